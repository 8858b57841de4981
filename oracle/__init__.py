"""Test infrastructure only: the plain CPU oracle of the paper's method."""
