"""The oracle's pins must catch plausible mistakes in the oracle itself.

Each case plants one mistake in a copy of oracle/grand_oracle.c (a
temporary directory; the repository's oracle is never touched), builds the
copy with the oracle's own compiler flags, and runs the oracle's CPU tests
against it: at least one must fail.  The mistakes are the ones a port of the
paper's steps could plausibly make (a swapped record direction, a reversed
order, an off-by-one boundary, a skipped filter)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = {
    # Alg. 6: the out-neighbour repair record is (y, w), y receiving w
    "out_repair_direction": (
        "{ rec[r].t = tmp[j].id; rec[r].s = w; rec[r].d = tmp[j].d; }",
        "{ rec[r].t = w; rec[r].s = tmp[j].id; rec[r].d = tmp[j].d; }"),
    # scratch cap: the P smallest (dist, src) records are kept
    "cap_keeps_farthest": (
        "    if (a->d != b->d) return a->d < b->d ? -1 : 1;\n    if (a->s != b->s) return a->s < b->s ? -1 : 1;\n"
        "    return 0;\n}\n\ntypedef struct {\n    uint32_t n_dirty;",
        "    if (a->d != b->d) return a->d < b->d ? 1 : -1;\n    if (a->s != b->s) return a->s < b->s ? -1 : 1;\n"
        "    return 0;\n}\n\ntypedef struct {\n    uint32_t n_dirty;"),
    # C_i: the first k_repair entries outside the batch, not the first
    # k_repair entries filtered afterwards
    "ci_cut_before_filter": (
        "for (uint32_t j = 0; j < s.nC && k < kr; j++)\n            if (!in_batch[s.C[j].id])",
        "for (uint32_t j = 0; j < s.nC && j < kr; j++)\n            if (!in_batch[s.C[j].id])"),
    # Alg. 6: an in-neighbour gets the c closest points of C_i
    "in_repair_farthest": (
        "                rec[r].s = j < m ? tmp[j].id : O_INVALID;\n                rec[r].d = j < m ? tmp[j].d : 0.0f;",
        "                rec[r].s = j < m ? tmp[m - 1 - j].id : O_INVALID;\n"
        "                rec[r].d = j < m ? tmp[m - 1 - j].d : 0.0f;"),
    # an in-neighbour is not its own replacement
    "in_repair_keeps_self": ("                if (ci[j] == z) continue;", ""),
    # bootstrap: the `want` nearest other batch points
    "bootstrap_half": (
        "        uint32_t k = m < want ? m : want;\n        memcpy(out",
        "        uint32_t k = (m < want ? m : want) / 2;\n        memcpy(out"),
    "bootstrap_self": ("            if (j == i) continue;\n            all[m].id", "            all[m].id"),
    # Alg. 4 prunes on alpha * dist <= D_p (equality included)
    "prune_strict": (
        "if (coef * (double)dij <= (double)cand[j].d) valid[j] = 0;",
        "if (coef * (double)dij < (double)cand[j].d) valid[j] = 0;"),
    # Alg. 1 keeps the l closest keys
    "beam_keeps_one_more": (
        "        if (nC > ell) nC = ell;",
        "        if (nC > ell + 1) nC = ell + 1;"),
    "search_reevaluates": ("            if (present) continue;\n            okey k", "            okey k"),
    # medoid ties keep the smaller id
    "medoid_tie_larger": (
        "        if (arg == O_INVALID || key < best) { best = key; arg = i; }",
        "        if (arg == O_INVALID || key <= best) { best = key; arg = i; }"),
    "medoid_not_reinstalled": (
        "    if (m0 != O_INVALID && in_batch[m0]) h->medoid = compute_medoid(h);\n}", "}"),
    "deleted_rows_kept": (
        "        for (uint32_t t = 0; t < h->cfg.R; t++) h->adj[(size_t)ids[i] * h->cfg.R + t] = O_INVALID;\n"
        "        h->deg[ids[i]] = 0;\n        h->active[ids[i]] = 0;\n    }\n    h->n_active -= n;",
        "        h->deg[ids[i]] = 0;\n        h->active[ids[i]] = 0;\n    }\n    h->n_active -= n;"),
    # Alg. 7: the shared neighbour at the highest slot is replaced
    "detour_lowest_slot": (
        "            for (int t = (int)R - 1; t >= 0; t--) {\n                int in = 0;",
        "            for (int t = 0; t < (int)R; t++) {\n                int in = 0;"),
    "empty_slot_ignored": (
        "            if (free_slot >= 0) { row[free_slot] = p; continue; }",
        "            if (free_slot >= 0 && 0) { row[free_slot] = p; continue; }"),
    # Alg. 8: PickOne starts at u's rank and skips batch points
    "pickone_start_zero": ("uint32_t r = L[(rank + j) % nl];", "uint32_t r = L[(0 + j) % nl];"),
    "pickone_takes_batch": (
        "                if (in_batch[r] || r == u) continue;", "                if (r == u) continue;"),
    # Section 5.4: the augmented coordinate is sqrt(M^2 - |x|^2)
    "mips_plus": ("    double t = M2 - s;", "    double t = M2 + s;"),
    # CAGRA construction: a route u -> z -> y counts when z is ranked before
    # y in L(u) and y's position in L(z) is below y's rank in L(u)
    "rank_route_condition": (
        "if (ry != O_INVALID && rz < ry && rzy < ry) routes[ry]++;",
        "if (ry != O_INVALID && rz < ry) routes[ry]++;"),
    # the merged list starts with the first R/2 pruned entries
    "merge_quarter": ("    const uint32_t half = R / 2;", "    const uint32_t half = R / 4;"),
    "merge_reverse_repeats": (
        "            if (!in_list(o, no, rv[k].s)) o[no++] = rv[k].s;", "            o[no++] = rv[k].s;"),
}


def _run_oracle_tests(tmp_path, mutation):
    """Copies the oracle, its tests and the workload generator, applies
    `mutation` (None: none) and returns the oracle tests' exit status."""
    dst = tmp_path / "repo"
    os.makedirs(dst)
    for d in ("oracle", "tests", "workloads"):
        shutil.copytree(os.path.join(ROOT, d), dst / d,
                        ignore=shutil.ignore_patterns("__pycache__", "*.so", "test_oracle_mutations.py"))
    src = dst / "oracle" / "grand_oracle.c"
    if mutation is not None:
        old, new = mutation
        text = src.read_text()
        assert text.count(old) == 1, "the mutated text is not unique in the oracle"
        src.write_text(text.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-w", "-ffp-contract=off", "-fopenmp", "-shared", "-fPIC",
                           "-o", str(dst / "oracle" / "libgrand_oracle.so"), str(src), "-lm"])
    tests = sorted(str(p.relative_to(dst)) for p in (dst / "tests").glob("test_oracle_*.py"))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *tests],
                       cwd=dst, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-2000:]


def test_unmutated_copy_passes(tmp_path):
    """The harness itself: the copied, unchanged oracle passes its tests."""
    rc, out = _run_oracle_tests(tmp_path, None)
    assert rc == 0, out


@pytest.mark.parametrize("name", list(MUTATIONS))
def test_oracle_pins_catch_mutation(name, tmp_path):
    rc, out = _run_oracle_tests(tmp_path, MUTATIONS[name])
    assert rc != 0, f"{name}: every oracle test passed with the planted mistake"
