// dispatch.h -- compile-time instantiation of the vector kernels.
//
// (kind, vector class) selects the element type / metric and the lane
// layout of row gathers:
//   class A: rows of <= 8 chunks of 16 B   -> 8 lanes per row, 1 chunk per lane
//   class B: rows of <= 32 chunks          -> 8 lanes per row, <= 4 chunks per lane
//   class C: rows of <= 256 chunks         -> 16 lanes per row, <= 16 chunks per lane
#pragma once
#include "index.h"
#include "vec.h"

#define GR_DISPATCH_KV(kind, vc, ...)                                                       \
  do {                                                                                      \
    const int k__ = (kind), v__ = (vc);                                                     \
    if (k__ == ::gr::kU8L2 && v__ == ::gr::kVcA) {                                          \
      constexpr int KIND = ::gr::kU8L2, LPV = 8, CPL = 1; __VA_ARGS__;                      \
    } else if (k__ == ::gr::kU8L2 && v__ == ::gr::kVcB) {                                   \
      constexpr int KIND = ::gr::kU8L2, LPV = 8, CPL = 4; __VA_ARGS__;                      \
    } else if (k__ == ::gr::kU8L2 && v__ == ::gr::kVcC) {                                   \
      constexpr int KIND = ::gr::kU8L2, LPV = 16, CPL = 16; __VA_ARGS__;                    \
    } else if (k__ == ::gr::kF32L2 && v__ == ::gr::kVcA) {                                  \
      constexpr int KIND = ::gr::kF32L2, LPV = 8, CPL = 1; __VA_ARGS__;                     \
    } else if (k__ == ::gr::kF32L2 && v__ == ::gr::kVcB) {                                  \
      constexpr int KIND = ::gr::kF32L2, LPV = 8, CPL = 4; __VA_ARGS__;                     \
    } else if (k__ == ::gr::kF32L2 && v__ == ::gr::kVcC) {                                  \
      constexpr int KIND = ::gr::kF32L2, LPV = 16, CPL = 16; __VA_ARGS__;                   \
    } else if (k__ == ::gr::kF32IP && v__ == ::gr::kVcA) {                                  \
      constexpr int KIND = ::gr::kF32IP, LPV = 8, CPL = 1; __VA_ARGS__;                     \
    } else if (k__ == ::gr::kF32IP && v__ == ::gr::kVcB) {                                  \
      constexpr int KIND = ::gr::kF32IP, LPV = 8, CPL = 4; __VA_ARGS__;                     \
    } else if (k__ == ::gr::kF32IP && v__ == ::gr::kVcC) {                                  \
      constexpr int KIND = ::gr::kF32IP, LPV = 16, CPL = 16; __VA_ARGS__;                   \
    } else {                                                                                \
      return hipErrorInvalidValue;                                                          \
    }                                                                                       \
  } while (0)

// Register rows (64 keys each) needed to hold `n` keys: 1, 2 or 4.
#define GR_DISPATCH_N(n, ...)                                                               \
  do {                                                                                      \
    const uint32_t n__ = (n);                                                               \
    if (n__ <= 64) {                                                                        \
      constexpr int NR = 1; __VA_ARGS__;                                                    \
    } else if (n__ <= 128) {                                                                \
      constexpr int NR = 2; __VA_ARGS__;                                                    \
    } else if (n__ <= 256) {                                                                \
      constexpr int NR = 4; __VA_ARGS__;                                                    \
    } else {                                                                                \
      return hipErrorInvalidValue;                                                          \
    }                                                                                       \
  } while (0)
