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

namespace gr {
// Workgroups of 64 lanes of `kern` (no dynamic LDS) that are resident on
// the current device at once, or 0 if the runtime cannot say.  A persistent
// loop over a queue split over exactly this many workgroups leaves no
// workgroup to start after the first ones finish.
static inline uint32_t resident_blocks(const void *kern) {
  int dev = 0, ncu = 0, per = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kern, 64, 0) != hipSuccess) return 0;
  return per > 0 && ncu > 0 ? (uint32_t)per * (uint32_t)ncu : 0u;
}
static inline uint32_t clamp_resident(uint32_t grid, uint32_t res) { return res && res < grid ? res : grid; }
}  // namespace gr
