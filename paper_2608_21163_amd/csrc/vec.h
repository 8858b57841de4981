// vec.h -- distance evaluation by a wavefront against gathered pool rows.
//
// Distance (the single Dist used everywhere in the method):
//   L2 : squared Euclidean distance;  IP : negated inner product.
// uint8 rows are summed exactly in 32-bit integers; fp32 rows are summed in
// fp64 (each difference and product is exact in fp64) and rounded once to
// fp32.  A zero result is returned as +0.
//
// Layout: every pool row is padded with zeros to a multiple of 16 bytes
// ("chunks").  A row is handled by LPV consecutive lanes ("a group"); lane
// `sub` of a group owns chunks sub, sub+LPV, ... (at most CPL of them).  The
// query (or the pivot of a prune) is held by every group in registers in the
// same chunk layout, so 64/LPV rows are evaluated per step and a step's
// partial sums are reduced with log2(LPV) shuffles.
#pragma once
#include "wave.h"

namespace gr {

enum { kF32L2 = 0, kF32IP = 1, kU8L2 = 2 };

__device__ __forceinline__ uint4 ld16(const uint8_t* p) { return *reinterpret_cast<const uint4*>(p); }
__device__ __forceinline__ uint32_t udot4(uint32_t a, uint32_t b, uint32_t c) {
  return __builtin_amdgcn_udot4(a, b, c, false);
}
__device__ __forceinline__ float canon0(float x) { return x == 0.0f ? 0.0f : x; }

// int8 matrix-core operands: uint8 rows are used as x ^ 0x80 = x - 128
// (signed), which leaves squared Euclidean distances unchanged, so
// Dist(i, j) = |y_i|^2 + |y_j|^2 - 2 y_i.y_j holds exactly in int32.
typedef int v4i __attribute__((ext_vector_type(4)));
__device__ __forceinline__ int sdot4(uint32_t a, uint32_t b, int c) {
  return __builtin_amdgcn_sdot4((int)a, (int)b, c, false);
}
__device__ __forceinline__ v4i to_i8x16(uint4 v) {
  v4i r;
  r[0] = (int)(v.x ^ 0x80808080u);
  r[1] = (int)(v.y ^ 0x80808080u);
  r[2] = (int)(v.z ^ 0x80808080u);
  r[3] = (int)(v.w ^ 0x80808080u);
  return r;
}
__device__ __forceinline__ int sq_i8x16(v4i a, int acc) {
#pragma unroll
  for (int w = 0; w < 4; w++) acc = sdot4((uint32_t)a[w], (uint32_t)a[w], acc);
  return acc;
}
__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

template <int KIND> struct Acc;
template <> struct Acc<kU8L2> { typedef uint32_t T; };
template <> struct Acc<kF32L2> { typedef double T; };
template <> struct Acc<kF32IP> { typedef double T; };

template <int KIND, int LPV, int CPL>
struct Slice {
  uint4 q[CPL];
  uint32_t qn;  // uint8 L2: this lane's part of |q|^2
};

template <int KIND, int LPV, int CPL>
__device__ __forceinline__ void load_slice(Slice<KIND, LPV, CPL>& s, const uint8_t* row, int nch) {
  const int sub = lane() % LPV;
  s.qn = 0;
#pragma unroll
  for (int k = 0; k < CPL; k++) {
    const int c = sub + k * LPV;
    s.q[k] = c < nch ? ld16(row + (size_t)c * 16) : make_uint4(0, 0, 0, 0);
    if (KIND == kU8L2) {
      s.qn = udot4(s.q[k].x, s.q[k].x, s.qn);
      s.qn = udot4(s.q[k].y, s.q[k].y, s.qn);
      s.qn = udot4(s.q[k].z, s.q[k].z, s.qn);
      s.qn = udot4(s.q[k].w, s.q[k].w, s.qn);
    }
  }
}

__device__ __forceinline__ double l2_4(uint4 a, uint4 b, double acc) {
  const float* fa = reinterpret_cast<const float*>(&a);
  const float* fb = reinterpret_cast<const float*>(&b);
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const double t = (double)fb[i] - (double)fa[i];
    acc = __builtin_fma(t, t, acc);
  }
  return acc;
}
__device__ __forceinline__ double ip_4(uint4 a, uint4 b, double acc) {
  const float* fa = reinterpret_cast<const float*>(&a);
  const float* fb = reinterpret_cast<const float*>(&b);
#pragma unroll
  for (int i = 0; i < 4; i++) acc = __builtin_fma((double)fa[i], (double)fb[i], acc);
  return acc;
}
__device__ __forceinline__ uint32_t u8l2_4(uint4 a, uint4 b, uint32_t acc) {
  // |b|^2 - 2 a.b over 16 bytes; with the query's |a|^2 added once this is
  // the exact sum of squared differences (modulo 2^32, exact in range)
  acc = udot4(b.x, b.x, acc);
  acc = udot4(b.y, b.y, acc);
  acc = udot4(b.z, b.z, acc);
  acc = udot4(b.w, b.w, acc);
  uint32_t ab = udot4(a.x, b.x, 0u);
  ab = udot4(a.y, b.y, ab);
  ab = udot4(a.z, b.z, ab);
  ab = udot4(a.w, b.w, ab);
  return acc - 2u * ab;
}

template <int KIND, int LPV, int CPL>
__device__ __forceinline__ typename Acc<KIND>::T partial(const Slice<KIND, LPV, CPL>& s, const uint4 (&b)[CPL]) {
  typename Acc<KIND>::T acc;
  if (KIND == kU8L2) acc = s.qn; else acc = 0;
#pragma unroll
  for (int k = 0; k < CPL; k++) {
    if (KIND == kU8L2) acc = u8l2_4(s.q[k], b[k], acc);
    else if (KIND == kF32L2) acc = l2_4(s.q[k], b[k], acc);
    else acc = ip_4(s.q[k], b[k], acc);
  }
  return acc;
}

template <int LPV>
__device__ __forceinline__ uint32_t group_sum(uint32_t v) {
#pragma unroll
  for (int o = 1; o < LPV; o <<= 1) v += xshfl(v, o);
  return v;
}
template <int LPV>
__device__ __forceinline__ double group_sum(double v) {
#pragma unroll
  for (int o = 1; o < LPV; o <<= 1) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = xshfl((uint32_t)b, o), hi = xshfl((uint32_t)(b >> 32), o);
    v += __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
  }
  return v;
}

template <int KIND>
__device__ __forceinline__ float finalize(typename Acc<KIND>::T t) {
  if (KIND == kU8L2) return canon0((float)t);
  if (KIND == kF32L2) return canon0((float)t);
  return canon0((float)(-t));
}

// Distances from the slice to rows ids[0..cnt) (ids in LDS), written to
// out[0..cnt) (LDS).  All gathers of RIF steps are issued before any is
// consumed so that many rows are in flight per wave.
template <int KIND, int LPV, int CPL>
__device__ __forceinline__ void wave_dists(const Slice<KIND, LPV, CPL>& s, const uint8_t* __restrict__ vecs,
                                           size_t stride, int nch, const uint32_t* ids, float* out, int cnt) {
  constexpr int G = 64 / LPV;
  constexpr int RIF = CPL >= 8 ? 1 : 8 / CPL;
  const int ln = lane(), grp = ln / LPV, sub = ln % LPV;
  for (int base = 0; base < cnt; base += G * RIF) {
    // steps whose rows all lie beyond cnt are skipped (uniform branches)
    const int steps = (cnt - base + G - 1) / G;
    uint4 b[RIF][CPL];
#pragma unroll
    for (int rr = 0; rr < RIF; rr++) {
      if (rr >= steps) break;
      const int c = base + rr * G + grp;
      const uint8_t* row = vecs + (size_t)(c < cnt ? ids[c] : 0u) * stride;
#pragma unroll
      for (int k = 0; k < CPL; k++) {
        const int ch = sub + k * LPV;
        b[rr][k] = (rr < steps && c < cnt && ch < nch) ? ld16(row + (size_t)ch * 16) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int rr = 0; rr < RIF; rr++) {
      if (rr >= steps) break;
      const int c = base + rr * G + grp;
      typename Acc<KIND>::T t = group_sum<LPV>(partial<KIND, LPV, CPL>(s, b[rr]));
      if (sub == 0 && c < cnt) out[c] = finalize<KIND>(t);
    }
  }
}

// Distance from the slice to a single row, returned in every lane.
template <int KIND, int LPV, int CPL>
__device__ __forceinline__ float wave_dist1(const Slice<KIND, LPV, CPL>& s, const uint8_t* row, int nch) {
  const int sub = lane() % LPV;
  uint4 b[CPL];
#pragma unroll
  for (int k = 0; k < CPL; k++) {
    const int ch = sub + k * LPV;
    b[k] = ch < nch ? ld16(row + (size_t)ch * 16) : make_uint4(0, 0, 0, 0);
  }
  typename Acc<KIND>::T t = group_sum<LPV>(partial<KIND, LPV, CPL>(s, b));
  return __shfl(finalize<KIND>(t), 0, 64);
}

}  // namespace gr
