// wave.h -- wavefront-level building blocks for gfx950 (wave64).
//
// Everything here is executed by one 64-lane wavefront cooperating through
// cross-lane shuffles, ballots and a little LDS; nothing synchronises across
// waves.  Keys are (distance, id) pairs ordered lexicographically; the top
// bit of an id is used as a per-entry "expanded" flag by the search, so key
// comparisons mask it.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gr {

constexpr uint32_t kInvalid = 0xFFFFFFFFu;
constexpr uint32_t kVisit = 0x80000000u;
constexpr uint32_t kIdMask = 0x7FFFFFFFu;

__device__ __forceinline__ float finf() { return __builtin_inff(); }
__device__ __forceinline__ int lane() { return (int)__lane_id(); }

// Key order and equality, written with non-short-circuit operators so that
// compare-exchange steps compile to compares and selects, not branches.
__device__ __forceinline__ bool kless(float a, uint32_t ia, float b, uint32_t ib) {
  return (a < b) | ((a == b) & ((ia & kIdMask) < (ib & kIdMask)));
}
__device__ __forceinline__ bool kequal(float a, uint32_t ia, float b, uint32_t ib) {
  return (a == b) & ((ia & kIdMask) == (ib & kIdMask));
}
__device__ __forceinline__ bool kvalid(uint32_t id) { return (id & kIdMask) != kIdMask; }

__device__ __forceinline__ uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }
// number of set bits of m strictly below this lane
__device__ __forceinline__ int mbcnt(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ int ffs64(uint64_t m) { return __ffsll((unsigned long long)m) - 1; }
__device__ __forceinline__ int fls64(uint64_t m) { return 63 - __clzll((unsigned long long)m); }

template <class T> __device__ __forceinline__ T rdlane(T v, int l);
template <> __device__ __forceinline__ uint32_t rdlane(uint32_t v, int l) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}
template <> __device__ __forceinline__ float rdlane(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// The value of lane (this lane ^ j), j a power of two below 64.  Distances
// up to 8 use DPP moves (quad permutes, half-row mirror, row rotate), 16 a
// swizzle within 32 lanes, and 32 a permute through the LDS crossbar.  After
// unrolling, j is a constant and the switch folds away.
__device__ __forceinline__ uint32_t xshfl(uint32_t v, int j) {
  switch (j) {
    case 1: return __builtin_amdgcn_update_dpp(0u, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    case 2: return __builtin_amdgcn_update_dpp(0u, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    case 4: {
      const uint32_t t = __builtin_amdgcn_update_dpp(0u, v, 0x141, 0xF, 0xF, false);  // row_half_mirror
      return __builtin_amdgcn_update_dpp(0u, t, 0x1B, 0xF, 0xF, false);                 // quad_perm [3,2,1,0]
    }
    case 8: return __builtin_amdgcn_update_dpp(0u, v, 0x128, 0xF, 0xF, false);  // row_ror:8
    case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);       // xor 16 within 32 lanes
    default: return (uint32_t)__shfl_xor((int)v, j, 64);
  }
}
__device__ __forceinline__ float xshfl(float v, int j) { return __uint_as_float(xshfl(__float_as_uint(v), j)); }

// The value of lane (this lane - 1); lane 0 gets its own value.
__device__ __forceinline__ uint32_t shfl_up1(uint32_t v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x138, 0xF, 0xF, false);  // wave_shr:1
}
__device__ __forceinline__ float shfl_up1(float v) { return __uint_as_float(shfl_up1(__float_as_uint(v))); }

// Compare-exchange of this lane's element with the element j lanes away.
// keep_min: this lane ends with the smaller key of the pair.
__device__ __forceinline__ void cx_lane(float& d, uint32_t& id, int j, bool keep_min) {
  const float od = xshfl(d, j);
  const uint32_t oi = xshfl(id, j);
  const bool take = (keep_min & kless(od, oi, d, id)) | (!keep_min & kless(d, id, od, oi));
  d = take ? od : d;
  id = take ? oi : id;
}

// Compare-exchange of register rows a (lower index) and b (higher index).
__device__ __forceinline__ void cx_reg(float& da, uint32_t& ia, float& db, uint32_t& ib, bool up) {
  const bool sw = (up & kless(db, ib, da, ia)) | (!up & kless(da, ia, db, ib));
  const float td = da;
  const uint32_t ti = ia;
  da = sw ? db : da;
  ia = sw ? ib : ia;
  db = sw ? td : db;
  ib = sw ? ti : ib;
}

// Bitonic sort, ascending, of N*64 keys held as element e = r*64 + lane.
template <int N>
__device__ __forceinline__ void wave_sort(float (&d)[N], uint32_t (&id)[N]) {
  const int ln = lane();
#pragma unroll
  for (int k = 2; k <= 64 * N; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j >= 64) {
        const int jr = j >> 6;
#pragma unroll
        for (int r = 0; r < N; r++) {
          const int p = r ^ jr;
          if (p > r) cx_reg(d[r], id[r], d[p], id[p], ((r * 64 + ln) & k) == 0);
        }
      } else {
#pragma unroll
        for (int r = 0; r < N; r++) {
          const bool up = ((r * 64 + ln) & k) == 0;
          const bool lower = (ln & j) == 0;
          cx_lane(d[r], id[r], j, lower == up);
        }
      }
    }
  }
}

// The same sort carrying a payload word with every key.
__device__ __forceinline__ void cx_lane3(float& d, uint32_t& id, uint32_t& pay, int j, bool keep_min) {
  const float od = xshfl(d, j);
  const uint32_t oi = xshfl(id, j);
  const uint32_t op = xshfl(pay, j);
  const bool take = (keep_min & kless(od, oi, d, id)) | (!keep_min & kless(d, id, od, oi));
  d = take ? od : d;
  id = take ? oi : id;
  pay = take ? op : pay;
}
__device__ __forceinline__ void cx_reg3(float& da, uint32_t& ia, uint32_t& pa, float& db, uint32_t& ib, uint32_t& pb,
                                        bool up) {
  const bool sw = (up & kless(db, ib, da, ia)) | (!up & kless(da, ia, db, ib));
  const float td = da;
  const uint32_t ti = ia, tp = pa;
  da = sw ? db : da;
  ia = sw ? ib : ia;
  pa = sw ? pb : pa;
  db = sw ? td : db;
  ib = sw ? ti : ib;
  pb = sw ? tp : pb;
}
template <int N>
__device__ __forceinline__ void wave_sort_pay(float (&d)[N], uint32_t (&id)[N], uint32_t (&pay)[N]) {
  const int ln = lane();
#pragma unroll
  for (int k = 2; k <= 64 * N; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (j >= 64) {
        const int jr = j >> 6;
#pragma unroll
        for (int r = 0; r < N; r++) {
          const int p = r ^ jr;
          if (p > r) cx_reg3(d[r], id[r], pay[r], d[p], id[p], pay[p], ((r * 64 + ln) & k) == 0);
        }
      } else {
#pragma unroll
        for (int r = 0; r < N; r++) {
          const bool up = ((r * 64 + ln) & k) == 0;
          const bool lower = (ln & j) == 0;
          cx_lane3(d[r], id[r], pay[r], j, lower == up);
        }
      }
    }
  }
}

// Bitonic merge (input bitonic) to ascending order.
template <int N>
__device__ __forceinline__ void wave_merge_up(float (&d)[N], uint32_t (&id)[N]) {
  const int ln = lane();
#pragma unroll
  for (int j = 32 * N; j > 0; j >>= 1) {
    if (j >= 64) {
      const int jr = j >> 6;
#pragma unroll
      for (int r = 0; r < N; r++) {
        const int p = r ^ jr;
        if (p > r) cx_reg(d[r], id[r], d[p], id[p], true);
      }
    } else {
#pragma unroll
      for (int r = 0; r < N; r++) cx_lane(d[r], id[r], j, (ln & j) == 0);
    }
  }
}

// Marks (in dup[]) every element of an ascending list whose key equals the
// key of the element just before it; returns the ballot of all marks.
template <int N>
__device__ __forceinline__ uint64_t wave_find_repeats(const float (&d)[N], const uint32_t (&id)[N],
                                                      uint64_t (&dm)[N]) {
  const int ln = lane();
  uint64_t any = 0;
#pragma unroll
  for (int r = 0; r < N; r++) {
    float pd = shfl_up1(d[r]);
    uint32_t pi = shfl_up1(id[r]);
    if (r > 0) {
      float qd = rdlane(d[r - 1], 63);
      uint32_t qi = rdlane(id[r - 1], 63);
      if (ln == 0) { pd = qd; pi = qi; }
    }
    const bool has_prev = (r > 0) || (ln > 0);
    const bool dup = has_prev && kvalid(id[r]) && kequal(d[r], id[r], pd, pi);
    dm[r] = ballot(dup);
    any |= dm[r];
  }
  return any;
}

// Sorts 64 keys (one per lane) ascending and removes repeated keys.
__device__ __forceinline__ void wave_sort_unique1(float& nd, uint32_t& ni) {
  float t1[1] = {nd};
  uint32_t t2[1] = {ni};
  wave_sort<1>(t1, t2);
  uint64_t dm[1];
  if (wave_find_repeats<1>(t1, t2, dm)) {
    if ((dm[0] >> lane()) & 1) { t1[0] = finf(); t2[0] = kInvalid; }
    wave_sort<1>(t1, t2);
  }
  nd = t1[0];
  ni = t2[0];
}

// min(C[i], B[N*64-1-i]) for ascending C and ascending B (64 keys, padded
// with +inf) is bitonic and holds the N*64 smallest keys of C and B; a
// bitonic merge then sorts it.
template <int N>
__device__ __forceinline__ void wave_merge_sorted64(float (&cd)[N], uint32_t (&ci)[N], float bd, uint32_t bi) {
  const int ln = lane();
  float rd = __shfl(bd, 63 - ln, 64);
  uint32_t ri = __shfl(bi, 63 - ln, 64);
  if (kless(rd, ri, cd[N - 1], ci[N - 1])) { cd[N - 1] = rd; ci[N - 1] = ri; }
  wave_merge_up<N>(cd, ci);
}

// Merges up to 64 new keys (one per lane, any order, invalid = (+inf,
// kInvalid)) into the ascending, repeat-free list C of N*64 keys, keeping
// the smallest `keep` distinct keys.  A new key equal to a key already in C
// is dropped (the entry in C, with its expanded flag, stays).  Repeats are
// rare, so they are found after merging: every new key equal to a repeated
// key is removed and the merge is redone from the saved C.  Removing repeats
// can expose others that the first merge had cut off, so this repeats until
// a merge has no repeat (each round removes at least one new key).  A merge
// without repeats holds the N*64 smallest distinct keys.
template <int N>
__device__ __forceinline__ void wave_merge_new(float (&cd)[N], uint32_t (&ci)[N], float nd, uint32_t ni,
                                               int keep) {
  const int ln = lane();
  wave_sort_unique1(nd, ni);
  float sd[N];
  uint32_t si[N];
#pragma unroll
  for (int r = 0; r < N; r++) { sd[r] = cd[r]; si[r] = ci[r]; }
  for (int round = 0; round <= 64; round++) {
    wave_merge_sorted64<N>(cd, ci, nd, ni);
    uint64_t dm[N];
    if (!wave_find_repeats<N>(cd, ci, dm)) break;
#pragma unroll
    for (int r = 0; r < N; r++) {
      uint64_t m = dm[r];
      while (m) {
        const int l = ffs64(m);
        m &= m - 1;
        const float kd = rdlane(cd[r], l);
        const uint32_t ki = rdlane(ci[r], l);
        if (kequal(nd, ni, kd, ki)) { nd = finf(); ni = kInvalid; }
      }
    }
    float t1[1] = {nd};
    uint32_t t2[1] = {ni};
    wave_sort<1>(t1, t2);
    nd = t1[0];
    ni = t2[0];
#pragma unroll
    for (int r = 0; r < N; r++) { cd[r] = sd[r]; ci[r] = si[r]; }
  }
#pragma unroll
  for (int r = 0; r < N; r++)
    if (r * 64 + ln >= keep) { cd[r] = finf(); ci[r] = kInvalid; }
}

// Same result as wave_merge_new (C <- the `keep` smallest distinct keys of
// C u new), cheaper when few new keys can enter.  C holds at most `keep`
// valid keys, sorted.  New keys not below C's key at position keep-1 (+inf
// while C is not full) cannot enter and are dropped first; up to kFewMax
// survivors are then inserted one at a time (rank by ballot, shift up by one
// element), repeats of keys already in C are skipped, and keys pushed past
// `keep` are dropped.  More survivors take the sort-and-merge path.
constexpr int kFewMax = 16;
template <int N>
__device__ __forceinline__ void wave_merge_new_fast(float (&cd)[N], uint32_t (&ci)[N], float nd, uint32_t ni,
                                                    int keep) {
  const int ln = lane();
  const int wr = (keep - 1) >> 6, wl = (keep - 1) & 63;
  float wd = 0.0f;
  uint32_t wi = 0;
#pragma unroll
  for (int r = 0; r < N; r++)
    if (r == wr) {
      wd = rdlane(cd[r], wl);
      wi = rdlane(ci[r], wl);
    }
  const bool in = kvalid(ni) && kless(nd, ni, wd, wi);
  uint64_t m = ballot(in);
  if (!m) return;
  if (popc(m) > kFewMax) {
    wave_merge_new<N>(cd, ci, in ? nd : finf(), in ? ni : kInvalid, keep);
    return;
  }
  while (m) {
    const int l = ffs64(m);
    m &= m - 1;
    const float xd = rdlane(nd, l);
    const uint32_t xi = rdlane(ni, l);
    int pos = 0;
    bool dup = false;
#pragma unroll
    for (int r = 0; r < N; r++) {
      pos += popc(ballot(kless(cd[r], ci[r], xd, xi)));
      dup |= ballot(kequal(cd[r], ci[r], xd, xi)) != 0;
    }
    if (dup || pos >= keep) continue;
    float pd = 0.0f;
    uint32_t pi = 0;
#pragma unroll
    for (int r = 0; r < N; r++) {
      const float top_d = rdlane(cd[r], 63);
      const uint32_t top_i = rdlane(ci[r], 63);
      float ud = shfl_up1(cd[r]);
      uint32_t ui = shfl_up1(ci[r]);
      ud = ln == 0 ? pd : ud;
      ui = ln == 0 ? pi : ui;
      const int e = r * 64 + ln;
      const bool at = e == pos, above = e > pos;
      cd[r] = at ? xd : (above ? ud : cd[r]);
      ci[r] = at ? xi : (above ? ui : ci[r]);
      pd = top_d;
      pi = top_i;
    }
  }
#pragma unroll
  for (int r = 0; r < N; r++)
    if (r * 64 + ln >= keep) { cd[r] = finf(); ci[r] = kInvalid; }
}

// 64-bit keys whose unsigned order is the (distance, id) order: the float's
// bits mapped to an order-preserving unsigned integer (negative values
// complemented, non-negative ones with the sign bit set) above the id with
// its expanded flag masked off.
__device__ __forceinline__ uint32_t sortable(float d) {
  const uint32_t b = __float_as_uint(d);
  return b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
}
__device__ __forceinline__ uint64_t key64(float d, uint32_t id) {
  return ((uint64_t)sortable(d) << 32) | (uint64_t)(id & kIdMask);
}
__device__ __forceinline__ uint64_t rdlane64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Same result as wave_merge_new_fast, with every survivor placed in one
// pass: survivors (new keys below C's key at position keep-1) that repeat a
// key of C are dropped; for the others, each C key counts the survivors
// below it and each survivor the C keys and other survivors below it, which
// gives every key its position in the merged order; keys at positions below
// `keep` are written to the LDS scratch (ld, li: 64*N entries each) and read
// back in order.  More than kBatchMax survivors take the sort-and-merge path.
constexpr int kBatchMax = 32;
template <int N>
__device__ __forceinline__ void wave_merge_lds(float (&cd)[N], uint32_t (&ci)[N], float nd, uint32_t ni, int keep,
                                               float *ld, uint32_t *li) {
  const int ln = lane();
  const int wr = (keep - 1) >> 6, wl = (keep - 1) & 63;
  uint64_t ck[N];
#pragma unroll
  for (int r = 0; r < N; r++) ck[r] = key64(cd[r], ci[r]);
  uint64_t wk = 0;
#pragma unroll
  for (int r = 0; r < N; r++)
    if (r == wr) wk = rdlane64(ck[r], wl);
  const uint64_t nk = key64(nd, ni);
  const bool in = kvalid(ni) && nk < wk;
  const uint64_t m = ballot(in);
  if (!m) return;
  if (popc(m) > kBatchMax) {
    wave_merge_new<N>(cd, ci, in ? nd : finf(), in ? ni : kInvalid, keep);
    return;
  }
  uint32_t cnt[N];
#pragma unroll
  for (int r = 0; r < N; r++) cnt[r] = 0;
  uint32_t ltc = 0, rk = 0;
  uint64_t live = 0, mm = m;
  while (mm) {
    const int l = ffs64(mm);
    mm &= mm - 1;
    const uint64_t xk = rdlane64(nk, l);
    bool lt[N];
    int below = 0;
    bool dup = false;
#pragma unroll
    for (int r = 0; r < N; r++) {
      lt[r] = ck[r] < xk;
      below += popc(ballot(lt[r]));
      dup |= ballot(ck[r] == xk) != 0;
    }
    if (dup) continue;
    live |= 1ull << l;
#pragma unroll
    for (int r = 0; r < N; r++) cnt[r] += lt[r] ? 0u : 1u;
    rk += xk < nk ? 1u : 0u;
    ltc = ln == l ? (uint32_t)below : ltc;
  }
#pragma unroll
  for (int r = 0; r < N; r++) {
    const int p = r * 64 + ln + (int)cnt[r];
    if (p < keep) { ld[p] = cd[r]; li[p] = ci[r]; }
  }
  if ((live >> ln) & 1) {
    const int p = (int)(ltc + rk);
    if (p < keep) { ld[p] = nd; li[p] = ni; }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < N; r++) {
    const int e = r * 64 + ln;
    const bool ok = e < keep;
    cd[r] = ok ? ld[e] : finf();
    ci[r] = ok ? li[e] : kInvalid;
  }
  __syncthreads();
}

// The float whose sortable() image is u.
__device__ __forceinline__ float unsortable(uint32_t u) {
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}
__device__ __forceinline__ uint64_t xshfl64(uint64_t v, int j) {
  return ((uint64_t)xshfl((uint32_t)(v >> 32), j) << 32) | (uint64_t)xshfl((uint32_t)v, j);
}

// Bitonic sort, ascending, of N*64 64-bit keys held as element e = r*64 + lane
// (one compare per exchange instead of the (distance, id) pair test).
template <int N>
__device__ __forceinline__ void wave_sort64(uint64_t (&k)[N]) {
  const int ln = lane();
#pragma unroll
  for (int kk = 2; kk <= 64 * N; kk <<= 1) {
#pragma unroll
    for (int j = kk >> 1; j > 0; j >>= 1) {
      if (j >= 64) {
        const int jr = j >> 6;
#pragma unroll
        for (int r = 0; r < N; r++) {
          const int p = r ^ jr;
          if (p > r) {
            const bool up = ((r * 64 + ln) & kk) == 0;
            const uint64_t a = k[r], b = k[p];
            const bool sw = (b < a) == up;
            k[r] = sw ? b : a;
            k[p] = sw ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < N; r++) {
          const bool up = ((r * 64 + ln) & kk) == 0;
          const bool keep_min = ((ln & j) == 0) == up;
          const uint64_t o = xshfl64(k[r], j);
          // equal keys may swap either way: the values are the same
          k[r] = ((o < k[r]) == keep_min) ? o : k[r];
        }
      }
    }
  }
}

// Bitonic sort, ascending, of N*64 32-bit keys held as element e = r*64 + lane.
template <int N>
__device__ __forceinline__ void wave_sort32(uint32_t (&k)[N]) {
  const int ln = lane();
#pragma unroll
  for (int kk = 2; kk <= 64 * N; kk <<= 1) {
#pragma unroll
    for (int j = kk >> 1; j > 0; j >>= 1) {
      if (j >= 64) {
        const int jr = j >> 6;
#pragma unroll
        for (int r = 0; r < N; r++) {
          const int p = r ^ jr;
          if (p > r) {
            const bool up = ((r * 64 + ln) & kk) == 0;
            const uint32_t a = k[r], b = k[p];
            const bool sw = (b < a) == up;
            k[r] = sw ? b : a;
            k[p] = sw ? a : b;
          }
        }
      } else {
#pragma unroll
        for (int r = 0; r < N; r++) {
          const bool up = ((r * 64 + ln) & kk) == 0;
          const bool keep_min = ((ln & j) == 0) == up;
          const uint32_t o = xshfl(k[r], j);
          k[r] = keep_min ? min(o, k[r]) : max(o, k[r]);
        }
      }
    }
  }
}

// Exclusive wave prefix sum of small non-negative ints.
__device__ __forceinline__ int wave_excl_scan(int v, int& total) {
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane() >= o) x += y;
  }
  total = __shfl(x, 63, 64);
  return x - v;
}

}  // namespace gr
