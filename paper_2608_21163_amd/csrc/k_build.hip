// k_build.hip -- CAGRA graph construction (Section 2.2 on CAGRA; Section
// 4.2, CAGRA graph construction): an approximate k-NN graph by NN-Descent,
// rank-based edge pruning to the fixed degree, then reverse edges merged in.
//
// Positions 0..n-1 stand for the points being built (pool row ids[p]).
// Every kernel runs one wavefront per node and reads only state that the
// previous kernel finished, so the result does not depend on scheduling:
//
// NN-Descent round (batch-synchronous): sample the first S new and the first
// S old entries of every list (sampled new entries turn old) and record each
// sample at its target; group the records by target; per node v gather
// Bn = its new samples and the S smallest (Dist, u) new reverse samples,
// Bo = the same for old minus Bn; the pairs within Bn and between Bn and Bo
// give proposals (b to a when (Dist, b) is below a's last key at the start
// of the round, and the other way); proposals are counted, then written in
// chunks that fit the record buffers, grouped by target and merged into a
// copy of the lists (the K smallest distinct keys; an existing key keeps its
// entry and flag).
//
// Rank-based pruning: per node u, for every neighbour y of rank r, count the
// z of rank rz < r whose list holds y at a rank below r (detourable routes);
// keep the R entries with the fewest routes, by (routes, rank).
// Reverse edges: every pruned edge u -> y at position t is recorded at y
// with key (t, u); y's output is the first R/2 of its pruned list, then its
// reverse neighbours in key order, then the rest of its pruned list,
// skipping ids already taken, up to R.
//
// Distances are evaluated one pair per lane along the dimensions in order,
// exactly (uint8) or with fp64 accumulation rounded once (fp32), the same
// value the searches and prunes produce for the pair.
#include "dispatch.h"

namespace gr {

constexpr uint32_t kNew = 0x80000000u;  // list entry not yet sampled; reverse records: an old sample

// Dist of two rows of nch 16-byte chunks, one lane, dimensions in order
// (zero padding adds nothing).
template <int KIND>
__device__ __forceinline__ float dist_seq(const uint8_t *a, const uint8_t *b, int nch) {
  if (KIND == kU8L2) {
    uint32_t s = 0;
    for (int c = 0; c < nch; c++) {
      const uint4 x = ld16(a + 16 * c), y = ld16(b + 16 * c);
      const uint32_t xw[4] = {x.x, x.y, x.z, x.w}, yw[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int w = 0; w < 4; w++)
#pragma unroll
        for (int k = 0; k < 4; k++) {
          const int t = (int)((xw[w] >> (8 * k)) & 0xFFu) - (int)((yw[w] >> (8 * k)) & 0xFFu);
          s += (uint32_t)(t * t);
        }
    }
    return canon0((float)s);
  } else {
    double s = 0.0;
    for (int c = 0; c < nch; c++) {
      const float4 x = *reinterpret_cast<const float4 *>(a + 16 * c);
      const float4 y = *reinterpret_cast<const float4 *>(b + 16 * c);
      const float xf[4] = {x.x, x.y, x.z, x.w}, yf[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
      for (int k = 0; k < 4; k++) {
        if (KIND == kF32L2) {
          const double t = (double)xf[k] - (double)yf[k];
          s = __builtin_fma(t, t, s);
        } else {
          s = __builtin_fma((double)xf[k], (double)yf[k], s);
        }
      }
    }
    return canon0(KIND == kF32IP ? (float)(-s) : (float)s);
  }
}

__device__ __forceinline__ const uint8_t *row_of(const BuildArgs &a, uint32_t pos) {
  return a.pool.vecs + (size_t)a.ids[pos] * a.pool.stride;
}

static __device__ void build_error(DevScalars *ds, uint32_t id) {
  if (atomicCAS(&ds->err_code, 0u, (uint32_t)kErrInit) == 0u) ds->err_id = id;
}

// Initial lists: K distinct positions other than u, each below n.
__global__ __launch_bounds__(64) void k_nnd_check(BuildArgs a) {
  const uint32_t u = blockIdx.x;
  if (u >= a.n) return;
  const int ln = lane();
  float d[2];
  uint32_t v[2];
  bool bad = false;
#pragma unroll
  for (int r = 0; r < 2; r++) {
    const uint32_t j = r * 64 + ln;
    const uint32_t x = j < a.K ? a.init[(size_t)u * a.K + j] : kInvalid;
    bad |= j < a.K && (x >= a.n || x == u);
    d[r] = j < a.K ? 0.0f : finf();
    v[r] = j < a.K ? x : kInvalid;
  }
  wave_sort<2>(d, v);
  uint64_t dm[2];
  if (ballot(bad) || wave_find_repeats<2>(d, v, dm)) {
    if (ln == 0) build_error(a.ds, u);
  }
}

// Lists from the initial positions, ascending by (Dist, position), all new.
template <int KIND>
__global__ __launch_bounds__(64) void k_nnd_init(BuildArgs a) {
  const uint32_t u = blockIdx.x;
  if (u >= a.n) return;
  const int ln = lane();
  const uint8_t *ru = row_of(a, u);
  float d[2];
  uint32_t v[2];
#pragma unroll
  for (int r = 0; r < 2; r++) {
    const uint32_t j = r * 64 + ln;
    v[r] = j < a.K ? a.init[(size_t)u * a.K + j] : kInvalid;
    d[r] = j < a.K ? dist_seq<KIND>(ru, row_of(a, v[r]), a.pool.nch) : finf();
  }
  wave_sort<2>(d, v);
#pragma unroll
  for (int r = 0; r < 2; r++) {
    const uint32_t j = r * 64 + ln;
    if (j < a.K) {
      a.lid[(size_t)u * a.K + j] = v[r] | kNew;
      a.ld[(size_t)u * a.K + j] = d[r];
    }
  }
}

// Samples of node u: the first S new entries (which turn old) and the first
// S old ones, in list order; each sample is also recorded at its target
// (old samples with the source's top bit set).
__global__ __launch_bounds__(64) void k_nnd_sample(BuildArgs a) {
  const uint32_t u = blockIdx.x;
  if (u >= a.n) return;
  const int ln = lane();
  const uint32_t S = a.S;
  uint32_t before_new = 0, before_old = 0;
#pragma unroll
  for (int r = 0; r < 2; r++) {
    const uint32_t j = r * 64 + ln;
    const bool in = j < a.K;
    const uint32_t e = in ? a.lid[(size_t)u * a.K + j] : 0u;
    const float dd = in ? a.ld[(size_t)u * a.K + j] : 0.0f;
    const bool isnew = in && (e & kNew);
    const bool isold = in && !(e & kNew);
    const uint64_t mn = ballot(isnew), mo = ballot(isold);
    const uint32_t kn = before_new + (uint32_t)mbcnt(mn), ko = before_old + (uint32_t)mbcnt(mo);
    const uint32_t v = e & kIdMask;
    if (isnew && kn < S) {
      a.ns[(size_t)u * S + kn] = v;
      const size_t q = (size_t)u * 2 * S + kn;
      a.rec_t[q] = v;
      a.rec_s[q] = u;
      a.rec_d[q] = dd;
      a.lid[(size_t)u * a.K + j] = v;
    }
    if (isold && ko < S) {
      a.os[(size_t)u * S + ko] = v;
      const size_t q = (size_t)u * 2 * S + S + ko;
      a.rec_t[q] = v;
      a.rec_s[q] = u | kNew;
      a.rec_d[q] = dd;
    }
    before_new += (uint32_t)popc(mn);
    before_old += (uint32_t)popc(mo);
  }
  for (uint32_t k = ln; k < S; k += 64) {
    if (k >= before_new) {
      a.ns[(size_t)u * S + k] = kInvalid;
      a.rec_t[(size_t)u * 2 * S + k] = kInvalid;
    }
    if (k >= before_old) {
      a.os[(size_t)u * S + k] = kInvalid;
      a.rec_t[(size_t)u * 2 * S + S + k] = kInvalid;
    }
  }
}

// Bn and Bo of node v (Bn ascending, then Bo ascending) into cand[v][0..4S),
// their sizes into cnb[v] = nb | no << 16.
__global__ __launch_bounds__(64) void k_nnd_cands(BuildArgs a) {
  const uint32_t v = blockIdx.x;
  if (v >= a.n) return;
  __shared__ uint32_t bnL[64];
  const int ln = lane();
  const uint32_t S = a.S;
  // the S smallest (Dist, u) reverse samples of each kind
  float rnd[1] = {finf()}, rod[1] = {finf()};
  uint32_t rni[1] = {kInvalid}, roi[1] = {kInvalid};
  const uint32_t g0 = a.goff[v], g1 = a.goff[v + 1];
  for (uint32_t b = g0; b < g1; b += 64) {
    const bool in = b + ln < g1;
    const uint32_t s = in ? a.gsrc[b + ln] : kInvalid;
    const float dd = in ? a.gd[b + ln] : finf();
    const bool old = in && (s & kNew);
    wave_merge_new<1>(rnd, rni, in && !old ? dd : finf(), in && !old ? s : kInvalid, (int)S);
    wave_merge_new<1>(rod, roi, old ? dd : finf(), old ? (s & kIdMask) : kInvalid, (int)S);
  }
  // Bn: the new samples and the new reverse samples, ascending, distinct
  {
    uint32_t x = kInvalid;
    const uint32_t rv = (uint32_t)__shfl((int)rni[0], (ln - (int)S) & 63, 64);
    if (ln < (int)S) x = a.ns[(size_t)v * S + ln];
    else if (ln < 2 * (int)S) x = rv;
    float kd = kvalid(x) ? 0.0f : finf();
    wave_sort_unique1(kd, x);
    bnL[ln] = x;
  }
  __syncthreads();
  const uint32_t bn = bnL[ln];
  const int nb = popc(ballot(kvalid(bn)));
  // Bo: the old samples and old reverse samples not in Bn
  uint32_t y = kInvalid;
  const uint32_t ro = (uint32_t)__shfl((int)roi[0], (ln - (int)S) & 63, 64);
  if (ln < (int)S) y = a.os[(size_t)v * S + ln];
  else if (ln < 2 * (int)S) y = ro;
  {
    float kd = kvalid(y) ? 0.0f : finf();
    wave_sort_unique1(kd, y);
  }
  bool keep = kvalid(y);
  if (keep) {
    int lo = 0, hi = nb;  // binary search in the ascending Bn
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (bnL[mid] < y) lo = mid + 1;
      else hi = mid;
    }
    keep = !(lo < nb && bnL[lo] == y);
  }
  const uint64_t km = ballot(keep);
  const int no = popc(km);
  uint32_t *c = a.cand + (size_t)v * 4 * S;
  if (ln < nb) c[ln] = bn;
  if (keep) c[nb + mbcnt(km)] = y;
  if (ln == 0) a.cnb[v] = (uint32_t)nb | ((uint32_t)no << 16);
}

// The pairs of node v: (i, j) for i < nb and i < j < nb + no.  WRITE = false
// counts the proposals into pcnt[v]; WRITE = true writes them from
// poff[v] - poff[v0] on (nodes v0 .. v1).  Rows are staged in LDS when the
// dynamic LDS holds them.
template <int KIND, bool WRITE>
__global__ __launch_bounds__(64) void k_nnd_join(BuildArgs a) {
  extern __shared__ uint4 rowsL[];
  __shared__ uint32_t cL[128];
  __shared__ float wdL[128];
  __shared__ uint32_t wiL[128];
  const uint32_t v = a.v0 + blockIdx.x;
  if (v >= a.v1) return;
  const int ln = lane();
  const uint32_t S = a.S, K = a.K;
  const uint32_t cc = a.cnb[v];
  const int nb = (int)(cc & 0xFFFFu), no = (int)(cc >> 16), m = nb + no;
  const uint32_t *c = a.cand + (size_t)v * 4 * S;
  // candidates and their last keys at the start of the round
  for (int i = ln; i < m; i += 64) {
    const uint32_t x = c[i];
    cL[i] = x;
    wdL[i] = a.ld[(size_t)x * K + K - 1];
    wiL[i] = a.lid[(size_t)x * K + K - 1] & kIdMask;
  }
  const int nch = a.pool.nch;
  const bool staged = a.stage_rows != 0;
  __syncthreads();
  if (staged) {
    for (int k = ln; k < m * nch; k += 64) {
      const int i = k / nch, ch = k - i * nch;
      rowsL[k] = ld16(row_of(a, cL[i]) + 16 * ch);
    }
  }
  __syncthreads();
  uint32_t cnt = 0;
  size_t base = 0;
  if (WRITE) base = (size_t)(a.poff[v] - a.poff[a.v0]);
  for (int i = 0; i < nb; i++) {
    const uint32_t pa = cL[i];
    const uint8_t *ra = staged ? reinterpret_cast<const uint8_t *>(rowsL + (size_t)i * nch) : row_of(a, pa);
    const float wda = wdL[i];
    const uint32_t wia = wiL[i];
    for (int j0 = i + 1; j0 < m; j0 += 64) {
      const int j = j0 + ln;
      bool pab = false, pba = false;
      float d = 0.0f;
      uint32_t pb = kInvalid;
      if (j < m) {
        pb = cL[j];
        const uint8_t *rb = staged ? reinterpret_cast<const uint8_t *>(rowsL + (size_t)j * nch) : row_of(a, pb);
        d = dist_seq<KIND>(ra, rb, nch);
        pab = kless(d, pb, wda, wia);       // b proposed to a
        pba = kless(d, pa, wdL[j], wiL[j]); // a proposed to b
      }
      const uint64_t m1 = ballot(pab), m2 = ballot(pba);
      if (WRITE) {
        const size_t o1 = base + cnt + (uint32_t)mbcnt(m1);
        const size_t o2 = base + cnt + (uint32_t)popc(m1) + (uint32_t)mbcnt(m2);
        if (pab) {
          a.rec_t[o1] = pa;
          a.rec_s[o1] = pb;
          a.rec_d[o1] = d;
        }
        if (pba) {
          a.rec_t[o2] = pb;
          a.rec_s[o2] = pa;
          a.rec_d[o2] = d;
        }
      }
      cnt += (uint32_t)(popc(m1) + popc(m2));
    }
  }
  if (!WRITE && ln == 0) a.pcnt[v] = cnt;
}

// Node u's next list <- the K smallest distinct keys of it and its grouped
// proposals (new entries flagged); one wavefront per node with proposals.
__global__ __launch_bounds__(64) void k_nnd_merge(BuildArgs a) {
  const int ln = lane();
  const uint32_t K = a.K, nd_total = *a.n_dirty;
  for (uint32_t it = blockIdx.x; it < nd_total; it += gridDim.x) {
    const uint32_t u = a.dirty[it];
    float cd[2];
    uint32_t ci[2];
#pragma unroll
    for (int r = 0; r < 2; r++) {
      const uint32_t j = r * 64 + ln;
      cd[r] = j < K ? a.nd[(size_t)u * K + j] : finf();
      ci[r] = j < K ? a.nid[(size_t)u * K + j] : kInvalid;
    }
    const uint32_t g0 = a.goff[u], g1 = a.goff[u + 1];
    for (uint32_t b = g0; b < g1; b += 64) {
      const bool in = b + ln < g1;
      const float pd = in ? a.gd[b + ln] : finf();
      const uint32_t ps = in ? (a.gsrc[b + ln] | kNew) : kInvalid;
      wave_merge_new<2>(cd, ci, pd, ps, (int)K);
    }
#pragma unroll
    for (int r = 0; r < 2; r++) {
      const uint32_t j = r * 64 + ln;
      if (j < K) {
        a.nd[(size_t)u * K + j] = cd[r];
        a.nid[(size_t)u * K + j] = ci[r];
      }
    }
  }
}

// Rank-based pruning of node u's list to R entries, and the reverse records
// (P(u)[t], u, t).
constexpr int kRankSlots = 256;
__global__ __launch_bounds__(64) void k_cagra_rank(BuildArgs a) {
  const uint32_t u = blockIdx.x;
  if (u >= a.n) return;
  __shared__ uint32_t hid[kRankSlots];
  __shared__ uint32_t hrk[kRankSlots];
  __shared__ uint32_t routes[128];
  __shared__ uint32_t lu[128];
  const int ln = lane();
  const uint32_t K = a.K;
  for (int s = ln; s < kRankSlots; s += 64) hid[s] = kInvalid;
  for (int r = ln; r < 128; r += 64) routes[r] = 0;
  __syncthreads();
  for (uint32_t r = ln; r < K; r += 64) {
    const uint32_t y = a.lid[(size_t)u * K + r] & kIdMask;
    lu[r] = y;
    uint32_t s = (y * 2654435761u) >> 24;
    while (atomicCAS(&hid[s], kInvalid, y) != kInvalid) s = (s + 1) & (kRankSlots - 1);
    hrk[s] = r;
  }
  __syncthreads();
  auto rank_of = [&](uint32_t y) -> uint32_t {
    uint32_t s = (y * 2654435761u) >> 24;
    for (;;) {
      const uint32_t h = hid[s];
      if (h == y) return hrk[s];
      if (h == kInvalid) return kInvalid;
      s = (s + 1) & (kRankSlots - 1);
    }
  };
  for (uint32_t rz = 0; rz < K; rz++) {
    const uint32_t z = lu[rz];
#pragma unroll
    for (int r = 0; r < 2; r++) {
      const uint32_t rzy = r * 64 + ln;
      if (rzy < K) {
        const uint32_t y = a.lid[(size_t)z * K + rzy] & kIdMask;
        const uint32_t ry = rank_of(y);
        if (ry != kInvalid && rz < ry && rzy < ry) atomicAdd(&routes[ry], 1u);
      }
    }
  }
  __syncthreads();
  float kd[2];
  uint32_t ki[2];
#pragma unroll
  for (int r = 0; r < 2; r++) {
    const uint32_t j = r * 64 + ln;
    kd[r] = j < K ? (float)routes[j] : finf();
    ki[r] = j < K ? j : kInvalid;
  }
  wave_sort<2>(kd, ki);
  const uint32_t R = a.R;
  if ((uint32_t)ln < R) {
    const uint32_t y = lu[ki[0]];
    a.prn[(size_t)u * R + ln] = y;
    const size_t q = (size_t)u * R + ln;
    a.rec_t[q] = y;
    a.rec_s[q] = u;
    a.rec_d[q] = (float)ln;
  }
}

// Output list of node y: the first R/2 of its pruned list, its reverse
// neighbours by (position, source), the rest of its pruned list, without
// repeats, up to R; written to the pool row of y.
__global__ __launch_bounds__(64) void k_cagra_out(BuildArgs a) {
  const uint32_t y = blockIdx.x;
  if (y >= a.n) return;
  __shared__ uint32_t outL[64];
  const int ln = lane();
  const uint32_t R = a.R, half = R / 2;
  const uint32_t p = (uint32_t)ln < R ? a.prn[(size_t)y * R + ln] : kInvalid;
  const uint32_t ph = (uint32_t)ln < half ? p : kInvalid;  // the first half
  // the R - half smallest (position, source) reverse neighbours outside the first half
  float rd[1] = {finf()};
  uint32_t ri[1] = {kInvalid};
  const uint32_t g0 = a.goff[y], g1 = a.goff[y + 1];
  for (uint32_t b = g0; b < g1; b += 64) {
    const bool in = b + ln < g1;
    uint32_t s = in ? a.gsrc[b + ln] : kInvalid;
    const float d = in ? a.gd[b + ln] : finf();
    bool dup = false;
    for (uint32_t t = 0; t < half; t++) dup |= s == rdlane(ph, (int)t);
    wave_merge_new<1>(rd, ri, in && !dup ? d : finf(), in && !dup ? s : kInvalid, (int)(R - half));
  }
  const uint32_t nr = (uint32_t)popc(ballot(kvalid(ri[0])));
  if ((uint32_t)ln < half) outL[ln] = p;
  if ((uint32_t)ln < nr) outL[half + ln] = ri[0];
  // the rest of the pruned list, skipping the reverse neighbours taken
  bool take = (uint32_t)ln >= half && (uint32_t)ln < R;
  if (take)
    for (uint32_t t = 0; t < nr; t++) take &= p != rdlane(ri[0], (int)t);
  const uint64_t tm = ballot(take);
  const uint32_t filled = half + nr;
  if (take && filled + (uint32_t)mbcnt(tm) < R) outL[filled + mbcnt(tm)] = p;
  __syncthreads();
  const uint32_t total = min(R, filled + (uint32_t)popc(tm));
  const uint32_t id = a.ids[y];
  if ((uint32_t)ln < R) a.pool.adj[(size_t)id * R + ln] = (uint32_t)ln < total ? a.ids[outL[ln]] : kInvalid;
  if (ln == 0) a.pool.deg[id] = total;
}

// ------------------------------------------------------------------ launches
hipError_t launch_build_check(const BuildArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_nnd_check, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_build_init(int kind, const BuildArgs &a, hipStream_t s) {
  if (kind == kU8L2) hipLaunchKernelGGL(k_nnd_init<kU8L2>, dim3(a.n), dim3(64), 0, s, a);
  else if (kind == kF32L2) hipLaunchKernelGGL(k_nnd_init<kF32L2>, dim3(a.n), dim3(64), 0, s, a);
  else hipLaunchKernelGGL(k_nnd_init<kF32IP>, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_build_sample(const BuildArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_nnd_sample, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_build_cands(const BuildArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_nnd_cands, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}
// rows of the 4S candidates staged in LDS when they fit in this many bytes
constexpr size_t kJoinLds = 32768;
size_t build_join_lds(const BuildArgs &a) {
  const size_t b = (size_t)4 * a.S * a.pool.stride;
  return b <= kJoinLds ? b : 0;
}
hipError_t launch_build_join(int kind, const BuildArgs &a0, bool write, hipStream_t s) {
  BuildArgs a = a0;
  const size_t lds = build_join_lds(a);
  a.stage_rows = lds ? 1 : 0;
  const uint32_t g = a.v1 - a.v0;
  if (g == 0) return hipSuccess;
#define GR_JOIN(K_)                                                                              \
  do {                                                                                           \
    if (write) hipLaunchKernelGGL((k_nnd_join<K_, true>), dim3(g), dim3(64), lds, s, a);          \
    else hipLaunchKernelGGL((k_nnd_join<K_, false>), dim3(g), dim3(64), lds, s, a);               \
  } while (0)
  if (kind == kU8L2) GR_JOIN(kU8L2);
  else if (kind == kF32L2) GR_JOIN(kF32L2);
  else GR_JOIN(kF32IP);
#undef GR_JOIN
  return hipGetLastError();
}
hipError_t launch_build_merge(const BuildArgs &a, uint32_t grid, hipStream_t s) {
  hipLaunchKernelGGL(k_nnd_merge, dim3(grid), dim3(64), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_build_rank(const BuildArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_cagra_rank, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_build_out(const BuildArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_cagra_out, dim3(a.n), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace gr
