// k_prune.hip -- GrANDRobustPrune (Alg. 4) executed by one wavefront, the
// forward prune of new nodes (Alg. 5, second loop) and the rebuild of every
// dirty node (Alg. 5 and Alg. 6, last loops), one wavefront per node.
#include "dispatch.h"

namespace gr {

// GrANDRobustPrune of node p.  Candidates (any order, invalid padded) come
// with their cached distances D_p (Section 3.1: reused, not recomputed).
// They are sorted by (D_p, id); repeats and p itself are dropped.  The
// first valid candidate p* is selected; selection stops at R; otherwise the
// distance from p* to every later valid candidate p' is evaluated by the
// wave (pivot p* held in registers, candidate rows gathered LPV lanes per
// row) and p' is invalidated when coef * Dist(p*, p') <= D_p[p'] (coef is
// alpha, or alpha^2 for the Euclidean reading, compared in fp64).
// On return lane t < nsel holds the t-th selected id and its distance.
template <int KIND, int LPV, int CPL, int NR>
__device__ int wave_prune(const PoolView &P, uint32_t p, uint32_t R, double coef, float (&cd)[NR],
                          uint32_t (&ci)[NR], uint32_t *lids, float *ldist, uint32_t &sel_id, float &sel_d,
                          unsigned long long &evals) {
  const int ln = lane();
#pragma unroll
  for (int r = 0; r < NR; r++)
    if ((ci[r] & kIdMask) == p || !kvalid(ci[r])) { cd[r] = finf(); ci[r] = kInvalid; }
  wave_sort<NR>(cd, ci);
  uint64_t dm[NR];
  if (wave_find_repeats<NR>(cd, ci, dm)) {
#pragma unroll
    for (int r = 0; r < NR; r++)
      if ((dm[r] >> ln) & 1) { cd[r] = finf(); ci[r] = kInvalid; }
    wave_sort<NR>(cd, ci);
  }
  bool valid[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) valid[r] = kvalid(ci[r]);
  sel_id = kInvalid;
  sel_d = finf();
  int nsel = 0;
  while (nsel < (int)R) {
    int e = -1;
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint64_t m = ballot(valid[r]);
      if (e < 0 && m) e = r * 64 + ffs64(m);
    }
    if (e < 0) break;
    const int er = e >> 6, el = e & 63;
    uint32_t pid = 0;
    float pd = 0.0f;
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (r == er) {
        pid = rdlane(ci[r], el);
        pd = rdlane(cd[r], el);
        if (ln == el) valid[r] = false;
      }
    if (ln == nsel) { sel_id = pid; sel_d = pd; }
    nsel++;
    if (nsel == (int)R) break;
    // compact the remaining valid candidates (all lie after p*)
    int cnt = 0;
    int cidx[NR];
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint64_t m = ballot(valid[r]);
      cidx[r] = cnt + mbcnt(m);
      if (valid[r]) lids[cidx[r]] = ci[r];
      cnt += popc(m);
    }
    if (cnt == 0) break;
    Slice<KIND, LPV, CPL> s;
    load_slice<KIND, LPV, CPL>(s, P.vecs + (size_t)pid * P.stride, P.nch);
    __syncthreads();
    wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, lids, ldist, cnt);
    __syncthreads();
    evals += (unsigned long long)cnt;
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (valid[r] && coef * (double)ldist[cidx[r]] <= (double)cd[r]) valid[r] = false;
    __syncthreads();
  }
  return nsel;
}

// Forward lists of new nodes: GrANDRobustPrune(p_i, V_i \ {p_i}, D_{p_i}),
// written to p_i's row (each new node owns its row), and the reverse-edge
// records (u, p_i, D_{p_i}[u]) for every selected u.
template <int KIND, int LPV, int CPL, int NR>
__global__ __launch_bounds__(64) void k_fwd_prune(FwdPruneArgs a) {
  __shared__ uint32_t lids[64 * NR];
  __shared__ float ldist[64 * NR];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t nv = a.v_n[i];
  float cd[NR];
  uint32_t ci[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) {
    const uint32_t e = r * 64 + ln;
    const bool in = e < nv;
    cd[r] = in ? a.v_d[(size_t)i * a.v_stride + e] : finf();
    ci[r] = in ? a.v_ids[(size_t)i * a.v_stride + e] : kInvalid;
  }
  unsigned long long evals = 0;
  uint32_t sid;
  float sdist;
  const int nsel = wave_prune<KIND, LPV, CPL, NR>(P, p, P.R, a.coef, cd, ci, lids, ldist, sid, sdist, evals);
  if (ln < (int)P.R) {
    const bool in = ln < nsel;
    P.adj[(size_t)p * P.R + ln] = in ? sid : kInvalid;
    a.rec_t[(size_t)i * P.R + ln] = in ? sid : kInvalid;
    a.rec_s[(size_t)i * P.R + ln] = p;
    a.rec_d[(size_t)i * P.R + ln] = in ? sdist : 0.0f;
  }
  if (ln == 0) {
    P.deg[p] = (uint32_t)nsel;
    atomicAdd(&a.ds->fwd_prunes, 1ull);
    atomicAdd(&a.ds->fwd_evals, evals);
    atomicAdd(&a.ds->records, (unsigned long long)nsel);
  }
}

// Rebuild of dirty nodes.  For dirty u: scratch_u = the P smallest distinct
// (distance, source) records addressed to u; C = (N_out(u) u scratch_u)
// minus u (and minus the delete batch); if |C| <= R, C is installed (kept
// entries in slot order, then new sources in record order); otherwise D_u
// is computed for the kept entries (records carry the distance of new
// sources) and GrANDRobustPrune(u, C, D_u) is installed.  One owner per
// dirty node, so rows are written without locks.
template <int KIND, int LPV, int CPL, int NP, int NC>
__global__ __launch_bounds__(64) void k_rebuild(RebuildArgs a) {
  __shared__ uint32_t rowL[64];
  __shared__ uint32_t lids[64 * NC];
  __shared__ float ldist[64 * NC];
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const uint32_t nd_total = a.ds->n_dirty;
  unsigned long long evals = 0, prunes = 0, nodes = 0, recs = 0, cand = 0;
  for (uint32_t it = blockIdx.x; it < nd_total; it += gridDim.x) {
    const uint32_t u = a.dirty[it];
    nodes++;
    const uint32_t g0 = a.goff[u], g1 = a.goff[u + 1];
    recs += g1 - g0;
    float sd[NP];
    uint32_t si[NP];
#pragma unroll
    for (int r = 0; r < NP; r++) { sd[r] = finf(); si[r] = kInvalid; }
    for (uint32_t base = g0; base < g1; base += 64) {
      const uint32_t j = base + ln;
      uint32_t sv = j < g1 ? a.gsrc[j] : kInvalid;
      float dv = j < g1 ? a.gd[j] : finf();
      if (!kvalid(sv)) { sv = kInvalid; dv = finf(); }
      wave_merge_new<NP>(sd, si, dv, sv, (int)a.P);
    }
    const uint32_t rv = ln < (int)R ? P.adj[(size_t)u * R + ln] : kInvalid;
    const bool keep = rv != kInvalid && rv != u && !(a.in_batch && a.in_batch[rv]);
    rowL[ln] = keep ? rv : kInvalid;
    __syncthreads();
    bool isnew[NP];
#pragma unroll
    for (int r = 0; r < NP; r++) {
      const uint32_t sv = si[r];
      bool ok = kvalid(sv) && sv != u && !(a.in_batch && a.in_batch[sv]);
      for (uint32_t t = 0; t < R; t++) ok = ok && rowL[t] != sv;
      isnew[r] = ok;
    }
    const uint64_t km = ballot(keep);
    const int kr = popc(km);
    int kn = 0;
    int npos[NP];
#pragma unroll
    for (int r = 0; r < NP; r++) {
      const uint64_t mm = ballot(isnew[r]);
      npos[r] = kn + mbcnt(mm);
      kn += popc(mm);
    }
    const int m = kr + kn;
    if (keep) lids[mbcnt(km)] = rv;
    if (m <= (int)R) {
#pragma unroll
      for (int r = 0; r < NP; r++)
        if (isnew[r]) lids[kr + npos[r]] = si[r];
      __syncthreads();
      if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < m ? lids[ln] : kInvalid;
      if (ln == 0) P.deg[u] = (uint32_t)m;
    } else {
      __syncthreads();
      Slice<KIND, LPV, CPL> s;
      load_slice<KIND, LPV, CPL>(s, P.vecs + (size_t)u * P.stride, P.nch);
      wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, lids, ldist, kr);
      evals += (unsigned long long)kr;
      __syncthreads();
#pragma unroll
      for (int r = 0; r < NP; r++)
        if (isnew[r]) { lids[kr + npos[r]] = si[r]; ldist[kr + npos[r]] = sd[r]; }
      __syncthreads();
      float cd[NC];
      uint32_t ci[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const int e = r * 64 + ln;
        cd[r] = e < m ? ldist[e] : finf();
        ci[r] = e < m ? lids[e] : kInvalid;
      }
      __syncthreads();
      uint32_t sid;
      float sdist;
      const int nsel = wave_prune<KIND, LPV, CPL, NC>(P, u, R, a.coef, cd, ci, lids, ldist, sid, sdist, evals);
      if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < nsel ? sid : kInvalid;
      if (ln == 0) P.deg[u] = (uint32_t)nsel;
      prunes++;
      cand += (unsigned long long)m + 1;
    }
    __syncthreads();
  }
  if (ln == 0) {
    atomicAdd(&a.ds->rb_prunes, prunes);
    atomicAdd(&a.ds->rb_evals, evals);
    atomicAdd(&a.ds->dirty, nodes);
    atomicAdd(&a.ds->rb_recs, recs);
    atomicAdd(&a.ds->rb_cand, cand);
  }
}

hipError_t launch_fwd_prune(int kind, int vc, uint32_t max_iters, const FwdPruneArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  GR_DISPATCH_KV(kind, vc, GR_DISPATCH_N(max_iters, {
    hipLaunchKernelGGL((k_fwd_prune<KIND, LPV, CPL, NR>), dim3(a.n), dim3(64), 0, st, a);
    return hipGetLastError();
  }));
  return hipErrorInvalidValue;
}

hipError_t launch_rebuild(int kind, int vc, uint32_t R, uint32_t P, const RebuildArgs &a, uint32_t grid,
                          hipStream_t st) {
  if (grid == 0) return hipSuccess;
  if (P > 128 || R + P > 256) return hipErrorInvalidValue;
  GR_DISPATCH_KV(kind, vc, {
    if (P <= 64 && R + P <= 128) {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, 1, 2>), dim3(grid), dim3(64), 0, st, a);
    } else if (P <= 64) {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, 1, 4>), dim3(grid), dim3(64), 0, st, a);
    } else {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, 2, 4>), dim3(grid), dim3(64), 0, st, a);
    }
    return hipGetLastError();
  });
  return hipErrorInvalidValue;
}

}  // namespace gr
