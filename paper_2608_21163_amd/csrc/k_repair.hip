// k_repair.hip -- in-place delete repair of GrAND-Vamana (Alg. 6).
//
// For every deleted p_i (one wavefront each):
//   in-neighbour repair : every z in N_in(p_i) outside the batch (exact, from
//     the reverse graph) gets the c points of C_i closest to z as scratch
//     records (z, y, Dist(z, y)), plus a marker record that makes z dirty
//     even when nothing is added;
//   out-neighbour repair: every w in N_out(p_i) outside the batch is added
//     to the scratch of the c points y of C_i closest to w: records
//     (y, w, Dist(w, y)).
// C_i is the first k_repair keys of the search from x_{p_i} outside the
// batch.  Records go to fixed offsets (a prefix sum of per-node counts), so
// no atomics are needed and the layout is deterministic.
#include "dispatch.h"

namespace gr {

__device__ __forceinline__ void rev_row(const RepairArgs &a, uint32_t i, uint32_t p, uint32_t &b0, uint32_t &b1) {
  const uint32_t r = a.rev_by_batch ? i : p;
  b0 = a.rev_off[r];
  b1 = a.rev_off[r + 1];
}

__global__ void k_repair_count(RepairArgs a, uint32_t *counts) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  const uint32_t p = a.ids[i];
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  uint32_t nin = 0, nout = 0;
  for (uint32_t j = b0; j < b1; j++) nin += a.in_batch[a.rev_src[j]] ? 0u : 1u;
  for (uint32_t t = 0; t < a.pool.R; t++) {
    const uint32_t w = a.pool.adj[(size_t)p * a.pool.R + t];
    nout += (w != kInvalid && !a.in_batch[w]) ? 1u : 0u;
  }
  counts[i] = nin * (a.c + 1) + nout * a.c;
}

hipError_t launch_repair_count(const RepairArgs &a, uint32_t *counts, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_repair_count, dim3((a.n + 255) / 256), dim3(256), 0, s, a, counts);
  return hipGetLastError();
}

// The c (distance, id)-smallest points of C_i other than x, measured from x.
// Lane t < c ends with the t-th one (invalid when C_i has fewer points).
template <int KIND, int LPV, int CPL>
__device__ __forceinline__ void closest_c(const RepairArgs &a, uint32_t cv, uint32_t x, uint32_t *lst, float *ldist,
                                          float &od, uint32_t &oi, unsigned long long &evals) {
  const int ln = lane();
  const PoolView &P = a.pool;
  const bool ok = kvalid(cv) && cv != x;
  const uint64_t m = ballot(ok);
  const int cnt = popc(m);
  if (ok) lst[mbcnt(m)] = cv;
  Slice<KIND, LPV, CPL> s;
  load_slice<KIND, LPV, CPL>(s, P.vecs + (size_t)x * P.stride, P.nch);
  __syncthreads();
  wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, lst, ldist, cnt);
  __syncthreads();
  evals += (unsigned long long)cnt;
  float d[1] = {ln < cnt ? ldist[ln] : finf()};
  uint32_t id[1] = {ln < cnt ? lst[ln] : kInvalid};
  __syncthreads();
  wave_sort<1>(d, id);
  od = d[0];
  oi = id[0];
}

template <int KIND, int LPV, int CPL>
__global__ __launch_bounds__(64) void k_repair(RepairArgs a) {
  __shared__ uint32_t lst[64];
  __shared__ float ldist[64];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t cv = ln < (int)a.kr ? a.ci[(size_t)i * a.kr + ln] : kInvalid;
  uint32_t r = a.rofs[i];
  unsigned long long evals = 0, rows = popc(ballot(kvalid(cv)));
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  for (uint32_t j = b0; j < b1; j++) {
    const uint32_t z = a.rev_src[j];
    if (a.in_batch[z]) continue;
    float od;
    uint32_t oi;
    closest_c<KIND, LPV, CPL>(a, cv, z, lst, ldist, od, oi, evals);
    rows++;
    if (ln < (int)a.c) {
      a.rec_t[r + ln] = z;
      a.rec_s[r + ln] = oi;
      a.rec_d[r + ln] = kvalid(oi) ? od : 0.0f;
    }
    if (ln == 0) {
      a.rec_t[r + a.c] = z;
      a.rec_s[r + a.c] = kInvalid;
      a.rec_d[r + a.c] = 0.0f;
    }
    r += a.c + 1;
  }
  for (uint32_t t = 0; t < P.R; t++) {
    const uint32_t w = P.adj[(size_t)p * P.R + t];
    if (w == kInvalid || a.in_batch[w]) continue;
    float od;
    uint32_t oi;
    closest_c<KIND, LPV, CPL>(a, cv, w, lst, ldist, od, oi, evals);
    rows++;
    if (ln < (int)a.c) {
      const bool v = kvalid(oi);
      a.rec_t[r + ln] = v ? oi : kInvalid;
      a.rec_s[r + ln] = v ? w : kInvalid;
      a.rec_d[r + ln] = v ? od : 0.0f;
    }
    r += a.c;
  }
  if (ln == 0) {
    atomicAdd(&a.ds->records, (unsigned long long)(r - a.rofs[i]));
    atomicAdd(&a.ds->rep_evals, evals);
    atomicAdd(&a.ds->rep_rows, rows);
    atomicAdd(&a.ds->rep_recs, (unsigned long long)(r - a.rofs[i]));
  }
}

hipError_t launch_repair(int kind, int vc, const RepairArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  GR_DISPATCH_KV(kind, vc, {
    hipLaunchKernelGGL((k_repair<KIND, LPV, CPL>), dim3(a.n), dim3(64), 0, st, a);
    return hipGetLastError();
  });
  return hipErrorInvalidValue;
}

}  // namespace gr
