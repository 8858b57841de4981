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

// Records per deleted node, one wavefront each: (c + 1) per in-neighbour
// and c per out-neighbour outside the batch.
__global__ __launch_bounds__(64) void k_repair_count(RepairArgs a, uint32_t *counts) {
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const int ln = lane();
  const uint32_t p = a.ids[i];
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  uint32_t nin = 0;
  for (uint32_t base = b0; base < b1; base += 64) {
    const uint32_t j = base + ln;
    const uint32_t z = j < b1 ? a.rev_src[j] : kInvalid;
    nin += (uint32_t)popc(ballot(z != kInvalid && !a.in_batch[z]));
  }
  const uint32_t w = ln < (int)a.pool.R ? a.pool.adj[(size_t)p * a.pool.R + ln] : kInvalid;
  const uint32_t nout = (uint32_t)popc(ballot(w != kInvalid && !a.in_batch[w]));
  if (ln == 0) counts[i] = nin * (a.c + 1) + nout * a.c;
}

hipError_t launch_repair_count(const RepairArgs &a, uint32_t *counts, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_repair_count, dim3(a.n), dim3(64), 0, s, a, counts);
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

// ---------------------------------------------------------------------------
// uint8 repair on the matrix cores, for rows of 64*NK bytes, k_repair <= 64
// and c <= K.  The "c closest points of C_i" of every repaired neighbour x
// are rows of one distance matrix {x} x C_i, so C_i (at most 4 tiles of 16
// candidates) is held in registers in the MFMA operand layout, the
// neighbours are taken 16 at a time as the other operand, and each
// 16 x 16 MFMA tile gives exact int32 distances (x ^ 0x80 operands).  Each
// lane keeps, for the 4 output rows it holds, the K smallest (distance, id)
// keys of its candidate column; the lists of the 16 lanes of a row are
// merged by a butterfly.  Records and their offsets are those of k_repair.

// Sorted list of the K smallest keys: inserts (d, id).
template <int K>
__device__ __forceinline__ void kl_insert(float (&ld)[K], uint32_t (&li)[K], float d, uint32_t id) {
  bool lt[K];
#pragma unroll
  for (int j = 0; j < K; j++) lt[j] = kless(d, id, ld[j], li[j]);
#pragma unroll
  for (int j = K - 1; j >= 0; j--) {
    const bool shift = j > 0 && lt[j > 0 ? j - 1 : 0];
    const float pd = ld[j > 0 ? j - 1 : 0];
    const uint32_t pi = li[j > 0 ? j - 1 : 0];
    ld[j] = shift ? pd : (lt[j] ? d : ld[j]);
    li[j] = shift ? pi : (lt[j] ? id : li[j]);
  }
}

template <int NK, int K>
__global__ __launch_bounds__(64) void k_repair_mfma(RepairArgs a) {
  constexpr int NT = 4;
  __shared__ uint32_t xl[64];
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const size_t goff = (size_t)g * 16;
  const int kr = (int)a.kr, nt = (kr + 15) >> 4;
  const int c = (int)a.c;
  v4i B[NT][NK];
  int nrmC[NT];
  uint32_t cid[NT];
  unsigned long long rows = 0;
#pragma unroll
  for (int t = 0; t < NT; t++) {
    cid[t] = kInvalid;
    nrmC[t] = 0;
    if (t < nt) {
      const int e = 16 * t + col;
      const uint32_t cv = e < kr ? a.ci[(size_t)i * kr + e] : kInvalid;
      cid[t] = cv;
      const uint8_t *row = P.vecs + (size_t)(kvalid(cv) ? cv : p) * P.stride + goff;
      int sq = 0;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) {
        B[t][kk] = to_i8x16(ld16(row + (size_t)kk * 64));
        sq = sq_i8x16(B[t][kk], sq);
      }
      sq += (int)xshfl((uint32_t)sq, 16);
      sq += (int)xshfl((uint32_t)sq, 32);
      nrmC[t] = sq;
    }
    rows += (unsigned long long)popc(ballot(g == 0 && kvalid(cid[t])));
  }
  const uint32_t r0 = a.rofs[i];
  uint32_t r = r0;
  uint32_t evals = 0;
  // xl[0..cnt): neighbours; inbound: in-neighbours z (records to z plus a
  // marker), else out-neighbours w (records to the chosen points)
  auto process = [&](int cnt, bool inbound) {
    for (int q = 0; q < cnt; q += 16) {
      const int e = q + col;
      const uint32_t x = xl[e < cnt ? e : q];
      const uint8_t *row = P.vecs + (size_t)x * P.stride + goff;
      v4i A[NK];
      int na = 0;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) {
        A[kk] = to_i8x16(ld16(row + (size_t)kk * 64));
        na = sq_i8x16(A[kk], na);
      }
      na += (int)xshfl((uint32_t)na, 16);
      na += (int)xshfl((uint32_t)na, 32);
      int rn[4];
      uint32_t rx[4];
#pragma unroll
      for (int ii = 0; ii < 4; ii++) {
        const int xe = q + 4 * g + ii;
        rn[ii] = __shfl(na, 4 * g + ii, 64);
        rx[ii] = xe < cnt ? xl[xe] : kInvalid;
      }
      float ld[4][K];
      uint32_t li[4][K];
#pragma unroll
      for (int ii = 0; ii < 4; ii++)
#pragma unroll
        for (int j = 0; j < K; j++) { ld[ii][j] = finf(); li[ii][j] = kInvalid; }
#pragma unroll
      for (int t = 0; t < NT; t++) {
        if (t >= nt) continue;
        v4i acc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < NK; kk++) acc = mfma_i8(A[kk], B[t][kk], acc);
#pragma unroll
        for (int ii = 0; ii < 4; ii++) {
          const bool ok = kvalid(cid[t]) && kvalid(rx[ii]) && cid[t] != rx[ii];
          const float d = canon0((float)(rn[ii] + nrmC[t] - 2 * acc[ii]));
          evals += ok ? 1u : 0u;
          kl_insert<K>(ld[ii], li[ii], ok ? d : finf(), ok ? cid[t] : kInvalid);
        }
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1)
#pragma unroll
        for (int ii = 0; ii < 4; ii++) {
          float od[K];
          uint32_t oi[K];
#pragma unroll
          for (int j = 0; j < K; j++) { od[j] = xshfl(ld[ii][j], o); oi[j] = xshfl(li[ii][j], o); }
#pragma unroll
          for (int j = 0; j < K; j++) kl_insert<K>(ld[ii], li[ii], od[j], oi[j]);
        }
#pragma unroll
      for (int ii = 0; ii < 4; ii++) {
        const int xe = q + 4 * g + ii;
        if (xe >= cnt) continue;
        const uint32_t xid = rx[ii];
        float yd = finf();
        uint32_t yi = kInvalid;
#pragma unroll
        for (int j = 0; j < K; j++)
          if (j == col) { yd = ld[ii][j]; yi = li[ii][j]; }
        const bool v = kvalid(yi);
        if (inbound) {
          const uint32_t base = r + (uint32_t)xe * (uint32_t)(c + 1);
          if (col < c) {
            a.rec_t[base + col] = xid;
            a.rec_s[base + col] = yi;
            a.rec_d[base + col] = v ? yd : 0.0f;
          } else if (col == c) {
            a.rec_t[base + c] = xid;
            a.rec_s[base + c] = kInvalid;
            a.rec_d[base + c] = 0.0f;
          }
        } else if (col < c) {
          const uint32_t base = r + (uint32_t)xe * (uint32_t)c;
          a.rec_t[base + col] = v ? yi : kInvalid;
          a.rec_s[base + col] = v ? xid : kInvalid;
          a.rec_d[base + col] = v ? yd : 0.0f;
        }
      }
    }
    r += (uint32_t)cnt * (uint32_t)(inbound ? c + 1 : c);
    rows += (unsigned long long)cnt;
  };
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  for (uint32_t base = b0; base < b1; base += 64) {
    const uint32_t j = base + ln;
    const uint32_t z = j < b1 ? a.rev_src[j] : kInvalid;
    const bool ok = z != kInvalid && !a.in_batch[z];
    const uint64_t m = ballot(ok);
    __syncthreads();
    if (ok) xl[mbcnt(m)] = z;
    __syncthreads();
    if (m) process(popc(m), true);
  }
  {
    const uint32_t w = ln < (int)P.R ? P.adj[(size_t)p * P.R + ln] : kInvalid;
    const bool ok = w != kInvalid && !a.in_batch[w];
    const uint64_t m = ballot(ok);
    __syncthreads();
    if (ok) xl[mbcnt(m)] = w;
    __syncthreads();
    if (m) process(popc(m), false);
  }
  unsigned long long ev = evals;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ev += __shfl_xor(ev, o, 64);
  if (ln == 0) {
    atomicAdd(&a.ds->records, (unsigned long long)(r - r0));
    atomicAdd(&a.ds->rep_evals, ev);
    atomicAdd(&a.ds->rep_rows, rows);
    atomicAdd(&a.ds->rep_recs, (unsigned long long)(r - r0));
  }
}

hipError_t launch_repair(int kind, int vc, const RepairArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  if (kind == kU8L2 && a.kr <= 64 && a.c <= 4 && (a.pool.nch == 4 || a.pool.nch == 8)) {
    if (a.pool.nch == 8) {
      if (a.c <= 2) hipLaunchKernelGGL((k_repair_mfma<2, 2>), dim3(a.n), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_repair_mfma<2, 4>), dim3(a.n), dim3(64), 0, st, a);
    } else {
      if (a.c <= 2) hipLaunchKernelGGL((k_repair_mfma<1, 2>), dim3(a.n), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_repair_mfma<1, 4>), dim3(a.n), dim3(64), 0, st, a);
    }
    return hipGetLastError();
  }
  GR_DISPATCH_KV(kind, vc, {
    hipLaunchKernelGGL((k_repair<KIND, LPV, CPL>), dim3(a.n), dim3(64), 0, st, a);
    return hipGetLastError();
  });
  return hipErrorInvalidValue;
}

}  // namespace gr
