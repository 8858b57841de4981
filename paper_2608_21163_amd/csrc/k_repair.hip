// k_repair.hip -- in-place delete repair of GrAND-Vamana (Alg. 6).
//
// For every deleted p_i:
//   in-neighbour repair : every z in N_in(p_i) outside the batch (exact, from
//     the reverse graph) gets the c points of C_i closest to z as scratch
//     records (z, y, Dist(z, y)), plus a marker record that makes z dirty
//     even when nothing is added;
//   out-neighbour repair: every w in N_out(p_i) outside the batch is added
//     to the scratch of the c points y of C_i closest to w: records
//     (y, w, Dist(w, y)).
// C_i is the first k_repair keys of the search from x_{p_i} outside the
// batch.
//
// Record layout (fixed, so every piece of work knows where its records go
// without a prefix over filtered neighbours): deleted node i owns
// nin_i*(c+1) + R*c records from rofs[i]; in-neighbour e (in reverse-row
// order) owns c+1 of them, out-slot t of N_out(p_i) owns c.  Neighbours in
// the batch, empty slots and missing points give records whose target is
// INVALID, which the grouping skips.
#include "dispatch.h"

namespace gr {

__device__ __forceinline__ void rev_row(const RepairArgs &a, uint32_t i, uint32_t p, uint32_t &b0, uint32_t &b1) {
  const uint32_t r = a.rev_by_batch ? i : p;
  b0 = a.rev_off[r];
  b1 = a.rev_off[r + 1];
}

// Work positions of deleted node i: its nin in-neighbours (positions
// 0 .. nin-1, in reverse-row order) followed by its R out-slots.  Position e
// owns c+1 records from rofs[i] + e*(c+1) when it is an in-neighbour, c
// records from rofs[i] + nin*(c+1) + (e-nin)*c when it is an out-slot.
// A work chunk is a run of at most a.cw positions of one node, so most nodes
// are one chunk (their C_i tiles loaded once) and a node with a long
// in-neighbour list is spread over several.
__global__ void k_repair_plan(RepairArgs a, uint32_t *counts, uint32_t *chunks) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.n) return;
  uint32_t b0, b1;
  rev_row(a, i, a.ids[i], b0, b1);
  const uint32_t nin = b1 - b0;
  counts[i] = nin * (a.c + 1) + a.pool.R * a.c;
  chunks[i] = (nin + a.pool.R + a.cw - 1) / a.cw;
}

// The descriptor of every work chunk j of deleted node i (one wave per
// node), so that a repair wave starts a chunk with one pair of loads instead
// of a chain of dependent ones.
__global__ void k_repair_map(RepairArgs a, uint4 *cdesc) {
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const uint32_t c0 = a.coff[i], c1 = a.coff[i + 1];
  const uint32_t p = a.ids[i];
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  const uint32_t nin = b1 - b0, npos = nin + a.pool.R;
  for (uint32_t q = c0 + threadIdx.x; q < c1; q += blockDim.x) {
    const uint32_t j = q - c0, e0 = j * a.cw;
    cdesc[2 * (size_t)q] = make_uint4(i, p, b0, nin);
    cdesc[2 * (size_t)q + 1] = make_uint4(a.rofs[i], e0, min(a.cw, npos - e0), j);
  }
}

// Position e of a chunk's node: its neighbour (INVALID when the slot is
// empty or the neighbour is in the batch) ...
__device__ __forceinline__ uint32_t repair_nbr(const RepairArgs &a, uint4 d0, uint32_t e) {
  const uint32_t p = d0.y, b0 = d0.z, nin = d0.w;
  const uint32_t x = e < nin ? a.rev_src[b0 + e] : a.pool.adj[(size_t)p * a.pool.R + (e - nin)];
  return (x != kInvalid && !a.in_batch[x]) ? x : kInvalid;
}
// ... and its records: c + 1 from `base` for an in-neighbour (the last one
// the marker), c for an out-slot.
__device__ __forceinline__ uint32_t repair_base(const RepairArgs &a, uint4 d0, uint32_t rbase, uint32_t e) {
  const uint32_t nin = d0.w, c = a.c;
  return rbase + (e < nin ? e * (c + 1) : nin * (c + 1) + (e - nin) * c);
}

hipError_t launch_repair_plan(const RepairArgs &a, uint32_t *counts, uint32_t *chunks, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_repair_plan, dim3((a.n + 255) / 256), dim3(256), 0, s, a, counts, chunks);
  return hipGetLastError();
}
hipError_t launch_repair_map(const RepairArgs &a, uint4 *cdesc, hipStream_t s) {
  if (a.n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_repair_map, dim3(a.n), dim3(64), 0, s, a, cdesc);
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

// One wavefront per deleted node, any element type: each neighbour's c
// closest points of C_i come from a gather and a sort of its distances.
template <int KIND, int LPV, int CPL>
__global__ __launch_bounds__(64) void k_repair(RepairArgs a) {
  __shared__ uint32_t lst[64];
  __shared__ float ldist[64];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n || (size_t)a.rofs[a.n] > a.rcap) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t c = a.c;
  const uint32_t cv = ln < (int)a.kr ? a.ci[(size_t)i * a.kr + ln] : kInvalid;
  unsigned long long evals = 0, rows = popc(ballot(kvalid(cv))), recs = 0;
  uint32_t b0, b1;
  rev_row(a, i, p, b0, b1);
  const uint32_t r0 = a.rofs[i];
  for (uint32_t e = 0; e < b1 - b0; e++) {
    const uint32_t z = a.rev_src[b0 + e];
    const uint32_t base = r0 + e * (c + 1);
    if (z == kInvalid || a.in_batch[z]) {
      for (uint32_t k = ln; k <= c; k += 64) a.rec_t[base + k] = kInvalid;
      continue;
    }
    float od;
    uint32_t oi;
    closest_c<KIND, LPV, CPL>(a, cv, z, lst, ldist, od, oi, evals);
    rows++;
    recs += c + 1;
    if (ln < (int)c) {
      a.rec_t[base + ln] = z;
      a.rec_s[base + ln] = oi;
      a.rec_d[base + ln] = kvalid(oi) ? od : 0.0f;
    }
    if (ln == 0) {
      a.rec_t[base + c] = z;
      a.rec_s[base + c] = kInvalid;
      a.rec_d[base + c] = 0.0f;
    }
  }
  const uint32_t ro = r0 + (b1 - b0) * (c + 1);
  for (uint32_t t = 0; t < P.R; t++) {
    const uint32_t w = P.adj[(size_t)p * P.R + t];
    const uint32_t base = ro + t * c;
    if (w == kInvalid || a.in_batch[w]) {
      for (uint32_t k = ln; k < c; k += 64) a.rec_t[base + k] = kInvalid;
      continue;
    }
    float od;
    uint32_t oi;
    closest_c<KIND, LPV, CPL>(a, cv, w, lst, ldist, od, oi, evals);
    rows++;
    const bool v = kvalid(oi);
    recs += (unsigned long long)popc(ballot(ln < (int)c && v));
    if (ln < (int)c) {
      a.rec_t[base + ln] = v ? oi : kInvalid;
      a.rec_s[base + ln] = v ? w : kInvalid;
      a.rec_d[base + ln] = v ? od : 0.0f;
    }
  }
  if (ln == 0) {
    stat_add(a.ds, kStRecords, recs);
    stat_add(a.ds, kStRepEvals, evals);
    stat_add(a.ds, kStRepRows, rows);
    stat_add(a.ds, kStRepRecs, recs);
  }
}

// ---------------------------------------------------------------------------
// uint8 repair on the matrix cores, for rows of 64*NK bytes, k_repair <= 64
// and c <= K.  The c closest points of C_i of each repaired neighbour x are
// found in one distance block {neighbours} x C_i (exact int32 from int8
// MFMA on x ^ 0x80).  Work is split in chunks of at most 64*NPL positions of
// one deleted node (persistent waves over the chunk list).  Per chunk the
// C_i tiles are the MFMA A operand and 16 neighbours at a time the B
// operand: lane (g, col) then holds 16 candidate distances of neighbour col,
// keeps its K + 1 smallest keys, and the four lanes of a neighbour merge
// their lists (two exchanges).
//
// C_i arrives in ascending id order (points first), so a candidate's slot
// is its rank among the ids and 32-bit keys 64 * Dist + slot order like
// (Dist, id) (Dist < 2^23 for 128 uint8 dimensions).  A slot without a point
// gets a key of at least 2^30.  The key of x itself (when x is in C_i) is its
// slot alone, Dist being 0, which is how it is excluded.
//
// Inside the step the keys of one neighbour x are handled as the signed
// values n = 128 x.c' - 64 |c'|^2 - slot = 64 |x|^2 - key (one shift-add per
// candidate from the MFMA product), largest first; the 64 |x|^2 term, the
// same for all of x's candidates, is added back when the key is written.
// The lists keep K + 1 values, x's own included, and x's value is taken out
// of the merged list.
// Every |n| stays below 2^31 (empty slots near -1.5 * 2^30), so the
// signed order is exact.

// Sorted (descending) list of the L largest values: entry j of the new list
// is the median of old entries j - 1 and j and the new value (one v_med3).
template <int L>
__device__ __forceinline__ void kl_insert_max(int32_t (&l)[L], int32_t k) {
#pragma unroll
  for (int j = L - 1; j > 0; j--) l[j] = max(min(l[j - 1], l[j]), min(max(l[j - 1], l[j]), k));
  l[0] = max(l[0], k);
}
// l <- the L largest of the two descending lists l and o.
template <int L>
__device__ __forceinline__ void kl_merge_max(int32_t (&l)[L], const int32_t (&o)[L]) {
#pragma unroll
  for (int j = 0; j < L; j++) kl_insert_max<L>(l, o[j]);
}
constexpr int32_t kSlotNone = 0x60000000;  // 64 |c'|^2 + slot of an empty candidate slot
constexpr int32_t kNone = INT32_MIN;       // below every value: a list entry not yet filled
constexpr uint32_t kKeyValid = 1u << 30;   // keys of points are below

template <int NK, int K, int NPL>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(4))) void k_repair_mfma(RepairArgs a) {
  constexpr int NT = 4;        // C_i tiles (k_repair <= 64)
  constexpr int W = 64 * NPL;  // positions per chunk
  __shared__ uint32_t cidL[64];                 // C_i ids by slot (ascending, points first)
  __shared__ __align__(16) int32_t ckeyL[64];   // -(64 |c'|^2 + slot) (-kSlotNone when empty)
  __shared__ uint32_t xL[W];                    // the chunk's neighbours
  __shared__ uint32_t rxL[W];                   // slot of each neighbour in C_i, or ~0
  // the chunk's records, staged and written out together at its end (one
  // contiguous range: at most c + 1 <= K + 1 per position)
  __shared__ uint32_t rtL[W * (K + 1)], rsL[W * (K + 1)];
  __shared__ float rdL[W * (K + 1)];
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const PoolView &P = a.pool;
  const size_t goff = (size_t)g * 16;
  const int kr = (int)a.kr;
  const uint32_t c = a.c;
  if ((size_t)a.rofs[a.n] > a.rcap) return;  // the host grows the buffers and launches again
  const uint32_t total = a.coff[a.n];
  unsigned long long evals = 0, rows = 0, recs = 0;
  for (uint32_t q = blockIdx.x; q < total; q += gridDim.x) {
    const uint4 d0 = a.cdesc[2 * (size_t)q], d1 = a.cdesc[2 * (size_t)q + 1];
    const uint32_t i = d0.x, p = d0.y, rbase = d1.x, e0 = d1.y, j = d1.w;
    const int cnt = (int)d1.z;
    // The chunk's C_i ids (A operand slot 16t + col) and its neighbours
    // (position e0 + e in xL[e]), then the C_i rows and the neighbours'
    // batch flags: all loads of a level issued together, their addresses
    // clamped to valid ones and the results selected afterwards.
    uint32_t cl[NT];
#pragma unroll
    for (int t = 0; t < NT; t++) {
      const int e = 16 * t + col;
      cl[t] = a.ci[(size_t)i * kr + (e < kr ? e : 0)];
    }
    uint32_t xv[NPL];
#pragma unroll
    for (int u = 0; u < NPL; u++) {
      const uint32_t pe = e0 + (uint32_t)(ln + 64 * u);
      const uint32_t *src = pe < d0.w ? a.rev_src + d0.z + pe : P.adj + (size_t)p * P.R + (pe - d0.w);
      xv[u] = *((ln + 64 * u) < cnt ? src : P.adj + (size_t)p * P.R);
    }
    // C_i rows (bytes 16g + 64kk of candidate 16t + col); slots past
    // k_repair or without a point hold the deleted node's row
    uint4 Cr[NT][NK];
#pragma unroll
    for (int t = 0; t < NT; t++) {
      cl[t] = 16 * t + col < kr ? cl[t] : kInvalid;
      const uint8_t *row = P.vecs + (size_t)(kvalid(cl[t]) ? cl[t] : p) * P.stride + goff;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) Cr[t][kk] = ld16(row + (size_t)kk * 64);
    }
    uint8_t inb[NPL];
#pragma unroll
    for (int u = 0; u < NPL; u++) inb[u] = a.in_batch[xv[u] != kInvalid ? xv[u] : 0u];
#pragma unroll
    for (int u = 0; u < NPL; u++) {
      const int e = ln + 64 * u;
      xv[u] = (e < cnt && xv[u] != kInvalid && !inb[u]) ? xv[u] : kInvalid;
      xL[e] = xv[u];
      rows += (unsigned long long)popc(ballot(xv[u] != kInvalid));
    }
    __syncthreads();
    // The rows of neighbours 16s .. 16s+15 (the B operand of step s): lane
    // (g, col) loads bytes 16g + 64kk of neighbour 16s + col.  The loads of
    // step s + 1 are issued before step s is computed.
    uint4 Xn[NK];
    uint32_t xsn;
    auto load_step = [&](int s) {
      xsn = xL[16 * s + col];
      const uint8_t *row = P.vecs + (size_t)(xsn != kInvalid ? xsn : p) * P.stride + goff;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) Xn[kk] = ld16(row + (size_t)kk * 64);
    };
    load_step(0);
    // C_i tiles (A operand) and their squared norms
    v4i Ct[NT][NK];
    int cnr[NT];
#pragma unroll
    for (int t = 0; t < NT; t++) {
      int sq = 0;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) {
        Ct[t][kk] = to_i8x16(Cr[t][kk]);
        sq = sq_i8x16(Ct[t][kk], sq);
      }
      sq += (int)xshfl((uint32_t)sq, 16);
      sq += (int)xshfl((uint32_t)sq, 32);
      cnr[t] = sq;
      if (g == 0) cidL[16 * t + col] = cl[t];
    }
    __syncthreads();
    const bool mvalid = kvalid(cidL[ln]);
    const uint32_t nv = (uint32_t)popc(ballot(mvalid));
    // lane ln holds slot ln's |c'|^2 in cnr[ln >> 4] (every group has it)
    int mycnr = cnr[0];
#pragma unroll
    for (int t = 1; t < NT; t++) mycnr = (ln >> 4) == t ? cnr[t] : mycnr;
    ckeyL[ln] = -(mvalid ? (mycnr << 6) | ln : kSlotNone);
    __syncthreads();
    // slot of each neighbour in C_i (binary search over the ascending ids)
#pragma unroll
    for (int u = 0; u < NPL; u++) {
      uint32_t lo = 0, hi = nv;
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (cidL[mid] < xv[u]) lo = mid + 1;
        else hi = mid;
      }
      rxL[ln + 64 * u] = (xv[u] != kInvalid && lo < nv && cidL[lo] == xv[u]) ? lo : ~0u;
    }
    __syncthreads();
    if (j == 0) rows += (unsigned long long)nv;
    const uint32_t rb0 = repair_base(a, d0, rbase, e0);
    for (int s = 0; 16 * s < cnt; s++) {
      // neighbours 16s .. 16s+15 as the B operand
      const uint32_t xs = xsn;
      const bool xsok = xs != kInvalid;
      const uint32_t rx = rxL[16 * s + col];
      v4i X[NK];
#pragma unroll
      for (int kk = 0; kk < NK; kk++) X[kk] = to_i8x16(Xn[kk]);
      if (16 * (s + 1) < cnt) load_step(s + 1);
      int nx = 0;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) nx = sq_i8x16(X[kk], nx);
      nx += (int)xshfl((uint32_t)nx, 16);
      nx += (int)xshfl((uint32_t)nx, 32);
      const uint32_t nx64 = (uint32_t)nx << 6;
      // x's own value (key rx) when x is in C_i; otherwise a value no
      // candidate takes (key ~0)
      const int32_t rxn = (int32_t)(nx64 - rx);
      constexpr int L = K + 1;
      int32_t l[L];
#pragma unroll
      for (int k = 0; k < L; k++) l[k] = kNone;
      // two tiles' products at a time
#pragma unroll
      for (int t0 = 0; t0 < NT; t0 += 2) {
        v4i acc[2];
#pragma unroll
        for (int u = 0; u < 2; u++) {
          acc[u] = v4i{0, 0, 0, 0};
#pragma unroll
          for (int kk = 0; kk < NK; kk++) acc[u] = mfma_i8(Ct[t0 + u][kk], X[kk], acc[u]);
        }
#pragma unroll
        for (int u = 0; u < 2; u++) {
          const int4 ck = *reinterpret_cast<const int4 *>(&ckeyL[16 * (t0 + u) + 4 * g]);
          const int32_t cks[4] = {ck.x, ck.y, ck.z, ck.w};
#pragma unroll
          for (int ii = 0; ii < 4; ii++) {
            const int32_t n = (int32_t)((uint32_t)acc[u][ii] << 7) + cks[ii];
            kl_insert_max<L>(l, n);
          }
        }
      }
#pragma unroll
      for (int o = 16; o < 64; o <<= 1) {
        int32_t ot[L];
#pragma unroll
        for (int k = 0; k < L; k++) ot[k] = (int32_t)xshfl((uint32_t)l[k], o);
        kl_merge_max<L>(l, ot);
      }
      // without x: the entries from x's value on move up by one
      bool has_x = false;
#pragma unroll
      for (int k = 0; k < L; k++) has_x |= l[k] == rxn;
#pragma unroll
      for (int k = 0; k < K; k++) l[k] = (has_x && l[k] <= rxn) ? l[k + 1] : l[k];
      if (g == 0 && xsok) evals += nv - (rx != ~0u ? 1u : 0u);
      // records of neighbour 16s + col (at most c + 1 <= K + 1): lane g
      // stages entries g, g + 4, ...
      const int e = 16 * s + col;
      if (e < cnt) {
        const uint32_t pos = e0 + (uint32_t)e;
        const bool inbound = pos < d0.w;
        const uint32_t nrec = inbound ? c + 1 : c;
        const uint32_t base = repair_base(a, d0, rbase, pos) - rb0;
#pragma unroll
        for (int kq = 0; kq < (K + 4) / 4; kq++) {
          const uint32_t k = (uint32_t)(g + 4 * kq);
          if (k >= nrec) break;
          int32_t n = kNone;
#pragma unroll
          for (int kk = 0; kk < K; kk++)
            if ((uint32_t)kk == k) n = l[kk];
          const uint32_t key = nx64 - (uint32_t)n;
          const bool v = key < kKeyValid;
          const uint32_t yi = v ? cidL[key & 63u] : kInvalid;
          const float yd = v ? (float)(key >> 6) : 0.0f;
          uint32_t rt = kInvalid, rs = kInvalid;
          float rd = 0.0f;
          if (xsok && inbound) {
            const bool marker = k == c;
            rt = xs;
            rs = marker ? kInvalid : yi;
            rd = marker ? 0.0f : yd;
            recs++;
          } else if (xsok) {
            rt = yi;
            rs = v ? xs : kInvalid;
            rd = yd;
            recs += v ? 1u : 0u;
          }
          rtL[base + k] = rt;
          rsL[base + k] = rs;
          rdL[base + k] = rd;
        }
      }
    }
    __syncthreads();
    // the chunk's records, written out in order
    const uint32_t nr = repair_base(a, d0, rbase, e0 + (uint32_t)cnt) - rb0;
    for (uint32_t o = (uint32_t)ln; o < nr; o += 64) {
      a.rec_t[rb0 + o] = rtL[o];
      a.rec_s[rb0 + o] = rsL[o];
      a.rec_d[rb0 + o] = rdL[o];
    }
    __syncthreads();
  }
  unsigned long long ev = evals, rc = recs;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    ev += __shfl_xor(ev, o, 64);
    rc += __shfl_xor(rc, o, 64);
  }
  if (ln == 0 && (ev | rc | rows)) {
    stat_add(a.ds, kStRecords, rc);
    stat_add(a.ds, kStRepEvals, ev);
    stat_add(a.ds, kStRepRows, rows);
    stat_add(a.ds, kStRepRecs, rc);
  }
}

// ---------------------------------------------------------------------------
// fp32 repair over the same work chunks: one lane per neighbour.  C_i is
// taken 16 candidates at a time; their rows pass through LDS in slices of 64
// floats (each value read once per slice, by every lane at the same address)
// while each lane streams its own neighbour's row in pieces of 16 floats and
// accumulates the 16 distances in fp64, in dimension order -- the summation
// the oracle performs, so the rounded distances are identical.  Each lane
// keeps its neighbour's K smallest (distance, id) keys; the records and their
// offsets are those of the uint8 form.
// Sorted list of the K smallest 64-bit (distance, id) keys.
template <int K>
__device__ __forceinline__ void kl_insert64(uint64_t (&l)[K], uint64_t k) {
#pragma unroll
  for (int j = 0; j < K; j++) {
    const uint64_t lo = k < l[j] ? k : l[j];
    k = k < l[j] ? l[j] : k;
    l[j] = lo;
  }
}

template <int KIND, int K>
__global__ __launch_bounds__(64) void k_repair_vec(RepairArgs a) {
  constexpr int GC = 16, SL = 64;
  __shared__ double cs[GC][SL];  // candidate slices, widened to fp64 once when staged
  __shared__ uint32_t cidL[64];
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const uint32_t c = a.c;
  const int kr = (int)a.kr;
  const int nfl = P.nch * 4;  // floats per padded row (padding is zero)
  if ((size_t)a.rofs[a.n] > a.rcap) return;  // the host grows the buffers and launches again
  const uint32_t total = a.coff[a.n];
  unsigned long long evals = 0, rows = 0, recs = 0;
  for (uint32_t q = blockIdx.x; q < total; q += gridDim.x) {
    const uint4 d0 = a.cdesc[2 * (size_t)q], d1 = a.cdesc[2 * (size_t)q + 1];
    const uint32_t i = d0.x, p = d0.y, rbase = d1.x, j = d1.w;
    const int cnt = (int)d1.z;
    const uint32_t pos = d1.y + (uint32_t)ln;  // this lane's position
    const bool inbound = pos < d0.w;
    const uint32_t x = ln < cnt ? repair_nbr(a, d0, pos) : kInvalid;
    const bool xok = x != kInvalid;
    cidL[ln] = ln < kr ? a.ci[(size_t)i * kr + ln] : kInvalid;
    __syncthreads();
    if (j == 0) rows += (unsigned long long)popc(ballot(ln < kr && kvalid(cidL[ln])));
    rows += (unsigned long long)popc(ballot(xok));
    const float *xrow = reinterpret_cast<const float *>(P.vecs + (size_t)(xok ? x : p) * P.stride);
    uint64_t l[K];
#pragma unroll
    for (int k = 0; k < K; k++) l[k] = ~0ull;
    for (int g0 = 0; g0 < kr; g0 += GC) {
      double acc[GC];
#pragma unroll
      for (int k = 0; k < GC; k++) acc[k] = 0.0;
      for (int d0 = 0; d0 < nfl; d0 += SL) {
        // candidates g0 .. g0+15, floats d0 .. d0+63 (zeros past the row or
        // for missing candidates), 16 floats per lane
        __syncthreads();
        {
          const int cand = ln >> 2, part = ln & 3;
          const int e = g0 + cand;
          const uint32_t cv = e < kr ? cidL[e] : kInvalid;
          const float *crow = reinterpret_cast<const float *>(P.vecs + (size_t)(kvalid(cv) ? cv : p) * P.stride);
          // all four loads issued before any is used (addresses clamped into
          // the row, the values past it replaced by zeros afterwards)
          uint4 v4[4];
#pragma unroll
          for (int h = 0; h < 4; h++) {
            const int f = d0 + 16 * part + 4 * h;
            v4[h] = *reinterpret_cast<const uint4 *>(crow + (f < nfl ? f : 0));
          }
#pragma unroll
          for (int h = 0; h < 4; h++) {
            const int f = d0 + 16 * part + 4 * h;
            const uint4 v = (kvalid(cv) && f < nfl) ? v4[h] : make_uint4(0, 0, 0, 0);
            double2 *dst = reinterpret_cast<double2 *>(&cs[cand][16 * part + 4 * h]);
            dst[0] = make_double2((double)__uint_as_float(v.x), (double)__uint_as_float(v.y));
            dst[1] = make_double2((double)__uint_as_float(v.z), (double)__uint_as_float(v.w));
          }
        }
        __syncthreads();
        for (int pc = 0; pc < SL && d0 + pc < nfl; pc += 16) {
          float xv[16];
          uint4 v4[4];
#pragma unroll
          for (int h = 0; h < 4; h++) {
            const int f = d0 + pc + 4 * h;  // rows hold nfl floats, a multiple of 4
            v4[h] = *reinterpret_cast<const uint4 *>(xrow + (f < nfl ? f : 0));
          }
#pragma unroll
          for (int h = 0; h < 4; h++) {
            const int f = d0 + pc + 4 * h;
            const uint4 v = f < nfl ? v4[h] : make_uint4(0, 0, 0, 0);
            xv[4 * h + 0] = __uint_as_float(v.x);
            xv[4 * h + 1] = __uint_as_float(v.y);
            xv[4 * h + 2] = __uint_as_float(v.z);
            xv[4 * h + 3] = __uint_as_float(v.w);
          }
#pragma unroll
          for (int k = 0; k < GC; k++)
#pragma unroll
            for (int t = 0; t < 16; t++) {
              if (KIND == kF32L2) {
                const double df = cs[k][pc + t] - (double)xv[t];
                acc[k] = __builtin_fma(df, df, acc[k]);
              } else {
                acc[k] = __builtin_fma((double)xv[t], cs[k][pc + t], acc[k]);
              }
            }
        }
      }
#pragma unroll
      for (int k = 0; k < GC; k++) {
        const int e = g0 + k;
        const uint32_t cv = e < kr ? cidL[e] : kInvalid;
        const bool ok = xok && kvalid(cv) && cv != x;
        evals += ok ? 1u : 0u;
        const float dk = finalize<KIND>(acc[k]);
        kl_insert64<K>(l, ok ? key64(dk, cv) : ~0ull);
      }
    }
    if (ln < cnt) {
      const uint32_t nrec = inbound ? c + 1 : c;
      const uint32_t base = repair_base(a, d0, rbase, pos);
      for (uint32_t k = 0; k < nrec; k++) {
        uint64_t key = ~0ull;
#pragma unroll
        for (int kk = 0; kk < K; kk++)
          if ((uint32_t)kk == k) key = l[kk];
        const bool v = key != ~0ull;
        const uint32_t yi = v ? (uint32_t)key : kInvalid;
        const float yd = v ? unsortable((uint32_t)(key >> 32)) : 0.0f;
        if (!xok) {
          a.rec_t[base + k] = kInvalid;
        } else if (inbound) {
          const bool marker = k == c;
          a.rec_t[base + k] = x;
          a.rec_s[base + k] = marker ? kInvalid : yi;
          a.rec_d[base + k] = marker ? 0.0f : yd;
          recs++;
        } else {
          a.rec_t[base + k] = yi;
          a.rec_s[base + k] = v ? x : kInvalid;
          a.rec_d[base + k] = yd;
          recs += v ? 1u : 0u;
        }
      }
    }
    __syncthreads();
  }
  unsigned long long ev = evals, rc = recs;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    ev += __shfl_xor(ev, o, 64);
    rc += __shfl_xor(rc, o, 64);
  }
  if (ln == 0 && (ev | rc | rows)) {
    stat_add(a.ds, kStRecords, rc);
    stat_add(a.ds, kStRepEvals, ev);
    stat_add(a.ds, kStRepRows, rows);
    stat_add(a.ds, kStRepRecs, rc);
  }
}

// Chunked forms (R <= 64, k_repair <= 64, c <= 4): the matrix-core form for
// uint8 rows of 64 or 128 bytes, the lane-per-neighbour form for fp32 rows;
// every other configuration takes one wave per deleted node.
bool repair_chunked(int kind, const PoolView &p, uint32_t kr, uint32_t c) {
  if (kr > 64 || c > 4 || p.R > 64) return false;
  if (kind == kU8L2) return p.nch == 4 || p.nch == 8;
  return kind == kF32L2 || kind == kF32IP;
}
// Positions per work chunk: two per lane on the matrix-core form (a node's
// in-neighbours and out-slots, about 2R, usually fit one chunk), one per lane
// on the fp32 form.
constexpr int kRepairNpl = 2;
uint32_t repair_chunk_width(int kind, const PoolView &p, uint32_t kr, uint32_t c) {
  return (kind == kU8L2 && repair_chunked(kind, p, kr, c)) ? 64u * kRepairNpl : 64u;
}

hipError_t launch_repair(int kind, int vc, const RepairArgs &a, uint32_t grid, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  if (kind == kU8L2 && repair_chunked(kind, a.pool, a.kr, a.c)) {
    // persistent waves over the chunk descriptors, twice the resident
    // workgroups: the second half starts as the first ones finish, which
    // evens out the work per wave (chunks differ in length)
    if (a.cw != 64u * kRepairNpl) return hipErrorInvalidValue;
    static const uint32_t r22 = resident_blocks((const void *)k_repair_mfma<2, 2, kRepairNpl>);
    static const uint32_t r24 = resident_blocks((const void *)k_repair_mfma<2, 4, kRepairNpl>);
    static const uint32_t r12 = resident_blocks((const void *)k_repair_mfma<1, 2, kRepairNpl>);
    static const uint32_t r14 = resident_blocks((const void *)k_repair_mfma<1, 4, kRepairNpl>);
    if (a.pool.nch == 8) {
      if (a.c <= 2)
        hipLaunchKernelGGL((k_repair_mfma<2, 2, kRepairNpl>), dim3(clamp_resident(grid, 2 * r22)), dim3(64), 0, st, a);
      else
        hipLaunchKernelGGL((k_repair_mfma<2, 4, kRepairNpl>), dim3(clamp_resident(grid, 2 * r24)), dim3(64), 0, st, a);
    } else {
      if (a.c <= 2)
        hipLaunchKernelGGL((k_repair_mfma<1, 2, kRepairNpl>), dim3(clamp_resident(grid, 2 * r12)), dim3(64), 0, st, a);
      else
        hipLaunchKernelGGL((k_repair_mfma<1, 4, kRepairNpl>), dim3(clamp_resident(grid, 2 * r14)), dim3(64), 0, st, a);
    }
    return hipGetLastError();
  }
  if (repair_chunked(kind, a.pool, a.kr, a.c)) {
    if (a.cw != 64u) return hipErrorInvalidValue;
    if (kind == kF32L2) {
      if (a.c <= 2) hipLaunchKernelGGL((k_repair_vec<kF32L2, 2>), dim3(grid), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_repair_vec<kF32L2, 4>), dim3(grid), dim3(64), 0, st, a);
    } else {
      if (a.c <= 2) hipLaunchKernelGGL((k_repair_vec<kF32IP, 2>), dim3(grid), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_repair_vec<kF32IP, 4>), dim3(grid), dim3(64), 0, st, a);
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
