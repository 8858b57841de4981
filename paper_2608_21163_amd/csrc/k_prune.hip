// k_prune.hip -- GrANDRobustPrune (Alg. 4) executed by one wavefront, the
// forward prune of new nodes (Alg. 5, second loop) and the rebuild of every
// dirty node (Alg. 5 and Alg. 6, last loops), one wavefront per node.
//
// When the candidate rows fit, a node's candidates and its own row are
// staged into LDS once (all gathers in flight together), and every distance
// of the prune -- D_p and the pairwise distances of the selection loop -- is
// evaluated from LDS.  LDS slots are assigned in ascending id order, so
// ordering keys by (distance, slot) breaks ties exactly as (distance, id).
// Rows too long for LDS are read from global memory (L2) instead.
#include "dispatch.h"

namespace gr {

// GrANDRobustPrune of node p over candidates addressed as rows of `vecs`.
// Candidates (any order, invalid padded) come with their distances D_p.
// They are sorted by (D_p, address); repeats and p itself are dropped.  The
// first valid candidate p* is selected; selection stops at R; otherwise the
// distance from p* to every later valid candidate p' is evaluated by the
// wave (pivot p* held in registers, candidate rows LPV lanes per row) and p'
// is invalidated when coef * Dist(p*, p') <= D_p[p'] (coef is alpha, or
// alpha^2 for the Euclidean reading, compared in fp64).
// On return lane t < nsel holds the t-th selection (address, distance).
template <int KIND, int LPV, int CPL, int NR>
__device__ int wave_prune(const uint8_t *vecs, size_t stride, int nch, uint32_t p, uint32_t R, double coef,
                          float (&cd)[NR], uint32_t (&ci)[NR], uint32_t *lids, float *ldist, uint32_t &sel_id,
                          float &sel_d, unsigned long long &evals) {
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
    load_slice<KIND, LPV, CPL>(s, vecs + (size_t)pid * stride, nch);
    __syncthreads();
    wave_dists<KIND, LPV, CPL>(s, vecs, stride, nch, lids, ldist, cnt);
    __syncthreads();
    evals += (unsigned long long)cnt;
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (valid[r] && coef * (double)ldist[cidx[r]] <= (double)cd[r]) valid[r] = false;
    __syncthreads();
  }
  return nsel;
}

// Bytes per LDS row: the pool stride plus one chunk, which staggers rows
// across LDS banks.
__host__ __device__ constexpr size_t lds_stride(size_t stride) { return stride + 16; }

// Copies rows ids[0..m) and row `extra` (slot m) of the pool into LDS slots
// 0..m, LPV lanes per row, with the gathers of RIF row groups in flight.
template <int LPV, int CPL>
__device__ __forceinline__ void stage_rows(const PoolView &P, const uint32_t *ids, int m, uint32_t extra,
                                           uint8_t *vbuf) {
  constexpr int G = 64 / LPV;
  constexpr int RIF = CPL >= 8 ? 1 : 8 / CPL;
  const int ln = lane(), grp = ln / LPV, sub = ln % LPV;
  const size_t ls = lds_stride(P.stride);
  for (int base = 0; base <= m; base += G * RIF) {
    uint4 b[RIF][CPL];
#pragma unroll
    for (int rr = 0; rr < RIF; rr++) {
      const int e = base + rr * G + grp;
      const uint32_t id = e < m ? ids[e] : extra;
      const uint8_t *row = P.vecs + (size_t)id * P.stride;
#pragma unroll
      for (int k = 0; k < CPL; k++) {
        const int ch = sub + k * LPV;
        b[rr][k] = (e <= m && ch < P.nch) ? ld16(row + (size_t)ch * 16) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int rr = 0; rr < RIF; rr++) {
      const int e = base + rr * G + grp;
#pragma unroll
      for (int k = 0; k < CPL; k++) {
        const int ch = sub + k * LPV;
        if (e <= m && ch < P.nch) *reinterpret_cast<uint4 *>(vbuf + (size_t)e * ls + (size_t)ch * 16) = b[rr][k];
      }
    }
  }
}

// GrANDRobustPrune of node p over the m distinct candidate ids in slot_id
// (LDS, any order), with every vector in LDS: the ids are sorted (slot =
// rank of the id), the rows of the candidates and of p are staged, D_p is
// evaluated from LDS (bit-identical to the distance evaluated during the
// search or carried by the records: the arithmetic and lane layout are the
// same), and the selection loop runs on LDS rows.  Lane t < nsel returns the
// t-th selected id and its distance.
template <int KIND, int LPV, int CPL, int NC>
__device__ int prune_staged(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, uint32_t *slot_id,
                            uint8_t *vbuf, uint32_t *lids, float *ldist, uint32_t &sel_id, float &sel_d,
                            unsigned long long &evals) {
  const int ln = lane();
  const size_t ls = lds_stride(P.stride);
  float kd[NC];
  uint32_t kid[NC];
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    kd[r] = e < m ? 0.0f : finf();
    kid[r] = e < m ? slot_id[e] : kInvalid;
  }
  wave_sort<NC>(kd, kid);
  __syncthreads();
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    if (e < m) {
      slot_id[e] = kid[r];
      lids[e] = (uint32_t)e;
    }
  }
  __syncthreads();
  stage_rows<LPV, CPL>(P, slot_id, m, p, vbuf);
  __syncthreads();
  Slice<KIND, LPV, CPL> su;
  load_slice<KIND, LPV, CPL>(su, vbuf + (size_t)m * ls, P.nch);
  wave_dists<KIND, LPV, CPL>(su, vbuf, ls, P.nch, lids, ldist, m);
  __syncthreads();
  evals += (unsigned long long)m;
  float cd[NC];
  uint32_t ci[NC];
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    cd[r] = e < m ? ldist[e] : finf();
    ci[r] = e < m ? (uint32_t)e : kInvalid;
  }
  __syncthreads();
  uint32_t ssl;
  const int nsel = wave_prune<KIND, LPV, CPL, NC>(vbuf, ls, P.nch, kIdMask - 1, R, coef, cd, ci, lids, ldist, ssl,
                                                  sel_d, evals);
  sel_id = ln < nsel ? slot_id[ssl] : kInvalid;
  __syncthreads();
  return nsel;
}

// ---------------------------------------------------------------------------
// uint8 GrANDRobustPrune on the matrix cores.  Rows are staged in LDS as in
// prune_staged.  The pairwise distances of the candidates form a dense Gram
// matrix (m x m x dim): with y = x - 128 (byte-wise x ^ 0x80, an exact int8
// view), Dist(i, j) = |y_i|^2 + |y_j|^2 - 2 y_i.y_j exactly in int32 (L2 is
// translation invariant), so the products run on v_mfma_i32_16x16x64_i8.
// Candidates are ordered by (D_p, slot); the greedy selection walks them in
// blocks of 16 pivots: a block's distance rows to every later candidate are
// produced by MFMA into LDS (blocks without a valid pivot are skipped), then
// the block's pivots are taken in order, each invalidating later candidates
// with coef * Dist(p*, p') <= D_p[p'].  Requires dim to be a multiple of 64.
struct MfmaLds {
  uint32_t *slot_id;   // [64*NC] candidate ids, then sorted by id (slot order)
  int32_t *nrm;        // [64*NC + 1] |y|^2 per slot (slot m = the node)
  float *dpos;         // [64*NC] D_p by sorted position
  uint32_t *spos;      // [64*NC] slot by sorted position
  float *blk;          // [16][64*NC] distance rows of the current pivot block
  uint8_t *vbuf;       // [(64*NC + 1) * lds_stride] rows
};

// Dynamic LDS of the matrix-core prune for up to MP candidates:
// blk | nrm | rows.
__host__ __device__ constexpr size_t mfma_blk_bytes(int MP) { return (size_t)16 * MP * 4; }
__host__ __device__ constexpr size_t mfma_nrm_bytes(int MP) { return ((size_t)(MP + 1) * 4 + 15) / 16 * 16; }
__host__ __device__ constexpr size_t mfma_lds_bytes(size_t stride, int MP) {
  return mfma_blk_bytes(MP) + mfma_nrm_bytes(MP) + (size_t)(MP + 1) * lds_stride(stride);
}
__device__ __forceinline__ MfmaLds mfma_lds(uint8_t *dyn, uint32_t *slot_id, uint32_t *spos, float *dpos, int MP) {
  MfmaLds L;
  L.slot_id = slot_id;
  L.spos = spos;
  L.dpos = dpos;
  L.blk = reinterpret_cast<float *>(dyn);
  L.nrm = reinterpret_cast<int32_t *>(dyn + mfma_blk_bytes(MP));
  L.vbuf = dyn + mfma_blk_bytes(MP) + mfma_nrm_bytes(MP);
  return L;
}

template <int LPV, int CPL, int NC>
__device__ int prune_mfma_u8(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, const MfmaLds &L,
                             uint32_t &sel_id, float &sel_d, unsigned long long &evals) {
  constexpr int MP = 64 * NC;
  const int ln = lane();
  const size_t ls = lds_stride(P.stride);
  const int nk = P.nch / 4;  // 64-byte K chunks
  sel_id = kInvalid;
  sel_d = finf();
  if (m <= 0) return 0;
  // slots in ascending id order
  {
    float kd[NC];
    uint32_t kid[NC];
#pragma unroll
    for (int r = 0; r < NC; r++) {
      const int e = r * 64 + ln;
      kd[r] = e < m ? 0.0f : finf();
      kid[r] = e < m ? L.slot_id[e] : kInvalid;
    }
    wave_sort<NC>(kd, kid);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < NC; r++)
      if (r * 64 + ln < m) L.slot_id[r * 64 + ln] = kid[r];
    __syncthreads();
  }
  stage_rows<LPV, CPL>(P, L.slot_id, m, p, L.vbuf);
  __syncthreads();
  // |y|^2 per slot and D_p = |y_p|^2 + |y_j|^2 - 2 y_p.y_j (exact)
  const uint8_t *prow = L.vbuf + (size_t)m * ls;
  int np = 0;
  for (int c = 0; c < P.nch; c++) {
    const uint4 v = ld16(prow + (size_t)c * 16);
    const uint32_t a0 = v.x ^ 0x80808080u, a1 = v.y ^ 0x80808080u, a2 = v.z ^ 0x80808080u, a3 = v.w ^ 0x80808080u;
    np = sdot4(a0, a0, np); np = sdot4(a1, a1, np); np = sdot4(a2, a2, np); np = sdot4(a3, a3, np);
  }
  float kd[NC];
  uint32_t kid[NC];
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    kd[r] = finf();
    kid[r] = kInvalid;
    if (e < m) {
      const uint8_t *row = L.vbuf + (size_t)e * ls;
      int nn = 0, dp = 0;
      for (int c = 0; c < P.nch; c++) {
        const uint4 v = ld16(row + (size_t)c * 16), w = ld16(prow + (size_t)c * 16);
        const uint32_t a0 = v.x ^ 0x80808080u, a1 = v.y ^ 0x80808080u, a2 = v.z ^ 0x80808080u, a3 = v.w ^ 0x80808080u;
        nn = sdot4(a0, a0, nn); nn = sdot4(a1, a1, nn); nn = sdot4(a2, a2, nn); nn = sdot4(a3, a3, nn);
        dp = sdot4(a0, w.x ^ 0x80808080u, dp); dp = sdot4(a1, w.y ^ 0x80808080u, dp);
        dp = sdot4(a2, w.z ^ 0x80808080u, dp); dp = sdot4(a3, w.w ^ 0x80808080u, dp);
      }
      L.nrm[e] = nn;
      kd[r] = canon0((float)(np + nn - 2 * dp));
      kid[r] = (uint32_t)e;
    }
  }
  evals += (unsigned long long)m;
  wave_sort<NC>(kd, kid);
  bool valid[NC];
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    valid[r] = e < m;
    L.spos[e] = kid[r];
    L.dpos[e] = kd[r];
  }
  __syncthreads();
  const int nt = (m + 15) / 16;
  int nsel = 0;
  bool done = false;
  for (int b = 0; b < nt && !done; b++) {
    // Sorted positions 16c .. 16c+15 (tile c) live in register row c/4,
    // lanes 16*(c%4) ..; tmask marks the tiles that still hold a valid
    // candidate, vb the valid pivots of block b.
    uint64_t vb = 0;
    uint32_t tmask = 0;
#pragma unroll
    for (int r = 0; r < NC; r++) {
      const uint64_t vm = ballot(valid[r]);
#pragma unroll
      for (int q = 0; q < 4; q++)
        if ((vm >> (16 * q)) & 0xFFFFull) tmask |= 1u << (4 * r + q);
      if (r == b / 4) vb = (vm >> (16 * (b % 4))) & 0xFFFFull;
    }
    if (!vb) continue;
    // distance rows of the block's candidates to every candidate of tile c >= b
    const int arow = 16 * b + (ln & 15);
    const uint32_t aslot = L.spos[arow < m ? arow : 0];
    const int kb = ln >> 4;
    for (int c = b; c < nt; c++) {
      if (!((tmask >> c) & 1u)) continue;
      const int bcol = 16 * c + (ln & 15);
      const uint32_t bslot = L.spos[bcol < m ? bcol : 0];
      v4i acc = {0, 0, 0, 0};
      for (int kk = 0; kk < nk; kk++) {
        const uint4 av = ld16(L.vbuf + (size_t)aslot * ls + (size_t)kk * 64 + (size_t)kb * 16);
        const uint4 bv = ld16(L.vbuf + (size_t)bslot * ls + (size_t)kk * 64 + (size_t)kb * 16);
        v4i A, B;
        A[0] = (int)(av.x ^ 0x80808080u); A[1] = (int)(av.y ^ 0x80808080u);
        A[2] = (int)(av.z ^ 0x80808080u); A[3] = (int)(av.w ^ 0x80808080u);
        B[0] = (int)(bv.x ^ 0x80808080u); B[1] = (int)(bv.y ^ 0x80808080u);
        B[2] = (int)(bv.z ^ 0x80808080u); B[3] = (int)(bv.w ^ 0x80808080u);
        acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(A, B, acc, 0, 0, 0);
      }
      const int ncol = L.nrm[bslot];
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const int rr = 4 * (ln >> 4) + i;
        const int rpos = 16 * b + rr;
        const int rn = L.nrm[L.spos[rpos < m ? rpos : 0]];
        L.blk[rr * MP + bcol] = canon0((float)(rn + ncol - 2 * acc[i]));
      }
    }
    evals += (unsigned long long)256 * __popc(tmask >> b);
    __syncthreads();
    for (int t = 0; t < 16; t++) {
      const int pos = 16 * b + t;
      if (pos >= m) break;
      if (!((vb >> t) & 1)) continue;
      // recheck: earlier pivots of this block may have invalidated it
      uint64_t still = 0;
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const uint64_t vm = ballot(valid[r]);
        if (r == b / 4) still = (vm >> (16 * (b % 4) + t)) & 1ull;
      }
      if (!still) continue;
      if (ln == nsel) { sel_id = L.slot_id[L.spos[pos]]; sel_d = L.dpos[pos]; }
      nsel++;
#pragma unroll
      for (int r = 0; r < NC; r++)
        if (r * 64 + ln == pos) valid[r] = false;
      if (nsel == (int)R) { done = true; break; }
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const int j = r * 64 + ln;
        if (valid[r] && j > pos && coef * (double)L.blk[t * MP + j] <= (double)L.dpos[j]) valid[r] = false;
      }
    }
    __syncthreads();
  }
  return nsel;
}

// ---------------------------------------------------------------------------
// uint8 GrANDRobustPrune with the candidate rows held in registers, for
// rows of 4*NK chunks (dim = 64*NK) and at most 64*NC candidates.  Same
// arithmetic as prune_mfma_u8 (exact int32 distances through int8 MFMA on
// x ^ 0x80), but nothing is staged in LDS, so many waves fit per CU:
//  1. the rows of the candidates (list order) and of p are loaded in the
//     MFMA operand layout (tile t = candidates 16t..16t+15; lane l holds
//     bytes 64kk + 16(l/16) .. +15 of candidate 16t + l%16), giving |y|^2 and
//     D_p exactly;
//  2. candidates are sorted by (D_p, id) and the rows reloaded in that order;
//  3. the greedy selection walks blocks of 16 pivots.  For a block b and a
//     tile c >= b one MFMA tile gives Dist(pivot, candidate) for 16 x 16
//     pairs; each lane turns the 4 values it holds into "kill" bits
//     (coef * Dist <= D_p[candidate]) and the bits of one candidate column
//     are OR-ed across the 4 lane groups into a 16-bit mask over the block's
//     pivots.  The block's pivots are resolved in order on the diagonal
//     tile's masks (scalar loop), and later candidates are invalidated when
//     their mask meets the set of selected pivots.
// cl[0..m): distinct candidate ids other than p (LDS).  spos/dpos: LDS
// scratch of 64*NC entries.  Lane t < nsel returns the t-th selection.
template <int NK, int NC>
__device__ int prune_mfma_reg(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, const uint32_t *cl,
                              uint32_t *spos, float *dpos, uint32_t &sel_id, float &sel_d,
                              unsigned long long &evals) {
  constexpr int T = 4 * NC;
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  sel_id = kInvalid;
  sel_d = finf();
  if (m <= 0) return 0;
  const int nt = (m + 15) >> 4;
  const size_t goff = (size_t)g * 16;
  v4i B[T][NK];
  int nrm[T];
  auto load_tile = [&](int t, uint32_t id) {
    const uint8_t *row = P.vecs + (size_t)id * P.stride + goff;
    int s = 0;
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      const uint4 v = ld16(row + (size_t)kk * 64);
      B[t][kk][0] = (int)(v.x ^ 0x80808080u);
      B[t][kk][1] = (int)(v.y ^ 0x80808080u);
      B[t][kk][2] = (int)(v.z ^ 0x80808080u);
      B[t][kk][3] = (int)(v.w ^ 0x80808080u);
#pragma unroll
      for (int w = 0; w < 4; w++) s = sdot4((uint32_t)B[t][kk][w], (uint32_t)B[t][kk][w], s);
    }
    s += (int)xshfl((uint32_t)s, 16);
    s += (int)xshfl((uint32_t)s, 32);
    nrm[t] = s;
  };
  // 1. rows in list order, the node's row, D_p
#pragma unroll
  for (int t = 0; t < T; t++)
    if (t < nt) {
      const int e = 16 * t + col;
      load_tile(t, e < m ? cl[e] : p);
    }
  v4i A[NK];
  int np = 0;
  {
    const uint8_t *row = P.vecs + (size_t)p * P.stride + goff;
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      const uint4 v = ld16(row + (size_t)kk * 64);
      A[kk][0] = (int)(v.x ^ 0x80808080u);
      A[kk][1] = (int)(v.y ^ 0x80808080u);
      A[kk][2] = (int)(v.z ^ 0x80808080u);
      A[kk][3] = (int)(v.w ^ 0x80808080u);
#pragma unroll
      for (int w = 0; w < 4; w++) np = sdot4((uint32_t)A[kk][w], (uint32_t)A[kk][w], np);
    }
    np += (int)xshfl((uint32_t)np, 16);
    np += (int)xshfl((uint32_t)np, 32);
  }
  float dt[T];
#pragma unroll
  for (int t = 0; t < T; t++) {
    dt[t] = finf();
    if (t < nt) {
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < NK; kk++) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(A[kk], B[t][kk], acc, 0, 0, 0);
      dt[t] = canon0((float)(np + nrm[t] - 2 * acc[0]));
    }
  }
  evals += (unsigned long long)m;
  // 2. sort by (D_p, id): position e = 16t + col of the list sits in
  //    register row t/4 at lane 16(t%4) + col
  float kd[NC];
  uint32_t kid[NC];
  bool valid[NC];
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    float d = dt[4 * r];
#pragma unroll
    for (int q = 1; q < 4; q++) d = g == q ? dt[4 * r + q] : d;
    kd[r] = e < m ? d : finf();
    kid[r] = e < m ? cl[e] : kInvalid;
  }
  wave_sort<NC>(kd, kid);
#pragma unroll
  for (int r = 0; r < NC; r++) {
    const int e = r * 64 + ln;
    valid[r] = e < m;
    spos[e] = kid[r];
    dpos[e] = kd[r];
  }
  __syncthreads();
  float dcol[T];
#pragma unroll
  for (int t = 0; t < T; t++) {
    dcol[t] = finf();
    if (t < nt) {
      const int e = 16 * t + col;
      load_tile(t, e < m ? spos[e] : p);
      dcol[t] = dpos[e];
    }
  }
  // 3. greedy selection over pivot blocks
  int nsel = 0;
  bool done = false;
#pragma unroll
  for (int b = 0; b < T; b++) {
    if (done || b >= nt) continue;
    const uint32_t vb = (uint32_t)(ballot(valid[b >> 2]) >> (16 * (b & 3))) & 0xFFFFu;
    if (!vb) continue;
    int rn[4];
#pragma unroll
    for (int i = 0; i < 4; i++) rn[i] = __shfl(nrm[b], 4 * g + i, 64);
    auto kill_mask = [&](int c) -> uint32_t {
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < NK; kk++) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(B[b][kk], B[c][kk], acc, 0, 0, 0);
      uint32_t km = 0;
#pragma unroll
      for (int i = 0; i < 4; i++) {
        const float d = canon0((float)(rn[i] + nrm[c] - 2 * acc[i]));
        km |= (coef * (double)d <= (double)dcol[c]) ? (1u << (4 * g + i)) : 0u;
      }
      km |= xshfl(km, 16);
      km |= xshfl(km, 32);
      return km;
    };
    const uint32_t kmd = kill_mask(b);
    const uint32_t bid = spos[16 * b + col];
    const float bd = dpos[16 * b + col];
    uint32_t S = 0, alive = vb;
    while (alive) {
      const int t = __ffs(alive) - 1;
      alive &= alive - 1;
      S |= 1u << t;
      const uint32_t sid = rdlane(bid, t);
      const float sd = rdlane(bd, t);
      if (ln == nsel) { sel_id = sid; sel_d = sd; }
      nsel++;
      if (nsel == (int)R) { done = true; break; }
      alive &= ~((uint32_t)ballot(g == 0 && ((kmd >> t) & 1u)) & 0xFFFFu);
    }
    evals += 256;
    if (done) continue;
#pragma unroll
    for (int c = b + 1; c < T; c++) {
      if (c >= nt) continue;
      if (!((ballot(valid[c >> 2]) >> (16 * (c & 3))) & 0xFFFFull)) continue;
      const uint32_t km = kill_mask(c);
      evals += 256;
      if (g == (c & 3) && (km & S)) valid[c >> 2] = false;
    }
  }
  __syncthreads();
  return nsel;
}

// Forward lists of new nodes: GrANDRobustPrune(p_i, V_i \ {p_i}, D_{p_i}),
// written to p_i's row (each new node owns its row), and the reverse-edge
// records (u, p_i, D_{p_i}[u]) for every selected u.
// MODE: kGlobal (rows read from global memory), kStaged (rows staged in
// LDS), kMfma (uint8 rows staged in LDS, pairwise distances on MFMA).
// kMfmaReg (uint8 rows of 64*NK bytes, candidate rows in registers).
enum { kGlobal = 0, kStaged = 1, kMfma = 2, kMfmaReg = 3 };

template <int KIND, int LPV, int CPL, int NR, int MODE>
__global__ __launch_bounds__(64) void k_fwd_prune(FwdPruneArgs a) {
  extern __shared__ __align__(16) uint8_t vbuf[];
  __shared__ uint32_t slot_id[64 * NR];
  __shared__ uint32_t lids[64 * NR];
  __shared__ float ldist[64 * NR];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t nv = a.v_n[i];
  unsigned long long evals = 0;
  uint32_t sid;
  float sdist;
  int nsel;
  if (MODE != kGlobal) {
    // V_i holds distinct ids other than p_i
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint32_t e = r * 64 + ln;
      if (e < nv) slot_id[e] = a.v_ids[(size_t)i * a.v_stride + e];
    }
    __syncthreads();
    if constexpr (MODE == kMfma)
      nsel = prune_mfma_u8<LPV, CPL, NR>(P, p, (int)nv, P.R, a.coef, mfma_lds(vbuf, slot_id, lids, ldist, 64 * NR),
                                         sid, sdist, evals);
    else
      nsel = prune_staged<KIND, LPV, CPL, NR>(P, p, (int)nv, P.R, a.coef, slot_id, vbuf, lids, ldist, sid, sdist,
                                              evals);
  } else {
    float cd[NR];
    uint32_t ci[NR];
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint32_t e = r * 64 + ln;
      const bool in = e < nv;
      cd[r] = in ? a.v_d[(size_t)i * a.v_stride + e] : finf();
      ci[r] = in ? a.v_ids[(size_t)i * a.v_stride + e] : kInvalid;
    }
    nsel = wave_prune<KIND, LPV, CPL, NR>(P.vecs, P.stride, P.nch, p, P.R, a.coef, cd, ci, lids, ldist, sid, sdist,
                                          evals);
  }
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
// entries in slot order, then new sources in record order); otherwise
// GrANDRobustPrune(u, C, D_u) is installed.  One owner per dirty node, so
// rows are written without locks.
template <int KIND, int LPV, int CPL, int NP, int NC, int MODE, int NK = 0>
__global__ __launch_bounds__(64) void k_rebuild(RebuildArgs a) {
  extern __shared__ __align__(16) uint8_t vbuf[];
  __shared__ uint32_t rowL[64];
  __shared__ uint32_t slot_id[64 * NC];
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
      wave_merge_new_fast<NP>(sd, si, dv, sv, (int)a.P);
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
    uint32_t *cl = MODE != kGlobal ? slot_id : lids;
    if (keep) cl[mbcnt(km)] = rv;
#pragma unroll
    for (int r = 0; r < NP; r++)
      if (isnew[r]) {
        cl[kr + npos[r]] = si[r];
        if (MODE == kGlobal) ldist[kr + npos[r]] = sd[r];
      }
    __syncthreads();
    if (m <= (int)R) {
      if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < m ? cl[ln] : kInvalid;
      if (ln == 0) P.deg[u] = (uint32_t)m;
    } else {
      uint32_t sid;
      float sdist;
      int nsel;
      if constexpr (MODE == kMfmaReg) {
        nsel = prune_mfma_reg<NK, NC>(P, u, m, R, a.coef, slot_id, lids, ldist, sid, sdist, evals);
      } else if constexpr (MODE == kMfma) {
        nsel = prune_mfma_u8<LPV, CPL, NC>(P, u, m, R, a.coef, mfma_lds(vbuf, slot_id, lids, ldist, 64 * NC), sid,
                                           sdist, evals);
      } else if constexpr (MODE == kStaged) {
        nsel = prune_staged<KIND, LPV, CPL, NC>(P, u, m, R, a.coef, slot_id, vbuf, lids, ldist, sid, sdist, evals);
      } else {
        // D_u of kept entries from global rows; new entries carry theirs
        Slice<KIND, LPV, CPL> s;
        load_slice<KIND, LPV, CPL>(s, P.vecs + (size_t)u * P.stride, P.nch);
        wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, lids, ldist, kr);
        evals += (unsigned long long)kr;
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
        nsel = wave_prune<KIND, LPV, CPL, NC>(P.vecs, P.stride, P.nch, u, R, a.coef, cd, ci, lids, ldist, sid, sdist,
                                              evals);
      }
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

// LDS bytes for staging `rows` candidate rows plus the node's own row.
static size_t staged_bytes(size_t stride, uint32_t rows) { return (size_t)(rows + 1) * lds_stride(stride); }
constexpr size_t kMaxStagedLds = 64 * 1024;

// The matrix-core prune applies to uint8 rows whose chunk count is a
// multiple of 4 (dim a multiple of 64), i.e. whole 64-byte MFMA K steps.
static bool mfma_ok(int kind, const PoolView &P) { return kind == kU8L2 && P.nch % 4 == 0; }

hipError_t launch_fwd_prune(int kind, int vc, uint32_t max_iters, const FwdPruneArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  GR_DISPATCH_KV(kind, vc, GR_DISPATCH_N(max_iters, {
    const size_t lds = staged_bytes(a.pool.stride, 64 * NR);
    const size_t mlds = mfma_lds_bytes(a.pool.stride, 64 * NR);
    if constexpr (KIND == kU8L2) {
      if (mfma_ok(kind, a.pool) && mlds <= kMaxStagedLds) {
        hipLaunchKernelGGL((k_fwd_prune<KIND, LPV, CPL, NR, kMfma>), dim3(a.n), dim3(64), mlds, st, a);
        return hipGetLastError();
      }
    }
    if (lds <= kMaxStagedLds) {
      hipLaunchKernelGGL((k_fwd_prune<KIND, LPV, CPL, NR, kStaged>), dim3(a.n), dim3(64), lds, st, a);
    } else {
      hipLaunchKernelGGL((k_fwd_prune<KIND, LPV, CPL, NR, kGlobal>), dim3(a.n), dim3(64), 0, st, a);
    }
    return hipGetLastError();
  }));
  return hipErrorInvalidValue;
}

template <int KIND, int LPV, int CPL, int NP, int NC>
static void launch_rebuild_t(const RebuildArgs &a, uint32_t grid, hipStream_t st) {
  const size_t lds = staged_bytes(a.pool.stride, 64 * NC);
  const size_t mlds = mfma_lds_bytes(a.pool.stride, 64 * NC);
  if constexpr (KIND == kU8L2 && NC == 2) {
    if (a.pool.nch == 8) {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, NP, NC, kMfmaReg, 2>), dim3(grid), dim3(64), 0, st, a);
      return;
    }
    if (a.pool.nch == 4) {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, NP, NC, kMfmaReg, 1>), dim3(grid), dim3(64), 0, st, a);
      return;
    }
  }
  if constexpr (KIND == kU8L2) {
    if (mfma_ok(KIND, a.pool) && mlds <= kMaxStagedLds) {
      hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, NP, NC, kMfma>), dim3(grid), dim3(64), mlds, st, a);
      return;
    }
  }
  if (lds <= kMaxStagedLds) {
    hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, NP, NC, kStaged>), dim3(grid), dim3(64), lds, st, a);
  } else {
    hipLaunchKernelGGL((k_rebuild<KIND, LPV, CPL, NP, NC, kGlobal>), dim3(grid), dim3(64), 0, st, a);
  }
}

hipError_t launch_rebuild(int kind, int vc, uint32_t R, uint32_t P, const RebuildArgs &a, uint32_t grid,
                          hipStream_t st) {
  if (grid == 0) return hipSuccess;
  if (P > 128 || R + P > 256) return hipErrorInvalidValue;
  GR_DISPATCH_KV(kind, vc, {
    if (P <= 64 && R + P <= 128) {
      launch_rebuild_t<KIND, LPV, CPL, 1, 2>(a, grid, st);
    } else if (P <= 64) {
      launch_rebuild_t<KIND, LPV, CPL, 1, 4>(a, grid, st);
    } else {
      launch_rebuild_t<KIND, LPV, CPL, 2, 4>(a, grid, st);
    }
    return hipGetLastError();
  });
  return hipErrorInvalidValue;
}

}  // namespace gr
