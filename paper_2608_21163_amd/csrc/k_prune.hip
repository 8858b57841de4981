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

// Greedy selection inside one block of 16 sorted positions, resolved in
// parallel: kb (lane col) holds the earlier positions that would kill col,
// vb the live positions.  Each round, an undecided position is rejected if
// a selected one kills it, and selected if no undecided earlier position
// can; the lowest undecided position is always decided, so this ends with
// exactly the set the one-by-one walk selects.
__device__ __forceinline__ uint32_t block_greedy(uint32_t kb, uint32_t vb, int col, int g) {
  uint32_t S = 0, U = vb;
  while (U) {
    const bool und = ((U >> col) & 1u) != 0;
    const bool rej = und && (kb & S) != 0u;
    const bool sel = und && !rej && (kb & U) == 0u;
    const uint32_t sm = (uint32_t)ballot(sel && g == 0) & 0xFFFFu;
    const uint32_t rm = (uint32_t)ballot(rej && g == 0) & 0xFFFFu;
    S |= sm;
    U &= ~(sm | rm);
  }
  return S;
}
// The lowest n set bits of m.
__device__ __forceinline__ uint32_t first_bits(uint32_t m, int n) {
  uint32_t r = 0;
  for (int k = 0; k < n && m; k++) {
    r |= m & (0u - m);
    m &= m - 1u;
  }
  return r;
}

// The largest integer distance d with coef * d <= D (fp64 product, as in the
// prune test), for an integer-valued D >= 0; every d up to it passes, since
// rounding is monotone.
// inv is 1 / coef (rounded): the quotient estimate is off by at most one,
// and the two exact tests correct it.
__device__ __forceinline__ int kill_threshold(double coef, double inv, float D) {
  if (!(coef > 0.0)) return 0x7FFFFFFF;
  const double dd = (double)D;
  if (!(dd < 2147483647.0)) return 0x7FFFFFFF;
  const double q = floor(dd * inv);
  if (!(q < 2147483646.0)) return 0x7FFFFFFF;
  int t = (int)q;
  t = coef * (double)(t + 1) <= dd ? t + 1 : t;
  t = coef * (double)t <= dd ? t : t - 1;
  return t;
}

// GrANDRobustPrune's greedy selection for uint8 rows of 64*NK bytes, over
// up to 64*NR candidates already sorted by (D_p, id): spos/dpos (LDS) hold
// the sorted ids and distances, valid[] marks positions < m (element
// e = r*64 + lane).  Blocks of 16 sorted positions are taken in order: the
// block's rows are loaded as the MFMA A operand; the diagonal tile's kill
// masks resolve the block's own pivots in order (scalar loop), then every
// later tile that still holds a valid candidate is loaded as the B operand
// and its candidates are invalidated when their mask meets the selected
// pivots.  Distances are exact int32 (x ^ 0x80 operands), and the test
// coef * Dist <= D_p is the integer test Dist <= kill_threshold(coef, D_p).
// Rows are read from global memory (L2) when needed, the later tiles of a
// block kGroup at a time with all their loads in flight; nothing is staged.
// Lane t < nsel returns the t-th selection.
constexpr int kGroup = 4;  // candidate tiles loaded together by greedy_u8

template <int NK, int NR>
__device__ int greedy_u8(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, const uint32_t *spos,
                         const float *dpos, bool (&valid)[NR], uint32_t &sid, float &sdist,
                         unsigned long long &evals) {
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const double inv = 1.0 / coef;
  const size_t goff = (size_t)g * 16;
  const int nt = (m + 15) >> 4;
  auto load_tile = [&](v4i (&dst)[NK], int t) -> int {
    const int e = 16 * t + col;
    const uint8_t *row = P.vecs + (size_t)(e < m ? spos[e] : p) * P.stride + goff;
    int sq = 0;
#pragma unroll
    for (int kk = 0; kk < NK; kk++) {
      dst[kk] = to_i8x16(ld16(row + (size_t)kk * 64));
      sq = sq_i8x16(dst[kk], sq);
    }
    sq += (int)xshfl((uint32_t)sq, 16);
    sq += (int)xshfl((uint32_t)sq, 32);
    return sq;
  };
  auto tile_valid = [&](int t) -> uint32_t {
    bool v = valid[0];
#pragma unroll
    for (int r = 1; r < NR; r++) v = r == (t >> 2) ? valid[r] : v;
    return (uint32_t)(ballot(v) >> (16 * (t & 3))) & 0xFFFFu;
  };
  sid = kInvalid;
  sdist = finf();
  int nsel = 0;
  bool done = false;
  uint32_t S_blk = 0;
  for (int b = 0; b < nt && !done; b++) {
    const uint32_t vb = tile_valid(b);
    if (!vb) continue;
    v4i A[NK];
    const int na = load_tile(A, b);
    int rn[4];
#pragma unroll
    for (int ii = 0; ii < 4; ii++) rn[ii] = __shfl(na, 4 * g + ii, 64);
    uint32_t kmd = 0;
    {
      const int thr = kill_threshold(coef, inv, dpos[16 * b + col]);
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < NK; kk++) acc = mfma_i8(A[kk], A[kk], acc);
#pragma unroll
      for (int ii = 0; ii < 4; ii++) kmd |= (rn[ii] + na - 2 * acc[ii] <= thr) ? (1u << (4 * g + ii)) : 0u;
      kmd |= xshfl(kmd, 16);
      kmd |= xshfl(kmd, 32);
    }
    evals += 256;
    {
      // kmd (lane col): positions of the block that kill col; only earlier
      // ones matter
      uint32_t S = block_greedy(kmd & ((1u << col) - 1u), vb, col, g);
      int ns = __popc(S);
      if (ns >= (int)R - nsel) {
        ns = (int)R - nsel;
        S = first_bits(S, ns);
        done = true;
      }
      // lane nsel + k takes the k-th selected position of the block
      const int k = ln - nsel;
      if (k >= 0 && k < ns) {
        const int t = __ffs(first_bits(S, k + 1) & ~first_bits(S, k)) - 1;
        sid = spos[16 * b + t];
        sdist = dpos[16 * b + t];
      }
      nsel += ns;
      S_blk = S;
    }
    const uint32_t S = S_blk;
    if (done) break;
    // later tiles that still hold a valid candidate, kGroup at a time: all
    // loads of a group are issued before any is used
    int c = b + 1;
    while (c < nt) {
      int cs[kGroup];
      int ng = 0;
#pragma unroll
      for (int q = 0; q < kGroup; q++) {
        cs[q] = -1;
        while (c < nt && cs[q] < 0) {
          if (tile_valid(c)) cs[q] = c;
          c++;
        }
        ng += cs[q] >= 0 ? 1 : 0;
      }
      if (ng == 0) break;
      v4i Bt[kGroup][NK];
      int nb[kGroup], thr[kGroup];
#pragma unroll
      for (int q = 0; q < kGroup; q++) {
        nb[q] = 0;
        thr[q] = 0;
        if (cs[q] >= 0) {
          const int e = 16 * cs[q] + col;
          const uint8_t *row = P.vecs + (size_t)(e < m ? spos[e] : p) * P.stride + goff;
#pragma unroll
          for (int kk = 0; kk < NK; kk++) Bt[q][kk] = to_i8x16(ld16(row + (size_t)kk * 64));
          thr[q] = kill_threshold(coef, inv, dpos[e]);
        }
      }
#pragma unroll
      for (int q = 0; q < kGroup; q++) {
        if (cs[q] < 0) continue;
        int sq = 0;
        v4i acc = {0, 0, 0, 0};
#pragma unroll
        for (int kk = 0; kk < NK; kk++) {
          sq = sq_i8x16(Bt[q][kk], sq);
          acc = mfma_i8(A[kk], Bt[q][kk], acc);
        }
        sq += (int)xshfl((uint32_t)sq, 16);
        sq += (int)xshfl((uint32_t)sq, 32);
        nb[q] = sq;
        uint32_t km = 0;
#pragma unroll
        for (int ii = 0; ii < 4; ii++) km |= (rn[ii] + nb[q] - 2 * acc[ii] <= thr[q]) ? (1u << (4 * g + ii)) : 0u;
        km |= xshfl(km, 16);
        km |= xshfl(km, 32);
        evals += 256;
        const int cc = cs[q];
        const bool dead = g == (cc & 3) && (km & S) != 0;
#pragma unroll
        for (int r = 0; r < NR; r++)
          if (r == (cc >> 2)) valid[r] = valid[r] && !dead;
      }
    }
  }
  return nsel;
}

// greedy_u8 with every candidate tile resident in registers: the NT tiles
// (16 sorted candidates each, at most 16*NT candidates) are loaded once, all
// loads in flight together.  Live positions are kept as lane masks (bit e of
// vm[e / 64] for sorted position e), and per tile column the kill threshold
// minus the row's norm, so a kill test is one multiply-add and a compare:
// Dist(i, j) <= thr_j  <=>  |y_i|^2 - 2 y_i.y_j <= thr_j - |y_j|^2.  Against
// a later tile the compares of the block's rows are ballots, masked with the
// rows the block selected, and folded to the killed columns.  The selected
// positions go to oid/od (LDS) in order; returns their number.
template <int NK, int NT>
__device__ int greedy_u8_reg(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, const uint32_t *spos,
                             const float *dpos, int *thr, int *nrmL, uint32_t *oid, float *od, uint32_t &ntile) {
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const double inv = 1.0 / coef;
  const size_t goff = (size_t)g * 16;
  const int nt = (m + 15) >> 4;
  constexpr int NR = (NT + 3) / 4;
  v4i T[NT][NK];
  {
    uint4 raw[NT][NK];
#pragma unroll
    for (int t = 0; t < NT; t++) {
      const int e = 16 * t + col;
      const uint8_t *row = P.vecs + (size_t)(e < m ? spos[e] : p) * P.stride + goff;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) raw[t][kk] = 16 * t < m ? ld16(row + (size_t)kk * 64) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int t = 0; t < NT; t++)
#pragma unroll
      for (int kk = 0; kk < NK; kk++) T[t][kk] = to_i8x16(raw[t][kk]);
  }
  // kill thresholds of the sorted positions (LDS), norms of the tile rows
#pragma unroll
  for (int r = 0; r < NR; r++) {
    const int e = r * 64 + ln;
    thr[e] = e < m ? kill_threshold(coef, inv, dpos[e]) : -1;
  }
  __syncthreads();
  int t2[NT];
#pragma unroll
  for (int t = 0; t < NT; t++) {
    int sq = 0;
#pragma unroll
    for (int kk = 0; kk < NK; kk++) sq = sq_i8x16(T[t][kk], sq);
    sq += (int)xshfl((uint32_t)sq, 16);
    sq += (int)xshfl((uint32_t)sq, 32);
    if (g == 0) nrmL[16 * t + col] = sq;
    t2[t] = thr[16 * t + col] - sq;
  }
  __syncthreads();
  uint64_t vm[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) vm[r] = ballot(r * 64 + ln < m);
  int nsel = 0;
  bool done = false;
#pragma unroll
  for (int b = 0; b < NT; b++) {
    if (b >= nt || done) break;
    const uint32_t vb = (uint32_t)(vm[b >> 2] >> (16 * (b & 3))) & 0xFFFFu;
    if (!vb) continue;
    int rn[4];
#pragma unroll
    for (int ii = 0; ii < 4; ii++) rn[ii] = nrmL[16 * b + 4 * g + ii];
    // kb (lane col < 16): the block's earlier positions that would kill col
    uint32_t kb = 0;
    {
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < NK; kk++) acc = mfma_i8(T[b][kk], T[b][kk], acc);
#pragma unroll
      for (int ii = 0; ii < 4; ii++) kb |= (rn[ii] - 2 * acc[ii] <= t2[b]) ? (1u << (4 * g + ii)) : 0u;
      kb |= xshfl(kb, 16);
      kb |= xshfl(kb, 32);
      kb &= (1u << col) - 1u;
    }
    ntile++;
    // the block's pivots in order: a live position is selected unless an
    // earlier selected one kills it
    uint32_t S = block_greedy(kb, vb, col, g);
    int ns = __popc(S);
    const int room = (int)R - nsel;
    if (ns >= room) {  // selection stops at R: keep the first `room`
      S = first_bits(S, room);
      ns = room;
      done = true;
    }
    if (g == 0 && ((S >> col) & 1u)) {
      const int pos = nsel + __popc(S & ((1u << col) - 1u));
      oid[pos] = spos[16 * b + col];
      od[pos] = dpos[16 * b + col];
    }
    nsel += ns;
    if (done) break;
    // whether block row 4g + ii (this lane's rows) was selected
    bool sb[4];
#pragma unroll
    for (int ii = 0; ii < 4; ii++) sb[ii] = ((S >> (4 * g + ii)) & 1u) != 0u;
#pragma unroll
    for (int c = b + 1; c < NT; c++) {
      if (c >= nt) break;
      if (!((vm[c >> 2] >> (16 * (c & 3))) & 0xFFFFull)) continue;
      v4i acc = {0, 0, 0, 0};
#pragma unroll
      for (int kk = 0; kk < NK; kk++) acc = mfma_i8(T[b][kk], T[c][kk], acc);
      // column col of tile c dies when a selected row of the block kills it
      bool k = false;
#pragma unroll
      for (int ii = 0; ii < 4; ii++) k |= sb[ii] && (rn[ii] - 2 * acc[ii] <= t2[c]);
      uint32_t kw = k ? 1u : 0u;
      kw |= xshfl(kw, 16);
      kw |= xshfl(kw, 32);
      const uint64_t d = ballot(kw != 0u && g == 0) & 0xFFFFull;
      vm[c >> 2] &= ~(d << (16 * (c & 3)));
      ntile++;
    }
  }
  __syncthreads();
  return nsel;
}

// ---------------------------------------------------------------------------
// Forward GrANDRobustPrune of a new uint8 point (rows of 64*NK bytes, R <=
// 64): V_i arrives with D_{p_i} from the search, so the keys are sorted at
// once and the greedy selection (greedy_u8) needs no gather beforehand.
template <int NK, int NR>
__global__ __launch_bounds__(64, 6) void k_fwd_prune_mr(FwdPruneArgs a) {
  __shared__ uint32_t spos[64 * NR];
  __shared__ float dpos[64 * NR];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t nv = a.v_n[i];
  const uint32_t R = P.R;
  float kd[NR];
  uint32_t kid[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) {
    const uint32_t e = r * 64 + ln;
    const bool in = e < nv;
    uint32_t id = in ? a.v_ids[(size_t)i * a.v_stride + e] : kInvalid;
    float d = in ? a.v_d[(size_t)i * a.v_stride + e] : finf();
    if (id == p || !kvalid(id)) { id = kInvalid; d = finf(); }
    kd[r] = d;
    kid[r] = id;
  }
  wave_sort<NR>(kd, kid);
  {
    uint64_t dm[NR];
    if (wave_find_repeats<NR>(kd, kid, dm)) {
#pragma unroll
      for (int r = 0; r < NR; r++)
        if ((dm[r] >> ln) & 1) { kd[r] = finf(); kid[r] = kInvalid; }
      wave_sort<NR>(kd, kid);
    }
  }
  bool valid[NR];
  int m = 0;
#pragma unroll
  for (int r = 0; r < NR; r++) {
    valid[r] = kvalid(kid[r]);
    m += popc(ballot(valid[r]));
    spos[r * 64 + ln] = kid[r];
    dpos[r * 64 + ln] = kd[r];
  }
  __syncthreads();
  uint32_t sid;
  float sdist;
  unsigned long long evals = 0;
  const int nsel = greedy_u8<NK, NR>(P, p, m, R, a.coef, spos, dpos, valid, sid, sdist, evals);
  if (ln < (int)R) {
    const bool in = ln < nsel;
    P.adj[(size_t)p * R + ln] = in ? sid : kInvalid;
    if (P.adjd) P.adjd[(size_t)p * R + ln] = in ? sdist : 0.0f;
    a.rec_t[(size_t)i * R + ln] = in ? sid : kInvalid;
    a.rec_s[(size_t)i * R + ln] = p;
    a.rec_d[(size_t)i * R + ln] = in ? sdist : 0.0f;
  }
  if (ln == 0) {
    P.deg[p] = (uint32_t)nsel;
    stat_add(a.ds, kStFwdPrunes, 1ull);
    stat_add(a.ds, kStFwdEvals, evals);
    stat_add(a.ds, kStRecords, (unsigned long long)nsel);
  }
}

// Forward lists of new nodes: GrANDRobustPrune(p_i, V_i \ {p_i}, D_{p_i}),
// written to p_i's row (each new node owns its row), and the reverse-edge
// records (u, p_i, D_{p_i}[u]) for every selected u.
// MODE: kGlobal (rows read from global memory), kStaged (rows staged in
// LDS), kMfma (uint8 rows staged in LDS, pairwise distances on MFMA).
enum { kGlobal = 0, kStaged = 1, kMfma = 2 };

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
    stat_add(a.ds, kStFwdPrunes, 1ull);
    stat_add(a.ds, kStFwdEvals, evals);
    stat_add(a.ds, kStRecords, (unsigned long long)nsel);
  }
}

// Rebuild of dirty nodes.  For dirty u: scratch_u = the P smallest distinct
// (distance, source) records addressed to u; C = (N_out(u) u scratch_u)
// minus u (and minus the delete batch); if |C| <= R, C is installed (kept
// entries in slot order, then new sources in record order); otherwise
// GrANDRobustPrune(u, C, D_u) is installed.  One owner per dirty node, so
// rows are written without locks.
template <int KIND, int LPV, int CPL, int NP, int NC, int MODE>
__global__ __launch_bounds__(64) void k_rebuild(RebuildArgs a) {
  extern __shared__ __align__(16) uint8_t vbuf[];
  __shared__ uint32_t rowL[64];
  __shared__ uint32_t slot_id[64 * NC];
  __shared__ uint32_t lids[64 * NC];
  __shared__ float ldist[64 * NC];
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const uint32_t nd_total = *a.list_n;
  unsigned long long evals = 0, prunes = 0, nodes = 0, recs = 0, cand = 0;
  for (uint32_t it = blockIdx.x; it < nd_total; it += gridDim.x) {
    const uint32_t u = a.list[it];
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
      if constexpr (MODE == kMfma) {
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
    stat_add(a.ds, kStRbPrunes, prunes);
    stat_add(a.ds, kStRbEvals, evals);
    stat_add(a.ds, kStRbCand, cand);
    if (a.count_nodes) {
      stat_add(a.ds, kStDirty, nodes);
      stat_add(a.ds, kStRbRecs, recs);
    }
  }
}

// C of dirty node u (R <= 64, P <= 64): the kept entries of N_out(u) (minus
// u and the delete batch) in slot order, then the sources of the P smallest
// distinct records that are not already kept; written to cl (LDS), and
// with cdl (LDS, given when the pool stores list distances) D_u of each:
// the stored distance of a kept entry, the record's distance of a new one.
// Returns |C|; nrec is the number of records addressed to u.
__device__ int collect_candidates(const RebuildArgs &a, uint32_t u, uint4 *rowL, uint32_t *cl, uint32_t &nrec,
                                  float *cdl = nullptr) {
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const uint32_t g0 = a.goff[u], g1 = a.goff[u + 1];
  const uint32_t rv = ln < (int)R ? P.adj[(size_t)u * R + ln] : kInvalid;
  const float rdv = cdl && ln < (int)R ? P.adjd[(size_t)u * R + ln] : 0.0f;
  nrec = g1 - g0;
  // the first 64 records, loaded beside the row (lanes past the records
  // read a valid one and drop it); then the batch flags of the row's ids and
  // of those records' sources together (index 0 stands in for an id that
  // is not checked)
  const uint32_t j0 = g0 + (uint32_t)ln;
  const uint32_t jc = j0 < g1 ? j0 : (g1 > g0 ? g0 : 0u);
  const uint32_t s0 = a.gsrc[jc];
  const float d0 = a.gd[jc];
  const bool rok = rv != kInvalid && rv != u;
  const bool sok = j0 < g1 && kvalid(s0);
  bool rin = false, sin = false;
  if (a.in_batch) {
    const uint8_t fr = a.in_batch[rok ? rv : 0u];
    const uint8_t fs = a.in_batch[sok ? s0 : 0u];
    rin = rok && fr;
    sin = sok && fs;
  }
  // the merged sources below are all among these records when there are
  // at most 64; then none of them needs its flag loaded again
  const bool recheck = a.in_batch && (g1 - g0 > 64u || ballot(sin) != 0);
  const bool keep = rok && !rin;
  const uint64_t kmask = ballot(keep);
  const int kr = popc(kmask);
  reinterpret_cast<uint32_t *>(rowL)[ln] = keep ? rv : kInvalid;
  if (keep) {
    cl[mbcnt(kmask)] = rv;
    if (cdl) cdl[mbcnt(kmask)] = rdv;
  }
  __syncthreads();
  // scratch_u: the P smallest distinct (distance, source) records
  float sd[1] = {finf()};
  uint32_t si[1] = {kInvalid};
  for (uint32_t base = g0; base < g1; base += 64) {
    const uint32_t j = base + ln;
    uint32_t sv = j < g1 ? (base == g0 ? s0 : a.gsrc[j]) : kInvalid;
    float dv = j < g1 ? (base == g0 ? d0 : a.gd[j]) : finf();
    if (!kvalid(sv)) { sv = kInvalid; dv = finf(); }
    wave_merge_new_fast<1>(sd, si, dv, sv, (int)a.P);
  }
  bool isnew;
  {
    const uint32_t sv = si[0];
    bool ok = kvalid(sv) && sv != u && !(recheck && a.in_batch[sv]);
#pragma unroll 4
    for (int t = 0; t < 16; t++) {
      const uint4 r4 = rowL[t];
      ok = ok & (r4.x != sv) & (r4.y != sv) & (r4.z != sv) & (r4.w != sv);
    }
    isnew = ok;
  }
  const uint64_t nmask = ballot(isnew);
  const int m = kr + popc(nmask);
  if (isnew) {
    cl[kr + mbcnt(nmask)] = si[0];
    if (cdl) cdl[kr + mbcnt(nmask)] = sd[0];
  }
  __syncthreads();
  return m;
}

// Candidate tiles a rebuild keeps in registers (|C| <= 80: the kept row and
// up to 16 records); larger candidate sets take greedy_u8.
constexpr int kRegTiles = 5;

// Rebuild of dirty nodes for uint8 rows of 64*NK bytes with R <= 64 and
// R + P <= 128 (the same steps as k_rebuild).  When a node prunes, D_u of
// every candidate comes from int8 MFMA of u's row against the candidates,
// 16 at a time (exact, so it equals the distances the records carry); the
// keys are sorted and greedy_u8 selects.  Only a few registers per
// candidate tile are live at a time, so many waves fit per SIMD to hide
// the gathers.
template <int NK>
__global__ __launch_bounds__(64, 4) void k_rebuild_mr(RebuildArgs a) {
  constexpr int NC = 2;
  __shared__ uint4 rowL[16];
  __shared__ uint32_t cl[64 * NC];
  __shared__ float cdL[64 * NC];  // D_u of the candidates, from the stored list distances
  __shared__ uint32_t spos[64 * NC];
  __shared__ float dpos[64 * NC];
  __shared__ int thrL[64 * NC];
  __shared__ int nrmL[64 * NC];
  __shared__ uint32_t oid[64];
  __shared__ float od[64];
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const uint32_t nd_total = *a.list_n;
  const size_t goff = (size_t)g * 16;
  unsigned long long evals = 0;
  uint32_t prunes = 0, nodes = 0, recs = 0, cand = 0;
  // the next node of this wave is read while the current one is rebuilt
  uint32_t u_next = blockIdx.x < nd_total ? a.list[blockIdx.x] : 0u;
  for (uint32_t it = blockIdx.x; it < nd_total; it += gridDim.x) {
    const uint32_t u = u_next;
    u_next = a.list[it + gridDim.x < nd_total ? it + gridDim.x : it];
    nodes++;
    uint32_t nrec;
    const int m = collect_candidates(a, u, rowL, cl, nrec, P.adjd ? cdL : nullptr);
    recs += nrec;
    if (m <= (int)R) {
      if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < m ? cl[ln] : kInvalid;
      if (P.adjd && ln < (int)R) P.adjd[(size_t)u * R + ln] = ln < m ? cdL[ln] : 0.0f;
      if (ln == 0) P.deg[u] = (uint32_t)m;
      __syncthreads();
      continue;
    }
    // D_u of every candidate (list order), into dpos: stored, or by int8
    // MFMA of u's row against the candidates
    if (P.adjd) {
#pragma unroll
      for (int r = 0; r < NC; r++)
        if (r * 64 + ln < m) dpos[r * 64 + ln] = cdL[r * 64 + ln];
    } else {
      v4i A[NK];
      int np = 0;
      const uint8_t *urow = P.vecs + (size_t)u * P.stride + goff;
#pragma unroll
      for (int kk = 0; kk < NK; kk++) {
        A[kk] = to_i8x16(ld16(urow + (size_t)kk * 64));
        np = sq_i8x16(A[kk], np);
      }
      np += (int)xshfl((uint32_t)np, 16);
      np += (int)xshfl((uint32_t)np, 32);
      // candidate tiles kRegTiles at a time (one batch when |C| <= 80), all
      // loads of a batch issued before the first is used
      for (int t0 = 0; 16 * t0 < m; t0 += kRegTiles) {
        uint4 raw[kRegTiles][NK];
#pragma unroll
        for (int h = 0; h < kRegTiles; h++) {
          const int e = 16 * (t0 + h) + col;
#pragma unroll
          for (int kk = 0; kk < NK; kk++)
            raw[h][kk] = e - col < m ? ld16(P.vecs + (size_t)(e < m ? cl[e] : u) * P.stride + goff + (size_t)kk * 64)
                                     : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int h = 0; h < kRegTiles; h++) {
          const int e = 16 * (t0 + h) + col;
          if (e - col >= m) break;
          int sq = 0;
          v4i acc = {0, 0, 0, 0};
#pragma unroll
          for (int kk = 0; kk < NK; kk++) {
            const v4i b = to_i8x16(raw[h][kk]);
            sq = sq_i8x16(b, sq);
            acc = mfma_i8(A[kk], b, acc);
          }
          sq += (int)xshfl((uint32_t)sq, 16);
          sq += (int)xshfl((uint32_t)sq, 32);
          if (g == 0) dpos[e] = canon0((float)(np + sq - 2 * acc[0]));
        }
      }
    }
    if (!P.adjd) evals += (unsigned long long)m;
    __syncthreads();
    // Candidates by (D_u, id): 32-bit keys D << 7 | list position (uint8
    // distances are integers below 2^23) order them when no two share a
    // distance; a tie, which the id decides, takes the 64-bit key sort.
    uint32_t k32[NC];
#pragma unroll
    for (int r = 0; r < NC; r++) {
      const int e = r * 64 + ln;
      k32[r] = e < m ? ((uint32_t)dpos[e] << 7) | (uint32_t)e : ~0u;
    }
    wave_sort32<NC>(k32);
    bool tie = false;
#pragma unroll
    for (int r = 0; r < NC; r++) {
      // the next element's key (lane 63 of a row: lane 0 of the next row)
      uint32_t nx = __shfl(k32[r], (ln + 1) & 63, 64);
      if (ln == 63) nx = r + 1 < NC ? rdlane(k32[r + 1 < NC ? r + 1 : r], 0) : ~0u;
      tie |= r * 64 + ln + 1 < m && (k32[r] >> 7) == (nx >> 7);
    }
    if (!ballot(tie)) {
      uint32_t sid[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) sid[r] = r * 64 + ln < m ? cl[k32[r] & 127u] : kInvalid;
#pragma unroll
      for (int r = 0; r < NC; r++) {
        spos[r * 64 + ln] = sid[r];
        dpos[r * 64 + ln] = r * 64 + ln < m ? (float)(k32[r] >> 7) : finf();
      }
    } else {
      uint64_t key[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const int e = r * 64 + ln;
        key[r] = e < m ? key64(dpos[e], cl[e]) : ~0ull;
      }
      __syncthreads();
      wave_sort64<NC>(key);
#pragma unroll
      for (int r = 0; r < NC; r++) {
        spos[r * 64 + ln] = (uint32_t)key[r];
        dpos[r * 64 + ln] = unsortable((uint32_t)(key[r] >> 32));
      }
    }
    __syncthreads();
    int nsel;
    if (m <= 16 * kRegTiles) {  // every candidate tile resident in registers
      uint32_t ntile = 0;
      nsel = greedy_u8_reg<NK, kRegTiles>(P, u, m, R, a.coef, spos, dpos, thrL, nrmL, oid, od, ntile);
      evals += 256ull * ntile;
    } else {  // more candidates (more than 16 records): tiles loaded per block
      bool valid[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) valid[r] = r * 64 + ln < m;
      uint32_t sid;
      float sdist;
      nsel = greedy_u8<NK, NC>(P, u, m, R, a.coef, spos, dpos, valid, sid, sdist, evals);
      if (ln < nsel) {
        oid[ln] = sid;
        od[ln] = sdist;
      }
      __syncthreads();
    }
    if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < nsel ? oid[ln] : kInvalid;
    if (P.adjd && ln < (int)R) P.adjd[(size_t)u * R + ln] = ln < nsel ? od[ln] : 0.0f;
    if (ln == 0) P.deg[u] = (uint32_t)nsel;
    prunes++;
    cand += (unsigned long long)m + (P.adjd ? 0u : 1u);
    __syncthreads();
  }
  if (ln == 0) {
    stat_add(a.ds, kStRbPrunes, prunes);
    stat_add(a.ds, kStRbEvals, evals);
    stat_add(a.ds, kStRbCand, cand);
    if (a.count_nodes) {
      stat_add(a.ds, kStDirty, nodes);
      stat_add(a.ds, kStRbRecs, recs);
    }
  }
}

// Rebuild, fast path (R <= 64, R a multiple of 4): four dirty nodes per
// wavefront, 16 lanes per node, four row slots per lane.  For dirty u the
// records fit when there are at most min(16, P) of them, so scratch_u is all
// of them; C = (N_out(u) u scratch_u) minus u, repeats and the delete batch.
// When C fits in R it is installed here (kept entries in slot order, then
// the new sources); every other node -- more records than that, or |C| > R,
// which needs GrANDRobustPrune -- is flagged in `qflag` and later compacted
// into `queue` for the general kernel.  No distance is needed on this path.
__global__ __launch_bounds__(64) void k_rebuild_fast(RebuildArgs a) {
  __shared__ uint4 rowL[64];
  __shared__ uint32_t srcL[64];
  __shared__ uint32_t outL[4 * 64];
  __shared__ float outD[4 * 64];  // stored list distances, when the pool keeps them
  const int ln = lane(), s = ln >> 4, q = ln & 15;
  const PoolView &P = a.pool;
  const uint32_t R = P.R, R4 = R >> 2;
  const uint32_t nd = *a.list_n;
  const uint32_t lim = a.P < 16u ? a.P : 16u;
  unsigned long long nodes = 0, recs = 0;
  for (uint32_t b = blockIdx.x * 4u; b < nd; b += gridDim.x * 4u) {
    const uint32_t idx = b + (uint32_t)s;
    const bool has = idx < nd;
    const uint32_t u = has ? a.list[idx] : 0u;
    uint32_t g0 = 0, g1 = 0;
    uint4 rw = make_uint4(kInvalid, kInvalid, kInvalid, kInvalid);
    float4 rd = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (has) {
      g0 = a.goff[u];
      g1 = a.goff[u + 1];
      if ((uint32_t)q < R4) {
        rw = *reinterpret_cast<const uint4 *>(P.adj + (size_t)u * R + 4 * q);
        if (P.adjd) rd = *reinterpret_cast<const float4 *>(P.adjd + (size_t)u * R + 4 * q);
      }
    }
    const uint32_t nrec = g1 - g0;
    const bool light = has && nrec <= lim;
    uint32_t src = kInvalid;
    float srd = 0.0f;
    if (light && (uint32_t)q < nrec) {
      src = a.gsrc[g0 + q];
      srd = a.gd[g0 + q];
    }
    const float dk[4] = {rd.x, rd.y, rd.z, rd.w};
    const uint32_t id[4] = {rw.x, rw.y, rw.z, rw.w};
    bool keep[4];
#pragma unroll
    for (int k = 0; k < 4; k++) keep[k] = id[k] != kInvalid && id[k] != u && !(a.in_batch && a.in_batch[id[k]]);
    bool nw = kvalid(src) && src != u && !(a.in_batch && a.in_batch[src]);
    rowL[ln] = make_uint4(keep[0] ? id[0] : kInvalid, keep[1] ? id[1] : kInvalid, keep[2] ? id[2] : kInvalid,
                          keep[3] ? id[3] : kInvalid);
    srcL[ln] = src;
    __syncthreads();
    // a source already in the kept row, or repeated by an earlier record
#pragma unroll 4
    for (int j = 0; j < 16; j++) {
      const uint4 r = rowL[s * 16 + j];
      const uint32_t o = srcL[s * 16 + j];
      nw = nw & (r.x != src) & (r.y != src) & (r.z != src) & (r.w != src) & !((j < q) & (o == src));
    }
    // positions: kept entries in slot order, then the new sources
    const int kc = (int)keep[0] + (int)keep[1] + (int)keep[2] + (int)keep[3];
    int x = kc;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int y = __shfl_up(x, o, 16);
      if (q >= o) x += y;
    }
    const int kr = __shfl(x, s * 16 + 15, 64);
    const uint32_t gm = (uint32_t)(ballot(nw) >> (16 * s)) & 0xFFFFu;
    const int m = kr + popc((uint64_t)gm);
    const bool install = light && m <= (int)R;
    if (install) {
      int pos = x - kc;
#pragma unroll
      for (int k = 0; k < 4; k++)
        if (keep[k]) {
          outL[s * 64 + pos] = id[k];
          outD[s * 64 + pos] = dk[k];
          pos++;
        }
      if (nw) {
        const int e = kr + popc((uint64_t)(gm & ((1u << q) - 1u)));
        outL[s * 64 + e] = src;
        outD[s * 64 + e] = srd;
      }
    }
    __syncthreads();
    if (install && (uint32_t)q < R4) {
      const int e = 4 * q;
      uint4 o;
      o.x = e + 0 < m ? outL[s * 64 + e + 0] : kInvalid;
      o.y = e + 1 < m ? outL[s * 64 + e + 1] : kInvalid;
      o.z = e + 2 < m ? outL[s * 64 + e + 2] : kInvalid;
      o.w = e + 3 < m ? outL[s * 64 + e + 3] : kInvalid;
      *reinterpret_cast<uint4 *>(P.adj + (size_t)u * R + e) = o;
      if (P.adjd) {
        float4 d;
        d.x = e + 0 < m ? outD[s * 64 + e + 0] : 0.0f;
        d.y = e + 1 < m ? outD[s * 64 + e + 1] : 0.0f;
        d.z = e + 2 < m ? outD[s * 64 + e + 2] : 0.0f;
        d.w = e + 3 < m ? outD[s * 64 + e + 3] : 0.0f;
        *reinterpret_cast<float4 *>(P.adjd + (size_t)u * R + e) = d;
      }
    }
    if (install && q == 0) P.deg[u] = (uint32_t)m;
    // nodes left for the general kernel are flagged by list position and
    // compacted afterwards (no shared counter on this path)
    if (has && q == 0) {
      a.qflag[idx] = install ? 0u : 1u;
      nodes++;
      recs += nrec;
    }
    __syncthreads();
  }
  // one atomic per wave: the counts live in lanes 0, 16, 32, 48
  unsigned long long tn = nodes, tr = recs;
#pragma unroll
  for (int k = 1; k < 4; k++) {
    tn += __shfl(nodes, 16 * k, 64);
    tr += __shfl(recs, 16 * k, 64);
  }
  if (ln == 0 && tn) {
    stat_add(a.ds, kStDirty, tn);
    stat_add(a.ds, kStRbRecs, tr);
  }
}

// ---------------------------------------------------------------------------
// fp32 GrANDRobustPrune with one lane per candidate position.  Distances
// are accumulated in fp64 in dimension order -- the oracle's summation, so
// every rounded distance is identical -- between each lane's own rows
// (streamed from the pool in pieces of 16 floats) and up to 16 rows staged in
// LDS, one slice of kVecSlice floats at a time, which every lane reads at the
// same address.
constexpr int kVecSlice = 64;

// st[k][0..kVecSlice) <- floats [d0, d0 + kVecSlice) of pool row ids[k],
// widened to fp64 once here rather than at every use (k < ns; zeros past
// the row or for an invalid id).  Lane (k, part) copies 16 floats.
__device__ __forceinline__ void vec_stage(const PoolView &P, const uint32_t *ids, int ns, int d0, int nfl,
                                          double (*st)[kVecSlice]) {
  const int ln = lane(), k = ln >> 2, part = ln & 3;
  if (k >= ns) return;
  const uint32_t id = ids[k];
  const float *row = reinterpret_cast<const float *>(P.vecs + (size_t)(kvalid(id) ? id : 0u) * P.stride);
  // all four loads issued before any is used: addresses clamped into the
  // row, the values past it replaced by zeros afterwards
  uint4 v4[4];
#pragma unroll
  for (int h = 0; h < 4; h++) {
    const int f = d0 + 16 * part + 4 * h;
    v4[h] = *reinterpret_cast<const uint4 *>(row + (f < nfl ? f : 0));
  }
#pragma unroll
  for (int h = 0; h < 4; h++) {
    const int f = d0 + 16 * part + 4 * h;
    const uint4 v = (kvalid(id) && f < nfl) ? v4[h] : make_uint4(0, 0, 0, 0);
    double2 *dst = reinterpret_cast<double2 *>(&st[k][16 * part + 4 * h]);
    dst[0] = make_double2((double)__uint_as_float(v.x), (double)__uint_as_float(v.y));
    dst[1] = make_double2((double)__uint_as_float(v.z), (double)__uint_as_float(v.w));
  }
}

// acc[r][k] += the terms of floats [d0, d0 + kVecSlice) between this lane's
// row own[r] and staged row k, for every register row r with work (act[r],
// uniform) and every k in kmask (uniform).
template <int KIND, int NCL, int NS>
__device__ __forceinline__ void vec_accumulate(const double (*st)[kVecSlice], const float *const (&own)[NCL],
                                               const bool (&act)[NCL], int d0, int nfl,
                                               double (&acc)[NCL][NS], uint32_t kmask = ~0u) {
  for (int pc = 0; pc < kVecSlice && d0 + pc < nfl; pc += 16) {
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      if (!act[r]) continue;
      float xv[16];
      // rows hold nfl floats, a multiple of 4; all four loads are issued
      // before any is used (addresses clamped into the row, the values past
      // it replaced by zeros afterwards)
      uint4 v4[4];
#pragma unroll
      for (int h = 0; h < 4; h++) {
        const int f = d0 + pc + 4 * h;
        v4[h] = *reinterpret_cast<const uint4 *>(own[r] + (f < nfl ? f : 0));
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
      for (int k = 0; k < NS; k++) {
        if (!((kmask >> k) & 1u)) continue;  // staged row k is not needed
#pragma unroll
        for (int t = 0; t < 16; t++) {
          if (KIND == kF32IP) {
            acc[r][k] = __builtin_fma((double)xv[t], st[k][pc + t], acc[r][k]);
          } else {
            const double df = st[k][pc + t] - (double)xv[t];
            acc[r][k] = __builtin_fma(df, df, acc[r][k]);
          }
        }
      }
    }
  }
}

// GrANDRobustPrune over m candidates sorted by (D_p, id) (spos/dpos in LDS,
// positions e = r*64 + lane, at most 64*NCL).  Positions are taken in blocks
// of NPB pivots: the block's rows are staged and the distances from them to
// every still-live position from the block on are computed, those positions
// packed onto the lanes (a block rarely leaves more than 64 of them, so the
// fp64 work follows the live positions, not the register rows); the block's
// own selections come from the parallel fixpoint, and later positions that a
// selected pivot kills (coef * Dist <= D, in fp64 on the rounded distance)
// are dropped.  Pivots already dead take no distance work.  The selections go to oid/od (LDS) in order; returns their
// number.
template <int KIND, int NCL, int NPB>
__device__ int prune_vec(const PoolView &P, uint32_t p, int m, uint32_t R, double coef, const uint32_t *spos,
                         const float *dpos, double (*st)[kVecSlice], uint32_t *oid, float *od, uint32_t &evals) {
  static_assert(NPB <= 16 && 64 % NPB == 0, "pivot blocks inside one register row");
  __shared__ uint32_t lpos[64 * NCL];  // live positions of the block, packed
  __shared__ uint32_t kmL[64 * NCL];   // kill masks by position
  const int ln = lane(), g = ln >> 4, col = ln & 15;
  const int nfl = P.nch * 4;
  uint64_t vm[NCL];
#pragma unroll
  for (int r = 0; r < NCL; r++) vm[r] = ballot(r * 64 + ln < m);
  int nsel = 0;
  const int nb = (m + NPB - 1) / NPB;
  for (int b = 0; b < nb; b++) {
    const int p0 = b * NPB;
    uint64_t vr = 0;
#pragma unroll
    for (int r = 0; r < NCL; r++)
      if (r == (p0 >> 6)) vr = vm[r];
    const uint32_t vb = (uint32_t)(vr >> (p0 & 63)) & ((1u << NPB) - 1u);
    if (!vb) continue;
    // live positions >= p0, in order, packed onto the lanes
    int nl = 0;
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      const int e = r * 64 + ln;
      const bool lv = e >= p0 && ((vm[r] >> ln) & 1ull);
      const uint64_t bm = ballot(lv);
      if (lv) lpos[nl + mbcnt(bm)] = (uint32_t)e;
      nl += popc(bm);
    }
    __syncthreads();
    bool act[NCL];
    const float *own[NCL];
    int ep[NCL];
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      act[r] = r * 64 < nl;
      const int c = r * 64 + ln;
      ep[r] = act[r] && c < nl ? (int)lpos[c] : -1;
      own[r] = reinterpret_cast<const float *>(P.vecs + (size_t)(ep[r] >= 0 ? spos[ep[r]] : p) * P.stride);
    }
    double acc[NCL][NPB];
#pragma unroll
    for (int r = 0; r < NCL; r++)
#pragma unroll
      for (int k = 0; k < NPB; k++) acc[r][k] = 0.0;
    for (int d0 = 0; d0 < nfl; d0 += kVecSlice) {
      __syncthreads();
      vec_stage(P, spos + p0, min(NPB, m - p0), d0, nfl, st);
      __syncthreads();
      vec_accumulate<KIND, NCL, NPB>(st, own, act, d0, nfl, acc, vb);
    }
    // kill masks of the packed positions, scattered back by position
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      const int e = ep[r];
      if (e < 0) continue;
      const double De = (double)dpos[e];
      uint32_t km = 0;
#pragma unroll
      for (int k = 0; k < NPB; k++) {
        const bool kill = ((vb >> k) & 1u) && e > p0 + k && coef * (double)finalize<KIND>(acc[r][k]) <= De;
        km |= kill ? (1u << k) : 0u;
      }
      kmL[e] = km;
    }
    evals += (uint32_t)(__popc(vb) * nl);
    __syncthreads();
    // km[r]: pivots of the block that kill this lane's position
    uint32_t km[NCL];
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      const int e = r * 64 + ln;
      km[r] = e >= p0 && ((vm[r] >> ln) & 1ull) ? kmL[e] : 0u;
    }
    // the block's own positions: lanes (p0 & 63) + col of register row p0 >> 6
    uint32_t kbr = 0;
#pragma unroll
    for (int r = 0; r < NCL; r++)
      if (r == (p0 >> 6)) kbr = km[r];
    const uint32_t kb = (uint32_t)__shfl((int)kbr, ((p0 & 63) + col) & 63, 64) & ((1u << col) - 1u);
    uint32_t S = block_greedy(kb, vb, col, g);
    int ns = __popc(S);
    const int room = (int)R - nsel;
    bool done = false;
    if (ns >= room) {
      S = first_bits(S, room);
      ns = room;
      done = true;
    }
    if (g == 0 && ((S >> col) & 1u)) {
      const int pos = nsel + __popc(S & ((1u << col) - 1u));
      oid[pos] = spos[p0 + col];
      od[pos] = dpos[p0 + col];
    }
    nsel += ns;
    if (done) break;
#pragma unroll
    for (int r = 0; r < NCL; r++) {
      const int e = r * 64 + ln;
      vm[r] &= ~ballot(e >= p0 + NPB && (km[r] & S) != 0u);
    }
    __syncthreads();
  }
  __syncthreads();
  return nsel;
}

// Rebuild of queued dirty nodes for fp32 rows with R <= 64 and R + P <= 128:
// C as in k_rebuild_mr; D_u of every candidate from u's staged row, a
// 64-bit-key sort, then prune_vec.
template <int KIND>
__global__ __launch_bounds__(64) void k_rebuild_vec(RebuildArgs a) {
  constexpr int NC = 2;
  __shared__ uint4 rowL[16];
  __shared__ uint32_t cl[64 * NC];
  __shared__ uint32_t spos[64 * NC];
  __shared__ float dpos[64 * NC];
  __shared__ double st[16][kVecSlice];
  __shared__ uint32_t oid[64];
  __shared__ float od[64];
  __shared__ uint32_t uid[1];
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t R = P.R;
  const int nfl = P.nch * 4;
  const uint32_t nd_total = *a.list_n;
  uint32_t evals = 0, prunes = 0, nodes = 0, recs = 0, cand = 0;
  for (uint32_t it = blockIdx.x; it < nd_total; it += gridDim.x) {
    const uint32_t u = a.list[it];
    nodes++;
    uint32_t nrec;
    const int m = collect_candidates(a, u, rowL, cl, nrec);
    recs += nrec;
    if (m <= (int)R) {
      if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < m ? cl[ln] : kInvalid;
      if (ln == 0) P.deg[u] = (uint32_t)m;
      __syncthreads();
      continue;
    }
    // D_u of every candidate (list order)
    {
      const float *own[NC];
      bool act[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const int e = r * 64 + ln;
        own[r] = reinterpret_cast<const float *>(P.vecs + (size_t)(e < m ? cl[e] : u) * P.stride);
        act[r] = r * 64 < m;
      }
      double du[NC][1];
#pragma unroll
      for (int r = 0; r < NC; r++) du[r][0] = 0.0;
      if (ln == 0) uid[0] = u;
      for (int d0 = 0; d0 < nfl; d0 += kVecSlice) {
        __syncthreads();
        vec_stage(P, uid, 1, d0, nfl, st);
        __syncthreads();
        vec_accumulate<KIND, NC, 1>(st, own, act, d0, nfl, du);
      }
      evals += (uint32_t)m;
      uint64_t key[NC];
#pragma unroll
      for (int r = 0; r < NC; r++) {
        const int e = r * 64 + ln;
        key[r] = e < m ? key64(finalize<KIND>(du[r][0]), cl[e]) : ~0ull;
      }
      __syncthreads();
      wave_sort64<NC>(key);
#pragma unroll
      for (int r = 0; r < NC; r++) {
        spos[r * 64 + ln] = (uint32_t)key[r];
        dpos[r * 64 + ln] = unsortable((uint32_t)(key[r] >> 32));
      }
      __syncthreads();
    }
    const int nsel = prune_vec<KIND, NC, 16>(P, u, m, R, a.coef, spos, dpos, st, oid, od, evals);
    if (ln < (int)R) P.adj[(size_t)u * R + ln] = ln < nsel ? oid[ln] : kInvalid;
    if (ln == 0) P.deg[u] = (uint32_t)nsel;
    prunes++;
    cand += (uint32_t)m + 1;
    __syncthreads();
  }
  if (ln == 0) {
    stat_add(a.ds, kStRbPrunes, (unsigned long long)prunes);
    stat_add(a.ds, kStRbEvals, (unsigned long long)evals);
    stat_add(a.ds, kStRbCand, (unsigned long long)cand);
    if (a.count_nodes) {
      stat_add(a.ds, kStDirty, (unsigned long long)nodes);
      stat_add(a.ds, kStRbRecs, (unsigned long long)recs);
    }
  }
}

// Forward GrANDRobustPrune of new fp32 points: V_i with the search's D, a
// 64-bit-key sort, then prune_vec (blocks of 8 pivots for 256 candidates).
template <int KIND, int NR>
__global__ __launch_bounds__(64) void k_fwd_prune_vec(FwdPruneArgs a) {
  constexpr int NPB = NR >= 4 ? 8 : 16;
  __shared__ uint32_t spos[64 * NR];
  __shared__ float dpos[64 * NR];
  __shared__ double st[16][kVecSlice];
  __shared__ uint32_t oid[64];
  __shared__ float od[64];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  const uint32_t nv = a.v_n[i];
  const uint32_t R = P.R;
  uint64_t key[NR];
  int m = 0;
#pragma unroll
  for (int r = 0; r < NR; r++) {
    const uint32_t e = r * 64 + ln;
    const uint32_t id = e < nv ? a.v_ids[(size_t)i * a.v_stride + e] : kInvalid;
    const bool ok = kvalid(id) && id != p;
    key[r] = ok ? key64(a.v_d[(size_t)i * a.v_stride + e], id) : ~0ull;
    m += popc(ballot(ok));
  }
  // V_i holds distinct ids: the sort alone gives the candidate order
  wave_sort64<NR>(key);
#pragma unroll
  for (int r = 0; r < NR; r++) {
    spos[r * 64 + ln] = (uint32_t)key[r];
    dpos[r * 64 + ln] = unsortable((uint32_t)(key[r] >> 32));
  }
  __syncthreads();
  uint32_t evals = 0;
  const int nsel = prune_vec<KIND, NR, NPB>(P, p, m, R, a.coef, spos, dpos, st, oid, od, evals);
  if (ln < (int)R) {
    const bool in = ln < nsel;
    const uint32_t sid = in ? oid[ln] : kInvalid;
    P.adj[(size_t)p * R + ln] = sid;
    a.rec_t[(size_t)i * R + ln] = sid;
    a.rec_s[(size_t)i * R + ln] = p;
    a.rec_d[(size_t)i * R + ln] = in ? od[ln] : 0.0f;
  }
  if (ln == 0) {
    P.deg[p] = (uint32_t)nsel;
    stat_add(a.ds, kStFwdPrunes, 1ull);
    stat_add(a.ds, kStFwdEvals, (unsigned long long)evals);
    stat_add(a.ds, kStRecords, (unsigned long long)nsel);
  }
}

// LDS bytes for staging `rows` candidate rows plus the node's own row.
static size_t staged_bytes(size_t stride, uint32_t rows) { return (size_t)(rows + 1) * lds_stride(stride); }
constexpr size_t kMaxStagedLds = 16 * 1024;  // larger footprints limit occupancy more than staging saves

// The matrix-core prune applies to uint8 rows whose chunk count is a
// multiple of 4 (dim a multiple of 64), i.e. whole 64-byte MFMA K steps.
static bool mfma_ok(int kind, const PoolView &P) { return kind == kU8L2 && P.nch % 4 == 0; }

hipError_t launch_fwd_prune(int kind, int vc, uint32_t max_iters, const FwdPruneArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  if (kind == kU8L2 && a.pool.R <= 64 && (a.pool.nch == 8 || a.pool.nch == 4)) {
    GR_DISPATCH_N(max_iters, {
      if (a.pool.nch == 8) hipLaunchKernelGGL((k_fwd_prune_mr<2, NR>), dim3(a.n), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_fwd_prune_mr<1, NR>), dim3(a.n), dim3(64), 0, st, a);
      return hipGetLastError();
    });
  }
  // fp32 rows longer than 32 floats: one lane per live candidate (the
  // per-pivot walk of the general kernel costs more there; measured at
  // d = 96 and 960)
  if (kind != kU8L2 && a.pool.R <= 64 && a.pool.nch > 8) {
    GR_DISPATCH_N(max_iters, {
      if (kind == kF32L2) hipLaunchKernelGGL((k_fwd_prune_vec<kF32L2, NR>), dim3(a.n), dim3(64), 0, st, a);
      else hipLaunchKernelGGL((k_fwd_prune_vec<kF32IP, NR>), dim3(a.n), dim3(64), 0, st, a);
      return hipGetLastError();
    });
  }
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
  if constexpr (KIND != kU8L2 && NC == 2 && NP == 1) {
    if (a.pool.R <= 64) {
      static const uint32_t res = resident_blocks((const void *)k_rebuild_vec<KIND>);
      hipLaunchKernelGGL((k_rebuild_vec<KIND>), dim3(clamp_resident(grid, 2 * res)), dim3(64), 0, st, a);
      return;
    }
  }
  if constexpr (KIND == kU8L2 && NC == 2 && NP == 1) {
    // persistent waves, twice the resident workgroups: the second half
    // starts as the first ones finish, which evens out the work per wave
    if (a.pool.R <= 64 && a.pool.nch == 8) {
      static const uint32_t res = resident_blocks((const void *)k_rebuild_mr<2>);
      hipLaunchKernelGGL(k_rebuild_mr<2>, dim3(clamp_resident(grid, 2 * res)), dim3(64), 0, st, a);
      return;
    }
    if (a.pool.R <= 64 && a.pool.nch == 4) {
      static const uint32_t res = resident_blocks((const void *)k_rebuild_mr<1>);
      hipLaunchKernelGGL(k_rebuild_mr<1>, dim3(clamp_resident(grid, 2 * res)), dim3(64), 0, st, a);
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

bool adj_dists_apply(int kind, uint32_t R, int nch, uint32_t P) {
  return kind == kU8L2 && R <= 64 && R % 4 == 0 && (nch == 8 || nch == 4) && P <= 64 && R + P <= 128;
}

// One wave per row, lane s for list entry s: the exact uint8 squared
// distance of u and its s-th neighbour (0 for an empty slot).
__global__ void k_adj_dists(PoolView P) {
  const int ln = threadIdx.x & 63;
  const uint32_t w0 = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, nw = (gridDim.x * blockDim.x) >> 6;
  for (uint32_t u = w0; u < P.cap; u += nw) {
    if (ln >= (int)P.R) continue;
    const uint32_t v = P.adj[(size_t)u * P.R + ln];
    float d = 0.0f;
    if (kvalid(v) && v < P.cap) {
      const uint4 *x = reinterpret_cast<const uint4 *>(P.vecs + (size_t)u * P.stride);
      const uint4 *y = reinterpret_cast<const uint4 *>(P.vecs + (size_t)v * P.stride);
      uint32_t acc = 0;
      for (int c = 0; c < P.nch; c++) {
        const uint4 a = x[c], b = y[c];
        acc = udot4(a.x, a.x, acc);
        acc = udot4(a.y, a.y, acc);
        acc = udot4(a.z, a.z, acc);
        acc = udot4(a.w, a.w, acc);
        acc = u8l2_4(a, b, acc);  // + |b|^2 - 2 a.b
      }
      d = canon0((float)acc);
    }
    P.adjd[(size_t)u * P.R + ln] = d;
  }
}
hipError_t launch_adj_dists(PoolView p, hipStream_t s) {
  if (!p.adjd || p.cap == 0) return hipSuccess;
  size_t g = ((size_t)p.cap * 64 + 255) / 256;
  if (g > 16384) g = 16384;
  hipLaunchKernelGGL(k_adj_dists, dim3((uint32_t)g), dim3(256), 0, s, p);
  return hipGetLastError();
}

// Dirty nodes are rebuilt by the fast kernel when the row layout allows it
// (R <= 64, R a multiple of 4); the nodes it leaves, and every node
// otherwise, by the general kernel of the configuration.
hipError_t launch_rebuild(int kind, int vc, uint32_t R, uint32_t P, const RebuildArgs &a0, uint32_t grid,
                          hipStream_t st) {
  if (grid == 0) return hipSuccess;
  if (P > 128 || R + P > 256) return hipErrorInvalidValue;
  RebuildArgs a = a0;
  a.list = a0.dirty;
  a.list_n = &a0.ds->n_dirty;
  a.count_nodes = 1;
  if (R <= 64 && R % 4 == 0) {
    // grid >= min(records, 8192) >= the blocks needed at four nodes per wave
    hipLaunchKernelGGL(k_rebuild_fast, dim3(grid), dim3(64), 0, st, a);
    hipError_t e = launch_compact_flags(a.qflag, a.list, a.list_n, a0.flag_cap, a.queue, a.queue_n, a.scan_tmp, st);
    if (e != hipSuccess) return e;
    a.list = a0.queue;
    a.list_n = a0.queue_n;
    a.count_nodes = 0;
  }
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
