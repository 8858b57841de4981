// k_cagra.hip -- GrAND-CAGRA updates (Alg. 7 and Alg. 8) on a fixed
// out-degree graph whose slot order is meaningful (slot 0 = closest).
//
// Insert (Alg. 7): N_out(p_i) is the R closest results of the search; the
// reverse edge q -> p_i replaces, in q's list, the element of
// N_out(q) n N_out(p_i) at the highest slot (the detour q -> p_i -> r
// remains), or fills q's first free slot.  Slots are updated with an atomic
// compare-and-swap.  Grouped mode: records are grouped per target and one
// wavefront applies them in (distance, p_i) order, so the result is
// deterministic.  Racing mode: one wavefront per record, concurrent
// compare-and-swap with re-reads on failure (lock-free, last writer wins).
//
// Delete (Alg. 8): for each u in N_in(B) \ B, each slot holding a deleted p
// (in slot order) is replaced by PickOne(N_out(p), u): a cyclic scan of p's
// valid entries starting at (rank of u among p's in-neighbours) mod |N_out(p)|
// for the first r outside the batch, r != u, r not already in u's list;
// INVALID if there is none.  No distances are computed.
#include "dispatch.h"

namespace gr {

__device__ __forceinline__ uint32_t load_acq(const uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Forward lists from the search results; records (q, p_i, dist) for q in
// N_out(p_i).
__global__ void k_cagra_fwd(PoolView P, const uint32_t *ids, uint32_t n, const uint32_t *c_ids, const float *c_d,
                            uint32_t *rec_t, uint32_t *rec_s, float *rec_d) {
  const uint32_t i = blockIdx.x;
  if (i >= n) return;
  const int ln = threadIdx.x;
  const uint32_t p = ids[i];
  if (ln < (int)P.R) {
    const uint32_t q = c_ids[(size_t)i * P.R + ln];
    P.adj[(size_t)p * P.R + ln] = q;
    rec_t[(size_t)i * P.R + ln] = q;
    rec_s[(size_t)i * P.R + ln] = p;
    rec_d[(size_t)i * P.R + ln] = c_d[(size_t)i * P.R + ln];
  }
  const uint64_t m = ballot(ln < (int)P.R && c_ids[(size_t)i * P.R + (ln < (int)P.R ? ln : 0)] != kInvalid);
  if (ln == 0) P.deg[p] = (uint32_t)popc(m);
}
hipError_t launch_cagra_fwd(PoolView p, const uint32_t *ids, uint32_t n, const uint32_t *c_ids, const float *c_d,
                            uint32_t *rec_t, uint32_t *rec_s, float *rec_d, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_cagra_fwd, dim3(n), dim3(64), 0, s, p, ids, n, c_ids, c_d, rec_t, rec_s, rec_d);
  return hipGetLastError();
}

// One reverse edge q -> p against q's row held by lane s in rv; fl4 (LDS,
// 64 ids, INVALID past R) holds N_out(p).  Returns the new value of this
// lane's slot.
__device__ __forceinline__ uint32_t detour_one(const CagraArgs &a, uint32_t q, uint32_t p, uint32_t rv,
                                               const uint4 *fl4) {
  const int ln = lane();
  const PoolView &P = a.pool;
  const bool inrow = ln < (int)P.R;
  if (ballot(inrow && rv == p)) return rv;
  const uint64_t fr = ballot(inrow && rv == kInvalid);
  if (fr) {
    const int s = ffs64(fr);
    if (ln == s) {
      atomicCAS(&P.adj[(size_t)q * P.R + s], kInvalid, p);
      return p;
    }
    return rv;
  }
  // this lane's entry is in N_out(p): 16-byte LDS reads, all lanes at the
  // same address
  bool mem = false;
#pragma unroll 4
  for (int t = 0; t < 16; t++) {
    const uint4 f = fl4[t];
    mem = mem | (f.x == rv) | (f.y == rv) | (f.z == rv) | (f.w == rv);
  }
  mem = mem && inrow && rv != kInvalid;
  const uint64_t mm = ballot(mem);
  if (mm) {
    const int s = fls64(mm);
    if (ln == s) {
      atomicCAS(&P.adj[(size_t)q * P.R + s], rv, p);
      return p;
    }
  }
  return rv;
}

__global__ __launch_bounds__(64) void k_cagra_detour(CagraArgs a) {
  constexpr int kFwdStage = 4;  // forward lists of records loaded together
  __shared__ uint4 fl4[kFwdStage][16];
  const int ln = lane();
  const PoolView &P = a.pool;
  const uint32_t nt = a.ds->n_dirty;
  uint32_t nodes = 0;
  for (uint32_t it = blockIdx.x; it < nt; it += gridDim.x) {
    const uint32_t q = a.list[it];
    const uint32_t g0 = a.goff[q], g1 = a.goff[q + 1];
    uint32_t rv = ln < (int)P.R ? P.adj[(size_t)q * P.R + ln] : kInvalid;
    // records in (dist, src) order: repeatedly take the 64 smallest keys
    // above the last one applied
    float lastd = -finf();
    uint32_t lasti = 0;
    bool first = true;
    uint32_t done = 0;
    while (done < g1 - g0) {
      float cd[1] = {finf()};
      uint32_t ci[1] = {kInvalid};
      for (uint32_t base = g0; base < g1; base += 64) {
        const uint32_t j = base + ln;
        float d = j < g1 ? a.gd[j] : finf();
        uint32_t s = j < g1 ? a.gsrc[j] : kInvalid;
        if (j >= g1 || (!first && !kless(lastd, lasti, d, s))) { d = finf(); s = kInvalid; }
        wave_merge_new_fast<1>(cd, ci, d, s, 64);
      }
      const int nb = popc(ballot(kvalid(ci[0])));
      if (nb == 0) break;
      for (int t0 = 0; t0 < nb; t0 += kFwdStage) {
        // N_out of the next kFwdStage records' sources, loaded together:
        // lane (h, part) copies 4 ids of record t0 + h
        {
          const int h = ln >> 4, part = ln & 15;
          const int t = t0 + h;
          const uint32_t p = (uint32_t)__shfl((int)ci[0], t < nb ? t : t0, 64);  // per-lane source lane
          uint4 v = make_uint4(kInvalid, kInvalid, kInvalid, kInvalid);
          if (t < nb && 4 * part < (int)P.R) {
            const uint32_t *row = a.fwd + (size_t)a.bidx[p] * P.R + 4 * part;
            if ((P.R & 3u) == 0) {
              v = *reinterpret_cast<const uint4 *>(row);
            } else {  // rows not 16-byte aligned: word loads, INVALID past R
              const int e = 4 * part;
              v.x = row[0];
              v.y = e + 1 < (int)P.R ? row[1] : kInvalid;
              v.z = e + 2 < (int)P.R ? row[2] : kInvalid;
              v.w = e + 3 < (int)P.R ? row[3] : kInvalid;
            }
          }
          fl4[h][part] = v;
        }
        __syncthreads();
        for (int h = 0; h < kFwdStage && t0 + h < nb; h++) {
          const uint32_t p = rdlane(ci[0], t0 + h);
          rv = detour_one(a, q, p, rv, fl4[h]);
        }
        __syncthreads();
      }
      lastd = rdlane(cd[0], nb - 1);
      lasti = rdlane(ci[0], nb - 1);
      first = false;
      done += nb;
    }
    const uint64_t m = ballot(ln < (int)P.R && rv != kInvalid);
    if (ln == 0) P.deg[q] = (uint32_t)popc(m);
    nodes++;
    __syncthreads();
  }
  if (ln == 0 && nodes) stat_add(a.ds, kStDirty, (unsigned long long)nodes);  // one counter update per wave
}
hipError_t launch_cagra_detour(const CagraArgs &a, uint32_t grid, hipStream_t s) {
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_cagra_detour, dim3(grid), dim3(64), 0, s, a);
  return hipGetLastError();
}

// Racing mode: every record independently; a failed compare-and-swap means
// another writer changed the slot, so the row is re-read and the decision
// retaken (bounded number of attempts).
__global__ __launch_bounds__(64) void k_cagra_racing(CagraArgs a) {
  __shared__ uint32_t fl[64];
  const int ln = lane();
  const PoolView &P = a.pool;
  const bool inrow = ln < (int)P.R;
  for (uint32_t it = blockIdx.x; it < a.nrec; it += gridDim.x) {
    const uint32_t q = a.rec_t[it], p = a.rec_s[it];
    if (q == kInvalid) continue;
    const uint32_t bi = a.bidx[p];
    fl[ln] = inrow ? a.fwd[(size_t)bi * P.R + ln] : kInvalid;
    __syncthreads();
    for (uint32_t attempt = 0; attempt < 2 * P.R + 2; attempt++) {
      const uint32_t rv = inrow ? load_acq(&P.adj[(size_t)q * P.R + ln]) : kInvalid;
      if (ballot(inrow && rv == p)) break;
      uint64_t cand = ballot(inrow && rv == kInvalid);
      int s;
      if (cand) {
        s = ffs64(cand);
      } else {
        bool mem = false;
        for (uint32_t t = 0; t < P.R; t++) mem = mem || (inrow && rv != kInvalid && fl[t] == rv);
        cand = ballot(mem);
        if (!cand) break;
        s = fls64(cand);
      }
      uint32_t ok = 0;
      if (ln == s) ok = atomicCAS(&P.adj[(size_t)q * P.R + s], rv, p) == rv ? 1u : 0u;
      if (rdlane(ok, s)) break;
    }
    __syncthreads();
  }
}
__global__ void k_cagra_degree(PoolView P) {
  const uint32_t u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= P.cap || !P.active[u]) return;
  uint32_t d = 0;
  for (uint32_t t = 0; t < P.R; t++) d += P.adj[(size_t)u * P.R + t] != kInvalid ? 1u : 0u;
  P.deg[u] = d;
}
hipError_t launch_cagra_racing(const CagraArgs &a, hipStream_t s) {
  if (a.nrec == 0) return hipSuccess;
  uint32_t g = a.nrec < 16384 ? a.nrec : 16384;
  hipLaunchKernelGGL(k_cagra_racing, dim3(g), dim3(64), 0, s, a);
  hipLaunchKernelGGL(k_cagra_degree, dim3((a.pool.cap + 255) / 256), dim3(256), 0, s, a.pool);
  return hipGetLastError();
}

// u in N_in(B) \ B, each once (epoch-stamped marks), appended to `list`.
__global__ void k_cagra_affected(const uint32_t *ids, uint32_t n, const uint8_t *in_batch, const uint32_t *rev_off,
                                 const uint32_t *rev_src, int by_batch, uint32_t *mark, uint32_t epoch,
                                 uint32_t *list, DevScalars *ds) {
  const uint32_t i = blockIdx.x;
  if (i >= n) return;
  const uint32_t row = by_batch ? i : ids[i];
  const uint32_t b0 = rev_off[row], b1 = rev_off[row + 1];
  for (uint32_t base = b0; base < b1; base += 64) {
    const uint32_t j = base + lane();
    const uint32_t z = j < b1 ? rev_src[j] : kInvalid;
    const bool add = z != kInvalid && !in_batch[z] && atomicExch(&mark[z], epoch) != epoch;
    // one list reservation per wave
    const uint64_t m = ballot(add);
    if (!m) continue;
    const int l0 = ffs64(m);
    uint32_t at = 0;
    if (lane() == l0) at = atomicAdd(&ds->n_dirty, (uint32_t)popc(m));
    at = rdlane(at, l0);
    if (add) list[at + (uint32_t)mbcnt(m)] = z;
  }
}
__global__ void k_zero_ndirty2(DevScalars *ds) { ds->n_dirty = 0; }
hipError_t launch_cagra_affected(const uint32_t *ids, uint32_t n, const uint8_t *in_batch, const uint32_t *rev_off,
                                 const uint32_t *rev_src, int by_batch, uint32_t *mark, uint32_t epoch,
                                 uint32_t *list, DevScalars *ds, hipStream_t s) {
  hipLaunchKernelGGL(k_zero_ndirty2, dim3(1), dim3(1), 0, s, ds);
  if (n == 0) return hipGetLastError();
  hipLaunchKernelGGL(k_cagra_affected, dim3(n), dim3(64), 0, s, ids, n, in_batch, rev_off, rev_src, by_batch, mark,
                     epoch, list, ds);
  return hipGetLastError();
}

__global__ __launch_bounds__(64) void k_cagra_pickone(CagraArgs a) {
  __shared__ uint32_t lc[64];
  __shared__ uint8_t lcb[64];  // batch flags of lc
  __shared__ uint4 uL[16];  // u's current row, for the membership test
  const int ln = lane();
  const PoolView &P = a.pool;
  const bool inrow = ln < (int)P.R;
  const uint32_t nt = *a.list_n;
  uint32_t nodes = 0;
  // the next entry of this wave is read during the current one; u's row is
  // loaded beside the mark that decides whether u is taken
  uint32_t u_next = blockIdx.x < nt ? a.list[blockIdx.x] : 0u;
  for (uint32_t it = blockIdx.x; it < nt; it += gridDim.x) {
    const uint32_t u = u_next;
    u_next = a.list[it + gridDim.x < nt ? it + gridDim.x : it];
    uint32_t rv = P.adj[(size_t)(u != kInvalid ? u : 0u) * P.R + (inrow ? ln : 0)];
    if (!inrow) rv = kInvalid;
    if (a.dedupe) {
      bool take = false;
      if (ln == 0) take = u != kInvalid && !a.in_batch[u] && atomicExch(&a.mark[u], a.epoch) != a.epoch;
      if (!__shfl((int)take, 0, 64)) continue;
    }
    reinterpret_cast<uint32_t *>(uL)[ln] = rv;
    // slots holding a deleted out-neighbour, found with one parallel lookup;
    // they are then handled in slot order (replacements only ever put
    // non-deleted ids into the row, so the set does not change)
    uint64_t dels = ballot(rv != kInvalid && a.in_batch[rv] != 0);
    while (dels) {
      const uint32_t s = (uint32_t)ffs64(dels);
      dels &= dels - 1;
      const uint32_t p = rdlane(rv, (int)s);
      // valid entries of N_out(p) in slot order (p's row is not edited here)
      // with their batch flags, and p's reverse row: the loads that do not
      // depend on each other are issued together
      const uint32_t lv = inrow ? P.adj[(size_t)p * P.R + ln] : kInvalid;
      const uint32_t row = a.rev_by_batch ? a.bidx[p] : p;
      const uint32_t b0 = a.rev_off[row], b1 = a.rev_off[row + 1];
      const bool lvb = a.in_batch[lv != kInvalid ? lv : 0u] != 0;
      const uint64_t vm = ballot(lv != kInvalid);
      const int nl = popc(vm);
      if (lv != kInvalid) {
        lc[mbcnt(vm)] = lv;
        lcb[mbcnt(vm)] = lvb ? 1 : 0;
      }
      // rank of u among p's in-neighbours (rows hold distinct sources)
      uint32_t below = 0;
      for (uint32_t j = b0 + ln; j < b1; j += 64) below += a.rev_src[j] < u ? 1u : 0u;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) below += __shfl_xor(below, o, 64);
      __syncthreads();
      uint32_t chosen = kInvalid;
      if (nl > 0) {
        const uint32_t start = below % (uint32_t)nl;
        uint32_t r = kInvalid;
        bool ok = false;
        if (ln < nl) {
          const uint32_t e = (start + (uint32_t)ln) % (uint32_t)nl;
          r = lc[e];
          ok = !lcb[e] && r != u;
        }
        // r must not already be in u's row (16-byte LDS reads, all lanes
        // at the same address)
#pragma unroll 4
        for (int t = 0; t < 16; t++) {
          const uint4 q = uL[t];
          ok = ok & (q.x != r) & (q.y != r) & (q.z != r) & (q.w != r);
        }
        const uint64_t om = ballot(ok);
        if (om) chosen = rdlane(r, ffs64(om));
      }
      if (ln == (int)s) {
        atomicCAS(&P.adj[(size_t)u * P.R + s], p, chosen);
        rv = chosen;
        reinterpret_cast<uint32_t *>(uL)[ln] = chosen;
      }
      __syncthreads();
    }
    const uint64_t m = ballot(inrow && rv != kInvalid);
    if (ln == 0) P.deg[u] = (uint32_t)popc(m);
    nodes++;
  }
  if (ln == 0 && nodes) stat_add(a.ds, kStDirty, (unsigned long long)nodes);  // one counter update per wave
}
hipError_t launch_cagra_pickone(const CagraArgs &a, uint32_t grid, hipStream_t s) {
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_cagra_pickone, dim3(grid), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace gr
