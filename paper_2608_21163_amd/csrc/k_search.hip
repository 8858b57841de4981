// k_search.hip -- BeamSearch (Alg. 1), one wavefront per query, and the
// brute-force candidate search that bootstraps an empty index.
//
// Search state of one wave:
//   C : the l closest (distance, id) keys seen so far, ascending, held in
//       registers as NR rows of 64 keys (element e = row*64 + lane); the top
//       id bit marks keys already expanded (the set V).
//   a lossy hash of ids whose distance was already evaluated, in LDS (16-bit
//       tags when the pool allows, so more waves fit per CU).  An
//       evaluated id either is in C or can never enter it again (the l-th
//       key only decreases once C is full), so skipping it is exact; the
//       hash may forget ids (they are then evaluated again and dropped by
//       the exact repeat check of the merge), but never reports an id that
//       was not evaluated.
// Each hop expands the smallest unexpanded key u, reads u's list (one slot
// per lane), drops ids found in the hash, gathers the remaining rows
// LPV lanes per row, and merges the new keys into C keeping the l smallest.
//
// Counting variant (EXACT): the hash is replaced by an exact visited bitmap
// per search in device memory, so every id is evaluated once and the
// evaluation count is the number of distinct ids whose distance the search
// needs ({start} and every neighbour of an expanded node).  The expansion
// order, and so C and V, are the same as with the hash (the hash only skips
// recomputation), which makes this variant a measurement of the method's
// own work.  It is launched only when counting is enabled.
#include "dispatch.h"

namespace gr {

constexpr int kHashBits = 11;
constexpr int kHashSize = 1 << kHashBits;
constexpr int kHashBits8 = 12;  // 8-bit tags: twice the slots in the same bytes

// Hash of evaluated ids.  With 8- or 16-bit entries an id v is split into a
// tag (v >> bits) and a slot ((v ^ tag * odd) & mask); tag and slot together
// determine v, so a stored tag matching the probe's tag is an exact hit.  The
// all-ones tag marks an empty slot, so the 8-bit form (4096 slots) needs ids
// below 0xFF << 12 and the 16-bit form (2048 slots) ids below 0xFFFF << 11;
// larger pools store whole 32-bit ids at a multiplicative hash slot.  Both
// narrow forms take 4 KB of LDS.
template <class HW> struct IdHash;
template <> struct IdHash<uint8_t> {
  static constexpr int kBits = kHashBits8;
  static constexpr int kSlots = 1 << kBits;
  static __device__ __forceinline__ uint32_t slot(uint32_t v) {
    return (v ^ ((v >> kBits) * 40503u)) & ((1u << kBits) - 1u);
  }
  static __device__ __forceinline__ uint8_t word(uint32_t v) { return (uint8_t)(v >> kBits); }
  static constexpr uint8_t kEmpty = 0xFFu;
};
template <> struct IdHash<uint16_t> {
  static constexpr int kBits = kHashBits;
  static constexpr int kSlots = 1 << kBits;
  static __device__ __forceinline__ uint32_t slot(uint32_t v) {
    return (v ^ ((v >> kHashBits) * 40503u)) & (kHashSize - 1);
  }
  static __device__ __forceinline__ uint16_t word(uint32_t v) { return (uint16_t)(v >> kHashBits); }
  static constexpr uint16_t kEmpty = 0xFFFFu;
};
template <> struct IdHash<uint32_t> {
  static constexpr int kBits = kHashBits;
  static constexpr int kSlots = 1 << kBits;
  static __device__ __forceinline__ uint32_t slot(uint32_t v) { return (v * 0x9E3779B1u) >> (32 - kHashBits); }
  static __device__ __forceinline__ uint32_t word(uint32_t v) { return v; }
  static constexpr uint32_t kEmpty = kInvalid;
};
bool hash16_ok(uint32_t cap) { return (uint64_t)cap <= ((uint64_t)0xFFFFu << kHashBits); }
bool hash8_ok(uint32_t cap) { return (uint64_t)cap <= ((uint64_t)0xFFu << kHashBits8); }

// 8-bit tags in S slots, S not necessarily a power of two: with t = v / S
// and r = v % S, v goes to slot (r + t * odd) % S and stores t.  Slot and tag
// determine v; tag 0xFF marks an empty slot, so ids must be below 255 * S.
// The searches of l <= 128 are held to five or six waves per SIMD by their
// registers, which leaves LDS for more slots than 4096 at no occupancy
// cost: 6144 slots for l in (64, 128] (7.5 KB a wave, 21 waves per CU) and
// 5120 for l <= 64 (6 KB, 26 waves per CU).  At 1M x 128 the 6144 slots cut
// the rows an insert search evaluates again from 24% to 18%.
template <int S> struct Slots8 {};
template <int S> struct IdHash<Slots8<S>> {
  static constexpr int kSlots = S;
  static __device__ __forceinline__ uint32_t slot(uint32_t v) {
    const uint32_t t = v / (uint32_t)S, r = v - t * (uint32_t)S;
    return (r + t * 2654435u) % (uint32_t)S;
  }
  static __device__ __forceinline__ uint8_t word(uint32_t v) { return (uint8_t)(v / (uint32_t)S); }
  static constexpr uint8_t kEmpty = 0xFFu;
};
template <int S> bool slots8_ok(uint32_t cap) { return (uint64_t)cap <= 255ull * S; }

template <int KIND, int LPV, int CPL, int NR, class HW, bool EXACT>
__device__ __forceinline__ void search_one(SearchArgs a) {
  typedef IdHash<HW> H;
  typedef decltype(H::word(0u)) Word;
  constexpr int kSlots = H::kSlots;
  __shared__ Word hsh[kSlots];
  // the merge's scratch; its first 64 entries also hold a hop's new ids and
  // their distances (read into registers before the merge writes)
  __shared__ uint32_t mid[64 * NR];
  __shared__ float mkey[64 * NR];
  uint32_t *const nid = mid;
  float *const nkey = mkey;
  const int ln = lane();
  const uint32_t qi = blockIdx.x;
  if (qi >= a.nq) return;
  const PoolView &P = a.pool;
  const uint8_t *qrow = a.qids ? P.vecs + (size_t)a.qids[qi] * P.stride : a.qbase + (size_t)qi * P.stride;
  const uint32_t start = a.start_ptr ? *a.start_ptr : a.start;
  Slice<KIND, LPV, CPL> s;
  load_slice<KIND, LPV, CPL>(s, qrow, P.nch);
  uint32_t *vrow = EXACT ? a.vis + (size_t)qi * a.vis_words : nullptr;
  if (!EXACT)
    for (int i = ln; i < kSlots; i += 64) hsh[i] = H::kEmpty;

  float cd[NR];
  uint32_t ci[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) { cd[r] = finf(); ci[r] = kInvalid; }
  if (start < P.cap) {  // an invalid start leaves C empty: no expansion
    const float d0 = wave_dist1<KIND, LPV, CPL>(s, P.vecs + (size_t)start * P.stride, P.nch);
    if (ln == 0) { cd[0] = d0; ci[0] = start; }
  }
  __syncthreads();
  if (ln == 0 && start < P.cap) {
    if (EXACT) atomicOr(&vrow[start >> 5], 1u << (start & 31));
    else hsh[H::slot(start)] = H::word(start);
  }
  __syncthreads();
  uint32_t nv = 0, evals = 1;
  // V in expansion order, written out 64 entries at a time: lane j holds the
  // entry of the hop nv with nv % 64 == j until its group of 64 is complete
  // (one store per 64 hops, so the waits for the lists of the others do not
  // also wait for stores)
  uint32_t vq = 0;
  float vdq = 0.0f;

  while (nv < a.max_iters) {
    // u = argmin over C \ V
    int e = -1;
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint64_t m = ballot(kvalid(ci[r]) && !(ci[r] & kVisit));
      if (e < 0 && m) e = r * 64 + ffs64(m);
    }
    if (e < 0) break;
    const int er = e >> 6, el = e & 63;
    uint32_t u = 0;
    float du = 0.0f;
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (r == er) {
        u = rdlane(ci[r], el) & kIdMask;
        du = rdlane(cd[r], el);
        if (ln == el) ci[r] |= kVisit;
      }
    if (a.v_ids) {
      if (ln == (int)(nv & 63u)) {
        vq = u;
        vdq = du;
      }
      if ((nv & 63u) == 63u) {
        const size_t o = (size_t)qi * a.v_stride + (nv - 63u) + (uint32_t)ln;
        a.v_ids[o] = vq;
        a.v_d[o] = vdq;
      }
    }
    nv++;
    // C <- C u N_out(u), skipping ids already evaluated
    const uint32_t v = ln < (int)P.R ? P.adj[(size_t)u * P.R + ln] : kInvalid;
    bool need;
    if (EXACT) {
      need = false;
      if (v != kInvalid) {
        const uint32_t bit = 1u << (v & 31);
        need = !(atomicOr(&vrow[v >> 5], bit) & bit);
      }
      __syncthreads();
    } else {
      const uint32_t hs = H::slot(v);
      const Word hw = H::word(v);
      need = v != kInvalid && hsh[hs] != hw;
      __syncthreads();
      if (need) hsh[hs] = hw;
    }
    const uint64_t m = ballot(need);
    const int cnt = popc(m);
    if (cnt == 0) continue;
    if (need) nid[mbcnt(m)] = v;
    __syncthreads();
    wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, nid, nkey, cnt);
    __syncthreads();
    evals += cnt;
    const float nd = ln < cnt ? nkey[ln] : finf();
    const uint32_t ni = ln < cnt ? nid[ln] : kInvalid;
    wave_merge_lds<NR>(cd, ci, nd, ni, (int)a.ell, mkey, mid);
    __syncthreads();
  }

  if (a.v_ids && ln < (int)(nv & 63u)) {  // the last, incomplete group
    const size_t o = (size_t)qi * a.v_stride + (nv & ~63u) + (uint32_t)ln;
    a.v_ids[o] = vq;
    a.v_d[o] = vdq;
  }
  if (a.v_n && ln == 0) a.v_n[qi] = nv;
  if (a.c_ids && a.c_by_id) {
    // the same set in ascending id order (delete repair candidates), through
    // LDS and a wave sort by id
    int base = 0;
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint32_t id = ci[r] & kIdMask;
      const bool ok = kvalid(ci[r]) && !(a.c_filter && a.c_filter[id]);
      const uint64_t mm = ballot(ok);
      const int pos = base + mbcnt(mm);
      if (ok && pos < (int)a.c_out) mid[pos] = id;
      base += popc(mm);
    }
    __syncthreads();
    const int m = base < (int)a.c_out ? base : (int)a.c_out;
    float sd[1] = {ln < m ? 0.0f : finf()};
    uint32_t si[1] = {ln < m ? mid[ln] : kInvalid};
    wave_sort<1>(sd, si);
    if (ln < (int)a.c_out) a.c_ids[(size_t)qi * a.c_out + ln] = si[0];
  } else if (a.c_ids) {
    int base = 0;
#pragma unroll
    for (int r = 0; r < NR; r++) {
      const uint32_t id = ci[r] & kIdMask;
      const bool ok = kvalid(ci[r]) && !(a.c_filter && a.c_filter[id]);
      const uint64_t mm = ballot(ok);
      const int pos = base + mbcnt(mm);
      if (ok && pos < (int)a.c_out) {
        a.c_ids[(size_t)qi * a.c_out + pos] = id;
        a.c_d[(size_t)qi * a.c_out + pos] = cd[r];
      }
      base += popc(mm);
    }
    for (int t = base + ln; t < (int)a.c_out; t += 64) {
      a.c_ids[(size_t)qi * a.c_out + t] = kInvalid;
      a.c_d[(size_t)qi * a.c_out + t] = finf();
    }
  }
  // stopped by the expansion cap with unexpanded keys left in C
  bool open = false;
#pragma unroll
  for (int r = 0; r < NR; r++) open |= ballot(kvalid(ci[r]) && !(ci[r] & kVisit)) != 0;
  if (ln == 0) {
    if (EXACT) {
      stat_add(a.ds, kStDistinct + a.which, (unsigned long long)evals);
    } else {
      stat_add(a.ds, kStHops + a.which, (unsigned long long)nv);
      stat_add(a.ds, kStEvals + a.which, (unsigned long long)evals);
      if (open && nv >= a.max_iters) stat_add(a.ds, kStCapped + a.which, 1ull);
    }
  }
}

template <int KIND, int LPV, int CPL, int NR, class HW, bool EXACT>
__global__ __launch_bounds__(64) void k_search(SearchArgs a) {
  search_one<KIND, LPV, CPL, NR, HW, EXACT>(a);
}

// Empty index at the start of a batch: the candidates of each new point are
// its `want` nearest other points of the batch, by brute force over the
// batch, kept sorted by (distance, id).
template <int KIND, int LPV, int CPL, int NR>
__global__ __launch_bounds__(64) void k_bootstrap(BootArgs a) {
  __shared__ uint32_t nid[64];
  __shared__ float nkey[64];
  const int ln = lane();
  const uint32_t i = blockIdx.x;
  if (i >= a.n) return;
  const PoolView &P = a.pool;
  const uint32_t p = a.ids[i];
  Slice<KIND, LPV, CPL> s;
  load_slice<KIND, LPV, CPL>(s, P.vecs + (size_t)p * P.stride, P.nch);
  float cd[NR];
  uint32_t ci[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) { cd[r] = finf(); ci[r] = kInvalid; }
  for (uint32_t base = 0; base < a.n; base += 64) {
    const uint32_t j = base + ln;
    const bool ok = j < a.n && j != i;
    const uint32_t v = j < a.n ? a.ids[j] : kInvalid;
    const uint64_t m = ballot(ok);
    const int cnt = popc(m);
    if (ok) nid[mbcnt(m)] = v;
    __syncthreads();
    wave_dists<KIND, LPV, CPL>(s, P.vecs, P.stride, P.nch, nid, nkey, cnt);
    __syncthreads();
    const float nd = ln < cnt ? nkey[ln] : finf();
    const uint32_t ni = ln < cnt ? nid[ln] : kInvalid;
    wave_merge_new_fast<NR>(cd, ci, nd, ni, (int)a.want);
    __syncthreads();
  }
  const uint32_t got = a.n - 1 < a.want ? a.n - 1 : a.want;
#pragma unroll
  for (int r = 0; r < NR; r++) {
    const int e = r * 64 + ln;
    if (e < (int)a.o_stride) {
      a.o_ids[(size_t)i * a.o_stride + e] = (uint32_t)e < got ? (ci[r] & kIdMask) : kInvalid;
      a.o_d[(size_t)i * a.o_stride + e] = (uint32_t)e < got ? cd[r] : finf();
    }
  }
  if (a.o_n && ln == 0) a.o_n[i] = got;
}

int vec_class(int nch) {
  if (nch <= 8) return kVcA;
  if (nch <= 32) return kVcB;
  if (nch <= 256) return kVcC;
  return -1;
}

hipError_t launch_search(int kind, int vc, const SearchArgs &a, hipStream_t st) {
  if (a.nq == 0) return hipSuccess;
  const bool h8 = hash8_ok(a.pool.cap), h16 = hash16_ok(a.pool.cap);
  GR_DISPATCH_KV(kind, vc, GR_DISPATCH_N(a.ell, {
    if (a.vis) hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, uint8_t, true>), dim3(a.nq), dim3(64), 0, st, a);
    else if (NR == 2 && slots8_ok<6144>(a.pool.cap))
      hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, Slots8<6144>, false>), dim3(a.nq), dim3(64), 0, st, a);
    else if (NR == 1 && slots8_ok<5120>(a.pool.cap))
      hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, Slots8<5120>, false>), dim3(a.nq), dim3(64), 0, st, a);
    else if (h8) hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, uint8_t, false>), dim3(a.nq), dim3(64), 0, st, a);
    else if (h16) hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, uint16_t, false>), dim3(a.nq), dim3(64), 0, st, a);
    else hipLaunchKernelGGL((k_search<KIND, LPV, CPL, NR, uint32_t, false>), dim3(a.nq), dim3(64), 0, st, a);
    return hipGetLastError();
  }));
  return hipErrorInvalidValue;
}

hipError_t launch_bootstrap(int kind, int vc, const BootArgs &a, hipStream_t st) {
  if (a.n == 0) return hipSuccess;
  GR_DISPATCH_KV(kind, vc, GR_DISPATCH_N(a.want, {
    hipLaunchKernelGGL((k_bootstrap<KIND, LPV, CPL, NR>), dim3(a.n), dim3(64), 0, st, a);
    return hipGetLastError();
  }));
  return hipErrorInvalidValue;
}

}  // namespace gr
