// k_graph.hip -- integer graph kernels: validation, staging of new rows,
// grouping of reverse-edge records by target (counting sort: histogram,
// prefix scan, scatter), the on-demand reverse graph in CSR form (Alg. 8,
// first two loops), clearing deleted rows, and the medoid.
#include <algorithm>

#include "dispatch.h"

namespace gr {

static inline uint32_t blocks_for(size_t n, uint32_t per) {
  size_t b = (n + per - 1) / per;
  if (b > 1u << 30) b = 1u << 30;
  return (uint32_t)(b == 0 ? 1 : b);
}

// ---------------------------------------------------------------- fills
__global__ void k_fill_u32(uint32_t *p, uint32_t v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}
__global__ void k_fill_u8(uint8_t *p, uint8_t v, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}
hipError_t launch_fill_u32(uint32_t *p, uint32_t v, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  uint32_t g = blocks_for(n, 256);
  if (g > 65536) g = 65536;
  hipLaunchKernelGGL(k_fill_u32, dim3(g), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}
hipError_t launch_fill_u8(uint8_t *p, uint8_t v, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  uint32_t g = blocks_for(n, 256);
  if (g > 65536) g = 65536;
  hipLaunchKernelGGL(k_fill_u8, dim3(g), dim3(256), 0, s, p, v, n);
  return hipGetLastError();
}

static __device__ void set_error(DevScalars *ds, uint32_t code, uint32_t id) {
  if (atomicCAS(&ds->err_code, 0u, code) == 0u) ds->err_id = id;
}

// ---------------------------------------------------------------- validation
// ids in range, not repeated within the batch (epoch-stamped marks), and
// in the expected active state.
__global__ void k_validate_ids(const uint32_t *ids, uint32_t n, uint32_t cap, const uint8_t *active, uint32_t *mark,
                               uint32_t epoch, int want_active, DevScalars *ds) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t id = ids[i];
  if (id >= cap) { set_error(ds, kErrRange, id); return; }
  if (atomicExch(&mark[id], epoch) == epoch) { set_error(ds, kErrRepeat, id); return; }
  if ((active[id] != 0) != (want_active != 0)) set_error(ds, kErrState, id);
}
hipError_t launch_validate_ids(const uint32_t *ids, uint32_t n, uint32_t cap, const uint8_t *active, uint32_t *mark,
                               uint32_t epoch, int want_active, DevScalars *ds, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_validate_ids, dim3(blocks_for(n, 256)), dim3(256), 0, s, ids, n, cap, active, mark, epoch,
                     want_active, ds);
  return hipGetLastError();
}

__global__ void k_check_finite(const uint8_t *rows, uint32_t n, size_t stride, uint32_t dim, DevScalars *ds) {
  const size_t total = (size_t)n * dim;
  for (size_t t = blockIdx.x * (size_t)blockDim.x + threadIdx.x; t < total; t += (size_t)gridDim.x * blockDim.x) {
    const size_t r = t / dim, c = t % dim;
    const float x = reinterpret_cast<const float *>(rows + r * stride)[c];
    if (!isfinite(x)) set_error(ds, kErrNonFinite, (uint32_t)r);
  }
}
hipError_t launch_check_finite(const uint8_t *rows, uint32_t n, size_t stride, uint32_t dim, DevScalars *ds,
                               hipStream_t s) {
  if (n == 0) return hipSuccess;
  uint32_t g = blocks_for((size_t)n * dim, 256);
  if (g > 16384) g = 16384;
  hipLaunchKernelGGL(k_check_finite, dim3(g), dim3(256), 0, s, rows, n, stride, dim, ds);
  return hipGetLastError();
}

__global__ void k_mips_augment(uint8_t *rows, size_t n, size_t stride, uint32_t dim, double M2, DevScalars *ds) {
  for (size_t r = blockIdx.x * (size_t)blockDim.x + threadIdx.x; r < n; r += (size_t)gridDim.x * blockDim.x) {
    float *x = reinterpret_cast<float *>(rows + r * stride);
    double s = 0.0;
    for (uint32_t j = 0; j < dim; j++) s = __builtin_fma((double)x[j], (double)x[j], s);
    if (s > M2) set_error(ds, kErrNorm, (uint32_t)r);
    const double t = M2 - s;
    x[dim] = (float)sqrt(t > 0.0 ? t : 0.0);
  }
}
hipError_t launch_mips_augment(uint8_t *rows, size_t n, size_t stride, uint32_t dim, float M, DevScalars *ds,
                               hipStream_t s) {
  if (n == 0) return hipSuccess;
  uint32_t g = blocks_for(n, 64);
  if (g > 65535) g = 65535;
  hipLaunchKernelGGL(k_mips_augment, dim3(g), dim3(64), 0, s, rows, n, stride, dim, (double)M * (double)M, ds);
  return hipGetLastError();
}

// ---------------------------------------------------------------- staging
// Alg. 5 / Alg. 7 first loop: write x_i into slot p_i, empty its list, mark
// it active; remember each id's batch position.  One wave per new point.
__global__ void k_stage(PoolView P, const uint8_t *rows, const uint32_t *ids, uint32_t n, uint32_t *bidx) {
  const uint32_t i = blockIdx.x;
  if (i >= n) return;
  const int ln = threadIdx.x;
  const uint32_t id = ids[i];
  const uint4 *src = reinterpret_cast<const uint4 *>(rows + (size_t)i * P.stride);
  uint4 *dst = reinterpret_cast<uint4 *>(P.vecs + (size_t)id * P.stride);
  for (int c = ln; c < P.nch; c += 64) dst[c] = src[c];
  if (ln < (int)P.R) P.adj[(size_t)id * P.R + ln] = kInvalid;
  if (ln == 0) {
    P.deg[id] = 0;
    P.active[id] = 1;
    bidx[id] = i;
  }
}
hipError_t launch_stage(PoolView p, const uint8_t *rows, const uint32_t *ids, uint32_t n, uint32_t *bidx,
                        hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_stage, dim3(n), dim3(64), 0, s, p, rows, ids, n, bidx);
  return hipGetLastError();
}

__global__ void k_mark_batch(const uint32_t *ids, uint32_t n, uint8_t *in_batch, uint32_t *bidx, uint8_t v) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  in_batch[ids[i]] = v;
  if (bidx) bidx[ids[i]] = i;
}
hipError_t launch_mark_batch(const uint32_t *ids, uint32_t n, uint8_t *in_batch, uint32_t *bidx, uint8_t v,
                             hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_mark_batch, dim3(blocks_for(n, 256)), dim3(256), 0, s, ids, n, in_batch, bidx, v);
  return hipGetLastError();
}

// Alg. 6 / Alg. 8 last loop: N_out(p_i) <- empty; the slot becomes free.
__global__ void k_clear_rows(PoolView P, const uint32_t *ids, uint32_t n) {
  const uint32_t i = blockIdx.x;
  if (i >= n) return;
  const int ln = threadIdx.x;
  const uint32_t id = ids[i];
  if (ln < (int)P.R) P.adj[(size_t)id * P.R + ln] = kInvalid;
  if (ln == 0) {
    P.deg[id] = 0;
    P.active[id] = 0;
  }
}
hipError_t launch_clear_rows(PoolView p, const uint32_t *ids, uint32_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_clear_rows, dim3(n), dim3(64), 0, s, p, ids, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------- scan
// Exclusive prefix sum of n u32 values into out[0..n], out[n] = total, in
// three passes over tiles of 4096 (tile sums, scan of tile sums, apply).
constexpr int kScanThreads = 256;
constexpr int kScanPer = 16;
constexpr int kScanTile = kScanThreads * kScanPer;

// Scratch words of launch_scan (and of the grouping scan, which keeps two
// tile-sum arrays).
size_t scan_tmp_words(size_t n) { return 2 * ((n + kScanTile - 1) / kScanTile + 2); }

__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t *wsum, uint32_t &total) {
  const int ln = lane(), w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (ln >= o) x += y;
  }
  if (ln == 63) wsum[w] = x;
  __syncthreads();
  uint32_t off = 0, tot = 0;
  for (int k = 0; k < (int)(blockDim.x >> 6); k++) {
    if (k < w) off += wsum[k];
    tot += wsum[k];
  }
  __syncthreads();
  total = tot;
  return off + x - v;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_tiles(const uint32_t *in, size_t n, uint32_t *tsum) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPer;
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) s += base + k < n ? in[base + k] : 0u;
  uint32_t total;
  block_excl_scan(s, wsum, total);
  if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}

// In-place exclusive scan of the nt tile sums (tsum[nt] <- their total) by
// one wave: it fits beside a kernel that holds nearly every wave slot of
// every CU, where a workgroup of many waves waits for one to drain.  Lane l
// owns 16 consecutive sums of each block of 1024, all loaded before the
// wave scan of the lane totals.
constexpr int kTsumPer = 16;
__global__ __launch_bounds__(64) void k_scan_tsum(uint32_t *tsum, uint32_t nt) {
  const int ln = lane();
  uint32_t carry = 0;
  for (uint32_t b0 = 0; b0 < nt; b0 += 64 * kTsumPer) {
    const uint32_t base = b0 + (uint32_t)ln * kTsumPer;
    uint32_t v[kTsumPer], sum = 0;
#pragma unroll
    for (int k = 0; k < kTsumPer; k++) {
      v[k] = base + k < nt ? tsum[base + k] : 0u;
      sum += v[k];
    }
    uint32_t x = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(x, o, 64);
      if (ln >= o) x += y;
    }
    uint32_t run = carry + x - sum;
#pragma unroll
    for (int k = 0; k < kTsumPer; k++) {
      if (base + k < nt) tsum[base + k] = run;
      run += v[k];
    }
    carry += __shfl(x, 63, 64);
  }
  if (ln == 0) tsum[nt] = carry;
}

__global__ __launch_bounds__(kScanThreads) void k_scan_apply(const uint32_t *in, size_t n, const uint32_t *tsum,
                                                             uint32_t nt, uint32_t *out) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPer;
  uint32_t v[kScanPer];
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    v[k] = base + k < n ? in[base + k] : 0u;
    s += v[k];
  }
  uint32_t total;
  uint32_t run = tsum[blockIdx.x] + block_excl_scan(s, wsum, total);
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    if (base + k < n) out[base + k] = run;
    run += v[k];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) out[n] = tsum[nt];
}

// Inputs of at most kSmallScan values: one workgroup, one launch.
constexpr int kSmallScanThreads = 1024, kSmallScanPer = 16;
constexpr size_t kSmallScan = (size_t)kSmallScanThreads * kSmallScanPer;
// With VEC, in and out are 16-byte aligned and a thread moves its values as
// 16-byte groups (a quarter of the load and store instructions).
template <bool VEC>
__global__ __launch_bounds__(kSmallScanThreads) void k_scan_small(const uint32_t *in, size_t n, uint32_t *out) {
  __shared__ uint32_t wsum[kSmallScanThreads / 64];
  const size_t base = (size_t)threadIdx.x * kSmallScanPer;
  uint32_t v[kSmallScanPer];
  uint32_t sum = 0;
  if (VEC && base + kSmallScanPer <= n) {
#pragma unroll
    for (int k = 0; k < kSmallScanPer / 4; k++) {
      const uint4 w = reinterpret_cast<const uint4 *>(in + base)[k];
      v[4 * k] = w.x;
      v[4 * k + 1] = w.y;
      v[4 * k + 2] = w.z;
      v[4 * k + 3] = w.w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kSmallScanPer; k++) v[k] = base + k < n ? in[base + k] : 0u;
  }
#pragma unroll
  for (int k = 0; k < kSmallScanPer; k++) sum += v[k];
  uint32_t total;
  uint32_t run = block_excl_scan(sum, wsum, total);
  if (VEC && base + kSmallScanPer <= n) {
#pragma unroll
    for (int k = 0; k < kSmallScanPer / 4; k++) {
      uint4 w;
      w.x = run;
      w.y = w.x + v[4 * k];
      w.z = w.y + v[4 * k + 1];
      w.w = w.z + v[4 * k + 2];
      run = w.w + v[4 * k + 3];
      reinterpret_cast<uint4 *>(out + base)[k] = w;
    }
  } else {
#pragma unroll
    for (int k = 0; k < kSmallScanPer; k++) {
      if (base + k < n) out[base + k] = run;
      run += v[k];
    }
  }
  if (threadIdx.x == 0) out[n] = total;
}

hipError_t launch_scan(const uint32_t *in, uint32_t *out, size_t n, uint32_t *tmp, hipStream_t s) {
  const uint32_t nt = (uint32_t)((n + kScanTile - 1) / kScanTile);
  if (nt == 0) return launch_fill_u32(out, 0u, 1, s);
  if (n <= kSmallScan) {
    if (((uintptr_t)in | (uintptr_t)out) % 16 == 0)
      hipLaunchKernelGGL(k_scan_small<true>, dim3(1), dim3(kSmallScanThreads), 0, s, in, n, out);
    else
      hipLaunchKernelGGL(k_scan_small<false>, dim3(1), dim3(kSmallScanThreads), 0, s, in, n, out);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_scan_tiles, dim3(nt), dim3(kScanThreads), 0, s, in, n, tmp);
  hipLaunchKernelGGL(k_scan_tsum, dim3(1), dim3(64), 0, s, tmp, nt);
  hipLaunchKernelGGL(k_scan_apply, dim3(nt), dim3(kScanThreads), 0, s, in, n, tmp, nt, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- grouping
// Reverse-edge records (target, src, dist) grouped by target (counting sort):
// a histogram of targets (non-returning atomics), one scan that yields both
// the group offsets and the dirty list (the targets with a record, compacted
// in ascending id order), and the scatter.  The scatter counts back down,
// so `cnt` is all zero again afterwards.  Order inside a group is arbitrary;
// consumers order records by (dist, src).
__global__ void k_group_hist(const uint32_t *rec_t, size_t nrec, uint32_t *cnt) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < nrec; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t t = rec_t[i];
    if (t != kInvalid) atomicAdd(&cnt[t], 1u);
  }
}

// Pass 1: per tile of kScanTile targets, the number of records and the
// number of targets holding at least one.  Thread t reads elements
// t, t + 256, ... of the tile (coalesced).
__global__ __launch_bounds__(kScanThreads) void k_gscan_tiles(const uint32_t *cnt, size_t n, uint32_t *tsum,
                                                              uint32_t *fsum) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t base = (size_t)blockIdx.x * kScanTile + threadIdx.x;
  uint32_t s = 0, f = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    const size_t i = base + (size_t)k * kScanThreads;
    const uint32_t c = i < n ? cnt[i] : 0u;
    s += c;
    f += c != 0u;
  }
  uint32_t ts, tf;
  block_excl_scan(s, wsum, ts);
  block_excl_scan(f, wsum, tf);
  if (threadIdx.x == 0) {
    tsum[blockIdx.x] = ts;
    fsum[blockIdx.x] = tf;
  }
}

// Pass 2: exclusive scans of both tile-sum arrays (one workgroup).
__global__ __launch_bounds__(1024) void k_gscan_tsum(uint32_t *tsum, uint32_t *fsum, uint32_t nt) {
  __shared__ uint32_t wsum[16];
  uint32_t carry = 0, fcarry = 0;
  for (uint32_t b0 = 0; b0 < nt; b0 += 1024) {
    const uint32_t i = b0 + threadIdx.x;
    const uint32_t v = i < nt ? tsum[i] : 0u, w = i < nt ? fsum[i] : 0u;
    uint32_t total, ftotal;
    const uint32_t ex = block_excl_scan(v, wsum, total);
    const uint32_t fx = block_excl_scan(w, wsum, ftotal);
    if (i < nt) {
      tsum[i] = carry + ex;
      fsum[i] = fcarry + fx;
    }
    carry += total;
    fcarry += ftotal;
  }
  if (threadIdx.x == 0) {
    tsum[nt] = carry;
    fsum[nt] = fcarry;
  }
}

// Pass 3: offsets of every target and the dirty list.  Each thread owns
// kScanPer consecutive targets of the tile.
__global__ __launch_bounds__(kScanThreads) void k_gscan_apply(const uint32_t *cnt, size_t n, const uint32_t *tsum,
                                                              const uint32_t *fsum, uint32_t nt, uint32_t *off,
                                                              uint32_t *dirty, DevScalars *ds) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPer;
  uint32_t v[kScanPer];
  uint32_t s = 0, f = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    v[k] = base + k < n ? cnt[base + k] : 0u;
    s += v[k];
    f += v[k] != 0u;
  }
  uint32_t total;
  uint32_t run = tsum[blockIdx.x] + block_excl_scan(s, wsum, total);
  uint32_t frun = fsum[blockIdx.x] + block_excl_scan(f, wsum, total);
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    if (base + k < n) off[base + k] = run;
    if (v[k]) dirty[frun++] = (uint32_t)(base + k);
    run += v[k];
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    off[n] = tsum[nt];
    ds->n_dirty = fsum[nt];
  }
}

// Stream compaction by flags, for a length known only on the device: the
// same three passes as the scan, over tiles of kScanTile flags; tiles at or
// beyond *n contribute nothing.
__global__ __launch_bounds__(kScanThreads) void k_cf_tiles(const uint32_t *flags, const uint32_t *np, uint32_t *tsum) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t n = *np;
  const size_t base = (size_t)blockIdx.x * kScanTile + threadIdx.x;
  // loads issued together: indices past n read flag 0 and are dropped
  uint32_t fl[kScanPer];
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    const size_t i = base + (size_t)k * kScanThreads;
    fl[k] = flags[i < n ? i : 0];
  }
  uint32_t f = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) f += (base + (size_t)k * kScanThreads < n && fl[k] != 0u) ? 1u : 0u;
  uint32_t total;
  block_excl_scan(f, wsum, total);
  if (threadIdx.x == 0) tsum[blockIdx.x] = total;
}
__global__ __launch_bounds__(kScanThreads) void k_cf_apply(const uint32_t *flags, const uint32_t *items,
                                                           const uint32_t *np, const uint32_t *tsum, uint32_t nt,
                                                           uint32_t *out, uint32_t *out_n) {
  __shared__ uint32_t wsum[kScanThreads / 64];
  const size_t n = *np;
  const size_t base = (size_t)blockIdx.x * kScanTile + (size_t)threadIdx.x * kScanPer;
  // flags and items loaded together: indices past n read entry 0 and are
  // dropped
  uint32_t f[kScanPer], it[kScanPer];
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    const size_t i = base + k < n ? base + k : 0;
    f[k] = flags[i];
    it[k] = items[i];
  }
#pragma unroll
  for (int k = 0; k < kScanPer; k++) {
    f[k] = (base + k < n && f[k] != 0u) ? 1u : 0u;
    s += f[k];
  }
  uint32_t total;
  uint32_t run = tsum[blockIdx.x] + block_excl_scan(s, wsum, total);
#pragma unroll
  for (int k = 0; k < kScanPer; k++)
    if (f[k]) out[run++] = it[k];
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *out_n = tsum[nt];
}
hipError_t launch_compact_flags(const uint32_t *flags, const uint32_t *items, const uint32_t *n, uint32_t cap,
                                uint32_t *out, uint32_t *out_n, uint32_t *tmp, hipStream_t s) {
  const uint32_t nt = (uint32_t)((cap + kScanTile - 1) / kScanTile);
  if (nt == 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_cf_tiles, dim3(nt), dim3(kScanThreads), 0, s, flags, n, tmp);
  hipLaunchKernelGGL(k_scan_tsum, dim3(1), dim3(64), 0, s, tmp, nt);
  hipLaunchKernelGGL(k_cf_apply, dim3(nt), dim3(kScanThreads), 0, s, flags, items, n, tmp, nt, out, out_n);
  return hipGetLastError();
}

__global__ void k_group_scatter(const uint32_t *rec_t, const uint32_t *rec_s, const float *rec_d, size_t nrec,
                                uint32_t *cnt, const uint32_t *off, uint32_t *gsrc, float *gd) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < nrec; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t t = rec_t[i];
    if (t == kInvalid) continue;
    const uint32_t pos = off[t] + atomicSub(&cnt[t], 1u) - 1u;
    gsrc[pos] = rec_s[i];
    gd[pos] = rec_d[i];
  }
}

// Two-level form (capacities up to 2^24 ids), with no global atomics:
//  count  per tile of kGrpTile records, LDS counts of the coarse buckets
//         (target >> kGrpShift), stored at mat[bucket * ntiles + tile];
//  scan   of mat (bucket-major): mato[bucket * ntiles + tile] is where the
//         tile's records of that bucket start;
//  part   the same tiles move their records there (LDS cursors);
//  bucket one workgroup per coarse bucket counts its records per target in
//         LDS, writes the group offsets of its kGrpWidth targets and its
//         targets with a record (ascending) to its pad row, and moves the
//         records into their groups (LDS cursors);
//  dirty  each pad row is copied after those of the buckets before it, so
//         the dirty list is in ascending id order as in the one-level form.
constexpr int kGrpShift = 12;
constexpr uint32_t kGrpWidth = 1u << kGrpShift;
constexpr int kGrpThreads = 256;
constexpr int kGrpPer = 8;
constexpr uint32_t kGrpTile = kGrpThreads * kGrpPer;
constexpr uint32_t kGrpMaxBuckets = 4096;
constexpr int kGrpBucketThreads = 1024;

uint32_t group_buckets(uint32_t cap) { return (uint32_t)(((size_t)cap + kGrpWidth - 1) >> kGrpShift); }
bool group_two_level(uint32_t cap) { return group_buckets(cap) <= kGrpMaxBuckets; }
size_t group_mat_words(uint32_t cap, size_t rcap) {
  return (size_t)group_buckets(cap) * ((rcap + kGrpTile - 1) / kGrpTile) + 1;
}
size_t group_pad_words(uint32_t cap) { return (size_t)group_buckets(cap) * kGrpWidth; }

__global__ __launch_bounds__(kGrpThreads) void k_grp_count(const uint32_t *rec_t, size_t nrec, uint32_t cap,
                                                           uint32_t nb1, uint32_t ntiles, uint32_t *mat) {
  __shared__ uint32_t h[kGrpMaxBuckets];
  for (uint32_t b = threadIdx.x; b < nb1; b += kGrpThreads) h[b] = 0;
  __syncthreads();
  const size_t base = (size_t)blockIdx.x * kGrpTile + threadIdx.x;
  uint32_t t[kGrpPer];
#pragma unroll
  for (int k = 0; k < kGrpPer; k++) {
    const size_t i = base + (size_t)k * kGrpThreads;
    t[k] = i < nrec ? rec_t[i] : kInvalid;
  }
#pragma unroll
  for (int k = 0; k < kGrpPer; k++)
    if (t[k] < cap) atomicAdd(&h[t[k] >> kGrpShift], 1u);
  __syncthreads();
  for (uint32_t b = threadIdx.x; b < nb1; b += kGrpThreads) mat[(size_t)b * ntiles + blockIdx.x] = h[b];
}

__global__ __launch_bounds__(kGrpThreads) void k_grp_part(const uint32_t *rec_t, const uint32_t *rec_s,
                                                          const float *rec_d, size_t nrec, uint32_t cap, uint32_t nb1,
                                                          uint32_t ntiles, const uint32_t *mato, uint32_t *pt,
                                                          uint32_t *ps, float *pd) {
  __shared__ uint32_t cur[kGrpMaxBuckets];
  for (uint32_t b = threadIdx.x; b < nb1; b += kGrpThreads) cur[b] = mato[(size_t)b * ntiles + blockIdx.x];
  __syncthreads();
  const size_t base = (size_t)blockIdx.x * kGrpTile + threadIdx.x;
  // every record of the thread is loaded before the first is placed
  // (indices past the records read record 0 and are dropped)
  uint32_t t[kGrpPer], sv[kGrpPer];
  float dv[kGrpPer];
#pragma unroll
  for (int k = 0; k < kGrpPer; k++) {
    const size_t i = base + (size_t)k * kGrpThreads;
    const size_t ic = i < nrec ? i : 0;
    t[k] = rec_t[ic];
    sv[k] = rec_s[ic];
    dv[k] = rec_d[ic];
    if (i >= nrec) t[k] = kInvalid;
  }
#pragma unroll
  for (int k = 0; k < kGrpPer; k++) {
    if (t[k] >= cap) continue;
    const uint32_t pos = atomicAdd(&cur[t[k] >> kGrpShift], 1u);
    pt[pos] = t[k];
    ps[pos] = sv[k];
    pd[pos] = dv[k];
  }
}

__global__ __launch_bounds__(kGrpBucketThreads) void k_grp_bucket(const uint32_t *pt, const uint32_t *ps,
                                                                  const float *pd, uint32_t cap, uint32_t nb1,
                                                                  uint32_t ntiles, const uint32_t *mato, uint32_t *off,
                                                                  uint32_t *gsrc, float *gd, uint32_t *dpad,
                                                                  uint32_t *dcnt) {
  constexpr int kq = kGrpWidth / kGrpBucketThreads;  // targets per thread in the scan
  __shared__ uint32_t h[kGrpWidth];
  __shared__ uint32_t wsum[kGrpBucketThreads / 64];
  const uint32_t b = blockIdx.x;
  const uint32_t lo = mato[(size_t)b * ntiles], hi = mato[(size_t)(b + 1) * ntiles];
  for (uint32_t k = threadIdx.x; k < kGrpWidth; k += kGrpBucketThreads) h[k] = 0;
  __syncthreads();
  for (uint32_t i = lo + threadIdx.x; i < hi; i += kGrpBucketThreads) atomicAdd(&h[pt[i] & (kGrpWidth - 1)], 1u);
  __syncthreads();
  uint32_t c[kq], sum = 0, nz = 0;
#pragma unroll
  for (int k = 0; k < kq; k++) {
    c[k] = h[kq * threadIdx.x + k];
    sum += c[k];
    nz += c[k] != 0u;
  }
  uint32_t total, ndirty;
  uint32_t run = lo + block_excl_scan(sum, wsum, total);
  uint32_t frun = block_excl_scan(nz, wsum, ndirty);
  const uint32_t t0 = (b << kGrpShift) + kq * threadIdx.x;
#pragma unroll
  for (int k = 0; k < kq; k++) {
    const uint32_t t = t0 + k;
    if (t < cap) off[t] = run;
    if (c[k]) dpad[(size_t)b * kGrpWidth + frun++] = t;
    h[kq * threadIdx.x + k] = run;  // this thread's own entries become cursors
    run += c[k];
  }
  if (threadIdx.x == 0) {
    dcnt[b] = ndirty;
    if (b == nb1 - 1) off[cap] = hi;
  }
  __syncthreads();
  for (uint32_t i = lo + threadIdx.x; i < hi; i += kGrpBucketThreads) {
    const uint32_t pos = atomicAdd(&h[pt[i] & (kGrpWidth - 1)], 1u);
    gsrc[pos] = ps[i];
    gd[pos] = pd[i];
  }
}

__global__ __launch_bounds__(kGrpThreads) void k_grp_dirty(const uint32_t *dpad, const uint32_t *dcnt, uint32_t nb1,
                                                           uint32_t *dirty, DevScalars *ds) {
  __shared__ uint32_t wsum[kGrpThreads / 64];
  const uint32_t b = blockIdx.x;
  uint32_t s = 0;
  for (uint32_t k = threadIdx.x; k < b; k += kGrpThreads) s += dcnt[k];
  uint32_t before;
  block_excl_scan(s, wsum, before);
  const uint32_t n = dcnt[b];
  for (uint32_t k = threadIdx.x; k < n; k += kGrpThreads) dirty[before + k] = dpad[(size_t)b * kGrpWidth + k];
  if (b == nb1 - 1 && threadIdx.x == 0) ds->n_dirty = before + n;
}

hipError_t launch_group(const uint32_t *rec_t, const uint32_t *rec_s, const float *rec_d, size_t nrec, uint32_t cap,
                        uint32_t *cnt, uint32_t *off, uint32_t *scan_tmp, uint32_t *gsrc, float *gd,
                        uint32_t *dirty, DevScalars *ds, const GroupBufs *gb, hipStream_t s) {
  if (gb && group_two_level(cap) && cap > 0) {
    if (nrec > gb->rcap) return hipErrorInvalidValue;
    const uint32_t nb1 = group_buckets(cap);
    const uint32_t ntiles = (uint32_t)((nrec + kGrpTile - 1) / kGrpTile);
    if (ntiles)
      hipLaunchKernelGGL(k_grp_count, dim3(ntiles), dim3(kGrpThreads), 0, s, rec_t, nrec, cap, nb1, ntiles, gb->mat);
    hipError_t e = launch_scan(gb->mat, gb->mato, (size_t)nb1 * ntiles, gb->tmp, s);
    if (e != hipSuccess) return e;
    if (ntiles)
      hipLaunchKernelGGL(k_grp_part, dim3(ntiles), dim3(kGrpThreads), 0, s, rec_t, rec_s, rec_d, nrec, cap, nb1,
                         ntiles, gb->mato, gb->pt, gb->ps, gb->pd);
    hipLaunchKernelGGL(k_grp_bucket, dim3(nb1), dim3(kGrpBucketThreads), 0, s, gb->pt, gb->ps, gb->pd, cap, nb1,
                       ntiles, gb->mato, off, gsrc, gd, gb->dpad, gb->dcnt);
    hipLaunchKernelGGL(k_grp_dirty, dim3(nb1), dim3(kGrpThreads), 0, s, gb->dpad, gb->dcnt, nb1, dirty, ds);
    return hipGetLastError();
  }
  uint32_t g = blocks_for(nrec, 256);
  if (g > 8192) g = 8192;
  if (nrec) hipLaunchKernelGGL(k_group_hist, dim3(g), dim3(256), 0, s, rec_t, nrec, cnt);
  const uint32_t nt = (uint32_t)((cap + kScanTile - 1) / kScanTile);
  uint32_t *tsum = scan_tmp, *fsum = scan_tmp + nt + 1;
  hipLaunchKernelGGL(k_gscan_tiles, dim3(nt), dim3(kScanThreads), 0, s, cnt, (size_t)cap, tsum, fsum);
  hipLaunchKernelGGL(k_gscan_tsum, dim3(1), dim3(1024), 0, s, tsum, fsum, nt);
  hipLaunchKernelGGL(k_gscan_apply, dim3(nt), dim3(kScanThreads), 0, s, cnt, (size_t)cap, tsum, fsum, nt, off, dirty,
                     ds);
  if (nrec) hipLaunchKernelGGL(k_group_scatter, dim3(g), dim3(256), 0, s, rec_t, rec_s, rec_d, nrec, cnt, off, gsrc, gd);
  return hipGetLastError();
}

// ---------------------------------------------------------------- reverse graph
// N_in as CSR (Alg. 8): every edge u -> v of an active row u is counted
// into v's row (by_batch: only edges into the delete batch, counted into
// the batch position of v), the counts are scanned, and sources are
// scattered.  Rows are in arbitrary order here; consumers that need an
// order derive it from the ids (rank of u = number of sources below u).
__global__ void k_rev_hist(PoolView P, int by_batch, const uint8_t *in_batch, const uint32_t *bidx, uint32_t *cnt) {
  const size_t total = (size_t)P.cap * P.R;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t v = P.adj[i];
    if (v == kInvalid) continue;
    const uint32_t u = (P.R & (P.R - 1)) == 0 ? (uint32_t)(i >> (__ffs(P.R) - 1)) : (uint32_t)(i / P.R);
    if (!P.active[u]) continue;
    if (by_batch) {
      if (in_batch[v]) atomicAdd(&cnt[bidx[v]], 1u);
    } else {
      atomicAdd(&cnt[v], 1u);
    }
  }
}
__global__ void k_rev_scatter(PoolView P, int by_batch, const uint8_t *in_batch, const uint32_t *bidx, uint32_t *cnt,
                              const uint32_t *off, uint32_t *src) {
  const size_t total = (size_t)P.cap * P.R;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t v = P.adj[i];
    if (v == kInvalid) continue;
    const uint32_t u = (P.R & (P.R - 1)) == 0 ? (uint32_t)(i >> (__ffs(P.R) - 1)) : (uint32_t)(i / P.R);
    if (!P.active[u]) continue;
    uint32_t row;
    if (by_batch) {
      if (!in_batch[v]) continue;
      row = bidx[v];
    } else {
      row = v;
    }
    const uint32_t pos = off[row] + atomicSub(&cnt[row], 1u) - 1u;
    src[pos] = u;
  }
}
// The naive in-neighbour detection a reverse graph replaces: for each id,
// a scan of every list for it.  Workgroup (x, i) scans the x-th of
// gridDim.x slices of the adjacency for ids[i] and adds the occurrences in
// active rows to counts[i] (counts zeroed by the caller).
__global__ __launch_bounds__(256) void k_scan_in_edges(PoolView P, const uint32_t *ids, uint32_t *counts) {
  const uint32_t p = ids[blockIdx.y];
  const size_t total = (size_t)P.cap * P.R;
  const size_t per = (total + gridDim.x - 1) / gridDim.x;
  const size_t e0 = (size_t)blockIdx.x * per, e1 = e0 + per < total ? e0 + per : total;
  uint32_t c = 0;
  for (size_t e = e0 + threadIdx.x; e < e1; e += blockDim.x)
    if (P.adj[e] == p && P.active[e / P.R]) c++;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0 && c) atomicAdd(&counts[blockIdx.y], c);
}
hipError_t launch_scan_in_edges(PoolView p, const uint32_t *ids, uint32_t n, uint32_t *counts, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipError_t e = launch_fill_u32(counts, 0u, n, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_scan_in_edges, dim3(256, n), dim3(256), 0, s, p, ids, counts);
  return hipGetLastError();
}
// counts[i] = off[row(i) + 1] - off[row(i)], row(i) = i (batch rows) or ids[i]
__global__ void k_row_lengths(const uint32_t *off, const uint32_t *ids, uint32_t n, uint32_t *counts) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t r = ids ? ids[i] : i;
  counts[i] = off[r + 1] - off[r];
}
hipError_t launch_row_lengths(const uint32_t *off, const uint32_t *ids, uint32_t n, uint32_t *counts, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(k_row_lengths, dim3(blocks_for(n, 256)), dim3(256), 0, s, off, ids, n, counts);
  return hipGetLastError();
}

__global__ void k_count_edges(const uint32_t *off, uint32_t nrows, DevScalars *ds) {
  if (threadIdx.x == 0) stat_add(ds, kStRevEdges, (unsigned long long)off[nrows]);
}

// Full reverse graph without global atomics, as a two-level counting sort:
//  1. every source chunk counts its edges per target bucket (LDS atomics);
//  2. the (bucket, chunk) counts are scanned bucket-major;
//  3. every chunk writes its edges as (src, target) pairs into its slice of
//     each bucket's segment (LDS atomics hand out the positions);
//  4. one workgroup per bucket counts its targets' in-degrees in LDS, scans
//     them into the CSR offsets and scatters the sources into the rows.
// HBM traffic: adj read twice, pairs written and read twice, sources
// written once; no global atomic operations.
constexpr int kRevThreads = 256;
constexpr uint32_t kRevMaxBuckets = 16384;  // LDS counters of steps 1 and 3 (64 KB)
constexpr int kRevMinShift = 8, kRevMaxShift = 13;  // bucket width 256 .. 8192 targets
constexpr uint32_t kRev2Coarse = 256;      // coarse buckets (two-level form)
constexpr int kRev2FineShift = 6;          // fine buckets of 64 targets
constexpr uint32_t kRev2FineChunks = 16;   // chunks per coarse bucket
constexpr uint32_t kRev2MaxSub = 256;      // fine buckets per coarse bucket
constexpr int kRev2Per = 16;               // edges per thread per local-sort step
constexpr int kRev2Step = kRevThreads * kRev2Per;  // edges per local-sort step
constexpr uint32_t kRev2Stage = 6144;      // sources a fine bucket stages in LDS (24 KB)

RevPlan rev_plan(uint32_t cap, uint32_t R) {
  RevPlan p{};
  int s = kRevMinShift;
  while (s < kRevMaxShift && (((size_t)cap + (1u << s) - 1) >> s) > 1024) s++;
  p.shift = s;
  p.nb = (uint32_t)(((size_t)cap + (1u << s) - 1) >> s);
  p.ng = std::max<uint32_t>(1, std::min<uint32_t>(1024, cap / 64));
  p.ch = (cap + p.ng - 1) / p.ng;
  const int idbits = cap > 1 ? 32 - __builtin_clz(cap - 1) : 1;
  p.packed = idbits + s <= 32;
  // 32-bit edge indices, with headroom for the loop strides
  p.ok = cap > 0 && p.nb <= kRevMaxBuckets && (uint64_t)cap * R + (1u << 20) < (1ull << 32);
  // two-level form: at most kRev2Coarse coarse buckets, fine buckets of
  // 2^kRev2FineShift targets, both partitions packed into 32 bits
  int s1 = kRev2FineShift + 1;
  while ((((size_t)cap + (1u << s1) - 1) >> s1) > kRev2Coarse) s1++;
  p.s1 = s1;
  p.s2 = kRev2FineShift;
  p.nb1 = (uint32_t)(((size_t)cap + (1u << s1) - 1) >> s1);
  p.nsub = 1u << (s1 - p.s2);
  p.nc2 = kRev2FineChunks;
  p.two = p.ok && idbits + s1 <= 32 && p.nsub <= kRev2MaxSub;
  p.rshift = (R & (R - 1)) == 0 ? __builtin_ctz(R) : -1;
  if (p.two) {  // more, smaller source chunks: more workgroups in flight
    p.ng = std::max<uint32_t>(1, std::min<uint32_t>(4096, cap / 64));
    p.ch = (cap + p.ng - 1) / p.ng;
  }
  return p;
}
size_t rev_pair_words(const RevPlan &rp, uint32_t cap, uint32_t R) {
  return rp.ok ? (size_t)cap * R * (rp.packed || rp.two ? 1 : 2) : 0;
}
size_t rev_bucket_words(const RevPlan &rp) {
  if (!rp.ok) return 0;
  return (rp.two ? (size_t)rp.nb1 * rp.ng : (size_t)rp.nb * rp.ng) + 1;
}
size_t rev_fine_words(const RevPlan &rp) { return rp.two ? (size_t)rp.nb1 * rp.nsub * rp.nc2 + 1 : 0; }

// Row of edge index i (the bucketed build requires cap * R < 2^32).
__device__ __forceinline__ uint32_t edge_row(const RevPlan &rp, uint32_t i, uint32_t R) {
  return rp.rshift >= 0 ? i >> rp.rshift : i / R;
}

// Reverse lists of the delete batch only (rows indexed by batch position).
// One pass over the adjacency: every workgroup (1024 threads, one per CU)
// first builds in LDS a bitmap of the batch ids (exact when the pool has at
// most 2^lbits ids; otherwise ids are folded onto the bits and a set bit is
// confirmed with the in_batch flag), then streams its rows with 16-byte
// loads and appends the edge index of each edge into the batch (from an
// active row) to its own region of `pairs` (the edge indices of its rows,
// so regions never overlap), positions from an LDS counter.  Then a
// histogram of the found edges per batch row, a scan, and a scatter of their
// sources.  Only the edges into the batch (about one in a hundred at 10K of
// 1M) reach global memory again.  Row order within a list is not fixed;
// consumers do not depend on it.
constexpr int kRevrThreads = 1024;
__global__ __launch_bounds__(kRevrThreads) void k_revr_find(PoolView P, const uint32_t *ids, uint32_t n,
                                                            const uint8_t *in_batch, uint32_t ch, uint32_t lbits,
                                                            uint32_t *pairs, uint32_t *wgcnt) {
  extern __shared__ uint32_t bm[];
  __shared__ uint32_t lcnt;
  const uint32_t nw = (1u << lbits) >> 5, mask = (1u << lbits) - 1u;
  for (uint32_t i = threadIdx.x; i < nw; i += blockDim.x) bm[i] = 0u;
  if (threadIdx.x == 0) lcnt = 0u;
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < n; i += blockDim.x) {
    const uint32_t v = ids[i] & mask;
    atomicOr(&bm[v >> 5], 1u << (v & 31u));
  }
  __syncthreads();
  const bool exact = P.cap <= (1u << lbits);
  const uint32_t r0 = blockIdx.x * ch;
  const uint32_t r1 = std::min<uint32_t>(P.cap, r0 + ch);
  auto test = [&](uint32_t e, uint32_t v) {
    if (v == kInvalid) return;
    const uint32_t f = v & mask;
    if (!((bm[f >> 5] >> (f & 31u)) & 1u)) return;
    if (!exact && !in_batch[v]) return;
    const uint32_t u = e / P.R;
    if (P.active[u]) pairs[r0 * P.R + atomicAdd(&lcnt, 1u)] = e;
  };
  if (r0 < r1) {
    const uint32_t e0 = r0 * P.R, e1 = r1 * P.R;
    if ((P.R & 3u) == 0) {
      // rows are whole 16-byte groups: four groups in flight per thread
      const uint4 *adj4 = reinterpret_cast<const uint4 *>(P.adj);
      const uint32_t q0 = e0 / 4, q1 = e1 / 4, step = blockDim.x;
      for (uint32_t q = q0 + threadIdx.x; q < q1; q += 4 * step) {
        // the four loads issued together (indices past the range read group
        // q0 and are dropped)
        uint4 w[4];
#pragma unroll
        for (int k = 0; k < 4; k++) {
          const uint32_t qk = q + k * step;
          w[k] = adj4[qk < q1 ? qk : q0];
          if (qk >= q1) w[k] = make_uint4(kInvalid, kInvalid, kInvalid, kInvalid);
        }
#pragma unroll
        for (int k = 0; k < 4; k++) {
          const uint32_t e = 4 * (q + k * step);
          test(e, w[k].x);
          test(e + 1, w[k].y);
          test(e + 2, w[k].z);
          test(e + 3, w[k].w);
        }
      }
    } else {
      const uint32_t step = blockDim.x;
      for (uint32_t i = e0 + threadIdx.x; i < e1; i += 4 * step) {
        uint32_t v[4];
#pragma unroll
        for (int k = 0; k < 4; k++) {
          const uint32_t ik = i + k * step;
          v[k] = P.adj[ik < e1 ? ik : e0];
          if (ik >= e1) v[k] = kInvalid;
        }
#pragma unroll
        for (int k = 0; k < 4; k++) test(i + k * step, v[k]);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) wgcnt[blockIdx.x] = lcnt;
}
__global__ __launch_bounds__(kRevThreads) void k_revr_hist(PoolView P, uint32_t ch, const uint32_t *bidx,
                                                           const uint32_t *pairs, const uint32_t *wgcnt,
                                                           uint32_t *cnt) {
  const uint32_t base = blockIdx.x * ch * P.R, m = wgcnt[blockIdx.x];
  for (uint32_t j = threadIdx.x; j < m; j += blockDim.x) atomicAdd(&cnt[bidx[P.adj[pairs[base + j]]]], 1u);
}
// cnt counts down to zero again, ready for the next use
__global__ __launch_bounds__(kRevThreads) void k_revr_scatter(PoolView P, uint32_t ch, const uint32_t *bidx,
                                                              const uint32_t *pairs, const uint32_t *wgcnt,
                                                              uint32_t *cnt, const uint32_t *off, uint32_t *src) {
  const uint32_t base = blockIdx.x * ch * P.R, m = wgcnt[blockIdx.x];
  for (uint32_t j = threadIdx.x; j < m; j += blockDim.x) {
    const uint32_t e = pairs[base + j];
    const uint32_t b = bidx[P.adj[e]];
    src[off[b] + atomicSub(&cnt[b], 1u) - 1u] = e / P.R;
  }
}

// Bits of the LDS batch bitmap (a power of two; the whole pool when it fits
// the workgroup's LDS) and the workgroups of the batch-rows build.
static uint32_t revr_lbits(uint32_t cap, int lds) {
  if (lds < 8192) lds = 65536;
  const uint64_t bits = (uint64_t)(lds - 1024) * 8;
  uint32_t lb = 5;
  while (lb < 31 && (2ull << lb) <= bits && (1u << lb) < cap) lb++;
  return lb;
}


// Edges of chunk blockIdx.x, four loads in flight per thread; f(u, v) for
// every edge u -> v of an active row.
template <class F>
__device__ __forceinline__ void for_chunk_edges(const PoolView &P, const RevPlan &rp, F f) {
  const uint32_t r0 = blockIdx.x * rp.ch;
  const uint32_t r1 = std::min<uint32_t>(P.cap, r0 + rp.ch);
  if (r0 >= r1) return;
  const uint32_t e0 = r0 * P.R, e1 = r1 * P.R;
  const uint32_t step = blockDim.x;
  for (uint32_t i = e0 + threadIdx.x; i < e1; i += 4 * step) {
    uint32_t v[4];
#pragma unroll
    for (int k = 0; k < 4; k++) v[k] = i + k * step < e1 ? P.adj[i + k * step] : kInvalid;
#pragma unroll
    for (int k = 0; k < 4; k++) {
      if (v[k] == kInvalid) continue;
      const uint32_t u = edge_row(rp, i + k * step, P.R);
      if (P.active[u]) f(u, v[k]);
    }
  }
}

__global__ __launch_bounds__(kRevThreads) void k_revb_count(PoolView P, RevPlan rp, uint32_t *bh) {
  extern __shared__ uint32_t lh[];
  for (uint32_t b = threadIdx.x; b < rp.nb; b += blockDim.x) lh[b] = 0;
  __syncthreads();
  for_chunk_edges(P, rp, [&](uint32_t, uint32_t v) { atomicAdd(&lh[v >> rp.shift], 1u); });
  __syncthreads();
  for (uint32_t b = threadIdx.x; b < rp.nb; b += blockDim.x) bh[(size_t)b * rp.ng + blockIdx.x] = lh[b];
}

template <bool PACKED>
__global__ __launch_bounds__(kRevThreads) void k_revb_part(PoolView P, RevPlan rp, const uint32_t *bo,
                                                           uint32_t *pairs) {
  extern __shared__ uint32_t lo[];
  for (uint32_t b = threadIdx.x; b < rp.nb; b += blockDim.x) lo[b] = bo[(size_t)b * rp.ng + blockIdx.x];
  __syncthreads();
  const uint32_t mask = (1u << rp.shift) - 1u;
  for_chunk_edges(P, rp, [&](uint32_t u, uint32_t v) {
    const uint32_t pos = atomicAdd(&lo[v >> rp.shift], 1u);
    if (PACKED) pairs[pos] = (u << rp.shift) | (v & mask);
    else reinterpret_cast<uint2 *>(pairs)[pos] = make_uint2(u, v);
  });
}

template <bool PACKED>
__global__ __launch_bounds__(kRevThreads) void k_revb_fill(RevPlan rp, uint32_t cap, const uint32_t *bo,
                                                           const uint32_t *pairs, uint32_t *off, uint32_t *src) {
  extern __shared__ uint32_t cnt[];
  __shared__ uint32_t wsum[kRevThreads / 64];
  const uint32_t b = blockIdx.x, W = 1u << rp.shift, mask = W - 1u;
  const uint32_t s0 = bo[(size_t)b * rp.ng], s1 = bo[(size_t)(b + 1) * rp.ng];
  for (uint32_t i = threadIdx.x; i < W; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
  auto target = [&](uint32_t j) -> uint32_t {
    return PACKED ? (pairs[j] & mask) : (reinterpret_cast<const uint2 *>(pairs)[j].y & mask);
  };
  auto source = [&](uint32_t j) -> uint32_t {
    return PACKED ? (pairs[j] >> rp.shift) : reinterpret_cast<const uint2 *>(pairs)[j].x;
  };
  for (uint32_t j = s0 + threadIdx.x; j < s1; j += blockDim.x) atomicAdd(&cnt[target(j)], 1u);
  __syncthreads();
  // exclusive scan of the W counts: thread t owns W / blockDim consecutive ones
  const uint32_t per = W / blockDim.x, base = threadIdx.x * per;
  uint32_t sum = 0;
  for (uint32_t k = 0; k < per; k++) sum += cnt[base + k];
  uint32_t total;
  uint32_t run = s0 + block_excl_scan(sum, wsum, total);
  for (uint32_t k = 0; k < per; k++) {
    const uint32_t c = cnt[base + k];
    const size_t v = (size_t)b * W + base + k;
    if (v < cap) off[v] = run;
    cnt[base + k] = run;
    run += c;
  }
  __syncthreads();
  for (uint32_t j = s0 + threadIdx.x; j < s1; j += blockDim.x) {
    const uint32_t pos = atomicAdd(&cnt[target(j)], 1u);
    src[pos] = source(j);
  }
  if (b == rp.nb - 1 && threadIdx.x == 0) off[cap] = s1;
}

// ---- two-level form.  Every write is a run of consecutive addresses:
// each partition step sorts a block of kRev2Step items by bucket in LDS
// (counting sort) and then writes the block bucket by bucket, so a bucket's
// items leave as one contiguous run instead of scattered words.
//  A  coarse counts per (coarse bucket, source chunk)       k_rev2_count
//  B  coarse partition: pairs (src << s1) | (target & m1)   k_rev2_part1
//  C  fine counts per (coarse, fine bucket, chunk)          k_rev2_count2
//  D  fine partition: pairs (src << s2) | (target & m2)     k_rev2_part2
//  E  one workgroup per fine bucket: in-degrees, offsets, sources staged
//     in LDS and written contiguously                      k_rev2_fill

// Local counting sort of up to kRev2Step items (key < nkey) of one block:
// returns, for this thread's items, their position in key order; fills
// lcnt (counts) and lstart (exclusive starts).  lcnt/lstart hold nkey
// entries (nkey <= blockDim.x * 4).
__device__ __forceinline__ void rev2_local_sort(const uint32_t (&key)[kRev2Per], const bool (&ok)[kRev2Per],
                                                uint32_t nkey, uint32_t *lcnt, uint32_t *lstart, uint32_t *wsum,
                                                uint32_t (&pos)[kRev2Per]) {
  for (uint32_t b = threadIdx.x; b < nkey; b += blockDim.x) lcnt[b] = 0;
  __syncthreads();
  uint32_t rk[kRev2Per];
#pragma unroll
  for (int k = 0; k < kRev2Per; k++) rk[k] = ok[k] ? atomicAdd(&lcnt[key[k]], 1u) : 0u;
  __syncthreads();
  // exclusive scan of lcnt: thread t owns keys 4t .. 4t+3
  uint32_t c[4], sum = 0;
#pragma unroll
  for (int q = 0; q < 4; q++) {
    const uint32_t b = threadIdx.x * 4 + q;
    c[q] = b < nkey ? lcnt[b] : 0u;
    sum += c[q];
  }
  uint32_t total;
  uint32_t run = block_excl_scan(sum, wsum, total);
#pragma unroll
  for (int q = 0; q < 4; q++) {
    const uint32_t b = threadIdx.x * 4 + q;
    if (b < nkey) lstart[b] = run;
    run += c[q];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kRev2Per; k++) pos[k] = ok[k] ? lstart[key[k]] + rk[k] : 0u;
}

// Edges of chunk blockIdx.x read as 16-byte groups of one row (R a power
// of two and a multiple of 4), four groups in flight per thread.
template <class F>
__device__ __forceinline__ void for_chunk_edges4(const PoolView &P, const RevPlan &rp, F f) {
  const uint32_t r0 = blockIdx.x * rp.ch;
  const uint32_t r1 = std::min<uint32_t>(P.cap, r0 + rp.ch);
  if (r0 >= r1) return;
  const uint32_t q0 = r0 * P.R / 4, q1 = r1 * P.R / 4;
  const uint32_t step = blockDim.x;
  const uint4 *adj4 = reinterpret_cast<const uint4 *>(P.adj);
  for (uint32_t q = q0 + threadIdx.x; q < q1; q += 4 * step) {
    uint4 v[4];
#pragma unroll
    for (int k = 0; k < 4; k++)
      v[k] = q + k * step < q1 ? adj4[q + k * step] : make_uint4(kInvalid, kInvalid, kInvalid, kInvalid);
#pragma unroll
    for (int k = 0; k < 4; k++) {
      if (q + k * step >= q1) continue;
      const uint32_t u = (4 * (q + k * step)) >> rp.rshift;
      if (!P.active[u]) continue;
      if (v[k].x != kInvalid) f(u, v[k].x);
      if (v[k].y != kInvalid) f(u, v[k].y);
      if (v[k].z != kInvalid) f(u, v[k].z);
      if (v[k].w != kInvalid) f(u, v[k].w);
    }
  }
}

__global__ __launch_bounds__(kRevThreads) void k_rev2_count(PoolView P, RevPlan rp, uint32_t *bh) {
  __shared__ uint32_t lh[kRev2Coarse];
  for (uint32_t b = threadIdx.x; b < rp.nb1; b += blockDim.x) lh[b] = 0;
  __syncthreads();
  auto add = [&](uint32_t, uint32_t v) { atomicAdd(&lh[v >> rp.s1], 1u); };
  if (rp.rshift >= 2) for_chunk_edges4(P, rp, add);
  else for_chunk_edges(P, rp, add);
  __syncthreads();
  for (uint32_t b = threadIdx.x; b < rp.nb1; b += blockDim.x) bh[(size_t)b * rp.ng + blockIdx.x] = lh[b];
}

__global__ __launch_bounds__(kRevThreads) void k_rev2_part1(PoolView P, RevPlan rp, const uint32_t *bo,
                                                            uint32_t *pairs) {
  __shared__ uint32_t gpos[kRev2Coarse], lcnt[kRev2Coarse], lstart[kRev2Coarse];
  __shared__ uint32_t wsum[kRevThreads / 64];
  __shared__ uint32_t sval[kRev2Step];
  __shared__ uint8_t skey[kRev2Step];
  for (uint32_t b = threadIdx.x; b < rp.nb1; b += blockDim.x) gpos[b] = bo[(size_t)b * rp.ng + blockIdx.x];
  const uint32_t r0 = blockIdx.x * rp.ch;
  const uint32_t r1 = std::min<uint32_t>(P.cap, r0 + rp.ch);
  const uint32_t e0 = r0 * P.R, e1 = r1 < r0 ? e0 : r1 * P.R;
  const uint32_t m1 = (1u << rp.s1) - 1u;
  for (uint32_t base = e0; base < e1; base += kRev2Step) {
    uint32_t key[kRev2Per], val[kRev2Per], pos[kRev2Per];
    bool ok[kRev2Per];
    if (rp.rshift >= 2) {
      // 16-byte groups of one row, all four loads in flight
      const uint4 *adj4 = reinterpret_cast<const uint4 *>(P.adj);
      uint4 w[kRev2Per / 4];
#pragma unroll
      for (int k4 = 0; k4 < kRev2Per / 4; k4++) {
        const uint32_t q = base / 4 + (uint32_t)k4 * blockDim.x + threadIdx.x;
        w[k4] = 4 * q < e1 ? adj4[q] : make_uint4(kInvalid, kInvalid, kInvalid, kInvalid);
      }
#pragma unroll
      for (int k4 = 0; k4 < kRev2Per / 4; k4++) {
        const uint32_t q = base / 4 + (uint32_t)k4 * blockDim.x + threadIdx.x;
        const uint32_t u = (4 * q) >> rp.rshift;
        const bool act = 4 * q < e1 && P.active[u] != 0;
        const uint32_t vv[4] = {w[k4].x, w[k4].y, w[k4].z, w[k4].w};
#pragma unroll
        for (int t = 0; t < 4; t++) {
          const int k = 4 * k4 + t;
          ok[k] = act && vv[t] != kInvalid;
          key[k] = ok[k] ? vv[t] >> rp.s1 : 0u;
          val[k] = (u << rp.s1) | (vv[t] & m1);
        }
      }
    } else {
#pragma unroll
      for (int k = 0; k < kRev2Per; k++) {
        const uint32_t i = base + (uint32_t)k * blockDim.x + threadIdx.x;
        const bool in = i < e1;
        const uint32_t v = in ? P.adj[i] : kInvalid;
        const uint32_t u = edge_row(rp, in ? i : e1 - 1, P.R);
        ok[k] = v != kInvalid && P.active[u] != 0;
        key[k] = ok[k] ? v >> rp.s1 : 0u;
        val[k] = (u << rp.s1) | (v & m1);
      }
    }
    rev2_local_sort(key, ok, rp.nb1, lcnt, lstart, wsum, pos);
#pragma unroll
    for (int k = 0; k < kRev2Per; k++)
      if (ok[k]) {
        sval[pos[k]] = val[k];
        skey[pos[k]] = (uint8_t)key[k];
      }
    __syncthreads();
    const uint32_t n = lstart[rp.nb1 - 1] + lcnt[rp.nb1 - 1];
    for (uint32_t j = threadIdx.x; j < n; j += blockDim.x) {
      const uint32_t b = skey[j];
      pairs[gpos[b] + (j - lstart[b])] = sval[j];
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < rp.nb1; b += blockDim.x) gpos[b] += lcnt[b];
    __syncthreads();
  }
}

// Range of chunk c (of nc2) of coarse bucket b1 in the coarse partition.
__device__ __forceinline__ void rev2_chunk(const RevPlan &rp, const uint32_t *bo, uint32_t b1, uint32_t c,
                                           uint32_t &x0, uint32_t &x1) {
  const uint32_t s0 = bo[(size_t)b1 * rp.ng], s1 = bo[(size_t)(b1 + 1) * rp.ng];
  const uint32_t n = s1 - s0;
  x0 = s0 + (uint32_t)((uint64_t)n * c / rp.nc2);
  x1 = s0 + (uint32_t)((uint64_t)n * (c + 1) / rp.nc2);
}

__global__ __launch_bounds__(kRevThreads) void k_rev2_count2(RevPlan rp, const uint32_t *bo, const uint32_t *pairs,
                                                             uint32_t *bh2) {
  __shared__ uint32_t lh[kRev2MaxSub];
  const uint32_t b1 = blockIdx.x / rp.nc2, c = blockIdx.x % rp.nc2;
  for (uint32_t b = threadIdx.x; b < rp.nsub; b += blockDim.x) lh[b] = 0;
  __syncthreads();
  uint32_t x0, x1;
  rev2_chunk(rp, bo, b1, c, x0, x1);
  const uint32_t m1 = (1u << rp.s1) - 1u;
  // unaligned head and tail word by word, the middle as 16-byte groups
  const uint32_t a0 = std::min(x1, (x0 + 3u) & ~3u), a1 = std::max(a0, x1 & ~3u);
  for (uint32_t j = x0 + threadIdx.x; j < a0; j += blockDim.x) atomicAdd(&lh[(pairs[j] & m1) >> rp.s2], 1u);
  for (uint32_t j = a1 + threadIdx.x; j < x1; j += blockDim.x) atomicAdd(&lh[(pairs[j] & m1) >> rp.s2], 1u);
  const uint4 *p4 = reinterpret_cast<const uint4 *>(pairs);
  const uint32_t qe = a1 / 4;
  for (uint32_t q = a0 / 4 + threadIdx.x; q < qe; q += 4 * blockDim.x) {
    uint4 v[4];  // four groups in flight per thread
#pragma unroll
    for (int k = 0; k < 4; k++) {
      const uint32_t qq = q + (uint32_t)k * blockDim.x;
      v[k] = qq < qe ? p4[qq] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < 4; k++) {
      if (q + (uint32_t)k * blockDim.x >= qe) break;
      atomicAdd(&lh[(v[k].x & m1) >> rp.s2], 1u);
      atomicAdd(&lh[(v[k].y & m1) >> rp.s2], 1u);
      atomicAdd(&lh[(v[k].z & m1) >> rp.s2], 1u);
      atomicAdd(&lh[(v[k].w & m1) >> rp.s2], 1u);
    }
  }
  __syncthreads();
  for (uint32_t b = threadIdx.x; b < rp.nsub; b += blockDim.x) bh2[((size_t)b1 * rp.nsub + b) * rp.nc2 + c] = lh[b];
}

__global__ __launch_bounds__(kRevThreads) void k_rev2_part2(RevPlan rp, const uint32_t *bo, const uint32_t *bo2,
                                                            const uint32_t *pairs, uint32_t *pairs2) {
  __shared__ uint32_t gpos[kRev2MaxSub], lcnt[kRev2MaxSub], lstart[kRev2MaxSub];
  __shared__ uint32_t wsum[kRevThreads / 64];
  __shared__ uint32_t sval[kRev2Step];
  __shared__ uint8_t skey[kRev2Step];
  const uint32_t b1 = blockIdx.x / rp.nc2, c = blockIdx.x % rp.nc2;
  for (uint32_t b = threadIdx.x; b < rp.nsub; b += blockDim.x)
    gpos[b] = bo2[((size_t)b1 * rp.nsub + b) * rp.nc2 + c];
  uint32_t x0, x1;
  rev2_chunk(rp, bo, b1, c, x0, x1);
  const uint32_t m1 = (1u << rp.s1) - 1u, m2 = (1u << rp.s2) - 1u;
  for (uint32_t base = x0; base < x1; base += kRev2Step) {
    uint32_t key[kRev2Per], val[kRev2Per], pos[kRev2Per];
    bool ok[kRev2Per];
#pragma unroll
    for (int k = 0; k < kRev2Per; k++) {
      const uint32_t j = base + (uint32_t)k * blockDim.x + threadIdx.x;
      const uint32_t x = j < x1 ? pairs[j] : 0u;
      ok[k] = j < x1;
      key[k] = (x & m1) >> rp.s2;
      val[k] = ((x >> rp.s1) << rp.s2) | (x & m2);
    }
    rev2_local_sort(key, ok, rp.nsub, lcnt, lstart, wsum, pos);
#pragma unroll
    for (int k = 0; k < kRev2Per; k++)
      if (ok[k]) {
        sval[pos[k]] = val[k];
        skey[pos[k]] = (uint8_t)key[k];
      }
    __syncthreads();
    const uint32_t n = lstart[rp.nsub - 1] + lcnt[rp.nsub - 1];
    for (uint32_t j = threadIdx.x; j < n; j += blockDim.x) {
      const uint32_t b = skey[j];
      pairs2[gpos[b] + (j - lstart[b])] = sval[j];
    }
    __syncthreads();
    for (uint32_t b = threadIdx.x; b < rp.nsub; b += blockDim.x) gpos[b] += lcnt[b];
    __syncthreads();
  }
}

constexpr int kFillThreads = 512;  // more loads in flight per fine bucket
__global__ __launch_bounds__(kFillThreads) void k_rev2_fill(RevPlan rp, uint32_t cap, const uint32_t *bo2,
                                                            const uint32_t *pairs2, uint32_t *off, uint32_t *src) {
  constexpr uint32_t W = 1u << kRev2FineShift;
  __shared__ uint32_t cnt[W];
  __shared__ uint32_t wsum[kFillThreads / 64];
  __shared__ uint32_t stage[kRev2Stage];
  const uint32_t fb = blockIdx.x;  // fine bucket = coarse * nsub + sub
  const size_t nfine = (size_t)rp.nb1 * rp.nsub;
  const uint32_t s0 = bo2[(size_t)fb * rp.nc2], s1 = bo2[(size_t)(fb + 1) * rp.nc2];
  const uint32_t m2 = W - 1u;
  const uint32_t n = s1 - s0;
  const bool staged = n <= kRev2Stage;
  for (uint32_t i = threadIdx.x; i < W; i += blockDim.x) cnt[i] = 0;
  __syncthreads();
  // a bucket that fits the stage is read once, all of a thread's pairs in
  // flight together, and kept in registers for the placement pass
  constexpr int kPer = kRev2Stage / kFillThreads;
  uint32_t xr[kPer];
  if (staged) {
#pragma unroll
    for (int k = 0; k < kPer; k++) {
      const uint32_t j = s0 + (uint32_t)k * blockDim.x + threadIdx.x;
      xr[k] = j < s1 ? pairs2[j] : 0u;
    }
#pragma unroll
    for (int k = 0; k < kPer; k++)
      if (s0 + (uint32_t)k * blockDim.x + threadIdx.x < s1) atomicAdd(&cnt[xr[k] & m2], 1u);
  } else {
    for (uint32_t j = s0 + threadIdx.x; j < s1; j += blockDim.x) atomicAdd(&cnt[pairs2[j] & m2], 1u);
  }
  __syncthreads();
  // offsets: W = 128 counts, thread t < W owns count t
  const uint32_t c = threadIdx.x < W ? cnt[threadIdx.x] : 0u;
  uint32_t total;
  const uint32_t ex = block_excl_scan(c, wsum, total);
  const size_t v = (size_t)fb * W + threadIdx.x;
  if (threadIdx.x < W && v < cap) off[v] = s0 + ex;
  __syncthreads();
  if (threadIdx.x < W) cnt[threadIdx.x] = ex;
  __syncthreads();
  if (staged) {
#pragma unroll
    for (int k = 0; k < kPer; k++)
      if (s0 + (uint32_t)k * blockDim.x + threadIdx.x < s1) stage[atomicAdd(&cnt[xr[k] & m2], 1u)] = xr[k] >> rp.s2;
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < n; j += blockDim.x) src[s0 + j] = stage[j];
  } else {
    for (uint32_t j = s0 + threadIdx.x; j < s1; j += blockDim.x) {
      const uint32_t x = pairs2[j];
      src[s0 + atomicAdd(&cnt[x & m2], 1u)] = x >> rp.s2;
    }
  }
  if (fb == nfine - 1 && threadIdx.x == 0) off[cap] = s1;
}

hipError_t launch_reverse(PoolView p, int by_batch, const uint8_t *in_batch, const uint32_t *bidx,
                          const uint32_t *ids, uint32_t nrows, uint32_t *cnt, uint32_t *off, uint32_t *scan_tmp,
                          uint32_t *src, const RevBufs &rb, DevScalars *ds, hipStream_t s) {
  const RevPlan &rp = rb.plan;
  if (!by_batch && rp.two) {
    hipLaunchKernelGGL(k_rev2_count, dim3(rp.ng), dim3(kRevThreads), 0, s, p, rp, rb.bh);
    hipError_t e = launch_scan(rb.bh, rb.bo, (size_t)rp.nb1 * rp.ng, scan_tmp, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_rev2_part1, dim3(rp.ng), dim3(kRevThreads), 0, s, p, rp, rb.bo, rb.pairs);
    hipLaunchKernelGGL(k_rev2_count2, dim3(rp.nb1 * rp.nc2), dim3(kRevThreads), 0, s, rp, rb.bo, rb.pairs, rb.bh2);
    e = launch_scan(rb.bh2, rb.bo2, (size_t)rp.nb1 * rp.nsub * rp.nc2, scan_tmp, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_rev2_part2, dim3(rp.nb1 * rp.nc2), dim3(kRevThreads), 0, s, rp, rb.bo, rb.bo2, rb.pairs,
                       rb.pairs2);
    hipLaunchKernelGGL(k_rev2_fill, dim3(rp.nb1 * rp.nsub), dim3(kFillThreads), 0, s, rp, p.cap, rb.bo2, rb.pairs2,
                       off, src);
    hipLaunchKernelGGL(k_count_edges, dim3(1), dim3(64), 0, s, off, nrows, ds);
    return hipGetLastError();
  }
  if (!by_batch && rp.ok) {
    const size_t lds_b = (size_t)rp.nb * 4, lds_w = (size_t)4 << rp.shift;
    hipLaunchKernelGGL(k_revb_count, dim3(rp.ng), dim3(kRevThreads), lds_b, s, p, rp, rb.bh);
    hipError_t e = launch_scan(rb.bh, rb.bo, (size_t)rp.nb * rp.ng, scan_tmp, s);
    if (e != hipSuccess) return e;
    if (rp.packed) {
      hipLaunchKernelGGL(k_revb_part<true>, dim3(rp.ng), dim3(kRevThreads), lds_b, s, p, rp, rb.bo, rb.pairs);
      hipLaunchKernelGGL(k_revb_fill<true>, dim3(rp.nb), dim3(kRevThreads), lds_w, s, rp, p.cap, rb.bo, rb.pairs,
                         off, src);
    } else {
      hipLaunchKernelGGL(k_revb_part<false>, dim3(rp.ng), dim3(kRevThreads), lds_b, s, p, rp, rb.bo, rb.pairs);
      hipLaunchKernelGGL(k_revb_fill<false>, dim3(rp.nb), dim3(kRevThreads), lds_w, s, rp, p.cap, rb.bo, rb.pairs,
                         off, src);
    }
    hipLaunchKernelGGL(k_count_edges, dim3(1), dim3(64), 0, s, off, nrows, ds);
    return hipGetLastError();
  }
  if (by_batch && rp.ok && rb.pairs && rb.bh && ids) {
    int dev = 0, ncu = 0, lds_max = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || ncu <= 0)
      ncu = 256;
    if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) lds_max = 65536;
    const uint32_t lbits = revr_lbits(p.cap, lds_max);
    // one workgroup per CU (its bitmap fills the LDS); wgcnt holds rp.ng words
    const uint32_t g = std::max<uint32_t>(1, std::min<uint32_t>((uint32_t)ncu, rp.ng));
    const uint32_t ch = (p.cap + g - 1) / g;
    const size_t lds = ((size_t)1 << lbits) / 8;
    hipLaunchKernelGGL(k_revr_find, dim3(g), dim3(kRevrThreads), lds, s, p, ids, nrows, in_batch, ch, lbits,
                       rb.pairs, rb.bh);
    hipLaunchKernelGGL(k_revr_hist, dim3(g), dim3(kRevThreads), 0, s, p, ch, bidx, rb.pairs, rb.bh, cnt);
    hipError_t e = launch_scan(cnt, off, nrows, scan_tmp, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_revr_scatter, dim3(g), dim3(kRevThreads), 0, s, p, ch, bidx, rb.pairs, rb.bh, cnt, off,
                       src);
    hipLaunchKernelGGL(k_count_edges, dim3(1), dim3(64), 0, s, off, nrows, ds);
    return hipGetLastError();
  }
  const size_t total = (size_t)p.cap * p.R;
  uint32_t g = blocks_for(total, 256);
  if (g > 16384) g = 16384;
  hipLaunchKernelGGL(k_rev_hist, dim3(g), dim3(256), 0, s, p, by_batch, in_batch, bidx, cnt);
  hipError_t e = launch_scan(cnt, off, nrows, scan_tmp, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rev_scatter, dim3(g), dim3(256), 0, s, p, by_batch, in_batch, bidx, cnt, off, src);
  hipLaunchKernelGGL(k_count_edges, dim3(1), dim3(64), 0, s, off, nrows, ds);
  return hipGetLastError();
}

// Rows of a CSR sorted ascending into dst (one wave per row; sources in a
// row are distinct).  Rows up to 64 use a register bitonic sort, longer rows
// a rank count.
__global__ __launch_bounds__(64) void k_sort_rows(const uint32_t *off, uint32_t nrows, const uint32_t *src,
                                                  uint32_t *dst) {
  const int ln = lane();
  for (uint32_t r = blockIdx.x; r < nrows; r += gridDim.x) {
    const uint32_t b = off[r], e = off[r + 1], len = e - b;
    if (len == 0) continue;
    if (len <= 64) {
      float d[1] = {0.0f};
      uint32_t v[1] = {ln < (int)len ? src[b + ln] : kInvalid};
      wave_sort<1>(d, v);
      if (ln < (int)len) dst[b + ln] = v[0];
    } else {
      for (uint32_t i = ln; i < len; i += 64) {
        const uint32_t x = src[b + i];
        uint32_t rank = 0;
        for (uint32_t j = 0; j < len; j++) rank += src[b + j] < x ? 1u : 0u;
        dst[b + rank] = x;
      }
    }
  }
}
hipError_t launch_sort_rows(const uint32_t *off, uint32_t nrows, const uint32_t *src, uint32_t *dst, hipStream_t s) {
  if (nrows == 0) return hipSuccess;
  uint32_t g = nrows < 65536 ? nrows : 65536;
  hipLaunchKernelGGL(k_sort_rows, dim3(g), dim3(64), 0, s, off, nrows, src, dst);
  return hipGetLastError();
}

// Copies the fixed-width lists of every node with each row sorted ascending
// (INVALID, the largest value, last): the canonical form of Vamana lists,
// whose order carries no meaning.  One wave per row, R <= 64.
__global__ __launch_bounds__(64) void k_sort_adj_rows(const uint32_t *adj, uint32_t cap, uint32_t R, uint32_t *dst) {
  const int ln = lane();
  for (uint32_t u = blockIdx.x; u < cap; u += gridDim.x) {
    float d[1] = {0.0f};
    uint32_t v[1] = {ln < (int)R ? adj[(size_t)u * R + ln] : kInvalid};
    wave_sort<1>(d, v);
    if (ln < (int)R) dst[(size_t)u * R + ln] = v[0];
  }
}
hipError_t launch_sort_adj_rows(const uint32_t *adj, uint32_t cap, uint32_t R, uint32_t *dst, hipStream_t s) {
  if (cap == 0) return hipSuccess;
  const uint32_t g = cap < 65536 ? cap : 65536;
  hipLaunchKernelGGL(k_sort_adj_rows, dim3(g), dim3(64), 0, s, adj, cap, R, dst);
  return hipGetLastError();
}

// ---------------------------------------------------------------- medoid
// The active id minimising (squared distance to the centroid, id).
//  uint8: exact.  With n active ids and per-dimension sums S_j, the squared
//    distance of x to S/n is |n x - S|^2 / n^2, so ids are compared by the
//    integer key sum_j (n x_j - S_j)^2, held in 128 bits (each term is below
//    2^78).  Three passes over the active ids find the smallest high word,
//    then the smallest low word among those, then the smallest id with
//    exactly that key.
//  fp32: blocks of 1024 consecutive ids summed in id order, block sums added
//    in block order, divided by the active count; the distance to it is a
//    fused multiply-add chain in fp64 in dimension order.  The smallest
//    distance is found with a 64-bit atomic min on its bit pattern
//    (non-negative doubles order like their bits), then the smallest id with
//    exactly that distance.
constexpr uint32_t kCentroidBlock = 1024;

size_t medoid_tmp_bytes(uint32_t cap, uint32_t dim) {
  const size_t nb = (cap + kCentroidBlock - 1) / kCentroidBlock;
  return (nb * dim + dim) * sizeof(double) + 64;
}

__global__ void k_centroid_part(PoolView P, int kind, uint32_t dim, double *part, const DevScalars *ds) {
  if (!ds->need_medoid) return;
  const uint32_t j = blockIdx.y * blockDim.x + threadIdx.x;
  const uint32_t b = blockIdx.x;
  if (j >= dim) return;
  const uint32_t i0 = b * kCentroidBlock;
  const uint32_t i1 = i0 + kCentroidBlock < P.cap ? i0 + kCentroidBlock : P.cap;
  if (kind == kU8L2) {
    unsigned long long s = 0;
    for (uint32_t i = i0; i < i1; i++)
      if (P.active[i]) s += P.vecs[(size_t)i * P.stride + j];
    reinterpret_cast<unsigned long long *>(part)[(size_t)b * dim + j] = s;
  } else {
    double s = 0.0;
    for (uint32_t i = i0; i < i1; i++)
      if (P.active[i]) s = s + (double)reinterpret_cast<const float *>(P.vecs + (size_t)i * P.stride)[j];
    part[(size_t)b * dim + j] = s;
  }
}
// fp32: cent[j] = the centroid coordinate; uint8: cent[j] holds S_j as a
// 64-bit integer.
__global__ void k_centroid_sum(int kind, uint32_t dim, uint32_t nb, const double *part, double *cent,
                               unsigned long long n, DevScalars *ds) {
  if (!ds->need_medoid) return;
  const uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j == 0) {
    ds->best_bits = ~0ull;
    ds->best_hi = ~0ull;
    ds->best_id = kInvalid;
  }
  if (j >= dim) return;
  if (kind == kU8L2) {
    const unsigned long long *pi = reinterpret_cast<const unsigned long long *>(part);
    unsigned long long s = 0;
    for (uint32_t b = 0; b < nb; b++) s += pi[(size_t)b * dim + j];
    reinterpret_cast<unsigned long long *>(cent)[j] = s;
  } else {
    double t = 0.0;
    for (uint32_t b = 0; b < nb; b++) t = t + part[(size_t)b * dim + j];
    cent[j] = t / (double)n;
  }
}
__device__ __forceinline__ double dist_to_centroid(const PoolView &P, uint32_t dim, uint32_t i, const double *cent) {
  double s = 0.0;
  const float *row = reinterpret_cast<const float *>(P.vecs + (size_t)i * P.stride);
  for (uint32_t j = 0; j < dim; j++) {
    const double t = (double)row[j] - cent[j];
    s = __builtin_fma(t, t, s);
  }
  return s;
}
__device__ __forceinline__ unsigned __int128 u8_centroid_key(const PoolView &P, uint32_t dim, uint32_t i,
                                                            const double *cent, unsigned long long n) {
  const unsigned long long *S = reinterpret_cast<const unsigned long long *>(cent);
  const uint8_t *row = P.vecs + (size_t)i * P.stride;
  unsigned __int128 key = 0;
  for (uint32_t j = 0; j < dim; j++) {
    const __int128 t = (__int128)n * row[j] - (__int128)S[j];
    key += (unsigned __int128)(t * t);
  }
  return key;
}
// pass 0: smallest high word (uint8) or smallest distance (fp32); pass 1
// (uint8 only): smallest low word among keys with the smallest high word;
// pass 2: smallest id with exactly the smallest key.
__global__ void k_medoid_pass(PoolView P, int kind, uint32_t dim, const double *cent, unsigned long long n,
                              int pass, DevScalars *ds) {
  if (!ds->need_medoid) return;
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= P.cap || !P.active[i]) return;
  if (kind == kU8L2) {
    const unsigned __int128 key = u8_centroid_key(P, dim, i, cent, n);
    const unsigned long long hi = (unsigned long long)(key >> 64), lo = (unsigned long long)key;
    if (pass == 0) atomicMin(&ds->best_hi, hi);
    else if (pass == 1) { if (hi == ds->best_hi) atomicMin(&ds->best_bits, lo); }
    else if (hi == ds->best_hi && lo == ds->best_bits) atomicMin(&ds->best_id, i);
  } else {
    const unsigned long long bits = (unsigned long long)__double_as_longlong(dist_to_centroid(P, dim, i, cent));
    if (pass == 0) atomicMin(&ds->best_bits, bits);
    else if (pass == 2 && bits == ds->best_bits) atomicMin(&ds->best_id, i);
  }
}
__global__ void k_medoid_store(DevScalars *ds) {
  if (ds->need_medoid) ds->medoid = ds->best_id;
  ds->need_medoid = 0;
}
// A new medoid is needed when the current one is in the delete batch.
__global__ void k_medoid_need(DevScalars *ds, const uint8_t *in_batch, int force) {
  const uint32_t m = ds->medoid;
  ds->need_medoid = force ? 1u : ((m != kInvalid && in_batch && in_batch[m]) ? 1u : 0u);
}
hipError_t launch_medoid_need(DevScalars *ds, const uint8_t *in_batch, int force, hipStream_t s) {
  hipLaunchKernelGGL(k_medoid_need, dim3(1), dim3(1), 0, s, ds, in_batch, force);
  return hipGetLastError();
}

hipError_t launch_medoid(PoolView p, int kind, uint32_t dim, uint64_t n_active, void *tmp, DevScalars *ds,
                         hipStream_t s) {
  if (n_active == 0) {
    hipLaunchKernelGGL(k_centroid_sum, dim3(1), dim3(64), 0, s, kind, 0u, 0u, (const double *)nullptr,
                       (double *)nullptr, 1ull, ds);
    hipLaunchKernelGGL(k_medoid_store, dim3(1), dim3(1), 0, s, ds);
    return hipGetLastError();
  }
  const uint32_t nb = (p.cap + kCentroidBlock - 1) / kCentroidBlock;
  double *part = reinterpret_cast<double *>(tmp);
  double *cent = part + (size_t)nb * dim;
  hipLaunchKernelGGL(k_centroid_part, dim3(nb, (dim + 63) / 64), dim3(64), 0, s, p, kind, dim, part,
                     (const DevScalars *)ds);
  hipLaunchKernelGGL(k_centroid_sum, dim3((dim + 63) / 64), dim3(64), 0, s, kind, dim, nb, part, cent,
                     (unsigned long long)n_active, ds);
  for (int pass = 0; pass < 3; pass++) {
    if (pass == 1 && kind != kU8L2) continue;
    hipLaunchKernelGGL(k_medoid_pass, dim3(blocks_for(p.cap, 256)), dim3(256), 0, s, p, kind, dim,
                       (const double *)cent, (unsigned long long)n_active, pass, ds);
  }
  hipLaunchKernelGGL(k_medoid_store, dim3(1), dim3(1), 0, s, ds);
  return hipGetLastError();
}

}  // namespace gr
