// api.hip -- the C ABI (include/grand.h): resource pool, argument
// validation before any mutation, and the fixed kernel sequence of each
// batch operation on one HIP stream (one host synchronisation per call).
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "index.h"
#include "vec.h"

using namespace gr;

// Device memory of grand_search_static: the staged query rows and the result
// lists of one call, in a fixed array that every GPU the library runs on
// holds from module load until the process ends.  In host code `scratch` is
// only a symbol; its device address on each GPU comes from
// hipGetSymbolAddress (scratch_of below) and is the only form passed on.
constexpr size_t kStaticScratchBytes = GRAND_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch[kMaxDevices] = {};

// Address of this device's `scratch`, looked up once per device with the
// device current.  Returns null (and the HIP error) when the lookup fails.
uint8_t *scratch_of(int dev, hipError_t *err) {
  *err = hipSuccess;
  if (dev < 0 || dev >= kMaxDevices) {
    *err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
      return nullptr;
    }
    g_scratch[dev] = static_cast<uint8_t *>(ptr);
  }
  return g_scratch[dev];
}
}  // namespace

struct grand_index {
  grand_params p{};
  hipStream_t stream = nullptr;
  uint8_t *static_scratch = nullptr;  // this device's address of `scratch`
  int kind = 0, vc = 0;
  size_t esize = 0, row_bytes = 0, stride = 0;  // caller row bytes; stored row bytes (16-byte multiple)
  uint32_t sdim = 0;   // stored elements per row: dim, or dim + 1 with GRAND_MIPS
  bool mips = false;
  int nch = 0;
  uint32_t iters = 0;
  double coef = 0.0;
  PoolView pool{};
  // pool-sized arrays (allocated once, Section 3.1 resource pool)
  uint8_t *in_batch = nullptr;
  uint32_t *bidx = nullptr, *mark = nullptr, *cnt = nullptr, *off = nullptr, *dirty = nullptr, *queue = nullptr, *qflag = nullptr;
  uint32_t *rev_off = nullptr, *rev_src = nullptr, *rev_sorted = nullptr, *scan_tmp = nullptr;
  RevBufs rev{};  // bucketed full reverse-graph build
  GroupBufs grp{};  // two-level grouping of records (null members: one-level form)
  size_t rev_sorted_cap = 0;
  void *med_tmp = nullptr;
  uint32_t epoch = 0;
  uint32_t medoid = GRAND_INVALID;
  uint64_t n_active = 0;
  DevScalars *ds = nullptr;       // device
  DevScalars *hs = nullptr;       // pinned host mirror
  // per-batch buffers
  uint32_t bcap = 0;
  uint32_t *b_ids = nullptr, *v_ids = nullptr, *v_n = nullptr, *c_ids = nullptr, *rcount = nullptr,
           *rofs = nullptr, *rchunk = nullptr, *coff = nullptr;
  uint4 *cdesc = nullptr;
  hipEvent_t ev_total = nullptr;  // record count of a delete batch copied to the host
  // second stream: a delete batch builds the reverse graph there while its
  // searches run on the main stream (both only read the graph)
  hipStream_t side = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  float *v_d = nullptr, *c_d = nullptr;
  uint8_t *b_vecs = nullptr;
  uint32_t c_stride = 0;
  size_t rcap = 0;
  uint32_t *rec_t = nullptr, *rec_s = nullptr, *gsrc = nullptr;
  float *rec_d = nullptr, *gd = nullptr;
  // query buffers
  uint32_t qcap = 0, qk = 0;
  uint8_t *q_vecs = nullptr;
  uint32_t *q_ids = nullptr;
  float *q_d = nullptr;
  // counting runs: an exact visited bitmap per search (measurement only)
  bool counting = false;
  uint32_t *vis = nullptr;
  size_t vis_cap = 0;  // words
  // timing and stats
  bool timing = false;
  std::vector<std::tuple<int, hipEvent_t, hipEvent_t>> pending;
  std::vector<hipEvent_t> spare_events;
  grand_stats_t st{};
  bool poisoned = false;
  std::string err;
};

namespace {

grand_status fail(grand_index *h, grand_status code, const std::string &msg) {
  h->err = msg;
  return code;
}

grand_status fail_dev(grand_index *h, hipError_t e, const char *what) {
  h->poisoned = true;
  h->err = std::string("HIP error in ") + what + ": " + hipGetErrorString(e);
  return GRAND_E_DEVICE;
}

#define HCHK(h, x)                                             \
  do {                                                         \
    hipError_t e_ = (x);                                       \
    if (e_ != hipSuccess) return fail_dev((h), e_, #x);        \
  } while (0)

template <class T>
hipError_t dalloc(T **p, size_t count) {
  *p = nullptr;
  if (count == 0) count = 1;
  return hipMalloc((void **)p, count * sizeof(T));
}

template <class T>
void dfree(T *&p) {
  if (p) (void)hipFree((void *)p);
  p = nullptr;
}

hipEvent_t get_event(grand_index *h) {
  if (!h->spare_events.empty()) {
    hipEvent_t e = h->spare_events.back();
    h->spare_events.pop_back();
    return e;
  }
  // phase markers need timestamps only: no system-scope fence
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Records HIP events around one phase of a call when timing is enabled.
// Phases of a few microseconds (validation, staging, clearing, the medoid
// check) are not timed: every recorded event leaves a gap of several
// microseconds between kernels on the stream.
static bool timed_phase(int ph) {
  return ph != GRAND_PH_VALIDATE && ph != GRAND_PH_STAGE && ph != GRAND_PH_CLEAR && ph != GRAND_PH_MEDOID;
}
struct Phase {
  grand_index *h;
  int ph;
  hipStream_t st;  // stream the phase's work goes to
  Phase(grand_index *h_, int ph_, hipStream_t st_ = nullptr) : h(h_), ph(ph_), st(st_ ? st_ : h_->stream) {
    if (!h->timing || !timed_phase(ph)) return;
    hipEvent_t e = get_event(h);
    if (!e) return;
    (void)hipEventRecord(e, st);
    h->pending.emplace_back(ph, e, nullptr);
  }
  ~Phase() {
    if (!h->timing || !timed_phase(ph) || h->pending.empty()) return;
    auto &last = h->pending.back();
    if (std::get<0>(last) != ph || std::get<2>(last) != nullptr) return;
    hipEvent_t e = get_event(h);
    if (!e) return;
    (void)hipEventRecord(e, st);
    std::get<2>(last) = e;
  }
};

// End of every call: wait for the stream, fold timings, refresh the host
// mirror of the device scalars (medoid, counters).
grand_status finish(grand_index *h) {
  HCHK(h, hipMemcpyAsync(h->hs, h->ds, kScalarBytes, hipMemcpyDeviceToHost, h->stream));
  HCHK(h, hipStreamSynchronize(h->stream));
  for (auto &t : h->pending) {
    float ms = 0.0f;
    if (std::get<2>(t)) {
      if (hipEventElapsedTime(&ms, std::get<1>(t), std::get<2>(t)) == hipSuccess) {
        h->st.phase_ms[std::get<0>(t)] += ms;
        h->st.phase_calls[std::get<0>(t)] += 1;
      }
      h->spare_events.push_back(std::get<2>(t));
    }
    h->spare_events.push_back(std::get<1>(t));
  }
  h->pending.clear();
  h->medoid = h->hs->medoid;
  return GRAND_OK;
}

grand_status check_usable(grand_index *h) {
  if (!h) return GRAND_E_ARG;
  if (h->poisoned) return GRAND_E_STATE;
  h->err.clear();
  return GRAND_OK;
}

// Reads the validation result (one synchronisation) and maps it to a status.
grand_status read_validation(grand_index *h) {
  HCHK(h, hipMemcpyAsync(h->hs, h->ds, kScalarBytes, hipMemcpyDeviceToHost, h->stream));
  HCHK(h, hipStreamSynchronize(h->stream));
  const uint32_t code = h->hs->err_code, id = h->hs->err_id;
  if (code == 0) return GRAND_OK;
  char buf[160];
  switch (code) {
    case kErrRange: snprintf(buf, sizeof buf, "id %u is out of range", id); return fail(h, GRAND_E_ID, buf);
    case kErrRepeat: snprintf(buf, sizeof buf, "id %u is repeated in the batch", id); return fail(h, GRAND_E_ID, buf);
    case kErrState: snprintf(buf, sizeof buf, "id %u is in the wrong active state", id); return fail(h, GRAND_E_ID, buf);
    case kErrNorm: snprintf(buf, sizeof buf, "row %u has a norm above mips_norm", id); return fail(h, GRAND_E_ARG, buf);
    case kErrInit:
      snprintf(buf, sizeof buf, "initial list of position %u is not knn distinct other positions below n", id);
      return fail(h, GRAND_E_ARG, buf);
    default: snprintf(buf, sizeof buf, "row %u holds a non-finite element", id); return fail(h, GRAND_E_ARG, buf);
  }
}

grand_status clear_errors(grand_index *h) {
  HCHK(h, launch_fill_u32(&h->ds->err_code, 0u, 2, h->stream));  // err_code and err_id
  return GRAND_OK;
}

grand_status ensure_batch(grand_index *h, uint32_t n) {
  if (n <= h->bcap) return GRAND_OK;
  HCHK(h, hipStreamSynchronize(h->stream));
  uint32_t nc = std::max<uint32_t>(n, h->bcap + h->bcap / 2);
  dfree(h->b_ids); dfree(h->v_ids); dfree(h->v_n); dfree(h->c_ids); dfree(h->rcount); dfree(h->rofs);
  dfree(h->v_d); dfree(h->c_d); dfree(h->b_vecs); dfree(h->rchunk); dfree(h->coff);
  dfree(h->cdesc);
  h->bcap = 0;
  // work chunks of a delete batch (64 or more positions each): at most
  // (in-edges of the batch) / 64 + 2 per deleted node, as R <= 64 there
  const size_t nchunk = (size_t)h->p.capacity * h->p.R / 64 + 2 * (size_t)nc + 1;
  const size_t vs = (size_t)nc * h->iters;
  if (dalloc(&h->b_ids, nc) || dalloc(&h->v_ids, vs) || dalloc(&h->v_d, vs) || dalloc(&h->v_n, nc) ||
      dalloc(&h->c_ids, (size_t)nc * h->c_stride) || dalloc(&h->c_d, (size_t)nc * h->c_stride) ||
      dalloc(&h->rcount, (size_t)nc + 1) || dalloc(&h->rofs, (size_t)nc + 1) ||
      dalloc(&h->rchunk, (size_t)nc + 1) || dalloc(&h->coff, (size_t)nc + 1) || dalloc(&h->cdesc, 2 * nchunk) ||
      dalloc(&h->b_vecs, (size_t)nc * h->stride)) {
    (void)hipGetLastError();
    return fail(h, GRAND_E_OOM, "device allocation of batch buffers failed");
  }
  HCHK(h, hipMemset(h->b_vecs, 0, (size_t)nc * h->stride));
  h->bcap = nc;
  return GRAND_OK;
}

grand_status ensure_records(grand_index *h, size_t n) {
  if (n <= h->rcap) return GRAND_OK;
  HCHK(h, hipStreamSynchronize(h->stream));
  size_t nc = std::max<size_t>(n, h->rcap + h->rcap / 2);
  dfree(h->rec_t); dfree(h->rec_s); dfree(h->rec_d); dfree(h->gsrc); dfree(h->gd);
  dfree(h->grp.pt); dfree(h->grp.ps); dfree(h->grp.pd); dfree(h->grp.mat); dfree(h->grp.mato); dfree(h->grp.tmp);
  h->rcap = 0;
  h->grp.rcap = 0;
  const bool two = group_two_level(h->p.capacity);
  const size_t mw = two ? group_mat_words(h->p.capacity, nc) : 0;
  if (dalloc(&h->rec_t, nc) || dalloc(&h->rec_s, nc) || dalloc(&h->rec_d, nc) || dalloc(&h->gsrc, nc) ||
      dalloc(&h->gd, nc) ||
      (two && (dalloc(&h->grp.pt, nc) || dalloc(&h->grp.ps, nc) || dalloc(&h->grp.pd, nc) ||
               dalloc(&h->grp.mat, mw) || dalloc(&h->grp.mato, mw) || dalloc(&h->grp.tmp, scan_tmp_words(mw))))) {
    (void)hipGetLastError();
    return fail(h, GRAND_E_OOM, "device allocation of record buffers failed");
  }
  h->rcap = nc;
  if (two) h->grp.rcap = nc;
  return GRAND_OK;
}

grand_status ensure_query(grand_index *h, uint32_t nq, uint32_t k) {
  if (nq <= h->qcap && k <= h->qk) return GRAND_OK;
  HCHK(h, hipStreamSynchronize(h->stream));
  const uint32_t nc = std::max(nq, h->qcap), kc = std::max(k, h->qk);
  dfree(h->q_vecs); dfree(h->q_ids); dfree(h->q_d);
  h->qcap = h->qk = 0;
  if (dalloc(&h->q_vecs, (size_t)nc * h->stride) || dalloc(&h->q_ids, (size_t)nc * kc) ||
      dalloc(&h->q_d, (size_t)nc * kc)) {
    (void)hipGetLastError();
    return fail(h, GRAND_E_OOM, "device allocation of query buffers failed");
  }
  HCHK(h, hipMemset(h->q_vecs, 0, (size_t)nc * h->stride));
  h->qcap = nc;
  h->qk = kc;
  return GRAND_OK;
}

// Copies n packed rows (host or device) into a padded staging buffer.
grand_status stage_rows(grand_index *h, uint8_t *dst, const void *src, uint32_t n) {
  HCHK(h, hipMemcpy2DAsync(dst, h->stride, src, h->row_bytes, h->row_bytes, n, hipMemcpyDefault, h->stream));
  return GRAND_OK;
}

uint32_t persistent_grid(size_t upper) {
  const size_t g = std::min<size_t>(upper, 256 * 32);
  return (uint32_t)std::max<size_t>(g, 1);
}

grand_status run_group(grand_index *h, size_t nrec) {
  Phase ph(h, GRAND_PH_GROUP);
  const GroupBufs *gb = h->grp.dpad && h->grp.rcap >= nrec ? &h->grp : nullptr;
  HCHK(h, launch_group(h->rec_t, h->rec_s, h->rec_d, nrec, h->p.capacity, h->cnt, h->off, h->scan_tmp, h->gsrc,
                       h->gd, h->dirty, h->ds, gb, h->stream));
  return GRAND_OK;
}

grand_status run_rebuild(grand_index *h, size_t nrec, const uint8_t *in_batch) {
  Phase ph(h, GRAND_PH_REBUILD);
  RebuildArgs a{};
  a.pool = h->pool;
  a.dirty = h->dirty;
  a.queue = h->queue;
  a.queue_n = &h->ds->n_queue;
  a.qflag = h->qflag;
  a.flag_cap = h->p.capacity;
  a.scan_tmp = h->scan_tmp;
  a.goff = h->off;
  a.gsrc = h->gsrc;
  a.gd = h->gd;
  a.in_batch = in_batch;
  a.P = h->p.P;
  a.coef = h->coef;
  a.ds = h->ds;
  HCHK(h, launch_rebuild(h->kind, h->vc, h->p.R, h->p.P, a, persistent_grid(nrec), h->stream));
  return GRAND_OK;
}

grand_status run_medoid(grand_index *h, const uint8_t *in_batch, int force) {
  Phase ph(h, GRAND_PH_MEDOID);
  HCHK(h, launch_medoid_need(h->ds, in_batch, force, h->stream));
  HCHK(h, launch_medoid(h->pool, h->kind, h->sdim, h->n_active, h->med_tmp, h->ds, h->stream));
  return GRAND_OK;
}

// Counting runs: gives a search launch a cleared visited bitmap of one bit
// per pool id for each of its nq searches (grown on demand).
grand_status prep_counting(grand_index *h, SearchArgs &a) {
  if (!h->counting || a.nq == 0) return GRAND_OK;
  const size_t words = ((size_t)h->p.capacity + 31) / 32;
  const size_t need = words * a.nq;
  if (need > h->vis_cap) {
    HCHK(h, hipStreamSynchronize(h->stream));
    dfree(h->vis);
    h->vis_cap = 0;
    if (dalloc(&h->vis, need)) {
      (void)hipGetLastError();
      return fail(h, GRAND_E_OOM, "device allocation of the counting bitmap failed");
    }
    h->vis_cap = need;
  }
  HCHK(h, launch_fill_u32(h->vis, 0u, need, h->stream));
  a.vis = h->vis;
  a.vis_words = (uint32_t)words;
  return GRAND_OK;
}

// The reverse graph of the current graph: rows of every id (full) or of the
// batch positions of the delete batch (by_batch).  The source array is part
// of the resource pool (capacity x R entries bound every reverse graph).
grand_status run_reverse(grand_index *h, int by_batch, uint32_t n, hipStream_t st = nullptr) {
  Phase ph(h, GRAND_PH_REVERSE, st);
  const uint32_t nrows = by_batch ? n : h->p.capacity;
  HCHK(h, launch_reverse(h->pool, by_batch, h->in_batch, h->bidx, by_batch ? h->b_ids : nullptr, nrows, h->cnt,
                         h->rev_off, h->scan_tmp, h->rev_src, h->rev, h->ds, st ? st : h->stream));
  return GRAND_OK;
}

grand_status vamana_insert(grand_index *h, uint32_t n, uint64_t n0) {
  const uint32_t R = h->p.R;
  if (n0 == 0) {
    Phase ph(h, GRAND_PH_BOOTSTRAP);
    BootArgs b{};
    b.pool = h->pool;
    b.ids = h->b_ids;
    b.n = n;
    b.want = std::min<uint32_t>(n - 1, h->p.L_build);
    b.o_ids = h->v_ids;
    b.o_d = h->v_d;
    b.o_n = h->v_n;
    b.o_stride = h->iters;
    HCHK(h, launch_bootstrap(h->kind, h->vc, b, h->stream));
  } else {
    Phase ph(h, GRAND_PH_SEARCH_INSERT);
    SearchArgs a{};
    a.pool = h->pool;
    a.qids = h->b_ids;
    a.nq = n;
    a.start = h->medoid;
    a.ell = h->p.L_build;
    a.max_iters = h->iters;
    a.which = 0;
    a.v_ids = h->v_ids;
    a.v_d = h->v_d;
    a.v_n = h->v_n;
    a.v_stride = h->iters;
    a.ds = h->ds;
    if (grand_status s_ = prep_counting(h, a)) return s_;
    HCHK(h, launch_search(h->kind, h->vc, a, h->stream));
  }
  grand_status s = ensure_records(h, (size_t)n * R);
  if (s != GRAND_OK) return s;
  {
    Phase ph(h, GRAND_PH_PRUNE_FWD);
    FwdPruneArgs f{};
    f.pool = h->pool;
    f.ids = h->b_ids;
    f.n = n;
    f.v_ids = h->v_ids;
    f.v_d = h->v_d;
    f.v_n = h->v_n;
    f.v_stride = h->iters;
    f.coef = h->coef;
    f.rec_t = h->rec_t;
    f.rec_s = h->rec_s;
    f.rec_d = h->rec_d;
    f.ds = h->ds;
    HCHK(h, launch_fwd_prune(h->kind, h->vc, h->iters, f, h->stream));
  }
  s = run_group(h, (size_t)n * R);
  if (s != GRAND_OK) return s;
  return run_rebuild(h, (size_t)n * R, nullptr);
}

grand_status cagra_insert(grand_index *h, uint32_t n, uint64_t n0) {
  const uint32_t R = h->p.R;
  if (n0 == 0) {
    Phase ph(h, GRAND_PH_BOOTSTRAP);
    BootArgs b{};
    b.pool = h->pool;
    b.ids = h->b_ids;
    b.n = n;
    b.want = std::min<uint32_t>(n - 1, R);
    b.o_ids = h->c_ids;
    b.o_d = h->c_d;
    b.o_n = nullptr;
    b.o_stride = R;
    HCHK(h, launch_bootstrap(h->kind, h->vc, b, h->stream));
  } else {
    Phase ph(h, GRAND_PH_SEARCH_INSERT);
    SearchArgs a{};
    a.pool = h->pool;
    a.qids = h->b_ids;
    a.nq = n;
    a.start = h->medoid;
    a.ell = h->p.L_build;
    a.max_iters = h->iters;
    a.which = 0;
    a.c_ids = h->c_ids;
    a.c_d = h->c_d;
    a.c_out = R;
    a.ds = h->ds;
    if (grand_status s_ = prep_counting(h, a)) return s_;
    HCHK(h, launch_search(h->kind, h->vc, a, h->stream));
  }
  grand_status s = ensure_records(h, (size_t)n * R);
  if (s != GRAND_OK) return s;
  {
    Phase ph(h, GRAND_PH_CAGRA_DETOUR);
    HCHK(h, launch_cagra_fwd(h->pool, h->b_ids, n, h->c_ids, h->c_d, h->rec_t, h->rec_s, h->rec_d, h->stream));
  }
  CagraArgs c{};
  c.pool = h->pool;
  c.bidx = h->bidx;
  c.fwd = h->c_ids;
  c.ds = h->ds;
  if (h->p.cas_mode == GRAND_CAS_RACING) {
    Phase ph(h, GRAND_PH_CAGRA_DETOUR);
    c.rec_t = h->rec_t;
    c.rec_s = h->rec_s;
    c.nrec = n * R;
    HCHK(h, launch_cagra_racing(c, h->stream));
    return GRAND_OK;
  }
  s = run_group(h, (size_t)n * R);
  if (s != GRAND_OK) return s;
  Phase ph(h, GRAND_PH_CAGRA_DETOUR);
  c.list = h->dirty;
  c.goff = h->off;
  c.gsrc = h->gsrc;
  c.gd = h->gd;
  HCHK(h, launch_cagra_detour(c, persistent_grid((size_t)n * R), h->stream));
  return GRAND_OK;
}

grand_status vamana_delete(grand_index *h, uint32_t n) {
  const uint32_t kr = h->p.k_repair;
  const int by_batch = h->p.rev_mode == GRAND_REV_BATCH;
  // the reverse graph (side stream) and the searches from the deleted
  // points (main stream) both only read the graph: they run together (the
  // searches are issued first), and the repair waits for both
  HCHK(h, hipEventRecord(h->ev_fork, h->stream));
  HCHK(h, hipStreamWaitEvent(h->side, h->ev_fork, 0));
  grand_status s;
  {
    Phase ph(h, GRAND_PH_SEARCH_DELETE);
    SearchArgs a{};
    a.pool = h->pool;
    a.qids = h->b_ids;
    a.nq = n;
    a.start = h->medoid;
    a.ell = h->p.L_build;
    a.max_iters = h->iters;
    a.which = 1;
    a.c_ids = h->c_ids;
    a.c_d = h->c_d;
    a.c_out = kr;
    a.c_filter = h->in_batch;
    a.c_by_id = 1;
    a.ds = h->ds;
    if (grand_status s_ = prep_counting(h, a)) return s_;
    HCHK(h, launch_search(h->kind, h->vc, a, h->stream));
  }
  s = run_reverse(h, by_batch, n, h->side);
  if (s != GRAND_OK) return s;
  HCHK(h, hipEventRecord(h->ev_join, h->side));
  HCHK(h, hipStreamWaitEvent(h->stream, h->ev_join, 0));
  RepairArgs r{};
  r.pool = h->pool;
  r.ids = h->b_ids;
  r.n = n;
  r.in_batch = h->in_batch;
  r.ci = h->c_ids;
  r.kr = kr;
  r.rev_off = h->rev_off;
  r.rev_src = h->rev_src;
  r.rev_by_batch = by_batch;
  r.c = h->p.c;
  r.rofs = h->rofs;
  r.coff = h->coff;
  r.cdesc = h->cdesc;
  r.cw = repair_chunk_width(h->kind, h->pool, kr, h->p.c);
  r.ds = h->ds;
  // record offsets and work chunks; the record count reaches the host
  // through an event while the repair runs, so the stream never drains
  HCHK(h, launch_repair_plan(r, h->rcount, h->rchunk, h->stream));
  HCHK(h, launch_scan(h->rcount, h->rofs, n, h->scan_tmp, h->stream));
  const bool chunked = repair_chunked(h->kind, h->pool, kr, h->p.c);
  if (chunked) {
    HCHK(h, launch_scan(h->rchunk, h->coff, n, h->scan_tmp, h->stream));
    HCHK(h, launch_repair_map(r, h->cdesc, h->stream));
  }
  HCHK(h, hipMemcpyAsync(&h->hs->n_dirty, h->rofs + n, sizeof(uint32_t), hipMemcpyDeviceToHost, h->stream));
  HCHK(h, hipEventRecord(h->ev_total, h->stream));
  const uint32_t grid = chunked ? persistent_grid((size_t)h->p.capacity * h->p.R / 64 + 2 * (size_t)n) : n;
  auto repair = [&]() -> grand_status {
    Phase ph(h, GRAND_PH_REPAIR);
    r.rec_t = h->rec_t;
    r.rec_s = h->rec_s;
    r.rec_d = h->rec_d;
    r.rcap = h->rcap;
    HCHK(h, launch_repair(h->kind, h->vc, r, grid, h->stream));
    return GRAND_OK;
  };
  if ((s = repair()) != GRAND_OK) return s;
  HCHK(h, hipEventSynchronize(h->ev_total));
  const size_t total = h->hs->n_dirty;
  if (total > h->rcap) {  // the launch above wrote nothing: grow and repeat it
    if ((s = ensure_records(h, total)) != GRAND_OK) return s;
    if ((s = repair()) != GRAND_OK) return s;
  }
  s = run_group(h, total);
  if (s != GRAND_OK) return s;
  return run_rebuild(h, total, h->in_batch);
}

grand_status cagra_delete(grand_index *h, uint32_t n) {
  const int by_batch = h->p.rev_mode == GRAND_REV_BATCH;
  grand_status s = run_reverse(h, by_batch, n);
  if (s != GRAND_OK) return s;
  Phase ph(h, GRAND_PH_CAGRA_PICKONE);
  h->epoch++;
  CagraArgs c{};
  if (by_batch) {
    // the batch's reverse rows are one contiguous array: every entry is an
    // in-neighbour of the batch, the first one to mark a node takes it
    c.list = h->rev_src;
    c.list_n = h->rev_off + n;
    c.dedupe = 1;
    c.mark = h->mark;
    c.epoch = h->epoch;
  } else {
    HCHK(h, launch_cagra_affected(h->b_ids, n, h->in_batch, h->rev_off, h->rev_src, by_batch, h->mark, h->epoch,
                                  h->dirty, h->ds, h->stream));
    c.list = h->dirty;
    c.list_n = &h->ds->n_dirty;
  }
  c.pool = h->pool;
  c.bidx = h->bidx;
  c.in_batch = h->in_batch;
  c.rev_off = h->rev_off;
  c.rev_src = h->rev_src;
  c.rev_by_batch = by_batch;
  c.ds = h->ds;
  HCHK(h, launch_cagra_pickone(c, persistent_grid(h->p.capacity), h->stream));
  return GRAND_OK;
}

bool params_ok(const grand_params *p, std::string &why) {
  if (!p || p->struct_size != sizeof(grand_params)) { why = "grand_params.struct_size mismatch"; return false; }
  if (p->algo != GRAND_VAMANA && p->algo != GRAND_CAGRA) { why = "unknown algo"; return false; }
  if (p->dtype != GRAND_F32 && p->dtype != GRAND_U8) { why = "unknown dtype"; return false; }
  if (p->metric != GRAND_L2 && p->metric != GRAND_IP && p->metric != GRAND_MIPS) { why = "unknown metric"; return false; }
  if (p->metric == GRAND_MIPS && (p->dtype != GRAND_F32 || !(p->mips_norm > 0.0f) || !isfinite(p->mips_norm))) {
    why = "GRAND_MIPS needs fp32 data and a finite mips_norm > 0";
    return false;
  }
  if (p->metric == GRAND_IP && (p->dtype != GRAND_F32 || p->algo != GRAND_CAGRA)) {
    why = "inner product is supported for fp32 CAGRA indexes (Vamana uses L2)";
    return false;
  }
  if (p->dim == 0) { why = "dim must be positive"; return false; }
  if (p->capacity == 0 || p->capacity >= 0x7FFFFFFFu) { why = "capacity must be in [1, 2^31-1)"; return false; }
  if (p->R == 0 || p->R > 64) { why = "R must be in [1, 64]"; return false; }
  if ((uint64_t)p->capacity * p->R >= 0xFFFFFFFFull) { why = "capacity * R must be < 2^32"; return false; }
  if (p->L_build == 0 || p->L_build > 256) { why = "L_build must be in [1, 256]"; return false; }
  const uint32_t it = p->max_iters ? p->max_iters : 2 * p->L_build;
  if (it < p->L_build || it > 256) { why = "max_iters must be in [L_build, 256]"; return false; }
  if (p->P == 0 || p->P > 128 || p->R + p->P > 256) { why = "P must be in [1, 128] with R + P <= 256"; return false; }
  if (p->k_repair == 0 || p->k_repair > 64) { why = "k_repair must be in [1, 64]"; return false; }
  if (p->c > 64) { why = "c must be <= 64"; return false; }
  if (!(p->alpha >= 0.0f) || !isfinite(p->alpha)) { why = "alpha must be finite and >= 0"; return false; }
  if (p->prune_rule != GRAND_ALPHA_ON_DIST && p->prune_rule != GRAND_ALPHA_ON_L2) { why = "bad prune_rule"; return false; }
  if (p->cas_mode != GRAND_CAS_GROUPED && p->cas_mode != GRAND_CAS_RACING) { why = "bad cas_mode"; return false; }
  if (p->rev_mode != GRAND_REV_FULL && p->rev_mode != GRAND_REV_BATCH) { why = "bad rev_mode"; return false; }
  return true;
}

void release(grand_index *h) {
  if (h->pool.vecs) (void)hipSetDevice(h->p.device);
  dfree(h->pool.vecs); dfree(h->pool.adj); dfree(h->pool.deg); dfree(h->pool.active); dfree(h->pool.adjd);
  dfree(h->in_batch); dfree(h->bidx); dfree(h->mark); dfree(h->cnt); dfree(h->off); dfree(h->dirty); dfree(h->queue); dfree(h->qflag);
  dfree(h->rev_off); dfree(h->rev_src); dfree(h->rev_sorted); dfree(h->scan_tmp); dfree(h->med_tmp);
  dfree(h->rev.pairs); dfree(h->rev.bh); dfree(h->rev.bo);
  dfree(h->rev.pairs2); dfree(h->rev.bh2); dfree(h->rev.bo2);
  dfree(h->ds);
  if (h->hs) (void)hipHostFree(h->hs);
  h->hs = nullptr;
  dfree(h->rchunk); dfree(h->coff); dfree(h->cdesc);
  if (h->ev_total) (void)hipEventDestroy(h->ev_total);
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  if (h->ev_join) (void)hipEventDestroy(h->ev_join);
  if (h->side) (void)hipStreamDestroy(h->side);
  h->ev_fork = h->ev_join = nullptr;
  h->side = nullptr;
  h->ev_total = nullptr;
  dfree(h->b_ids); dfree(h->v_ids); dfree(h->v_n); dfree(h->c_ids); dfree(h->rcount); dfree(h->rofs);
  dfree(h->v_d); dfree(h->c_d); dfree(h->b_vecs);
  dfree(h->rec_t); dfree(h->rec_s); dfree(h->rec_d); dfree(h->gsrc); dfree(h->gd);
  dfree(h->grp.pt); dfree(h->grp.ps); dfree(h->grp.pd); dfree(h->grp.mat); dfree(h->grp.mato); dfree(h->grp.tmp);
  dfree(h->grp.dpad); dfree(h->grp.dcnt);
  dfree(h->q_vecs); dfree(h->q_ids); dfree(h->q_d);
  dfree(h->vis);
  for (auto &t : h->pending) {
    if (std::get<1>(t)) (void)hipEventDestroy(std::get<1>(t));
    if (std::get<2>(t)) (void)hipEventDestroy(std::get<2>(t));
  }
  for (auto e : h->spare_events) (void)hipEventDestroy(e);
}

}  // namespace

extern "C" {

void grand_default_params(grand_params *p) {
  if (!p) return;
  memset(p, 0, sizeof *p);
  p->struct_size = sizeof(grand_params);
  p->algo = GRAND_VAMANA;
  p->dtype = GRAND_F32;
  p->metric = GRAND_L2;
  p->dim = 128;
  p->capacity = 1u << 20;
  p->R = 64;
  p->L_build = 128;
  p->P = 64;
  p->c = 2;
  p->k_repair = 50;
  p->max_iters = 0;
  p->alpha = 1.2f;
  p->prune_rule = GRAND_ALPHA_ON_DIST;
  p->cas_mode = GRAND_CAS_GROUPED;
  p->rev_mode = GRAND_REV_BATCH;
  p->max_batch = 10000;
  p->device = 0;
  p->stream = nullptr;
}

grand_status grand_create(const grand_params *p, grand_index **out) {
  if (!out) return GRAND_E_ARG;
  *out = nullptr;
  std::string why;
  if (!params_ok(p, why)) {
    fprintf(stderr, "grand_create: %s\n", why.c_str());
    return GRAND_E_ARG;
  }
  grand_index *h = new grand_index();
  h->p = *p;
  if (hipSetDevice(p->device) != hipSuccess) {
    (void)hipGetLastError();
    delete h;
    return GRAND_E_DEVICE;
  }
  h->stream = (hipStream_t)p->stream;
  {
    hipError_t e = hipSuccess;
    h->static_scratch = scratch_of(p->device, &e);
    if (!h->static_scratch) {
      (void)hipGetLastError();
      fprintf(stderr, "grand_create: no address for the static search scratch: %s\n", hipGetErrorString(e));
      delete h;
      return GRAND_E_DEVICE;
    }
  }
  h->kind = p->dtype == GRAND_U8 ? kU8L2 : (p->metric == GRAND_IP ? kF32IP : kF32L2);
  h->esize = p->dtype == GRAND_U8 ? 1 : 4;
  h->mips = p->metric == GRAND_MIPS;
  h->sdim = p->dim + (h->mips ? 1 : 0);
  h->row_bytes = (size_t)p->dim * h->esize;
  h->stride = ((size_t)h->sdim * h->esize + 15) / 16 * 16;
  h->nch = (int)(h->stride / 16);
  h->vc = vec_class(h->nch);
  if (h->vc < 0) {
    fprintf(stderr, "grand_create: vectors of %zu bytes are too long (max 4096)\n", h->row_bytes);
    delete h;
    return GRAND_E_ARG;
  }
  h->iters = p->max_iters ? p->max_iters : 2 * p->L_build;
  const double a = (double)p->alpha;
  h->coef = p->prune_rule == GRAND_ALPHA_ON_L2 ? a * a : a;
  h->c_stride = std::max(p->R, p->k_repair);
  const size_t cap = p->capacity;
  h->rev.plan = rev_plan(p->capacity, p->R);
  PoolView &P = h->pool;
  P.stride = h->stride;
  P.nch = h->nch;
  P.R = p->R;
  P.cap = p->capacity;
  P.adjd = nullptr;
  const bool stored = p->algo == GRAND_VAMANA && adj_dists_apply(h->kind, p->R, h->nch, p->P);
  bool bad = dalloc(&P.vecs, cap * h->stride) || dalloc(&P.adj, cap * p->R) || dalloc(&P.deg, cap) ||
             (stored && dalloc(&P.adjd, cap * p->R)) ||
             dalloc(&P.active, cap) || dalloc(&h->in_batch, cap) || dalloc(&h->bidx, cap) ||
             dalloc(&h->mark, cap) || dalloc(&h->cnt, cap + 1) || dalloc(&h->off, cap + 1) ||
             dalloc(&h->dirty, cap) || dalloc(&h->queue, cap) || dalloc(&h->qflag, cap) || dalloc(&h->rev_off, cap + 1) || dalloc(&h->rev_src, cap * p->R) ||
             dalloc(&h->scan_tmp, scan_tmp_words(std::max(std::max(cap + 1, rev_bucket_words(h->rev.plan)),
                                                          rev_fine_words(h->rev.plan)))) ||
             (h->rev.plan.ok && (dalloc(&h->rev.pairs, rev_pair_words(h->rev.plan, p->capacity, p->R)) ||
                                 dalloc(&h->rev.bh, rev_bucket_words(h->rev.plan)) ||
                                 dalloc(&h->rev.bo, rev_bucket_words(h->rev.plan)))) ||
             (h->rev.plan.two && (dalloc(&h->rev.pairs2, rev_pair_words(h->rev.plan, p->capacity, p->R)) ||
                                  dalloc(&h->rev.bh2, rev_fine_words(h->rev.plan)) ||
                                  dalloc(&h->rev.bo2, rev_fine_words(h->rev.plan)))) ||
             (group_two_level(p->capacity) && (dalloc(&h->grp.dpad, group_pad_words(p->capacity)) ||
                                               dalloc(&h->grp.dcnt, group_buckets(p->capacity)))) ||
             dalloc(&h->ds, 1) ||
             hipMalloc(&h->med_tmp, medoid_tmp_bytes(p->capacity, p->dim + 1)) != hipSuccess ||
             hipHostMalloc((void **)&h->hs, sizeof(DevScalars), hipHostMallocDefault) != hipSuccess ||
             hipEventCreateWithFlags(&h->ev_total, hipEventDisableTiming) != hipSuccess ||
             hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming) != hipSuccess ||
             hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming) != hipSuccess ||
             hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking) != hipSuccess;
  if (bad) {
    (void)hipGetLastError();
    release(h);
    delete h;
    return GRAND_E_OOM;
  }
  hipStream_t s = h->stream;
  bool err = hipMemsetAsync(P.vecs, 0, cap * h->stride, s) != hipSuccess ||
             launch_fill_u32(P.adj, GRAND_INVALID, cap * p->R, s) != hipSuccess ||
             hipMemsetAsync(P.deg, 0, cap * 4, s) != hipSuccess || hipMemsetAsync(P.active, 0, cap, s) != hipSuccess ||
             hipMemsetAsync(h->in_batch, 0, cap, s) != hipSuccess || hipMemsetAsync(h->mark, 0, cap * 4, s) != hipSuccess ||
             hipMemsetAsync(h->cnt, 0, (cap + 1) * 4, s) != hipSuccess ||
             hipMemsetAsync(h->ds, 0, sizeof(DevScalars), s) != hipSuccess;
  memset(h->hs, 0, sizeof(DevScalars));
  h->hs->medoid = GRAND_INVALID;
  if (!err) err = hipMemcpyAsync(h->ds, h->hs, sizeof(DevScalars), hipMemcpyHostToDevice, s) != hipSuccess;
  if (!err) err = hipStreamSynchronize(s) != hipSuccess;
  if (err) {
    (void)hipGetLastError();
    release(h);
    delete h;
    return GRAND_E_DEVICE;
  }
  h->st.struct_size = sizeof(grand_stats_t);
  grand_status bs = ensure_batch(h, std::max<uint32_t>(p->max_batch, 1));
  if (bs == GRAND_OK) bs = ensure_records(h, (size_t)std::max<uint32_t>(p->max_batch, 1) * p->R);
  if (bs != GRAND_OK) {
    release(h);
    delete h;
    return bs;
  }
  *out = h;
  return GRAND_OK;
}

grand_status grand_destroy(grand_index *h) {
  if (!h) return GRAND_OK;
  if (!h->poisoned) (void)hipStreamSynchronize(h->stream);
  release(h);
  delete h;
  return GRAND_OK;
}

grand_status grand_set_stream(grand_index *h, void *stream) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  HCHK(h, hipStreamSynchronize(h->stream));
  h->stream = (hipStream_t)stream;
  return GRAND_OK;
}

grand_status grand_insert_batch(grand_index *h, const void *vecs, const uint32_t *ids, uint32_t n) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (n == 0) return GRAND_OK;
  if (!vecs || !ids) return fail(h, GRAND_E_ARG, "null argument");
  if (h->n_active + n > h->p.capacity) return fail(h, GRAND_E_CAPACITY, "batch exceeds the free capacity");
  HCHK(h, hipSetDevice(h->p.device));
  if ((s = ensure_batch(h, n)) != GRAND_OK) return s;
  {
    Phase ph(h, GRAND_PH_VALIDATE);
    HCHK(h, hipMemcpyAsync(h->b_ids, ids, (size_t)n * 4, hipMemcpyDefault, h->stream));
    if ((s = stage_rows(h, h->b_vecs, vecs, n)) != GRAND_OK) return s;
    if ((s = clear_errors(h)) != GRAND_OK) return s;
    h->epoch++;
    HCHK(h, launch_validate_ids(h->b_ids, n, h->p.capacity, h->pool.active, h->mark, h->epoch, 0, h->ds, h->stream));
    if (h->p.dtype == GRAND_F32)
      HCHK(h, launch_check_finite(h->b_vecs, n, h->stride, h->p.dim, h->ds, h->stream));
    if (h->mips) HCHK(h, launch_mips_augment(h->b_vecs, n, h->stride, h->p.dim, h->p.mips_norm, h->ds, h->stream));
  }
  if ((s = read_validation(h)) != GRAND_OK) {
    (void)finish(h);
    return s;
  }
  {
    Phase ph(h, GRAND_PH_STAGE);
    HCHK(h, launch_stage(h->pool, h->b_vecs, h->b_ids, n, h->bidx, h->stream));
  }
  const uint64_t n0 = h->n_active;
  h->n_active += n;
  s = h->p.algo == GRAND_CAGRA ? cagra_insert(h, n, n0) : vamana_insert(h, n, n0);
  if (s != GRAND_OK) return s;
  if (n0 == 0 && (s = run_medoid(h, nullptr, 1)) != GRAND_OK) return s;
  h->st.inserted += n;
  return finish(h);
}

// Device buffers of one graph construction; freed when the call ends.
struct BuildBufs {
  uint32_t *init = nullptr, *lid = nullptr, *nid = nullptr, *ns = nullptr, *os = nullptr, *cand = nullptr,
           *cnb = nullptr, *pcnt = nullptr, *poff = nullptr, *prn = nullptr;
  float *ld = nullptr, *nd = nullptr;
  ~BuildBufs() {
    dfree(init); dfree(lid); dfree(nid); dfree(ns); dfree(os); dfree(cand); dfree(cnb); dfree(pcnt);
    dfree(poff); dfree(prn); dfree(ld); dfree(nd);
  }
};

grand_status grand_build_cagra(grand_index *h, const void *vecs, const uint32_t *ids, uint32_t n,
                               const uint32_t *init, uint32_t knn, uint32_t iters, uint32_t sample) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (!vecs || !ids || !init) return fail(h, GRAND_E_ARG, "null argument");
  if (h->p.algo != GRAND_CAGRA) return fail(h, GRAND_E_ARG, "graph construction is for the CAGRA variant");
  if (h->n_active != 0) return fail(h, GRAND_E_ARG, "graph construction needs an empty index");
  const uint32_t R = h->p.R, K = knn, S = sample;
  if (K < R || K > 128 || n <= K || S == 0 || S > 32)
    return fail(h, GRAND_E_ARG, "need R <= knn <= 128, knn < n and 1 <= sample <= 32");
  if (n > h->p.capacity) return fail(h, GRAND_E_CAPACITY, "more points than the capacity");
  const uint64_t max_prop = 12ull * S * S - 2ull * S;  // proposals of one node in one round
  if ((uint64_t)n * max_prop >= (1ull << 32)) return fail(h, GRAND_E_CAPACITY, "sample too large for n points");
  HCHK(h, hipSetDevice(h->p.device));
  if ((s = ensure_batch(h, n)) != GRAND_OK) return s;
  BuildBufs b;
  const size_t nk = (size_t)n * K, nsz = (size_t)n * S;
  if (dalloc(&b.init, nk) || dalloc(&b.lid, nk) || dalloc(&b.nid, nk) || dalloc(&b.ld, nk) || dalloc(&b.nd, nk) ||
      dalloc(&b.ns, nsz) || dalloc(&b.os, nsz) || dalloc(&b.cand, 4 * nsz) || dalloc(&b.cnb, n) ||
      dalloc(&b.pcnt, n) || dalloc(&b.poff, (size_t)n + 1) || dalloc(&b.prn, (size_t)n * R)) {
    (void)hipGetLastError();
    return fail(h, GRAND_E_OOM, "device allocation of the construction buffers failed");
  }
  // the record buffers the index holds for its batches, grown to the sample
  // and reverse-edge records if needed; the proposals of a round are written
  // in chunks of nodes that fit them
  const size_t need = std::max<size_t>(std::max<size_t>((size_t)n * 2 * S, (size_t)n * R), max_prop);
  if ((s = ensure_records(h, need)) != GRAND_OK) return s;
  BuildArgs a{};
  a.pool = h->pool;
  a.ids = h->b_ids;
  a.n = n;
  a.K = K;
  a.S = S;
  a.R = R;
  a.init = b.init;
  a.lid = b.lid;
  a.ld = b.ld;
  a.nid = b.nid;
  a.nd = b.nd;
  a.ns = b.ns;
  a.os = b.os;
  a.cand = b.cand;
  a.cnb = b.cnb;
  a.pcnt = b.pcnt;
  a.poff = b.poff;
  a.rec_t = h->rec_t;
  a.rec_s = h->rec_s;
  a.rec_d = h->rec_d;
  a.goff = h->off;
  a.gsrc = h->gsrc;
  a.gd = h->gd;
  a.dirty = h->dirty;
  a.n_dirty = &h->ds->n_dirty;
  a.prn = b.prn;
  a.ds = h->ds;
  {
    Phase ph(h, GRAND_PH_VALIDATE);
    HCHK(h, hipMemcpyAsync(h->b_ids, ids, (size_t)n * 4, hipMemcpyDefault, h->stream));
    HCHK(h, hipMemcpyAsync(b.init, init, nk * 4, hipMemcpyDefault, h->stream));
    if ((s = stage_rows(h, h->b_vecs, vecs, n)) != GRAND_OK) return s;
    if ((s = clear_errors(h)) != GRAND_OK) return s;
    h->epoch++;
    HCHK(h, launch_validate_ids(h->b_ids, n, h->p.capacity, h->pool.active, h->mark, h->epoch, 0, h->ds, h->stream));
    if (h->p.dtype == GRAND_F32)
      HCHK(h, launch_check_finite(h->b_vecs, n, h->stride, h->p.dim, h->ds, h->stream));
    HCHK(h, launch_build_check(a, h->stream));
  }
  if ((s = read_validation(h)) != GRAND_OK) {
    (void)finish(h);
    return s;
  }
  {
    Phase ph(h, GRAND_PH_STAGE);
    HCHK(h, launch_stage(h->pool, h->b_vecs, h->b_ids, n, h->bidx, h->stream));
  }
  h->n_active = n;
  HCHK(h, launch_build_init(h->kind, a, h->stream));
  std::vector<uint32_t> poff((size_t)n + 1);
  for (uint32_t it = 0; it < iters; it++) {
    // samples, recorded at their targets and grouped
    HCHK(h, launch_build_sample(a, h->stream));
    if ((s = run_group(h, (size_t)n * 2 * S)) != GRAND_OK) return s;
    HCHK(h, launch_build_cands(a, h->stream));
    HCHK(h, hipMemcpyAsync(a.nid, a.lid, nk * 4, hipMemcpyDeviceToDevice, h->stream));
    HCHK(h, hipMemcpyAsync(a.nd, a.ld, nk * 4, hipMemcpyDeviceToDevice, h->stream));
    // proposals per node, then written and merged chunk by chunk
    a.v0 = 0;
    a.v1 = n;
    HCHK(h, launch_build_join(h->kind, a, false, h->stream));
    HCHK(h, launch_scan(b.pcnt, b.poff, n, h->scan_tmp, h->stream));
    HCHK(h, hipMemcpyAsync(poff.data(), b.poff, poff.size() * 4, hipMemcpyDeviceToHost, h->stream));
    HCHK(h, hipStreamSynchronize(h->stream));
    uint32_t v0 = 0;
    while (v0 < n) {
      uint32_t v1 = v0 + 1;
      while (v1 < n && (size_t)(poff[v1 + 1] - poff[v0]) <= h->rcap) v1++;
      const size_t nrec = poff[v1] - poff[v0];  // at most rcap: one node proposes at most max_prop
      if (nrec) {
        a.v0 = v0;
        a.v1 = v1;
        HCHK(h, launch_build_join(h->kind, a, true, h->stream));
        if ((s = run_group(h, nrec)) != GRAND_OK) return s;
        HCHK(h, launch_build_merge(a, persistent_grid(v1 - v0 + n / 8), h->stream));
      }
      v0 = v1;
    }
    std::swap(a.lid, a.nid);
    std::swap(a.ld, a.nd);
  }
  // rank-based pruning, then the reverse edges
  HCHK(h, launch_build_rank(a, h->stream));
  if ((s = run_group(h, (size_t)n * R)) != GRAND_OK) return s;
  HCHK(h, launch_build_out(a, h->stream));
  if ((s = run_medoid(h, nullptr, 1)) != GRAND_OK) return s;
  h->st.inserted += n;
  s = finish(h);
  HCHK(h, hipStreamSynchronize(h->stream));  // the construction buffers are freed on return
  return s;
}

grand_status grand_delete_batch(grand_index *h, const uint32_t *ids, uint32_t n) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (n == 0) return GRAND_OK;
  if (!ids) return fail(h, GRAND_E_ARG, "null argument");
  HCHK(h, hipSetDevice(h->p.device));
  if ((s = ensure_batch(h, n)) != GRAND_OK) return s;
  {
    Phase ph(h, GRAND_PH_VALIDATE);
    HCHK(h, hipMemcpyAsync(h->b_ids, ids, (size_t)n * 4, hipMemcpyDefault, h->stream));
    if ((s = clear_errors(h)) != GRAND_OK) return s;
    h->epoch++;
    HCHK(h, launch_validate_ids(h->b_ids, n, h->p.capacity, h->pool.active, h->mark, h->epoch, 1, h->ds, h->stream));
  }
  if ((s = read_validation(h)) != GRAND_OK) {
    (void)finish(h);
    return s;
  }
  HCHK(h, launch_mark_batch(h->b_ids, n, h->in_batch, h->bidx, 1, h->stream));
  s = h->p.algo == GRAND_CAGRA ? cagra_delete(h, n) : vamana_delete(h, n);
  if (s != GRAND_OK) return s;
  {
    Phase ph(h, GRAND_PH_CLEAR);
    HCHK(h, launch_clear_rows(h->pool, h->b_ids, n, h->stream));
  }
  h->n_active -= n;
  // whether the medoid was deleted reaches the host with the call's final
  // copy of the device scalars; only then are the medoid kernels launched
  HCHK(h, launch_medoid_need(h->ds, h->in_batch, 0, h->stream));
  HCHK(h, launch_mark_batch(h->b_ids, n, h->in_batch, nullptr, 0, h->stream));
  h->st.deleted += n;
  if ((s = finish(h)) != GRAND_OK) return s;
  if (!h->hs->need_medoid) return GRAND_OK;
  {
    Phase ph(h, GRAND_PH_MEDOID);
    HCHK(h, launch_medoid(h->pool, h->kind, h->sdim, h->n_active, h->med_tmp, h->ds, h->stream));
  }
  return finish(h);
}

grand_status grand_search(grand_index *h, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                          uint32_t *out_ids, float *out_dists) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (k == 0 || beam == 0 || k > beam || beam > 256) return fail(h, GRAND_E_ARG, "need 1 <= k <= beam <= 256");
  if (nq == 0) return GRAND_OK;
  if (!queries || !out_ids || !out_dists) return fail(h, GRAND_E_ARG, "null argument");
  HCHK(h, hipSetDevice(h->p.device));
  if ((s = ensure_query(h, nq, k)) != GRAND_OK) return s;
  if (h->p.dtype == GRAND_F32) {
    Phase ph(h, GRAND_PH_VALIDATE);
    if ((s = stage_rows(h, h->q_vecs, queries, nq)) != GRAND_OK) return s;
    if ((s = clear_errors(h)) != GRAND_OK) return s;
    HCHK(h, launch_check_finite(h->q_vecs, nq, h->stride, h->p.dim, h->ds, h->stream));
    if ((s = read_validation(h)) != GRAND_OK) {
      (void)finish(h);
      return s;
    }
  } else {
    if ((s = stage_rows(h, h->q_vecs, queries, nq)) != GRAND_OK) return s;
  }
  if (h->n_active == 0) {
    HCHK(h, launch_fill_u32(h->q_ids, GRAND_INVALID, (size_t)nq * k, h->stream));
    HCHK(h, launch_fill_u32(reinterpret_cast<uint32_t *>(h->q_d), 0x7F800000u, (size_t)nq * k, h->stream));
  } else {
    Phase ph(h, GRAND_PH_SEARCH_QUERY);
    SearchArgs a{};
    a.pool = h->pool;
    a.qbase = h->q_vecs;
    a.nq = nq;
    a.start = h->medoid;
    a.ell = beam;
    a.max_iters = 2 * beam;
    a.which = 2;
    a.c_ids = h->q_ids;
    a.c_d = h->q_d;
    a.c_out = k;
    a.ds = h->ds;
    if (grand_status s_ = prep_counting(h, a)) return s_;
    HCHK(h, launch_search(h->kind, h->vc, a, h->stream));
  }
  HCHK(h, hipMemcpyAsync(out_ids, h->q_ids, (size_t)nq * k * 4, hipMemcpyDefault, h->stream));
  HCHK(h, hipMemcpyAsync(out_dists, h->q_d, (size_t)nq * k * 4, hipMemcpyDefault, h->stream));
  h->st.queried += nq;
  return finish(h);
}

grand_status grand_search_static(grand_index *h, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                                 uint32_t *out_ids, float *out_dists) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (k == 0 || beam == 0 || k > beam || beam > 256) return fail(h, GRAND_E_ARG, "need 1 <= k <= beam <= 256");
  if (nq == 0) return GRAND_OK;
  if (!queries || !out_ids || !out_dists) return fail(h, GRAND_E_ARG, "null argument");
  // layout in `scratch`: query rows (nq x stride), ids (nq x k), distances
  // (nq x k), each region 256-byte aligned
  const size_t qb = ((size_t)nq * h->stride + 255) / 256 * 256;
  const size_t rb = ((size_t)nq * k * 4 + 255) / 256 * 256;
  if (qb + 2 * rb > kStaticScratchBytes)
    return fail(h, GRAND_E_CAPACITY, "queries and results exceed the static search scratch");
  HCHK(h, hipSetDevice(h->p.device));
  uint8_t *q_vecs = h->static_scratch;
  uint32_t *q_ids = reinterpret_cast<uint32_t *>(h->static_scratch + qb);
  float *q_d = reinterpret_cast<float *>(h->static_scratch + qb + rb);
  // the array keeps the previous call's contents: zero the rows' padding
  if (h->stride != h->row_bytes) HCHK(h, launch_fill_u32(reinterpret_cast<uint32_t *>(q_vecs), 0u, qb / 4, h->stream));
  if ((s = stage_rows(h, q_vecs, queries, nq)) != GRAND_OK) return s;
  if (h->p.dtype == GRAND_F32) {
    if ((s = clear_errors(h)) != GRAND_OK) return s;
    HCHK(h, launch_check_finite(q_vecs, nq, h->stride, h->p.dim, h->ds, h->stream));
    if ((s = read_validation(h)) != GRAND_OK) {
      (void)finish(h);
      return s;
    }
  }
  if (h->n_active == 0) {
    HCHK(h, launch_fill_u32(q_ids, GRAND_INVALID, (size_t)nq * k, h->stream));
    HCHK(h, launch_fill_u32(reinterpret_cast<uint32_t *>(q_d), 0x7F800000u, (size_t)nq * k, h->stream));
  } else {
    SearchArgs a{};
    a.pool = h->pool;
    a.qbase = q_vecs;
    a.nq = nq;
    a.start = h->medoid;
    a.ell = beam;
    a.max_iters = 2 * beam;
    a.which = 2;
    a.c_ids = q_ids;
    a.c_d = q_d;
    a.c_out = k;
    a.ds = h->ds;
    HCHK(h, launch_search(h->kind, h->vc, a, h->stream));
  }
  HCHK(h, hipMemcpyAsync(out_ids, q_ids, (size_t)nq * k * 4, hipMemcpyDefault, h->stream));
  HCHK(h, hipMemcpyAsync(out_dists, q_d, (size_t)nq * k * 4, hipMemcpyDefault, h->stream));
  h->st.queried += nq;
  return finish(h);
}

grand_status grand_count_in_edges(grand_index *h, const uint32_t *ids, uint32_t n, int method, uint32_t *out_counts,
                                  float *ms) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (ms) *ms = 0.0f;
  if (n == 0) return GRAND_OK;
  if (!ids || !out_counts) return fail(h, GRAND_E_ARG, "null argument");
  if (method != GRAND_INDEG_SCAN && method != GRAND_INDEG_REV_BATCH && method != GRAND_INDEG_REV_FULL)
    return fail(h, GRAND_E_ARG, "unknown method");
  if (method == GRAND_INDEG_SCAN && n > 65535) return fail(h, GRAND_E_ARG, "the scan method takes at most 65535 ids");
  HCHK(h, hipSetDevice(h->p.device));
  if ((s = ensure_batch(h, n)) != GRAND_OK) return s;
  HCHK(h, hipMemcpyAsync(h->b_ids, ids, (size_t)n * 4, hipMemcpyDefault, h->stream));
  if ((s = clear_errors(h)) != GRAND_OK) return s;
  h->epoch++;
  HCHK(h, launch_validate_ids(h->b_ids, n, h->p.capacity, h->pool.active, h->mark, h->epoch, 1, h->ds, h->stream));
  if ((s = read_validation(h)) != GRAND_OK) {
    (void)finish(h);
    return s;
  }
  HCHK(h, launch_mark_batch(h->b_ids, n, h->in_batch, h->bidx, 1, h->stream));
  hipEvent_t e0 = get_event(h), e1 = get_event(h);
  if (!e0 || !e1) return fail(h, GRAND_E_DEVICE, "event creation failed");
  HCHK(h, hipEventRecord(e0, h->stream));
  if (method == GRAND_INDEG_SCAN) {
    HCHK(h, launch_scan_in_edges(h->pool, h->b_ids, n, h->rcount, h->stream));
  } else {
    const int by_batch = method == GRAND_INDEG_REV_BATCH;
    if ((s = run_reverse(h, by_batch, by_batch ? n : h->p.capacity)) != GRAND_OK) return s;
    HCHK(h, launch_row_lengths(h->rev_off, by_batch ? nullptr : h->b_ids, n, h->rcount, h->stream));
  }
  HCHK(h, hipEventRecord(e1, h->stream));
  HCHK(h, launch_mark_batch(h->b_ids, n, h->in_batch, nullptr, 0, h->stream));
  HCHK(h, hipMemcpyAsync(out_counts, h->rcount, (size_t)n * 4, hipMemcpyDefault, h->stream));
  if ((s = finish(h)) != GRAND_OK) return s;
  float t = 0.0f;
  HCHK(h, hipEventElapsedTime(&t, e0, e1));
  h->spare_events.push_back(e0);
  h->spare_events.push_back(e1);
  if (ms) *ms = t;
  return GRAND_OK;
}

// ---------------------------------------------------------------- readers
struct grand_reader {
  grand_index *h = nullptr;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  uint8_t *q_vecs = nullptr;
  uint32_t *q_ids = nullptr;
  float *q_d = nullptr;
  uint32_t qcap = 0, qk = 0;
  DevScalars *ds = nullptr;  // the reader's own error flags and counters
  DevScalars *hs = nullptr;  // pinned host mirror
  std::string err;
};

namespace {
void reader_release(grand_reader *r) {
  dfree(r->q_vecs); dfree(r->q_ids); dfree(r->q_d); dfree(r->ds);
  if (r->hs) (void)hipHostFree(r->hs);
  if (r->own_stream && r->stream) (void)hipStreamDestroy(r->stream);
}
grand_status rfail(grand_reader *r, grand_status code, const std::string &msg) {
  r->err = msg;
  return code;
}
#define RCHK(r, x)                                                                     \
  do {                                                                                 \
    hipError_t e_ = (x);                                                               \
    if (e_ != hipSuccess) return rfail((r), GRAND_E_DEVICE, std::string(#x ": ") + hipGetErrorString(e_)); \
  } while (0)
}  // namespace

grand_status grand_reader_create(grand_index *h, void *stream, grand_reader **out) {
  if (!out) return GRAND_E_ARG;
  *out = nullptr;
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  HCHK(h, hipSetDevice(h->p.device));
  grand_reader *r = new grand_reader();
  r->h = h;
  bool bad = false;
  if (stream) {
    r->stream = (hipStream_t)stream;
  } else {
    bad = hipStreamCreateWithFlags(&r->stream, hipStreamNonBlocking) != hipSuccess;  // default priority
    r->own_stream = !bad;
  }
  bad = bad || dalloc(&r->ds, 1) || hipHostMalloc((void **)&r->hs, sizeof(DevScalars), hipHostMallocDefault) != hipSuccess;
  if (!bad) bad = hipMemsetAsync(r->ds, 0, sizeof(DevScalars), r->stream) != hipSuccess ||
                  hipStreamSynchronize(r->stream) != hipSuccess;
  if (bad) {
    (void)hipGetLastError();
    reader_release(r);
    delete r;
    return fail(h, GRAND_E_OOM, "reader allocation failed");
  }
  *out = r;
  return GRAND_OK;
}

grand_status grand_reader_destroy(grand_reader *r) {
  if (!r) return GRAND_OK;
  (void)hipSetDevice(r->h->p.device);
  (void)hipStreamSynchronize(r->stream);
  reader_release(r);
  delete r;
  return GRAND_OK;
}

grand_status grand_reader_search(grand_reader *r, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                                 uint32_t *out_ids, float *out_dists) {
  if (!r) return GRAND_E_ARG;
  grand_index *h = r->h;
  r->err.clear();
  if (h->poisoned) return GRAND_E_STATE;
  if (k == 0 || beam == 0 || k > beam || beam > 256) return rfail(r, GRAND_E_ARG, "need 1 <= k <= beam <= 256");
  if (nq == 0) return GRAND_OK;
  if (!queries || !out_ids || !out_dists) return rfail(r, GRAND_E_ARG, "null argument");
  RCHK(r, hipSetDevice(h->p.device));
  if (nq > r->qcap || k > r->qk) {
    RCHK(r, hipStreamSynchronize(r->stream));
    const uint32_t nc = std::max(nq, r->qcap), kc = std::max(k, r->qk);
    dfree(r->q_vecs); dfree(r->q_ids); dfree(r->q_d);
    r->qcap = r->qk = 0;
    if (dalloc(&r->q_vecs, (size_t)nc * h->stride) || dalloc(&r->q_ids, (size_t)nc * kc) ||
        dalloc(&r->q_d, (size_t)nc * kc)) {
      (void)hipGetLastError();
      return rfail(r, GRAND_E_OOM, "device allocation of reader buffers failed");
    }
    RCHK(r, hipMemsetAsync(r->q_vecs, 0, (size_t)nc * h->stride, r->stream));
    r->qcap = nc;
    r->qk = kc;
  }
  RCHK(r, hipMemcpy2DAsync(r->q_vecs, h->stride, queries, h->row_bytes, h->row_bytes, nq, hipMemcpyDefault, r->stream));
  if (h->p.dtype == GRAND_F32) {
    RCHK(r, launch_fill_u32(&r->ds->err_code, 0u, 2, r->stream));
    RCHK(r, launch_check_finite(r->q_vecs, nq, h->stride, h->p.dim, r->ds, r->stream));
    RCHK(r, hipMemcpyAsync(r->hs, r->ds, kScalarBytes, hipMemcpyDeviceToHost, r->stream));
    RCHK(r, hipStreamSynchronize(r->stream));
    if (r->hs->err_code) return rfail(r, GRAND_E_ARG, "a query holds a non-finite element");
  }
  SearchArgs a{};
  a.pool = h->pool;
  a.qbase = r->q_vecs;
  a.nq = nq;
  a.start = GRAND_INVALID;
  a.start_ptr = &h->ds->medoid;  // the index's medoid as the search starts
  a.ell = beam;
  a.max_iters = 2 * beam;
  a.which = 2;
  a.c_ids = r->q_ids;
  a.c_d = r->q_d;
  a.c_out = k;
  a.ds = r->ds;
  RCHK(r, launch_search(h->kind, h->vc, a, r->stream));
  RCHK(r, hipMemcpyAsync(out_ids, r->q_ids, (size_t)nq * k * 4, hipMemcpyDefault, r->stream));
  RCHK(r, hipMemcpyAsync(out_dists, r->q_d, (size_t)nq * k * 4, hipMemcpyDefault, r->stream));
  RCHK(r, hipStreamSynchronize(r->stream));
  return GRAND_OK;
}

const char *grand_reader_last_error(const grand_reader *r) { return r ? r->err.c_str() : "null reader"; }

grand_status grand_export_graph(grand_index *h, uint32_t *adj, uint32_t *deg, uint8_t *active, uint32_t *medoid,
                                uint32_t *rev_offsets, uint32_t *rev_srcs, uint64_t *nnz) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  HCHK(h, hipSetDevice(h->p.device));
  const size_t cap = h->p.capacity;
  if (adj && h->p.algo == GRAND_VAMANA) {
    // Vamana lists are sets: returned with each row ascending (the reverse
    // graph's source array is free scratch between delete batches)
    HCHK(h, launch_sort_adj_rows(h->pool.adj, (uint32_t)cap, h->p.R, h->rev_src, h->stream));
    HCHK(h, hipMemcpyAsync(adj, h->rev_src, cap * h->p.R * 4, hipMemcpyDefault, h->stream));
  } else if (adj) {
    HCHK(h, hipMemcpyAsync(adj, h->pool.adj, cap * h->p.R * 4, hipMemcpyDefault, h->stream));
  }
  if (deg) HCHK(h, hipMemcpyAsync(deg, h->pool.deg, cap * 4, hipMemcpyDefault, h->stream));
  if (active) HCHK(h, hipMemcpyAsync(active, h->pool.active, cap, hipMemcpyDefault, h->stream));
  if (rev_offsets || rev_srcs || nnz) {
      if ((s = run_reverse(h, 0, 0)) != GRAND_OK) return s;
    uint32_t e32 = 0;
    HCHK(h, hipMemcpyAsync(&h->hs->err_id, h->rev_off + cap, sizeof(uint32_t), hipMemcpyDeviceToHost, h->stream));
    HCHK(h, hipStreamSynchronize(h->stream));
    e32 = h->hs->err_id;
    const size_t e = e32;
    if (rev_offsets) HCHK(h, hipMemcpyAsync(rev_offsets, h->rev_off, (cap + 1) * 4, hipMemcpyDefault, h->stream));
    if (rev_srcs && e) {
      if (h->rev_sorted_cap < e) {
        HCHK(h, hipStreamSynchronize(h->stream));
        dfree(h->rev_sorted);
        h->rev_sorted_cap = 0;
        if (dalloc(&h->rev_sorted, e)) {
          (void)hipGetLastError();
          return fail(h, GRAND_E_OOM, "device allocation for the sorted reverse graph failed");
        }
        h->rev_sorted_cap = e;
      }
      HCHK(h, launch_sort_rows(h->rev_off, (uint32_t)cap, h->rev_src, h->rev_sorted, h->stream));
      HCHK(h, hipMemcpyAsync(rev_srcs, h->rev_sorted, e * 4, hipMemcpyDefault, h->stream));
    }
    if (nnz) *nnz = e;
  }
  if ((s = finish(h)) != GRAND_OK) return s;
  if (medoid) *medoid = h->medoid;
  return GRAND_OK;
}

__global__ void k_import_check(PoolView P, DevScalars *ds) {
  const size_t total = (size_t)P.cap * P.R;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total; i += (size_t)gridDim.x * blockDim.x) {
    const uint32_t v = P.adj[i];
    const uint32_t u = (uint32_t)(i / P.R);
    const bool bad = v != GRAND_INVALID && (v >= P.cap || v == u || !P.active[u] || !P.active[v]);
    if (bad && atomicCAS(&ds->err_code, 0u, (uint32_t)kErrState) == 0u) ds->err_id = u;
  }
}

__global__ void k_count_active(const uint8_t *active, uint32_t cap, DevScalars *ds) {
  unsigned long long c = 0;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < cap; i += gridDim.x * blockDim.x) c += active[i] ? 1 : 0;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) c += __shfl_xor(c, o, 64);
  if ((threadIdx.x & 63) == 0 && c) atomicAdd(&ds->n_count, c);
}

// Installs medoid m if it is an active id, else INVALID.
__global__ void k_set_medoid(DevScalars *ds, const uint8_t *active, uint32_t cap, uint32_t m) {
  ds->medoid = (m < cap && active[m]) ? m : GRAND_INVALID;
}

grand_status grand_import_graph(grand_index *h, const void *vecs, const uint32_t *adj, const uint32_t *deg,
                                const uint8_t *active, uint32_t medoid) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (!vecs || !adj || !deg || !active) return fail(h, GRAND_E_ARG, "null argument");
  HCHK(h, hipSetDevice(h->p.device));
  const size_t cap = h->p.capacity;
  HCHK(h, hipMemcpy2DAsync(h->pool.vecs, h->stride, vecs, h->row_bytes, h->row_bytes, cap, hipMemcpyDefault,
                           h->stream));
  HCHK(h, hipMemcpyAsync(h->pool.adj, adj, cap * h->p.R * 4, hipMemcpyDefault, h->stream));
  HCHK(h, hipMemcpyAsync(h->pool.deg, deg, cap * 4, hipMemcpyDefault, h->stream));
  HCHK(h, hipMemcpyAsync(h->pool.active, active, cap, hipMemcpyDefault, h->stream));
  if ((s = clear_errors(h)) != GRAND_OK) return s;
  if (h->mips) HCHK(h, launch_mips_augment(h->pool.vecs, cap, h->stride, h->p.dim, h->p.mips_norm, h->ds, h->stream));
  HCHK(h, launch_adj_dists(h->pool, h->stream));
  HCHK(h, hipMemsetAsync(&h->ds->n_count, 0, sizeof(unsigned long long), h->stream));
  hipLaunchKernelGGL(k_import_check, dim3(4096), dim3(256), 0, h->stream, h->pool, h->ds);
  hipLaunchKernelGGL(k_count_active, dim3(1024), dim3(256), 0, h->stream, h->pool.active, h->p.capacity, h->ds);
  hipLaunchKernelGGL(k_set_medoid, dim3(1), dim3(1), 0, h->stream, h->ds, h->pool.active, h->p.capacity, medoid);
  HCHK(h, hipGetLastError());
  if ((s = finish(h)) != GRAND_OK) return s;
  h->n_active = h->hs->n_count;
  if (h->hs->err_code) {
    // malformed lists: leave an empty index rather than an inconsistent one
    char buf[128];
    if (h->hs->err_code == kErrNorm)
      snprintf(buf, sizeof buf, "row %u has a norm above mips_norm", h->hs->err_id);
    else
      snprintf(buf, sizeof buf, "list of node %u holds an invalid, inactive or self edge", h->hs->err_id);
    HCHK(h, launch_fill_u32(h->pool.adj, GRAND_INVALID, cap * h->p.R, h->stream));
    HCHK(h, hipMemsetAsync(h->pool.deg, 0, cap * 4, h->stream));
    HCHK(h, hipMemsetAsync(h->pool.active, 0, cap, h->stream));
    hipLaunchKernelGGL(k_set_medoid, dim3(1), dim3(1), 0, h->stream, h->ds, h->pool.active, h->p.capacity,
                       GRAND_INVALID);
    if ((s = finish(h)) != GRAND_OK) return s;
    h->n_active = 0;
    return fail(h, GRAND_E_ARG, buf);
  }
  if (h->n_active > 0 && h->medoid == GRAND_INVALID) {
    // no usable medoid was given: install one (as after a bootstrap)
    if ((s = run_medoid(h, nullptr, 1)) != GRAND_OK) return s;
    if ((s = finish(h)) != GRAND_OK) return s;
  }
  return GRAND_OK;
}

grand_status grand_set_timing(grand_index *h, int enable) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  h->timing = enable != 0;
  h->st.timing_enabled = h->timing ? 1 : 0;
  return GRAND_OK;
}

grand_status grand_set_counting(grand_index *h, int enable) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  HCHK(h, hipStreamSynchronize(h->stream));
  h->counting = enable != 0;
  if (!h->counting) {
    dfree(h->vis);
    h->vis_cap = 0;
  }
  return GRAND_OK;
}

grand_status grand_stats(grand_index *h, void *out_v, size_t size) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if (!out_v || size < sizeof(grand_stats_t)) return fail(h, GRAND_E_ARG, "stats buffer smaller than grand_stats_t");
  grand_stats_t *out = static_cast<grand_stats_t *>(out_v);
  if ((s = finish(h)) != GRAND_OK) return s;
  HCHK(h, hipMemcpyAsync(h->hs->stat, h->ds->stat, sizeof(h->hs->stat), hipMemcpyDeviceToHost, h->stream));
  HCHK(h, hipStreamSynchronize(h->stream));
  unsigned long long c[kStatCount] = {};
  for (int slot = 0; slot < kStatSlots; slot++)
    for (int k = 0; k < kStatCount; k++) c[k] += h->hs->stat[(size_t)slot * kStatWords + k];
  grand_stats_t r = h->st;
  for (int i = 0; i < 3; i++) {
    r.search_hops[i] = c[kStHops + i];
    r.search_evals[i] = c[kStEvals + i];
  }
  r.fwd_evals = c[kStFwdEvals];
  r.fwd_prunes = c[kStFwdPrunes];
  r.rebuild_evals = c[kStRbEvals];
  r.rebuild_prunes = c[kStRbPrunes];
  r.dirty = c[kStDirty];
  r.rebuild_records = c[kStRbRecs];
  r.records = c[kStRecords];
  r.rev_edges = c[kStRevEdges];
  r.repair_evals = c[kStRepEvals];
  r.rebuild_rows = c[kStRbCand];
  r.repair_rows = c[kStRepRows];
  r.repair_records = c[kStRepRecs];
  for (int i = 0; i < 3; i++) {
    r.search_distinct[i] = c[kStDistinct + i];
    r.search_capped[i] = c[kStCapped + i];
  }
  r.struct_size = sizeof(grand_stats_t);
  *out = r;
  return GRAND_OK;
}

grand_status grand_reset_stats(grand_index *h) {
  grand_status s = check_usable(h);
  if (s != GRAND_OK) return s;
  if ((s = finish(h)) != GRAND_OK) return s;
  const uint32_t t = h->st.timing_enabled;
  memset(&h->st, 0, sizeof h->st);
  h->st.struct_size = sizeof(grand_stats_t);
  h->st.timing_enabled = t;
  HCHK(h, hipMemsetAsync(h->ds->stat, 0, sizeof(h->ds->stat), h->stream));
  HCHK(h, hipStreamSynchronize(h->stream));
  return GRAND_OK;
}

const char *grand_last_error(const grand_index *h) { return h ? h->err.c_str() : "null handle"; }

}  // extern "C"
