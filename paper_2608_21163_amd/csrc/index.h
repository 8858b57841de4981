// index.h -- internal definitions shared by the host orchestration and the
// kernel translation units of the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/grand.h"

namespace gr {

// Work counters.  Many workgroups finish at the same moment, and device
// atomics on one address are serialised, so every counter is spread over
// kStatSlots slots (slot rows of kStatWords words, 256 bytes apart):
// workgroup b adds into slot b % kStatSlots, and the host sums the slots
// when it reads the counters.
enum StatId {
  kStHops = 0,     // nodes expanded by [insert, delete, query] searches (3)
  kStEvals = 3,    // row gathers of those searches (3)
  kStFwdEvals = 6, // pairwise distances in forward prunes
  kStFwdPrunes,
  kStRbEvals,      // distances in dirty rebuilds (D_u and pairwise)
  kStRbPrunes,     // rebuilds that pruned
  kStDirty,        // dirty nodes rebuilt / CAGRA targets / affected nodes
  kStRbRecs,       // scratch records read by rebuilds
  kStRecords,      // reverse-edge and repair records emitted
  kStRevEdges,
  kStRepEvals,     // distances in delete repair
  kStRbCand,       // vector rows a pruning rebuild needs: |C| + 1
  kStRepRows,      // vector rows a repair needs: neighbours + |C_i|
  kStRepRecs,      // records written by repairs
  kStDistinct,     // distinct distance evaluations of [insert, delete, query] searches (counting runs) (3)
  kStCapped = kStDistinct + 3,  // searches stopped by the expansion cap with candidates left (3)
  kStatCount = kStCapped + 3
};
constexpr int kStatWords = 32;
constexpr int kStatSlots = 256;
static_assert(kStatCount <= kStatWords, "stat slot too small");

// Device-side scalars and the work counters, one struct per index.  The
// scalars come first: the host copies only them after each call.
struct DevScalars {
  uint32_t err_code;                // first validation error (0 = none)
  uint32_t err_id;
  uint32_t n_dirty;                 // number of entries in the dirty / affected list
  uint32_t n_queue;                 // dirty nodes left by the fast rebuild for the general one
  uint32_t medoid;
  uint32_t best_id;
  unsigned long long best_bits;     // medoid search: smallest squared distance (fp32 data: bit pattern;
                                    // uint8 data: low 64 bits of the exact integer key)
  unsigned long long best_hi;       // uint8 medoid search: high 64 bits of the smallest key
  uint32_t need_medoid;             // medoid kernels run only when set
  uint32_t pad_;
  unsigned long long n_count;       // scratch counter (active ids at import)
  unsigned long long stat[kStatSlots * kStatWords];
};
constexpr size_t kScalarBytes = offsetof(DevScalars, stat);

__device__ __forceinline__ void stat_add(DevScalars *ds, int id, unsigned long long v) {
  if (v) atomicAdd(&ds->stat[(size_t)(blockIdx.x % kStatSlots) * kStatWords + id], v);
}

enum { kErrRange = 1, kErrRepeat = 2, kErrState = 3, kErrNonFinite = 4, kErrNorm = 5, kErrInit = 6 };

// Vector-layout classes: lanes per row (LPV) and 16-byte chunks per lane
// (CPL) of the distance machinery, chosen from the padded row length.
enum { kVcA = 0, kVcB = 1, kVcC = 2 };  // <= 8 chunks, <= 32 chunks, <= 256 chunks

// Pool view passed to kernels.
struct PoolView {
  uint8_t *vecs;
  uint32_t *adj;
  uint32_t *deg;
  uint8_t *active;
  float *adjd;     // Dist(u, N_out(u)[s]) beside every list entry, when stored (else null)
  size_t stride;   // bytes per pool row (multiple of 16)
  int nch;         // 16-byte chunks per row
  uint32_t R;
  uint32_t cap;
};

struct SearchArgs {
  PoolView pool;
  const uint8_t *qbase;       // query rows (padded to the pool stride) ...
  const uint32_t *qids;       // ... or pool ids used as queries (if non-null)
  uint32_t nq;
  uint32_t start;
  const uint32_t *start_ptr;  // if non-null, the start id is read here when a search begins
  uint32_t ell;
  uint32_t max_iters;
  int which;                  // 0 insert, 1 delete, 2 query (counter slot)
  // V output: expanded nodes with their distances
  uint32_t *v_ids;
  float *v_d;
  uint32_t *v_n;
  uint32_t v_stride;
  // C output: the first c_out entries of C whose id is not flagged in c_filter
  uint32_t *c_ids;
  float *c_d;
  uint32_t c_out;
  const uint8_t *c_filter;
  int c_by_id;                // write that set in ascending id order instead (c_out <= 64; c_d untouched)
  // counting runs only: an exact visited bitmap of vis_words words per
  // search (cleared by the caller) replaces the lossy hash
  uint32_t *vis;
  uint32_t vis_words;
  DevScalars *ds;
};

struct BootArgs {
  PoolView pool;
  const uint32_t *ids;        // batch ids (already staged in the pool)
  uint32_t n;
  uint32_t want;              // neighbours kept per point
  uint32_t *o_ids;            // n x o_stride, sorted by (distance, id)
  float *o_d;
  uint32_t *o_n;              // count per point (may be null)
  uint32_t o_stride;
};

struct FwdPruneArgs {
  PoolView pool;
  const uint32_t *ids;
  uint32_t n;
  const uint32_t *v_ids;
  const float *v_d;
  const uint32_t *v_n;
  uint32_t v_stride;
  double coef;                // alpha (or alpha^2) in fp64
  uint32_t *rec_t, *rec_s;    // n x R reverse-edge records
  float *rec_d;
  DevScalars *ds;
};

struct RebuildArgs {
  PoolView pool;
  const uint32_t *dirty;      // dirty nodes (count in ds->n_dirty)
  const uint32_t *list;       // nodes this launch rebuilds ...
  const uint32_t *list_n;     // ... and their number (device)
  uint32_t *queue;            // fast rebuild: nodes left for the general kernel ...
  uint32_t *queue_n;          // ... and their number (device)
  uint32_t *qflag;            // per list position: 1 if left for the general kernel
  uint32_t flag_cap;          // entries of qflag (bounds the list length)
  uint32_t *scan_tmp;         // compaction scratch (scan_tmp_words(flag_cap))
  int count_nodes;            // this launch counts dirty nodes and records read
  const uint32_t *goff;       // group offsets by target id (cap + 1)
  const uint32_t *gsrc;
  const float *gd;
  const uint8_t *in_batch;    // delete: ids of the batch (null for insert)
  uint32_t P;
  double coef;
  DevScalars *ds;
};

struct RepairArgs {
  PoolView pool;
  const uint32_t *ids;
  uint32_t n;
  const uint8_t *in_batch;
  const uint32_t *ci;         // n x kr repair candidates, ascending ids, INVALID padded at the end
  uint32_t kr;
  const uint32_t *rev_off;
  const uint32_t *rev_src;
  int rev_by_batch;           // reverse rows indexed by batch position (1) or by id (0)
  uint32_t c;
  const uint32_t *rofs;       // record offsets per deleted node (n + 1)
  const uint32_t *coff;       // work-chunk offsets per deleted node (n + 1)
  const uint4 *cdesc;         // two words per work chunk: {node, id, reverse-row start, in-degree}, {record base of the node, first position, positions, chunk index}
  uint32_t cw;                // positions per work chunk (a multiple of 64)
  size_t rcap;                // record capacity: nothing is written when rofs[n] exceeds it
  uint32_t *rec_t, *rec_s;
  float *rec_d;
  DevScalars *ds;
};

// CAGRA graph construction (k_build.hip); positions 0..n-1 stand for pool
// rows ids[0..n-1].
struct BuildArgs {
  PoolView pool;
  const uint32_t *ids;        // position -> pool id
  uint32_t n, K, S, R;        // points, k-NN degree, sample size, output degree
  const uint32_t *init;       // n x K initial positions
  uint32_t *lid;              // n x K lists, ascending by (Dist, position); top bit: not yet sampled
  float *ld;
  uint32_t *nid;              // the lists the merges of a round write
  float *nd;
  uint32_t *ns, *os;          // n x S new and old samples
  uint32_t *cand, *cnb;       // n x 4S join candidates (Bn, then Bo) and nb | no << 16
  uint32_t *pcnt;             // proposals per node
  const uint32_t *poff;       // their exclusive scan (n + 1)
  uint32_t v0, v1;            // nodes of one join chunk
  int stage_rows;             // join: candidate rows staged in dynamic LDS
  uint32_t *rec_t, *rec_s;    // records (target, source, key)
  float *rec_d;
  const uint32_t *goff, *gsrc;  // grouped records (offsets per target, sources, keys)
  const float *gd;
  const uint32_t *dirty;      // targets with records and their number (device)
  const uint32_t *n_dirty;
  uint32_t *prn;              // n x R pruned lists
  DevScalars *ds;
};
hipError_t launch_build_check(const BuildArgs &a, hipStream_t s);
hipError_t launch_build_init(int kind, const BuildArgs &a, hipStream_t s);
hipError_t launch_build_sample(const BuildArgs &a, hipStream_t s);
hipError_t launch_build_cands(const BuildArgs &a, hipStream_t s);
hipError_t launch_build_join(int kind, const BuildArgs &a, bool write, hipStream_t s);
hipError_t launch_build_merge(const BuildArgs &a, uint32_t grid, hipStream_t s);
hipError_t launch_build_rank(const BuildArgs &a, hipStream_t s);
hipError_t launch_build_out(const BuildArgs &a, hipStream_t s);

struct CagraArgs {
  PoolView pool;
  const uint32_t *list;       // dirty targets (detour) or affected nodes (pickone)
  const uint32_t *goff;       // detour: group offsets by target
  const uint32_t *gsrc;
  const float *gd;
  const uint32_t *bidx;       // batch position of each batch id
  const uint32_t *fwd;        // n x R forward lists of the new nodes (snapshot)
  const uint8_t *in_batch;
  const uint32_t *rev_off;
  const uint32_t *rev_src;
  int rev_by_batch;
  const uint32_t *rec_t, *rec_s;   // racing mode: raw records
  uint32_t nrec;
  DevScalars *ds;
  // pickone: number of list entries (device); with `dedupe` the list may
  // repeat a node and hold nodes of the batch: an entry is taken when its
  // node is outside the batch and its mark is first set to `epoch`
  const uint32_t *list_n;
  int dedupe;
  uint32_t *mark;
  uint32_t epoch;
};

// ---- launchers (defined in the kernel translation units) ----------------
int vec_class(int nch);
hipError_t launch_search(int kind, int vc, const SearchArgs &a, hipStream_t s);
hipError_t launch_bootstrap(int kind, int vc, const BootArgs &a, hipStream_t s);
hipError_t launch_fwd_prune(int kind, int vc, uint32_t max_iters, const FwdPruneArgs &a, hipStream_t s);
hipError_t launch_rebuild(int kind, int vc, uint32_t R, uint32_t P, const RebuildArgs &a, uint32_t grid,
                          hipStream_t s);
hipError_t launch_repair(int kind, int vc, const RepairArgs &a, uint32_t grid, hipStream_t s);
hipError_t launch_repair_plan(const RepairArgs &a, uint32_t *counts, uint32_t *chunks, hipStream_t s);
hipError_t launch_repair_map(const RepairArgs &a, uint4 *cdesc, hipStream_t s);
bool repair_chunked(int kind, const PoolView &p, uint32_t kr, uint32_t c);
uint32_t repair_chunk_width(int kind, const PoolView &p, uint32_t kr, uint32_t c);

hipError_t launch_fill_u32(uint32_t *p, uint32_t v, size_t n, hipStream_t s);
hipError_t launch_fill_u8(uint8_t *p, uint8_t v, size_t n, hipStream_t s);
hipError_t launch_validate_ids(const uint32_t *ids, uint32_t n, uint32_t cap, const uint8_t *active,
                               uint32_t *mark, uint32_t epoch, int want_active, DevScalars *ds, hipStream_t s);
// Augmentation of inner-product rows into L2 rows (Section 5.4): row[dim] =
// fp32(sqrt(M^2 - sum_j row[j]^2)), the sum in fp64 in dimension order;
// rows whose squared norm exceeds M^2 raise kErrNorm.
hipError_t launch_mips_augment(uint8_t *rows, size_t n, size_t stride, uint32_t dim, float M, DevScalars *ds,
                               hipStream_t s);
hipError_t launch_check_finite(const uint8_t *rows, uint32_t n, size_t stride, uint32_t dim, DevScalars *ds,
                               hipStream_t s);
// Stored list distances apply to Vamana uint8 pools whose list writers are
// the forward prune and rebuild kernels that maintain them (R <= 64, R a
// multiple of 4, rows of 64 or 128 bytes, P <= 64, R + P <= 128).
bool adj_dists_apply(int kind, uint32_t R, int nch, uint32_t P);
// Dist(u, v) for every entry of every list (after a bulk import).
hipError_t launch_adj_dists(PoolView p, hipStream_t s);
hipError_t launch_stage(PoolView p, const uint8_t *rows, const uint32_t *ids, uint32_t n, uint32_t *bidx,
                        hipStream_t s);
hipError_t launch_mark_batch(const uint32_t *ids, uint32_t n, uint8_t *in_batch, uint32_t *bidx, uint8_t v,
                             hipStream_t s);
hipError_t launch_clear_rows(PoolView p, const uint32_t *ids, uint32_t n, hipStream_t s);
// Buffers of the two-level grouping (capacities up to 2^24 ids).
struct GroupBufs {
  uint32_t *pt, *ps;  // records moved to their coarse buckets: targets, sources
  float *pd;          // and distances (rcap each)
  uint32_t *mat;      // per (coarse bucket, record tile) counts, group_mat_words
  uint32_t *mato;     // their exclusive scan, group_mat_words
  uint32_t *tmp;      // scan scratch, scan_tmp_words(group_mat_words)
  uint32_t *dpad;     // targets with a record, per coarse bucket, group_pad_words
  uint32_t *dcnt;     // their number per coarse bucket, group_buckets
  size_t rcap;        // records the buffers hold
};
uint32_t group_buckets(uint32_t cap);
bool group_two_level(uint32_t cap);
size_t group_mat_words(uint32_t cap, size_t rcap);
size_t group_pad_words(uint32_t cap);
// Groups the records by target: off[0..cap] group offsets, gsrc/gd the
// grouped sources and distances, dirty[0..n_dirty) the targets with a
// record in ascending order (ds->n_dirty).  gb selects the two-level form
// (no global atomics) when the capacity allows it; else the one-level form
// with `cnt` (all zero before and after).
hipError_t launch_group(const uint32_t *rec_t, const uint32_t *rec_s, const float *rec_d, size_t nrec,
                        uint32_t cap, uint32_t *cnt, uint32_t *off, uint32_t *scan_tmp, uint32_t *gsrc,
                        float *gd, uint32_t *dirty, DevScalars *ds, const GroupBufs *gb, hipStream_t s);
hipError_t launch_scan(const uint32_t *in, uint32_t *out, size_t n, uint32_t *tmp, hipStream_t s);
// out[0..k) = the items[i] with flags[i] != 0, i < *n (n on the device, at
// most cap), in order; *out_n = k.
hipError_t launch_compact_flags(const uint32_t *flags, const uint32_t *items, const uint32_t *n, uint32_t cap,
                                uint32_t *out, uint32_t *out_n, uint32_t *tmp, hipStream_t s);
size_t scan_tmp_words(size_t n);
// Plan of the bucketed full reverse-graph build: targets are split into
// nb buckets of 2^shift ids and sources into ng chunks of ch rows.
struct RevPlan {
  int ok;          // the bucketed build applies (else per-edge global atomics)
  int shift;       // log2 of the bucket width
  int packed;      // (src << shift) | (target & (width - 1)) fits 32 bits
  uint32_t nb, ng, ch;
  // two-level form (ids of at most 20 bits): nb1 coarse buckets of 2^s1
  // targets, each split into nsub sub-buckets of 2^s2 targets; the coarse
  // partition is counted in ng source chunks, the fine one in nc2 chunks of
  // each coarse bucket
  int two, s1, s2;
  uint32_t nb1, nsub, nc2;
  int rshift;      // log2 R when R is a power of two, else -1 (row of an edge index)
};
RevPlan rev_plan(uint32_t cap, uint32_t R);
size_t rev_pair_words(const RevPlan &rp, uint32_t cap, uint32_t R);  // u32 words of each pair buffer
size_t rev_bucket_words(const RevPlan &rp);                          // u32 words of each coarse table
size_t rev_fine_words(const RevPlan &rp);                            // u32 words of each fine table
struct RevBufs {
  RevPlan plan;
  uint32_t *pairs;  // rev_pair_words (one-level pairs, or the coarse partition)
  uint32_t *bh;     // per (bucket, chunk) counts, rev_bucket_words
  uint32_t *bo;     // their exclusive scan, rev_bucket_words
  uint32_t *pairs2; // fine partition (two-level form), rev_pair_words
  uint32_t *bh2;    // per (coarse bucket, sub-bucket, chunk) counts, rev_fine_words
  uint32_t *bo2;    // their exclusive scan
};
// by_batch: rows of the nrows batch positions (ids: the batch's ids; a batch
// id's position is bidx[id] and in_batch[id] is set), else rows of every id
hipError_t launch_reverse(PoolView p, int by_batch, const uint8_t *in_batch, const uint32_t *bidx,
                          const uint32_t *ids, uint32_t nrows, uint32_t *cnt, uint32_t *off, uint32_t *scan_tmp,
                          uint32_t *src, const RevBufs &rb, DevScalars *ds, hipStream_t s);
hipError_t launch_scan_in_edges(PoolView p, const uint32_t *ids, uint32_t n, uint32_t *counts, hipStream_t s);
hipError_t launch_row_lengths(const uint32_t *off, const uint32_t *ids, uint32_t n, uint32_t *counts, hipStream_t s);
hipError_t launch_sort_adj_rows(const uint32_t *adj, uint32_t cap, uint32_t R, uint32_t *dst, hipStream_t s);
hipError_t launch_sort_rows(const uint32_t *off, uint32_t nrows, const uint32_t *src, uint32_t *dst,
                            hipStream_t s);
hipError_t launch_medoid(PoolView p, int kind, uint32_t dim, uint64_t n_active, void *tmp, DevScalars *ds,
                         hipStream_t s);
size_t medoid_tmp_bytes(uint32_t cap, uint32_t dim);
hipError_t launch_medoid_need(DevScalars *ds, const uint8_t *in_batch, int force, hipStream_t s);
hipError_t launch_cagra_fwd(PoolView p, const uint32_t *ids, uint32_t n, const uint32_t *c_ids, const float *c_d,
                            uint32_t *rec_t, uint32_t *rec_s, float *rec_d, hipStream_t s);
hipError_t launch_cagra_detour(const CagraArgs &a, uint32_t grid, hipStream_t s);
hipError_t launch_cagra_racing(const CagraArgs &a, hipStream_t s);
hipError_t launch_cagra_affected(const uint32_t *ids, uint32_t n, const uint8_t *in_batch, const uint32_t *rev_off,
                                 const uint32_t *rev_src, int by_batch, uint32_t *mark, uint32_t epoch,
                                 uint32_t *list, DevScalars *ds, hipStream_t s);
hipError_t launch_cagra_pickone(const CagraArgs &a, uint32_t grid, hipStream_t s);

}  // namespace gr
