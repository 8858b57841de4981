/*
 * grand.h -- C ABI of the MI355X (gfx950) library for batched dynamic
 * updates of fixed-degree proximity-graph ANN indexes, following
 * "GrAND: GPU-based Dynamic Graph Indexes for Approximate Nearest Neighbour
 * Search": Vamana with GrANDRobustPrune (Alg. 4-6) and a CAGRA-style fixed
 * out-degree variant with lock-free find-and-replace (Alg. 7-8), both
 * searched by BeamSearch (Alg. 1).
 *
 * Conventions for every entry point
 *  - Status codes are returned; nothing is thrown across the ABI.
 *  - Pointer arguments may point to host memory or to device memory of the
 *    index's GPU; the library detects which.  The caller owns every buffer
 *    it passes; the library copies what it needs and keeps no pointer after
 *    the call returns.
 *  - All work is ordered on the index's HIP stream and every call returns
 *    after its work has completed (one host synchronisation per call).
 *  - Arguments are validated before any state changes: a call that fails
 *    validation leaves the index exactly as it was, and grand_last_error()
 *    describes the problem.  A HIP failure during a call returns
 *    GRAND_E_DEVICE and poisons the handle; every later call on it returns
 *    GRAND_E_STATE.
 *  - One index must not be used by two host threads at the same time.
 *  - Ids are the slots of the resource pool (Section 4: a pool of a fixed
 *    peak size N, ids in [0, N-1], deleted ids reusable).
 */
#ifndef GRAND_H
#define GRAND_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GRAND_INVALID 0xFFFFFFFFu

typedef struct grand_index grand_index;

typedef enum {
  GRAND_OK = 0,
  GRAND_E_ARG = -1,       /* malformed argument (sizes, k > beam, NaN/inf vector element, ...) */
  GRAND_E_ID = -2,        /* id out of range, repeated in a batch, or in the wrong active state */
  GRAND_E_CAPACITY = -3,  /* a size limit of the library would be exceeded */
  GRAND_E_DEVICE = -4,    /* a HIP call failed; the handle is poisoned */
  GRAND_E_OOM = -5,       /* device allocation failed (state unchanged) */
  GRAND_E_STATE = -6      /* the handle was poisoned by an earlier device failure */
} grand_status;

enum { GRAND_VAMANA = 0, GRAND_CAGRA = 1 };
enum { GRAND_F32 = 0, GRAND_U8 = 1 };
/* GRAND_MIPS: inner-product (maximum inner product) search through the L2
 * augmentation of Section 5.4: a stored vector is [x, sqrt(M^2 - |x|^2)]
 * and a query [q, 0], where M (grand_params.mips_norm) bounds every stored
 * norm, so that |x' - q'|^2 = M^2 + |q|^2 - 2 <x, q> orders points like
 * -<x, q>.  Callers pass vectors of `dim` elements; the extra coordinate is
 * computed as the fp32 rounding of the fp64 square root of M^2 - sum x_j^2
 * (the sum in dimension order).  Search distances are the squared L2
 * distances in the augmented space.  fp32 only, Vamana or CAGRA. */
enum { GRAND_L2 = 0, GRAND_IP = 1, GRAND_MIPS = 2 };
/* alpha test of GrANDRobustPrune (Alg. 4): alpha * Dist(p*, p') <= D_p[p']
 * on the squared distance (default), or on the Euclidean distance. */
enum { GRAND_ALPHA_ON_DIST = 0, GRAND_ALPHA_ON_L2 = 1 };
/* CAGRA reverse edges (Alg. 7): grouped per target and applied in
 * (distance, id) order by one owner (deterministic, default), or applied by
 * independent racing compare-and-swap updates as in the paper's lock-free
 * last-writer-wins form. */
enum { GRAND_CAS_GROUPED = 0, GRAND_CAS_RACING = 1 };
/* In-neighbour discovery for deletes (Alg. 8): the reverse lists of the
 * deleted nodes only (default): one pass over every list that keeps the
 * edges into the batch, then a histogram, prefix scan and scatter into CSR
 * rows indexed by batch position; or the full reverse graph of every node in
 * CSR form (the transpose that grand_export_graph also returns). */
enum { GRAND_REV_FULL = 0, GRAND_REV_BATCH = 1 };

typedef struct {
  uint32_t struct_size;  /* sizeof(grand_params) */
  int32_t algo;          /* GRAND_VAMANA | GRAND_CAGRA */
  int32_t dtype;         /* GRAND_F32 | GRAND_U8 (U8 requires L2) */
  int32_t metric;        /* GRAND_L2 | GRAND_IP (IP requires CAGRA and F32) | GRAND_MIPS (F32) */
  uint32_t dim;          /* vector length; f32 <= 1024, u8 <= 4096 */
  uint32_t capacity;     /* pool size N (ids in [0, N)), < 2^31 */
  uint32_t R;            /* degree bound (Vamana) / fixed degree (CAGRA), 1..64 */
  uint32_t L_build;      /* beam width of insert/delete searches (CAGRA: internal top-k), <= 256 */
  uint32_t P;            /* scratch capacity per node (Alg. 5 and 6), 1..128 */
  uint32_t c;            /* replacement edges per repaired neighbour (Alg. 6), <= 64 */
  uint32_t k_repair;     /* top-k of the delete search used for repair (Alg. 6), <= 64 */
  uint32_t max_iters;    /* expansion cap of insert/delete searches; 0 = 2 * L_build; <= 256 */
  float alpha;           /* pruning factor of GrANDRobustPrune */
  int32_t prune_rule;    /* GRAND_ALPHA_ON_DIST | GRAND_ALPHA_ON_L2 */
  int32_t cas_mode;      /* GRAND_CAS_GROUPED | GRAND_CAS_RACING */
  int32_t rev_mode;      /* GRAND_REV_FULL | GRAND_REV_BATCH */
  uint32_t max_batch;    /* batch size the per-batch buffers are first sized for (grown on demand) */
  float mips_norm;       /* GRAND_MIPS: M, at least the norm of every vector inserted or imported */
  int32_t device;        /* HIP device ordinal */
  void *stream;          /* hipStream_t for all work; NULL = the null stream */
} grand_params;

/* Fills p with the defaults (Vamana, f32, L2, R 64, L_build 128, P 64,
 * c 2, k_repair 50, alpha 1.2 -- the parameters of Section 5.4; reverse
 * lists of the delete batch only). */
void grand_default_params(grand_params *p);

/* Creates an index and allocates its whole resource pool on the device
 * (Section 3.1, resource-pool reuse; Section 4, peak size N).  *out
 * receives the handle.  Errors: GRAND_E_ARG for unsupported parameters,
 * GRAND_E_OOM, GRAND_E_DEVICE. */
grand_status grand_create(const grand_params *p, grand_index **out);

/* Frees the index and all its device memory.  NULL is accepted. */
grand_status grand_destroy(grand_index *h);

/* Sets the HIP stream used by later calls (e.g. torch's current stream). */
grand_status grand_set_stream(grand_index *h, void *stream);

/* BatchInsert (Alg. 3; Vamana Alg. 5; CAGRA Alg. 7).
 * vecs: n rows of dim elements of the index dtype, row-major, packed.
 * ids:  n distinct ids in [0, capacity) that are not active.
 * Every point is searched for on the graph as it was at the start of the
 * batch; forward lists are pruned per point; reverse edges are grouped per
 * target and applied once per target.  An index empty at the start of the
 * batch is bootstrapped from the batch itself (each point's candidates are
 * its nearest other batch points) and its medoid computed.
 * n == 0 is a no-op.  Errors: GRAND_E_ID, GRAND_E_ARG (non-finite element;
 * with GRAND_MIPS a vector whose norm exceeds mips_norm). */
grand_status grand_insert_batch(grand_index *h, const void *vecs, const uint32_t *ids, uint32_t n);

/* CAGRA graph construction (Section 2.2 on CAGRA; Section 4.2, CAGRA graph
 * construction): builds the fixed-degree graph of an empty GRAND_CAGRA
 * index over n points in one call, instead of growing it by batches.
 *   1. an approximate k-NN graph of degree knn by NN-Descent, `iters` rounds
 *      with `sample` new and `sample` old entries sampled per list per round
 *      (local joins between the sampled neighbours and reverse neighbours;
 *      every round reads the lists of the round's start);
 *   2. rank-based pruning: per node, the R neighbours with the fewest
 *      detourable routes (a route u -> z -> y with both ranks below the rank
 *      of y in u's list), by (routes, rank);
 *   3. reverse edges: the output list of y is the first R/2 of its pruned
 *      list, then the nodes whose pruned list holds y (ascending by that
 *      position, then id), then the rest of its pruned list, up to R.
 * vecs, ids: as for grand_insert_batch (n distinct inactive ids).
 * init: n x knn row-major batch positions (host or device): row p holds knn
 *   distinct positions in [0, n) other than p, the random initial neighbours
 *   (drawn by the caller, so that a run can be reproduced).
 * Requires R <= knn <= 128, knn < n, 1 <= sample <= 32, and
 * n * (12 sample^2 - 2 sample) < 2^32 (proposals of one round).  The medoid
 * is computed at the end.  Argument and validation errors change nothing.
 * Errors: GRAND_E_ARG
 * (wrong variant, index not empty, bad sizes or initial lists, non-finite
 * element), GRAND_E_ID, GRAND_E_CAPACITY, GRAND_E_OOM. */
grand_status grand_build_cagra(grand_index *h, const void *vecs, const uint32_t *ids, uint32_t n,
                               const uint32_t *init, uint32_t knn, uint32_t iters, uint32_t sample);

/* BatchDelete (Alg. 3; Vamana Alg. 6; CAGRA Alg. 8), in place.
 * ids: n distinct active ids.  In-neighbours of the deleted nodes are found
 * exactly from a reverse graph built on the GPU for this batch; their lists
 * and those of the repair targets are rebuilt so that no edge points to a
 * deleted id; the deleted rows are cleared and their ids become free.  If
 * the medoid is deleted a new one is installed.
 * n == 0 is a no-op.  Errors: GRAND_E_ID. */
grand_status grand_delete_batch(grand_index *h, const uint32_t *ids, uint32_t n);

/* BeamSearch (Alg. 1) from the medoid with l = beam and at most 2*beam
 * expansions, for nq queries (nq rows of dim elements, packed).
 * out_ids / out_dists: nq x k, the k closest (distance, id) found, padded
 * with GRAND_INVALID / +inf (an empty index returns only padding).
 * Requires 1 <= k <= beam <= 256.  Errors: GRAND_E_ARG. */
grand_status grand_search(grand_index *h, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                          uint32_t *out_ids, float *out_dists);

/* Bytes of the fixed device array that grand_search_static works in. */
#define GRAND_STATIC_SCRATCH_BYTES (8u << 20)

/* grand_search for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, semantics and errors as grand_search, and the same
 * kernels; the staged query rows and the result lists live in a fixed
 * device array of GRAND_STATIC_SCRATCH_BYTES that the library holds on
 * every GPU it runs on until the process ends, so the call allocates
 * nothing (no phase timing and no counting run apply to it).
 * Limit: align256(nq * row) + 2 * align256(nq * k * 4) <= that size, where
 * row is the vector length in bytes rounded up to 16 (for 128-byte rows
 * and k = 10 about 40,000 queries); larger calls return GRAND_E_CAPACITY
 * with nothing done.  Every call on one GPU shares that GPU's array: calls
 * that overlap in time on one GPU (from several threads, or several indexes
 * on different streams) race on it and must be serialised by the caller. */
grand_status grand_search_static(grand_index *h, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                                 uint32_t *out_ids, float *out_dists);

/* In-neighbour detection, the step a delete batch needs before it can
 * repair (Alg. 8 builds a reverse graph for it; Section 4.2 reports that
 * building it is an order of magnitude faster than a linear scan of the
 * graph for each deleted point).  Counts, for each of n distinct active ids,
 * the lists of active nodes that hold it, by one of three methods so that
 * their costs can be compared:
 *   GRAND_INDEG_SCAN      a scan of every list for each id (n passes over
 *                         the adjacency; n <= 65535);
 *   GRAND_INDEG_REV_BATCH the reverse lists of the ids only, as a delete
 *                         batch builds them (one pass);
 *   GRAND_INDEG_REV_FULL  the full reverse graph of every node.
 * out_counts: n counts (host or device).  ms (may be NULL): GPU time of the
 * method, from events on the index's stream.  The index is not changed.
 * Errors: GRAND_E_ID (ids out of range, repeated or inactive), GRAND_E_ARG. */
enum { GRAND_INDEG_SCAN = 0, GRAND_INDEG_REV_BATCH = 1, GRAND_INDEG_REV_FULL = 2 };
grand_status grand_count_in_edges(grand_index *h, const uint32_t *ids, uint32_t n, int method, uint32_t *out_counts,
                                  float *ms);

/* Readers: searches that may run while the index's own host thread
 * inserts or deletes (Section 2.3 overlaps kernels on several streams;
 * Section 3.1 names the read-write race of a search reading a list that a
 * delete repairs).  A reader has its own HIP stream (`stream`, or a new
 * non-blocking stream of default priority when NULL), its own staging
 * buffers and counters; grand_reader_search may be called from one other
 * host thread at a time per reader, concurrently with any insert, delete or
 * search call on the index.  Readers must be destroyed before the index;
 * grand_import_graph must not overlap a reader's search.
 * Consistency model of a search that overlaps an update batch: every list
 * entry it reads is a pool id below the capacity or INVALID (lists are
 * rewritten one 32-bit entry at a time); a list that the batch rewrites is
 * read before, after, or part-way through its rewrite, so it may mix old
 * and new entries; a node deleted by the batch may still be reached and
 * returned, and an id that the batch re-inserts may be read with its old
 * or new vector (or, while its row is being copied, a mix of the two).  The
 * start node is the index's medoid as each search begins.  A search that
 * overlaps no update sees the state after the last completed call and
 * returns exactly what grand_search returns.
 * grand_reader_search has the arguments, results and errors of
 * grand_search, and returns after its work on the reader's stream has
 * completed. */
typedef struct grand_reader grand_reader;
grand_status grand_reader_create(grand_index *h, void *stream, grand_reader **out);
grand_status grand_reader_search(grand_reader *r, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                                 uint32_t *out_ids, float *out_dists);
grand_status grand_reader_destroy(grand_reader *r);
const char *grand_reader_last_error(const grand_reader *r);

/* Copies the index state out.  Any output pointer may be NULL.
 *   adj: capacity x R lists, GRAND_INVALID padding.  Vamana lists are sets
 *        (their order carries no meaning) and are returned canonically:
 *        each row's ids ascending, padding last.  CAGRA lists are returned
 *        in slot order, which the find-and-replace rules depend on;
 *   deg: capacity;
 *   active: capacity bytes (0/1);  medoid: 1 id (GRAND_INVALID if empty).
 *   rev_offsets (capacity + 1) / rev_srcs: the reverse graph of the current
 *        graph in CSR form, rows ascending by source id (Alg. 8).  With
 *        rev_srcs NULL only the offsets and *nnz are produced, so the caller
 *        can size rev_srcs and call again.  nnz: number of edges. */
grand_status grand_export_graph(grand_index *h, uint32_t *adj, uint32_t *deg, uint8_t *active, uint32_t *medoid,
                                uint32_t *rev_offsets, uint32_t *rev_srcs, uint64_t *nnz);

/* Replaces the whole state: vecs (capacity rows, packed), adj (capacity x
 * R), deg, active (capacity bytes), medoid.  Lists must hold only active ids
 * without repeats.  Used to resume from an exported state and by tests.
 * Errors: GRAND_E_ARG (malformed lists). */
grand_status grand_import_graph(grand_index *h, const void *vecs, const uint32_t *adj, const uint32_t *deg,
                                const uint8_t *active, uint32_t medoid);

/* Per-phase timing and work counters. */
enum {
  GRAND_PH_VALIDATE = 0, GRAND_PH_STAGE, GRAND_PH_SEARCH_INSERT, GRAND_PH_BOOTSTRAP, GRAND_PH_PRUNE_FWD,
  GRAND_PH_GROUP, GRAND_PH_REBUILD, GRAND_PH_SEARCH_DELETE, GRAND_PH_REVERSE, GRAND_PH_REPAIR,
  GRAND_PH_CLEAR, GRAND_PH_MEDOID, GRAND_PH_SEARCH_QUERY, GRAND_PH_CAGRA_DETOUR, GRAND_PH_CAGRA_PICKONE,
  GRAND_NPHASE
};

typedef struct {
  uint32_t struct_size;            /* sizeof(grand_stats_t) */
  uint32_t timing_enabled;
  uint64_t inserted, deleted, queried;
  uint64_t search_hops[3];         /* [insert, delete, query] searches: nodes expanded */
  uint64_t search_evals[3];        /* distance evaluations (row gathers) of those searches */
  uint64_t fwd_evals;              /* pairwise distance evaluations in forward prunes */
  uint64_t fwd_prunes;             /* forward GrANDRobustPrune invocations */
  uint64_t rebuild_evals;          /* distance evaluations in dirty rebuilds (D_u and pairwise) */
  uint64_t rebuild_prunes;         /* dirty rebuilds that ran GrANDRobustPrune */
  uint64_t dirty;                  /* dirty nodes rebuilt (or CAGRA targets / affected nodes) */
  uint64_t rebuild_records;        /* scratch records read by dirty rebuilds */
  uint64_t records;                /* reverse-edge / repair records emitted */
  uint64_t rev_edges;              /* edges found by reverse-graph builds */
  uint64_t repair_evals;           /* distance evaluations in delete repair */
  uint64_t rebuild_rows;           /* vector rows pruning rebuilds need (|C| + 1 each) */
  uint64_t repair_rows;            /* vector rows repairs need (neighbours + |C_i|) */
  uint64_t repair_records;         /* records written by repairs */
  uint64_t search_distinct[3];     /* distinct ids whose distance a search needs: {start} and every
                                      neighbour of an expanded node (counting runs only) */
  uint64_t search_capped[3];       /* searches stopped by max_iters with unexpanded candidates left */
  double phase_ms[GRAND_NPHASE];   /* summed kernel time per phase (timing enabled) */
  uint64_t phase_calls[GRAND_NPHASE];
} grand_stats_t;

/* Enables (1) or disables (0) per-phase HIP event timing on the stream.
 * Phases of a few microseconds (validate, stage, clear, medoid) are not
 * timed, since each recorded event adds a short gap on the stream; their
 * phase_ms stay 0. */
grand_status grand_set_timing(grand_index *h, int enable);

/* Enables (1) or disables (0) counting runs, a measurement mode: every
 * search then uses an exact visited bitmap of one bit per pool id in device
 * memory (capacity/8 bytes per search of a launch, allocated on demand)
 * instead of its lossy visited hash, so that each needed distance is
 * evaluated once and search_distinct counts the method's own distance
 * evaluations (Alg. 1 needs Dist for the start and for every neighbour of
 * an expanded node).  Results are the same as without counting; searches
 * are slower.  Errors: GRAND_E_OOM when the bitmap cannot be allocated. */
grand_status grand_set_counting(grand_index *h, int enable);

/* Copies the counters into out, which must point to at least `size` >=
 * sizeof(grand_stats_t) bytes laid out as grand_stats_t (its struct_size
 * is set).  Errors: GRAND_E_ARG for a null or smaller buffer. */
grand_status grand_stats(grand_index *h, void *out, size_t size);
grand_status grand_reset_stats(grand_index *h);

/* Text of the last error on this handle ("" if none). */
const char *grand_last_error(const grand_index *h);

#ifdef __cplusplus
}
#endif
#endif /* GRAND_H */
