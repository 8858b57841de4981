/*
 * grand_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU implementation of the batched dynamic
 * update of a fixed-degree proximity-graph ANN index described in
 * "GrAND: GPU-based Dynamic Graph Indexes for ANN Search" (Vamana with
 * GrANDRobustPrune, Alg. 4-6; CAGRA find-and-replace variant, Alg. 7-8;
 * BeamSearch, Alg. 1).  It exists so that tests, the smoke check and the
 * benchmark's CPU-baseline leg can check the GPU library against the paper.
 * Nothing in the product path may link, load or call it, and it shares no
 * code, header or constant with the GPU library.
 *
 * Conventions (each reading of the paper is restated where it is applied):
 *   - Every batch step reads the state at the start of the batch (or of the
 *     previous phase) and writes only state owned by the item it processes,
 *     so the OpenMP loops below give the same result for any thread count.
 *   - All orders are the total order on (distance, id).
 *   - INVALID = 0xFFFFFFFF pads adjacency rows.
 *
 * Parity pins: see tests/test_oracle_*.py.  The whole-graph state after many
 * batches is "parity unpinned" beyond the invariants and property checks
 * those tests apply: the paper prints no worked example of it.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <omp.h>

#define O_INVALID 0xFFFFFFFFu

enum { O_OK = 0, O_E_ARG = -1, O_E_ID = -2, O_E_CAPACITY = -3, O_E_OOM = -5 };
enum { O_VAMANA = 0, O_CAGRA = 1 };
enum { O_F32 = 0, O_U8 = 1 };
enum { O_L2 = 0, O_IP = 1, O_MIPS = 2 };
enum { O_ALPHA_ON_DIST = 0, O_ALPHA_ON_L2 = 1 };

typedef struct {
    int32_t algo, dtype, metric, prune_rule;
    uint32_t dim, capacity, R, L_build, P, c, k_repair, max_iters;
    float alpha;
    int32_t threads;
    float mips_norm;           /* O_MIPS: M, the bound on every stored norm */
} ocfg;

typedef struct {
    uint64_t searches, hops, dist_evals, prunes, dirty, records, cap_dropped;
} ostats;

typedef struct {
    ocfg cfg;
    uint32_t sdim;             /* stored elements per row: dim, or dim + 1 for O_MIPS */
    size_t esize;              /* bytes per element */
    uint8_t *vecs;             /* capacity x dim */
    uint32_t *adj;             /* capacity x R */
    uint32_t *deg;             /* capacity */
    uint8_t *active;           /* capacity */
    uint32_t medoid;
    uint64_t n_active;
    ostats st;
    char err[256];
} oindex;

typedef struct { float d; uint32_t id; } okey;

static int key_less(okey a, okey b) { return a.d < b.d || (a.d == b.d && a.id < b.id); }

static int key_cmp(const void *pa, const void *pb) {
    okey a = *(const okey *)pa, b = *(const okey *)pb;
    if (key_less(a, b)) return -1;
    if (key_less(b, a)) return 1;
    return 0;
}

static int nthreads(const oindex *h) { return h->cfg.threads > 0 ? h->cfg.threads : omp_get_max_threads(); }

static const void *vec_of(const oindex *h, uint32_t id) {
    return h->vecs + (size_t)id * h->sdim * h->esize;
}

/* ------------------------------------------------------------------------
 * MIPS to L2 (Section 5.4): inner-product data are searched as L2 data by
 * storing x' = [x, sqrt(M^2 - |x|^2)] (M bounds every norm) and querying
 * with q' = [q, 0]: |x' - q'|^2 = M^2 + |q|^2 - 2 <x, q>, an increasing
 * function of -<x, q>.  The squared norm is an fp64 sum in dimension order,
 * the square root is taken in fp64 and rounded once to fp32.  Returns 0, or
 * -1 when |x|^2 exceeds M^2.
 * ---------------------------------------------------------------------- */
static int mips_row(const oindex *h, const float *x, float *out, int is_query) {
    const uint32_t d = h->cfg.dim;
    double s = 0.0;
    for (uint32_t j = 0; j < d; j++) { out[j] = x[j]; s = fma((double)x[j], (double)x[j], s); }
    if (is_query) { out[d] = 0.0f; return 0; }
    double M2 = (double)h->cfg.mips_norm * (double)h->cfg.mips_norm;
    double t = M2 - s;
    out[d] = (float)sqrt(t > 0.0 ? t : 0.0);
    return s > M2 ? -1 : 0;
}

/* A caller row (dim elements) as stored (sdim elements): copied, or
 * augmented for O_MIPS.  out holds sdim elements. */
static int store_row(const oindex *h, const void *x, void *out, int is_query) {
    if (h->cfg.metric == O_MIPS) return mips_row(h, x, out, is_query);
    memcpy(out, x, (size_t)h->cfg.dim * h->esize);
    return 0;
}

/* ------------------------------------------------------------------------
 * Dist (Alg. 1 takes a distance function; Section 5.1 uses Euclidean and
 * inner-product datasets).  Reading: one function Dist everywhere,
 *   L2: squared Euclidean distance, IP: negated inner product,
 * accumulated exactly for uint8 (integers) and in fp64 for fp32, one fused
 * multiply-add per dimension in dimension order, rounded once to fp32.
 * A zero result is returned as +0.
 * ---------------------------------------------------------------------- */
static float dist_raw(const oindex *h, const void *a, const void *b) {
    uint32_t d = h->sdim;
    float r;
    if (h->cfg.dtype == O_U8) {
        const uint8_t *x = a, *y = b;
        int64_t s = 0;
        if (h->cfg.metric == O_L2) {
            for (uint32_t j = 0; j < d; j++) { int64_t t = (int64_t)x[j] - (int64_t)y[j]; s += t * t; }
            r = (float)s;
        } else {
            for (uint32_t j = 0; j < d; j++) s += (int64_t)x[j] * (int64_t)y[j];
            r = (float)(-s);
        }
    } else {
        const float *x = a, *y = b;
        double s = 0.0;
        if (h->cfg.metric != O_IP) {
            for (uint32_t j = 0; j < d; j++) { double t = (double)x[j] - (double)y[j]; s = fma(t, t, s); }
            r = (float)s;
        } else {
            for (uint32_t j = 0; j < d; j++) s = fma((double)x[j], (double)y[j], s);
            r = (float)(-s);
        }
    }
    if (r == 0.0f) r = 0.0f;
    return r;
}

static float dist_ids(const oindex *h, uint32_t a, uint32_t b) {
    return dist_raw(h, vec_of(h, a), vec_of(h, b));
}

/* ------------------------------------------------------------------------
 * BeamSearch (Alg. 1).  C starts as {s}; V is empty.  While some element of
 * C is not in V (and |V| < max_iters, a cap added so the visited list has a
 * bound): expand u, the (Dist, id)-smallest element of C \ V, add it to V,
 * add every out-neighbour of u not already in C, and keep the l smallest.
 * Dedupe is against C only: an id evicted from C can never re-enter, since
 * the l-th smallest key never increases once C is full.
 * Returns C (sorted, |C| <= l) and V in expansion order, with distances.
 * ---------------------------------------------------------------------- */
typedef struct {
    okey *C; uint8_t *vis; uint32_t nC;
    okey *V; uint32_t nV;
    uint64_t evals;
} osearch;

static void beam_search(const oindex *h, const void *q, uint32_t s, uint32_t ell,
                        uint32_t max_iters, osearch *out) {
    const uint32_t R = h->cfg.R;
    okey *C = out->C;
    uint8_t *vis = out->vis;
    uint32_t nC = 0, nV = 0;
    uint64_t evals = 0;
    C[0].d = dist_raw(h, q, vec_of(h, s));
    C[0].id = s;
    vis[0] = 0;
    nC = 1;
    evals++;
    while (nV < max_iters) {
        uint32_t i;
        for (i = 0; i < nC; i++) if (!vis[i]) break;      /* argmin of C \ V */
        if (i == nC) break;
        vis[i] = 1;
        out->V[nV++] = C[i];
        uint32_t u = C[i].id;
        for (uint32_t t = 0; t < R; t++) {
            uint32_t v = h->adj[(size_t)u * R + t];
            if (v == O_INVALID) continue;
            int present = 0;
            for (uint32_t j = 0; j < nC; j++) if (C[j].id == v) { present = 1; break; }
            if (present) continue;
            okey k = { dist_raw(h, q, vec_of(h, v)), v };
            evals++;
            /* sorted insert; C holds at most ell + R entries before the cut */
            uint32_t pos = nC;
            while (pos > 0 && key_less(k, C[pos - 1])) { C[pos] = C[pos - 1]; vis[pos] = vis[pos - 1]; pos--; }
            C[pos] = k;
            vis[pos] = 0;
            nC++;
        }
        if (nC > ell) nC = ell;                             /* keep the l closest */
    }
    out->nC = nC;
    out->nV = nV;
    out->evals = evals;
}

static int search_alloc(osearch *s, uint32_t ell, uint32_t R, uint32_t max_iters) {
    s->C = malloc(sizeof(okey) * (ell + R + 1));
    s->vis = malloc(ell + R + 1);
    s->V = malloc(sizeof(okey) * (max_iters + 1));
    return s->C && s->vis && s->V;
}

static void search_free(osearch *s) { free(s->C); free(s->vis); free(s->V); }

/* ------------------------------------------------------------------------
 * GrANDRobustPrune (Alg. 4).  Candidates come with cached distances D_p
 * (Section 3.1: distances from the search are reused, never recomputed).
 * Candidates equal to p, INVALID or repeated are dropped; the rest are
 * taken in (D_p, id) order.  The first valid candidate p* is selected; if R
 * are selected the loop ends; otherwise every later valid p' with
 * alpha * Dist(p*, p') <= D_p[p'] is invalidated.  Reading of the alpha
 * test: alpha multiplies the same Dist used everywhere (squared L2), in
 * fp64; the variant ALPHA_ON_L2 applies alpha to the Euclidean distance,
 * i.e. alpha^2 * Dist <= D.  Output in selection order; returns |L|.
 * ---------------------------------------------------------------------- */
static uint32_t robust_prune(const oindex *h, uint32_t p, const okey *cand_in, uint32_t n,
                             uint32_t *L, uint64_t *evals) {
    const uint32_t R = h->cfg.R;
    okey *cand = malloc(sizeof(okey) * (n + 1));
    uint8_t *valid = malloc(n + 1);
    uint32_t m = 0;
    for (uint32_t i = 0; i < n; i++) {
        if (cand_in[i].id == p || cand_in[i].id == O_INVALID) continue;
        cand[m++] = cand_in[i];
    }
    qsort(cand, m, sizeof(okey), key_cmp);
    uint32_t w = 0;                     /* drop repeated ids (adjacent after the sort
                                           only if their D agree; check all) */
    for (uint32_t i = 0; i < m; i++) {
        int dup = 0;
        for (uint32_t j = 0; j < w; j++) if (cand[j].id == cand[i].id) { dup = 1; break; }
        if (!dup) cand[w++] = cand[i];
    }
    m = w;
    for (uint32_t i = 0; i < m; i++) valid[i] = 1;
    double a = (double)h->cfg.alpha;
    double coef = h->cfg.prune_rule == O_ALPHA_ON_L2 ? a * a : a;
    uint32_t nl = 0;
    for (uint32_t i = 0; i < m; i++) {
        if (!valid[i]) continue;
        L[nl++] = cand[i].id;             /* p* = argmin over valid candidates */
        valid[i] = 0;
        if (nl == R) break;
        for (uint32_t j = i + 1; j < m; j++) {
            if (!valid[j]) continue;
            float dij = dist_ids(h, cand[i].id, cand[j].id);
            (*evals)++;
            if (coef * (double)dij <= (double)cand[j].d) valid[j] = 0;
        }
    }
    free(cand);
    free(valid);
    return nl;
}

/* ------------------------------------------------------------------------
 * Medoid (Alg. 5 starts from a pre-computed medoid; Section 6.2 notes a new
 * medoid is installed when the medoid is deleted).  Reading: the active id
 * minimising (squared distance to the centroid, id).
 *   uint8: exact.  With n active points and per-dimension sums S_j, the
 *     squared distance of x to the centroid S/n is |n x - S|^2 / n^2, so the
 *     comparison uses the integer key sum_j (n x_j - S_j)^2 (128-bit).
 *   fp32: the centroid sums each dimension in a fixed order (blocks of 1024
 *     consecutive ids summed in ascending id order, block sums added in
 *     block order) and divides by n; the distance to it is a fused
 *     multiply-add chain in fp64, in dimension order.
 * ---------------------------------------------------------------------- */
#define O_CENTROID_BLOCK 1024u

static uint32_t medoid_u8(const oindex *h, uint64_t n) {
    const uint32_t d = h->sdim, cap = h->cfg.capacity;
    uint64_t *S = calloc(d, sizeof(uint64_t));
    for (uint32_t i = 0; i < cap; i++) {
        if (!h->active[i]) continue;
        const uint8_t *x = vec_of(h, i);
        for (uint32_t j = 0; j < d; j++) S[j] += x[j];
    }
    unsigned __int128 best = 0;
    uint32_t arg = O_INVALID;
    for (uint32_t i = 0; i < cap; i++) {
        if (!h->active[i]) continue;
        const uint8_t *x = vec_of(h, i);
        unsigned __int128 key = 0;
        for (uint32_t j = 0; j < d; j++) {
            __int128 t = (__int128)n * x[j] - (__int128)S[j];
            key += (unsigned __int128)(t * t);
        }
        if (arg == O_INVALID || key < best) { best = key; arg = i; }  /* ascending ids: ties keep the smaller id */
    }
    free(S);
    return arg;
}

static uint32_t compute_medoid(const oindex *h) {
    const uint32_t d = h->sdim, cap = h->cfg.capacity;
    uint64_t n = 0;
    for (uint32_t i = 0; i < cap; i++) n += h->active[i] ? 1 : 0;
    if (n == 0) return O_INVALID;
    if (h->cfg.dtype == O_U8) return medoid_u8(h, n);
    double *c = calloc(d, sizeof(double));
    for (uint32_t j = 0; j < d; j++) {
        double t = 0.0;
        for (uint32_t b0 = 0; b0 < cap; b0 += O_CENTROID_BLOCK) {
            double sb = 0.0;
            for (uint32_t i = b0; i < cap && i < b0 + O_CENTROID_BLOCK; i++)
                if (h->active[i]) sb = sb + (double)((const float *)vec_of(h, i))[j];
            t = t + sb;
        }
        c[j] = t / (double)n;
    }
    double best = INFINITY;
    uint32_t arg = O_INVALID;
    for (uint32_t i = 0; i < cap; i++) {
        if (!h->active[i]) continue;
        double s = 0.0;
        for (uint32_t j = 0; j < d; j++) {
            double t = (double)((const float *)vec_of(h, i))[j] - c[j];
            s = fma(t, t, s);
        }
        if (s < best) { best = s; arg = i; }   /* ascending ids: ties keep the smaller id */
    }
    free(c);
    return arg;
}

/* ------------------------------------------------------------------------
 * Reverse graph in CSR (Alg. 8, first two loops; Section 4.2): the exact
 * transpose of all out-lists of active nodes.  Filling sources in ascending
 * id order makes every row ascending by source id.
 * ---------------------------------------------------------------------- */
static uint64_t reverse_csr(const uint32_t *adj, const uint8_t *active, uint32_t cap, uint32_t R,
                            uint32_t *offsets, uint32_t *srcs) {
    uint32_t *cnt = calloc((size_t)cap + 1, sizeof(uint32_t));
    for (uint32_t u = 0; u < cap; u++) {
        if (!active[u]) continue;
        for (uint32_t t = 0; t < R; t++) {
            uint32_t v = adj[(size_t)u * R + t];
            if (v != O_INVALID) cnt[v]++;
        }
    }
    uint64_t acc = 0;
    for (uint32_t v = 0; v < cap; v++) { offsets[v] = (uint32_t)acc; acc += cnt[v]; }
    offsets[cap] = (uint32_t)acc;
    if (srcs) {
        for (uint32_t v = 0; v < cap; v++) cnt[v] = offsets[v];
        for (uint32_t u = 0; u < cap; u++) {
            if (!active[u]) continue;
            for (uint32_t t = 0; t < R; t++) {
                uint32_t v = adj[(size_t)u * R + t];
                if (v != O_INVALID) srcs[cnt[v]++] = u;
            }
        }
    }
    free(cnt);
    return acc;
}

/* ------------------------------------------------------------------------
 * Reverse-edge records and their grouping (Alg. 5 and Alg. 6 scratch
 * buffers).  A record (target, src, dist) asks to add src to target's list.
 * Reading of the scratch capacity P: per target, records are taken as a
 * set of sources (repeated (target, src) pairs count once) ordered by
 * (dist, src), and the first P are kept; the race-dependent "first come"
 * of the paper is replaced by this order.  Every target is dirty, also when
 * its records were dropped by the cap.  A record with src == INVALID only
 * marks its target dirty.
 * ---------------------------------------------------------------------- */
typedef struct { uint32_t t, s; float d; } orec;

static int rec_cmp(const void *pa, const void *pb) {
    const orec *a = pa, *b = pb;
    if (a->t != b->t) return a->t < b->t ? -1 : 1;
    int ai = a->s == O_INVALID, bi = b->s == O_INVALID;     /* markers last */
    if (ai != bi) return ai ? 1 : -1;
    if (a->d != b->d) return a->d < b->d ? -1 : 1;
    if (a->s != b->s) return a->s < b->s ? -1 : 1;
    return 0;
}

typedef struct {
    uint32_t n_dirty;
    uint32_t *dirty;     /* ascending */
    uint32_t *gofs;      /* n_dirty + 1 offsets into gsrc */
    uint32_t *gsrc;      /* kept sources per dirty node, in (dist, src) order */
    uint64_t cap_dropped;
} ogroups;

static void group_records(const oindex *h, orec *rec, uint64_t n, ogroups *g) {
    qsort(rec, n, sizeof(orec), rec_cmp);
    g->dirty = malloc(sizeof(uint32_t) * (n + 1));
    g->gofs = malloc(sizeof(uint32_t) * (n + 2));
    g->gsrc = malloc(sizeof(uint32_t) * (n + 1));
    g->n_dirty = 0;
    g->cap_dropped = 0;
    uint64_t ns = 0;
    uint64_t i = 0;
    while (i < n) {
        uint64_t j = i;
        while (j < n && rec[j].t == rec[i].t) j++;
        g->dirty[g->n_dirty] = rec[i].t;
        g->gofs[g->n_dirty] = (uint32_t)ns;
        uint32_t kept = 0;
        for (uint64_t k = i; k < j; k++) {
            if (rec[k].s == O_INVALID) continue;
            int dup = 0;
            for (uint64_t q = g->gofs[g->n_dirty]; q < ns; q++) if (g->gsrc[q] == rec[k].s) { dup = 1; break; }
            if (dup) continue;
            if (kept < h->cfg.P) { g->gsrc[ns++] = rec[k].s; kept++; }
            else g->cap_dropped++;
        }
        g->n_dirty++;
        i = j;
    }
    g->gofs[g->n_dirty] = (uint32_t)ns;
}

static void groups_free(ogroups *g) { free(g->dirty); free(g->gofs); free(g->gsrc); }

/* ------------------------------------------------------------------------
 * Dirty rebuild (Alg. 5 final loop; Alg. 6 "Rebuild neighbourhood"):
 * C = (N_out(u) U scratch_u) minus u and minus the delete batch; if |C| <= R
 * it is installed as is (existing entries first, then new sources in group
 * order), otherwise D_u is computed and GrANDRobustPrune(u, C, D_u) is
 * installed.  Each dirty node owns its row, so the loop is race-free.
 * ---------------------------------------------------------------------- */
static void rebuild_dirty(oindex *h, const ogroups *g, const uint8_t *in_batch) {
    const uint32_t R = h->cfg.R;
    uint64_t prunes = 0, evals = 0;
    #pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads(h)) reduction(+:prunes, evals)
    for (uint32_t k = 0; k < g->n_dirty; k++) {
        uint32_t u = g->dirty[k];
        uint32_t ng = g->gofs[k + 1] - g->gofs[k];
        uint32_t *C = malloc(sizeof(uint32_t) * (R + ng + 1));
        uint32_t m = 0;
        for (uint32_t pass = 0; pass < 2; pass++) {
            uint32_t cnt = pass == 0 ? R : ng;
            for (uint32_t t = 0; t < cnt; t++) {
                uint32_t v = pass == 0 ? h->adj[(size_t)u * R + t] : g->gsrc[g->gofs[k] + t];
                if (v == O_INVALID || v == u) continue;
                if (in_batch && in_batch[v]) continue;
                int dup = 0;
                for (uint32_t q = 0; q < m; q++) if (C[q] == v) { dup = 1; break; }
                if (!dup) C[m++] = v;
            }
        }
        uint32_t *row = h->adj + (size_t)u * R;
        if (m <= R) {
            for (uint32_t t = 0; t < R; t++) row[t] = t < m ? C[t] : O_INVALID;
            h->deg[u] = m;
        } else {
            okey *cand = malloc(sizeof(okey) * m);
            for (uint32_t q = 0; q < m; q++) { cand[q].id = C[q]; cand[q].d = dist_ids(h, u, C[q]); }
            evals += m;
            uint32_t *L = malloc(sizeof(uint32_t) * R);
            uint32_t nl = robust_prune(h, u, cand, m, L, &evals);
            for (uint32_t t = 0; t < R; t++) row[t] = t < nl ? L[t] : O_INVALID;
            h->deg[u] = nl;
            prunes++;
            free(L);
            free(cand);
        }
        free(C);
    }
    h->st.prunes += prunes;
    h->st.dist_evals += evals;
    h->st.dirty += g->n_dirty;
}

/* ------------------------------------------------------------------------
 * Validation (done before any state changes; a failing batch leaves the
 * index untouched).
 * ---------------------------------------------------------------------- */
static int validate_ids(oindex *h, const uint32_t *ids, uint32_t n, int want_active) {
    uint8_t *seen = calloc(h->cfg.capacity, 1);
    int rc = O_OK;
    for (uint32_t i = 0; i < n && rc == O_OK; i++) {
        uint32_t id = ids[i];
        if (id >= h->cfg.capacity) { snprintf(h->err, sizeof h->err, "id %u out of range", id); rc = O_E_ID; }
        else if (seen[id]) { snprintf(h->err, sizeof h->err, "id %u repeated in batch", id); rc = O_E_ID; }
        else if ((h->active[id] != 0) != (want_active != 0)) {
            snprintf(h->err, sizeof h->err, "id %u is %s", id, want_active ? "not active" : "already active");
            rc = O_E_ID;
        }
        else seen[id] = 1;
    }
    free(seen);
    return rc;
}

static int validate_vectors(oindex *h, const void *vecs, uint32_t n, int is_query) {
    if (h->cfg.dtype != O_F32) return O_OK;
    const float *x = vecs;
    for (uint64_t i = 0; i < (uint64_t)n * h->cfg.dim; i++)
        if (!isfinite(x[i])) { snprintf(h->err, sizeof h->err, "non-finite vector element"); return O_E_ARG; }
    if (h->cfg.metric == O_MIPS && !is_query) {
        float *tmp = malloc(sizeof(float) * h->sdim);
        int bad = 0;
        for (uint32_t i = 0; i < n && !bad; i++) bad = mips_row(h, x + (size_t)i * h->cfg.dim, tmp, 0) != 0;
        free(tmp);
        if (bad) { snprintf(h->err, sizeof h->err, "vector norm above mips_norm"); return O_E_ARG; }
    }
    return O_OK;
}

/* ========================================================================
 * Public entry points (ctypes).
 * ====================================================================== */
void *oracle_create(const ocfg *cfg) {
    if (!cfg || cfg->dim == 0 || cfg->capacity == 0 || cfg->R == 0 || cfg->R > 4096 ||
        cfg->L_build == 0) return NULL;
    oindex *h = calloc(1, sizeof(oindex));
    h->cfg = *cfg;
    if (h->cfg.max_iters == 0) h->cfg.max_iters = 2 * h->cfg.L_build;
    h->esize = cfg->dtype == O_U8 ? 1 : 4;
    h->sdim = cfg->dim + (cfg->metric == O_MIPS ? 1 : 0);
    size_t cap = cfg->capacity;
    h->vecs = calloc(cap * h->sdim, h->esize);
    h->adj = malloc(cap * cfg->R * sizeof(uint32_t));
    h->deg = calloc(cap, sizeof(uint32_t));
    h->active = calloc(cap, 1);
    if (!h->vecs || !h->adj || !h->deg || !h->active) return NULL;
    memset(h->adj, 0xFF, cap * cfg->R * sizeof(uint32_t));
    h->medoid = O_INVALID;
    return h;
}

void oracle_destroy(void *hv) {
    oindex *h = hv;
    if (!h) return;
    free(h->vecs); free(h->adj); free(h->deg); free(h->active); free(h);
}

const char *oracle_last_error(void *hv) { return ((oindex *)hv)->err; }
void oracle_set_threads(void *hv, int32_t t) { ((oindex *)hv)->cfg.threads = t; }
void oracle_get_stats(void *hv, ostats *out) { *out = ((oindex *)hv)->st; }

/* Stage (Alg. 5 first loop / Alg. 7 first loop): write the vector into its
 * slot, empty its list, mark it active. */
static void stage(oindex *h, const void *vecs, const uint32_t *ids, uint32_t n) {
    size_t row = (size_t)h->cfg.dim * h->esize;
    for (uint32_t i = 0; i < n; i++) {
        store_row(h, (const uint8_t *)vecs + (size_t)i * row, h->vecs + (size_t)ids[i] * h->sdim * h->esize, 0);
        for (uint32_t t = 0; t < h->cfg.R; t++) h->adj[(size_t)ids[i] * h->cfg.R + t] = O_INVALID;
        h->deg[ids[i]] = 0;
        h->active[ids[i]] = 1;
    }
    h->n_active += n;
}

/* Bootstrap for an index that is empty at the start of the batch (the
 * paper starts from seed graphs; reading: the candidates of each new point
 * are its `want` nearest other points of the batch, found by brute force). */
static void bootstrap_candidates(const oindex *h, const uint32_t *ids, uint32_t n, uint32_t want,
                                 okey *out /* n x want */, uint32_t *nout) {
    #pragma omp parallel for schedule(dynamic, 16) num_threads(nthreads(h))
    for (uint32_t i = 0; i < n; i++) {
        okey *all = malloc(sizeof(okey) * (n + 1));
        uint32_t m = 0;
        for (uint32_t j = 0; j < n; j++) {
            if (j == i) continue;
            all[m].id = ids[j];
            all[m].d = dist_ids(h, ids[i], ids[j]);
            m++;
        }
        qsort(all, m, sizeof(okey), key_cmp);
        uint32_t k = m < want ? m : want;
        memcpy(out + (size_t)i * want, all, sizeof(okey) * k);
        nout[i] = k;
        free(all);
    }
}

/* GrAND-Vamana BatchInsert (Alg. 5). */
static int vamana_insert(oindex *h, const void *vecs, const uint32_t *ids, uint32_t n) {
    const uint32_t R = h->cfg.R, ell = h->cfg.L_build, mi = h->cfg.max_iters;
    uint64_t n_active0 = h->n_active;
    uint32_t m0 = h->medoid;
    stage(h, vecs, ids, n);
    uint32_t cmax = n_active0 == 0 ? ell : mi;
    okey *cand = malloc(sizeof(okey) * (size_t)n * cmax);
    uint32_t *ncand = malloc(sizeof(uint32_t) * n);
    if (n_active0 == 0) {
        bootstrap_candidates(h, ids, n, ell, cand, ncand);
    } else {
        uint64_t hops = 0, evals = 0;
        /* forward search on the batch-start snapshot: new nodes have empty
           lists and no in-edges, so they are unreachable from the medoid */
        #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:hops, evals)
        for (uint32_t i = 0; i < n; i++) {
            osearch s;
            search_alloc(&s, ell, R, mi);
            beam_search(h, vec_of(h, ids[i]), m0, ell, mi, &s);
            memcpy(cand + (size_t)i * cmax, s.V, sizeof(okey) * s.nV);   /* V_i with D_{p_i} */
            ncand[i] = s.nV;
            hops += s.nV; evals += s.evals;
            search_free(&s);
        }
        h->st.searches += n; h->st.hops += hops; h->st.dist_evals += evals;
    }
    /* forward GrANDRobustPrune of V_i \ {p_i}; each item owns row p_i */
    uint32_t *L = malloc(sizeof(uint32_t) * (size_t)n * R);
    uint32_t *nL = malloc(sizeof(uint32_t) * n);
    uint64_t evals = 0;
    #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:evals)
    for (uint32_t i = 0; i < n; i++)
        nL[i] = robust_prune(h, ids[i], cand + (size_t)i * cmax, ncand[i], L + (size_t)i * R, &evals);
    h->st.dist_evals += evals;
    h->st.prunes += n;
    uint64_t nrec = 0;
    for (uint32_t i = 0; i < n; i++) {
        uint32_t *row = h->adj + (size_t)ids[i] * R;
        for (uint32_t t = 0; t < R; t++) row[t] = t < nL[i] ? L[(size_t)i * R + t] : O_INVALID;
        h->deg[ids[i]] = nL[i];
        nrec += nL[i];
    }
    /* reverse edges (u, p_i, D_{p_i}[u]) into per-target scratch */
    orec *rec = malloc(sizeof(orec) * (nrec + 1));
    uint64_t r = 0;
    for (uint32_t i = 0; i < n; i++) {
        const okey *ci = cand + (size_t)i * cmax;
        for (uint32_t t = 0; t < nL[i]; t++) {
            uint32_t u = L[(size_t)i * R + t];
            float du = NAN;
            for (uint32_t q = 0; q < ncand[i]; q++) if (ci[q].id == u) { du = ci[q].d; break; }
            rec[r].t = u; rec[r].s = ids[i]; rec[r].d = du; r++;
        }
    }
    ogroups g;
    group_records(h, rec, nrec, &g);
    h->st.records += nrec;
    h->st.cap_dropped += g.cap_dropped;
    rebuild_dirty(h, &g, NULL);
    groups_free(&g);
    free(rec); free(L); free(nL); free(cand); free(ncand);
    if (n_active0 == 0) h->medoid = compute_medoid(h);
    return O_OK;
}

/* GrAND-CAGRA BatchInsert (Alg. 7). */
static int cagra_insert(oindex *h, const void *vecs, const uint32_t *ids, uint32_t n) {
    const uint32_t R = h->cfg.R, ell = h->cfg.L_build, mi = h->cfg.max_iters;
    uint64_t n_active0 = h->n_active;
    uint32_t m0 = h->medoid;
    stage(h, vecs, ids, n);
    okey *fwd = malloc(sizeof(okey) * (size_t)n * R);   /* N_out(p_i) with distances */
    uint32_t *nf = malloc(sizeof(uint32_t) * n);
    if (n_active0 == 0) {
        bootstrap_candidates(h, ids, n, R, fwd, nf);
    } else {
        uint64_t hops = 0, evals = 0;
        #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:hops, evals)
        for (uint32_t i = 0; i < n; i++) {
            osearch s;
            search_alloc(&s, ell, R, mi);
            beam_search(h, vec_of(h, ids[i]), m0, ell, mi, &s);
            uint32_t k = s.nC < R ? s.nC : R;               /* the R closest (k = R) */
            memcpy(fwd + (size_t)i * R, s.C, sizeof(okey) * k);
            nf[i] = k;
            hops += s.nV; evals += s.evals;
            search_free(&s);
        }
        h->st.searches += n; h->st.hops += hops; h->st.dist_evals += evals;
    }
    uint64_t nrec = 0;
    for (uint32_t i = 0; i < n; i++) {
        uint32_t *row = h->adj + (size_t)ids[i] * R;
        for (uint32_t t = 0; t < R; t++) row[t] = t < nf[i] ? fwd[(size_t)i * R + t].id : O_INVALID;
        h->deg[ids[i]] = nf[i];
        nrec += nf[i];
    }
    /* backward edges: records (q, p_i) grouped by q, taken in (dist, p_i) order */
    orec *rec = malloc(sizeof(orec) * (nrec + 1));
    uint32_t *owner = malloc(sizeof(uint32_t) * (nrec + 1));  /* batch index of src */
    uint64_t r = 0;
    for (uint32_t i = 0; i < n; i++)
        for (uint32_t t = 0; t < nf[i]; t++) {
            rec[r].t = fwd[(size_t)i * R + t].id; rec[r].s = ids[i]; rec[r].d = fwd[(size_t)i * R + t].d; r++;
        }
    qsort(rec, nrec, sizeof(orec), rec_cmp);
    /* map src id -> batch index (ids are unique within the batch) */
    uint32_t *bidx = malloc(sizeof(uint32_t) * h->cfg.capacity);
    for (uint32_t i = 0; i < n; i++) bidx[ids[i]] = i;
    for (uint64_t k = 0; k < nrec; k++) owner[k] = bidx[rec[k].s];
    /* group starts */
    uint64_t *gstart = malloc(sizeof(uint64_t) * (nrec + 1));
    uint64_t ng = 0;
    for (uint64_t k = 0; k < nrec; k++) if (k == 0 || rec[k].t != rec[k - 1].t) gstart[ng++] = k;
    gstart[ng] = nrec;
    /* one owner per target q: for each record, if q's list has a free slot
       the new node fills the first one; otherwise pick the element of
       N_out(q) n N_out(p_i) at the highest slot of q's list and replace it by
       p_i (detour find-and-replace).  N_out(p_i) is read from the forward
       lists as written above (a snapshot), never from a list being edited. */
    #pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads(h))
    for (uint64_t gi = 0; gi < ng; gi++) {
        uint32_t q = rec[gstart[gi]].t;
        uint32_t *row = h->adj + (size_t)q * R;
        for (uint64_t k = gstart[gi]; k < gstart[gi + 1]; k++) {
            uint32_t p = rec[k].s;
            int has = 0, free_slot = -1;
            for (uint32_t t = 0; t < R; t++) {
                if (row[t] == p) has = 1;
                if (row[t] == O_INVALID && free_slot < 0) free_slot = (int)t;
            }
            if (has) continue;
            if (free_slot >= 0) { row[free_slot] = p; continue; }
            const okey *fp = fwd + (size_t)owner[k] * R;
            uint32_t nfp = nf[owner[k]];
            for (int t = (int)R - 1; t >= 0; t--) {
                int in = 0;
                for (uint32_t j = 0; j < nfp; j++) if (fp[j].id == row[t]) { in = 1; break; }
                if (in) { row[t] = p; break; }
            }
        }
        uint32_t dg = 0;
        for (uint32_t t = 0; t < R; t++) dg += row[t] != O_INVALID;
        h->deg[q] = dg;
    }
    h->st.records += nrec;
    h->st.dirty += ng;
    free(gstart); free(bidx); free(owner); free(rec); free(fwd); free(nf);
    if (n_active0 == 0) h->medoid = compute_medoid(h);
    return O_OK;
}

int32_t oracle_insert_batch(void *hv, const void *vecs, const uint32_t *ids, uint32_t n) {
    oindex *h = hv;
    h->err[0] = 0;
    if (n == 0) return O_OK;
    if (!vecs || !ids) { snprintf(h->err, sizeof h->err, "null argument"); return O_E_ARG; }
    int rc = validate_ids(h, ids, n, 0);
    if (rc) return rc;
    rc = validate_vectors(h, vecs, n, 0);
    if (rc) return rc;
    return h->cfg.algo == O_CAGRA ? cagra_insert(h, vecs, ids, n) : vamana_insert(h, vecs, ids, n);
}

/* Clear the deleted rows and re-install the medoid if it was deleted
 * (Alg. 6 last loop; Alg. 8 last loop; Section 6.2). */
static void clear_batch(oindex *h, const uint32_t *ids, uint32_t n, uint8_t *in_batch, uint32_t m0) {
    for (uint32_t i = 0; i < n; i++) {
        for (uint32_t t = 0; t < h->cfg.R; t++) h->adj[(size_t)ids[i] * h->cfg.R + t] = O_INVALID;
        h->deg[ids[i]] = 0;
        h->active[ids[i]] = 0;
    }
    h->n_active -= n;
    if (m0 != O_INVALID && in_batch[m0]) h->medoid = compute_medoid(h);
}

/* GrAND-Vamana BatchDelete (Alg. 6) with in-neighbours taken exactly from
 * the on-demand reverse graph (Section 1 contribution (iii), Alg. 3). */
static int vamana_delete(oindex *h, const uint32_t *ids, uint32_t n) {
    const uint32_t R = h->cfg.R, ell = h->cfg.L_build, mi = h->cfg.max_iters;
    const uint32_t cap = h->cfg.capacity, kr = h->cfg.k_repair, cc = h->cfg.c;
    uint32_t m0 = h->medoid;
    uint8_t *in_batch = calloc(cap, 1);
    for (uint32_t i = 0; i < n; i++) in_batch[ids[i]] = 1;
    /* C_i: the first k_repair of BeamSearch(x_{p_i}).C outside the batch */
    uint32_t *Ci = malloc(sizeof(uint32_t) * (size_t)n * (kr + 1));
    uint32_t *nCi = calloc(n, sizeof(uint32_t));
    uint64_t hops = 0, evals = 0;
    #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:hops, evals)
    for (uint32_t i = 0; i < n; i++) {
        osearch s;
        search_alloc(&s, ell, R, mi);
        beam_search(h, vec_of(h, ids[i]), m0, ell, mi, &s);
        uint32_t k = 0;
        for (uint32_t j = 0; j < s.nC && k < kr; j++)
            if (!in_batch[s.C[j].id]) Ci[(size_t)i * (kr + 1) + k++] = s.C[j].id;
        nCi[i] = k;
        hops += s.nV; evals += s.evals;
        search_free(&s);
    }
    h->st.searches += n; h->st.hops += hops; h->st.dist_evals += evals;
    /* reverse graph of the batch-start graph */
    uint32_t *offs = malloc(sizeof(uint32_t) * ((size_t)cap + 1));
    uint64_t nnz = reverse_csr(h->adj, h->active, cap, R, offs, NULL);
    uint32_t *srcs = malloc(sizeof(uint32_t) * (nnz + 1));
    reverse_csr(h->adj, h->active, cap, R, offs, srcs);
    /* record counts per deleted node: c per surviving in- and out-neighbour
       plus one dirty marker per surviving in-neighbour */
    uint64_t *rofs = malloc(sizeof(uint64_t) * (n + 1));
    rofs[0] = 0;
    for (uint32_t i = 0; i < n; i++) {
        uint32_t p = ids[i], nin = 0, nout = 0;
        for (uint32_t q = offs[p]; q < offs[p + 1]; q++) nin += !in_batch[srcs[q]];
        for (uint32_t t = 0; t < R; t++) {
            uint32_t w = h->adj[(size_t)p * R + t];
            nout += w != O_INVALID && !in_batch[w];
        }
        rofs[i + 1] = rofs[i] + (uint64_t)nin * (cc + 1) + (uint64_t)nout * cc;
    }
    uint64_t nrec = rofs[n];
    orec *rec = malloc(sizeof(orec) * (nrec + 1));
    uint64_t used_total = 0;
    evals = 0;
    #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:evals, used_total)
    for (uint32_t i = 0; i < n; i++) {
        uint32_t p = ids[i];
        const uint32_t *ci = Ci + (size_t)i * (kr + 1);
        okey *tmp = malloc(sizeof(okey) * (nCi[i] + 1));
        uint64_t r = rofs[i];
        /* in-neighbour repair: z gets the c points of C_i closest to z */
        for (uint32_t q = offs[p]; q < offs[p + 1]; q++) {
            uint32_t z = srcs[q];
            if (in_batch[z]) continue;
            uint32_t m = 0;
            for (uint32_t j = 0; j < nCi[i]; j++) {
                if (ci[j] == z) continue;
                tmp[m].id = ci[j]; tmp[m].d = dist_ids(h, z, ci[j]); m++;
            }
            evals += m;
            qsort(tmp, m, sizeof(okey), key_cmp);
            for (uint32_t j = 0; j < cc; j++) {
                rec[r].t = z;
                rec[r].s = j < m ? tmp[j].id : O_INVALID;
                rec[r].d = j < m ? tmp[j].d : 0.0f;
                r++;
            }
            rec[r].t = z; rec[r].s = O_INVALID; rec[r].d = 0.0f; r++;     /* z is dirty */
        }
        /* out-neighbour repair: w is added to the lists of the c points of
           C_i closest to w */
        for (uint32_t t = 0; t < R; t++) {
            uint32_t w = h->adj[(size_t)p * R + t];
            if (w == O_INVALID || in_batch[w]) continue;
            uint32_t m = 0;
            for (uint32_t j = 0; j < nCi[i]; j++) {
                if (ci[j] == w) continue;
                tmp[m].id = ci[j]; tmp[m].d = dist_ids(h, w, ci[j]); m++;
            }
            evals += m;
            qsort(tmp, m, sizeof(okey), key_cmp);
            for (uint32_t j = 0; j < cc; j++) {
                if (j < m) { rec[r].t = tmp[j].id; rec[r].s = w; rec[r].d = tmp[j].d; }
                else { rec[r].t = O_INVALID; rec[r].s = O_INVALID; rec[r].d = 0.0f; }
                r++;
            }
        }
        used_total += r - rofs[i];
        free(tmp);
    }
    h->st.dist_evals += evals;
    /* drop empty records (target INVALID) before grouping */
    uint64_t w = 0;
    for (uint64_t k = 0; k < nrec; k++) if (rec[k].t != O_INVALID) rec[w++] = rec[k];
    ogroups g;
    group_records(h, rec, w, &g);
    h->st.records += w;
    h->st.cap_dropped += g.cap_dropped;
    rebuild_dirty(h, &g, in_batch);
    groups_free(&g);
    clear_batch(h, ids, n, in_batch, m0);
    free(rec); free(rofs); free(srcs); free(offs); free(Ci); free(nCi); free(in_batch);
    return O_OK;
}

/* GrAND-CAGRA BatchDelete (Alg. 8).  Reading of PickOne's round-robin: the
 * in-neighbour u of a deleted p starts its cyclic scan of N_out(p) (valid
 * entries in slot order) at (rank of u in N_in(p)) mod |N_out(p)| and takes
 * the first r outside the batch, different from u and not already in
 * N_out(u); with no such r the slot becomes INVALID.  Each affected u owns
 * its list and handles its deleted out-neighbours in slot order. */
static int cagra_delete(oindex *h, const uint32_t *ids, uint32_t n) {
    const uint32_t R = h->cfg.R, cap = h->cfg.capacity;
    uint32_t m0 = h->medoid;
    uint8_t *in_batch = calloc(cap, 1);
    for (uint32_t i = 0; i < n; i++) in_batch[ids[i]] = 1;
    uint32_t *offs = malloc(sizeof(uint32_t) * ((size_t)cap + 1));
    uint64_t nnz = reverse_csr(h->adj, h->active, cap, R, offs, NULL);
    uint32_t *srcs = malloc(sizeof(uint32_t) * (nnz + 1));
    reverse_csr(h->adj, h->active, cap, R, offs, srcs);
    uint8_t *affected = calloc(cap, 1);
    for (uint32_t i = 0; i < n; i++)
        for (uint32_t q = offs[ids[i]]; q < offs[ids[i] + 1]; q++)
            if (!in_batch[srcs[q]]) affected[srcs[q]] = 1;
    uint64_t n_aff = 0;
    #pragma omp parallel for schedule(dynamic, 256) num_threads(nthreads(h)) reduction(+:n_aff)
    for (uint32_t u = 0; u < cap; u++) {
        if (!affected[u]) continue;
        n_aff++;
        uint32_t *row = h->adj + (size_t)u * R;
        for (uint32_t s = 0; s < R; s++) {
            uint32_t p = row[s];
            if (p == O_INVALID || !in_batch[p]) continue;
            uint32_t L[4096];
            uint32_t nl = 0;
            for (uint32_t t = 0; t < R; t++) {
                uint32_t v = h->adj[(size_t)p * R + t];   /* p's list is never edited here */
                if (v != O_INVALID) L[nl++] = v;
            }
            uint32_t rank = 0;
            for (uint32_t q = offs[p]; q < offs[p + 1]; q++) if (srcs[q] == u) { rank = q - offs[p]; break; }
            uint32_t chosen = O_INVALID;
            for (uint32_t j = 0; j < nl; j++) {
                uint32_t r = L[(rank + j) % nl];
                if (in_batch[r] || r == u) continue;
                int in = 0;
                for (uint32_t t = 0; t < R; t++) if (row[t] == r) { in = 1; break; }
                if (in) continue;
                chosen = r;
                break;
            }
            row[s] = chosen;
        }
        uint32_t dg = 0;
        for (uint32_t t = 0; t < R; t++) dg += row[t] != O_INVALID;
        h->deg[u] = dg;
    }
    h->st.dirty += n_aff;
    clear_batch(h, ids, n, in_batch, m0);
    free(affected); free(srcs); free(offs); free(in_batch);
    return O_OK;
}

int32_t oracle_delete_batch(void *hv, const uint32_t *ids, uint32_t n) {
    oindex *h = hv;
    h->err[0] = 0;
    if (n == 0) return O_OK;
    if (!ids) { snprintf(h->err, sizeof h->err, "null argument"); return O_E_ARG; }
    int rc = validate_ids(h, ids, n, 1);
    if (rc) return rc;
    return h->cfg.algo == O_CAGRA ? cagra_delete(h, ids, n) : vamana_delete(h, ids, n);
}

/* Search: BeamSearch from the medoid with l = beam and a cap of 2 * beam
 * expansions; the first k of C, padded with INVALID / +inf. */
/* ------------------------------------------------------------------------
 * CAGRA graph construction (Section 2.2 on CAGRA; Section 4.2, CAGRA graph
 * construction): an approximate k-NN graph by NN-Descent, optimised into a
 * fixed-degree graph by rank-based edge reordering and pruning, then
 * reverse-edge addition.  The paper names these steps without their
 * parameters; the readings used here:
 *
 * NN-Descent, batch-synchronous.  Node u keeps a list L(u) of K entries
 * (Dist, v, new flag), ascending by (Dist, v).  L(u) starts from the K
 * caller-drawn random neighbours init[u] (all new).  One round:
 *   1. samples: NS(u) = the first S new entries of L(u) in list order, OS(u)
 *      = the first S old ones; the sampled new entries become old;
 *   2. reverse samples: RN(v) = the S smallest (Dist, u) over the u with v in
 *      NS(u) (Dist from u's entry), RO(v) likewise from OS;
 *   3. local join at every v: Bn = NS(v) u RN(v), Bo = (OS(v) u RO(v)) \ Bn;
 *      every pair {a, b} of distinct points of Bn, and every (a in Bn, b in
 *      Bo), gives Dist(a, b); b is proposed to a when (Dist, b) is below the
 *      key of the last entry of L(a) at the start of the round, and a to b
 *      likewise;
 *   4. merge: L(u) <- the K smallest distinct keys of L(u) and u's
 *      proposals; a proposal whose key is already in L(u) is dropped (the
 *      entry keeps its flag), the others enter as new.
 * Rank-based pruning: the rank of v in L(u) is its position.  An edge u -> y
 * of rank r has a detourable route through z when z has rank rz < r in L(u)
 * and y has rank ry < r in L(z).  The pruned list P(u) is the R entries with
 * the fewest detourable routes, ascending by (routes, r).
 * Reverse edges: y's reverse neighbours are the u with y in P(u), ascending
 * by (position of y in P(u), u).  The output list of y is the first R/2
 * entries of P(y), then its reverse neighbours in order, then the rest of
 * P(y), skipping ids already taken, up to R.
 * Positions 0..n-1 stand for ids[0..n-1] until the output is written.
 * ---------------------------------------------------------------------- */
typedef struct { float d; uint32_t v; uint8_t isnew; } oent;

static int ent_less(const oent *a, const oent *b) { return a->d < b->d || (a->d == b->d && a->v < b->v); }
static int ent_cmp(const void *pa, const void *pb) {
    const oent *a = pa, *b = pb;
    if (ent_less(a, b)) return -1;
    if (ent_less(b, a)) return 1;
    return 0;
}
static int okey_cmp_u(const void *pa, const void *pb) { return key_cmp(pa, pb); }

/* the S smallest (d, id) keys over all records (t, id, d) with target t, per
 * target; out: n x S ids, INVALID padded */
static void smallest_per_target(uint32_t n, uint32_t S, const orec *rec, uint64_t nrec, uint32_t *out) {
    uint64_t *cnt = calloc((size_t)n + 1, sizeof(uint64_t));
    for (uint64_t k = 0; k < nrec; k++) cnt[rec[k].t + 1]++;
    for (uint32_t t = 0; t < n; t++) cnt[t + 1] += cnt[t];
    okey *all = malloc(sizeof(okey) * (nrec + 1));
    uint64_t *fill = malloc(sizeof(uint64_t) * ((size_t)n + 1));
    memcpy(fill, cnt, sizeof(uint64_t) * ((size_t)n + 1));
    for (uint64_t k = 0; k < nrec; k++) { okey e = { rec[k].d, rec[k].s }; all[fill[rec[k].t]++] = e; }
    for (uint32_t t = 0; t < n; t++) {
        uint64_t a = cnt[t], b = cnt[t + 1];
        qsort(all + a, b - a, sizeof(okey), okey_cmp_u);
        for (uint32_t j = 0; j < S; j++) out[(size_t)t * S + j] = a + j < b ? all[a + j].id : O_INVALID;
    }
    free(cnt); free(all); free(fill);
}

static int in_list(const uint32_t *a, uint32_t m, uint32_t v) {
    for (uint32_t i = 0; i < m; i++) if (a[i] == v) return 1;
    return 0;
}

/* NN-Descent over positions 0..n-1 (point p is row ids[p] of the index);
 * L: n x K, the result, ascending per node. */
static void nn_descent(const oindex *h, const uint32_t *ids, uint32_t n, const uint32_t *init, uint32_t K,
                       uint32_t iters, uint32_t S, oent *L) {
    const int nt = nthreads(h);
    #pragma omp parallel for schedule(static) num_threads(nt)
    for (uint32_t u = 0; u < n; u++) {
        oent *l = L + (size_t)u * K;
        for (uint32_t j = 0; j < K; j++) {
            uint32_t v = init[(size_t)u * K + j];
            l[j].d = dist_ids(h, ids[u], ids[v]); l[j].v = v; l[j].isnew = 1;
        }
        qsort(l, K, sizeof(oent), ent_cmp);
    }
    uint32_t *NS = malloc(sizeof(uint32_t) * (size_t)n * S), *OS = malloc(sizeof(uint32_t) * (size_t)n * S);
    uint32_t *RN = malloc(sizeof(uint32_t) * (size_t)n * S), *RO = malloc(sizeof(uint32_t) * (size_t)n * S);
    orec *rn = malloc(sizeof(orec) * ((size_t)n * S + 1)), *ro = malloc(sizeof(orec) * ((size_t)n * S + 1));
    for (uint32_t it = 0; it < iters; it++) {
        /* 1. samples */
        uint64_t nrn = 0, nro = 0;
        for (uint32_t u = 0; u < n; u++) {
            oent *l = L + (size_t)u * K;
            uint32_t cn = 0, co = 0;
            for (uint32_t j = 0; j < K; j++) {
                if (l[j].isnew) {
                    if (cn < S) {
                        NS[(size_t)u * S + cn++] = l[j].v;
                        orec r = { l[j].v, u, l[j].d }; rn[nrn++] = r;
                        l[j].isnew = 0;
                    }
                } else if (co < S) {
                    OS[(size_t)u * S + co++] = l[j].v;
                    orec r = { l[j].v, u, l[j].d }; ro[nro++] = r;
                }
            }
            for (; cn < S; cn++) NS[(size_t)u * S + cn] = O_INVALID;
            for (; co < S; co++) OS[(size_t)u * S + co] = O_INVALID;
        }
        /* 2. reverse samples */
        smallest_per_target(n, S, rn, nrn, RN);
        smallest_per_target(n, S, ro, nro, RO);
        /* 3. local joins: proposals against the keys of the round's start */
        okey *worst = malloc(sizeof(okey) * n);
        for (uint32_t u = 0; u < n; u++) { worst[u].d = L[(size_t)u * K + K - 1].d; worst[u].id = L[(size_t)u * K + K - 1].v; }
        uint64_t cap = 1024, np = 0;
        orec *prop = malloc(sizeof(orec) * cap);
        for (uint32_t v = 0; v < n; v++) {
            uint32_t bn[64], bo[64], nb = 0, no = 0;
            for (uint32_t j = 0; j < S; j++) {
                uint32_t x = NS[(size_t)v * S + j];
                if (x != O_INVALID && !in_list(bn, nb, x)) bn[nb++] = x;
                x = RN[(size_t)v * S + j];
                if (x != O_INVALID && !in_list(bn, nb, x)) bn[nb++] = x;
            }
            for (uint32_t j = 0; j < S; j++) {
                uint32_t x = OS[(size_t)v * S + j];
                if (x != O_INVALID && !in_list(bn, nb, x) && !in_list(bo, no, x)) bo[no++] = x;
                x = RO[(size_t)v * S + j];
                if (x != O_INVALID && !in_list(bn, nb, x) && !in_list(bo, no, x)) bo[no++] = x;
            }
            for (uint32_t i = 0; i < nb; i++) {
                for (uint32_t j = 0; j < nb + no; j++) {
                    if (j < nb && j <= i) continue;             /* unordered pairs within Bn */
                    uint32_t a = bn[i], b = j < nb ? bn[j] : bo[j - nb];
                    float d = dist_ids(h, ids[a], ids[b]);
                    okey kb = { d, b }, ka = { d, a };
                    if (np + 2 > cap) { cap *= 2; prop = realloc(prop, sizeof(orec) * cap); }
                    if (key_less(kb, worst[a])) { orec r = { a, b, d }; prop[np++] = r; }
                    if (key_less(ka, worst[b])) { orec r = { b, a, d }; prop[np++] = r; }
                }
            }
        }
        free(worst);
        /* 4. merge, per node, its list with its proposals in (Dist, id) order */
        qsort(prop, np, sizeof(orec), rec_cmp);
        uint64_t k0 = 0;
        oent *m = malloc(sizeof(oent) * 2 * K);
        while (k0 < np) {
            uint64_t k1 = k0;
            while (k1 < np && prop[k1].t == prop[k0].t) k1++;
            oent *l = L + (size_t)prop[k0].t * K;
            uint32_t nm = 0, i = 0;
            uint64_t k = k0;
            while (nm < K && (i < K || k < k1)) {
                oent c;
                oent pk = { k < k1 ? prop[k].d : 0.0f, k < k1 ? prop[k].s : 0u, 1 };
                if (k >= k1 || (i < K && !ent_less(&pk, &l[i]))) c = l[i++];   /* ties: the entry first */
                else { c = pk; k++; }
                if (nm > 0 && m[nm - 1].d == c.d && m[nm - 1].v == c.v) continue;  /* a repeat: the earlier stays */
                m[nm++] = c;
            }
            memcpy(l, m, sizeof(oent) * K);
            k0 = k1;
        }
        free(m);
        free(prop);
    }
    free(NS); free(OS); free(RN); free(RO); free(rn); free(ro);
}

/* Rank-based pruning of the K-lists `lists` (positions, each ascending) to
 * P (n x R): per node, the R entries with the fewest detourable routes,
 * ascending by (routes, rank). */
static void rank_prune(const uint32_t *lists, uint32_t n, uint32_t K, uint32_t R, uint32_t *P, int nt) {
    #pragma omp parallel num_threads(nt)
    {
        uint32_t *rank = malloc(sizeof(uint32_t) * n);
        for (uint32_t i = 0; i < n; i++) rank[i] = O_INVALID;
        okey *cnt = malloc(sizeof(okey) * K);   /* (routes, rank) */
        #pragma omp for schedule(dynamic, 64)
        for (uint32_t u = 0; u < n; u++) {
            const uint32_t *l = lists + (size_t)u * K;
            for (uint32_t r = 0; r < K; r++) rank[l[r]] = r;
            uint32_t routes[128] = { 0 };
            for (uint32_t rz = 0; rz < K; rz++) {
                const uint32_t *lz = lists + (size_t)l[rz] * K;
                for (uint32_t rzy = 0; rzy < K; rzy++) {
                    uint32_t ry = rank[lz[rzy]];
                    if (ry != O_INVALID && rz < ry && rzy < ry) routes[ry]++;
                }
            }
            for (uint32_t r = 0; r < K; r++) { cnt[r].d = (float)routes[r]; cnt[r].id = r; }
            qsort(cnt, K, sizeof(okey), okey_cmp_u);
            for (uint32_t t = 0; t < R; t++) P[(size_t)u * R + t] = l[cnt[t].id];
            for (uint32_t r = 0; r < K; r++) rank[l[r]] = O_INVALID;
        }
        free(rank); free(cnt);
    }
}

/* Reverse edges merged into the pruned lists P (n x R) -> out (n x R, with
 * the list lengths in nout). */
static void reverse_merge(const uint32_t *P, uint32_t n, uint32_t R, uint32_t *out, uint32_t *nout, int nt) {
    orec *rv = malloc(sizeof(orec) * ((size_t)n * R + 1));
    uint64_t nrv = 0;
    for (uint32_t u = 0; u < n; u++)
        for (uint32_t t = 0; t < R; t++) { orec r = { P[(size_t)u * R + t], u, (float)t }; rv[nrv++] = r; }
    qsort(rv, nrv, sizeof(orec), rec_cmp);          /* (target, position, source) */
    uint64_t *rs = calloc((size_t)n + 1, sizeof(uint64_t));
    for (uint64_t k = 0; k < nrv; k++) rs[rv[k].t + 1]++;
    for (uint32_t t = 0; t < n; t++) rs[t + 1] += rs[t];
    const uint32_t half = R / 2;
    #pragma omp parallel for schedule(static) num_threads(nt)
    for (uint32_t y = 0; y < n; y++) {
        uint32_t *o = out + (size_t)y * R, no = 0;
        const uint32_t *py = P + (size_t)y * R;
        for (uint32_t t = 0; t < half; t++) o[no++] = py[t];
        for (uint64_t k = rs[y]; k < rs[y + 1] && no < R; k++)
            if (!in_list(o, no, rv[k].s)) o[no++] = rv[k].s;
        for (uint32_t t = half; t < R && no < R; t++)
            if (!in_list(o, no, py[t])) o[no++] = py[t];
        nout[y] = no;
        for (uint32_t t = no; t < R; t++) o[t] = O_INVALID;
    }
    free(rv); free(rs);
}

static int check_init(oindex *h, const uint32_t *init, uint32_t n, uint32_t K) {
    for (uint32_t u = 0; u < n; u++)
        for (uint32_t j = 0; j < K; j++) {
            uint32_t v = init[(size_t)u * K + j];
            if (v >= n || v == u || in_list(init + (size_t)u * K, j, v)) {
                snprintf(h->err, sizeof h->err, "initial list of position %u is not K distinct other positions", u);
                return O_E_ARG;
            }
        }
    return O_OK;
}

int32_t oracle_build_cagra(void *hv, const void *vecs, const uint32_t *ids, uint32_t n, const uint32_t *init,
                           uint32_t K, uint32_t iters, uint32_t S) {
    oindex *h = hv;
    const uint32_t R = h->cfg.R;
    if (h->cfg.algo != O_CAGRA) { snprintf(h->err, sizeof h->err, "graph construction is for the CAGRA variant"); return O_E_ARG; }
    if (h->n_active != 0) { snprintf(h->err, sizeof h->err, "graph construction needs an empty index"); return O_E_ARG; }
    if (K < R || K > 128 || n <= K || S == 0 || S > 32) {
        snprintf(h->err, sizeof h->err, "need R <= K <= 128, K < n and 1 <= S <= 32");
        return O_E_ARG;
    }
    int rc = validate_ids(h, ids, n, 0);
    if (rc == O_OK) rc = validate_vectors(h, vecs, n, 0);
    if (rc == O_OK) rc = check_init(h, init, n, K);
    if (rc != O_OK) return rc;
    stage(h, vecs, ids, n);
    const int nt = nthreads(h);
    oent *L = malloc(sizeof(oent) * (size_t)n * K);
    nn_descent(h, ids, n, init, K, iters, S, L);
    uint32_t *lists = malloc(sizeof(uint32_t) * (size_t)n * K);
    for (size_t i = 0; i < (size_t)n * K; i++) lists[i] = L[i].v;
    free(L);
    uint32_t *P = malloc(sizeof(uint32_t) * (size_t)n * R), *out = malloc(sizeof(uint32_t) * (size_t)n * R);
    uint32_t *nout = malloc(sizeof(uint32_t) * n);
    rank_prune(lists, n, K, R, P, nt);
    reverse_merge(P, n, R, out, nout, nt);
    for (uint32_t y = 0; y < n; y++) {
        uint32_t *row = h->adj + (size_t)ids[y] * R;
        for (uint32_t t = 0; t < R; t++) row[t] = t < nout[y] ? ids[out[(size_t)y * R + t]] : O_INVALID;
        h->deg[ids[y]] = nout[y];
    }
    free(lists); free(P); free(out); free(nout);
    h->medoid = compute_medoid(h);
    return O_OK;
}

/* The three steps on their own (positions, no index state changed). */
int32_t oracle_nn_descent(void *hv, const void *vecs, uint32_t n, const uint32_t *init, uint32_t K, uint32_t iters,
                          uint32_t S, uint32_t *out_ids, float *out_d) {
    oindex *h = hv;
    if (K == 0 || K > 128 || n <= K || S == 0 || S > 32 || n > h->cfg.capacity || h->n_active != 0) {
        snprintf(h->err, sizeof h->err, "bad NN-Descent arguments");
        return O_E_ARG;
    }
    if (check_init(h, init, n, K) != O_OK) return O_E_ARG;
    uint32_t *ids = malloc(sizeof(uint32_t) * n);
    for (uint32_t i = 0; i < n; i++) ids[i] = i;
    size_t row = (size_t)h->cfg.dim * h->esize;
    for (uint32_t i = 0; i < n; i++)
        store_row(h, (const uint8_t *)vecs + (size_t)i * row, h->vecs + (size_t)i * h->sdim * h->esize, 0);
    oent *L = malloc(sizeof(oent) * (size_t)n * K);
    nn_descent(h, ids, n, init, K, iters, S, L);
    for (size_t i = 0; i < (size_t)n * K; i++) { out_ids[i] = L[i].v; out_d[i] = L[i].d; }
    free(L); free(ids);
    return O_OK;
}
void oracle_rank_prune(const uint32_t *lists, uint32_t n, uint32_t K, uint32_t R, uint32_t *P) {
    rank_prune(lists, n, K, R, P, 1);
}
void oracle_reverse_merge(const uint32_t *P, uint32_t n, uint32_t R, uint32_t *out, uint32_t *nout) {
    reverse_merge(P, n, R, out, nout, 1);
}

int32_t oracle_search(void *hv, const void *queries, uint32_t nq, uint32_t k, uint32_t beam,
                      uint32_t *out_ids, float *out_d) {
    oindex *h = hv;
    h->err[0] = 0;
    if (k == 0 || beam == 0 || k > beam) { snprintf(h->err, sizeof h->err, "need 1 <= k <= beam"); return O_E_ARG; }
    if (nq == 0) return O_OK;
    if (validate_vectors(h, queries, nq, 1)) return O_E_ARG;
    size_t row = (size_t)h->cfg.dim * h->esize;
    uint64_t hops = 0, evals = 0;
    #pragma omp parallel for schedule(dynamic, 4) num_threads(nthreads(h)) reduction(+:hops, evals)
    for (uint32_t i = 0; i < nq; i++) {
        uint32_t got = 0;
        if (h->n_active > 0) {
            osearch s;
            uint8_t *qs = malloc((size_t)h->sdim * h->esize);
            store_row(h, (const uint8_t *)queries + (size_t)i * row, qs, 1);
            search_alloc(&s, beam, h->cfg.R, 2 * beam);
            beam_search(h, qs, h->medoid, beam, 2 * beam, &s);
            free(qs);
            for (; got < k && got < s.nC; got++) {
                out_ids[(size_t)i * k + got] = s.C[got].id;
                out_d[(size_t)i * k + got] = s.C[got].d;
            }
            hops += s.nV; evals += s.evals;
            search_free(&s);
        }
        for (; got < k; got++) { out_ids[(size_t)i * k + got] = O_INVALID; out_d[(size_t)i * k + got] = INFINITY; }
    }
    h->st.searches += nq; h->st.hops += hops; h->st.dist_evals += evals;
    return O_OK;
}

/* Export: lists (Vamana lists are sets and are returned with each row
 * ascending, INVALID last; CAGRA lists in slot order), degrees, active map,
 * medoid, and optionally the reverse CSR (offsets: capacity + 1 entries). */
static int u32_cmp(const void *pa, const void *pb) {
    uint32_t a = *(const uint32_t *)pa, b = *(const uint32_t *)pb;
    return a < b ? -1 : a > b ? 1 : 0;
}

int32_t oracle_export_graph(void *hv, uint32_t *adj, uint32_t *deg, uint8_t *active, uint32_t *medoid,
                            uint32_t *rev_offsets, uint32_t *rev_srcs, uint64_t *nnz) {
    oindex *h = hv;
    size_t cap = h->cfg.capacity;
    if (adj) {
        memcpy(adj, h->adj, cap * h->cfg.R * sizeof(uint32_t));
        if (h->cfg.algo == O_VAMANA)
            for (size_t u = 0; u < cap; u++) qsort(adj + u * h->cfg.R, h->cfg.R, sizeof(uint32_t), u32_cmp);
    }
    if (deg) memcpy(deg, h->deg, cap * sizeof(uint32_t));
    if (active) memcpy(active, h->active, cap);
    if (medoid) *medoid = h->medoid;
    if (rev_offsets) {
        uint64_t z = reverse_csr(h->adj, h->active, h->cfg.capacity, h->cfg.R, rev_offsets, rev_srcs);
        if (nnz) *nnz = z;
    }
    return O_OK;
}

/* Import a full state (vectors for every slot, lists, degrees, active map,
 * medoid).  Used by tests to set up hand-made graphs. */
int32_t oracle_import_graph(void *hv, const void *vecs, const uint32_t *adj, const uint32_t *deg,
                            const uint8_t *active, uint32_t medoid) {
    oindex *h = hv;
    size_t cap = h->cfg.capacity;
    const size_t row = (size_t)h->cfg.dim * h->esize;
    for (size_t i = 0; i < cap; i++)
        store_row(h, (const uint8_t *)vecs + i * row, h->vecs + i * h->sdim * h->esize, 0);
    memcpy(h->adj, adj, cap * h->cfg.R * sizeof(uint32_t));
    memcpy(h->deg, deg, cap * sizeof(uint32_t));
    memcpy(h->active, active, cap);
    h->medoid = medoid;
    h->n_active = 0;
    for (size_t i = 0; i < cap; i++) h->n_active += active[i] ? 1 : 0;
    return O_OK;
}

/* ---- pieces exposed for the pin tests ---------------------------------- */
/* Dist of two stored rows (sdim elements each). */
float oracle_dist(void *hv, const void *a, const void *b) { return dist_raw(hv, a, b); }

/* A caller row as stored (sdim elements): is_query selects the query form
 * of the MIPS augmentation.  Returns -1 for a norm above mips_norm. */
int32_t oracle_store_row(void *hv, const void *x, void *out, int32_t is_query) {
    return store_row(hv, x, out, is_query);
}

/* BeamSearch on the current state from start s; writes C (ids, dists) and V
 * (ids, dists); returns |C| and stores |V| in *nV. */
uint32_t oracle_beam_search(void *hv, const void *q, uint32_t s, uint32_t ell, uint32_t max_iters,
                            uint32_t *C_ids, float *C_d, uint32_t *V_ids, float *V_d, uint32_t *nV) {
    oindex *h = hv;
    osearch st;
    uint8_t *qs = malloc((size_t)h->sdim * h->esize);
    store_row(h, q, qs, 1);
    search_alloc(&st, ell, h->cfg.R, max_iters);
    beam_search(h, qs, s, ell, max_iters, &st);
    free(qs);
    for (uint32_t i = 0; i < st.nC; i++) { C_ids[i] = st.C[i].id; C_d[i] = st.C[i].d; }
    for (uint32_t i = 0; i < st.nV; i++) { V_ids[i] = st.V[i].id; V_d[i] = st.V[i].d; }
    *nV = st.nV;
    uint32_t nc = st.nC;
    search_free(&st);
    return nc;
}

/* GrANDRobustPrune of node p over explicit candidates with their D_p. */
uint32_t oracle_robust_prune(void *hv, uint32_t p, const uint32_t *ids, const float *D, uint32_t n,
                             uint32_t *L) {
    okey *cand = malloc(sizeof(okey) * (n + 1));
    for (uint32_t i = 0; i < n; i++) { cand[i].id = ids[i]; cand[i].d = D[i]; }
    uint64_t ev = 0;
    uint32_t nl = robust_prune(hv, p, cand, n, L, &ev);
    free(cand);
    return nl;
}

uint32_t oracle_medoid(void *hv) { return compute_medoid(hv); }

uint64_t oracle_reverse_csr(const uint32_t *adj, const uint8_t *active, uint32_t cap, uint32_t R,
                            uint32_t *offsets, uint32_t *srcs) {
    return reverse_csr(adj, active, cap, R, offsets, srcs);
}

/* Exact k nearest active neighbours by brute force (ground truth, the
 * recall@k definition of Section 5.5). */
int32_t oracle_bruteforce_knn(void *hv, const void *queries, uint32_t nq, uint32_t k,
                              uint32_t *out_ids, float *out_d) {
    oindex *h = hv;
    size_t row = (size_t)h->cfg.dim * h->esize;
    const uint32_t cap = h->cfg.capacity;
    #pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads(h))
    for (uint32_t i = 0; i < nq; i++) {
        uint8_t *q = malloc((size_t)h->sdim * h->esize);
        store_row(h, (const uint8_t *)queries + (size_t)i * row, q, 1);
        okey *best = malloc(sizeof(okey) * (k + 1));
        uint32_t nb = 0;
        for (uint32_t v = 0; v < cap; v++) {
            if (!h->active[v]) continue;
            okey key = { dist_raw(h, q, vec_of(h, v)), v };
            if (nb == k && !key_less(key, best[k - 1])) continue;
            uint32_t pos = nb < k ? nb++ : k - 1;
            while (pos > 0 && key_less(key, best[pos - 1])) { best[pos] = best[pos - 1]; pos--; }
            best[pos] = key;
        }
        for (uint32_t j = 0; j < k; j++) {
            out_ids[(size_t)i * k + j] = j < nb ? best[j].id : O_INVALID;
            out_d[(size_t)i * k + j] = j < nb ? best[j].d : INFINITY;
        }
        free(best);
        free(q);
    }
    return O_OK;
}
