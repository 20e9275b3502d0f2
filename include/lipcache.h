/*
 * lipcache.h - C ABI of the certified feature cache (LipCache) on gfx950.
 *
 * The library implements the certified cache path of "LipCache: A Local
 * Inference Proxy with Certified Caching for Edge Image Classification
 * Service": the spectral norm of the guard network's linear head, the
 * per-entry certified reuse radius, the batched strict-ball lookup with
 * nearest-hit selection, and the write-back of misses.
 *
 * Conventions shared by every entry point
 *  - Pointers are DEVICE pointers owned by the caller unless marked (host).
 *    The library allocates no device memory and retains no caller pointer:
 *    scratch memory is passed in as a workspace (`ws`, `ws_bytes`); each
 *    entry point has a *_workspace_bytes query.  `ws` must be 256-byte
 *    aligned.  Its only state outlives a call: the static workspace of
 *    lipcache_lookup_noalloc, and a 4 KiB pinned host buffer through which
 *    the synchronous calls read a few bytes back (allocated on first use,
 *    a slot per concurrent call); calls on different streams are
 *    independent.
 *  - Matrices are row-major and contiguous; a feature is one row of d
 *    elements.  Supported feature sizes: 32 <= d <= 1024, d % 32 == 0.
 *  - Arguments are validated on the host before any device work; a
 *    validation failure (LIPCACHE_EINVAL, LIPCACHE_EUNSUPPORTED,
 *    LIPCACHE_EWORKSPACE, LIPCACHE_ECAPACITY) writes nothing.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls marked
 *    (async) only enqueue work: outputs are valid once the stream reaches
 *    that point.  Calls marked (sync) block until their result is on the
 *    host.  A failing HIP call returns LIPCACHE_EHIP.
 *  - Inputs are assumed finite with |component| < 1e15.  A query holding a
 *    NaN misses; an entry whose radius is NaN or <= 0 is never a hit.
 */
#ifndef LIPCACHE_H
#define LIPCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LIPCACHE_ABI_VERSION 7

/* Same type as hipStream_t. */
typedef struct ihipStream_t* lipcache_stream_t;

typedef enum lipcache_status {
  LIPCACHE_OK = 0,
  LIPCACHE_EINVAL = 1,        /* invalid argument (null pointer, size, enum)          */
  LIPCACHE_EDEGENERATE = 2,   /* sigma_max(W) <= 0: construction stops (Alg. 1)        */
  LIPCACHE_ENOCONV = 3,       /* power iteration hit max_iters; sigma still written    */
  LIPCACHE_ECAPACITY = 4,     /* insert would exceed the cache capacity; nothing added */
  LIPCACHE_EUNSUPPORTED = 5,  /* valid request the library does not implement          */
  LIPCACHE_EWORKSPACE = 6,    /* workspace missing, too small or misaligned            */
  LIPCACHE_EHIP = 7           /* a HIP runtime call or kernel launch failed            */
} lipcache_status;

/* Element types.  Storage of cache features (store_dtype): F32 or BF16.
 * Matrix-core precision of the lookup's distance filter (precision): F16
 * (float16 operands, float32 accumulation) or F32. */
enum { LIPCACHE_F32 = 0, LIPCACHE_BF16 = 1, LIPCACHE_F16 = 2 };

/* Lookup option, ORed into `precision` (LIPCACHE_F16 | LIPCACHE_LOOKUP_PRUNE):
 * prefix pruning.  The squared distance over the first 32 features is a
 * lower bound of the full one (Eq. (13) sums non-negative terms), so a block
 * of query-entry pairs whose prefix filter (the same rigorous slack, with
 * the ball widened to r_i (1 + 3e-5) so that every pair of the boundary
 * band survives) rejects every pair cannot hold a hit or a band pair, and
 * the rest of its contraction is skipped.  Every output equals the lookup
 * without the option except stats[LIPCACHE_STAT_RECHECKED], which counts
 * fewer pairs the filter let through that were not hits.  Applies to the
 * float16 filter with 64 <= d <= 512 on caches of n >= 32768 rows with a
 * float16 image (other cases run the full contraction, with the same
 * answers); the workspace grows by about
 * 4 B + 4 n bytes (the entry thresholds padded to a multiple of 1024 rows). */
#define LIPCACHE_LOOKUP_PRUNE 0x100

/* Radius modes (policy component rho, Sec. 4.3): the conservative radius of
 * Eq. (21) or the tight per-pair radius of Remark 5.1, Eq. (29). */
enum { LIPCACHE_RADIUS_CONSERVATIVE = 0 /* Eq. (21) */, LIPCACHE_RADIUS_TIGHT = 1 /* Remark 5.1 */ };

/* Reuse boundaries compared with the certified radius (Sec. 6). */
enum {
  LIPCACHE_BOUNDARY_SCALED = 0,     /* factor * r_i (radius tightening)               */
  LIPCACHE_BOUNDARY_GLOBAL = 1,     /* one nearest-neighbour threshold for all        */
  LIPCACHE_BOUNDARY_INTERCLASS = 2  /* empirical: half the nearest class-mean gap     */
};

/* Cache selection strategies S of the offline construction (Alg. 1). */
enum {
  LIPCACHE_SELECT_RADIUS_DEDUP = 0, /* by decreasing radius, skipping duplicates  */
  LIPCACHE_SELECT_PRIORITY = 1,     /* by decreasing caller priority (random keys) */
  LIPCACHE_SELECT_KCENTER = 2       /* farthest-first traversal                   */
};

/* Label written for a query whose hit set is empty (falls back to MainNet,
 * Eq. (15)). */
#define LIPCACHE_MISS (-1)

/* Indices of the lookup statistics counters (uint64_t stats[4]). */
enum {
  LIPCACHE_STAT_HITS = 0,        /* queries with a non-empty hit set                   */
  LIPCACHE_STAT_RECHECKED = 1,   /* (query, entry) pairs the exact re-check evaluated  */
  LIPCACHE_STAT_BAND_PAIRS = 2,  /* re-checked pairs with |D - r| <= 1e-5 r            */
  LIPCACHE_STAT_BAND_QUERIES = 3 /* queries with at least one such pair                */
};

/*
 * The feature cache C = {(z_i, y~_i, r_i)} (Sec. 4.1; Alg. 2 input) with its
 * budget B_C (`capacity`, Alg. 1).  Struct-of-arrays, every device array
 * holds `capacity` rows, rows [0, n) are live.  The caller owns the arrays;
 * lipcache_insert writes rows and advances `n`.
 */
typedef struct lipcache_cache {
  void*    z;           /* [capacity][d] features; float (F32) or bf16 bits (BF16)   */
  void*    zimg;        /* [capacity][d] float16 image of the stored features for
                           the F16 distance filter, or NULL.  Insert keeps it
                           equal to f16(stored z) (round to nearest even after
                           clamping to +-65504).  The F16 lookup streams it (half
                           the bytes of an F32 store); without it each workgroup
                           converts z on the fly.                                   */
  float*   r;           /* [capacity] certified radius r_i                           */
  int32_t* label;       /* [capacity] payload y~_i                                   */
  float*   norm2;       /* [capacity] ||z_i||^2 of the stored values (derived)       */
  int64_t  n;           /* live rows; host-side value                                */
  int64_t  capacity;    /* rows allocated in each array                              */
  int32_t  d;           /* feature size                                              */
  int32_t  store_dtype; /* LIPCACHE_F32 or LIPCACHE_BF16                             */
} lipcache_cache;

/*
 * sigma_max(W), the spectral norm of the head f(z) = W z + b (Sec. 5.1,
 * Eq. (18)): the Lipschitz constant every certificate divides by.  Alg. 1
 * computes it before certifying any candidate and stops when it is <= 0.
 *
 * Power iteration in float64 on the Gram matrix of W (W W^T when C <= d,
 * else W^T W; same non-zero spectrum): v <- G v / ||G v||, with the estimate
 * sigma_k = sqrt(v_k^T G v_k) (= ||W v_k|| for unit v_k).  Stops after two
 * consecutive iterations with |sigma_k - sigma_{k-1}| <= rel_tol sigma_k.
 *
 *  W          [C][d] float head, C >= 1, 1 <= d, min(C, d) <= 1024
 *  max_iters  >= 1
 *  rel_tol    > 0 (1e-13 gives sigma to about 1e-12 relative)
 *  sigma      (host) out: the estimate, written on OK, ENOCONV and EDEGENERATE
 *  iterations (host, nullable) out: iterations run
 *  ws         lipcache_spectral_norm_workspace_bytes(C, d) bytes
 * Returns OK, ENOCONV (max_iters reached), EDEGENERATE (sigma <= 0). (sync)
 */
lipcache_status lipcache_spectral_norm(const float* W, int32_t C, int32_t d,
                                       int32_t max_iters, double rel_tol,
                                       double* sigma, int32_t* iterations,
                                       void* ws, size_t ws_bytes,
                                       lipcache_stream_t stream);
size_t lipcache_spectral_norm_workspace_bytes(int32_t C, int32_t d);

/*
 * Certification of N candidate features (Sec. 4.3, Alg. 1; Sec. 5.2).
 * For every row z_i (rounded to bf16, ties to even, first when store_dtype
 * is BF16: the stored centre is what is certified):
 *   logits s = W z_i + b accumulated in float64 (Eq. (5)),
 *   label y_i = argmax_c s_c, lowest index on ties (Eq. (6)),
 *   margin m_i = s_y - max_{j != y} s_j (Eq. (20)),
 *   radius r_i = m_i / (sigma sqrt 2) (Eq. (21)) in float64,
 *   or with LIPCACHE_RADIUS_TIGHT the per-pair radius of Remark 5.1,
 *   r*_i = min_{j != y} (s_y - s_j) / ||W_y - W_j||_2 (float64),
 *   where a class with W_j = W_y sets no finite constraint (r*_i = +inf when
 *   no class does).  r*_i >= r_i.  The radius is stored rounded toward
 *   zero, so the float32 ball never reaches past the certified one.
 * A radius <= 0 (a tie) marks a candidate that must be discarded (Alg. 1).
 *
 *  z [N][d] float; W [C][d] float, C >= 2; b [C] float or NULL (= 0)
 *  sigma       > 0, normally lipcache_spectral_norm's result (used by the
 *              conservative radius only, but validated in both modes)
 *  radius_mode LIPCACHE_RADIUS_CONSERVATIVE or LIPCACHE_RADIUS_TIGHT; the
 *              tight mode needs a C x C float64 table of row distances in
 *              the workspace, and evaluates the logits a second time only
 *              for the rows whose minimum its first pass cannot prove
 *  label_out [N] int32, r_out [N] float (required)
 *  margin_out [N] float, norm2_out [N] float (nullable): m_i and ||z_i||^2
 *  ws          lipcache_certify_workspace_bytes(C, d, radius_mode) bytes
 * N = 0 is valid and does nothing. (async)
 */
lipcache_status lipcache_certify(const float* z, int64_t N, int32_t d,
                                 const float* W, const float* b, int32_t C,
                                 double sigma, int32_t radius_mode,
                                 int32_t store_dtype, int32_t* label_out,
                                 float* r_out, float* margin_out,
                                 float* norm2_out, void* ws, size_t ws_bytes,
                                 lipcache_stream_t stream);
size_t lipcache_certify_workspace_bytes(int32_t C, int32_t d, int32_t radius_mode);

/*
 * Batched certified lookup (Sec. 4.4, Eq. (13)-(15); Alg. 2).  For every
 * query q the hit set is H(q) = {i < n : ||q - z_i||_2 < r_i} (strict) and
 * the answer is the nearest hit i* (least distance, lowest index among equal
 * float32-rounded distances) with its payload, or a miss.
 *
 * Distances are filtered on the matrix cores (float16 or float32 MFMA) with
 * a rigorous error slack, so no true hit is ever dropped; every surviving
 * pair is re-checked as sum_k (q_k - z_ik)^2 in float64, which decides the
 * hit.
 *
 *  c          cache (host struct; its arrays on the device), n >= 0
 *  zq         [B][c->d] float queries, B >= 0
 *  precision  LIPCACHE_F16 or LIPCACHE_F32 (F32 requires d <= 512), either
 *             optionally | LIPCACHE_LOOKUP_PRUNE
 *  label_out  [B] int32: y~_{i*}, or LIPCACHE_MISS (required)
 *  index_out  [B] int64: i*, or -1 (nullable)
 *  dist2_out  [B] float: ||q - z_{i*}||^2 rounded to nearest, +inf on a miss (nullable)
 *  stats      [4] uint64 counters, see LIPCACHE_STAT_* (nullable; overwritten)
 *  band_flag  [B] uint8: 1 if a re-checked pair of the query lies within
 *             relative 1e-5 of its ball boundary (nullable)
 *  ws         lipcache_lookup_workspace_bytes(B, n, d, precision) bytes
 * (async)
 */
lipcache_status lipcache_lookup(const lipcache_cache* c, const float* zq, int64_t B,
                                int32_t precision, int32_t* label_out,
                                int64_t* index_out, float* dist2_out,
                                uint64_t* stats, uint8_t* band_flag,
                                void* ws, size_t ws_bytes, lipcache_stream_t stream);
size_t lipcache_lookup_workspace_bytes(int64_t B, int64_t N, int32_t d, int32_t precision);

/* 1 if lipcache_lookup(c, ..., precision, ...) takes the pruned path of
 * LIPCACHE_LOOKUP_PRUNE for this cache (float16 filter with a float16
 * image, 64 <= d <= 512, n >= 32768), 0 if it runs the full contraction
 * (always the case without the option, or for an invalid argument).  Host
 * only. */
int32_t lipcache_lookup_prunes(const lipcache_cache* c, int32_t precision);

/*
 * lipcache_lookup for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same arguments and results as lipcache_lookup without `ws`/`ws_bytes`.
 * The workspace is a static device array of LIPCACHE_NOALLOC_SCRATCH_BYTES
 * (32 MiB) per GPU, held until the process ends; the call allocates nothing.
 * It serves lookups with lipcache_lookup_workspace_bytes(B, c->n, c->d,
 * precision) <= LIPCACHE_NOALLOC_SCRATCH_BYTES (e.g. B = 65,536 queries
 * against 4.5M entries) and returns LIPCACHE_EWORKSPACE, with nothing
 * written, for larger ones.  Every call on one GPU uses that GPU's array:
 * calls that overlap on one GPU (other streams or host threads) race, so
 * serialise them.  (async)
 */
#define LIPCACHE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
lipcache_status lipcache_lookup_noalloc(const lipcache_cache* c, const float* zq, int64_t B,
                                        int32_t precision, int32_t* label_out,
                                        int64_t* index_out, float* dist2_out,
                                        uint64_t* stats, uint8_t* band_flag,
                                        lipcache_stream_t stream);

/*
 * Write-back (Sec. 4.4, Alg. 2; construction, Alg. 1): append, in ascending
 * row order, every row j of z_src with r_src[j] > 0 and (miss_selector ==
 * NULL or miss_selector[j] == LIPCACHE_MISS).  The feature is stored in the
 * cache's dtype (bf16 rounded to nearest even), with its label, radius and
 * the squared norm of the stored values.  All-or-nothing: when the selected
 * rows do not fit into capacity - n, returns ECAPACITY and appends nothing.
 *
 *  c              cache; c->n is advanced by the rows appended
 *  z_src [k][c->d] float, 16-byte aligned; label_src [k] int32,
 *                 r_src [k] float (required); c->z must be 16-byte and
 *                 c->zimg 8-byte aligned (rows move as 16-byte vectors)
 *  miss_selector  [k] int32 or NULL (e.g. lipcache_lookup's label_out)
 *  inserted       (host, nullable) out: rows appended
 *  ws             lipcache_insert_workspace_bytes(k) bytes
 * (sync: one device-to-host read of the selected count)
 */
lipcache_status lipcache_insert(lipcache_cache* c, const float* z_src,
                                const int32_t* label_src, const float* r_src,
                                const int32_t* miss_selector, int64_t k,
                                int64_t* inserted, void* ws, size_t ws_bytes,
                                lipcache_stream_t stream);
size_t lipcache_insert_workspace_bytes(int64_t k);

/*
 * Offline construction of the feature store (Sec. 4.3, Alg. 1): select at
 * most `budget` of N candidates (z_i, label_i, r_i) and append them to the
 * cache.  r_i and label_i normally come from lipcache_certify (payload =
 * proxy label) or carry another payload source.  A candidate is eligible
 * when r_i > 0, guard_label_i == label_i if guard_label is given (the
 * cache-centre label-consistency flag), its priority is not NaN, and, with
 * a per-class budget, 0 <= label_i < n_classes.  Distances are exact
 * (float64) over the stored values (bf16-rounded for a bf16 store).
 *
 *  strategy LIPCACHE_SELECT_RADIUS_DEDUP: visit eligible candidates by
 *           decreasing r_i (ties: lower index); skip one whose class already
 *           holds per_class entries; skip a duplicate - a candidate strictly
 *           inside the ball ||z_i - z_j|| < r_j of an entry already in the
 *           cache (present before the call or appended earlier in it);
 *           append the rest in visit order until `budget` are appended.
 *           LIPCACHE_SELECT_PRIORITY: the same visit by decreasing
 *           priority_i, with no duplicate test (random keys give the random
 *           strategy; the caller draws them).
 *           LIPCACHE_SELECT_KCENTER: farthest-first traversal - start at the
 *           largest-radius eligible candidate (ties: lower index), then
 *           repeatedly append the candidate whose squared distance to the
 *           nearest chosen one is largest (ties: lower index).  With a
 *           per-class budget each class 0 .. n_classes-1 is traversed on its
 *           own, in that order; entries present before the call are not used.
 *  z [N][c->d] float, 16-byte aligned; label [N] int32; r [N] float
 *  guard_label [N] int32 or NULL; priority [N] float (PRIORITY only, else
 *           ignored)
 *  budget   maximum rows to append; < 0 means the free capacity; more than
 *           the free capacity returns ECAPACITY (nothing appended)
 *  per_class, n_classes  per-label budget (0 = none) and label range
 *           (1 <= n_classes <= 16384 when per_class > 0)
 *  selected_out [budget] int64 or NULL: candidate indices in append order
 *  appended (host, nullable) out: rows appended; c->n advances by it
 *  ws       lipcache_construct_workspace_bytes(c, N, n_classes, budget)
 *           bytes (depends on the cache's capacity and d)
 * (sync: the host drives the visit in chunks of 1024 candidates)
 */
lipcache_status lipcache_construct(lipcache_cache* c, const float* z, const int32_t* label,
                                   const float* r, const int32_t* guard_label,
                                   const float* priority, int64_t N, int32_t strategy,
                                   int64_t budget, int32_t per_class, int32_t n_classes,
                                   int64_t* selected_out, int64_t* appended,
                                   void* ws, size_t ws_bytes, lipcache_stream_t stream);
size_t lipcache_construct_workspace_bytes(const lipcache_cache* c, int64_t N, int32_t n_classes,
                                          int64_t budget);

/*
 * Exact cluster index for a sublinear lookup (the paper points to an exact
 * sublinear index for large caches).  Rows 0 .. n_indexed-1 of a cache are
 * partitioned into K clusters (a few Lloyd iterations of k-means from
 * evenly spaced rows, on an evenly strided sample of about 512 rows per
 * cluster, then one assignment of every row); entry i of cluster c can
 * contain a query q only if
 * ||q - mu_c|| < R_c with R_c >= max over its live members of
 * (||z_i - mu_c|| + r_i) (triangle inequality), so the indexed lookup scans
 * only the clusters a query may need and returns exactly what
 * lipcache_lookup returns.  Rows appended after the build are scanned in
 * full.  All arrays are caller-owned device memory.
 */
typedef struct lipcache_index {
  lipcache_cache sorted; /* the indexed rows in cluster order (same d and store_dtype as the
                            cache, capacity >= n_indexed; zimg as for a cache)               */
  int64_t* perm;         /* [n_indexed] cache row held by sorted row j                       */
  int64_t* offsets;      /* [K + 1] cluster c = sorted rows [offsets[c], offsets[c + 1])     */
  float* centers;        /* [K][d] cluster centres mu_c (16-byte aligned)                    */
  float* bound;          /* [K] R_c, rounded up; -inf when no member can be hit              */
  int32_t K;
  int64_t n_indexed;     /* rows of the cache covered (the cache's n at build time)          */
} lipcache_index;

/*
 * Build an index over rows 0 .. c->n-1 (K clusters, `iters` Lloyd
 * iterations; 1 <= K <= 65536, K <= c->n).  Sets idx->K, idx->n_indexed and
 * idx->sorted.n; the arrays of idx must be allocated by the caller.
 * c->z, idx->sorted.z, idx->sorted.zimg and idx->centers must be 16-byte
 * aligned and c->zimg 8-byte aligned (LIPCACHE_EINVAL otherwise).
 *  ws lipcache_index_build_workspace_bytes(c->n, c->d, K) bytes
 * (async)
 */
lipcache_status lipcache_index_build(const lipcache_cache* c, int32_t K, int32_t iters,
                                     lipcache_index* idx, void* ws, size_t ws_bytes,
                                     lipcache_stream_t stream);
size_t lipcache_index_build_workspace_bytes(int64_t n, int32_t d, int32_t K);

/*
 * lipcache_lookup through an index built on this cache: the same label,
 * index into the cache, d^2 and band flags as lipcache_lookup on the same
 * cache, and the same stats except LIPCACHE_STAT_RECHECKED, which counts the
 * indexed scan's re-checks.  pairs (host, nullable) out: query-entry pairs
 * the filter scanned (B * c->n for the dense lookup).  Rows 0 .. n_indexed-1
 * of the cache must be the ones the index was built on; rows appended since
 * are scanned in full.  zq 16-byte aligned.
 *  ws lipcache_lookup_indexed_workspace_bytes(B, c->n, c->d, idx->K,
 *     idx->n_indexed) bytes
 * (sync: one read-back of the work-list size)
 */
lipcache_status lipcache_lookup_indexed(const lipcache_cache* c, const lipcache_index* idx,
                                        const float* zq, int64_t B, int32_t precision,
                                        int32_t* label_out, int64_t* index_out, float* dist2_out,
                                        uint64_t* stats, uint8_t* band_flag, int64_t* pairs,
                                        void* ws, size_t ws_bytes, lipcache_stream_t stream);
size_t lipcache_lookup_indexed_workspace_bytes(int64_t B, int64_t n, int32_t d, int32_t K,
                                               int64_t n_indexed);

/*
 * Reuse boundaries for the comparison of Sec. 6: a radius per cache entry,
 * written to r_out [c->n] float, for use with lipcache_lookup on a copy of
 * the cache descriptor whose `r` points at r_out (features, labels and
 * norms are shared).  Entries whose certified radius c->r[i] is not
 * positive get 0.
 *  mode LIPCACHE_BOUNDARY_SCALED: factor * r_i (0 <= factor; factor <= 1 is
 *       the paper's radius tightening and keeps every hit certified)
 *       LIPCACHE_BOUNDARY_GLOBAL: factor for every live entry (a global
 *       nearest-neighbour threshold tau: the nearest entry within tau is
 *       reused)
 *       LIPCACHE_BOUNDARY_INTERCLASS: factor * 1/2 * min over other labels o
 *       of ||mu_{y_i} - mu_o||, mu_c = mean of the live cached features of
 *       label c (float64); +inf when no other label is cached.  Labels must
 *       lie in [0, n_classes) (1 <= n_classes <= 65536); an entry outside
 *       gets 0 and is left out of the means.
 *  ws   lipcache_boundary_radius_workspace_bytes(c->d, n_classes) bytes
 *       (INTERCLASS only; may be NULL otherwise)
 * (async)
 */
lipcache_status lipcache_boundary_radius(const lipcache_cache* c, int32_t mode, double factor,
                                         int32_t n_classes, float* r_out, void* ws, size_t ws_bytes,
                                         lipcache_stream_t stream);
size_t lipcache_boundary_radius_workspace_bytes(int32_t d, int32_t n_classes);

/*
 * Certified-consistency count (Sec. 6): counts[0] = hits (lookup_label !=
 * LIPCACHE_MISS), counts[1] = hits whose label equals head_label, the
 * head's argmax at the same query (e.g. lipcache_certify's label_out for
 * the queries).  The consistency rate is counts[1] / counts[0].
 *  lookup_label [B], head_label [B] int32; counts [2] uint64 (device)
 * (async)
 */
lipcache_status lipcache_consistency(const int32_t* lookup_label, const int32_t* head_label, int64_t B,
                                     uint64_t* counts, lipcache_stream_t stream);

/*
 * Diagnostic view of the lookup's distance filter for small problems.  For
 * every pair (q, i < n) writes the matrix-core dot product g_hat = q . z_i
 * as the lookup kernel computes it, and cand = 1 if the pair passes the
 * filter (and is re-checked by lipcache_lookup), else 0.  Where the bf16
 * filter starts its accumulators at -Q_q (d <= 128 with a bf16 image or
 * store), g_hat is that accumulator plus Q_q in float32; cand is always the
 * kernel's own decision.
 *
 *  g_hat [B][n] float, cand [B][n] uint8 (required); B * n <= 2^26
 *  ws    lipcache_lookup_workspace_bytes(B, n, d, precision) bytes
 * (async)
 */
lipcache_status lipcache_lookup_filter_dump(const lipcache_cache* c, const float* zq,
                                            int64_t B, int32_t precision,
                                            float* g_hat, uint8_t* cand,
                                            void* ws, size_t ws_bytes,
                                            lipcache_stream_t stream);

/* Static description of a status code. */
const char* lipcache_status_string(lipcache_status status);

/* LIPCACHE_ABI_VERSION of the built library. */
int32_t lipcache_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LIPCACHE_H */
