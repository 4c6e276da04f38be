/*
 * nv.h -- C ABI of the approximate-caching cache-hit generation path on MI355X.
 *
 * Method (Agarwal et al., "Approximate Caching for Efficiently Serving
 * Diffusion Models"): a request's prompt embedding is matched against the
 * cached prompt embeddings (Sec. 4.3, Alg. 1); the best cosine similarity is
 * mapped to a skip count K by the cache selector (Sec. 5.3.1); the matched
 * entry's intermediate latent after K denoising steps is fetched
 * (Sec. 5.3, storage) and the remaining N - K guided DDIM steps of the
 * latent-diffusion UNet are run for the new prompt (Sec. 4.1, Sec. 2.1, Sec. 6).
 *
 * Conventions shared by every entry point:
 *   - Every tensor pointer is a DEVICE pointer unless its comment says "host".
 *     The caller owns all buffers; the library never frees caller memory.
 *     Only nv_unet_create allocates (weights), released by nv_unet_destroy.
 *   - Work is enqueued on `stream` (a hipStream_t, NULL = default stream) and
 *     is asynchronous unless stated.  Host arrays are read before return.
 *   - Validation failures return synchronously before any launch and leave
 *     outputs untouched.  nv_last_error() gives a message for the last
 *     failing call on the calling thread.
 *   - Handles are not thread-safe: concurrent calls on one nv_unet, or calls
 *     sharing a workspace, race.
 */
#ifndef NV_H
#define NV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NV_OK = 0,
  NV_ERR_INVALID_ARG = -1,   /* null pointer, bad size, bad table, K out of range */
  NV_ERR_UNSUPPORTED = -2,   /* legal but not implemented (e.g. d % 8 != 0) */
  NV_ERR_OUT_OF_MEMORY = -3, /* device allocation failed (nv_unet_create only) */
  NV_ERR_HIP = -4,           /* a HIP runtime call or kernel launch failed */
  NV_ERR_WORKSPACE = -5      /* workspace pointer null or smaller than required */
} nv_status;

typedef enum { NV_F32 = 0, NV_BF16 = 1 } nv_dtype;

/* Text for a status code.  Never NULL. */
const char* nv_status_string(int32_t status);
/* Detail of the last error on this thread ("" if none).  Never NULL. */
const char* nv_last_error(void);
/* Library version string. */
const char* nv_version(void);

/* ------------------------------------------------------------------------ *
 * Cache lookup + cache selector (Sec. 4.3 Alg. 1 search and K choice;
 * Sec. 5.3.1 selector table).
 *
 * For each query q_j (float32 [m][d], row-major) and cache row c_i
 * ([n][d] row-major, float32 or bfloat16), the canonical similarity is the
 * float64 sum of (double)q_jk * (double)c_ik over k = 0..d-1 taken strictly
 * left to right (every product is exact in float64).  The result is
 *   idx_out[j] = lowest i with the maximal canonical similarity,
 *   sim_out[j] = that similarity rounded to float32 (nearest even),
 *   k_out[j]   = k_values[t] for the first t with sim_out[j] > thresholds[t]
 *                (float32 compare, strict), or 0 when none does.
 * These outputs are exact, not approximate: a reduced-precision scan (bf16
 * matrix cores) keeps every row within a proven error margin of the best
 * and only those rows are rescored canonically.
 * n == 0 is legal: idx = -1, sim = -inf, K = 0 (the "no suitable cache" branch).
 *
 * Arguments: queries device f32 [m][d]; cache device [n][d] of c_dtype;
 * thresholds/k_values HOST arrays of length J (1..16), thresholds finite and
 * strictly descending, k_values >= 0; idx_out device int64 [m], sim_out
 * device f32 [m], k_out device int32 [m].  Limits: 1 <= m <= 4096,
 * 0 <= n < 2^31, 1 <= d <= 4096; d % 8 != 0 or d > 2048 gives NV_ERR_UNSUPPORTED.
 * workspace: device, >= nv_cache_lookup_workspace(m, n, d) bytes, 256-byte
 * aligned, contents need not be initialised.
 * ------------------------------------------------------------------------ */
size_t nv_cache_lookup_workspace(int32_t m, int64_t n, int32_t d);
int32_t nv_cache_lookup(const float* queries, int32_t m, const void* cache, int32_t c_dtype,
                        int64_t n, int32_t d, const float* thresholds, const int32_t* k_values,
                        int32_t J, int64_t* idx_out, float* sim_out, int32_t* k_out,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Capacity of the scratch array behind nv_cache_lookup_static (64 MiB per GPU). */
#define NV_LOOKUP_STATIC_BYTES ((size_t)64 << 20)

/* nv_cache_lookup_static: nv_cache_lookup without a workspace, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  It allocates nothing: its
 * scratch is a device array of NV_LOOKUP_STATIC_BYTES inside the library, one
 * copy per GPU (the device current at the call), held until the process ends.
 * Arguments, results and errors are those of nv_cache_lookup, plus
 * NV_ERR_UNSUPPORTED (before any launch) when the lookup needs more scratch
 * than the array holds; it needs at most nv_cache_lookup_workspace(m, n, d)
 * bytes: with d = 768, 8 queries fit up to 85M rows and 256 queries up to
 * 4.1M.  Every call on one GPU shares the array and leaves its scratch
 * behind (the next call initialises what it reads): calls in stream order are
 * safe, calls that overlap on one GPU (unordered streams) race. */
int32_t nv_cache_lookup_static(const float* queries, int32_t m, const void* cache,
                               int32_t c_dtype, int64_t n, int32_t d, const float* thresholds,
                               const int32_t* k_values, int32_t J, int64_t* idx_out,
                               float* sim_out, int32_t* k_out, void* stream);

/* ------------------------------------------------------------------------ *
 * State fetch (Sec. 5.3 storage; Alg. 1 retrieval of the state after step K).
 *
 * store: device f32 [n_store][n_slots][latent_elems]; slot s holds the
 * state after slot_k[s] steps (slot_k HOST int32 [n_slots], each > 0).
 * payload: device int32 [n_rows] mapping a cache row to its store entry
 * (NULL = identity, n_store >= n_rows).  idx, k: device [B] (lookup outputs).
 * noise: device f32 [B][latent_elems], used for samples with K = 0.
 * out[b] = store[payload[idx[b]]][slot of k[b]] when k[b] > 0, else noise[b].
 * A sample whose K has no slot, or whose idx/payload is out of range, gets
 * noise[b] and its k is rewritten to 0 in k (device, in place), so the
 * caller's later nv_denoise runs it from scratch.
 * ------------------------------------------------------------------------ */
/* Cache insertion after a miss: rows (device f32 [m][d], finite) become
 * cache rows n .. n+m-1 of cache (device [capacity][d] of c_dtype; bf16 rows
 * are rounded to nearest even), and payload[n + i] = entry[i] (device int32
 * [capacity] and [m]; both NULL to leave the payload alone).  The caller
 * owns n and capacity and passes n + m as the new row count afterwards.
 * Errors: NV_ERR_INVALID_ARG for null rows / cache, m < 1, d < 1, n < 0,
 * n + m > capacity, a bad c_dtype, or only one of entry / payload. */
int32_t nv_cache_insert(const float* rows, int32_t m, int32_t d, void* cache, int32_t c_dtype,
                        int64_t n, int64_t capacity, const int32_t* entry, int32_t* payload,
                        void* stream);

int32_t nv_gather_states(const float* store, int64_t n_store, int32_t n_slots,
                         const int32_t* slot_k, const int32_t* payload, int64_t n_rows,
                         const int64_t* idx, int32_t* k, const float* noise, int32_t B,
                         int64_t latent_elems, float* out, void* stream);

/* ------------------------------------------------------------------------ *
 * Maintained cache (Sec. 5.4: LCBFU eviction, holes, dropping prompts).
 *
 * States live in a pool: device f32 [n_pool][latent_elems].  The table,
 * device int32 [n_entries][n_slots], names for prompt (entry) e the pool
 * state saved after slot_k[s] steps, or -1 for a hole.  payload (device
 * int32 [n_rows], NULL = identity) maps a vector-DB row to its entry.
 *
 * nv_gather_pool: the hole-aware fetch.  For sample b with match idx[b] and
 * selector K k[b], the state served is the one with the largest slot_k[s]
 * <= k[b] whose table entry is in [0, n_pool); out[b] is that pool state and
 * k[b] (device, in place) becomes its slot_k[s].  No such state (or
 * k[b] <= 0, or idx / payload out of range): out[b] = noise[b], k[b] = 0.
 * latent_elems a multiple of 4; pool, noise, out 16-byte aligned.
 *
 * nv_table_update: rec (device int32 [u][1 + n_slots]) holds an entry id
 * then its new table row; rows with an id outside [0, n_entries) are
 * ignored.  Ids must be distinct within one call.
 *
 * nv_cache_move_rows: row src[i] of the cache (device [n][d] of c_dtype)
 * and payload[src[i]] (payload may be NULL) move to dst[i], for i < count
 * (src, dst device int64 [count]); pairs outside [0, n) are ignored.  The
 * dst values must be distinct and none may equal any src (the maintainer's
 * compaction plan meets this: every dst is below every src).  d even.
 *
 * nv_denoise_store_pool: nv_denoise_store with the destinations given per
 * state: dst HOST int32 [B][n_slots], pool index or -1 (not stored); the
 * state of sample b after slot_k[s] steps goes to pool[dst[b][s]].  Each
 * pool index may appear once.
 * ------------------------------------------------------------------------ */
int32_t nv_gather_pool(const float* pool, int64_t n_pool, const int32_t* table,
                       int64_t n_entries, int32_t n_slots, const int32_t* slot_k,
                       const int32_t* payload, int64_t n_rows, const int64_t* idx, int32_t* k,
                       const float* noise, int32_t B, int64_t latent_elems, float* out,
                       void* stream);
int32_t nv_table_update(int32_t* table, int64_t n_entries, int32_t n_slots, const int32_t* rec,
                        int32_t u, void* stream);
int32_t nv_cache_move_rows(void* cache, int32_t c_dtype, int64_t n, int32_t d, int32_t* payload,
                           const int64_t* src, const int64_t* dst, int32_t count, void* stream);

/* LCBFU maintainer (host only; no GPU work).  Each stored state has the
 * score f * K: f counts the requests served from it, starting at 1 when it
 * is stored; K is its slot's step count.  Equal scores go to the state
 * stored first.
 *
 * nv_lcbfu_create: slot_k HOST int32 [n_slots] (1..16 distinct values >= 1);
 * state_capacity = the limit on stored states = pool size; entry_capacity
 * >= state_capacity bounds entry ids (every live prompt holds a state).
 * Returns the handle in *out; release it with nv_lcbfu_destroy.
 *
 * nv_lcbfu_access: B served requests (HOST row [B], HOST k [B], the k
 * nv_gather_pool returned): each with k > 0 raises its state's f by one.
 * A row out of range or a k naming no stored state is NV_ERR_INVALID_ARG
 * (nothing is changed).
 *
 * nv_lcbfu_insert: makes room for and stores m new prompts (m * n_slots <=
 * state_capacity).  First it evicts the fewest lowest-scored states that let
 * m * n_slots new ones fit (exactly n_slots per prompt once full); a prompt
 * left with no state is dropped: the live rows at or past the new row count
 * (*n_kept) move, in ascending order, into the dropped rows below it.  Then
 * prompt i gets the lowest free entry id entry_out[i] and the lowest free
 * pool states state_out[i][s] (slot order), and row *n_kept + i.  All
 * outputs are HOST arrays sized by the caller: entry_out [m], state_out
 * [m][n_slots], move_src / move_dst [m * n_slots] (*n_moves used), upd
 * [m * n_slots + m][1 + n_slots] (*n_upd records for nv_table_update: every
 * entry whose table row changed, ascending, with its new row).
 *
 * nv_lcbfu_info: info HOST int64 [5] = rows, stored states, evictions so far,
 * prompts dropped so far, states ever stored.
 * nv_lcbfu_export: copies (each may be NULL) the table HOST int32
 * [entry_capacity][n_slots], the row -> entry map HOST int32 [rows], and
 * counts HOST int64 [state_capacity] (f of each pool state, 0 if free).
 * ------------------------------------------------------------------------ */
typedef struct nv_lcbfu nv_lcbfu;
int32_t nv_lcbfu_create(int32_t n_slots, const int32_t* slot_k, int64_t state_capacity,
                        int64_t entry_capacity, nv_lcbfu** out);
void nv_lcbfu_destroy(nv_lcbfu* h);
int32_t nv_lcbfu_access(nv_lcbfu* h, int32_t B, const int64_t* row, const int32_t* k);
int32_t nv_lcbfu_insert(nv_lcbfu* h, int32_t m, int32_t* entry_out, int32_t* state_out,
                        int64_t* move_src, int64_t* move_dst, int32_t* n_moves, int32_t* upd,
                        int32_t* n_upd, int64_t* n_kept);
int32_t nv_lcbfu_info(const nv_lcbfu* h, int64_t* info);
int32_t nv_lcbfu_export(const nv_lcbfu* h, int32_t* table, int32_t* rows, int64_t* counts);

/* ------------------------------------------------------------------------ *
 * IVF approximate index over the cached embeddings (the paper's vector DB
 * searches through an index, Sec. 5.3 / Sec. 6; an exact scan is
 * nv_cache_lookup).  Scores are the lookup's canonical float64 scores; every
 * order is total (ties to the lower list / row), so results are
 * reproducible bit for bit.
 *
 * nv_ivf_build: cache device [n][d] of c_dtype (d a multiple of 8, <= 2048);
 * init HOST int64 [L] (1 <= L <= min(n, 4096)): the rows that start the
 * centroids.  iters Lloyd steps (0..100) each assign every row to its best
 * centroid (lower list on ties) and replace each non-empty list's centroid
 * by its normalised mean: the float64 sum of its rows in ascending row
 * order, divided by the correctly rounded square root of the left-to-right
 * sum of squares, rounded to float32 and then to the cache type.  A final
 * assignment gives lists (device int64 [n]); perm (device int64 [n]) holds
 * the row ids grouped by list, ascending within a list; offsets (device
 * int64 [L + 1]) delimit the lists; ivf_rows (device [n][d] of c_dtype)
 * receives the rows in perm order; cents (device [L][d] of c_dtype) the
 * centroids; *max_list (HOST) the longest list.  Synchronous on `stream`.
 * workspace >= nv_ivf_build_workspace(n, d, L), 256-byte aligned.
 *
 * nv_ivf_search: queries device f32 [m][d] (1 <= m <= 4096); the index as
 * built; 1 <= nprobe <= min(L, 256).  Each query ranks the lists by its
 * score against their centroids (higher first, lower list on ties), scans
 * the first nprobe, and returns the best row among them (higher score
 * first, lower row on ties): idx_out (device int64 [m], the original row
 * id, -1 if every probed list is empty), sim_out (device f32 [m], the score
 * rounded to float32, -inf if none) and k_out (device int32 [m], the
 * selector's K as in nv_cache_lookup).  probed_out (device int32
 * [m][nprobe], may be NULL) receives the lists probed, in rank order.
 * workspace >= nv_ivf_search_workspace(m, L, nprobe, max_list).
 * nprobe = L gives the exact lookup's results.
 * ------------------------------------------------------------------------ */
size_t nv_ivf_build_workspace(int64_t n, int32_t d, int32_t L);
int32_t nv_ivf_build(const void* cache, int32_t c_dtype, int64_t n, int32_t d,
                     const int64_t* init, int32_t L, int32_t iters, void* cents, int64_t* lists,
                     int64_t* perm, int64_t* offsets, void* ivf_rows, int64_t* max_list,
                     void* workspace, size_t workspace_bytes, void* stream);
size_t nv_ivf_search_workspace(int32_t m, int32_t L, int32_t nprobe, int64_t max_list);
int32_t nv_ivf_search(const float* queries, int32_t m, int32_t d, const void* cents, int32_t L,
                      const void* ivf_rows, int32_t c_dtype, const int64_t* perm,
                      const int64_t* offsets, int64_t max_list, int32_t nprobe,
                      const float* thresholds, const int32_t* k_values, int32_t J,
                      int64_t* idx_out, float* sim_out, int32_t* k_out, int32_t* probed_out,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ *
 * Match predictor (Sec. 5.2, Sec. 6: a one-class SVM over the cached prompt
 * embeddings decides whether a close match is likely; if not, the request
 * skips the cache and is generated from scratch, Alg. 1).
 *
 * Model: linear, decision value s(q) = w.q - rho, match predicted iff
 * s(q) >= tau.  Training minimises
 *   J(w, rho) = nu/2 |w|^2 - nu rho + (1/n) sum_i max(0, rho - w.x_i)
 * by plain SGD in float64 from w = 0, rho = 0: at step t (0-based) over row
 * i = order[t], eta = eta0 / (1 + eta0 nu t); if rho - w.x_i > 0,
 * w -= eta (nu w - x_i) and rho -= eta (1 - nu), else w -= eta nu w and
 * rho += eta nu.  Every w.x is a left-to-right sum of rounded float64
 * products with no fused multiply-add, so results are bit-reproducible.
 *
 * nv_ocsvm_train (host only): rows HOST [n][d] of c_dtype (the vector DB's
 * embeddings), order HOST int64 [T] (the visiting order; the caller draws
 * it), w_out HOST float64 [d], rho_out HOST.
 *
 * nv_match_gate: scores the queries (device f32 [m][d]) with w (device
 * float64 [d]) and, when idx / sim / k (device, a lookup's outputs for the
 * same queries) are given, turns every query with s < tau into "no match":
 * idx = -1, sim = -inf, k = 0.  score_out (device float64 [m]) may be NULL
 * when idx is given, and idx / sim / k NULL to only score.  Applied after
 * the lookup, it gives Alg. 1's result with the predictor in front.
 * ------------------------------------------------------------------------ */
int32_t nv_ocsvm_train(const void* rows, int32_t c_dtype, int64_t n, int32_t d, double nu,
                       double eta0, const int64_t* order, int64_t T, double* w_out,
                       double* rho_out);
int32_t nv_match_gate(const float* queries, int32_t m, int32_t d, const double* w, double rho,
                      double tau, double* score_out, int64_t* idx, float* sim, int32_t* k,
                      void* stream);

/* nv_cache_lookup_gated: Alg. 1 with the predictor in front of the search.
 * Each query's decision value s = w.q - rho is computed as by nv_match_gate;
 * the queries with s >= tau are compacted (ascending order) and searched by
 * the exact lookup, the others get the "no suitable cache" result (idx -1,
 * sim -inf, K 0) without touching the cache.  Arguments and results as
 * nv_cache_lookup (idx_out, sim_out, k_out for every query) and
 * nv_match_gate (w, rho, tau; score_out device float64 [m] or NULL), plus
 * *n_searched (HOST) = the number of queries searched.  Synchronous on
 * `stream` (that number sizes the search).  workspace >=
 * nv_cache_lookup_gated_workspace(m, n, d), 256-byte aligned.  Errors: those
 * of nv_cache_lookup, NV_ERR_INVALID_ARG for null w / n_searched, a
 * non-finite rho or a NaN tau. */
size_t nv_cache_lookup_gated_workspace(int32_t m, int64_t n, int32_t d);
int32_t nv_cache_lookup_gated(const float* queries, int32_t m, const void* cache,
                              int32_t c_dtype, int64_t n, int32_t d, const float* thresholds,
                              const int32_t* k_values, int32_t J, const double* w, double rho,
                              double tau, int64_t* idx_out, float* sim_out, int32_t* k_out,
                              double* score_out, int32_t* n_searched, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ *
 * Latent-diffusion UNet (Sec. 2.1: UNet backbone, text conditioning through
 * cross-attention, operating on latents).  Topology rule:
 *   conv_in; per level l: n_res ResBlocks (+ transformer of depth[l] if > 0),
 *   stride-2 conv except at the last level; middle Res / Transformer
 *   (mid_depth, skipped if 0) / Res; per level from the last: n_res + 1
 *   ResBlocks on [h, skip] channel concatenations (+ transformer), nearest x2
 *   upsample + conv except at level 0; GroupNorm, SiLU, conv_out.
 *   Time embedding: [cos(t f_k), sin(t f_k)], f_k = exp(-ln(1e4) k / (ch0/2)),
 *   Linear(ch0, 4 ch0), SiLU, Linear(4 ch0, 4 ch0), + pooled (pooled_dim
 *   must then equal 4 ch0).  Heads: n_heads if > 0, else C / head_dim.
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t in_ch, out_ch;  /* latent channels (4, 4) */
  int32_t H, W;           /* latent size, divisible by 2^(n_levels-1) */
  int32_t n_levels;       /* 1..4 */
  int32_t ch[4];          /* channels per level, multiples of 32 and of gn_groups */
  int32_t depth[4];       /* transformer depth per level (0 = none) */
  int32_t mid_depth;      /* transformer depth of the middle block */
  int32_t n_res;          /* ResBlocks per down level (n_res + 1 per up level) */
  int32_t n_heads;        /* > 0: fixed head count */
  int32_t head_dim;       /* used when n_heads == 0 */
  int32_t gn_groups;      /* GroupNorm groups */
  int32_t ctx_len, ctx_dim; /* conditioning tokens and their width */
  int32_t pooled_dim;     /* 0, or 4*ch[0]: pooled vector added to the time embedding */
  float gn_eps, ln_eps;
} nv_unet_config;

typedef struct nv_unet nv_unet;

/* Number of float weights of a topology (-1 if the config is invalid). */
int64_t nv_unet_param_count(const nv_unet_config* cfg);

/* Name and element count of parameter i (0-based) in canonical order;
 * name is NUL-terminated and truncated to name_len bytes. */
int32_t nv_unet_param_info(const nv_unet_config* cfg, int64_t i, char* name, int32_t name_len,
                           int64_t* numel);

/* weights_host: HOST float32 array of nv_unet_param_count(cfg) values, the
 * tensors concatenated in canonical order (conv weights [Cout][Cin][3][3],
 * linear [out][in], row-major):
 *   time.l1.{w,b} time.l2.{w,b} conv_in.{w,b}
 *   per down level, per ResBlock: res, then transformer if depth > 0;
 *     then ds.{w,b} unless last level
 *   mid.res0, mid.attn (if mid_depth > 0), mid.res1
 *   per up level from the last, per ResBlock (n_res + 1): res, transformer;
 *     then us.{w,b} unless level 0
 *   out.gn.{g,b} conv_out.{w,b}
 * res(cin, cout) = gn1.{g,b} conv1.{w,b} temb.{w,b} gn2.{g,b} conv2.{w,b}
 *   [skip.{w,b} (linear [cout][cin]) when cin != cout]
 * transformer(c, depth) = gn.{g,b} proj_in.{w,b}, per block:
 *   ln1.{g,b} attn1.q.w attn1.k.w attn1.v.w attn1.o.{w,b} ln2.{g,b}
 *   attn2.q.w attn2.k.w ([c][ctx_dim]) attn2.v.w attn2.o.{w,b} ln3.{g,b}
 *   ff1.{w,b} ([8c][c], output [a | g]) ff2.{w,b} ([c][4c]); then proj_out.{w,b}.
 * Matrices are converted to float16 on the device (exact for bfloat16-valued
 * weights of magnitude in [2^-17, 65504]); norms and biases stay float32.
 * The model computes with float16 matrix-core operands, float32 accumulation
 * and float32 statistics.  *out receives the handle. */
int32_t nv_unet_create(const nv_unet_config* cfg, const float* weights_host, int64_t n_weights,
                       nv_unet** out);
void nv_unet_destroy(nv_unet* net);

/* DDIM schedule: T training steps (T % N == 0), scaled-linear betas
 * beta_t = (sqrt(beta_start) + (sqrt(beta_end) - sqrt(beta_start)) t/(T-1))^2,
 * abar_t = prod_{s<=t}(1 - beta_s); grid t_i = (N-1-i) T/N + 1; step i goes
 * t_i -> t_{i+1}, the last step to abar_0.  Deterministic (eta = 0). */
typedef struct {
  int32_t T, N;
  float beta_start, beta_end;
} nv_schedule;

/* Device workspace needed by nv_denoise / nv_unet_eps for B samples (2B rows). */
size_t nv_denoise_workspace(const nv_unet* net, int32_t B);

/* Resume B samples from their cached states (Sec. 4.1): sample b holds, in
 * latent (device f32 [B][in_ch][H][W]), the state after k[b] steps, and
 * runs steps k[b] .. N-1; on return latent holds x_0 for every sample.
 * k: HOST int32 [B], 0 <= k[b] <= N (k[b] == N: returned unchanged; k[b] == 0:
 * full generation from x_N).  cond, uncond: device f32 [B][ctx_len][ctx_dim]
 * (the prompt's and the empty prompt's encodings).  pooled: device f32
 * [B][pooled_dim], or NULL when pooled_dim == 0 (applied to both rows).
 * Each step evaluates the UNet on 2 rows per sample (uncond, cond), combines
 * eps = eps_u + guidance (eps_c - eps_u) and applies the DDIM update.
 * Samples with different k run together: at iteration j sample b is at
 * step k[b] + j and leaves the batch after step N-1.  1 <= B <= 64. */
int32_t nv_denoise(nv_unet* net, const nv_schedule* sched, float* latent, const int32_t* k,
                   int32_t B, const float* cond, const float* uncond, const float* pooled,
                   float guidance, void* workspace, size_t workspace_bytes, void* stream);

/* nv_denoise with DDIM's stochastic samplers (eta in [0, 1]): each update is
 *   x <- sqrt(a_p) x0 + sqrt(1 - a_p - sigma^2) eps + sigma z,
 *   sigma = eta sqrt((1 - a_p) / (1 - a_t)) sqrt(1 - a_t / a_p),
 * with x0 = (x - sqrt(1 - a_t) eps) / sqrt(a_t) and z = noise[b][i] for
 * sample b at grid step i; noise: device f32 [B][N][in_ch][H][W] of standard
 * normal draws that the caller makes (a new seed after a cache hit makes the
 * tail of the trajectory, and the image, differ: the diversity remedy of
 * Sec. 9).  eta = 0 is the deterministic update of nv_denoise. */
int32_t nv_denoise_eta(nv_unet* net, const nv_schedule* sched, float* latent, const int32_t* k,
                       int32_t B, const float* cond, const float* uncond, const float* pooled,
                       float guidance, float eta, const float* noise, void* workspace,
                       size_t workspace_bytes, void* stream);

/* The cache-miss side of Alg. 1 (Sec. 4.3: a request without a suitable
 * cache generates from scratch and its intermediate states join the cache):
 * exactly nv_denoise, and in addition, whenever sample b has completed
 * slot_k[s] steps (including k[b] itself: the state it was given), its
 * latent is copied to store[entry[b]][s], store being device f32
 * [n_store][n_slots][in_ch][H][W] (the layout nv_gather_states reads).
 * slot_k: HOST int32 [n_slots], 1 <= n_slots <= 16, each in [0, N].
 * entry: HOST int64 [B], -1 (store nothing for b) or in [0, n_store).
 * Slots a sample never reaches (slot_k < k[b]) are left as they were.
 * Errors: those of nv_denoise, plus NV_ERR_INVALID_ARG for bad slots or
 * entries, or a null store with entries to write. */
int32_t nv_denoise_store(nv_unet* net, const nv_schedule* sched, float* latent,
                         const int32_t* k, int32_t B, const float* cond, const float* uncond,
                         const float* pooled, float guidance, float* store, int64_t n_store,
                         int32_t n_slots, const int32_t* slot_k, const int64_t* entry,
                         void* workspace, size_t workspace_bytes, void* stream);
int32_t nv_denoise_store_pool(nv_unet* net, const nv_schedule* sched, float* latent,
                              const int32_t* k, int32_t B, const float* cond,
                              const float* uncond, const float* pooled, float guidance,
                              float* pool, int64_t n_pool, int32_t n_slots,
                              const int32_t* slot_k, const int32_t* dst, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Execution options of a handle (flags, default NV_UNET_GRAPHS); the results
 * are bit-identical under every setting.
 *   NV_UNET_GRAPHS: the denoise entry points capture each step (the UNet on
 *     the active rows, guidance, the DDIM update) once into a HIP graph per
 *     active row count and replay it: the same kernels in the same order with
 *     one host call per step instead of one per kernel.  The graphs belong to
 *     the handle and are rebuilt when the workspace, the batch size, the
 *     guidance, eta, the noise pointer or N change between calls; while launch
 *     tracing is on, steps are launched kernel by kernel.
 * Setting options drops the captured graphs.  Not thread-safe with
 * concurrent calls on the handle.  NV_ERR_INVALID_ARG for a null handle or
 * unknown flags. */
enum { NV_UNET_GRAPHS = 1 };
int32_t nv_unet_set_options(nv_unet* net, int32_t flags);

/* One UNet evaluation per row for teacher-forced checks: sample b at step
 * index step_idx[b] (HOST int32 [B], 0 <= step_idx < N, timestep t_i of the
 * grid) gives eps_uncond[b], eps_cond[b] (device f32 [B][out_ch][H][W]). */
int32_t nv_unet_eps(nv_unet* net, const nv_schedule* sched, const float* x,
                    const int32_t* step_idx, int32_t B, const float* cond, const float* uncond,
                    const float* pooled, float* eps_uncond, float* eps_cond, void* workspace,
                    size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------ *
 * Single layers of the UNet on the same kernels the plan uses, for
 * per-layer parity checks and kernel measurement.  Activations are float16
 * (IEEE binary16), weights float16, bias float32; workspace: device,
 * >= nv_op_workspace() bytes, 256-byte aligned (split-K partials).
 *
 * nv_op_linear:  out[m][n] = sum_k a[m][k] w[n][k] (+ bias[n]) (+ residual[m][n]),
 *   a = [x | x2] the channel concatenation of x [M][K1] and x2 [M][K2] (x2 NULL,
 *   K2 = 0 for one source); w [N][K1+K2], residual/out [M][N]; K1, K2 % 8 == 0.
 * nv_op_conv3x3: out = conv3x3([x | x2], w) + bias, zero padding 1, NHWC:
 *   x [B][H][W][Cin1], x2 [B][H][W][Cin2] (NULL, 0 for one source),
 *   w [Cout][3][3][Cin1+Cin2], out [B][Ho][Wo][Cout] with (Ho, Wo) = (H, W) for
 *   stride 1, (H/2, W/2) for stride 2 (H, W even), (2H, 2W) when upsample = 1
 *   (nearest x2 before the convolution); Cin1, Cin2 % 8 == 0.
 * ------------------------------------------------------------------------ */
size_t nv_op_workspace(void);
int32_t nv_op_linear(const void* x, const void* x2, const void* w, const float* bias,
                     const void* residual, void* out, int64_t M, int32_t N, int32_t K1,
                     int32_t K2, void* workspace, size_t workspace_bytes, void* stream);
int32_t nv_op_conv3x3(const void* x, const void* x2, const void* w, const float* bias, void* out,
                      int32_t B, int32_t H, int32_t W, int32_t Cin1, int32_t Cin2, int32_t Cout,
                      int32_t stride, int32_t upsample, void* workspace, size_t workspace_bytes,
                      void* stream);

/* nv_op_attention: multi-head softmax(q k^T * scale) v per row, float16 in and
 * out, float32 softmax (Sec. 2.1: the UNet's self- and cross-attention).
 *   q [rows][S][ldq] and k [rows][L][ldk] with head h in columns
 *   [h*dh, (h+1)*dh); v given TRANSPOSED: channel c of key j of row r at
 *   vt[c * vt_ld + r * vt_row + j], with vt_row >= L, vt_row % 8 == 0 and
 *   vt_ld >= rows * vt_row, vt_ld % 8 == 0 (keys L..vt_row-1 are never used);
 *   out [rows][S][ldo].  dh in {16, 32, 40, 64, 80, 128, 160}; ldq, ldk, ldo
 *   % 8 == 0.  No workspace. */
int32_t nv_op_attention(const void* q, const void* k, const void* vt, void* out, int32_t rows,
                        int32_t S, int32_t L, int32_t heads, int32_t dh, int32_t ldq, int32_t ldk,
                        int32_t ldo, int64_t vt_ld, int64_t vt_row, float scale, void* stream);

/* ------------------------------------------------------------------------ *
 * Launch tracing for measurement.  While enabled, every kernel launch of the
 * families in family_mask carries a pair of HIP events that the dispatch
 * timestamps at the kernel's start and end (the first max_launches launches
 * are kept), i.e. the kernel's execution time alone; each
 * record carries the launch's algorithmic FLOPs (2 M N K for matrix
 * products) and bytes.  nv_trace_read waits for the recorded events and
 * returns the sums over the launches of `family` (a mask).  Enabling again
 * discards earlier records.  Process-wide, not thread-safe across streams.
 * ------------------------------------------------------------------------ */
enum {
  NV_FAM_CONV = 1,    /* 3x3 implicit-GEMM convolutions (main kernel) */
  NV_FAM_LINEAR = 2,  /* dense GEMMs (main kernel) */
  NV_FAM_ATTN = 4,    /* attention */
  NV_FAM_SCAN = 8     /* cache scan of the lookup */
};
int32_t nv_trace_enable(int32_t family_mask, int32_t max_launches);
int32_t nv_trace_disable(void);
int32_t nv_trace_read(int32_t family, int64_t* launches, double* ms, double* flops,
                      double* bytes);
/* Record i (0-based, in launch order) of the current trace: its family, shape
 * (HOST int64 [4]: for matrix products M, N, K and the tile code
 * BM * 10000 + BN * 10 + splits; for attention S, L, heads * dh and
 * dh * 10000 + QB * 1000 + KB; for scans m, n, d, 0), kernel time in ms
 * (waits for the launch) and algorithmic FLOPs.  NV_ERR_INVALID_ARG when i is
 * out of range. */
int32_t nv_trace_get(int32_t i, int32_t* family, int64_t* shape, double* ms, double* flops);

/* ------------------------------------------------------------------------ *
 * Matrix-core throughput probe (measurement support, not part of the path).
 * Launches `blocks` workgroups of 256 threads; every wave issues iters x 8
 * independent v_mfma_f32_16x16x32_{f16,bf16} (bf16 != 0 selects bf16) on
 * register operands, i.e. blocks * 4 * iters * 8 * 16384 FLOPs.  Time it with
 * events on `stream` to obtain the achieved dense matrix peak.  sink: device
 * float[256], never written in practice (keeps the work live).
 * Errors: NV_ERR_INVALID_ARG for a null sink or non-positive sizes.
 * ------------------------------------------------------------------------ */
int32_t nv_probe_mfma(int32_t bf16, int32_t iters, int32_t blocks, float* sink, void* stream);
/* HBM read probe: reads bytes / 16 16-byte chunks of the device buffer buf
 * once (`blocks` workgroups of 256 threads, grid-stride); time it with events
 * for the achieved read bandwidth.  sink as above.  Errors: NV_ERR_INVALID_ARG
 * for null pointers, bytes < 16 or blocks <= 0. */
int32_t nv_probe_read(const void* buf, int64_t bytes, int32_t blocks, float* sink, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* NV_H */
