/*
 * libsalt -- batched centroid + residual LoRA apply for MI355X (gfx950).
 *
 * The serving-time composition of SALT ("Pin Once, Swap Light", Sec. 3.3): the
 * weight served to request i is W_base + gamma * Wbar + delta_i, where the domain
 * centroid Wbar is a high-rank LoRA that stays pinned in GPU memory (Sec. 3.1)
 * and the user residual delta_i is a rank <= 2 LoRA that is swapped in from host
 * memory on demand (Sec. 3.1, Sec. 4.4).  With y already holding x * W_base, the
 * library adds, for every token t of a mixed batch,
 *
 *     y_t += gamma_t * (x_t A_{c_t}) B_{c_t}  +  (x_t A_{u_t}) B_{u_t}
 *
 * (row vectors; A is in x r, B is r x out; c_t = centroid id, u_t = residual slot).
 *
 * Conventions for every entry point
 *   - Returns a salt_status; no exception or abort crosses the ABI.
 *   - An invalid call (SALT_ERR_INVALID_ARG, _OUT_OF_RANGE, _NOT_PINNED,
 *     _SLOT_EMPTY) changes no state.  A failing HIP call returns SALT_ERR_HIP and
 *     poisons the context: every later call on it returns SALT_ERR_BAD_STATE.
 *     salt_last_error() gives a message for the last failure.
 *   - A context is externally synchronised (not thread-safe).
 *   - "stream" arguments are hipStream_t values passed as void*; NULL is the
 *     legacy default stream.  Work is enqueued asynchronously unless stated.
 *   - Adapter layout is rank-major: A is stored transposed, At[r][in], and B as
 *     B[r][out], both row-major in the context dtype.  Concatenating a centroid
 *     and a residual (the single r_c + r_u adapter of Sec. 3.3) is then a stack
 *     of rows.
 *   - in_dim and out_dim must be multiples of 8; x, y and every host buffer must
 *     be 16-byte aligned.
 */
#ifndef SALT_H_
#define SALT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SALT_VERSION 1

#if defined(__GNUC__)
#define SALT_API __attribute__((visibility("default")))
#else
#define SALT_API
#endif

typedef enum {
  SALT_OK = 0,
  SALT_ERR_INVALID_ARG = 1,   /* null pointer, bad size, misaligned buffer        */
  SALT_ERR_OUT_OF_RANGE = 2,  /* table / centroid / slot / rank / token count     */
  SALT_ERR_OUT_OF_MEMORY = 3, /* device or pinned allocation failed               */
  SALT_ERR_NOT_PINNED = 4,    /* residual blob is not page-locked host memory     */
  SALT_ERR_SLOT_EMPTY = 5,    /* a map references a slot that was never loaded    */
  SALT_ERR_HIP = 6,           /* a HIP runtime call failed; the context is poisoned */
  SALT_ERR_BAD_STATE = 7      /* poisoned context, stale plan, unpinned centroids */
} salt_status;

typedef enum { SALT_F32 = 0, SALT_BF16 = 1 } salt_dtype;

/* One adapted linear projection ("table"): x[T][in_dim] -> y[T][out_dim]. */
typedef struct {
  int32_t in_dim;
  int32_t out_dim;
} salt_shape;

typedef struct {
  salt_dtype dtype;          /* storage type of x, y and every adapter; math is fp32 */
  int32_t n_tables;          /* >= 1: projections served by this context            */
  const salt_shape* tables;  /* [n_tables]; copied by salt_create                  */
  int32_t n_centroids;       /* C in [0, 64]: centroid library size (Sec. 3.2)     */
  int32_t r_c;               /* centroid rank in [0, 128], a multiple of 8 (0 iff C == 0) */
  int32_t n_slots;           /* residual slot-pool size, >= 1                      */
  int32_t r_u_max;           /* largest residual rank a slot holds, in [0, 72]: ranks
                                up to 2 are the SALT residuals, larger ones serve
                                long-tail adapters that concatenate a centroid and a
                                residual (Sec. 3.3, e.g. r = 17 / 33 / 65)           */
  int32_t max_tokens;        /* largest batch a plan accepts, in [1, 65536]         */
  int32_t device;            /* HIP device ordinal                                  */
  int32_t flags;             /* reserved, must be 0                                 */
} salt_config;

/* Results are reproducible: the split-K partial sums of the shrink are added
 * in a fixed order, so the same call on equal inputs gives bit-identical y on
 * every run.  The K split depends on the tables that share a launch, so one
 * table applied alone and inside a salt_apply_batch may differ in the last
 * bits (both within fp32 accumulation error). */

typedef struct salt_ctx salt_ctx;
typedef struct salt_plan salt_plan;

/* ---- context ----------------------------------------------------------------
 * salt_create validates cfg, then allocates on cfg->device: the centroid store
 * (per table, At[C][r_c][in] and B[C][r_c][out]), the residual slot pool
 * (n_slots slots of salt_residual_bytes(ctx, r_u_max) bytes each) and a side
 * stream for residual swaps.  The context owns all of these; salt_destroy waits
 * for the context's outstanding work and frees them.  Fails with
 * SALT_ERR_OUT_OF_MEMORY (nothing leaked) if the pool does not fit. */
SALT_API salt_status salt_create(const salt_config* cfg, salt_ctx** out);
SALT_API void salt_destroy(salt_ctx* ctx);

/* Pin centroids c0 .. c0+n-1 of one table into device memory (Sec. 3.1: the
 * centroid is pre-loaded and pinned; Sec. 3.3: done once at node start-up).
 *   At_host: [n][r_c][in] host array (pageable is fine), B_host: [n][r_c][out].
 * Blocking: the copy has completed when the call returns and the host arrays may
 * be freed.  salt_apply on a table refuses to run (SALT_ERR_BAD_STATE) until all
 * n_centroids of that table have been pinned at least once. */
SALT_API salt_status salt_pin_centroids(salt_ctx* ctx, int32_t table, int32_t c0, int32_t n,
                               const void* At_host, const void* B_host);

/* Size in bytes of one user's residual blob of rank r_u over all tables of the
 * context: r_u * sum_t(in_t + out_t) * element size (the per-adapter swap size
 * of Table 1 and the appendix tables).  Returns 0 for an invalid rank. */
SALT_API size_t salt_residual_bytes(const salt_ctx* ctx, int32_t r_u);
/* Same count without a context (host-only; no HIP call). */
SALT_API size_t salt_residual_bytes_for(salt_dtype dtype, int32_t n_tables, const salt_shape* tables,
                               int32_t r_u);

/* Swap one user's residual into a slot of the HBM pool (Sec. 3.1: only the
 * residual is swapped; Sec. 4.4: the H2D PCIe transfer this minimises).
 *   blob: page-locked host memory (salt_host_alloc / hipHostMalloc), laid out as,
 *         for each table in order, At_u[r_u][in] followed by B_u[r_u][out];
 *         bytes must equal salt_residual_bytes(ctx, r_u).  r_u == 0 empties the
 *         residual term of the slot (bytes == 0, blob may be NULL).
 * Asynchronous, on the context's side stream: a blob inside memory from
 * salt_host_alloc is read by the device directly (the gather kernel of
 * salt_load_residuals); any other page-locked blob takes one hipMemcpyAsync.
 * The copy first
 * waits for every enqueued salt_apply whose plan references this slot, so an
 * in-flight apply still sees the slot's previous residual.  Every later
 * salt_apply whose plan references the slot waits for this copy.  The blob must
 * stay valid and unmodified until the copy completes (salt_wait_loads).
 * The event that orders the copy behind those applies is recorded on their
 * stream when it is needed (here, at the plan's next salt_plan_set_maps, or when
 * the plan moves to another stream), not after every apply, so it also covers
 * work enqueued on that stream since; the stream of a plan's latest applies must
 * therefore stay valid until one of those calls or salt_plan_destroy.
 * Errors: SALT_ERR_OUT_OF_RANGE (slot, r_u > r_u_max), SALT_ERR_INVALID_ARG
 * (bytes mismatch), SALT_ERR_NOT_PINNED (pageable blob; no synchronous fallback). */
SALT_API salt_status salt_load_residual(salt_ctx* ctx, int32_t slot, int32_t r_u, const void* blob,
                               size_t bytes);

/* A batch of swaps (Sec. 4.4: the per-step H2D traffic of the users that come
 * in): slots[i] <- blobs[i] of rank ranks[i] and bytes[i] bytes, for i < n, as
 * salt_load_residual would do them one by one, but validated as a whole first
 * (an invalid entry fails the call and changes no state) and ordered with one
 * event for the whole batch.  Blobs inside memory from salt_host_alloc need no
 * pointer query; when every blob of the call lies in such memory and no slot
 * repeats, one kernel per 64 blobs reads them all over PCIe into their slots
 * (no per-blob DMA set-up), else each blob takes its own hipMemcpyAsync, in
 * order.  A slot listed twice receives its last blob. */
SALT_API salt_status salt_load_residuals(salt_ctx* ctx, int32_t n, const int32_t* slots, const int32_t* ranks,
                                         const void* const* blobs, const size_t* bytes);

/* Block the host until every residual swap enqueued so far has completed. */
SALT_API salt_status salt_wait_loads(salt_ctx* ctx);

/* Page-locked host buffers for residual blobs (hipHostMalloc / hipHostFree),
 * mapped for the device current at the call, so that swaps of a context on that
 * device can read them in place (on another device they take DMA copies). */
SALT_API salt_status salt_host_alloc(size_t bytes, void** out);
SALT_API void salt_host_free(void* p);

/* ---- plans --------------------------------------------------------------------
 * A plan is the canonical grouping of one batch (Sec. 3.3: the frontend groups
 * requests by their centroid): tokens ordered by (centroid id, residual slot,
 * token index) ascending, -1 first.  Built once per batch on the device, then
 * reused by every table's apply.  A plan owns device buffers sized for
 * max_tokens, including the apply's scratch (split-K partials: two K ranges per
 * token row of a 16-table launch, or up to 64 MiB for small batches so that
 * their launches can split K finely enough to fill the device): the work of one
 * plan is ordered by the library, also across streams (a call on a stream other
 * than the one of the plan's last work first waits for that work), so several
 * streams that run concurrently need one plan each.
 * Why four calls (create / set_maps / build / destroy) instead of one build
 * that allocates: a serving loop keeps one plan per stream and reuses its
 * buffers batch after batch, so no call on the hot path allocates; the maps
 * are staged (host validation, one H2D copy) separately from the device build
 * so that the copy can be issued early.  salt_apply_map is the one-shot form. */
SALT_API salt_status salt_plan_create(salt_ctx* ctx, salt_plan** out);
SALT_API void salt_plan_destroy(salt_ctx* ctx, salt_plan* plan);

/* Stage a batch's maps (host arrays, pageable or pinned, read before return):
 *   tok_c[T]: centroid id in [-1, C)        (-1: no centroid term)
 *   tok_u[T]: residual slot in [-1, n_slots) (-1: no residual term)
 *   tok_gamma[T]: centroid scale per token (Sec. 3.3's discrete gamma bins), or
 *                 NULL for gamma = 1.  Must be finite.
 * Validates the maps on the host (SALT_ERR_OUT_OF_RANGE, SALT_ERR_SLOT_EMPTY for
 * a slot never loaded), snapshots the residual rank of every referenced slot and
 * enqueues one H2D copy of the packed maps on `stream`.  0 <= T <= max_tokens;
 * T == 0 gives an empty plan whose applies do nothing. */
SALT_API salt_status salt_plan_set_maps(salt_ctx* ctx, salt_plan* plan, int32_t T, const int32_t* tok_c,
                               const int32_t* tok_u, const float* tok_gamma, void* stream);

/* Build the plan on the device from the staged maps (enqueued on `stream`):
 * the sorted order, the segments of equal (centroid, slot) and the groups of
 * equal centroid.  Integer work; the result is bit-exact and unique.  One
 * kernel for batches of up to 4096 tokens, three above.  The tiles the apply
 * kernels walk (runs of at most 16 / 32 / 64 tokens of one centroid group) are
 * cut on the host by salt_plan_set_maps from its per-centroid token counts; the
 * build checks them against the sorted order (salt_plan_errors). */
SALT_API salt_status salt_plan_build(salt_ctx* ctx, salt_plan* plan, void* stream);

/* Copy a built plan to host arrays (synchronises `stream`).  Sizes: perm[T],
 * seg_off[n_seg + 1], seg_c[n_seg], seg_u[n_seg], grp_off[n_grp + 1] where
 * n_seg, n_grp <= T; pass arrays of T + 1 entries.  Any pointer may be NULL. */
SALT_API salt_status salt_plan_download(salt_ctx* ctx, const salt_plan* plan, void* stream, int32_t* perm,
                               int32_t* seg_off, int32_t* seg_c, int32_t* seg_u, int32_t* grp_off,
                               int32_t* n_seg, int32_t* n_grp);

/* ---- the hot path ---------------------------------------------------------------
 * y[t] += gamma_t * (x[t] A_{c_t}) B_{c_t} + (x[t] A_{u_t}) B_{u_t} for one table,
 * every token of a built plan (Sec. 3.3's served weight minus W_base).
 *   x: device [T][in_dim], y: device [T][out_dim], context dtype, row-major,
 *      16-byte aligned; y is read and written once per element, rounded once
 *      (round-to-nearest-even) from fp32 y + fp32 delta.
 * Accumulation is fp32: the centroid contractions run on MFMA with fp32
 * accumulation (bf16 contexts: the expand splits the fp32 v into two bf16
 * terms), the residual contractions on fp32 vector ALUs.  Two kernel launches
 * on `stream` (the shrink, then the expand), enqueued after the swaps of every
 * slot the plan references; no block of either waits for another block.
 * Errors: SALT_ERR_OUT_OF_RANGE (table), SALT_ERR_BAD_STATE (plan not built;
 * centroids of the table not all pinned; a referenced slot was reloaded with a
 * different rank after salt_plan_set_maps), SALT_ERR_INVALID_ARG (null or
 * misaligned x / y).  T == 0 is a no-op. */
SALT_API salt_status salt_apply(salt_ctx* ctx, int32_t table, salt_plan* plan, const void* x, void* y,
                       void* stream);

/* The apply of n tables on one plan (a decoder layer's projections, Sec. 3.3:
 * every table of a batch shares its grouping): tables[i] with xs[i] -> ys[i]
 * for i < n, the same result as n calls of salt_apply, in launches of up to 16
 * tables (each launch two kernels, whatever n).  Tables may repeat and x
 * pointers may be shared (q / k / v read one x); y buffers must not overlap.
 * Errors as salt_apply, for any entry; nothing is enqueued then. */
SALT_API salt_status salt_apply_batch(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan,
                                      const void* const* xs, void* const* ys, void* stream);

/* salt_apply_batch for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * same arguments and kernels, but the launches keep their split-K partial sums
 * in a static device array of the library (64 MiB per device, set up by
 * salt_create) instead of the plan's buffer, whose capacity still bounds the
 * K split.  The call allocates nothing and calls no allocating routine.
 * Whenever the plan's partial capacity (two K ranges per token row of a
 * 16-table launch, raised to up to 16 Mi floats for small batches; it fits the
 * array when max_tokens x padded(r_c + r_u) <= 512 Ki) fits the array,
 * the launches are exactly those of salt_apply_batch and y is bit-identical;
 * beyond that a launch may split K more coarsely (same accuracy bound).  The
 * array is shared by every salt_apply_batch_noalloc on the device: calls whose
 * work overlaps in time (on different streams) race on it and give wrong y;
 * calls on one stream are ordered and safe.  Every partial a launch reads was
 * written by that launch, so nothing needs clearing.  SALT_ERR_OUT_OF_RANGE
 * (nothing enqueued) if a launch's partials cannot fit even with one K range
 * per table: T x padded(r_c + r_u) floats per table of the launch must total
 * at most 16 Mi. */
SALT_API salt_status salt_apply_batch_noalloc(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan,
                                              const void* const* xs, void* const* ys, void* stream);

/* salt_apply_batch for measurement (n <= 16: one launch): events[0] and
 * events[1] (hipEvent_t, timing enabled) record the start and end of the
 * shrink kernel, events[2] and events[3] those of the expand kernel
 * (hipExtLaunchKernel), so hipEventElapsedTime gives each kernel's own
 * duration without the dispatch gaps.  SALT_ERR_INVALID_ARG for a null
 * event; SALT_ERR_OUT_OF_RANGE for n > 16. */
SALT_API salt_status salt_apply_batch_timed(salt_ctx* ctx, int32_t n, const int32_t* tables, salt_plan* plan,
                                            const void* const* xs, void* const* ys, void* stream,
                                            void* const* events);

/* One-shot apply on host maps (the frontend call of Sec. 3.3: group the
 * incoming requests, then serve them): salt_plan_set_maps + salt_plan_build +
 * salt_apply on a plan the context owns and reuses (created on the first call;
 * no allocation after that), all on `stream`.  Maps as salt_plan_set_maps, x /
 * y as salt_apply; the host arrays are read before the call returns.  Calls
 * that share the context's plan are ordered by the library. */
SALT_API salt_status salt_apply_map(salt_ctx* ctx, int32_t table, int32_t T, const int32_t* tok_c,
                                    const int32_t* tok_u, const float* tok_gamma, const void* x, void* y,
                                    void* stream);

/* Synchronise `stream`, then report in *n_errors how many tile records the
 * device build found inconsistent with the sorted order (a tile holding a
 * token of another centroid, or a malformed tile); 0 in normal operation.
 * SALT_ERR_BAD_STATE (and *n_errors >= 1) if the device plan's token or tile
 * count differs from what the host staged.  The apply kernels clamp every
 * index they read from a plan, so an inconsistent plan cannot make them access
 * memory outside their buffers; it would make y wrong, which this call reports. */
SALT_API salt_status salt_plan_errors(salt_ctx* ctx, const salt_plan* plan, void* stream,
                                      int32_t* n_errors);

/* How the applies of a plan whose maps are set run (host-only; no HIP call):
 *   *tile_tokens: tokens per tile (16, 32 or 64; the tiles of a centroid group
 *                 cut its tokens into near-equal runs of at most this many),
 *   *n_tiles:     tiles of the batch,
 *   *launches:    kernel launches per apply of up to 16 tables: 2 (shrink,
 *                 then expand), 0 for an empty batch.
 * Any pointer may be NULL.  SALT_ERR_BAD_STATE if no maps were set. */
SALT_API salt_status salt_plan_tiling(salt_ctx* ctx, const salt_plan* plan, int32_t* tile_tokens,
                                      int32_t* n_tiles, int32_t* launches);

/* ---- a centroid fused into the base weight -------------------------------------------
 * Sec. 3.3: for a high-frequency domain the provider folds the scaled centroid
 * into the base weight at node start-up; such a node then serves its tokens with
 * the residual alone (maps with c = -1).  For one pinned centroid c of `table`:
 *
 *     W[i][o] <- rne(W[i][o] + gamma * sum_r A_c[i][r] B_c[r][o])
 *
 *   W: device, the table's base weight in the context dtype, row-major
 *      [in_dim][ldw] (ldw elements between rows, a multiple of 8, >= out_dim;
 *      columns past out_dim are not touched), 16-byte aligned, owned by the
 *      caller.  Each element is read and written once; the rank-r_c product is
 *      accumulated in fp32 (bf16 MFMA for bf16 contexts) and added with one
 *      rounding (round-to-nearest-even).
 * Enqueued on `stream`.  The same call with -gamma takes the centroid out again
 * up to one rounding per call (not bit-exact in bf16).  Errors:
 * SALT_ERR_OUT_OF_RANGE (table, c), SALT_ERR_BAD_STATE (centroid never pinned),
 * SALT_ERR_INVALID_ARG (null or misaligned W, bad ldw, non-finite gamma). */
SALT_API salt_status salt_fuse_centroid(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w,
                                        int64_t ldw, void* stream);
/* salt_fuse_centroid for measurement: the HIP events `start_event` and
 * `stop_event` record the start and end of its kernel (as salt_apply_timed). */
SALT_API salt_status salt_fuse_centroid_timed(salt_ctx* ctx, int32_t table, int32_t c, float gamma, void* w,
                                              int64_t ldw, void* stream, void* start_event, void* stop_event);

/* ---- adapter similarity in factor space -------------------------------------------------
 * Sec. 3.1, Eq. 2: the alignment penalty between two low-rank updates is one
 * minus their matrix cosine, L_align(dW1, dW2) = 1 - Tr(dW1^T dW2) /
 * (||dW1||_F ||dW2||_F + 1e-8); Sec. 4.5 compares adapters and the centroid layer
 * by layer with the same cosine.  With dW = A B (A in x r, B r x out) the three
 * terms are sums over r x r Gram products, so the in x out updates are never
 * formed:  Tr(dW1^T dW2) = sum_ab (A1^T A2)_ab (B1 B2^T)_ab and
 * ||dW||_F^2 = sum_ab (A^T A)_ab (B B^T)_ab.
 *   blob1, blob2: device, 16-byte aligned, laid out like residual blobs of the
 *       context (for each table, At[r][in] then B[r][out], context dtype), ranks
 *       r1, r2 in [1, 256]; a centroid is passed the same way.
 *   out: host, [n_tables][3] doubles: Tr(dW1^T dW2), ||dW1||_F^2, ||dW2||_F^2 per table.
 * The Grams accumulate in fp32 (MFMA over in and over out), their elementwise
 * products in fp64.  Keeps its device scratch in the context (allocated on the
 * first call, grown when a call needs more, freed by salt_destroy), enqueues on
 * `stream` and synchronises it before returning (the results are host values).  Errors: SALT_ERR_OUT_OF_RANGE (rank),
 * SALT_ERR_INVALID_ARG (null or misaligned pointer), SALT_ERR_OUT_OF_MEMORY. */
SALT_API salt_status salt_adapter_gram(salt_ctx* ctx, const void* blob1, int32_t r1, const void* blob2,
                                       int32_t r2, double* out, void* stream);

/* ---- centroid routing (host only) ------------------------------------------------------
 * Sec. 3.2: a user's dataset is routed to a centroid of the library, or to the
 * standard-LoRA fallback, from the token-normalised displacement norms N_k its
 * profiling subset induces under each of the K centroids and the per-centroid
 * statistics calibrated at the end of Phase 1:
 *   stage 1 (out-of-distribution): Z_N,k = |N_k - mu_N,k| / sigma_N,k; the data is
 *       rejected when min_k Z_N,k > tau_N;
 *   stage 2 (expert routing): R_k = N_k / (mean of N_j over j != k),
 *       Z_R,k = |R_k - mu_R,k| / sigma_R,k, k* = argmin_k Z_R,k (lowest k on ties);
 *       the data is sent to the fallback as blended when Z_R,k* > tau_R.
 * Inputs are host arrays of K >= 2 finite values (N_k >= 0, sigma > 0, the other
 * norms of every k not all zero); z_n / z_r (may be NULL) receive Z_N,k / Z_R,k
 * (Z_R only when stage 1 passes).  No GPU work; no context needed.
 * Errors: SALT_ERR_INVALID_ARG. */
typedef struct {
  int32_t k_star;      /* routed centroid, or -1 for the fallback               */
  int32_t ood;         /* 1: rejected by stage 1                                  */
  int32_t blended;     /* 1: passed stage 1, rejected by stage 2's threshold      */
  double z_n_min;      /* min_k Z_N,k                                             */
  double z_r_min;      /* min_k Z_R,k (0 when stage 1 rejected)                   */
} salt_route_result;
SALT_API salt_status salt_route(int32_t K, const double* n_k, const double* mu_n, const double* sigma_n,
                                const double* mu_r, const double* sigma_r, double tau_n, double tau_r,
                                double* z_n, double* z_r, salt_route_result* out);

/* ---- diagnostics -------------------------------------------------------------------- */
SALT_API const char* salt_status_str(salt_status s);
SALT_API const char* salt_last_error(const salt_ctx* ctx);
SALT_API int32_t salt_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SALT_H_ */
