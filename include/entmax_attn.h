/*
 * entmax_attn.h -- C ABI of the MI355X (gfx950) alpha-entmax flash attention
 * library (AdaSplash, arXiv 2502.12082).
 *
 * Operation (per batch b, head h; Q, K, V, O in R^{n x d}):
 *   x_ij  = (alpha-1) * scale * <q_i, k_j>          (Eq. 1 scores in Eq. 2 coordinates)
 *   tau_i : sum_j [x_ij - tau_i]_+^{1/(alpha-1)} = 1  (Eq. 3; Algorithm 1, Halley-bisection)
 *   P_ij  = [x_ij - tau_i]_+^{1/(alpha-1)}           (Eq. 2)
 *   O     = P V                                      (Eq. 1 with pi = alpha-entmax)
 * and its gradients dQ, dK, dV (Sec. 3.2.2, Eq. 11-13, App. A.2).  Key blocks
 * whose probabilities are all zero are skipped (block mask, Eq. 8; lookup
 * tables, Sec. 3.2.1).  Causal attention is top-left aligned (key j <= query i).
 *
 * Memory: every tensor argument is a DEVICE pointer (HIP), contiguous,
 * [batch, heads, seqlen, head_dim] with head_dim fastest unless stated.  The
 * caller allocates and owns everything; the library never allocates, frees or
 * synchronises.  Calls are asynchronous on `stream` (a hipStream_t; NULL =
 * the default stream).  Buffers written by entmax_attn_fwd and read by
 * entmax_attn_bwd (the residuals) must stay alive and unmodified in between.
 *
 * Errors: arguments are checked before anything is launched; on failure
 * nothing is written and a non-zero ea_status is returned.  NaN/Inf inside
 * the tensors is not checked and propagates.  No C++ exception crosses this
 * interface.  All functions are reentrant.
 */
#ifndef ENTMAX_ATTN_H
#define ENTMAX_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  EA_OK = 0,
  EA_ERR_INVALID_ARG = 1, /* null/misaligned pointer, bad size or parameter */
  EA_ERR_UNSUPPORTED = 2, /* head_dim not 64/128, unknown dtype, seqlen too large */
  EA_ERR_WORKSPACE = 3,   /* workspace smaller than entmax_attn_sizes() says */
  EA_ERR_HIP = 4          /* a kernel launch failed */
} ea_status;

typedef enum { EA_BF16 = 0, EA_F32 = 1 } ea_dtype;

/* Problem shape.  seqlen n is the number of queries and of keys (1..131072). */
typedef struct {
  int32_t batch, heads, seqlen, head_dim; /* head_dim in {64, 128} */
  int32_t dtype;                          /* ea_dtype of Q, K, V, dO and O */
} ea_shape;

typedef struct {
  float alpha;      /* > 1; 2 = sparsemax, 1.5 = 1.5-entmax; finite */
  float scale;      /* > 0, finite; usually 1/sqrt(head_dim) */
  int32_t causal;   /* 0 or 1 */
  int32_t max_iter; /* Halley-bisection updates after the initial midpoint (Algorithm 1's T), 0..64 */
  float tol;        /* >= 0: the solver stops on a tile of query rows (256; 128 without a mask)
                       once every row has |f(tau)| <= tol */
  int32_t need_bwd; /* 1: also write o2 for a later entmax_attn_bwd */
} ea_params;

/*
 * Forward outputs other than O, consumed by the backward.  T = ceil(n / 64)
 * blocks of 64 rows; BH = batch * heads.
 *   tau        fp32  [BH, n]       threshold in Eq. 2 coordinates (x - tau)
 *   o2         fp32  [BH, n, d]    O^(2) = U V / rowsum(U), U = P^{2-alpha} (App. A.2);
 *                                  required iff need_bwd
 *   block_mask u8    [BH, T, T]    1 iff some p in the 64x64 block is > 0 (Eq. 8 at the
 *                                  returned tau); 0 for causally dead blocks
 *   q_count    i32   [BH, T]       |Q_i|, key blocks listed for query block i
 *   q_index    i32   [BH, T, T]    row (b,h,i): Q_i ascending in its first q_count entries
 *   k_count    i32   [BH, T]       |K_j|, query blocks listed for key block j
 *   k_index    i32   [BH, T, T]    row (b,h,j): K_j ascending in its first k_count entries
 *                                  (k_count, k_index: written only when need_bwd)
 *   stats      i32   [2, BH, T]    optional (may be NULL), per 64-row query block: [0] the K
 *                                  passes the solver streamed (1 max pass + evaluations that
 *                                  did not run on cached scores), [1] its evaluations of
 *                                  f, f', f'' (Algorithm 1 iterations, Eq. 3-7)
 *   tau_lo     fp32  [BH, n]       fp32 inputs only (required then; ignored, may be NULL,
 *                                  for bf16): the threshold is tau + tau_lo to ~fp64
 *                                  precision.  For alpha not in {1.25, 1.5, 2} the fp32
 *                                  path refines tau in fp64 and recomputes x - tau in fp64
 *                                  near the support edge, where u = p^(2-alpha) is
 *                                  ill-conditioned (Sec. 3.2.2); tau_lo is 0 otherwise.
 */
typedef struct {
  float* tau;
  float* o2;
  uint8_t* block_mask;
  int32_t* q_count;
  int32_t* q_index;
  int32_t* k_count;
  int32_t* k_index;
  int32_t* stats;
  float* tau_lo;
} ea_residuals;

/* Byte sizes of every residual buffer and of the workspaces. */
typedef struct {
  size_t tau, o2, block_mask, q_count, q_index, k_count, k_index, stats;
  size_t ws_fwd; /* workspace entmax_attn_fwd can use: the solver's candidate cache */
  size_t ws_bwd; /* workspace entmax_attn_bwd needs: fp32 [BH, n] for delta */
  size_t tau_lo; /* fp32 [BH, n] for fp32 inputs, 0 for bf16 */
} ea_sizes;

/* Library defaults: alpha 1.5, scale 1/sqrt(64), non-causal, max_iter 12,
 * tol 1e-5, need_bwd 1. */
void entmax_attn_default_params(ea_params* p);

/* Fills *out for this shape/params.  Errors as for entmax_attn_fwd's shape
 * and parameter checks. */
ea_status entmax_attn_sizes(const ea_shape* shape, const ea_params* params, ea_sizes* out);

/*
 * Forward: solves tau (Algorithm 1/3), writes the block mask and the lookup
 * tables, then O (and o2 if need_bwd), visiting only listed key blocks.
 *   q, k, v  [BH, n, d] in shape->dtype, 16-byte aligned
 *   o        [BH, n, d] in shape->dtype, 16-byte aligned (written)
 *   res      residual buffers (written), 4-byte aligned, o2 16-byte aligned
 *   workspace optional, 16-byte aligned: the solver's candidate cache, in
 *            1.125 MiB slots.  sizes.ws_fwd holds min(tiles, 512) slots (a
 *            tile is 256 query rows of one head), so it does not grow with
 *            B * H * n beyond 576 MiB.  With S slots and more tiles than
 *            slots the solver runs the tiles in launches of S workgroups,
 *            one slot each (2 S workgroups of 128 rows, half a slot each, in
 *            the one-group form the solver takes for small grids and at
 *            d = 64 for n <= 32768).  A tile stores, while it finds the row maxima, the
 *            scores above each row's lower bracket end and runs its
 *            evaluations on them instead of streaming K again (when the
 *            stored scores do not fit, it streams K, and collects once more
 *            if its first streamed evaluation counts few enough scores above
 *            the lower end).  Without a workspace (NULL, or too small for
 *            one slot) every tile streams K on every pass.  Results agree up
 *            to rounding either way.  Contents are scratch.
 * Launches 2 kernels on `stream` (the solver one more per S workgroups
 * beyond the first S).
 */
ea_status entmax_attn_fwd(const ea_shape* shape, const ea_params* params, const void* q,
                          const void* k, const void* v, void* o, const ea_residuals* res,
                          void* workspace, size_t ws_bytes, void* stream);

/*
 * Backward: dQ, dK, dV (fp32, [BH, n, d], 16-byte aligned, fully written) of
 * sum(dO * O), from Q, K, V, dO (shape->dtype) and the residuals of the
 * matching forward (tau, o2, tables; params must equal the forward's).
 * workspace: at least sizes.ws_bwd bytes, 16-byte aligned.  Launches 3
 * kernels on `stream`.
 */
ea_status entmax_attn_bwd(const ea_shape* shape, const ea_params* params, const void* q,
                          const void* k, const void* v, const void* dout,
                          const ea_residuals* res, float* dq, float* dk, float* dv,
                          void* workspace, size_t ws_bytes, void* stream);

/*
 * The same passes one kernel launch at a time, for callers that schedule or
 * time the stages themselves; entmax_attn_fwd is exactly stages 0, 1 and
 * entmax_attn_bwd stages 0, 1, 2, in order, with the same argument rules.
 *   forward  stage 0: tau, block_mask, q_count/q_index and stats (solver,
 *                     Algorithm 1/3, Eq. 8; row tables, Sec. 3.2.1)
 *            stage 1: O (and o2 if need_bwd) from tau and the row tables
 *                     (Algorithm 2, App. A.5), and if need_bwd
 *                     k_count/k_index from block_mask (Sec. 3.2.1)
 *   backward stage 0: delta = rowsum(dO * o2) into the workspace (App. A.2)
 *            stage 1: dK, dV over each key block's list (Algorithm 4, Eq. 12-13)
 *            stage 2: dQ over each query block's list (Algorithm 5, Eq. 11)
 * A stage reads what the earlier stages of the same pass wrote.  stage outside
 * 0..1 (forward) or 0..2 (backward) returns EA_ERR_INVALID_ARG.
 */
ea_status entmax_attn_fwd_stage(int stage, const ea_shape* shape, const ea_params* params,
                                const void* q, const void* k, const void* v, void* o,
                                const ea_residuals* res, void* workspace, size_t ws_bytes,
                                void* stream);
ea_status entmax_attn_bwd_stage(int stage, const ea_shape* shape, const ea_params* params,
                                const void* q, const void* k, const void* v, const void* dout,
                                const ea_residuals* res, float* dq, float* dk, float* dv,
                                void* workspace, size_t ws_bytes, void* stream);

/*
 * The backward without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Arguments, results and errors are those of
 * entmax_attn_bwd; delta lives in a scratch array inside the library instead
 * of a caller workspace: EA_NOALLOC_MAX_ROWS fp32 values (4 MiB), one copy per
 * device, held until the process ends.  batch * heads * seqlen above
 * EA_NOALLOC_MAX_ROWS returns EA_ERR_UNSUPPORTED before anything is launched.
 * Nothing is allocated: the first call on a device looks up the array's
 * address there (hipGetSymbolAddress, no allocation).  Every call on one
 * device shares that array, so calls that overlap on one device (concurrent
 * streams, or threads) race and must be serialised by the caller; calls on
 * one stream are ordered.  Launches 3 kernels on `stream`.
 */
#define EA_NOALLOC_MAX_ROWS 1048576
ea_status entmax_attn_bwd_noalloc(const ea_shape* shape, const ea_params* params, const void* q,
                                  const void* k, const void* v, const void* dout,
                                  const ea_residuals* res, float* dq, float* dk, float* dv,
                                  void* stream);

/*
 * No-mask ("memory-efficient") mode, Algorithm 2 as written (Sec. 3.2.1): the
 * forward solves tau and accumulates O (and, if need_bwd, o2) in one kernel
 * per 128-row query tile, visiting every valid key block; no block mask or
 * tables exist, so memory beyond the inputs and outputs is O(n) per head.
 *   tau  fp32 [BH, n] (written); o2 fp32 [BH, n, d] (written if need_bwd)
 *   tau_lo  fp32 [BH, n], fp32 inputs only (required then, written by the
 *        forward and read by the backward; ignored, may be NULL, for bf16):
 *        the low part of the threshold, as ea_residuals.tau_lo
 *   workspace  optional candidate cache, as for entmax_attn_fwd
 * The backward visits every valid block (no tables) and otherwise follows
 * entmax_attn_bwd: workspace >= sizes.ws_bwd bytes.  Results equal those of
 * entmax_attn_fwd / entmax_attn_bwd up to rounding.  One kernel launch
 * (forward) or three (backward) on `stream`.
 */
ea_status entmax_attn_fwd_dense(const ea_shape* shape, const ea_params* params, const void* q,
                                const void* k, const void* v, void* o, float* tau, float* tau_lo,
                                float* o2, void* workspace, size_t ws_bytes, void* stream);
ea_status entmax_attn_bwd_dense(const ea_shape* shape, const ea_params* params, const void* q,
                                const void* k, const void* v, const void* dout, const float* tau,
                                const float* tau_lo, const float* o2, float* dq, float* dk,
                                float* dv, void* workspace, size_t ws_bytes, void* stream);

/*
 * Row-wise alpha-entmax of a materialized score matrix s, [rows, n] row-major
 * in `dtype` (Sec. 3.1): per row, x = (alpha-1) * scale * s, tau from the
 * hybrid Halley-bisection iteration of Algorithm 1 (Eq. 3-7; the same update
 * rules, max_iter, tol and early exit as the attention solver), and
 * p_j = [x_j - tau]_+^(1/(alpha-1)) (Eq. 2).
 *   params  alpha, scale, max_iter, tol are used; causal and need_bwd are not
 *   p       fp32 [rows, n] (written), tau fp32 [rows] (written)
 * 1 <= n <= 32768 (longer rows return EA_ERR_UNSUPPORTED), rows >= 1.  All
 * pointers are device pointers, 16-byte aligned.  One kernel launch on
 * `stream`; nothing is allocated.
 */
ea_status entmax_rows_fwd(int64_t rows, int32_t n, ea_dtype dtype, const ea_params* params,
                          const void* s, float* p, float* tau, void* stream);

/*
 * Backward of entmax_rows_fwd: ds = scale * u * (dp - <u, dp> / sum(u)) per
 * row, u_j = [x_j - tau]_+^(1/(alpha-1) - 1) on the support (the Jacobian
 * Diag(u) - u u^T / |u|_1 of Sec. 3.2.2).  s and tau as given to / returned
 * by the forward; dp, ds fp32 [rows, n].  Same argument rules.
 */
ea_status entmax_rows_bwd(int64_t rows, int32_t n, ea_dtype dtype, const ea_params* params,
                          const void* s, const float* tau, const float* dp, float* ds,
                          void* stream);

/* Static, human-readable name of a status code. */
const char* entmax_attn_status_string(ea_status s);

/* Name of the HIP error (e.g. "hipErrorInvalidConfiguration") behind the calling
 * thread's most recent EA_ERR_HIP, or "" if that thread has seen none. Static
 * storage; the caller does not free it. */
const char* entmax_attn_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ENTMAX_ATTN_H */
