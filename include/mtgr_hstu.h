/*
 * mtgr_hstu.h — C ABI of the MI355X (gfx950) implementation of MTGR's jagged
 * dynamic-mask HSTU attention and the gated Group-LayerNorm that follows it
 * (MTGR, arXiv 2505.18654, Sec. 4.2, Eq. 5 and Eq. 6).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is DEVICE memory owned by the caller (borrowed; the
 *     library keeps no reference after the call returns).  The library never
 *     allocates device memory and never synchronises the stream.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null stream).
 *   - Outputs are overwritten, never accumulated into (this includes the
 *     parameter gradients dgamma, dbeta and drab).
 *   - On any status other than MTGR_SUCCESS nothing has been launched and every
 *     output is untouched, except MTGR_ERROR_DEVICE, which reports a failed
 *     launch (outputs then undefined).  mtgr_last_error_message() names the
 *     offending argument.
 *   - Jagged batches: user b owns tokens offsets[b] .. offsets[b+1]-1 of a
 *     [T, ...] tensor.  offsets (int32, B+1 entries, device) must satisfy
 *     offsets[0] = 0, offsets[b] <= offsets[b+1], offsets[B] = total_tokens and
 *     offsets[b+1] - offsets[b] <= max_seqlen; seg[t] must lie in 0..3 and
 *     group ids in 0..G-1.  These device-resident preconditions are not checked
 *     by the hot-path calls (checking them would need a synchronisation);
 *     violating them is undefined.  mtgr_debug_validate_inputs checks them.
 *   - B = 0 or T = 0 is a successful no-op (outputs of size zero; parameter
 *     gradients are zero-filled).
 *   - Every function is stateless and may be called concurrently from several
 *     host threads.
 */
#ifndef MTGR_HSTU_H
#define MTGR_HSTU_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MTGR_HSTU_VERSION 100           /* major * 100 + minor */

typedef enum {
    MTGR_SUCCESS = 0,
    MTGR_ERROR_NULL_POINTER = 1,        /* a required pointer is NULL */
    MTGR_ERROR_INVALID_ARGUMENT = 2,    /* a size, stride or alignment is invalid */
    MTGR_ERROR_UNSUPPORTED = 3,         /* valid but not implemented (head_dim, dtype, ...) */
    MTGR_ERROR_WORKSPACE_TOO_SMALL = 4, /* workspace_bytes below the queried size */
    MTGR_ERROR_DEVICE = 5               /* a HIP call or kernel launch failed */
} mtgr_status_t;

typedef enum {
    MTGR_DTYPE_BF16 = 0,                /* bf16 storage, fp32 accumulation */
    MTGR_DTYPE_FP32 = 1                 /* fp32 storage and arithmetic (parity mode) */
} mtgr_dtype_t;

/* Token segments of the sequence [U | S | R | I] (Sec. 4.1, Eq. 4). */
enum {
    MTGR_SEG_USER = 0,                  /* user-feature token (static) */
    MTGR_SEG_HIST = 1,                  /* history item (static) */
    MTGR_SEG_RT = 2,                    /* real-time item (dynamic) */
    MTGR_SEG_CAND = 3                   /* candidate (cross + item features) */
};

/* Bits of mtgr_hstu_problem_t.flags. */
#define MTGR_ATTN_PLANNED 1u   /* the workspace already holds this batch's plan
                                  (mtgr_hstu_attn_plan); skip rebuilding it */
#define MTGR_BWD_SKIP_DQ 2u    /* backward: do not form dq (dq may be NULL) */
#define MTGR_BWD_SKIP_DKDV 4u  /* backward: do not form dk, dv (both may be NULL) */
#define MTGR_BWD_KEEP_DS 8u    /* backward with MTGR_BWD_SKIP_DQ: also leave dS in the
                                  workspace (needs the backward = 1 workspace size) for a
                                  later dq-only call with MTGR_BWD_DS_READY */
#define MTGR_BWD_DS_READY 16u  /* backward with MTGR_BWD_SKIP_DKDV: form dq from the dS that
                                  a previous MTGR_BWD_KEEP_DS call left in this workspace for
                                  the same batch, plan and inputs; drab must be NULL (that
                                  call formed it) */
#define MTGR_FWD_CAND_ROWS 32u /* forward only: form and write only the output rows of
                                  candidate tokens (seg = MTGR_SEG_CAND); every other row of
                                  out is left untouched.  Work is skipped for 128-row query
                                  tiles without a candidate.  Not valid for the backward. */

#define MTGR_MAX_RAB_BUCKETS 64
#define MTGR_MAX_HEADS 255
#define MTGR_MAX_GROUPS 127
#define MTGR_MAX_LD (1ll << 24)   /* largest attention token stride (elements); larger strides
                                     return MTGR_ERROR_UNSUPPORTED */

typedef void* mtgr_stream_t;            /* hipStream_t */

/* Shape of one attention call.
 *   num_users B >= 0, total_tokens T >= 0 (T < 2^31), max_seqlen >= every user's length.
 *   num_heads H in 1..255; head_dim dh in {16, 32, 64, 128} for both dtypes.  bf16 at
 *     dh = 32..128 runs on the bf16 matrix cores; bf16 at dh = 16 runs on vector-ALU kernels
 *     with bf16 storage and fp32 arithmetic (a pair then holds 64 flop of products against
 *     the SiLU's transcendental work, so the matrix cores would not pay), as does fp32.
 *   A problem whose work list would reach 2^24 workgroups returns MTGR_ERROR_UNSUPPORTED
 *     (one launch holds at most 2^32 - 1 work-items).
 *   alpha: multiplier of q.k inside the SiLU (Eq. 5 has none: pass 1.0).
 *   num_rab_buckets: 0 = no relative bias, else 1..64 (rab is [H][num_rab_buckets] fp32;
 *     a gap whose log-time bucket is >= num_rab_buckets uses the last bucket).
 *   ld_*: token strides in ELEMENTS (>= H*dh, <= MTGR_MAX_LD); q, k, v may be views into one fused
 *     projection output.  Gradients share the layout of their primal:
 *     dq uses ld_q, dk ld_k, dv ld_v, and dout uses ld_o.
 *   flags: MTGR_ATTN_PLANNED, MTGR_BWD_SKIP_DQ / _DKDV, MTGR_BWD_KEEP_DS / _DS_READY,
 *     MTGR_FWD_CAND_ROWS (see their definitions above).
 * Alignment: every tensor pointer 16-byte aligned; every ld a multiple of 16 bytes. */
typedef struct {
    int32_t num_users;
    int32_t max_seqlen;
    int64_t total_tokens;
    int32_t num_heads;
    int32_t head_dim;
    int32_t dtype;                      /* mtgr_dtype_t */
    float alpha;
    int32_t num_rab_buckets;
    uint32_t flags;                     /* MTGR_ATTN_PLANNED, MTGR_BWD_*, MTGR_FWD_* bits (0 = none) */
    int64_t ld_q, ld_k, ld_v, ld_o;
} mtgr_hstu_problem_t;

/* Shape of one gate + Group-LN call.
 *   num_tokens T in 0 .. 2^28 - 1, dim d (bf16: multiple of 8 and <= 4096; fp32: multiple of 4
 *   and <= 2048),
 *   num_groups G in 1..127, eps > 0.
 *   ld_*: token strides in elements (>= d).  Gradients share the layout of their
 *   primal: dx uses ld_x, du ld_u, dy ld_y. */
typedef struct {
    int64_t num_tokens;
    int32_t dim;
    int32_t num_groups;
    int32_t dtype;                      /* mtgr_dtype_t */
    float eps;
    int64_t ld_x, ld_u, ld_y;
} mtgr_gln_problem_t;

/* Bytes of device workspace for problem `p`.  Pure host arithmetic.
 *   backward = 0: the plan; enough for mtgr_hstu_attn_plan, _fwd and a backward that
 *     recomputes S and dP in its dq kernel.
 *   backward = 1: the plan plus room for dS as bf16 64 x 64 blocks (an upper bound of
 *     H * sum_b ceil(n_b / 64)^2 blocks of 8 KB, from T, B and max_seqlen).  With it the
 *     bf16 backward stores dS from its dk/dv kernel and forms dq from it (fewer operations;
 *     the same dS operand, so dq differs from the recomputing form only in the order of its
 *     float sums).  The first bytes have the backward = 0 layout, so one plan serves.
 *     For fp32 and for bf16 at head_dim 16 (vector-ALU kernels) both sizes are equal. */
mtgr_status_t mtgr_hstu_attn_workspace_size(const mtgr_hstu_problem_t* p, int backward,
                                            size_t* bytes);

/* Builds the batch plan into `workspace`: per 64-token tile of every user, the segment
 * flags and time range that classify each (query tile, key tile) pair as fully visible,
 * partially visible or fully masked under the dynamic mask (Sec. 4.2), and a work list of
 * (user, head, tile) items ordered longest user first.  The plan depends only on
 * offsets, seg, ts and the problem shape, so one plan serves every forward and backward
 * call on the same batch (all layers of the encoder) when they pass MTGR_ATTN_PLANNED.
 * Without that flag, mtgr_hstu_attn_fwd/bwd rebuild the plan themselves. */
mtgr_status_t mtgr_hstu_attn_plan(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                  const int8_t* seg, const int32_t* ts, void* workspace,
                                  size_t workspace_bytes, mtgr_stream_t stream);

/* Forward of Eq. 5 (Sec. 4.2) for every user b, head h and token i of b:
 *   out[i,h,:] = sum over tokens j of b with M_ij = 1 of
 *                silu(alpha * q[i,h,:].k[j,h,:] + rab[h, bucket(|ts_i - ts_j|)]) / n_b * v[j,h,:]
 * where n_b is the user's token count (candidates included) and M is the
 * dynamic mask of Sec. 4.2 ("Dynamic Masking"), evaluated from seg and ts:
 *   M_ij = 1 iff i == j, or seg_j is USER/HIST (static, rule 1), or seg_j is RT and
 *   seg_i is RT/CAND and ts_j < ts_i (rule 2); candidates are seen only by
 *   themselves (rule 3).
 * The bias term is present only when rab != NULL (requires num_rab_buckets > 0); its values
 * must be finite and below 1e29 in magnitude (the bf16 forward hides masked pairs by driving
 * alpha * s + rab to about -1e30 when |alpha| >= 1e-7);
 * bucket(g) = g for g < 2, else 2e + [g >= 1.5 * 2^e] with e = floor(log2 g), g as uint32.
 *   offsets [B+1] int32, seg [T] int8, ts [T] int32 (seconds; any epoch).
 *   q, k, v [T, H, dh] (dtype), out [T, H, dh] (dtype, stride ld_o).
 *   workspace: at least mtgr_hstu_attn_workspace_size(p, 0) bytes, 256-byte aligned.
 * With MTGR_FWD_CAND_ROWS only the candidates' rows are formed: the one pass per user that
 * scores all of its candidates (user sample aggregation, Sec. 4.1, Eq. 3), e.g. at serving
 * time when the user-side rows of the layer are not needed.  Each candidate row is the same
 * as in a full forward of the batch (n_b still counts every token of the user). */
mtgr_status_t mtgr_hstu_attn_fwd(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                 const int8_t* seg, const int32_t* ts, const void* q,
                                 const void* k, const void* v, const float* rab, void* out,
                                 void* workspace, size_t workspace_bytes, mtgr_stream_t stream);

/* Serving with the user side cached across requests (user sample aggregation, Sec. 4.1, Eq. 3;
 * its serving cost, Sec. 6.5).  Candidates see the static tokens, the real-time tokens earlier
 * than themselves, and themselves only (Sec. 4.2), and no user-side token sees a candidate, so
 * a user's user-side keys and values (U | S | R) can be held by the caller across requests and
 * each request brings only its candidates.  For every user b and candidate i of the request:
 *   out[i,h,:] = ( sum over cached tokens j of b with M_ij = 1 of p_ij vc[j,h,:]  +  p_ii v[i,h,:] )
 * with p_ij = silu(alpha q_i.kc_j + rab[h, bucket(|ts_i - ts_c[j]|)]) / n_b,
 *      p_ii = silu(alpha q_i.k_i + rab[h, 0]) / n_b,  n_b = cached tokens of b + candidates of b
 * (every token of the user, as in mtgr_hstu_attn_fwd), M_ij the mask of Sec. 4.2 from the
 * cached tokens' segments (in the cache plan) and timestamps.  This equals the candidate rows
 * of mtgr_hstu_attn_fwd on the concatenated sequence [cached | candidates] up to the order of
 * the float sums.  (The user side of the first layer depends only on the user; at deeper layers
 * it also depends on n_b, so a cache serves requests with the same candidate count.)
 *   p: the request: B users, T = all candidates, max_seqlen >= candidates of any user; its
 *     tokens should be candidates (seg = MTGR_SEG_CAND); q, k, v, out [T, H, dh] bf16.
 *     head_dim 32, 64 or 128 (bf16 matrix cores; other shapes MTGR_ERROR_UNSUPPORTED).
 *     Only MTGR_ATTN_PLANNED may be set (the request's plan in workspace).
 *   pc: the cache: the same B, num_heads, head_dim and dtype; total_tokens, max_seqlen of the
 *     cached tokens; ld_k / ld_v are the token strides of kc / vc.
 *   offsets_c [B+1], ts_c [Tc] int32; kc, vc [Tc, H, dh] bf16 (device).
 *   cache_plan: a workspace of at least mtgr_hstu_attn_workspace_size(pc, 0) bytes that
 *     mtgr_hstu_attn_plan(pc, offsets_c, seg_c, ts_c, ...) filled (once per cache contents).
 *   workspace: at least mtgr_hstu_attn_workspace_size(p, 0) bytes (the request's plan). */
mtgr_status_t mtgr_hstu_attn_fwd_cached(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                        const int8_t* seg, const int32_t* ts, const void* q,
                                        const void* k, const void* v, const float* rab, void* out,
                                        const mtgr_hstu_problem_t* pc, const int32_t* offsets_c,
                                        const int32_t* ts_c, const void* kc, const void* vc,
                                        const void* cache_plan, size_t cache_plan_bytes,
                                        void* workspace, size_t workspace_bytes,
                                        mtgr_stream_t stream);

/* Bytes of the per-GPU device array that holds the plan of mtgr_hstu_attn_fwd_noalloc. */
#define MTGR_NOALLOC_SCRATCH_BYTES (16u * 1024u * 1024u)

/* For callers that cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  mtgr_hstu_attn_fwd without a workspace: the plan (tile
 * summaries, work list, token codes) is built on every call into a file-scope device array of
 * the library, MTGR_NOALLOC_SCRATCH_BYTES on each GPU it runs on, kept until the process ends.
 * Same arguments and results as mtgr_hstu_attn_fwd otherwise (same kernels and plan, so the
 * output is bit for bit that of mtgr_hstu_attn_fwd).
 *   - Calls nothing that allocates (no hipMalloc / hipFree).  Its first call on a device looks
 *     up that device's array address (hipGetSymbolAddress), with that device current.
 *   - stream must belong to the current device (MTGR_ERROR_INVALID_ARGUMENT otherwise).
 *   - Every call on one GPU shares that GPU's array, which keeps the last call's plan: calls
 *     that overlap on one GPU (different streams, or host threads) race and give undefined
 *     output; order them on one stream.
 *   - A problem whose plan (mtgr_hstu_attn_workspace_size(p, 0)) exceeds
 *     MTGR_NOALLOC_SCRATCH_BYTES returns MTGR_ERROR_UNSUPPORTED before any launch (the five
 *     workloads of the benchmark need at most 7.4 MB: 1024 users, 1.5M tokens, 6 heads).
 *   - MTGR_ATTN_PLANNED is rejected (MTGR_ERROR_INVALID_ARGUMENT): there is no plan kept for
 *     the caller between calls. */
mtgr_status_t mtgr_hstu_attn_fwd_noalloc(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                         const int8_t* seg, const int32_t* ts, const void* q,
                                         const void* k, const void* v, const float* rab, void* out,
                                         mtgr_stream_t stream);

/* Backward of Eq. 5: given dout = dL/dout, writes dq, dk, dv (same dtype and
 * layout as q, k, v) and, when drab != NULL, drab = dL/drab ([H][num_rab_buckets]
 * fp32; requires rab != NULL).  With s = alpha q.k + rab, sg = sigmoid(s):
 *   dS_ij = M_ij (dout_i . v_j) sg (1 + s (1 - sg)) / n_b,
 *   dv_j = sum_i M_ij silu(s_ij)/n_b dout_i,  dq_i = alpha sum_j dS_ij k_j,
 *   dk_j = alpha sum_i dS_ij q_i,  drab[h, x] = sum over pairs in bucket x of dS_ij.
 * The forward saves nothing (no softmax statistics), so the same inputs are passed.
 * Two kernels, no atomics on dq/dk/dv (results are deterministic):
 *   - workspace of at least mtgr_hstu_attn_workspace_size(p, 1) bytes (bf16): the dk/dv
 *     kernel also stores dS (bf16, the operand of its dk product) in the workspace and a
 *     second kernel forms dq = alpha sum_j dS_ij k_j from it;
 *   - otherwise (at least the backward = 0 size; always for fp32): the dq kernel
 *     recomputes S, dP and dS itself.
 * MTGR_BWD_SKIP_DQ / _DKDV form only one side; with MTGR_BWD_KEEP_DS / _DS_READY the two
 * halves of the stored-dS path can be issued as two calls.  drab is formed by the call
 * that runs the dk/dv kernel, or by a dq-only call without MTGR_BWD_DS_READY (fp32: by the
 * call that forms dq). */
mtgr_status_t mtgr_hstu_attn_bwd(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                 const int8_t* seg, const int32_t* ts, const void* q,
                                 const void* k, const void* v, const float* rab,
                                 const void* dout, void* dq, void* dk, void* dv, float* drab,
                                 void* workspace, size_t workspace_bytes, mtgr_stream_t stream);

/* Bytes of device workspace for the Group-LN calls: 0 for the forward; the backward
 * keeps per-workgroup dgamma/dbeta partials (about 512 x 2 G d floats at most). */
mtgr_status_t mtgr_group_layernorm_workspace_size(const mtgr_gln_problem_t* p, int backward,
                                                  size_t* bytes);

/* Eq. 6 up to the MLP (Sec. 4.2): y = GroupLN(x (*) u) per token t:
 *   z = x[t] (*) u[t]  (u == NULL: z = x[t], the input Group-LN before the projections)
 *   mean[t] = mean(z), rstd[t] = 1/sqrt(mean((z - mean)^2) + eps)  (biased variance)
 *   y[t] = gamma[g] (*) (z - mean[t]) rstd[t] + beta[g],  g = group_ids[t].
 *   x, u, y [T, d] (dtype); group_ids [T] int8; gamma, beta [G][d] fp32;
 *   mean, rstd [T] fp32 (may be NULL when not needed for a backward). */
mtgr_status_t mtgr_group_layernorm_fwd(const mtgr_gln_problem_t* p, const void* x, const void* u,
                                       const int8_t* group_ids, const float* gamma,
                                       const float* beta, void* y, float* mean, float* rstd,
                                       mtgr_stream_t stream);

/* Backward of mtgr_group_layernorm_fwd, using its saved mean and rstd:
 *   with zhat = (z - mean) rstd and g = dy (*) gamma[g_t]:
 *   dz = rstd (g - mean(g) - zhat mean(g (*) zhat)),  dx = dz (*) u,  du = dz (*) x,
 *   dgamma[g] = sum over tokens of group g of dy (*) zhat,  dbeta[g] = sum of dy.
 *   du must be non-NULL iff u is non-NULL.  dgamma, dbeta [G][d] fp32 are
 *   overwritten: summed per workgroup (LDS atomics among its waves, order not fixed),
 *   then over workgroups in a fixed order.  workspace: at least
 *   mtgr_group_layernorm_workspace_size(p, 1) bytes, 16-byte aligned. */
mtgr_status_t mtgr_group_layernorm_bwd(const mtgr_gln_problem_t* p, const void* dy, const void* x,
                                       const void* u, const int8_t* group_ids, const float* gamma,
                                       const float* mean, const float* rstd, void* dx, void* du,
                                       float* dgamma, float* dbeta, void* workspace,
                                       size_t workspace_bytes, mtgr_stream_t stream);

/* Projection activation of the encoder layer built around the attention (Sec. 4.2: the
 * Group-LN'd input is projected to K, Q, V, U by MLPs; read here as one fused linear map
 * followed by SiLU, as in HSTU, with the GEMM left to a BLAS library):
 *   out[r, c] = silu(h[r, c] + bias[c])        (bias may be NULL: no bias)
 *   h, out [rows, cols] (dtype), row strides ld_h, ld_out in elements (>= cols; out may be h
 *   with ld_out = ld_h); bias [cols] fp32.  cols a multiple of 8 (bf16) or 4 (fp32); h, out
 *   16-byte aligned and their rows too (ld * element size a multiple of 16). */
mtgr_status_t mtgr_bias_silu_fwd(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* h,
                                 int64_t ld_h, const float* bias, void* out, int64_t ld_out,
                                 mtgr_stream_t stream);

/* Backward of mtgr_bias_silu_fwd:
 *   dh[r, c] = dout[r, c] * silu'(z),  z = h[r, c] + bias[c],
 *   silu'(z) = s (1 + z (1 - s)),  s = 1 / (1 + exp(-z)).
 * Same layout rules as the forward (dh may be dout with equal strides); the bias gradient
 * (the column sums of dh) is left to the caller. */
mtgr_status_t mtgr_bias_silu_bwd(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* h,
                                 int64_t ld_h, const float* bias, const void* dout, int64_t ld_dout,
                                 void* dh, int64_t ld_dh, mtgr_stream_t stream);

/* Elementwise out = a + b on [rows, cols] (the residual branch of the encoder layer's
 * backward); the same layout rules as mtgr_bias_silu_fwd (out may be a or b). */
mtgr_status_t mtgr_add(int64_t rows, int32_t cols, mtgr_dtype_t dtype, const void* a, int64_t ld_a,
                       const void* b, int64_t ld_b, void* out, int64_t ld_out, mtgr_stream_t stream);

/* Dense bf16 products of the encoder layer built around the attention (Sec. 4.2: the MLPs that
 * project the Group-LN'd input to K, Q, V, U, read as one fused linear map followed by SiLU, and
 * the top MLP of Eq. 6 read as one linear map plus the residual), fp32 accumulation on the bf16
 * matrix cores, with the layer's elementwise work fused into the product:
 *   layout MTGR_GEMM_NN: C[M,N] = A B,    A [M,K] (lda >= K), B [K,N] (ldb >= N)
 *          MTGR_GEMM_NT: C[M,N] = A B^T,  A [M,K], B [N,K] (ldb >= K)   (input gradients)
 *          MTGR_GEMM_TN: C[M,N] = A^T B,  A [K,M] (lda >= M), B [K,N]   (weight gradients;
 *            colsum, if not NULL, receives the column sums of B over K as fp32 [N]: the bias
 *            gradient; needs the workspace of mtgr_gemm_workspace_size)
 *   epilogue MTGR_GEMM_EPI_NONE:          C = AB
 *            MTGR_GEMM_EPI_BIAS_SILU:     C = AB (pre-activation), C2 = silu(AB + bias)
 *            MTGR_GEMM_EPI_BIAS_RESIDUAL: C = AB + bias + R
 *     (bias [N] fp32, 16-byte aligned; R, C2 [M,N] bf16 with strides ldr, ldc2; TN takes only
 *     MTGR_GEMM_EPI_NONE)
 * All matrices bf16 row-major with element strides; pointers 16-byte aligned, strides multiples
 * of 8 elements and below 2^22.  Shapes: K >= 1; N a multiple of 8; K a multiple of 32 for
 * NN / NT (any K for TN); M a multiple of 8 for TN (any M for NN / NT).  Other shapes return
 * MTGR_ERROR_UNSUPPORTED; M = 0 or N = 0 does nothing.  The TN sums over K are split into fp32 partials that are added in a
 * fixed order (the result is deterministic). */
#define MTGR_GEMM_NN 0
#define MTGR_GEMM_NT 1
#define MTGR_GEMM_TN 2
#define MTGR_GEMM_EPI_NONE 0
#define MTGR_GEMM_EPI_BIAS_SILU 1
#define MTGR_GEMM_EPI_BIAS_RESIDUAL 2
mtgr_status_t mtgr_gemm_workspace_size(int32_t layout, int64_t M, int64_t N, int64_t K, size_t* bytes);
mtgr_status_t mtgr_gemm_bf16(int32_t layout, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                             const void* B, int64_t ldb, void* C, int64_t ldc, int32_t epilogue,
                             const float* bias, const void* R, int64_t ldr, void* C2, int64_t ldc2,
                             float* colsum, void* workspace, size_t workspace_bytes,
                             mtgr_stream_t stream);

/* Measurement aid (no part of the method): the shader clock while the matrix cores are busy.
 * Launches `blocks` workgroups of 256 threads that each issue `mfma_iterations` x 4
 * v_mfma_f32_32x32x16_bf16 per wave back to back, and writes per workgroup
 * out[3 b] = shader-clock cycles and out[3 b + 1] = constant-rate counter ticks around that
 * loop (out[3 b + 2] is a checksum), device memory, int64, 3 * blocks entries.
 * *wall_clock_khz (host) receives the constant counter's rate; the clock in kHz is
 * out[3 b] / out[3 b + 1] * *wall_clock_khz.  blocks in [1, 65536]. */
mtgr_status_t mtgr_debug_clock_probe(int32_t mfma_iterations, int32_t blocks, int64_t* out,
                                     int32_t* wall_clock_khz, mtgr_stream_t stream);

/* Bytes of device scratch that mtgr_debug_validate_inputs needs. */
#define MTGR_VALIDATE_SCRATCH_BYTES 64

/* Debugging aid, not for the hot path: checks the device-resident preconditions that the
 * other calls assume of a jagged batch (the layout of Sec. 4.1, Eq. 3 and Eq. 4) and
 * WAITS for the result (it synchronises `stream`).
 *   offsets [B+1] int32: offsets[0] = 0, offsets[b] <= offsets[b+1], offsets[B] = T and
 *     offsets[b+1] - offsets[b] <= max_seqlen, with B, T, max_seqlen from `p`;
 *   seg [T] int8 in 0..3 (MTGR_SEG_*);
 *   group_ids [T] int8 in 0..num_groups-1, checked only when group_ids is not NULL.
 * scratch: device memory of at least MTGR_VALIDATE_SCRATCH_BYTES, 8-byte aligned; its
 * contents are overwritten.  Returns MTGR_SUCCESS when every condition holds, else
 * MTGR_ERROR_INVALID_ARGUMENT with mtgr_last_error_message() naming the first index of each
 * violated condition.  Only p->num_users, p->total_tokens and p->max_seqlen are read.
 * Reads offsets[0..B] and seg[0..T-1] (group_ids[0..T-1]) only, so invalid values cannot
 * make it read out of bounds. */
mtgr_status_t mtgr_debug_validate_inputs(const mtgr_hstu_problem_t* p, const int32_t* offsets,
                                         const int8_t* seg, const int8_t* group_ids,
                                         int32_t num_groups, void* scratch, size_t scratch_bytes,
                                         mtgr_stream_t stream);

/* Static string for a status code. */
const char* mtgr_status_string(mtgr_status_t status);

/* Message of the last failing call on the calling host thread ("" if none). */
const char* mtgr_last_error_message(void);

/* MTGR_HSTU_VERSION of the loaded library. */
int32_t mtgr_version(void);

#ifdef __cplusplus
}
#endif
#endif /* MTGR_HSTU_H */
