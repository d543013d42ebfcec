/*
 * CPU oracle for MTGR's jagged dynamic-mask HSTU attention and the gated
 * Group-LayerNorm that follows it (MTGR, arXiv 2505.18654, Sec. 4.2).
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, obviously-correct fp64
 * reference used by the test-suite, the benchmark's CPU-baseline leg and the
 * smoke check.  The product library never links, loads or calls it, and it
 * shares no code, header, table or constant with the HIP implementation.
 *
 * Conventions
 *   - Host pointers; every floating-point tensor is double, densely packed.
 *   - Jagged users: offsets[B+1] (int64, offsets[0] = 0, non-decreasing);
 *     user b owns tokens offsets[b] .. offsets[b+1]-1, n_b = its length.
 *   - seg[T] in {0 user-feature, 1 history, 2 real-time, 3 candidate}; ts[T] int32.
 *   - q, k, v, out, dout, dq, dk, dv: [T][H][dh].  x, u, y, dy, dx, du: [T][d].
 *   - rab: [H][nbuckets] or NULL.  gamma, beta, dgamma, dbeta: [G][d].
 */
#ifndef MTGR_ORACLE_H
#define MTGR_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Dynamic mask (Sec. 4.2, "Dynamic Masking", its three rules): may query token
 * i use key token j?  `same` is nonzero when i and j are the same token. */
int mtgr_oracle_visible(int seg_i, int32_t ts_i, int seg_j, int32_t ts_j, int same);

/* Log-time bucket of a time gap (relative bias; not in the paper, see the
 * bucket definition in the source). */
int mtgr_oracle_rab_bucket(uint32_t delta);

/* Number of visible (i, j) pairs of the whole batch. */
int64_t mtgr_oracle_count_visible(int32_t B, const int64_t* offsets, const int8_t* seg,
                                  const int32_t* ts);

/* Eq. 5: out_i = sum_j M_ij * silu(alpha q_i.k_j + rab) / n_b * v_j, per head. */
void mtgr_oracle_attn_fwd(int32_t B, const int64_t* offsets, const int8_t* seg, const int32_t* ts,
                          int32_t H, int32_t dh, double alpha,
                          const double* q, const double* k, const double* v,
                          const double* rab, int32_t nbuckets, double* out);

/* Chain rule of Eq. 5.  drab may be NULL (then rab's gradient is not formed). */
void mtgr_oracle_attn_bwd(int32_t B, const int64_t* offsets, const int8_t* seg, const int32_t* ts,
                          int32_t H, int32_t dh, double alpha,
                          const double* q, const double* k, const double* v,
                          const double* rab, int32_t nbuckets, const double* dout,
                          double* dq, double* dk, double* dv, double* drab);

/* Eq. 6 (gate then Group-LN): z = x (*) u (u may be NULL: plain Group-LN),
 * y = gamma[g] (*) (z - mean) * rstd + beta[g], g = gid[t]. */
void mtgr_oracle_gln_fwd(int64_t T, int32_t d, int32_t G, double eps,
                         const double* x, const double* u, const int8_t* gid,
                         const double* gamma, const double* beta,
                         double* y, double* mean, double* rstd);

void mtgr_oracle_gln_bwd(int64_t T, int32_t d, int32_t G, double eps,
                         const double* x, const double* u, const int8_t* gid,
                         const double* gamma, const double* dy,
                         double* dx, double* du, double* dgamma, double* dbeta);

#ifdef __cplusplus
}
#endif
#endif
