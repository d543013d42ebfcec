/*
 * CPU oracle for MTGR's jagged dynamic-mask HSTU attention and gated Group-LN.
 *
 * TEST INFRASTRUCTURE ONLY: used by tests, the benchmark's CPU-baseline leg and
 * the smoke check; the product library never touches it.  Plain dense loops in
 * double precision, one OpenMP task per (user, head); no blocking, fusion or
 * reordering beyond the definitions below.
 *
 * Parity pins (all in the CPU test-suite): the worked mask example of
 * Sec. 4.2; the all-static, causal and zero-query reductions of Eq. 5 to
 * library routines; autograd of a dense formulation and central finite
 * differences for the backward; torch's layer_norm for Group-LN with one group;
 * an integer table and bit-length identity for the bias bucket.
 */
#include "mtgr_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

enum { SEG_USER = 0, SEG_HIST = 1, SEG_RT = 2, SEG_CAND = 3 };

/* Sec. 4.2, Dynamic Masking.
 *  Rule 1: the static sequence (user features and history) is visible to every token.
 *  Rule 2: a real-time token is visible only to tokens that occur after it in time,
 *          real-time tokens and candidates alike (strictly later: ties are hidden).
 *  Rule 3: a candidate is visible to itself only.
 * A static token comes from before the aggregation window, so it sees only the
 * static sequence (and itself); every token sees itself. */
int mtgr_oracle_visible(int seg_i, int32_t ts_i, int seg_j, int32_t ts_j, int same)
{
    if (same) return 1;
    if (seg_j == SEG_USER || seg_j == SEG_HIST) return 1;                 /* rule 1 */
    if (seg_j == SEG_RT)                                                   /* rule 2 */
        return (seg_i == SEG_RT || seg_i == SEG_CAND) && ts_j < ts_i;
    return 0;                                                              /* rule 3 */
}

/* Half-octave log-time bucket of a gap delta >= 0:
 *   delta < 2           -> delta
 *   2^e <= delta < 2^(e+1), e >= 1
 *       -> 2e     if delta < 1.5 * 2^e
 *       -> 2e + 1 otherwise
 * Every uint32 gap lands in 0..63. */
int mtgr_oracle_rab_bucket(uint32_t delta)
{
    if (delta < 2u) return (int)delta;
    uint64_t g = delta;
    int e = 0;
    while ((g >> (e + 1)) != 0u) e++;          /* e = floor(log2(delta)) */
    uint64_t lo = (uint64_t)1 << e;
    return 2 * e + (g * 2u >= 3u * lo ? 1 : 0);
}

static uint32_t abs_gap(int32_t a, int32_t b)
{
    int64_t d = (int64_t)a - (int64_t)b;
    return (uint32_t)(d < 0 ? -d : d);
}

static int bias_bucket(int32_t ts_i, int32_t ts_j, int32_t nbuckets)
{
    int bk = mtgr_oracle_rab_bucket(abs_gap(ts_i, ts_j));
    return bk < nbuckets ? bk : nbuckets - 1;
}

static double silu(double x) { return x / (1.0 + exp(-x)); }

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

int64_t mtgr_oracle_count_visible(int32_t B, const int64_t* offsets, const int8_t* seg,
                                  const int32_t* ts)
{
    int64_t total = 0;
    for (int32_t b = 0; b < B; b++)
        for (int64_t i = offsets[b]; i < offsets[b + 1]; i++)
            for (int64_t j = offsets[b]; j < offsets[b + 1]; j++)
                total += mtgr_oracle_visible(seg[i], ts[i], seg[j], ts[j], i == j);
    return total;
}

/* Score s_ij of Eq. 5 for head h: alpha * q_i . k_j (+ relative bias). */
static double score(const double* q, const double* k, const double* rab, int32_t nbuckets,
                    const int32_t* ts, int32_t H, int32_t dh, double alpha,
                    int64_t i, int64_t j, int32_t h)
{
    const double* qi = q + ((size_t)i * H + h) * dh;
    const double* kj = k + ((size_t)j * H + h) * dh;
    double dot = 0.0;
    for (int32_t c = 0; c < dh; c++) dot += qi[c] * kj[c];
    double s = alpha * dot;
    if (rab) s += rab[(size_t)h * nbuckets + bias_bucket(ts[i], ts[j], nbuckets)];
    return s;
}

void mtgr_oracle_attn_fwd(int32_t B, const int64_t* offsets, const int8_t* seg, const int32_t* ts,
                          int32_t H, int32_t dh, double alpha,
                          const double* q, const double* k, const double* v,
                          const double* rab, int32_t nbuckets, double* out)
{
    int64_t T = B > 0 ? offsets[B] : 0;
    memset(out, 0, sizeof(double) * (size_t)T * H * dh);
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int32_t b = 0; b < B; b++) {
        for (int32_t h = 0; h < H; h++) {
            int64_t o = offsets[b], n = offsets[b + 1] - offsets[b];
            for (int64_t i = o; i < o + n; i++) {
                double* oi = out + ((size_t)i * H + h) * dh;
                for (int64_t j = o; j < o + n; j++) {
                    if (!mtgr_oracle_visible(seg[i], ts[i], seg[j], ts[j], i == j)) continue;
                    double s = score(q, k, rab, nbuckets, ts, H, dh, alpha, i, j, h);
                    double p = silu(s) / (double)n;          /* divided by the user's length */
                    const double* vj = v + ((size_t)j * H + h) * dh;
                    for (int32_t c = 0; c < dh; c++) oi[c] += p * vj[c];
                }
            }
        }
    }
}

/* Backward of Eq. 5 per visible pair (i, j), with s = s_ij, sg = sigmoid(s):
 *   p = silu(s)/n,  dP = dout_i . v_j,  dS = dP * silu'(s)/n,
 *   silu'(s) = sg * (1 + s * (1 - sg)),
 *   dv_j += p dout_i,  dq_i += alpha dS k_j,  dk_j += alpha dS q_i,
 *   drab[h, bucket(i, j)] += dS. */
void mtgr_oracle_attn_bwd(int32_t B, const int64_t* offsets, const int8_t* seg, const int32_t* ts,
                          int32_t H, int32_t dh, double alpha,
                          const double* q, const double* k, const double* v,
                          const double* rab, int32_t nbuckets, const double* dout,
                          double* dq, double* dk, double* dv, double* drab)
{
    int64_t T = B > 0 ? offsets[B] : 0;
    size_t nel = (size_t)T * H * dh;
    memset(dq, 0, sizeof(double) * nel);
    memset(dk, 0, sizeof(double) * nel);
    memset(dv, 0, sizeof(double) * nel);
    int32_t nb = (rab && drab) ? nbuckets : 0;
    double* part = nb ? (double*)calloc((size_t)B * H * nb, sizeof(double)) : NULL;
    #pragma omp parallel for collapse(2) schedule(dynamic)
    for (int32_t b = 0; b < B; b++) {
        for (int32_t h = 0; h < H; h++) {
            int64_t o = offsets[b], n = offsets[b + 1] - offsets[b];
            double* pb = part ? part + ((size_t)b * H + h) * nb : NULL;
            for (int64_t i = o; i < o + n; i++) {
                const double* doi = dout + ((size_t)i * H + h) * dh;
                const double* qi = q + ((size_t)i * H + h) * dh;
                double* dqi = dq + ((size_t)i * H + h) * dh;
                for (int64_t j = o; j < o + n; j++) {
                    if (!mtgr_oracle_visible(seg[i], ts[i], seg[j], ts[j], i == j)) continue;
                    double s = score(q, k, rab, nbuckets, ts, H, dh, alpha, i, j, h);
                    double sg = sigmoid(s);
                    double p = s * sg / (double)n;
                    const double* vj = v + ((size_t)j * H + h) * dh;
                    const double* kj = k + ((size_t)j * H + h) * dh;
                    double* dkj = dk + ((size_t)j * H + h) * dh;
                    double* dvj = dv + ((size_t)j * H + h) * dh;
                    double dP = 0.0;
                    for (int32_t c = 0; c < dh; c++) dP += doi[c] * vj[c];
                    double dS = dP * sg * (1.0 + s * (1.0 - sg)) / (double)n;
                    for (int32_t c = 0; c < dh; c++) {
                        dvj[c] += p * doi[c];
                        dqi[c] += alpha * dS * kj[c];
                        dkj[c] += alpha * dS * qi[c];
                    }
                    if (pb) pb[bias_bucket(ts[i], ts[j], nbuckets)] += dS;
                }
            }
        }
    }
    if (drab && rab) {
        memset(drab, 0, sizeof(double) * (size_t)H * nbuckets);
        for (int32_t b = 0; b < B; b++)
            for (int32_t h = 0; h < H; h++)
                for (int32_t x = 0; x < nb; x++)
                    drab[(size_t)h * nbuckets + x] += part[((size_t)b * H + h) * nb + x];
    }
    free(part);
}

/* Eq. 6 without the MLP and residual: y = GroupLN(x (*) u).  One LayerNorm per
 * token over its d features (biased variance), with the affine parameters of
 * the token's group. */
void mtgr_oracle_gln_fwd(int64_t T, int32_t d, int32_t G, double eps,
                         const double* x, const double* u, const int8_t* gid,
                         const double* gamma, const double* beta,
                         double* y, double* mean, double* rstd)
{
    (void)G;
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; t++) {
        const double* xt = x + (size_t)t * d;
        const double* ut = u ? u + (size_t)t * d : NULL;
        double* z = (double*)malloc(sizeof(double) * (size_t)d);
        double mu = 0.0, var = 0.0;
        for (int32_t c = 0; c < d; c++) { z[c] = ut ? xt[c] * ut[c] : xt[c]; mu += z[c]; }
        mu /= d;
        for (int32_t c = 0; c < d; c++) var += (z[c] - mu) * (z[c] - mu);
        var /= d;
        double r = 1.0 / sqrt(var + eps);
        const double* ga = gamma + (size_t)gid[t] * d;
        const double* be = beta + (size_t)gid[t] * d;
        for (int32_t c = 0; c < d; c++) y[(size_t)t * d + c] = ga[c] * (z[c] - mu) * r + be[c];
        if (mean) mean[t] = mu;
        if (rstd) rstd[t] = r;
        free(z);
    }
}

/* LayerNorm backward with zhat = (z - mean) rstd and g = dy (*) gamma[g_t]:
 *   dz = rstd (g - mean(g) - zhat mean(g (*) zhat)),
 *   dx = dz (*) u, du = dz (*) x,
 *   dgamma[g] = sum over the group's tokens of dy (*) zhat, dbeta[g] = sum of dy. */
void mtgr_oracle_gln_bwd(int64_t T, int32_t d, int32_t G, double eps,
                         const double* x, const double* u, const int8_t* gid,
                         const double* gamma, const double* dy,
                         double* dx, double* du, double* dgamma, double* dbeta)
{
    double* zhat = (double*)malloc(sizeof(double) * (size_t)(T > 0 ? T : 1) * d);
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; t++) {
        const double* xt = x + (size_t)t * d;
        const double* ut = u ? u + (size_t)t * d : NULL;
        const double* dyt = dy + (size_t)t * d;
        const double* ga = gamma + (size_t)gid[t] * d;
        double* zh = zhat + (size_t)t * d;
        double mu = 0.0, var = 0.0;
        for (int32_t c = 0; c < d; c++) { zh[c] = ut ? xt[c] * ut[c] : xt[c]; mu += zh[c]; }
        mu /= d;
        for (int32_t c = 0; c < d; c++) var += (zh[c] - mu) * (zh[c] - mu);
        var /= d;
        double r = 1.0 / sqrt(var + eps);
        for (int32_t c = 0; c < d; c++) zh[c] = (zh[c] - mu) * r;
        double m1 = 0.0, m2 = 0.0;
        for (int32_t c = 0; c < d; c++) { double g = dyt[c] * ga[c]; m1 += g; m2 += g * zh[c]; }
        m1 /= d;
        m2 /= d;
        for (int32_t c = 0; c < d; c++) {
            double dz = r * (dyt[c] * ga[c] - m1 - zh[c] * m2);
            dx[(size_t)t * d + c] = ut ? dz * ut[c] : dz;
            if (du && ut) du[(size_t)t * d + c] = dz * xt[c];
        }
    }
    memset(dgamma, 0, sizeof(double) * (size_t)G * d);
    memset(dbeta, 0, sizeof(double) * (size_t)G * d);
    for (int64_t t = 0; t < T; t++) {
        const double* dyt = dy + (size_t)t * d;
        const double* zh = zhat + (size_t)t * d;
        double* dg = dgamma + (size_t)gid[t] * d;
        double* db = dbeta + (size_t)gid[t] * d;
        for (int32_t c = 0; c < d; c++) { dg[c] += dyt[c] * zh[c]; db[c] += dyt[c]; }
    }
    free(zhat);
}
