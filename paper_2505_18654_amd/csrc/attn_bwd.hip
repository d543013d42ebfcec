// Backward of the jagged dynamic-mask SiLU attention (chain rule of Eq. 5).
//
// With s = alpha q_i.k_j + rab, sg = sigmoid(s), p = silu(s)/n_b and dP = dout_i . v_j:
//     dS_ij = M_ij dP_ij sg (1 + s (1 - sg)) / n_b
//     dV_j = sum_i M_ij p_ij dout_i,   dK_j = alpha sum_i dS_ij q_i,
//     dQ_i = alpha sum_j dS_ij k_j,    drab[h, bucket] += dS_ij.
// There is no softmax, so nothing is saved by the forward and no row statistic is needed.
//
// No atomics on dQ/dK/dV (results are deterministic).  Two bf16 paths:
//   stored dS (workspace of the backward size):
//     dkdv kernel (column-parallel): per wave 32 keys; the workgroup's 128 keys of K sit in LDS
//       and V in VGPRs; the visible queries stream through LDS 32 at a time (Q, dO, codes,
//       double-buffered).  Per unit: S = Q K^T, dP = dO V^T (lane = key column), then
//       dV += P^T dO and dK += dS^T Q with dO and Q read transposed from their row-major
//       tiles.  It writes dS (bf16, exactly the operand of its dK product, without 1 / n_b) as
//       64 x 64 blocks in its register-fragment order (512 contiguous bytes per store) and
//       forms drab (per-lane runs of equal buckets into an LDS histogram, one global atomic
//       per bucket per workgroup).
//     dq-from-dS kernel (row-parallel): dQ^T += K^T dS^T from K tiles and the stored blocks,
//       16 MFMAs per 32 x 64 tile and no elementwise work.
//   recompute (smaller workspace, or a dq-only call): the dq kernel (row-parallel, like the
//     forward) keeps Q and dO in VGPRs, streams K and V tiles, recomputes S^T = K Q^T,
//     dP^T = V dO^T and dS^T in registers, and forms dQ^T += K^T dS^T with K^T read by
//     ds_read_b64_tr_b16; the dkdv kernel is the same as above without the dS store.
#include <type_traits>

#include "attn_bwd_common.h"

namespace mtgr {

namespace {
using bwd::BM;
using bwd::BN;
}  // namespace

// ------------------------------------------------------------------ vector-ALU kernels
// fp32 storage (the parity mode) or bf16 storage at head_dim 16 (see the forward's vector
// kernel); arithmetic in fp32.  dq kernel: 64 query rows, 4 threads per row (dh/4 features each); keys staged 32 at a time.
template <int DH, bool RAB, class E>
__global__ __launch_bounds__(256) void attn_bwd_dq_vec_kernel(AttnArgs a) {
    constexpr int BMF = 64, SUB = 32, Q4 = DH / 4, KP = DH + 1;
    __shared__ float sK[SUB * KP];
    __shared__ float sV[SUB * KP];
    __shared__ int sKcode[SUB];
    __shared__ int sKts[SUB];
    __shared__ float sRab[MTGR_RAB_LDS];
    __shared__ float sHist[MTGR_RAB_LDS];
    const int tid = threadIdx.x;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const bool want_drab = RAB && a.drab != nullptr;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BMF;
    const int ntk = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const int4* summ = a.summ + (long long)b * a.ntile;
    const TileSummary sq = load_summary(summ, qt);
    const int qi = q0 + (tid >> 2), part = tid & 3;
    const bool qvalid = qi < nb;
    const E* Q = (const E*)a.q;
    const E* K = (const E*)a.k;
    const E* V = (const E*)a.v;
    const E* DO = (const E*)a.dout;
    float qv[Q4], gv[Q4], acc[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        qv[c] = qvalid ? ld_elem(Q, (long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c) : 0.f;
        gv[c] = qvalid ? ld_elem(DO, (long long)(ob + qi) * a.ld_o + h * DH + part * Q4 + c) : 0.f;
        acc[c] = 0.f;
    }
    int qcode = 0, qts = 0;
    if (qvalid) {
        qcode = token_code(a.seg[ob + qi]);
        qts = a.ts[ob + qi];
    }
    if (RAB && tid < MTGR_RAB_LDS) {
        sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;
        sHist[tid] = 0.f;
    }
    for (int t = 0; t < ntk; t++) {
        const bool overlap = (t * BN < q0 + BMF) && (q0 < t * BN + BN);
        if (tile_class(sq, load_summary(summ, t), overlap) == TILE_MASKED) continue;
        for (int sub = 0; sub < BN / SUB; sub++) {
            const int kb = t * BN + sub * SUB;
            __syncthreads();
            for (int i = tid; i < SUB * DH; i += 256) {
                const int row = i / DH, c = i % DH, key = kb + row;
                sK[row * KP + c] = key < nb ? ld_elem(K, (long long)(ob + key) * a.ld_k + h * DH + c) : 0.f;
                sV[row * KP + c] = key < nb ? ld_elem(V, (long long)(ob + key) * a.ld_v + h * DH + c) : 0.f;
            }
            if (tid < SUB) {
                const int key = kb + tid;
                sKcode[tid] = key < nb ? token_code(a.seg[ob + key]) : 0;
                sKts[tid] = key < nb ? a.ts[ob + key] : 0;
            }
            __syncthreads();
            for (int j = 0; j < SUB; j++) {
                float s = 0.f, dp = 0.f;
#pragma unroll
                for (int c = 0; c < Q4; c++) {
                    s = fmaf(qv[c], sK[j * KP + part * Q4 + c], s);
                    dp = fmaf(gv[c], sV[j * KP + part * Q4 + c], dp);
                }
                s += __shfl_xor(s, 1, 64);
                s += __shfl_xor(s, 2, 64);
                dp += __shfl_xor(dp, 1, 64);
                dp += __shfl_xor(dp, 2, 64);
                float x = s * a.alpha;
                int bk = 0;
                if (RAB) {
                    bk = rab_bucket(qts, sKts[j], a.nbuckets);
                    x += sRab[bk];
                }
                const float sg = 1.0f / (1.0f + expf(-x));
                const float ds = dp * sg * (1.0f + x * (1.0f - sg)) * inv_n;
                if (visible(qcode, qts, qi, sKcode[j], sKts[j], kb + j)) {
#pragma unroll
                    for (int c = 0; c < Q4; c++) acc[c] = fmaf(ds, sK[j * KP + part * Q4 + c], acc[c]);
                    if (want_drab && part == 0) atomicAdd(&sHist[bk], ds);
                }
            }
        }
    }
    __syncthreads();
    if (want_drab && tid < a.nbuckets && sHist[tid] != 0.f) atomicAdd(&a.drab[h * a.nbuckets + tid], sHist[tid]);
    if (qvalid) {
        E* DQ = (E*)a.dq;
#pragma unroll
        for (int c = 0; c < Q4; c++)
            st_elem(DQ, (long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c, a.alpha * acc[c]);
    }
}

// dkdv kernel: 64 key rows, 4 threads per key; queries staged 32 at a time.
template <int DH, bool RAB, class E>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_vec_kernel(AttnArgs a) {
    constexpr int BMF = 64, SUB = 32, Q4 = DH / 4, KP = DH + 1;
    __shared__ float sQ[SUB * KP];
    __shared__ float sG[SUB * KP];
    __shared__ int sQcode[SUB];
    __shared__ int sQts[SUB];
    __shared__ float sRab[MTGR_RAB_LDS];
    const int tid = threadIdx.x;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, kt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int k0 = kt * BMF;
    const int ntq = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const int4* summ = a.summ + (long long)b * a.ntile;
    const TileSummary sk = load_summary(summ, kt);
    const int kj = k0 + (tid >> 2), part = tid & 3;
    const bool kvalid = kj < nb;
    const E* Q = (const E*)a.q;
    const E* K = (const E*)a.k;
    const E* V = (const E*)a.v;
    const E* DO = (const E*)a.dout;
    float kv[Q4], vv[Q4], dk[Q4], dv[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        kv[c] = kvalid ? ld_elem(K, (long long)(ob + kj) * a.ld_k + h * DH + part * Q4 + c) : 0.f;
        vv[c] = kvalid ? ld_elem(V, (long long)(ob + kj) * a.ld_v + h * DH + part * Q4 + c) : 0.f;
        dk[c] = 0.f;
        dv[c] = 0.f;
    }
    int kcode = 0, kts = 0;
    if (kvalid) {
        kcode = token_code(a.seg[ob + kj]);
        kts = a.ts[ob + kj];
    }
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;
    for (int t = 0; t < ntq; t++) {
        const bool overlap = (t * BN < k0 + BMF) && (k0 < t * BN + BN);
        if (tile_class(load_summary(summ, t), sk, overlap) == TILE_MASKED) continue;
        for (int sub = 0; sub < BN / SUB; sub++) {
            const int qb = t * BN + sub * SUB;
            __syncthreads();
            for (int i = tid; i < SUB * DH; i += 256) {
                const int row = i / DH, c = i % DH, qr = qb + row;
                sQ[row * KP + c] = qr < nb ? ld_elem(Q, (long long)(ob + qr) * a.ld_q + h * DH + c) : 0.f;
                sG[row * KP + c] = qr < nb ? ld_elem(DO, (long long)(ob + qr) * a.ld_o + h * DH + c) : 0.f;
            }
            if (tid < SUB) {
                const int qr = qb + tid;
                sQcode[tid] = qr < nb ? token_code(a.seg[ob + qr]) : 0;
                sQts[tid] = qr < nb ? a.ts[ob + qr] : 0;
            }
            __syncthreads();
            for (int i = 0; i < SUB; i++) {
                float s = 0.f, dp = 0.f;
#pragma unroll
                for (int c = 0; c < Q4; c++) {
                    s = fmaf(sQ[i * KP + part * Q4 + c], kv[c], s);
                    dp = fmaf(sG[i * KP + part * Q4 + c], vv[c], dp);
                }
                s += __shfl_xor(s, 1, 64);
                s += __shfl_xor(s, 2, 64);
                dp += __shfl_xor(dp, 1, 64);
                dp += __shfl_xor(dp, 2, 64);
                float x = s * a.alpha;
                if (RAB) x += sRab[rab_bucket(sQts[i], kts, a.nbuckets)];
                const float sg = 1.0f / (1.0f + expf(-x));
                const float p = x * sg * inv_n;
                const float ds = dp * sg * (1.0f + x * (1.0f - sg)) * inv_n;
                if (visible(sQcode[i], sQts[i], qb + i, kcode, kts, kj)) {
#pragma unroll
                    for (int c = 0; c < Q4; c++) {
                        dv[c] = fmaf(p, sG[i * KP + part * Q4 + c], dv[c]);
                        dk[c] = fmaf(ds, sQ[i * KP + part * Q4 + c], dk[c]);
                    }
                }
            }
        }
    }
    if (kvalid) {
        E* DK = (E*)a.dk;
        E* DV = (E*)a.dv;
#pragma unroll
        for (int c = 0; c < Q4; c++) {
            st_elem(DK, (long long)(ob + kj) * a.ld_k + h * DH + part * Q4 + c, a.alpha * dk[c]);
            st_elem(DV, (long long)(ob + kj) * a.ld_v + h * DH + part * Q4 + c, dv[c]);
        }
    }
}

// The relative bias enters the scores of both kernels (RAB_IN).  drab (a.drab) is formed by the
// dK/dV kernel when it runs, else by the recomputing dQ kernel.
template <int DH, bool RAB_IN>
static hipError_t bwd_bf16_dh(const AttnArgs& a, int slots, const BwdPlan& plan, hipStream_t s) {
    if (plan.dkdv) {
        if (plan.store_ds) attn_bwd_dkdv_bf16_kernel<DH, RAB_IN, true><<<slots, 256, 0, s>>>(a);
        else attn_bwd_dkdv_bf16_kernel<DH, RAB_IN, false><<<slots, 256, 0, s>>>(a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (plan.dq_from_ds) {
        attn_bwd_dq_ds_bf16_kernel<DH><<<slots, 256, 0, s>>>(a);
        return hipGetLastError();
    }
    if (plan.dq_recompute) {
        AttnArgs b = a;
        if (plan.dkdv) b.drab = nullptr;
        attn_bwd_dq_bf16_kernel<DH, RAB_IN><<<slots, 256, 0, s>>>(b);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <int DH, bool RAB_IN, class E>
static hipError_t bwd_vec_dh(const AttnArgs& a, int slots, bool dq, bool dkdv, hipStream_t s) {
    if (dq) {
        attn_bwd_dq_vec_kernel<DH, RAB_IN, E><<<slots, 256, 0, s>>>(a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dkdv) {
        attn_bwd_dkdv_vec_kernel<DH, RAB_IN, E><<<slots, 256, 0, s>>>(a);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_attn_bwd_bf16(const AttnArgs& a, int head_dim, int slots, const BwdPlan& plan,
                                hipStream_t s) {
    const bool rab = a.rab != nullptr;
    switch (head_dim) {
        case 32: return rab ? bwd_bf16_dh<32, true>(a, slots, plan, s) : bwd_bf16_dh<32, false>(a, slots, plan, s);
        case 64: return rab ? bwd_bf16_dh<64, true>(a, slots, plan, s) : bwd_bf16_dh<64, false>(a, slots, plan, s);
        case 128: return rab ? bwd_bf16_dh<128, true>(a, slots, plan, s) : bwd_bf16_dh<128, false>(a, slots, plan, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_bwd_vec(const AttnArgs& a, bool bf16, int head_dim, int slots, bool dq, bool dkdv,
                               hipStream_t s) {
    const bool rab = a.rab != nullptr;
    if (bf16) {
        if (head_dim != 16) return hipErrorInvalidValue;
        return rab ? bwd_vec_dh<16, true, uint16_t>(a, slots, dq, dkdv, s)
                   : bwd_vec_dh<16, false, uint16_t>(a, slots, dq, dkdv, s);
    }
    switch (head_dim) {
        case 16: return rab ? bwd_vec_dh<16, true, float>(a, slots, dq, dkdv, s) : bwd_vec_dh<16, false, float>(a, slots, dq, dkdv, s);
        case 32: return rab ? bwd_vec_dh<32, true, float>(a, slots, dq, dkdv, s) : bwd_vec_dh<32, false, float>(a, slots, dq, dkdv, s);
        case 64: return rab ? bwd_vec_dh<64, true, float>(a, slots, dq, dkdv, s) : bwd_vec_dh<64, false, float>(a, slots, dq, dkdv, s);
        case 128: return rab ? bwd_vec_dh<128, true, float>(a, slots, dq, dkdv, s) : bwd_vec_dh<128, false, float>(a, slots, dq, dkdv, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mtgr
