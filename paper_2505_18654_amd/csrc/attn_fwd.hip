// Forward of the jagged dynamic-mask SiLU attention (Eq. 5, Sec. 4.2).
//
// bf16 kernel: one workgroup = 4 waves = 128 query rows of one (user, head); each wave owns
// 32 query rows.  The user's 64-key tiles that are not fully masked stream through two LDS
// buffers: while the waves compute on one tile, the next tile's K and V rows (and its
// timestamps and mask codes) are copied straight from global memory into the other buffer
// (global_load_lds, no staging registers).  Per 32-key half of a tile each wave computes
//     S^T (32 keys x 32 queries) = K Q^T          v_mfma_f32_32x32x16_bf16, Q held in VGPRs
//     P = silu(alpha S + rab) / n_b, masked        in registers, straight from the accumulators
//     O^T (dh x 32 queries)     += V^T P^T         V^T read with ds_read_b64_tr_b16
// Computing the transposed products lets the accumulator layout of S^T (lane = query column,
// registers = keys) serve directly as the B operand of the second product, so P never goes
// through LDS, and the transposing LDS read gives V^T without a transposed copy.  The mask
// is evaluated only on PARTIAL tiles.
#include <type_traits>

#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

namespace {

constexpr int BM = 128;   // query rows per workgroup
constexpr int BN = 64;    // keys per tile

__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *(const uint4*)p; }

}  // namespace

template <int DH, bool RAB>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8;       // 16-byte chunks per row
    constexpr int KSTEPS = DH / 16;   // k-steps of S^T = K Q^T
    constexpr int DBLK = DH / 32;     // 32-row blocks of O^T
    constexpr int TILE = BN * DH;     // elements of one 64-row tile

    __shared__ __align__(16) uint16_t sK0[TILE];
    __shared__ __align__(16) uint16_t sK1[TILE];
    __shared__ __align__(16) uint16_t sV0[TILE];
    __shared__ __align__(16) uint16_t sV1[TILE];
    __shared__ int sKts[2][BN];
    __shared__ int sKcode[2][BN];
    __shared__ float sRab[MTGR_RAB_LDS];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BM;
    const int ntk = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const float alpha = a.alpha;
    const int4* summ = a.summ + (long long)b * a.ntile;

    TileSummary sq = load_summary(summ, 2 * qt);
    if (2 * qt + 1 < ntk) sq = combine(sq, load_summary(summ, 2 * qt + 1));

    const int col = lane & 31, hh = lane >> 5;
    const int qi = q0 + w * 32 + col;
    const bool qvalid = qi < nb;
    int qcode = 0, qts = 0;
    if (qvalid) {
        qcode = token_code(a.seg[ob + qi]);
        qts = a.ts[ob + qi];
    }
    const uint16_t* Kb = (const uint16_t*)a.k + (long long)ob * a.ld_k;
    const uint16_t* Vb = (const uint16_t*)a.v + (long long)ob * a.ld_v;
    const uint16_t* Q = (const uint16_t*)a.q;
    bf16x8 qreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; kk++) {
        uint4 u = make_uint4(0, 0, 0, 0);
        if (qvalid) u = ldg16(Q + (long long)(ob + qi) * a.ld_q + h * DH + 16 * kk + 8 * hh);
        qreg[kk] = as_bf16x8(u);
    }
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;

    floatx16 oacc[DBLK];
#pragma unroll
    for (int i = 0; i < DBLK; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) oacc[i][r] = 0.f;

    auto class_of = [&](int t) {
        const bool overlap = (t * BN < q0 + BM) && (q0 < t * BN + BN);
        return tile_class(sq, load_summary(summ, t), overlap);
    };
    TileWalker<decltype(class_of)> walk(class_of, ntk);
    auto issue = [&](int t, int buf) {
        tile_dma<DH>(buf ? sK1 : sK0, Kb, a.ld_k, t * BN, nb, h * DH, tid);
        tile_dma<DH>(buf ? sV1 : sV0, Vb, a.ld_v, t * BN, nb, h * DH, tid);
        codes_dma(sKts[buf], sKcode[buf], a.ts + ob, a.tok_code + ob, t * BN, nb, tid);
    };

    int cls, cls_n;
    int t = walk.next(0, &cls);
    int cur = 0;
    if (t < ntk) issue(t, 0);
    while (t < ntk) {
        wait_vmem();                                   // this wave's copies of tile t landed
        if (tid < BN && t * BN + tid >= nb) sKcode[cur][tid] = 0;
        __syncthreads();                               // ... and every other wave's
        const int tn = walk.next(t + 1, &cls_n);
        if (tn < ntk) issue(tn, cur ^ 1);              // overlaps the compute below
        const uint16_t* sK = cur ? sK1 : sK0;
        const uint16_t* sV = cur ? sV1 : sV0;
        const int* kts = sKts[cur];
        const int* kcode = sKcode[cur];

        // One straight-line body per tile class (the branch is per tile, not per element), so
        // the scheduler can overlap one half's SiLU epilogue with the other half's MFMAs.
        auto body = [&](auto masked_tag) {
            constexpr bool MASKED = decltype(masked_tag)::value;
            // --- scores of both 32-key halves, operands read one k-step ahead
            floatx16 sacc[2];
#pragma unroll
            for (int blk = 0; blk < 2; blk++)
#pragma unroll
                for (int r = 0; r < 16; r++) sacc[blk][r] = 0.f;
            bf16x8 ka0 = tile_read8<CPR>(sK, col, hh);
            bf16x8 ka1 = tile_read8<CPR>(sK, 32 + col, hh);
#pragma unroll
            for (int kk = 0; kk < KSTEPS; kk++) {
                bf16x8 nx0 = ka0, nx1 = ka1;
                if (kk + 1 < KSTEPS) {
                    nx0 = tile_read8<CPR>(sK, col, 2 * kk + 2 + hh);
                    nx1 = tile_read8<CPR>(sK, 32 + col, 2 * kk + 2 + hh);
                }
                sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka0, qreg[kk], sacc[0], 0, 0, 0);
                sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka1, qreg[kk], sacc[1], 0, 0, 0);
                ka0 = nx0;
                ka1 = nx1;
                __builtin_amdgcn_sched_barrier(0);
            }
            // --- SiLU epilogue in quarters (8 keys each), p = (alpha s / n_b) / (1 + 2^(-alpha s log2 e))
            const float c_exp = -1.4426950408889634f * alpha;
            const float c_out = alpha * inv_n;
            auto epilogue = [&](int blk, int q4, uint32_t* dst) {
#pragma unroll
                for (int r = 8 * q4; r < 8 * q4 + 8; r += 2) {
                    float pv[2];
#pragma unroll
                    for (int e = 0; e < 2; e++) {
                        const int rr = r + e;
                        const int kl = 32 * blk + 8 * (rr >> 2) + 4 * hh + (rr & 3);
                        const float sv = sacc[blk][rr];
                        float p;
                        if (RAB) {
                            const float x = sv * alpha + sRab[rab_bucket(qts, kts[kl], a.nbuckets)];
                            float sg;
                            p = silu_sig(x, sg) * inv_n;
                        } else {
                            p = (sv * c_out) * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(sv * c_exp));
                        }
                        if (MASKED) p = visible(qcode, qts, qi, kcode[kl], kts[kl], t * BN + kl) ? p : 0.f;
                        pv[e] = p;
                    }
                    dst[(r & 7) >> 1] = pack_bf16x2(pv[0], pv[1]);
                }
            };
            // --- O^T += V^T P^T, 16 keys (one k-step) at a time; each group of 4 MFMAs is
            // followed by the epilogue of the next 16 keys, which the MFMAs do not depend on.
            uint32_t pk[4][4];
            epilogue(0, 0, pk[0]);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int ks = 0; ks < 4; ks++) {
                const int blk = ks >> 1, kq = ks & 1;
                const bf16x8 pb = as_bf16x8(make_uint4(pk[ks][0], pk[ks][1], pk[ks][2], pk[ks][3]));
#pragma unroll
                for (int db = 0; db < DBLK; db++) {
                    const bf16x8 va = tile_read_tr<CPR>(sV, 32 * blk + 16 * kq, 32 * db, lane);
                    oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, oacc[db], 0, 0, 0);
                }
                if (ks + 1 < 4) epilogue((ks + 1) >> 1, (ks + 1) & 1, pk[ks + 1]);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (cls == TILE_PARTIAL)
            body(std::true_type{});
        else
            body(std::false_type{});
        __syncthreads();                               // buffer `cur` is refilled next round
        t = tn;
        cls = cls_n;
        cur ^= 1;
    }

    // Output: O^T accumulators -> bf16 rows of this wave staged in LDS (swizzled 32-row
    // tile inside the K buffers) -> 16-byte coalesced stores.
    uint16_t* sO = (w < 2 ? sK0 : sK1) + (w & 1) * 32 * DH;
#pragma unroll
    for (int db = 0; db < DBLK; db++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int d = 32 * db + 8 * g + 4 * hh;
            *(uint2*)&sO[8 * tile_chunk<CPR>(col, d >> 3) + (d & 7)] =
                make_uint2(pack_bf16x2(oacc[db][4 * g + 0], oacc[db][4 * g + 1]),
                           pack_bf16x2(oacc[db][4 * g + 2], oacc[db][4 * g + 3]));
        }
    }
    __syncthreads();
    uint16_t* O = (uint16_t*)a.out;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; i++) {
        const int c = lane + 64 * i, row = c / CPR, cc = c % CPR;
        const int qr = q0 + w * 32 + row;
        if (qr < nb)
            *(uint4*)(O + (long long)(ob + qr) * a.ld_o + h * DH + cc * 8) =
                *(const uint4*)&sO[8 * tile_chunk<CPR>(row, cc)];
    }
}

// fp32 parity kernel: 64 query rows per workgroup, 4 threads per row each owning dh/4
// features; keys staged 32 at a time in LDS; plain FMA loops.
template <int DH, bool RAB>
__global__ __launch_bounds__(256) void attn_fwd_f32_kernel(AttnArgs a) {
    constexpr int BMF = 64, SUB = 32, Q4 = DH / 4, KP = DH + 1;
    __shared__ float sK[SUB * KP];
    __shared__ float sV[SUB * KP];
    __shared__ int sKcode[SUB];
    __shared__ int sKts[SUB];
    __shared__ float sRab[MTGR_RAB_LDS];
    const int tid = threadIdx.x;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BMF;
    const int ntk = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const int4* summ = a.summ + (long long)b * a.ntile;
    const TileSummary sq = load_summary(summ, qt);

    const int qi = q0 + (tid >> 2), part = tid & 3;
    const bool qvalid = qi < nb;
    int qcode = 0, qts = 0;
    const float* Q = (const float*)a.q;
    const float* K = (const float*)a.k;
    const float* V = (const float*)a.v;
    float qv[Q4], ov[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        qv[c] = qvalid ? Q[(long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c] : 0.f;
        ov[c] = 0.f;
    }
    if (qvalid) {
        qcode = token_code(a.seg[ob + qi]);
        qts = a.ts[ob + qi];
    }
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;

    for (int t = 0; t < ntk; t++) {
        const bool overlap = (t * BN < q0 + BMF) && (q0 < t * BN + BN);
        const int cls = tile_class(sq, load_summary(summ, t), overlap);
        if (cls == TILE_MASKED) continue;
        for (int sub = 0; sub < BN / SUB; sub++) {
            const int kb = t * BN + sub * SUB;
            __syncthreads();
            for (int i = tid; i < SUB * DH; i += 256) {
                const int row = i / DH, c = i % DH, key = kb + row;
                sK[row * KP + c] = key < nb ? K[(long long)(ob + key) * a.ld_k + h * DH + c] : 0.f;
                sV[row * KP + c] = key < nb ? V[(long long)(ob + key) * a.ld_v + h * DH + c] : 0.f;
            }
            if (tid < SUB) {
                const int key = kb + tid;
                sKcode[tid] = key < nb ? token_code(a.seg[ob + key]) : 0;
                sKts[tid] = key < nb ? a.ts[ob + key] : 0;
            }
            __syncthreads();
            for (int j = 0; j < SUB; j++) {
                float s = 0.f;
#pragma unroll
                for (int c = 0; c < Q4; c++) s = fmaf(qv[c], sK[j * KP + part * Q4 + c], s);
                s += __shfl_xor(s, 1, 64);
                s += __shfl_xor(s, 2, 64);
                float x = s * a.alpha;
                if (RAB) x += sRab[rab_bucket(qts, sKts[j], a.nbuckets)];
                const float p = x / (1.0f + expf(-x)) * inv_n;
                const bool vis = visible(qcode, qts, qi, sKcode[j], sKts[j], kb + j);
                if (vis) {
#pragma unroll
                    for (int c = 0; c < Q4; c++) ov[c] = fmaf(p, sV[j * KP + part * Q4 + c], ov[c]);
                }
            }
        }
    }
    if (qvalid) {
        float* O = (float*)a.out;
#pragma unroll
        for (int c = 0; c < Q4; c++) O[(long long)(ob + qi) * a.ld_o + h * DH + part * Q4 + c] = ov[c];
    }
}

template <int DH>
static hipError_t fwd_bf16_dh(const AttnArgs& a, int slots, hipStream_t s) {
    if (a.rab)
        attn_fwd_bf16_kernel<DH, true><<<slots, 256, 0, s>>>(a);
    else
        attn_fwd_bf16_kernel<DH, false><<<slots, 256, 0, s>>>(a);
    return hipGetLastError();
}

template <int DH>
static hipError_t fwd_f32_dh(const AttnArgs& a, int slots, hipStream_t s) {
    if (a.rab)
        attn_fwd_f32_kernel<DH, true><<<slots, 256, 0, s>>>(a);
    else
        attn_fwd_f32_kernel<DH, false><<<slots, 256, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_attn_fwd_bf16(const AttnArgs& a, int head_dim, int slots, hipStream_t s) {
    switch (head_dim) {
        case 32: return fwd_bf16_dh<32>(a, slots, s);
        case 64: return fwd_bf16_dh<64>(a, slots, s);
        case 128: return fwd_bf16_dh<128>(a, slots, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_fwd_f32(const AttnArgs& a, int head_dim, int slots, hipStream_t s) {
    switch (head_dim) {
        case 16: return fwd_f32_dh<16>(a, slots, s);
        case 32: return fwd_f32_dh<32>(a, slots, s);
        case 64: return fwd_f32_dh<64>(a, slots, s);
        case 128: return fwd_f32_dh<128>(a, slots, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mtgr
