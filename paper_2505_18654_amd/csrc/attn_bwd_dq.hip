// dQ (and drab) of the attention backward, recomputing S, dP and dS (bf16).
#include "attn_bwd_common.h"

namespace mtgr {
using bwd::BM;
using bwd::BN;
using bwd::ldg16;
using bwd::zero;

// ------------------------------------------------------------------ dQ (+ drab), bf16
template <int DH, bool RAB>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8, KSTEPS = DH / 16, DBLK = DH / 32, TILE = BN * DH;
    __shared__ __align__(16) uint16_t sK0[TILE];
    __shared__ __align__(16) uint16_t sK1[TILE];
    __shared__ __align__(16) uint16_t sV0[TILE];
    __shared__ __align__(16) uint16_t sV1[TILE];
    __shared__ int sKts[2][BN];
    __shared__ int sKcode[2][BN];
    __shared__ float sRab[MTGR_RAB_LDS];
    __shared__ float sHist[RAB ? bwd::HIST_WORDS : 1];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const bool want_drab = RAB && a.drab != nullptr;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BM;
    const int ntk = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const float alpha = a.alpha;
    const float c_exp = -1.4426950408889634f * alpha;   // sigmoid(alpha s) = 1 / (1 + 2^(c_exp s))
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
    const uint16_t* Q = (const uint16_t*)a.q;
    const uint16_t* DO = (const uint16_t*)a.dout;
    const uint16_t* Kb = (const uint16_t*)a.k + (long long)ob * a.ld_k;
    const uint16_t* Vb = (const uint16_t*)a.v + (long long)ob * a.ld_v;
    bf16x8 qreg[KSTEPS], doreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; kk++) {
        uint4 u = make_uint4(0, 0, 0, 0), g = make_uint4(0, 0, 0, 0);
        if (qvalid) {
            u = ldg16(Q + (long long)(ob + qi) * a.ld_q + h * DH + 16 * kk + 8 * hh);
            g = ldg16(DO + (long long)(ob + qi) * a.ld_o + h * DH + 16 * kk + 8 * hh);
        }
        qreg[kk] = as_bf16x8(u);
        doreg[kk] = as_bf16x8(g);
    }
    if (RAB) {
        if (tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? NEG_LOG2E * a.rab[h * a.nbuckets + tid] : 0.f;
        bwd::hist_zero(sHist, tid);
    }
    floatx16 dqacc[DBLK];
#pragma unroll
    for (int i = 0; i < DBLK; i++) zero(dqacc[i]);

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
    bwd::HistRun run;   // drab: this lane's current run of equal buckets
    if (t < ntk) issue(t, 0);
    while (t < ntk) {
        wait_vmem();
        if (tid < BN && t * BN + tid >= nb) sKcode[cur][tid] = 0;
        lds_barrier();
        const int tn = walk.next(t + 1, &cls_n);
        if (tn < ntk) issue(tn, cur ^ 1);
        const uint16_t* sK = cur ? sK1 : sK0;
        const uint16_t* sV = cur ? sV1 : sV0;
        const int* kts = sKts[cur];
        const int* kcode = sKcode[cur];

#pragma unroll
        for (int blk = 0; blk < 2; blk++) {
            floatx16 sacc, dpacc;
            zero(sacc);
            zero(dpacc);
#pragma unroll
            for (int kk = 0; kk < KSTEPS; kk++) {
                const bf16x8 ka = tile_read8<CPR>(sK, 32 * blk + col, 2 * kk + hh);
                const bf16x8 va = tile_read8<CPR>(sV, 32 * blk + col, 2 * kk + hh);
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[kk], sacc, 0, 0, 0);
                dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, doreg[kk], dpacc, 0, 0, 0);
            }
            uint32_t dsk[2][4];
            // Element rr belongs to key 32 blk + 8 (rr / 4) + 4 hh + rr % 4.  Straight-line code
            // per group of GRP elements (one mask branch per group, after it) so that their
            // exp / rcp chains interleave; 16 without a bias, 4 with one (timestamps and bias
            // values read first) to stay within the register budget.
            constexpr int GRP = RAB ? 4 : 16;
#pragma unroll
            for (int g0 = 0; g0 < 16; g0 += GRP) {
                float dv[GRP];
                int bk[GRP];
                if (RAB) {
#pragma unroll
                    for (int e = 0; e < GRP; e++) {
                        const int rr = g0 + e;
                        bk[e] = rab_bucket(qts, kts[32 * blk + 8 * (rr >> 2) + 4 * hh + (rr & 3)], a.nbuckets);
                    }
                }
#pragma unroll
                for (int e = 0; e < GRP; e++) {
                    const int rr = g0 + e;
                    // ds is dS without the per-user factor 1 / n_b, applied once to dQ and drab.
                    if (RAB) {
                        float sg;
                        const float p = silu_scaled(__builtin_fmaf(sacc[rr], c_exp, sRab[bk[e]]), sg);
                        dv[e] = dpacc[rr] * __builtin_fmaf(NEG_LN2, __builtin_fmaf(-p, sg, p), sg);
                    } else {
                        const float sv = sacc[rr];
                        const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(sv * c_exp));
                        dv[e] = (dpacc[rr] * sg) * __builtin_fmaf(alpha, __builtin_fmaf(-sv, sg, sv), 1.0f);
                    }
                }
                if (cls == TILE_PARTIAL) {
#pragma unroll
                    for (int e = 0; e < GRP; e++) {
                        const int rr = g0 + e, kl = 32 * blk + 8 * (rr >> 2) + 4 * hh + (rr & 3);
                        dv[e] = visible(qcode, qts, qi, kcode[kl], kts[kl], t * BN + kl) ? dv[e] : 0.f;
                    }
                } else if (!qvalid) {
#pragma unroll
                    for (int e = 0; e < GRP; e++) dv[e] = 0.f;
                }
#pragma unroll
                for (int e = 0; e < GRP; e += 2) {
                    const int r = g0 + e;
                    dsk[r >> 3][(r & 7) >> 1] = pack_bf16x2(dv[e], dv[e + 1]);
                }
                if (want_drab) {
#pragma unroll
                    for (int e = 0; e < GRP; e++) run.add(sHist, lane, bk[e], dv[e]);
                }
            }
#pragma unroll
            for (int kq = 0; kq < 2; kq++) {
                const bf16x8 db = as_bf16x8(make_uint4(dsk[kq][0], dsk[kq][1], dsk[kq][2], dsk[kq][3]));
#pragma unroll
                for (int d = 0; d < DBLK; d++) {
                    const bf16x8 kt = tile_read_tr<CPR>(sK, 32 * blk + 16 * kq, 32 * d, lane);
                    dqacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kt, db, dqacc[d], 0, 0, 0);
                }
            }
        }
        t = tn;
        cls = cls_n;
        cur ^= 1;
    }
    // One barrier per tile suffices: the copy into a buffer is issued only after the barrier
    // that every wave passes once done with the tile that buffer held.  The tiles' LDS is
    // reused below.
    __syncthreads();

    if (want_drab) {
        run.flush(sHist, lane);
        __syncthreads();   // zeroing (when no tile was visited) and every histogram update
        if (tid < a.nbuckets) {
            const float v = bwd::hist_total(sHist, tid);
            if (v != 0.f) atomicAdd(&a.drab[h * a.nbuckets + tid], v * inv_n);
        }
    }
    uint16_t* sO = (w < 2 ? sK0 : sK1) + (w & 1) * 32 * DH;
    const float dq_scale = alpha * inv_n;
#pragma unroll
    for (int d = 0; d < DBLK; d++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int dd = 32 * d + 8 * g + 4 * hh;
            *(uint2*)&sO[8 * tile_chunk<CPR>(col, dd >> 3) + (dd & 7)] =
                make_uint2(pack_bf16x2(dq_scale * dqacc[d][4 * g + 0], dq_scale * dqacc[d][4 * g + 1]),
                           pack_bf16x2(dq_scale * dqacc[d][4 * g + 2], dq_scale * dqacc[d][4 * g + 3]));
        }
    }
    __syncthreads();
    uint16_t* DQ = (uint16_t*)a.dq;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; i++) {
        const int c = lane + 64 * i, row = c / CPR, cc = c % CPR;
        const int qr = q0 + w * 32 + row;
        if (qr < nb)
            store_nt16(DQ + (long long)(ob + qr) * a.ld_q + h * DH + cc * 8, &sO[8 * tile_chunk<CPR>(row, cc)]);
    }
}

template __global__ void attn_bwd_dq_bf16_kernel<32, false>(AttnArgs);
template __global__ void attn_bwd_dq_bf16_kernel<32, true>(AttnArgs);
template __global__ void attn_bwd_dq_bf16_kernel<64, false>(AttnArgs);
template __global__ void attn_bwd_dq_bf16_kernel<64, true>(AttnArgs);
template __global__ void attn_bwd_dq_bf16_kernel<128, false>(AttnArgs);
template __global__ void attn_bwd_dq_bf16_kernel<128, true>(AttnArgs);
}  // namespace mtgr
