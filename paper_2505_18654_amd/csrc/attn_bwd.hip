// Backward of the jagged dynamic-mask SiLU attention (chain rule of Eq. 5).
//
// With s = alpha q_i.k_j + rab, sg = sigmoid(s), p = silu(s)/n_b and dP = dout_i . v_j:
//     dS_ij = M_ij dP_ij sg (1 + s (1 - sg)) / n_b
//     dV_j = sum_i M_ij p_ij dout_i,   dK_j = alpha sum_i dS_ij q_i,
//     dQ_i = alpha sum_j dS_ij k_j,    drab[h, bucket] += dS_ij.
// There is no softmax, so nothing is saved by the forward and no row statistic is needed.
//
// Two kernels, no atomics on dQ/dK/dV (results are deterministic):
//   dq kernel (row-parallel, like the forward): per wave 32 queries, Q and dO in VGPRs; the
//     user's visible 64-key tiles stream through two LDS buffers (global_load_lds); per
//     32-key half: S^T = K Q^T, dP^T = V dO^T, dS^T in registers, dQ^T += K^T dS^T with K^T
//     read by ds_read_b64_tr_b16.  It also forms drab (LDS histogram, one global atomic per
//     bucket per workgroup).
//   dkdv kernel (column-parallel): per wave 32 keys, K and V in VGPRs; the visible 64-query
//     tiles of Q and dO stream through two LDS buffers; per 32-query half: S = Q K^T,
//     dP = dO V^T (lane = key column), then dV += P^T dO and dK += dS^T Q with dO and Q read
//     transposed from their row-major tiles.
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

namespace {
constexpr int BM = 128;   // rows (queries or keys) per workgroup
constexpr int BN = 64;    // columns per inner tile
__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *(const uint4*)p; }

__device__ __forceinline__ void zero(floatx16& x) {
#pragma unroll
    for (int r = 0; r < 16; r++) x[r] = 0.f;
}
}  // namespace

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
    __shared__ float sHist[MTGR_RAB_LDS];

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
    if (RAB && tid < MTGR_RAB_LDS) {
        sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;
        sHist[tid] = 0.f;
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
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                float dv[2];
#pragma unroll
                for (int e = 0; e < 2; e++) {
                    const int rr = r + e;
                    const int kl = 32 * blk + 8 * (rr >> 2) + 4 * hh + (rr & 3);
                    float x = sacc[rr] * alpha;
                    int bk = 0;
                    if (RAB) {
                        bk = rab_bucket(qts, kts[kl], a.nbuckets);
                        x += sRab[bk];
                    }
                    float sg;
                    silu_sig(x, sg);
                    float ds = dpacc[rr] * sg * (1.0f + x * (1.0f - sg)) * inv_n;
                    if (cls == TILE_PARTIAL)
                        ds = visible(qcode, qts, qi, kcode[kl], kts[kl], t * BN + kl) ? ds : 0.f;
                    else if (!qvalid)
                        ds = 0.f;
                    if (want_drab && ds != 0.f) atomicAdd(&sHist[bk], ds);
                    dv[e] = ds;
                }
                dsk[r >> 3][(r & 7) >> 1] = pack_bf16x2(dv[0], dv[1]);
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
        lds_barrier();
        t = tn;
        cls = cls_n;
        cur ^= 1;
    }

    if (want_drab && tid < a.nbuckets && sHist[tid] != 0.f) atomicAdd(&a.drab[h * a.nbuckets + tid], sHist[tid]);
    uint16_t* sO = (w < 2 ? sK0 : sK1) + (w & 1) * 32 * DH;
#pragma unroll
    for (int d = 0; d < DBLK; d++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int dd = 32 * d + 8 * g + 4 * hh;
            *(uint2*)&sO[8 * tile_chunk<CPR>(col, dd >> 3) + (dd & 7)] =
                make_uint2(pack_bf16x2(alpha * dqacc[d][4 * g + 0], alpha * dqacc[d][4 * g + 1]),
                           pack_bf16x2(alpha * dqacc[d][4 * g + 2], alpha * dqacc[d][4 * g + 3]));
        }
    }
    __syncthreads();
    uint16_t* DQ = (uint16_t*)a.dq;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; i++) {
        const int c = lane + 64 * i, row = c / CPR, cc = c % CPR;
        const int qr = q0 + w * 32 + row;
        if (qr < nb)
            *(uint4*)(DQ + (long long)(ob + qr) * a.ld_q + h * DH + cc * 8) =
                *(const uint4*)&sO[8 * tile_chunk<CPR>(row, cc)];
    }
}

// ------------------------------------------------------------------ dK, dV, bf16
template <int DH, bool RAB>
__global__ __launch_bounds__(256, 2) void attn_bwd_dkdv_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8, KSTEPS = DH / 16, DBLK = DH / 32, TILE = BN * DH;
    __shared__ __align__(16) uint16_t sQ0[TILE];
    __shared__ __align__(16) uint16_t sQ1[TILE];
    __shared__ __align__(16) uint16_t sG0[TILE];
    __shared__ __align__(16) uint16_t sG1[TILE];
    __shared__ int sQts[2][BN];
    __shared__ int sQcode[2][BN];
    __shared__ float sRab[MTGR_RAB_LDS];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, kt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int k0 = kt * BM;
    const int ntq = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const float alpha = a.alpha;
    const int4* summ = a.summ + (long long)b * a.ntile;
    TileSummary sk = load_summary(summ, 2 * kt);
    if (2 * kt + 1 < ntq) sk = combine(sk, load_summary(summ, 2 * kt + 1));
    else sk.flags &= ~TS_ALL_STATIC;   // a lone half tile is never fully visible

    const int col = lane & 31, hh = lane >> 5;
    const int kj = k0 + w * 32 + col;
    const bool kvalid = kj < nb;
    int kcode = 0, kts = 0;
    if (kvalid) {
        kcode = token_code(a.seg[ob + kj]);
        kts = a.ts[ob + kj];
    }
    const uint16_t* K = (const uint16_t*)a.k;
    const uint16_t* V = (const uint16_t*)a.v;
    const uint16_t* Qb = (const uint16_t*)a.q + (long long)ob * a.ld_q;
    const uint16_t* Gb = (const uint16_t*)a.dout + (long long)ob * a.ld_o;
    bf16x8 kreg[KSTEPS], vreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; kk++) {
        uint4 u = make_uint4(0, 0, 0, 0), g = make_uint4(0, 0, 0, 0);
        if (kvalid) {
            u = ldg16(K + (long long)(ob + kj) * a.ld_k + h * DH + 16 * kk + 8 * hh);
            g = ldg16(V + (long long)(ob + kj) * a.ld_v + h * DH + 16 * kk + 8 * hh);
        }
        kreg[kk] = as_bf16x8(u);
        vreg[kk] = as_bf16x8(g);
    }
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;
    floatx16 dkacc[DBLK], dvacc[DBLK];
#pragma unroll
    for (int i = 0; i < DBLK; i++) {
        zero(dkacc[i]);
        zero(dvacc[i]);
    }

    // A query tile that runs past the user's end holds copies of its last row; it must take
    // the masked path so that those rows contribute nothing.
    auto class_of = [&](int t) {
        const bool overlap = (t * BN < k0 + BM) && (k0 < t * BN + BN);
        const int c = tile_class(load_summary(summ, t), sk, overlap);
        return (c == TILE_FULL && t * BN + BN > nb) ? TILE_PARTIAL : c;
    };
    TileWalker<decltype(class_of)> walk(class_of, ntq);
    auto issue = [&](int t, int buf) {
        tile_dma_tracked<DH>(buf ? sQ1 : sQ0, Qb, a.ld_q, t * BN, nb, h * DH, tid);
        tile_dma_tracked<DH>(buf ? sG1 : sG0, Gb, a.ld_o, t * BN, nb, h * DH, tid);
        codes_dma_tracked(sQts[buf], sQcode[buf], a.ts + ob, a.tok_code + ob, t * BN, nb, tid);
    };

    int cls, cls_n;
    int t = walk.next(0, &cls);
    int cur = 0;
    if (t < ntq) issue(t, 0);
    while (t < ntq) {
        wait_vmem();
        if (tid < BN && t * BN + tid >= nb) sQcode[cur][tid] = 0;
        lds_barrier();
        const int tn = walk.next(t + 1, &cls_n);
        if (tn < ntq) issue(tn, cur ^ 1);
        const uint16_t* sQ = cur ? sQ1 : sQ0;
        const uint16_t* sG = cur ? sG1 : sG0;
        const int* qts = sQts[cur];
        const int* qcode = sQcode[cur];
        const int qb = t * BN;

#pragma unroll
        for (int half = 0; half < 2; half++) {
            // S (32 q x 32 keys) = Q K^T and dP = dO V^T: lane = key column, registers = queries.
            floatx16 sacc, dpacc;
            zero(sacc);
            zero(dpacc);
#pragma unroll
            for (int kk = 0; kk < KSTEPS; kk++) {
                const bf16x8 qa = tile_read8<CPR>(sQ, 32 * half + col, 2 * kk + hh);
                const bf16x8 ga = tile_read8<CPR>(sG, 32 * half + col, 2 * kk + hh);
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kreg[kk], sacc, 0, 0, 0);
                dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga, vreg[kk], dpacc, 0, 0, 0);
            }
            uint32_t pk[2][4], dsk[2][4];
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                float pv[2], dv[2];
#pragma unroll
                for (int e = 0; e < 2; e++) {
                    const int rr = r + e;
                    const int ql = 32 * half + 8 * (rr >> 2) + 4 * hh + (rr & 3);
                    float x = sacc[rr] * alpha;
                    if (RAB) x += sRab[rab_bucket(qts[ql], kts, a.nbuckets)];
                    float sg;
                    float p = silu_sig(x, sg) * inv_n;
                    float ds = dpacc[rr] * sg * (1.0f + x * (1.0f - sg)) * inv_n;
                    if (cls == TILE_PARTIAL) {
                        const bool vis = visible(qcode[ql], qts[ql], qb + ql, kcode, kts, kj);
                        p = vis ? p : 0.f;
                        ds = vis ? ds : 0.f;
                    }
                    pv[e] = p;
                    dv[e] = ds;
                }
                pk[r >> 3][(r & 7) >> 1] = pack_bf16x2(pv[0], pv[1]);
                dsk[r >> 3][(r & 7) >> 1] = pack_bf16x2(dv[0], dv[1]);
            }
            // dV (32 keys x dh) += P^T dO ; dK += dS^T Q.  A = P^T / dS^T from registers,
            // B = dO / Q read transposed (lane = feature column, slots = queries).
#pragma unroll
            for (int kq = 0; kq < 2; kq++) {
                const bf16x8 pa = as_bf16x8(make_uint4(pk[kq][0], pk[kq][1], pk[kq][2], pk[kq][3]));
                const bf16x8 da = as_bf16x8(make_uint4(dsk[kq][0], dsk[kq][1], dsk[kq][2], dsk[kq][3]));
#pragma unroll
                for (int d = 0; d < DBLK; d++) {
                    const bf16x8 gb = tile_read_tr<CPR>(sG, 32 * half + 16 * kq, 32 * d, lane);
                    const bf16x8 qbv = tile_read_tr<CPR>(sQ, 32 * half + 16 * kq, 32 * d, lane);
                    dvacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa, gb, dvacc[d], 0, 0, 0);
                    dkacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, qbv, dkacc[d], 0, 0, 0);
                }
            }
        }
        lds_barrier();
        t = tn;
        cls = cls_n;
        cur ^= 1;
    }

    // dK / dV accumulators: lane = feature column, registers = key rows.  Each wave stages
    // its 32 rows in a swizzled 32-row tile inside the Q buffers.
    uint16_t* sO = (w < 2 ? sQ0 : sQ1) + (w & 1) * 32 * DH;
    uint16_t* DK = (uint16_t*)a.dk;
    uint16_t* DV = (uint16_t*)a.dv;
#pragma unroll
    for (int which = 0; which < 2; which++) {
        __syncthreads();
#pragma unroll
        for (int d = 0; d < DBLK; d++) {
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int krow = 8 * (r >> 2) + 4 * hh + (r & 3);
                const int dd = 32 * d + col;
                const float val = which == 0 ? alpha * dkacc[d][r] : dvacc[d][r];
                sO[8 * tile_chunk<CPR>(krow, dd >> 3) + (dd & 7)] = (uint16_t)f32_to_bf16_bits(val);
            }
        }
        __syncthreads();
        uint16_t* dst = which == 0 ? DK : DV;
        const long long ld = which == 0 ? a.ld_k : a.ld_v;
#pragma unroll
        for (int i = 0; i < 32 * CPR / 64; i++) {
            const int c = lane + 64 * i, row = c / CPR, cc = c % CPR;
            const int kr = k0 + w * 32 + row;
            if (kr < nb)
                *(uint4*)(dst + (long long)(ob + kr) * ld + h * DH + cc * 8) =
                    *(const uint4*)&sO[8 * tile_chunk<CPR>(row, cc)];
        }
    }
}

// ------------------------------------------------------------------ fp32 parity kernels
// dq kernel: 64 query rows, 4 threads per row (dh/4 features each); keys staged 32 at a time.
template <int DH, bool RAB>
__global__ __launch_bounds__(256) void attn_bwd_dq_f32_kernel(AttnArgs a) {
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
    const float* Q = (const float*)a.q;
    const float* K = (const float*)a.k;
    const float* V = (const float*)a.v;
    const float* DO = (const float*)a.dout;
    float qv[Q4], gv[Q4], acc[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        qv[c] = qvalid ? Q[(long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c] : 0.f;
        gv[c] = qvalid ? DO[(long long)(ob + qi) * a.ld_o + h * DH + part * Q4 + c] : 0.f;
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
        float* DQ = (float*)a.dq;
#pragma unroll
        for (int c = 0; c < Q4; c++)
            DQ[(long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c] = a.alpha * acc[c];
    }
}

// dkdv kernel: 64 key rows, 4 threads per key; queries staged 32 at a time.
template <int DH, bool RAB>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_f32_kernel(AttnArgs a) {
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
    const float* Q = (const float*)a.q;
    const float* K = (const float*)a.k;
    const float* V = (const float*)a.v;
    const float* DO = (const float*)a.dout;
    float kv[Q4], vv[Q4], dk[Q4], dv[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        kv[c] = kvalid ? K[(long long)(ob + kj) * a.ld_k + h * DH + part * Q4 + c] : 0.f;
        vv[c] = kvalid ? V[(long long)(ob + kj) * a.ld_v + h * DH + part * Q4 + c] : 0.f;
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
                sQ[row * KP + c] = qr < nb ? Q[(long long)(ob + qr) * a.ld_q + h * DH + c] : 0.f;
                sG[row * KP + c] = qr < nb ? DO[(long long)(ob + qr) * a.ld_o + h * DH + c] : 0.f;
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
        float* DK = (float*)a.dk;
        float* DV = (float*)a.dv;
#pragma unroll
        for (int c = 0; c < Q4; c++) {
            DK[(long long)(ob + kj) * a.ld_k + h * DH + part * Q4 + c] = a.alpha * dk[c];
            DV[(long long)(ob + kj) * a.ld_v + h * DH + part * Q4 + c] = dv[c];
        }
    }
}

// The relative bias enters the scores of both kernels (RAB_IN); drab is formed by the dq
// kernel only when the caller asked for it (a.drab != nullptr).
template <int DH, bool RAB_IN>
static hipError_t bwd_bf16_dh(const AttnArgs& a, int slots, bool dq, bool dkdv, hipStream_t s) {
    if (dq) {
        attn_bwd_dq_bf16_kernel<DH, RAB_IN><<<slots, 256, 0, s>>>(a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dkdv) {
        attn_bwd_dkdv_bf16_kernel<DH, RAB_IN><<<slots, 256, 0, s>>>(a);
        return hipGetLastError();
    }
    return hipSuccess;
}

template <int DH, bool RAB_IN>
static hipError_t bwd_f32_dh(const AttnArgs& a, int slots, bool dq, bool dkdv, hipStream_t s) {
    if (dq) {
        attn_bwd_dq_f32_kernel<DH, RAB_IN><<<slots, 256, 0, s>>>(a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (dkdv) {
        attn_bwd_dkdv_f32_kernel<DH, RAB_IN><<<slots, 256, 0, s>>>(a);
        return hipGetLastError();
    }
    return hipSuccess;
}

hipError_t launch_attn_bwd_bf16(const AttnArgs& a, int head_dim, int slots, bool dq, bool dkdv,
                                hipStream_t s) {
    const bool rab = a.rab != nullptr;
    switch (head_dim) {
        case 32: return rab ? bwd_bf16_dh<32, true>(a, slots, dq, dkdv, s) : bwd_bf16_dh<32, false>(a, slots, dq, dkdv, s);
        case 64: return rab ? bwd_bf16_dh<64, true>(a, slots, dq, dkdv, s) : bwd_bf16_dh<64, false>(a, slots, dq, dkdv, s);
        case 128: return rab ? bwd_bf16_dh<128, true>(a, slots, dq, dkdv, s) : bwd_bf16_dh<128, false>(a, slots, dq, dkdv, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_bwd_f32(const AttnArgs& a, int head_dim, int slots, bool dq, bool dkdv,
                               hipStream_t s) {
    const bool rab = a.rab != nullptr;
    switch (head_dim) {
        case 16: return rab ? bwd_f32_dh<16, true>(a, slots, dq, dkdv, s) : bwd_f32_dh<16, false>(a, slots, dq, dkdv, s);
        case 32: return rab ? bwd_f32_dh<32, true>(a, slots, dq, dkdv, s) : bwd_f32_dh<32, false>(a, slots, dq, dkdv, s);
        case 64: return rab ? bwd_f32_dh<64, true>(a, slots, dq, dkdv, s) : bwd_f32_dh<64, false>(a, slots, dq, dkdv, s);
        case 128: return rab ? bwd_f32_dh<128, true>(a, slots, dq, dkdv, s) : bwd_f32_dh<128, false>(a, slots, dq, dkdv, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mtgr
