// dK, dV (and drab, and optionally the stored dS blocks) of the attention backward (bf16).
#include "attn_bwd_common.h"

namespace mtgr {
using bwd::BM;
using bwd::BN;
using bwd::ldg16;
using bwd::zero;

// ------------------------------------------------------------------ dK, dV, bf16
// A workgroup owns 128 keys (32 per wave) of one (user, head).  K of those keys stays in LDS
// for the whole kernel and V in VGPRs; the visible queries stream through LDS 32 at a time
// (Q and dO rows plus their timestamps and mask codes, double-buffered, copied with
// global_load_lds one unit ahead).  Per unit a wave forms S and dP (32 queries x its 32 keys),
// then P and dS in registers, and accumulates dV += P^T dO and dK += dS^T Q.  Reading K from
// LDS instead of registers keeps the wave within 256 VGPRs without spilling: a scratch reload
// issued after a prefetch would have to wait for that prefetch (vector-memory operations
// complete in issue order), serialising copy and compute.
// With STORE it also writes dS (bf16, the A operand of its dK product, masked but without the
// factor 1 / n_b) as 64 x 64 blocks for the dQ-from-dS kernel; it forms drab when a.drab is set.
template <int DH, bool RAB, bool STORE>
__global__ __launch_bounds__(256, 2) void attn_bwd_dkdv_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8, KSTEPS = DH / 16, DBLK = DH / 32, UNIT = 32 * DH;
    __shared__ __align__(16) uint16_t sK[BM * DH];
    // Query unit buffers: Q then dO of one unit in one array, so that a dO operand sits a constant
    // distance from the Q operand read with the same lane offset (one address for both reads).
    __shared__ __align__(16) uint16_t sQG[2][2 * UNIT];
    __shared__ __align__(16) int sQts[2][32];
    __shared__ __align__(16) int sQcode[2][32];
    __shared__ float sRab[MTGR_RAB_LDS];
    __shared__ float sHist[RAB ? bwd::HIST_WORDS : 1];

    const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, kt = item.y >> 8, h = item.y & 255;
    const bool want_drab = RAB && a.drab != nullptr;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int k0 = kt * BM;
    const int ntq = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const float alpha = a.alpha;
    const float c_exp = -1.4426950408889634f * alpha;   // sigmoid(alpha s) = 1 / (1 + 2^(c_exp s))
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
    const uint16_t* V = (const uint16_t*)a.v;
    const uint16_t* Kb = (const uint16_t*)a.k + (long long)ob * a.ld_k;
    const uint16_t* Qb = (const uint16_t*)a.q + (long long)ob * a.ld_q;
    const uint16_t* Gb = (const uint16_t*)a.dout + (long long)ob * a.ld_o;
    bf16x8 vreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; kk++) {
        uint4 g = make_uint4(0, 0, 0, 0);
        if (kvalid) g = ldg16(V + (long long)(ob + kj) * a.ld_v + h * DH + 16 * kk + 8 * hh);
        vreg[kk] = as_bf16x8(g);
    }
    if (RAB) {
        if (tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;
        bwd::hist_zero(sHist, tid);
    }
    // stored dS: block (query tile q, key tile k) of this (user, head) is ds_blk + q ntq + k;
    // this wave's 32 keys are keys 32 (w & 1) .. 32 (w & 1) + 31 of key tile kblk.
    const int kblk = (k0 + 32 * w) >> 6;
    const bool store_rows = STORE && kblk < ntq;
    const long long ds_blk = STORE ? a.ds_off[b] + (long long)h * ntq * ntq + kblk : 0;
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
    // Unit (t, half): queries 64 t + 32 half .. + 31 (the second half of a tile is skipped
    // when it starts past the user's end, so every copied unit holds a valid row).
    auto issue = [&](int t, int half, int buf) {
        const int r0 = t * BN + 32 * half;
        tile_dma_pair<DH, 32>(sQG[buf], Qb, a.ld_q, sQG[buf] + UNIT, Gb, a.ld_o, r0, nb, h * DH, tid);
        codes_dma<32>(sQts[buf], sQcode[buf], a.ts + ob, a.tok_code + ob, r0, nb, tid);
    };

    int cls, cls_n;
    int t = walk.next(0, &cls), half = 0, buf = 0;
    if (t < ntq) {
        tile_dma<DH, BM>(sK, Kb, a.ld_k, k0, nb, h * DH, tid);
        issue(t, 0, 0);
    }
    wait_vmcnt_seen<0>();   // K, V, the first unit
    bwd::HistRun run;   // drab: this lane's current run of equal buckets
    bool first = true;
    while (t < ntq) {
        // The copy of this unit was issued before the previous unit's 4 dS stores.
        if (!first) {
            if (STORE && store_rows) wait_vmcnt_seen<4>();
            else wait_vmcnt_seen<0>();
        }
        first = false;
        const int qb = t * BN + 32 * half;
        if (tid < 32 && qb + tid >= nb) sQcode[buf][tid] = 0;
        lds_barrier();
        int tn = t, hn = 1;
        cls_n = cls;
        if (half == 1 || t * BN + 32 >= nb) {
            tn = walk.next(t + 1, &cls_n);
            hn = 0;
        }
        if (tn < ntq) issue(tn, hn, buf ^ 1);
        const uint16_t* sQ = sQG[buf];
        const uint16_t* sG = sQ + UNIT;
        const int* qts = sQts[buf];
        const int* qcode = sQcode[buf];

        // S (32 q x 32 keys) = Q K^T and dP = dO V^T: lane = key column, registers = queries.
        // The LDS operands of k-step kk + PF_S are read while k-step kk's MFMAs issue; the
        // scheduling fence after each step keeps the compiler from sinking the reads next to
        // their use (it did, to save registers, and every MFMA then waited a full LDS round trip).
        floatx16 sacc, dpacc;
        zero(sacc);
        zero(dpacc);
        constexpr int PF_S = 1;
        bf16x8 qa[KSTEPS], ga[KSTEPS], kb[KSTEPS];
        auto load_s = [&](int kk) {
            qa[kk] = tile_read8<CPR>(sQ, col, 2 * kk + hh);
            ga[kk] = tile_read8<CPR>(sG, col, 2 * kk + hh);
            kb[kk] = tile_read8<CPR>(sK, 32 * w + col, 2 * kk + hh);
        };
#pragma unroll
        for (int kk = 0; kk < PF_S && kk < KSTEPS; kk++) load_s(kk);
#pragma unroll
        for (int kk = 0; kk < KSTEPS; kk++) {
            if (kk + PF_S < KSTEPS) load_s(kk + PF_S);
            sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[kk], kb[kk], sacc, 0, 0, 0);
            dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ga[kk], vreg[kk], dpacc, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        uint32_t pk[2][4], dsk[2][4];
        // dV (32 keys x dh) += P^T dO ; dK += dS^T Q.  A = P^T / dS^T from registers,
        // B = dO / Q read transposed (lane = feature column, slots = queries).  Step j =
        // (kq, d) = (j / DBLK, j % DBLK); its operands are read PF_D steps ahead, as above.
        constexpr int NJ = 2 * DBLK, PF_D = 2;
        bf16x8 gbs[NJ], qbs[NJ];
        auto load_d = [&](int j) {
            gbs[j] = tile_read_tr<CPR>(sG, 16 * (j / DBLK), 32 * (j % DBLK), lane);
            qbs[j] = tile_read_tr<CPR>(sQ, 16 * (j / DBLK), 32 * (j % DBLK), lane);
        };
        bf16x8 pa[2], da[2];
        auto operands = [&](int kq) {
            pa[kq] = as_bf16x8(make_uint4(pk[kq][0], pk[kq][1], pk[kq][2], pk[kq][3]));
            da[kq] = as_bf16x8(make_uint4(dsk[kq][0], dsk[kq][1], dsk[kq][2], dsk[kq][3]));
        };
        auto product = [&](int j) {
            const int kq = j / DBLK, d = j % DBLK;
            dvacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa[kq], gbs[j], dvacc[d], 0, 0, 0);
            dkacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da[kq], qbs[j], dkacc[d], 0, 0, 0);
        };
        // Element rr belongs to query 8 (rr / 4) + 4 hh + rr % 4.  p and ds are P and dS
        // without the per-user factor 1 / n_b (and, without a relative bias, P without alpha):
        // the factors are applied once to dK, dV, dQ and drab.  silu'(x) = sg + x sg (1 - sg),
        // and x sg = alpha p (without a bias; p itself with one), so dS = dP (sg + alpha p (1 - sg))
        // reuses p: p (1 - sg) is one fma.
        auto mask = [&](int rr, float& p, float& ds) {
            const int ql = 8 * (rr >> 2) + 4 * hh + (rr & 3);
            const bool vis = visible(qcode[ql], qts[ql], qb + ql, kcode, kts, kj);
            p = vis ? p : 0.f;
            ds = vis ? ds : 0.f;
        };
        if constexpr (!RAB) {
            // Elements 0..7 (queries 0..15) first; then elements 8..15 interleave with the
            // dV / dK products of queries 0..15, so that one wave overlaps its own VALU and
            // MFMA work; then the products of queries 16..31.  The mask of a PARTIAL unit is
            // one branch per half, after its straight-line element math.
            // The fmas are explicit, so that every instantiation (with and without the dS store)
            // rounds alike and their dK / dV agree bit for bit.
            auto element = [&](int rr, float& p, float& ds) {
                const float sv = sacc[rr];
                const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(sv * c_exp));
                p = sv * sg;
                ds = dpacc[rr] * __builtin_fmaf(alpha, __builtin_fmaf(-p, sg, p), sg);
            };
            float pv[16], dv[16];
#pragma unroll
            for (int rr = 0; rr < 8; rr++) element(rr, pv[rr], dv[rr]);
            if (cls == TILE_PARTIAL) {
#pragma unroll
                for (int rr = 0; rr < 8; rr++) mask(rr, pv[rr], dv[rr]);
            }
#pragma unroll
            for (int r = 0; r < 8; r += 2) {
                pk[0][r >> 1] = pack_bf16x2(pv[r], pv[r + 1]);
                dsk[0][r >> 1] = pack_bf16x2(dv[r], dv[r + 1]);
            }
            operands(0);
            // Operands one step ahead here (two spilled); 8 / DBLK elements per step.
            constexpr int EPS = 8 / DBLK;
            load_d(0);
#pragma unroll
            for (int j = 0; j < DBLK; j++) {
                load_d(j + 1);
                product(j);
#pragma unroll
                for (int e = 8 + EPS * j; e < 8 + EPS * (j + 1); e++) element(e, pv[e], dv[e]);
                // Pin the products here: their results are read only by later products, and
                // the compiler otherwise sinks them all behind the element math.
                asm volatile("" : "+v"(dvacc[j]), "+v"(dkacc[j]));
                __builtin_amdgcn_sched_barrier(0);
            }
            if (cls == TILE_PARTIAL) {
#pragma unroll
                for (int rr = 8; rr < 16; rr++) mask(rr, pv[rr], dv[rr]);
            }
#pragma unroll
            for (int r = 8; r < 16; r += 2) {
                pk[1][(r - 8) >> 1] = pack_bf16x2(pv[r], pv[r + 1]);
                dsk[1][(r - 8) >> 1] = pack_bf16x2(dv[r], dv[r + 1]);
            }
        } else {
            // With a relative bias: groups of 4 elements (their bucket indices, then their bias
            // values read from LDS) keep the live registers within budget.  As without a bias,
            // elements 0..7 (queries 0..15) come first and elements 8..15 interleave with the
            // dV / dK products of queries 0..15, so that the wave overlaps its own VALU and
            // MFMA work.
            // The 4 queries of a group are consecutive (8 (g0 / 4) + 4 hh + 0..3): their
            // timestamps (and, for a partial unit, mask codes) are one 16-byte LDS read each.
            typedef int i32x4 __attribute__((ext_vector_type(4)));
            auto group = [&](int g0) {
                float pv[4], dv[4];
                int bk[4];
                const int qb0 = 8 * (g0 >> 2) + 4 * hh;
                const i32x4 qt4 = *(const i32x4*)&qts[qb0];
#pragma unroll
                for (int e = 0; e < 4; e++) bk[e] = rab_bucket(qt4[e], kts, a.nbuckets);
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    // (the forward's scaled exponent, one operation fewer here, spilled two more
                    // registers into this loop and was 3 % slower)
                    const float x = sacc[g0 + e] * alpha + sRab[bk[e]];
                    const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(NEG_LOG2E * x));
                    pv[e] = x * sg;
                    dv[e] = dpacc[g0 + e] * (__builtin_fmaf(-pv[e], sg, pv[e]) + sg);
                }
                if (cls == TILE_PARTIAL) {
                    const i32x4 qc4 = *(const i32x4*)&qcode[qb0];
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const bool vis = visible(qc4[e], qt4[e], qb + qb0 + e, kcode, kts, kj);
                        pv[e] = vis ? pv[e] : 0.f;
                        dv[e] = vis ? dv[e] : 0.f;
                    }
                }
#pragma unroll
                for (int e = 0; e < 4; e += 2) {
                    const int r = g0 + e;
                    pk[r >> 3][(r & 7) >> 1] = pack_bf16x2(pv[e], pv[e + 1]);
                    dsk[r >> 3][(r & 7) >> 1] = pack_bf16x2(dv[e], dv[e + 1]);
                }
                if (want_drab) {
#pragma unroll
                    for (int e = 0; e < 4; e++) run.add(sHist, lane, bk[e], dv[e]);
                }
            };
            group(0);
            group(4);
            operands(0);
            load_d(0);
#pragma unroll
            for (int j = 0; j < DBLK; j++) {
                load_d(j + 1);
                product(j);
                // groups 8 and 12 spread over the DBLK products of queries 0..15
#pragma unroll
                for (int gi = 0; gi < 2; gi++)
                    if (gi * DBLK / 2 == j) group(8 + 4 * gi);
                asm volatile("" : "+v"(dvacc[j]), "+v"(dkacc[j]));
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (store_rows) {
            // Sub-block (query half, key half) of block (t, kblk), 2 KB in register-fragment
            // order: chunk (kq, g, lane) = 4 bf16 of dS for key 32 (w & 1) + lane % 32 and
            // queries 32 half + 16 kq + 8 g + 4 (lane / 32) + 0..3, i.e. dsk[kq][2g], dsk[kq][2g+1].
            // Each of the 4 store instructions writes 512 contiguous bytes (non-temporal: the dQ
            // kernel reads the block once, later).
            uint2* sub = (uint2*)(a.ds + ((ds_blk + (long long)t * ntq) << 12)) + (2 * half + (w & 1)) * 256;
#pragma unroll
            for (int kq = 0; kq < 2; kq++)
#pragma unroll
                for (int g = 0; g < 2; g++)
                    store_nt8(&sub[(2 * kq + g) * 64 + lane], dsk[kq][2 * g], dsk[kq][2 * g + 1]);
        }
        // Operands 0 .. DBLK have been read (one step ahead); the rest go two steps ahead.
        operands(1);
        if constexpr (DBLK + 1 < NJ) load_d(DBLK + 1);
#pragma unroll
        for (int j = DBLK; j < NJ; j++) {
            if (j + PF_D < NJ) load_d(j + PF_D);
            product(j);
            __builtin_amdgcn_sched_barrier(0);
        }
        t = tn;
        half = hn;
        cls = cls_n;
        buf ^= 1;
    }

    if (want_drab) {
        run.flush(sHist, lane);
        __syncthreads();   // every wave's histogram updates have landed
        if (tid < a.nbuckets) {
            const float v = bwd::hist_total(sHist, tid);
            if (v != 0.f) atomicAdd(&a.drab[h * a.nbuckets + tid], v * inv_n);
        }
    }
    // dK / dV accumulators: lane = feature column, registers = key rows.  Each wave stages
    // its 32 rows in a swizzled 32-row tile inside the K tile.
    uint16_t* sO = sK + w * 32 * DH;
    const float dk_scale = alpha * inv_n, dv_scale = RAB ? inv_n : alpha * inv_n;
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
                const float val = which == 0 ? dk_scale * dkacc[d][r] : dv_scale * dvacc[d][r];
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
                store_nt16(dst + (long long)(ob + kr) * ld + h * DH + cc * 8, &sO[8 * tile_chunk<CPR>(row, cc)]);
        }
    }
}

template __global__ void attn_bwd_dkdv_bf16_kernel<32, false, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<32, false, true>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<32, true, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<32, true, true>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<64, false, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<64, false, true>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<64, true, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<64, true, true>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<128, false, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<128, false, true>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<128, true, false>(AttnArgs);
template __global__ void attn_bwd_dkdv_bf16_kernel<128, true, true>(AttnArgs);
}  // namespace mtgr
