// dQ of the attention backward from the dS blocks stored by the dK/dV kernel (bf16).
#include "attn_bwd_common.h"

namespace mtgr {
using bwd::BM;
using bwd::BN;
using bwd::ldg16;
using bwd::zero;

// ------------------------------------------------------------------ dQ from stored dS, bf16
// dQ^T (dh x 32 queries) += K^T dS^T over the user's visible 64-key tiles, with dS read from the
// blocks the dK/dV kernel stored (64 keys x 64 queries, already masked; 1 / n_b is applied here,
// in that kernel's register-fragment order: four 2 KB sub-blocks (query half, key half), each
// chunk (kq, g, lane) holding 4 queries 16 kq + 8 g + 4 (lane / 32) + 0..3 of key lane % 32).
// Per key tile the K tile and the two dS blocks of the workgroup's 128 queries stream through
// LDS.  Both MFMA operands come from ds_read_b64_tr_b16: K^T from the swizzled K tile, dS^T
// by pointing each supplier lane at the fragment chunk of (key, 4 queries) that the transpose
// must deliver.  A block exists only if the dK/dV kernel visited its (64 queries, 128 keys)
// pair; otherwise all its pairs are masked and the wave skips it.
template <int DH>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_ds_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8, DBLK = DH / 32, TILE = BN * DH, DSB = 64 * 64;
    __shared__ __align__(16) uint16_t sK0[TILE];
    __shared__ __align__(16) uint16_t sK1[TILE];
    __shared__ __align__(16) uint16_t sD0[2 * DSB];
    __shared__ __align__(16) uint16_t sD1[2 * DSB];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BM;
    const int ntk = (nb + BN - 1) / BN;
    const float scale = a.alpha / (float)nb;   // the stored dS lacks the factor 1 / n_b
    const int4* summ = a.summ + (long long)b * a.ntile;
    TileSummary sq = load_summary(summ, 2 * qt);
    if (2 * qt + 1 < ntk) sq = combine(sq, load_summary(summ, 2 * qt + 1));

    const int col = lane & 31, hh = lane >> 5;
    const int q64 = 2 * qt + (w >> 1);
    const bool qblk = q64 < ntk;
    const TileSummary sq64 = load_summary(summ, qblk ? q64 : ntk - 1);
    const long long blk0 = a.ds_off[b] + (long long)h * ntk * ntk;
    const uint16_t* Kb = (const uint16_t*)a.k + (long long)ob * a.ld_k;
    floatx16 dqacc[DBLK];
#pragma unroll
    for (int i = 0; i < DBLK; i++) zero(dqacc[i]);

    auto class_of = [&](int t) {
        const bool overlap = (t * BN < q0 + BM) && (q0 < t * BN + BN);
        return tile_class(sq, load_summary(summ, t), overlap);
    };
    TileWalker<decltype(class_of)> walk(class_of, ntk);
    // Blocks of this wave's 64 queries that the dK/dV kernel wrote (its key tiles are 128 wide).
    auto written_of = [&](int t) {
        const int kt = t >> 1;
        TileSummary sk = load_summary(summ, 2 * kt);
        if (2 * kt + 1 < ntk) sk = combine(sk, load_summary(summ, 2 * kt + 1));
        else sk.flags &= ~TS_ALL_STATIC;
        const bool overlap = (q64 * BN < kt * BM + BM) && (kt * BM < q64 * BN + BN);
        return tile_class(sq64, sk, overlap);
    };
    TileWalker<decltype(written_of)> written(written_of, ntk);
    // 8 KB block (read once: non-temporal copy): instruction i of wave w fills bytes
    // [1024 (4 i + w), +1024) of the LDS copy.
    // The 16-byte unit u = 128 sub-block + 32 row + v of the block (row = 2 kq + g, v = 16-byte
    // half of a fragment row) sits at u ^ dsw(u), which permutes units only inside aligned groups
    // of 16.  Stored as is, the 32 lanes of one transposing read below (4 rows x 8 chunks of one
    // fragment column range) hit 4 bank pairs, 8 lanes each; swizzled, 32 distinct ones.
    auto dsw = [](int u) {
        const int row = (u >> 5) & 3;
        return ((row & 1) << 1) | ((row >> 1) << 2) | (((u >> 4) & 1) << 3);
    };
    auto block_dma = [&](uint16_t* dst, const uint16_t* src) {
#pragma unroll
        for (int i = 0; i < 2; i++) {
            const int part = __builtin_amdgcn_readfirstlane(i * 4 + w);
            const int u = part * 64 + lane;
            lds_dma16_nt(__builtin_amdgcn_readfirstlane(lds_address(dst) + (uint32_t)part * 1024u),
                         uniform_ptr(src + part * 512), (uint32_t)((u ^ dsw(u)) & 63) * 16u);
        }
    };
    auto issue = [&](int t, int buf) {
        tile_dma<DH>(buf ? sK1 : sK0, Kb, a.ld_k, t * BN, nb, h * DH, tid);
#pragma unroll
        for (int j = 0; j < 2; j++)
            if (2 * qt + j < ntk)
                block_dma((buf ? sD1 : sD0) + j * DSB, a.ds + ((blk0 + (long long)(2 * qt + j) * ntk + t) << 12));
    };
    // Supplier address of this lane for the dS^T operand (query half w & 1 of its block):
    // group G = lane / 16 and index 4 s + q deliver key 8 p' + 4 (G / 2) + s and queries
    // 16 (G % 2) + 4 q .. + 3, i.e. chunk (kq = G % 2, g = q / 2, lane' = key % 32 + 32 (q % 2)).
    // k-step ks, half p of its 8 slots adds key offset 8 (2 ks + p): sub-block (2 ks + p) / 4,
    // chunk offset 8 ((2 ks + p) % 4).
    // In the swizzled copy the lane's unit moves by dsw (its row and v bit 4 fix it: the same for
    // every k-step), and the k-step's offset of 4 units is applied by XOR (the two touch the
    // same unit bits).
    const int gq = lane >> 4, sq_ = (lane & 15) >> 2, qq = lane & 3;
    const uint32_t ds_lane = (uint32_t)(w & 1) * 4096u +
                             ((uint32_t)(((2 * (gq & 1) + (qq >> 1)) * 64 + 32 * (qq & 1) + 4 * (gq >> 1) + sq_) * 8) ^
                              (uint32_t)((((qq >> 1) << 1) | ((gq & 1) << 2) | ((qq & 1) << 3)) * 16));
    auto ds_operand = [&](const uint16_t* blk, int ks) {
        const char* base = (const char*)blk;
        const int c0 = 2 * ks, c1 = 2 * ks + 1;
        const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_short4*)(base + (c0 >> 2) * 2048 + (ds_lane ^ (64u * (c0 & 3)))));
        const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_short4*)(base + (c1 >> 2) * 2048 + (ds_lane ^ (64u * (c1 & 3)))));
        const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, v);
    };

    int cls_unused, cls_n;
    int t = walk.next(0, &cls_unused);
    int cur = 0;
    if (t < ntk) issue(t, 0);
    while (t < ntk) {
        wait_vmem();
        lds_barrier();
        const int tn = walk.next(t + 1, &cls_n);
        if (tn < ntk) issue(tn, cur ^ 1);
        int wc;
        const bool use = qblk && written.next(t, &wc) == t;
        if (use) {
            const uint16_t* sK = cur ? sK1 : sK0;
            const uint16_t* sD = (cur ? sD1 : sD0) + (w >> 1) * DSB;
#pragma unroll
            for (int ks = 0; ks < 4; ks++) {
                const bf16x8 dst = ds_operand(sD, ks);
#pragma unroll
                for (int d = 0; d < DBLK; d++) {
                    const bf16x8 ktr = tile_read_tr<CPR>(sK, 16 * ks, 32 * d, lane);
                    dqacc[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ktr, dst, dqacc[d], 0, 0, 0);
                }
            }
        }
        t = tn;
        cur ^= 1;
    }
    // One barrier per tile suffices: the copy into a buffer is issued only after the barrier
    // that every wave passes once done with the tile that buffer held.  The tiles' LDS is
    // reused below.
    __syncthreads();

    uint16_t* sO = (w < 2 ? sK0 : sK1) + (w & 1) * 32 * DH;
#pragma unroll
    for (int d = 0; d < DBLK; d++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int dd = 32 * d + 8 * g + 4 * hh;
            *(uint2*)&sO[8 * tile_chunk<CPR>(col, dd >> 3) + (dd & 7)] =
                make_uint2(pack_bf16x2(scale * dqacc[d][4 * g + 0], scale * dqacc[d][4 * g + 1]),
                           pack_bf16x2(scale * dqacc[d][4 * g + 2], scale * dqacc[d][4 * g + 3]));
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

template __global__ void attn_bwd_dq_ds_bf16_kernel<32>(AttnArgs);
template __global__ void attn_bwd_dq_ds_bf16_kernel<64>(AttnArgs);
template __global__ void attn_bwd_dq_ds_bf16_kernel<128>(AttnArgs);
}  // namespace mtgr
