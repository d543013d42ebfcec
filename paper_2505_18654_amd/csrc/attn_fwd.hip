// Forward of the jagged dynamic-mask SiLU attention (Eq. 5, Sec. 4.2).
//
// bf16 kernel: one workgroup = 4 waves = 128 query rows of one (user, head); each wave owns
// 32 query rows.  For every 64-key tile of the user that is not fully masked, K and V are
// staged row-major through LDS (the next tile's rows are fetched into registers while the
// current one is computed) and the wave computes, per 32-key half of the tile,
//     S^T (32 keys x 32 queries) = K Q^T          v_mfma_f32_32x32x16_bf16, Q held in VGPRs
//     P = silu(alpha S + rab) / n_b, masked        in registers, straight from the accumulators
//     O^T (dh x 32 queries)     += V^T P^T         V^T read with ds_read_b64_tr_b16
// Computing the transposed products lets the accumulator layout of S^T (lane = query column,
// registers = keys) serve directly as the B operand of the second product, so P never goes
// through LDS, and the transposing LDS read gives V^T without a transposed copy.  The mask
// is evaluated only on PARTIAL tiles, from segment codes and timestamps staged with the keys.
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
    constexpr int KP = DH + 8;        // padded LDS row (elements)
    constexpr int OP = DH + 8;        // padded output staging row
    constexpr int KSTEPS = DH / 16;   // k-steps of S^T = K Q^T
    constexpr int DBLK = DH / 32;     // 32-row blocks of O^T
    constexpr int CPR = DH / 8;       // 16-byte chunks per row
    constexpr int KCH = BN * CPR / 256;
    constexpr int KV_BYTES = 2 * BN * KP * 2;
    constexpr int O_BYTES = BM * OP * 2;
    constexpr int BYTES = KV_BYTES > O_BYTES ? KV_BYTES : O_BYTES;

    __shared__ __align__(16) char smem[BYTES];
    __shared__ int sKcode[BN];
    __shared__ int sKts[BN];
    __shared__ float sRab[MTGR_RAB_LDS];
    uint16_t* sK = (uint16_t*)smem;
    uint16_t* sV = sK + BN * KP;

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
    const uint16_t* Q = (const uint16_t*)a.q;
    const uint16_t* K = (const uint16_t*)a.k;
    const uint16_t* V = (const uint16_t*)a.v;
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

    auto klass = [&](int t) {
        const bool overlap = (t * BN < q0 + BM) && (q0 < t * BN + BN);
        return tile_class(sq, load_summary(summ, t), overlap);
    };
    auto next_visible = [&](int t) {
        while (t < ntk && klass(t) == TILE_MASKED) ++t;
        return t;
    };

    uint4 kreg[KCH], vreg[KCH];
    int kcode_reg = 0, kts_reg = 0;
    auto gload = [&](int t) {
        const int kb = t * BN;
#pragma unroll
        for (int i = 0; i < KCH; i++) {
            const int c = tid + 256 * i, row = c / CPR, cc = c % CPR;
            const int key = kb + row;
            const bool ok = key < nb;
            kreg[i] = ok ? ldg16(K + (long long)(ob + key) * a.ld_k + h * DH + cc * 8) : make_uint4(0, 0, 0, 0);
            vreg[i] = ok ? ldg16(V + (long long)(ob + key) * a.ld_v + h * DH + cc * 8) : make_uint4(0, 0, 0, 0);
        }
        if (tid < BN) {
            const int key = kb + tid;
            kcode_reg = key < nb ? token_code(a.seg[ob + key]) : 0;
            kts_reg = key < nb ? a.ts[ob + key] : 0;
        }
    };
    auto sstore = [&]() {
#pragma unroll
        for (int i = 0; i < KCH; i++) {
            const int c = tid + 256 * i, row = c / CPR, cc = c % CPR;
            *(uint4*)&sK[row * KP + cc * 8] = kreg[i];
            *(uint4*)&sV[row * KP + cc * 8] = vreg[i];
        }
        if (tid < BN) {
            sKcode[tid] = kcode_reg;
            sKts[tid] = kts_reg;
        }
    };

    int t = next_visible(0);
    if (t < ntk) gload(t);
    while (t < ntk) {
        const int cls = klass(t);
        __syncthreads();
        sstore();
        __syncthreads();
        const int tn = next_visible(t + 1);
        if (tn < ntk) gload(tn);

#pragma unroll
        for (int blk = 0; blk < 2; blk++) {
            floatx16 sacc;
#pragma unroll
            for (int r = 0; r < 16; r++) sacc[r] = 0.f;
#pragma unroll
            for (int kk = 0; kk < KSTEPS; kk++) {
                const bf16x8 ka = *(const bf16x8*)&sK[(32 * blk + col) * KP + 16 * kk + 8 * hh];
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qreg[kk], sacc, 0, 0, 0);
            }
            // P in bf16 in B-operand order: pk[kq] holds keys 32 blk + 16 kq + 8(s/4) + 4hh + s%4.
            uint32_t pk[2][4];
#pragma unroll
            for (int r = 0; r < 16; r += 2) {
                float pv[2];
#pragma unroll
                for (int e = 0; e < 2; e++) {
                    const int rr = r + e;
                    const int kl = 32 * blk + 8 * (rr >> 2) + 4 * hh + (rr & 3);
                    float x = sacc[rr] * alpha;
                    if (RAB) x += sRab[rab_bucket(qts, sKts[kl], a.nbuckets)];
                    float sg;
                    float p = silu_sig(x, sg) * inv_n;
                    if (cls == TILE_PARTIAL)
                        p = visible(qcode, qts, qi, sKcode[kl], sKts[kl], t * BN + kl) ? p : 0.f;
                    pv[e] = p;
                }
                pk[r >> 3][(r & 7) >> 1] = pack_bf16x2(pv[0], pv[1]);
            }
#pragma unroll
            for (int kq = 0; kq < 2; kq++) {
                const bf16x8 pb = as_bf16x8(make_uint4(pk[kq][0], pk[kq][1], pk[kq][2], pk[kq][3]));
#pragma unroll
                for (int db = 0; db < DBLK; db++) {
                    const bf16x8 va = lds_read_tr(sV, KP, 32 * blk + 16 * kq, 32 * db, lane);
                    oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, oacc[db], 0, 0, 0);
                }
            }
        }
        t = tn;
    }

    // Output: O^T accumulators -> bf16 rows staged in LDS -> 16-byte coalesced stores.
    __syncthreads();
    uint16_t* sO = (uint16_t*)smem;
#pragma unroll
    for (int db = 0; db < DBLK; db++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int d = 32 * db + 8 * g + 4 * hh;
            *(uint2*)&sO[(w * 32 + col) * OP + d] =
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
                *(const uint4*)&sO[(w * 32 + row) * OP + cc * 8];
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
