// Dense bf16 products of the encoder layer around the attention (Sec. 4.2: the projection MLPs
// that form Q, K, V, U, and the top MLP of Eq. 6), with the layer's elementwise work fused:
//   C = op(A) op(B) with op(A) [M, K], op(B) [K, N], fp32 accumulation on the bf16 matrix cores;
//   epilogue NONE:          C = acc
//            BIAS_SILU:     C = acc (the pre-activation, kept for the backward),
//                           C2 = silu(acc + bias)          (the projection's activation)
//            BIAS_RESIDUAL: C = acc + bias + R             (the top MLP plus the residual)
//   layout NN: A [M, K], B [K, N] row-major          (forward products)
//          NT: A [M, K], B [N, K] row-major, C = A B^T (input gradients: dY W^T)
//          TN: A [K, M], B [K, N] row-major, C = A^T B (weight gradients: X^T dY, K = tokens),
//              split over K into fp32 partials that a second kernel adds in a fixed order, with
//              the column sums of B (the bias gradient) formed on the way.
//
// Workgroup: 4 waves, a 256 (m) x 128 (n) tile of C, k in steps of 32 through three LDS stages
// filled by global_load_lds one or two steps ahead.  The products are computed transposed,
// C^T block = B^T A^T (v_mfma_f32_32x32x16_bf16), so that a lane's accumulators hold one row of
// C at 4 consecutive columns per register group: the epilogue reads bias / residual and writes
// C in 8-byte pieces per row without an LDS round trip.  An operand whose k index is contiguous
// in memory (A of NN / NT, B of NT) sits in LDS as [rows][32 k] and is read 16 bytes per lane;
// one whose k index runs over rows (B of NN / TN, A of TN) sits as [32 k][cols] and is read
// with the transposing ds_read_b64_tr_b16, the supplier rows chosen so that both operands use
// the natural k order of the instruction (lane half hf holds k = 8 hf .. 8 hf + 7).
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

namespace {

constexpr int GBM = 256, GBN = 128, GBK = 32, GSTAGES = 3;
constexpr int A_ELEMS = GBM * GBK, B_ELEMS = GBN * GBK;

// Operand read from a [32 k][cols] tile (CPR 16-byte chunks per row): lane l receives column
// c0 + l % 32 at k rows k0 + 8 hf + 0..7 (hf = l / 32), the natural k order of the MFMA operand.
template <int CPR>
__device__ __forceinline__ bf16x8 kr_read(const uint16_t* tile, int k0, int c0, int lane) {
    const int j = lane & 15, hf = lane >> 5;
    const int row = k0 + 8 * hf + (j >> 2);
    const int colx = c0 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const uint16_t* p0 = tile + 8 * tile_chunk<CPR>(row, colx >> 3) + (colx & 7);
    const uint16_t* p1 = tile + 8 * tile_chunk<CPR>(row + 4, colx >> 3) + (colx & 7);
    const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p0);
    const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p1);
    const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Operand read from a [rows][32 k] tile: row r, k16 step ks, natural k order.
__device__ __forceinline__ bf16x8 kc_read(const uint16_t* tile, int r, int ks, int lane) {
    return tile_read8<4>(tile, r, 2 * ks + (lane >> 5));
}

__device__ __forceinline__ float silu(float z) {
    return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}

}  // namespace

template <int LAYOUT, int EPI, bool COLSUM>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmArgs g) {
    constexpr bool A_KR = LAYOUT == GEMM_TN;      // A stored [K][M]
    constexpr bool B_KR = LAYOUT != GEMM_NT;      // B stored [K][N]
    constexpr bool SPLIT = LAYOUT == GEMM_TN;     // fp32 partials per K split
    __shared__ __align__(16) uint16_t sA[GSTAGES][A_ELEMS];
    __shared__ __align__(16) uint16_t sB[GSTAGES][B_ELEMS];
    __shared__ float sCol[COLSUM ? 2 * GBN : 1];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int col = lane & 31, hf = lane >> 5;
    // workgroups of one XCD (blockIdx % 8) take the n blocks of one m block one after another,
    // so the A rows of that block stay in the XCD's L2
    const int bid = blockIdx.x, x = bid % XCDS, jx = bid / XCDS;
    const int mb = x + XCDS * (jx / g.nblocks), nb = jx % g.nblocks;
    if (mb >= g.mblocks) return;
    const int m0 = mb * GBM, n0 = nb * GBN;
    const int split = blockIdx.y;
    const int nks = (int)((g.K + GBK - 1) / GBK);
    const int ks_begin = split * g.ks_per_split;
    const int ks_end = min(nks, ks_begin + g.ks_per_split);
    const int nk = max(ks_end - ks_begin, 0);
    const uint16_t* A = (const uint16_t*)g.A;
    const uint16_t* B = (const uint16_t*)g.B;
    const bool colsum = COLSUM && mb == 0;

    auto issue = [&](int i) {
        const int st = i % GSTAGES;
        const int k0 = (ks_begin + i) * GBK;
        if constexpr (A_KR) tile_dma<GBM, GBK>(sA[st], A, g.lda, k0, (int)g.K, m0, tid);
        else tile_dma<GBK, GBM>(sA[st], A, g.lda, m0, (int)g.M, k0, tid);
        if constexpr (B_KR) tile_dma<GBN, GBK>(sB[st], B, g.ldb, k0, (int)g.K, n0, tid);
        else tile_dma<GBK, GBN>(sB[st], B, g.ldb, n0, (int)g.N, k0, tid);
    };
    constexpr int NI = GBM * GBK / 8 / 256 + GBN * GBK / 8 / 256;   // copy instructions per stage

    floatx16 acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; a++)
#pragma unroll
        for (int b = 0; b < 2; b++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[a][b][r] = 0.f;
    float csum = 0.f;

    if (nk > 0) issue(0);
    if (nk > 1) issue(1);
    for (int i = 0; i < nk; i++) {
        const int st = i % GSTAGES;
        if (i + 1 < nk) wait_vmcnt<NI>(); else wait_vmem();
        const int k0 = (ks_begin + i) * GBK;
        if constexpr (A_KR) {
            // the last k step of a ragged K: rows past K hold copies of row K - 1 (the copy
            // clamps); zero them in both tiles so that they add nothing
            const int valid = (int)min(g.K - k0, (long long)GBK);
            if (valid < GBK) {
                lds_barrier();
                uint4* za = (uint4*)sA[st];
                uint4* zb = (uint4*)sB[st];
                for (int c = tid; c < (GBK - valid) * (GBM / 8); c += 256) za[valid * (GBM / 8) + c] = make_uint4(0, 0, 0, 0);
                for (int c = tid; c < (GBK - valid) * (GBN / 8); c += 256) zb[valid * (GBN / 8) + c] = make_uint4(0, 0, 0, 0);
            }
        }
        lds_barrier();
        if (i + 2 < nk) issue(i + 2);      // into the stage read in step i - 1
        const uint16_t* tA = sA[st];
        const uint16_t* tB = sB[st];
        if (COLSUM && colsum) {
            // bias gradient: column sums of B over this K split (two threads per column)
            const int c = tid & (GBN - 1), h = tid >> 7;
#pragma unroll 4
            for (int r = 16 * h; r < 16 * h + 16; r++)
                csum += bf16_to_f32(tB[8 * tile_chunk<GBN / 8>(r, c >> 3) + (c & 7)]);
        }
#pragma unroll
        for (int ks = 0; ks < GBK / 16; ks++) {
            bf16x8 aop[4], bop[2];
#pragma unroll
            for (int a = 0; a < 4; a++) {
                if constexpr (B_KR) aop[a] = kr_read<GBN / 8>(tB, 16 * ks, 32 * a, lane);
                else aop[a] = kc_read(tB, 32 * a + col, ks, lane);
            }
#pragma unroll
            for (int b = 0; b < 2; b++) {
                if constexpr (A_KR) bop[b] = kr_read<GBM / 8>(tA, 16 * ks, 64 * w + 32 * b, lane);
                else bop[b] = kc_read(tA, 64 * w + 32 * b + col, ks, lane);
            }
#pragma unroll
            for (int a = 0; a < 4; a++)
#pragma unroll
                for (int b = 0; b < 2; b++)
                    acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aop[a], bop[b], acc[a][b], 0, 0, 0);
        }
    }

    // acc[a][b] holds C^T of rows n0 + 32 a + 8 (r / 4) + 4 hf + r % 4, columns m0 + 64 w + 32 b + col:
    // lane row gm of C, columns gn .. gn + 3 per register group q = r / 4.
#pragma unroll
    for (int b = 0; b < 2; b++) {
        const long long gm = m0 + 64 * w + 32 * b + col;
        if (gm >= g.M) continue;
#pragma unroll
        for (int a = 0; a < 4; a++) {
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const int gn = n0 + 32 * a + 8 * q + 4 * hf;
                float v[4] = {acc[a][b][4 * q], acc[a][b][4 * q + 1], acc[a][b][4 * q + 2], acc[a][b][4 * q + 3]};
                if constexpr (SPLIT) {
                    float* P = g.partial + ((long long)split * g.M + gm) * g.N + gn;
                    *(float4*)P = make_float4(v[0], v[1], v[2], v[3]);
                    continue;
                }
                uint16_t* C = (uint16_t*)g.C + gm * g.ldc + gn;
                if constexpr (EPI == GEMM_EPI_BIAS_SILU) {
                    *(uint2*)C = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                    const float4 bi = *(const float4*)(g.bias + gn);
                    uint16_t* C2 = (uint16_t*)g.C2 + gm * g.ldc2 + gn;
                    *(uint2*)C2 = make_uint2(pack_bf16x2(silu(v[0] + bi.x), silu(v[1] + bi.y)),
                                             pack_bf16x2(silu(v[2] + bi.z), silu(v[3] + bi.w)));
                } else if constexpr (EPI == GEMM_EPI_BIAS_RESIDUAL) {
                    const float4 bi = *(const float4*)(g.bias + gn);
                    const uint2 rr = *(const uint2*)((const uint16_t*)g.R + gm * g.ldr + gn);
                    v[0] += bi.x + __uint_as_float(rr.x << 16);
                    v[1] += bi.y + __uint_as_float(rr.x & 0xffff0000u);
                    v[2] += bi.z + __uint_as_float(rr.y << 16);
                    v[3] += bi.w + __uint_as_float(rr.y & 0xffff0000u);
                    *(uint2*)C = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                } else {
                    *(uint2*)C = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
                }
            }
        }
    }
    if (COLSUM && colsum) {
        sCol[tid] = csum;
        __syncthreads();
        if (tid < GBN) g.colsum_partial[(long long)split * g.N + n0 + tid] = sCol[tid] + sCol[tid + GBN];
    }
}

// Sum of the K-split partials in a fixed order: C = bf16(sum_s partial[s]) and, with column
// sums, colsum = sum_s colsum_partial[s] (fp32).
__global__ __launch_bounds__(256) void gemm_split_reduce_kernel(GemmArgs g) {
    const long long MN4 = g.M * g.N / 4;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i < MN4; i += (long long)gridDim.x * 256) {
        const long long e = 4 * i, m = e / g.N, n = e % g.N;
        float4 s = *(const float4*)(g.partial + e);
        for (int p = 1; p < g.splits; p++) {
            const float4 t = *(const float4*)(g.partial + (long long)p * g.M * g.N + e);
            s.x += t.x; s.y += t.y; s.z += t.z; s.w += t.w;
        }
        *(uint2*)((uint16_t*)g.C + m * g.ldc + n) = make_uint2(pack_bf16x2(s.x, s.y), pack_bf16x2(s.z, s.w));
    }
    if (g.colsum && blockIdx.x == 0) {
        for (int n = threadIdx.x; n < g.N; n += 256) {
            float s = 0.f;
            for (int p = 0; p < g.splits; p++) s += g.colsum_partial[(long long)p * g.N + n];
            g.colsum[n] = s;
        }
    }
}

void gemm_plan(int layout, long long M, long long N, long long K, int* mblocks, int* nblocks, int* splits,
               int* ks_per_split) {
    *mblocks = (int)((M + GBM - 1) / GBM);
    *nblocks = (int)(N / GBN);
    const int nks = (int)((K + GBK - 1) / GBK);
    int s = 1;
    if (*mblocks == 0 || *nblocks == 0 || nks == 0) {     // empty product: nothing is launched
        *splits = 1;
        *ks_per_split = 0;
        return;
    }
    if (layout == GEMM_TN) {
        // enough workgroups for two per CU, each split at least 8 k steps
        const long long tiles = (long long)*mblocks * *nblocks;
        s = (int)((512 + tiles - 1) / tiles);
        s = max(1, min(s, nks / 8));
        s = min(s, 64);
    }
    *ks_per_split = (nks + s - 1) / s;
    *splits = (nks + *ks_per_split - 1) / *ks_per_split;
    if (*splits < 1) *splits = 1;
}

size_t gemm_workspace_bytes(int layout, long long M, long long N, long long K) {
    if (layout != GEMM_TN) return 0;
    int mb, nb, s, per;
    gemm_plan(layout, M, N, K, &mb, &nb, &s, &per);
    return (size_t)s * (size_t)(M * N + N) * sizeof(float);
}

template <int LAYOUT, int EPI, bool COLSUM>
static hipError_t gemm_launch(const GemmArgs& g, hipStream_t s) {
    const int gx = XCDS * ((g.mblocks + XCDS - 1) / XCDS) * g.nblocks;
    gemm_bf16_kernel<LAYOUT, EPI, COLSUM><<<dim3(gx, g.splits), 256, 0, s>>>(g);
    return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& g, hipStream_t s) {
    hipError_t e = hipSuccess;
    switch (g.layout) {
        case GEMM_NN:
            if (g.epilogue == GEMM_EPI_BIAS_SILU) e = gemm_launch<GEMM_NN, GEMM_EPI_BIAS_SILU, false>(g, s);
            else if (g.epilogue == GEMM_EPI_BIAS_RESIDUAL) e = gemm_launch<GEMM_NN, GEMM_EPI_BIAS_RESIDUAL, false>(g, s);
            else e = gemm_launch<GEMM_NN, GEMM_EPI_NONE, false>(g, s);
            return e;
        case GEMM_NT:
            if (g.epilogue == GEMM_EPI_BIAS_SILU) e = gemm_launch<GEMM_NT, GEMM_EPI_BIAS_SILU, false>(g, s);
            else if (g.epilogue == GEMM_EPI_BIAS_RESIDUAL) e = gemm_launch<GEMM_NT, GEMM_EPI_BIAS_RESIDUAL, false>(g, s);
            else e = gemm_launch<GEMM_NT, GEMM_EPI_NONE, false>(g, s);
            return e;
        case GEMM_TN:
            e = g.colsum ? gemm_launch<GEMM_TN, GEMM_EPI_NONE, true>(g, s) : gemm_launch<GEMM_TN, GEMM_EPI_NONE, false>(g, s);
            if (e != hipSuccess) return e;
            gemm_split_reduce_kernel<<<(int)min((g.M * g.N / 4 + 255) / 256, 8192ll), 256, 0, s>>>(g);
            return hipGetLastError();
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mtgr
