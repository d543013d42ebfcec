// Bias + SiLU of the encoder layer's projection (forward) and its derivative (backward).
// Memory-bound elementwise work on [rows, cols] matrices with row strides; one 16-byte chunk
// (8 bf16 or 4 fp32) per thread and step.  Every byte is read or written once: the bf16 chunks
// move with the non-temporal hint (measured on [69563, 4096]: bias + SiLU backward 0.303 ->
// 0.291 ms, the residual add on [69563, 1024] 0.077 -> 0.071 ms).
#include "mtgr_internal.h"
#include "mtgr_device.h"

namespace mtgr {

namespace {

template <bool BF16>
struct Chunk;

template <>
struct Chunk<true> {
    static constexpr int N = 8;
    __device__ static void load(const void* base, long long idx, float* out) {
        const u32x4_nt u = __builtin_nontemporal_load((const u32x4_nt*)((const uint16_t*)base + idx));
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ static void store(void* base, long long idx, const float* v) {
        const u32x4_nt u = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                            pack_bf16x2(v[6], v[7])};
        __builtin_nontemporal_store(u, (u32x4_nt*)((uint16_t*)base + idx));
    }
};

template <>
struct Chunk<false> {
    static constexpr int N = 4;
    __device__ static void load(const void* base, long long idx, float* out) {
        const float4 f = *(const float4*)((const float*)base + idx);
        out[0] = f.x;
        out[1] = f.y;
        out[2] = f.z;
        out[3] = f.w;
    }
    __device__ static void store(void* base, long long idx, const float* v) {
        *(float4*)((float*)base + idx) = make_float4(v[0], v[1], v[2], v[3]);
    }
};

// z = h + bias; forward: out = silu(z) = z sigmoid(z); backward: out = g silu'(z) with
// silu'(z) = sigmoid(z) (1 + z (1 - sigmoid(z))).
template <bool BF16, bool BWD>
__global__ __launch_bounds__(256) void bias_silu_kernel(long long rows, int cols, const void* h, long long ld_h,
                                                        const float* bias, const void* g, long long ld_g,
                                                        void* out, long long ld_out) {
    using C = Chunk<BF16>;
    constexpr int N = C::N;
    const int nch = cols / N;
    for (long long r = blockIdx.x; r < rows; r += gridDim.x) {
        for (int ch = threadIdx.x; ch < nch; ch += blockDim.x) {
            const int c = ch * N;
            float z[N];
            C::load(h, r * ld_h + c, z);
            if (bias != nullptr) {
#pragma unroll
                for (int i = 0; i < N; i++) z[i] += bias[c + i];
            }
            float o[N];
            if (BWD) C::load(g, r * ld_g + c, o);
#pragma unroll
            for (int i = 0; i < N; i++) {
                const float sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z[i]));
                o[i] = BWD ? o[i] * sg * (1.0f + z[i] * (1.0f - sg)) : z[i] * sg;
            }
            C::store(out, r * ld_out + c, o);
        }
    }
}

// out = a + b (the encoder layer's residual branch in the backward).
template <bool BF16>
__global__ __launch_bounds__(256) void add_kernel(long long rows, int cols, const void* a, long long lda,
                                                  const void* b, long long ldb, void* out, long long ldo) {
    using C = Chunk<BF16>;
    constexpr int N = C::N;
    const int nch = cols / N;
    for (long long r = blockIdx.x; r < rows; r += gridDim.x) {
        for (int ch = threadIdx.x; ch < nch; ch += blockDim.x) {
            float x[N], y[N];
            C::load(a, r * lda + ch * N, x);
            C::load(b, r * ldb + ch * N, y);
#pragma unroll
            for (int i = 0; i < N; i++) x[i] += y[i];
            C::store(out, r * ldo + ch * N, x);
        }
    }
}

}  // namespace

hipError_t launch_add(long long rows, int cols, bool bf16, const void* a, long long lda, const void* b,
                      long long ldb, void* out, long long ldo, hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int grid = (int)(rows < 16384 ? rows : 16384);
    if (bf16) add_kernel<true><<<grid, 256, 0, s>>>(rows, cols, a, lda, b, ldb, out, ldo);
    else add_kernel<false><<<grid, 256, 0, s>>>(rows, cols, a, lda, b, ldb, out, ldo);
    return hipGetLastError();
}

hipError_t launch_bias_silu(long long rows, int cols, bool bf16, bool backward, const void* h, long long ld_h,
                            const float* bias, const void* g, long long ld_g, void* out, long long ld_out,
                            hipStream_t s) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int grid = (int)(rows < 16384 ? rows : 16384);
    if (bf16) {
        if (backward) bias_silu_kernel<true, true><<<grid, 256, 0, s>>>(rows, cols, h, ld_h, bias, g, ld_g, out, ld_out);
        else bias_silu_kernel<true, false><<<grid, 256, 0, s>>>(rows, cols, h, ld_h, bias, g, ld_g, out, ld_out);
    } else {
        if (backward) bias_silu_kernel<false, true><<<grid, 256, 0, s>>>(rows, cols, h, ld_h, bias, g, ld_g, out, ld_out);
        else bias_silu_kernel<false, false><<<grid, 256, 0, s>>>(rows, cols, h, ld_h, bias, g, ld_g, out, ld_out);
    }
    return hipGetLastError();
}

}  // namespace mtgr
