// Shader clock under matrix-core load, for stating a kernel's fraction of the peak at the clock
// it actually ran at.  Every workgroup keeps its four SIMDs issuing v_mfma_f32_32x32x16_bf16
// back to back (four independent accumulator chains per wave) and records, around that loop,
// the shader-clock counter (s_memtime) and the constant-rate counter (s_memrealtime).
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

__global__ __launch_bounds__(256) void clock_probe_kernel(int iters, long long* out) {
    const int lane = threadIdx.x & 63;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; e++) {
        a[e] = (__bf16)(1.0f + 0.001f * (float)((lane + e) & 7));
        b[e] = (__bf16)(1.0f - 0.001f * (float)((lane * 3 + e) & 7));
    }
    floatx16 acc[4];
#pragma unroll
    for (int k = 0; k < 4; k++)
#pragma unroll
        for (int r = 0; r < 16; r++) acc[k][r] = 0.f;
    __syncthreads();
    const long long t0 = (long long)__builtin_amdgcn_s_memtime();
    const long long r0 = (long long)__builtin_amdgcn_s_memrealtime();
    for (int i = 0; i < iters; i++) {
#pragma unroll
        for (int k = 0; k < 4; k++) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < 4; k++) s += acc[k][0] + acc[k][15];
    __syncthreads();
    const long long t1 = (long long)__builtin_amdgcn_s_memtime();
    const long long r1 = (long long)__builtin_amdgcn_s_memrealtime();
    if (threadIdx.x == 0) {
        out[3 * blockIdx.x] = t1 - t0;
        out[3 * blockIdx.x + 1] = r1 - r0;
        out[3 * blockIdx.x + 2] = (long long)s;      // keeps the MFMA chains live
    }
}

hipError_t launch_clock_probe(int iters, int blocks, long long* out, hipStream_t s) {
    clock_probe_kernel<<<blocks, 256, 0, s>>>(iters, out);
    return hipGetLastError();
}

}  // namespace mtgr
