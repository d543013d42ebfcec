// Gate + Group-LayerNorm (Eq. 6 up to the MLP: y = GroupLN(x (*) u)), forward and backward.
//
// Memory-bound: one wave per token row, 16-byte vector loads, wave reductions through
// cross-lane shuffles, two-pass variance on values held in registers.  Each wave walks a
// run of consecutive tokens; since a user's tokens come segment by segment ([U|S|R|I]) and
// the groups are the segments, gamma/beta rows stay in registers across a run and are only
// re-read when the group changes.  The backward keeps dgamma/dbeta partials for the current
// group in registers and flushes them with fp32 atomics when the group changes.
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

namespace {
constexpr int WAVES = 4;
constexpr int TOKENS_PER_WAVE = 16;

template <bool BF16>
struct Vec;   // 16-byte chunk of the storage type

template <>
struct Vec<true> {
    static constexpr int N = 8;
    __device__ static void load(const void* base, long long idx, float* out) {
        const uint4 u = *(const uint4*)((const uint16_t*)base + idx);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ static void store(void* base, long long idx, const float* v) {
        uint4 u;
        u.x = pack_bf16x2(v[0], v[1]);
        u.y = pack_bf16x2(v[2], v[3]);
        u.z = pack_bf16x2(v[4], v[5]);
        u.w = pack_bf16x2(v[6], v[7]);
        *(uint4*)((uint16_t*)base + idx) = u;
    }
};

template <>
struct Vec<false> {
    static constexpr int N = 4;
    __device__ static void load(const void* base, long long idx, float* out) {
        const float4 f = *(const float4*)((const float*)base + idx);
        out[0] = f.x; out[1] = f.y; out[2] = f.z; out[3] = f.w;
    }
    __device__ static void store(void* base, long long idx, const float* v) {
        *(float4*)((float*)base + idx) = make_float4(v[0], v[1], v[2], v[3]);
    }
};

__device__ __forceinline__ void load_param(const float* p, int off, float* out, int n) {
    for (int i = 0; i < n; i += 4) {
        const float4 f = *(const float4*)(p + off + i);
        out[i] = f.x; out[i + 1] = f.y; out[i + 2] = f.z; out[i + 3] = f.w;
    }
}
}  // namespace

// NCH = 16-byte chunks per lane (d <= 64 * NCH * N).
template <bool BF16, int NCH, bool GATE>
__global__ __launch_bounds__(WAVES * 64) void gln_fwd_kernel(GlnArgs a) {
    using V = Vec<BF16>;
    constexpr int N = V::N;
    const int lane = threadIdx.x & 63;
    const long long wave = (long long)blockIdx.x * WAVES + (threadIdx.x >> 6);
    const long long t0 = wave * TOKENS_PER_WAVE;
    const int d = a.d;
    const int nch = d / N;                       // chunks per row
    const float inv_d = 1.0f / (float)d;
    float gam[NCH][N], bet[NCH][N];
    int gcur = -1;
    for (long long t = t0; t < t0 + TOKENS_PER_WAVE && t < a.T; t++) {
        float z[NCH][N];
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (ch < nch) {
                V::load(a.x, t * a.ld_x + ch * N, z[c]);
                if (GATE) {
                    float uu[N];
                    V::load(a.u, t * a.ld_u + ch * N, uu);
#pragma unroll
                    for (int i = 0; i < N; i++) z[c][i] *= uu[i];
                }
#pragma unroll
                for (int i = 0; i < N; i++) sum += z[c][i];
            }
        }
        const float mean = wave_sum(sum) * inv_d;
        float sq = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            if (lane + 64 * c < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) {
                    const float dz = z[c][i] - mean;
                    sq += dz * dz;
                }
            }
        }
        const float var = wave_sum(sq) * inv_d;
        const float rstd = rsqrtf(var + a.eps);
        const int g = a.gid[t];
        if (g != gcur) {
            gcur = g;
#pragma unroll
            for (int c = 0; c < NCH; c++) {
                const int ch = lane + 64 * c;
                if (ch < nch) {
                    load_param(a.gamma, g * d + ch * N, gam[c], N);
                    load_param(a.beta, g * d + ch * N, bet[c], N);
                }
            }
        }
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (ch < nch) {
                float y[N];
#pragma unroll
                for (int i = 0; i < N; i++) y[i] = gam[c][i] * ((z[c][i] - mean) * rstd) + bet[c][i];
                V::store(a.y, t * a.ld_y + ch * N, y);
            }
        }
        if (lane == 0) {
            if (a.mean) a.mean[t] = mean;
            if (a.rstd) a.rstd[t] = rstd;
        }
    }
}

template <bool BF16, int NCH, bool GATE>
__global__ __launch_bounds__(WAVES * 64) void gln_bwd_kernel(GlnArgs a) {
    using V = Vec<BF16>;
    constexpr int N = V::N;
    const int lane = threadIdx.x & 63;
    const long long wave = (long long)blockIdx.x * WAVES + (threadIdx.x >> 6);
    const long long t0 = wave * TOKENS_PER_WAVE;
    const int d = a.d;
    const int nch = d / N;
    const float inv_d = 1.0f / (float)d;
    float gam[NCH][N], pg[NCH][N], pb[NCH][N];
    int gcur = -1;
    auto flush = [&]() {
        if (gcur < 0) return;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (ch < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) {
                    atomicAdd(&a.dgamma[gcur * d + ch * N + i], pg[c][i]);
                    atomicAdd(&a.dbeta[gcur * d + ch * N + i], pb[c][i]);
                }
            }
        }
    };
    for (long long t = t0; t < t0 + TOKENS_PER_WAVE && t < a.T; t++) {
        const int g = a.gid[t];
        if (g != gcur) {
            flush();
            gcur = g;
#pragma unroll
            for (int c = 0; c < NCH; c++) {
                const int ch = lane + 64 * c;
                if (ch < nch) load_param(a.gamma, g * d + ch * N, gam[c], N);
#pragma unroll
                for (int i = 0; i < N; i++) {
                    pg[c][i] = 0.f;
                    pb[c][i] = 0.f;
                }
            }
        }
        const float mean = a.mean[t], rstd = a.rstd[t];
        float xh[NCH][N], gy[NCH][N];
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (ch < nch) {
                float xx[N], dy[N];
                V::load(a.x, t * a.ld_x + ch * N, xx);
                V::load(a.dy, t * a.ld_y + ch * N, dy);
                if (GATE) {
                    float uu[N];
                    V::load(a.u, t * a.ld_u + ch * N, uu);
#pragma unroll
                    for (int i = 0; i < N; i++) xx[i] *= uu[i];
                }
#pragma unroll
                for (int i = 0; i < N; i++) {
                    xh[c][i] = (xx[i] - mean) * rstd;
                    gy[c][i] = dy[i];
                    const float gg = dy[i] * gam[c][i];
                    s1 += gg;
                    s2 += gg * xh[c][i];
                    pg[c][i] += dy[i] * xh[c][i];
                    pb[c][i] += dy[i];
                }
            }
        }
        const float m1 = wave_sum(s1) * inv_d;
        const float m2 = wave_sum(s2) * inv_d;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (ch < nch) {
                float dz[N];
#pragma unroll
                for (int i = 0; i < N; i++) dz[i] = rstd * (gy[c][i] * gam[c][i] - m1 - xh[c][i] * m2);
                if (GATE) {
                    float xx[N], uu[N], dx[N], du[N];
                    V::load(a.x, t * a.ld_x + ch * N, xx);
                    V::load(a.u, t * a.ld_u + ch * N, uu);
#pragma unroll
                    for (int i = 0; i < N; i++) {
                        dx[i] = dz[i] * uu[i];
                        du[i] = dz[i] * xx[i];
                    }
                    V::store(a.dx, t * a.ld_x + ch * N, dx);
                    V::store(a.du, t * a.ld_u + ch * N, du);
                } else {
                    V::store(a.dx, t * a.ld_x + ch * N, dz);
                }
            }
        }
    }
    flush();
}

template <bool BF16, int NCH>
static hipError_t gln_launch(const GlnArgs& a, bool bwd, hipStream_t s) {
    const long long waves = (a.T + TOKENS_PER_WAVE - 1) / TOKENS_PER_WAVE;
    const int blocks = (int)((waves + WAVES - 1) / WAVES);
    const bool gate = a.u != nullptr;
    if (!bwd) {
        if (gate) gln_fwd_kernel<BF16, NCH, true><<<blocks, WAVES * 64, 0, s>>>(a);
        else gln_fwd_kernel<BF16, NCH, false><<<blocks, WAVES * 64, 0, s>>>(a);
    } else {
        if (gate) gln_bwd_kernel<BF16, NCH, true><<<blocks, WAVES * 64, 0, s>>>(a);
        else gln_bwd_kernel<BF16, NCH, false><<<blocks, WAVES * 64, 0, s>>>(a);
    }
    return hipGetLastError();
}

template <bool BF16>
static hipError_t gln_dispatch(const GlnArgs& a, bool bwd, hipStream_t s) {
    const int n = Vec<BF16>::N;
    const int chunks_per_lane = (a.d / n + 63) / 64;
    if (chunks_per_lane <= 1) return gln_launch<BF16, 1>(a, bwd, s);
    if (chunks_per_lane <= 2) return gln_launch<BF16, 2>(a, bwd, s);
    if (chunks_per_lane <= 4) return gln_launch<BF16, 4>(a, bwd, s);
    if (chunks_per_lane <= 8) return gln_launch<BF16, 8>(a, bwd, s);
    return hipErrorInvalidValue;
}

hipError_t launch_gln_fwd(const GlnArgs& a, bool bf16, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    return bf16 ? gln_dispatch<true>(a, false, s) : gln_dispatch<false>(a, false, s);
}

hipError_t launch_gln_bwd(const GlnArgs& a, bool bf16, hipStream_t s) {
    hipError_t e = launch_fill_f32(a.dgamma, (long long)a.G * a.d, 0.f, s);
    if (e != hipSuccess) return e;
    e = launch_fill_f32(a.dbeta, (long long)a.G * a.d, 0.f, s);
    if (e != hipSuccess || a.T == 0) return e;
    return bf16 ? gln_dispatch<true>(a, true, s) : gln_dispatch<false>(a, true, s);
}

}  // namespace mtgr
