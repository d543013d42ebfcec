// Gate + Group-LayerNorm (Eq. 6 up to the MLP: y = GroupLN(x (*) u)), forward and backward.
//
// Memory-bound: one wave per token row, 16-byte vector loads, wave reductions through
// cross-lane shuffles, two-pass variance on values held in registers.  Each wave walks a
// run of consecutive tokens; since a user's tokens come segment by segment ([U|S|R|I]) and
// the groups are the segments, gamma/beta rows stay in registers across a run and are only
// re-read when the group changes.
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

namespace {
constexpr int WAVES = 4;            // forward: waves per workgroup
constexpr int TOKENS_PER_WAVE = 4;   // forward: consecutive tokens per wave
constexpr int BWD_WAVES = 8;         // backward: waves per workgroup

template <bool BF16>
struct Vec;   // 16-byte chunk of the storage type

template <>
struct Vec<true> {
    static constexpr int N = 8;
    __device__ static uint4 raw(const void* base, long long idx) {
        typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = __builtin_nontemporal_load((const u32x4*)((const uint16_t*)base + idx));
        return make_uint4(v.x, v.y, v.z, v.w);
    }
    __device__ static void unpack(const uint4 u, float* out) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
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
        // streaming store: the outputs are not read again by this kernel (measured: the forward
        // 0.082 -> 0.069 ms on the mtgr_large batch)
        typedef unsigned int u32x4s __attribute__((ext_vector_type(4)));
        const u32x4s w = {u.x, u.y, u.z, u.w};
        __builtin_nontemporal_store(w, (u32x4s*)((uint16_t*)base + idx));
    }
};

template <>
struct Vec<false> {
    static constexpr int N = 4;
    __device__ static uint4 raw(const void* base, long long idx) {
        typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
        const u32x4 v = __builtin_nontemporal_load((const u32x4*)((const float*)base + idx));
        return make_uint4(v.x, v.y, v.z, v.w);
    }
    __device__ static void unpack(const uint4 u, float* out) {
        out[0] = __uint_as_float(u.x); out[1] = __uint_as_float(u.y);
        out[2] = __uint_as_float(u.z); out[3] = __uint_as_float(u.w);
    }
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
// FULL: every lane owns exactly NCH chunks (d = 64 NCH N), so no chunk guard is needed.  Otherwise
// a lane past the row's last chunk loads that last chunk again and ignores it: a guard would put
// a branch around the loads, and the counters of loads in flight are waited to zero at the join,
// which serialises the prefetch (the serving workload's d = 768 ran its forward at 5.1 TB/s).
template <bool BF16, int NCH, bool GATE, bool FULL>
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
    // raw rows of the next token, loaded while the current one is normalised
    float xr[NCH][N] = {}, ur[NCH][N] = {};
    auto load_rows = [&](long long t) {
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = FULL ? lane + 64 * c : min(lane + 64 * c, nch - 1);
            V::load(a.x, t * a.ld_x + ch * N, xr[c]);
            if (GATE) V::load(a.u, t * a.ld_u + ch * N, ur[c]);
        }
    };
    const long long t_end = min(t0 + TOKENS_PER_WAVE, a.T);
    if (t0 < t_end) load_rows(t0);
    for (long long t = t0; t < t_end; t++) {
        float z[NCH][N];
        float sum = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
#pragma unroll
            for (int i = 0; i < N; i++) z[c][i] = GATE ? xr[c][i] * ur[c][i] : xr[c][i];
            if (FULL || lane + 64 * c < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) sum += z[c][i];
            }
        }
        const int g = a.gid[t];
        if (t + 1 < t_end) load_rows(t + 1);
        const float mean = wave_sum(sum) * inv_d;
        float sq = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            if (FULL || lane + 64 * c < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) {
                    const float dz = z[c][i] - mean;
                    sq += dz * dz;
                }
            }
        }
        const float var = wave_sum(sq) * inv_d;
        const float rstd = rsqrtf(var + a.eps);
        if (g != gcur) {
            gcur = g;
#pragma unroll
            for (int c = 0; c < NCH; c++) {
                const int ch = lane + 64 * c;
                if (FULL || ch < nch) {
                    load_param(a.gamma, g * d + ch * N, gam[c], N);
                    load_param(a.beta, g * d + ch * N, bet[c], N);
                }
            }
        }
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (FULL || ch < nch) {
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

// Backward.  Workgroup = BWD_WAVES waves over a contiguous chunk of tokens, each wave a
// contiguous run of `tpw` tokens (the next token's rows are loaded while the current one is
// processed).  dgamma/dbeta: each wave keeps the partial sums of its current group in
// registers and adds them into a per-workgroup accumulator [2][G][d] when the group changes
// (LDS atomics among the workgroup's waves, or the workgroup's own workspace slot when
// 2 G d floats do not fit in LDS); the accumulator is then stored to the workgroup's slot
// and gln_param_reduce_kernel sums the slots in a fixed order.  No device-wide atomics.
// Rows of more than 2 chunks per lane (d > 1024 bf16, > 512 fp32) need more than the 256
// registers of two waves per SIMD: there the workgroup runs half as many waves, each taking the
// token runs of two.
template <int NCH>
constexpr int bwd_real_waves() { return NCH >= 4 ? BWD_WAVES / 2 : BWD_WAVES; }

template <bool BF16, int NCH, bool GATE, bool LDS_ACC, bool FULL>
__global__ __launch_bounds__(bwd_real_waves<NCH>() * 64) void gln_bwd_kernel(GlnArgs a, float* __restrict__ part,
                                                                              int tpw) {
    using V = Vec<BF16>;
    constexpr int N = V::N;
    constexpr int RW = bwd_real_waves<NCH>(), WPW = BWD_WAVES / RW;
    extern __shared__ float sAcc[];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int d = a.d;
    const int nch = d / N;
    const int accn = 2 * a.G * d;
    float* slot = part + (long long)blockIdx.x * accn;
    float* acc = LDS_ACC ? sAcc : slot;
    for (int i = threadIdx.x; i < accn; i += RW * 64) acc[i] = 0.f;
    // With the LDS accumulator, gamma [G][d] is staged in LDS behind it, so that reloading a
    // wave's gamma rows on a group change is an LDS read: a global load there would be counted
    // with the rows in flight, and the wait for it would drain the prefetch.
    const float* gsrc = a.gamma;
    if constexpr (LDS_ACC) {
        float* sGam = sAcc + accn;
        for (int i = threadIdx.x; i < a.G * d; i += RW * 64) sGam[i] = a.gamma[i];
        gsrc = sGam;
    }
    __syncthreads();
    const long long t0 = ((long long)blockIdx.x * BWD_WAVES + (long long)w * WPW) * tpw;
    const long long t1 = min(t0 + (long long)WPW * tpw, a.T);
    const float inv_d = 1.0f / (float)d;
    float gam[NCH][N], pg[NCH][N], pb[NCH][N];
    int gcur = -1;
    auto flush = [&]() {
        if (gcur < 0) return;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (FULL || ch < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) {
                    atomicAdd(&acc[gcur * d + ch * N + i], pg[c][i]);
                    atomicAdd(&acc[(a.G + gcur) * d + ch * N + i], pb[c][i]);
                }
            }
        }
    };
    // Rows and statistics of the tokens ahead, kept as the raw 16-byte chunks as loaded.  Up to
    // two chunks per lane the next two tokens are in flight while the current one is
    // processed (three rows are read per token, and one token per wave in flight leaves HBM
    // idle), the next one up to four chunks, none at eight (no registers left).
    struct Rows {
        uint4 x[NCH], y[NCH], u[NCH];
        int g;
        float m, r;
    };
    auto fetch = [&](long long t, Rows& r) {
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            if constexpr (FULL || NCH <= 4) {
                // past the row's last chunk: that chunk again, ignored (no branch around the loads,
                // which would wait for the rows in flight); at 8 chunks nothing is prefetched
                const int ch = FULL ? lane + 64 * c : min(lane + 64 * c, nch - 1);
                r.x[c] = V::raw(a.x, t * a.ld_x + ch * N);
                r.y[c] = V::raw(a.dy, t * a.ld_y + ch * N);
                if (GATE) r.u[c] = V::raw(a.u, t * a.ld_u + ch * N);
            } else {
                const int ch = lane + 64 * c;
                if (ch < nch) {
                    r.x[c] = V::raw(a.x, t * a.ld_x + ch * N);
                    r.y[c] = V::raw(a.dy, t * a.ld_y + ch * N);
                    if (GATE) r.u[c] = V::raw(a.u, t * a.ld_u + ch * N);
                }
            }
        }
        r.g = a.gid[t];
        r.m = a.mean[t];
        r.r = a.rstd[t];
    };
    // PFD + 1 row buffers used round robin, the loop unrolled by PFD + 1 so that every buffer
    // index is a compile-time constant: no register of a load in flight is ever copied (a copy
    // would wait for that load and serialise the prefetch).  Token t + PFD is requested into the
    // buffer that token t - 1 used, before token t is processed.
    constexpr int PFD = NCH <= 2 ? 2 : NCH <= 4 ? 1 : 0;
    constexpr int NB = PFD + 1;
    auto process = [&](long long t, const Rows& cur) {
        float xx[NCH][N], uu[NCH][N], dy[NCH][N];
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            V::unpack(cur.x[c], xx[c]);
            V::unpack(cur.y[c], dy[c]);
#pragma unroll
            for (int i = 0; i < N; i++) uu[c][i] = 1.f;
            if (GATE) V::unpack(cur.u[c], uu[c]);
        }
        const int g = cur.g;
        const float mean = cur.m, rstd = cur.r;
        if (g != gcur) {
            flush();
            gcur = g;
#pragma unroll
            for (int c = 0; c < NCH; c++) {
                const int ch = lane + 64 * c;
                if (FULL || ch < nch) load_param(gsrc, g * d + ch * N, gam[c], N);
#pragma unroll
                for (int i = 0; i < N; i++) {
                    pg[c][i] = 0.f;
                    pb[c][i] = 0.f;
                }
            }
        }
        float xh[NCH][N];
        float s1 = 0.f, s2 = 0.f;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            if (FULL || lane + 64 * c < nch) {
#pragma unroll
                for (int i = 0; i < N; i++) {
                    xh[c][i] = (xx[c][i] * uu[c][i] - mean) * rstd;
                    const float gg = dy[c][i] * gam[c][i];
                    s1 += gg;
                    s2 += gg * xh[c][i];
                    pg[c][i] += dy[c][i] * xh[c][i];
                    pb[c][i] += dy[c][i];
                }
            }
        }
        const float m1 = wave_sum(s1) * inv_d;
        const float m2 = wave_sum(s2) * inv_d;
#pragma unroll
        for (int c = 0; c < NCH; c++) {
            const int ch = lane + 64 * c;
            if (FULL || ch < nch) {
                float dz[N];
#pragma unroll
                for (int i = 0; i < N; i++) dz[i] = rstd * (dy[c][i] * gam[c][i] - m1 - xh[c][i] * m2);
                if (GATE) {
                    float dx[N], du[N];
#pragma unroll
                    for (int i = 0; i < N; i++) {
                        dx[i] = dz[i] * uu[c][i];
                        du[i] = dz[i] * xx[c][i];
                    }
                    V::store(a.dx, t * a.ld_x + ch * N, dx);
                    V::store(a.du, t * a.ld_u + ch * N, du);
                } else {
                    V::store(a.dx, t * a.ld_x + ch * N, dz);
                }
            }
        }
    };
    if constexpr (PFD == 0) {
        for (long long t = t0; t < t1; t++) {
            Rows cur = {};
            fetch(t, cur);
            process(t, cur);
        }
    } else {
        Rows buf[NB] = {};
#pragma unroll
        for (int k = 0; k < PFD; k++) fetch(min(t0 + k, t1 - 1), buf[k]);
        for (long long tb = t0; tb < t1; tb += NB) {
#pragma unroll
            for (int j = 0; j < NB; j++) {
                const long long t = tb + j;
                if (t >= t1) break;
                // unconditional (near the end the last token is fetched again), so that every
                // iteration issues the same loads and the wait counts stay exact
                fetch(min(t + PFD, t1 - 1), buf[(j + PFD) % NB]);
                process(t, buf[j]);
            }
        }
    }
    flush();
    __syncthreads();
    if (LDS_ACC)
        for (int i = threadIdx.x; i < accn; i += RW * 64) slot[i] = sAcc[i];
}

// dgamma/dbeta = sum over workgroup slots (fixed order).  Block = 32 columns x 8 slot sets
// (slot s goes to set s % 8); each thread keeps four partial sums so that four loads are in
// flight, then the partials and the sets are added in a fixed order (deterministic).
constexpr int RED_COLS = 32, RED_SETS = 8;
__global__ __launch_bounds__(256) void gln_param_reduce_kernel(const float* __restrict__ part,
                                                               int nslots, int accn, int gd,
                                                               float* __restrict__ dgamma,
                                                               float* __restrict__ dbeta) {
    __shared__ float sRed[RED_SETS][RED_COLS];
    const int c = threadIdx.x % RED_COLS, r = threadIdx.x / RED_COLS;
    const int e = blockIdx.x * RED_COLS + c;
    float s4[4] = {0.f, 0.f, 0.f, 0.f};
    if (e < accn) {
        int s = r;
#pragma unroll 1
        for (; s + 3 * RED_SETS < nslots; s += 4 * RED_SETS) {
#pragma unroll
            for (int k = 0; k < 4; k++) s4[k] += part[(long long)(s + k * RED_SETS) * accn + e];
        }
#pragma unroll
        for (int k = 0; k < 4; k++)
            if (s + k * RED_SETS < nslots) s4[k] += part[(long long)(s + k * RED_SETS) * accn + e];
    }
    sRed[r][c] = (s4[0] + s4[1]) + (s4[2] + s4[3]);
    __syncthreads();
    if (r == 0 && e < accn) {
        float tot = 0.f;
#pragma unroll
        for (int k = 0; k < RED_SETS; k++) tot += sRed[k][c];
        if (e < gd) dgamma[e] = tot;
        else dbeta[e - gd] = tot;
    }
}

template <bool BF16, int NCH>
static hipError_t gln_launch(const GlnArgs& a, bool bwd, hipStream_t s) {
    const bool gate = a.u != nullptr;
    const bool full = a.d == 64 * NCH * Vec<BF16>::N;
    if (!bwd) {
        const long long waves = (a.T + TOKENS_PER_WAVE - 1) / TOKENS_PER_WAVE;
        const int blocks = (int)((waves + WAVES - 1) / WAVES);
        if (full) {
            if (gate) gln_fwd_kernel<BF16, NCH, true, true><<<blocks, WAVES * 64, 0, s>>>(a);
            else gln_fwd_kernel<BF16, NCH, false, true><<<blocks, WAVES * 64, 0, s>>>(a);
        } else {
            if (gate) gln_fwd_kernel<BF16, NCH, true, false><<<blocks, WAVES * 64, 0, s>>>(a);
            else gln_fwd_kernel<BF16, NCH, false, false><<<blocks, WAVES * 64, 0, s>>>(a);
        }
        return hipGetLastError();
    }
    int nslots, tpw;
    gln_bwd_partition(a.T, &nslots, &tpw);
    const int accn = 2 * a.G * a.d;
    const bool lds = accn * (int)sizeof(float) <= GLN_LDS_ACC_BYTES;
    const size_t shm = lds ? (accn + a.G * a.d) * sizeof(float) : 0;   // accumulator, then gamma
    float* part = a.workspace;
    constexpr int threads = bwd_real_waves<NCH>() * 64;
    if (lds && full) {
        if (gate) gln_bwd_kernel<BF16, NCH, true, true, true><<<nslots, threads, shm, s>>>(a, part, tpw);
        else gln_bwd_kernel<BF16, NCH, false, true, true><<<nslots, threads, shm, s>>>(a, part, tpw);
    } else if (lds) {
        if (gate) gln_bwd_kernel<BF16, NCH, true, true, false><<<nslots, threads, shm, s>>>(a, part, tpw);
        else gln_bwd_kernel<BF16, NCH, false, true, false><<<nslots, threads, shm, s>>>(a, part, tpw);
    } else {
        if (gate) gln_bwd_kernel<BF16, NCH, true, false, false><<<nslots, threads, 0, s>>>(a, part, tpw);
        else gln_bwd_kernel<BF16, NCH, false, false, false><<<nslots, threads, 0, s>>>(a, part, tpw);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    gln_param_reduce_kernel<<<(accn + RED_COLS - 1) / RED_COLS, 256, 0, s>>>(part, nslots, accn, a.G * a.d, a.dgamma,
                                                            a.dbeta);
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

void gln_bwd_partition(long long T, int* nslots, int* tpw) {
    const long long per_wave = (T + (long long)GLN_BWD_SLOTS * BWD_WAVES - 1) / ((long long)GLN_BWD_SLOTS * BWD_WAVES);
    *tpw = (int)(per_wave < 1 ? 1 : per_wave);
    *nslots = (int)((T + (long long)*tpw * BWD_WAVES - 1) / ((long long)*tpw * BWD_WAVES));
    if (*nslots < 1) *nslots = 1;
}

size_t gln_bwd_workspace_bytes(long long T, int d, int G) {
    int nslots, tpw;
    gln_bwd_partition(T, &nslots, &tpw);
    return (size_t)nslots * 2 * G * d * sizeof(float);
}

hipError_t launch_gln_fwd(const GlnArgs& a, bool bf16, hipStream_t s) {
    if (a.T == 0) return hipSuccess;
    return bf16 ? gln_dispatch<true>(a, false, s) : gln_dispatch<false>(a, false, s);
}

hipError_t launch_gln_bwd(const GlnArgs& a, bool bf16, hipStream_t s) {
    if (a.T == 0) {
        hipError_t e = launch_fill_f32(a.dgamma, (long long)a.G * a.d, 0.f, s);
        if (e != hipSuccess) return e;
        return launch_fill_f32(a.dbeta, (long long)a.G * a.d, 0.f, s);
    }
    return bf16 ? gln_dispatch<true>(a, true, s) : gln_dispatch<false>(a, true, s);
}

}  // namespace mtgr
