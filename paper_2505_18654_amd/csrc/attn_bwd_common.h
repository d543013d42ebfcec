// Shared pieces of the attention backward kernels, which live in separate translation units
// (attn_bwd_dq.hip, attn_bwd_dkdv.hip, attn_bwd_dqds.hip): compiled together, the register
// allocation of one kernel changed with the others (the dK/dV kernel spilled about twice as
// much), so each kernel family is compiled on its own and instantiated explicitly.
#pragma once

#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {
namespace bwd {
constexpr int BM = 128;   // rows (queries or keys) per workgroup
constexpr int BN = 64;    // columns per inner tile
__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *(const uint4*)p; }

__device__ __forceinline__ void zero(floatx16& x) {
#pragma unroll
    for (int r = 0; r < 16; r++) x[r] = 0.f;
}

// drab histogram of one workgroup in LDS.  Log-time buckets put most (query, key) pairs of a
// tile into a handful of buckets, so one histogram would serialise the 64 lanes of each LDS
// atomic.  Lane l adds into copy l % 32 (at most two lanes of an instruction share a copy),
// and the copies are HIST_STRIDE = 65 words apart so that one bucket of different copies sits
// in different banks.  8.3 KB.
constexpr int HIST_COPIES = 32;
constexpr int HIST_STRIDE = MTGR_RAB_LDS + 1;
constexpr int HIST_WORDS = HIST_COPIES * HIST_STRIDE;
__device__ __forceinline__ void hist_zero(float* hist, int tid) {
    for (int i = tid; i < HIST_WORDS; i += 256) hist[i] = 0.f;
}
__device__ __forceinline__ void hist_add(float* hist, int lane, int bucket, float v) {
    atomicAdd(&hist[(lane & (HIST_COPIES - 1)) * HIST_STRIDE + bucket], v);
}
// Per-lane run of equal buckets: consecutive scores of a lane (queries of one key, or keys of
// one query, in token order) mostly fall into the same log-time bucket, so each lane sums its
// run in a register and touches the LDS histogram only when the bucket changes (and once at
// the end).  LDS float atomics are slow on this chip; this makes them rare.
struct HistRun {
    int bucket = 0;
    float sum = 0.f;
    __device__ __forceinline__ void add(float* hist, int lane, int b, float v) {
        if (v != 0.f) {
            if (b != bucket) {
                if (sum != 0.f) hist_add(hist, lane, bucket, sum);
                bucket = b;
                sum = 0.f;
            }
            sum += v;
        }
    }
    __device__ __forceinline__ void flush(float* hist, int lane) {
        if (sum != 0.f) hist_add(hist, lane, bucket, sum);
        sum = 0.f;
    }
};
__device__ __forceinline__ float hist_total(const float* hist, int bucket) {
    float s = 0.f;
#pragma unroll 8
    for (int c = 0; c < HIST_COPIES; c++) s += hist[c * HIST_STRIDE + bucket];
    return s;
}
}  // namespace bwd

template <int DH, bool RAB>
__global__ void attn_bwd_dq_bf16_kernel(AttnArgs a);
template <int DH, bool RAB, bool STORE>
__global__ void attn_bwd_dkdv_bf16_kernel(AttnArgs a);
template <int DH>
__global__ void attn_bwd_dq_ds_bf16_kernel(AttnArgs a);

}  // namespace mtgr
