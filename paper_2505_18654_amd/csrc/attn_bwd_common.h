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
}  // namespace bwd

template <int DH, bool RAB>
__global__ void attn_bwd_dq_bf16_kernel(AttnArgs a);
template <int DH, bool RAB, bool STORE>
__global__ void attn_bwd_dkdv_bf16_kernel(AttnArgs a);
template <int DH>
__global__ void attn_bwd_dq_ds_bf16_kernel(AttnArgs a);

}  // namespace mtgr
