// Debug-time check of the device-resident preconditions of a jagged batch (offsets, segment
// codes, group ids).  Not on the hot path: the entry point that launches it synchronises.
#include "mtgr_internal.h"

namespace mtgr {

namespace {

// first[c] = smallest index at which condition c fails (~0 = none):
//   0 offsets[0] != 0, 1 offsets[b+1] < offsets[b], 2 offsets[B] != T,
//   3 offsets[b+1] - offsets[b] > max_seqlen, 4 seg[t] outside 0..3, 5 group_ids[t] outside 0..G-1.
__global__ void validate_init_kernel(unsigned long long* first) {
    if (threadIdx.x < VALIDATE_CONDITIONS) first[threadIdx.x] = ~0ull;
}

__global__ void validate_kernel(const int* offsets, int num_users, long long total, int max_seqlen,
                                const int8_t* seg, const int8_t* group_ids, int groups,
                                unsigned long long* first) {
    const long long i0 = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    const long long stride = (long long)gridDim.x * blockDim.x;
    for (long long b = i0; b <= num_users; b += stride) {
        const long long o = offsets[b];
        if (b == 0 && o != 0) atomicMin(&first[0], 0ull);
        if (b < num_users) {
            const long long o1 = offsets[b + 1];
            if (o1 < o) atomicMin(&first[1], (unsigned long long)b);
            else if (o1 - o > max_seqlen) atomicMin(&first[3], (unsigned long long)b);
        } else if (o != total) {
            atomicMin(&first[2], (unsigned long long)b);
        }
    }
    for (long long t = i0; t < total; t += stride) {
        const int s = seg[t];
        if (s < 0 || s > 3) atomicMin(&first[4], (unsigned long long)t);
        if (group_ids != nullptr) {
            const int g = group_ids[t];
            if (g < 0 || g >= groups) atomicMin(&first[5], (unsigned long long)t);
        }
    }
}

}  // namespace

hipError_t launch_validate(const int* offsets, int num_users, long long total, int max_seqlen,
                           const int8_t* seg, const int8_t* group_ids, int groups,
                           unsigned long long* first, hipStream_t s) {
    validate_init_kernel<<<1, 64, 0, s>>>(first);
    const long long n = total > num_users + 1 ? total : (long long)num_users + 1;
    const long long blocks = (n + 255) / 256;
    validate_kernel<<<(int)(blocks < 2048 ? blocks : 2048), 256, 0, s>>>(offsets, num_users, total, max_seqlen,
                                                                         seg, group_ids, groups, first);
    return hipGetLastError();
}

}  // namespace mtgr
