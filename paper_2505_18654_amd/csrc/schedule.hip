// Tile metadata and work scheduling for the jagged attention kernels.
//
// 1. tile_summaries: for every user and every 64-token tile of that user (tiles start at
//    the user's first token), the segment flags and the time range that decide whether a
//    (query tile, key tile) pair is fully visible, partially visible or fully masked under
//    the dynamic mask of Sec. 4.2.  Fully masked pairs are skipped by the attention kernels.
//    It also writes each token's mask code (static / real-time / dynamic / valid bits), which
//    the attention kernels copy into LDS next to the tile's timestamps.
// 2. build_schedule: one work item per (user, head, tile of `bm` rows).  Users are sorted
//    longest first (jagged lengths are long-tailed, Sec. 5 "Load balance"), (user, head)
//    groups are dealt round-robin to the 8 XCDs so that all tiles of one group run on one
//    XCD and share its L2, and each XCD's queue is laid out at slots x, x + 8, x + 16, ...
//    because the hardware dispatches workgroup i to XCD i mod 8.
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {

__global__ __launch_bounds__(256) void tile_summaries_kernel(const int* __restrict__ offsets,
                                                             const int8_t* __restrict__ seg,
                                                             const int* __restrict__ ts, int ntile,
                                                             int4* __restrict__ summ,
                                                             int* __restrict__ tok_code) {
    const int b = blockIdx.y;
    const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int ob = offsets[b];
    const int nb = offsets[b + 1] - ob;
    if (t >= ntile) return;
    const int rel = t * SUMMARY_TILE + lane;
    const bool valid = rel < nb;
    int sg = -1, tv = 0;
    if (valid) {
        sg = seg[ob + rel];
        tv = ts[ob + rel];
        tok_code[ob + rel] = token_code(sg);
    }
    const bool is_static = valid && sg <= SEG_HIST;
    const bool is_rt = valid && sg == SEG_RT;
    const bool is_dyn = valid && sg >= SEG_RT;
    const unsigned long long st = __ballot(is_static);
    int flags = 0;
    if (st) flags |= TS_ANY_STATIC;
    if (st == ~0ull) flags |= TS_ALL_STATIC;
    if (__ballot(is_rt)) flags |= TS_ANY_RT;
    if (__ballot(is_dyn)) flags |= TS_ANY_DYN;
    if (__ballot(valid && sg == SEG_CAND)) flags |= TS_ANY_CAND;
    const int mn = wave_min(is_rt ? tv : 0x7fffffff);
    const int mx = wave_max(is_dyn ? tv : (int)0x80000000);
    if (lane == 0) summ[(long long)b * ntile + t] = make_int4(flags, mn, mx, 0);
}

// Exclusive prefix sum over the 1024 threads of the block; returns the block total in *total.
__device__ int block_exclusive_scan(int v, int* scratch, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    if (lane == 63) scratch[w] = incl;
    __syncthreads();
    if (threadIdx.x == 0) {
        int run = 0;
        for (int i = 0; i < 16; i++) {
            int x = scratch[i];
            scratch[i] = run;
            run += x;
        }
        scratch[16] = run;
    }
    __syncthreads();
    const int res = scratch[w] + incl - v;
    *total = scratch[16];
    __syncthreads();
    return res;
}

__global__ __launch_bounds__(1024) void build_schedule_kernel(const int* __restrict__ offsets,
                                                              int num_users, int heads, int bm,
                                                              int2* __restrict__ items, int slots,
                                                              int* __restrict__ sorted_users) {
    __shared__ int hist[SCHED_BUCKETS];
    __shared__ int scratch[32];
    const int tid = threadIdx.x;
    for (int i = tid; i < slots; i += 1024) items[i] = make_int2(-1, 0);
    for (int i = tid; i < SCHED_BUCKETS; i += 1024) hist[i] = 0;
    __syncthreads();
    for (int b = tid; b < num_users; b += 1024) {
        const int n = offsets[b + 1] - offsets[b];
        const int key = min((n + SUMMARY_TILE - 1) / SUMMARY_TILE, SCHED_BUCKETS - 1);
        atomicAdd(&hist[key], 1);
    }
    __syncthreads();
    // Descending bucket order: position of bucket k = number of users in buckets > k.
    {
        constexpr int PER = SCHED_BUCKETS / 1024;
        int local[PER];
        int sum = 0;
#pragma unroll
        for (int i = 0; i < PER; i++) {
            local[i] = hist[SCHED_BUCKETS - 1 - (tid * PER + i)];
            sum += local[i];
        }
        int total;
        int run = block_exclusive_scan(sum, scratch, &total);
#pragma unroll
        for (int i = 0; i < PER; i++) {
            hist[SCHED_BUCKETS - 1 - (tid * PER + i)] = run;
            run += local[i];
        }
    }
    __syncthreads();
    for (int b = tid; b < num_users; b += 1024) {
        const int n = offsets[b + 1] - offsets[b];
        const int key = min((n + SUMMARY_TILE - 1) / SUMMARY_TILE, SCHED_BUCKETS - 1);
        const int rank = atomicAdd(&hist[key], 1);
        sorted_users[rank] = b;
    }
    __threadfence_block();
    __syncthreads();
    // Group g = rank * heads + h goes to XCD g % 8 at queue position
    // sum of tile counts of the earlier groups with the same residue.  One pass over 1024
    // groups at a time: a scan with stride 8 inside each wave, then per residue over the
    // 16 waves, with a running carry per residue.
    __shared__ int wsum[16][XCDS];
    __shared__ int carry[XCDS];
    if (tid < XCDS) carry[tid] = 0;
    const int lane = tid & 63, wv = tid >> 6, x = tid % XCDS;
    const long long groups = (long long)num_users * heads;
    for (long long base = 0; base < groups; base += 1024) {
        const long long g = base + tid;
        int nq = 0, b = -1, h = 0;
        if (g < groups) {
            b = sorted_users[g / heads];
            h = (int)(g % heads);
            const int n = offsets[b + 1] - offsets[b];
            nq = (n + bm - 1) / bm;
        }
        int incl = nq;
#pragma unroll
        for (int off = XCDS; off < 64; off <<= 1) {
            const int o = __shfl_up(incl, off, 64);
            if (lane >= off) incl += o;
        }
        if (lane >= 64 - XCDS) wsum[wv][x] = incl;   // this wave's total of residue x
        __syncthreads();
        if (tid < XCDS) {
            int run = carry[tid];
            for (int i = 0; i < 16; i++) {
                const int t = wsum[i][tid];
                wsum[i][tid] = run;
                run += t;
            }
            carry[tid] = run;
        }
        __syncthreads();
        const int pos = wsum[wv][x] + incl - nq;
        for (int t = 0; t < nq; t++) {
            const long long slot = (long long)(pos + t) * XCDS + x;
            if (slot < slots) items[slot] = make_int2(b, (t << 8) | h);
        }
        __syncthreads();   // wsum is rewritten by the next pass
    }
}

// First stored-dS block of every user: exclusive prefix sum of H * ceil(n_b / 64)^2.
__global__ __launch_bounds__(1024) void ds_offsets_kernel(const int* __restrict__ offsets, int num_users,
                                                          int heads, long long* __restrict__ ds_off) {
    __shared__ long long scratch[17];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    long long carry = 0;
    for (int base = 0; base < num_users; base += 1024) {
        const int b = base + tid;
        long long v = 0;
        if (b < num_users) {
            const long long nt = (offsets[b + 1] - offsets[b] + 63) / 64;
            v = (long long)heads * nt * nt;
        }
        long long incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const long long o = __shfl_up(incl, off, 64);
            if (lane >= off) incl += o;
        }
        if (lane == 63) scratch[w] = incl;
        __syncthreads();
        if (tid == 0) {
            long long run = 0;
            for (int i = 0; i < 16; i++) {
                const long long x = scratch[i];
                scratch[i] = run;
                run += x;
            }
            scratch[16] = run;
        }
        __syncthreads();
        if (b < num_users) ds_off[b] = carry + scratch[w] + incl - v;
        carry += scratch[16];
        __syncthreads();
    }
    if (tid == 0) ds_off[num_users] = carry;
}

hipError_t launch_ds_offsets(const int* offsets, int num_users, int heads, long long* ds_off,
                             hipStream_t s) {
    ds_offsets_kernel<<<1, 1024, 0, s>>>(offsets, num_users, heads, ds_off);
    return hipGetLastError();
}

__global__ void fill_f32_kernel(float* __restrict__ p, long long n, float value) {
    for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (long long)gridDim.x * blockDim.x)
        p[i] = value;
}

long long schedule_slots(long long total_tokens, int num_users, int max_seqlen, int heads, int bm) {
    // Items <= heads * sum_b ceil(n_b / bm) <= heads * (T / bm + B).  Groups are sorted by
    // tile count, so queue x holds at most max_b ceil(n_b / bm) + items / 8 entries.
    const long long items = (long long)heads * (total_tokens / bm + num_users);
    const long long per_xcd = (max_seqlen + bm - 1) / bm + (items + XCDS - 1) / XCDS;
    return per_xcd * XCDS;
}

hipError_t launch_tile_summaries(const int* offsets, const int8_t* seg, const int* ts, int num_users,
                                 int ntile, int4* summ, int* tok_code, hipStream_t s) {
    if (num_users == 0 || ntile == 0) return hipSuccess;
    dim3 grid((ntile + 3) / 4, num_users);
    tile_summaries_kernel<<<grid, 256, 0, s>>>(offsets, seg, ts, ntile, summ, tok_code);
    return hipGetLastError();
}

hipError_t launch_build_schedule(const int* offsets, int num_users, int heads, int bm, int2* items,
                                 int slots, int* sorted_users, hipStream_t s) {
    build_schedule_kernel<<<1, 1024, 0, s>>>(offsets, num_users, heads, bm, items, slots,
                                             sorted_users);
    return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, long long n, float value, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const long long blocks = (n + 255) / 256;
    fill_f32_kernel<<<(int)(blocks < 1024 ? blocks : 1024), 256, 0, s>>>(p, n, value);
    return hipGetLastError();
}

}  // namespace mtgr
