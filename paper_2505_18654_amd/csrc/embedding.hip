// Dynamic embedding table of MTGR's training framework (Sec. 5, "Dynamic Hash Table" and
// "Embedding Lookup"): a compact key store (open addressing, linear probing over 64-bit IDs)
// decoupled from the value store (embedding rows plus an occurrence counter and the time of
// the last lookup per row), a hash-set de-duplication of each batch, lookup with insertion,
// the gather of a batch's rows, a sparse SGD step, eviction by time and a rebuild of the key
// store at another capacity.
//
// Every kernel is a bounded grid-stride loop; every probe loop is bounded by the capacity it
// walks.  Concurrency inside one call: distinct IDs race only for free slots (atomicCAS on the
// 64-bit key) and for free rows (atomic counters); an ID's own slot and row are touched by one
// thread, so its metadata needs no atomics.
#include "../../include/mtgr_embedding.h"
#include "mtgr_device.h"
#include "mtgr_internal.h"

namespace mtgr {
namespace {

constexpr uint64_t KEY_EMPTY = 0xFFFFFFFFFFFFFFFFull;
constexpr uint64_t KEY_DELETED = 0xFFFFFFFFFFFFFFFEull;
constexpr int THREADS = 256;

// 64-bit finalizer of MurmurHash3 (public domain): spreads every input bit over the word.
__device__ __forceinline__ uint64_t mix64(uint64_t k) {
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdull;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ull;
    k ^= k >> 33;
    return k;
}

__device__ __forceinline__ uint64_t load_key(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t cas_key(uint64_t* p, uint64_t expect, uint64_t value) {
    return atomicCAS((unsigned long long*)p, (unsigned long long)expect, (unsigned long long)value);
}

__device__ __forceinline__ long long grid_threads() { return (long long)gridDim.x * blockDim.x; }
__device__ __forceinline__ long long thread_id() { return (long long)blockIdx.x * blockDim.x + threadIdx.x; }

__global__ void fill_u64_kernel(uint64_t* p, long long n, uint64_t v) {
    for (long long i = thread_id(); i < n; i += grid_threads()) p[i] = v;
}
__global__ void fill_i32_kernel(int* p, long long n, int v) {
    for (long long i = thread_id(); i < n; i += grid_threads()) p[i] = v;
}
__global__ void fill_f32_kernel(float* p, long long n, float v) {
    for (long long i = thread_id(); i < n; i += grid_threads()) p[i] = v;
}
__global__ void zero_i64_kernel(long long* p) { *p = 0; }

// ------------------------------------------------------------------------ de-duplication
// Each workgroup takes DEDUP_CHUNK consecutive IDs and first de-duplicates them in an LDS hash
// set (LDS integer atomics are cheap), then inserts each of its distinct IDs once into the
// global set (capacity tmask + 1 >= 2 n) and adds its local count there with one atomic.
// Skewed batches repeat a few hot IDs thousands of times; counting them in LDS first keeps the
// global atomics on a hot ID to one per workgroup.  pos[i] = the global slot of ids[i].
constexpr int DEDUP_PER_THREAD = 4;
constexpr int DEDUP_CHUNK = THREADS * DEDUP_PER_THREAD;   // 1024 IDs
constexpr int DEDUP_LCAP = 2 * DEDUP_CHUNK;               // LDS set: 2048 entries, 32 KB

__global__ __launch_bounds__(THREADS) void dedup_insert_kernel(long long n, const uint64_t* __restrict__ ids,
                                                               uint64_t* tkeys, int* tocc, int* __restrict__ pos,
                                                               long long tmask) {
    __shared__ uint64_t lkeys[DEDUP_LCAP];
    __shared__ int lcount[DEDUP_LCAP];
    __shared__ int lslot[DEDUP_LCAP];
    const long long i0 = (long long)blockIdx.x * DEDUP_CHUNK;
    for (int e = threadIdx.x; e < DEDUP_LCAP; e += THREADS) {
        lkeys[e] = KEY_EMPTY;
        lcount[e] = 0;
    }
    __syncthreads();
    int mine[DEDUP_PER_THREAD];
#pragma unroll
    for (int k = 0; k < DEDUP_PER_THREAD; k++) {
        const long long i = i0 + threadIdx.x + (long long)k * THREADS;
        mine[k] = -1;
        if (i >= n) continue;
        const uint64_t key = ids[i];
        int p = (int)(mix64(key) & (DEDUP_LCAP - 1));
        for (int step = 0; step < DEDUP_LCAP; step++) {
            const uint64_t old = atomicCAS((unsigned long long*)&lkeys[p], (unsigned long long)KEY_EMPTY,
                                           (unsigned long long)key);
            if (old == KEY_EMPTY || old == key) break;
            p = (p + 1) & (DEDUP_LCAP - 1);
        }
        atomicAdd(&lcount[p], 1);
        mine[k] = p;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < DEDUP_LCAP; e += THREADS) {
        const uint64_t key = lkeys[e];
        if (key == KEY_EMPTY) continue;
        long long p = (long long)(mix64(key) & (uint64_t)tmask);
        for (long long step = 0; step <= tmask; step++) {
            const uint64_t k = load_key(tkeys + p);
            if (k == key) break;
            if (k == KEY_EMPTY) {
                const uint64_t old = cas_key(tkeys + p, KEY_EMPTY, key);
                if (old == KEY_EMPTY || old == key) break;
            }
            p = (p + 1) & tmask;
        }
        atomicAdd(tocc + p, lcount[e]);
        lslot[e] = (int)p;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < DEDUP_PER_THREAD; k++) {
        const long long i = i0 + threadIdx.x + (long long)k * THREADS;
        if (i < n) pos[i] = lslot[mine[k]];
    }
}

// Scan of the set's occupancy in blocks of SCAN_BLOCK slots (THREADS x 4).
constexpr int SCAN_PER_THREAD = 4;
constexpr int SCAN_BLOCK = THREADS * SCAN_PER_THREAD;

__device__ __forceinline__ int block_scan_exclusive(int v, int* total) {
    __shared__ int wsum[THREADS / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < THREADS / 64; i++) {
        before += i < w ? wsum[i] : 0;
        all += wsum[i];
    }
    __syncthreads();   // wsum is reused by the next call
    *total = all;
    return before + incl - v;
}

__global__ __launch_bounds__(THREADS) void scan_count_kernel(const uint64_t* __restrict__ tkeys,
                                                             long long tcap, int* __restrict__ bsum) {
    const long long base = (long long)blockIdx.x * SCAN_BLOCK + threadIdx.x * SCAN_PER_THREAD;
    int c = 0;
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) c += (base + e < tcap && tkeys[base + e] != KEY_EMPTY) ? 1 : 0;
    int total;
    block_scan_exclusive(c, &total);
    if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

// Exclusive scan of the nblk block counts (one workgroup, in chunks); *count = their sum.
__global__ __launch_bounds__(THREADS) void scan_top_kernel(int* bsum, long long nblk, long long* count) {
    long long carry = 0;
    for (long long base = 0; base < nblk; base += THREADS) {
        const long long i = base + threadIdx.x;
        const int v = i < nblk ? bsum[i] : 0;
        int total;
        const int ex = block_scan_exclusive(v, &total);
        if (i < nblk) bsum[i] = (int)(carry + ex);
        carry += total;
    }
    if (threadIdx.x == 0) *count = carry;
}

__global__ __launch_bounds__(THREADS) void scan_emit_kernel(const uint64_t* __restrict__ tkeys,
                                                            const int* __restrict__ tocc, long long tcap,
                                                            const int* __restrict__ bsum, int* __restrict__ rank,
                                                            uint64_t* __restrict__ unique,
                                                            int* __restrict__ occ_out) {
    const long long base = (long long)blockIdx.x * SCAN_BLOCK + threadIdx.x * SCAN_PER_THREAD;
    bool occ[SCAN_PER_THREAD];
    int c = 0;
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) {
        occ[e] = base + e < tcap && tkeys[base + e] != KEY_EMPTY;
        c += occ[e] ? 1 : 0;
    }
    int total;
    int r = bsum[blockIdx.x] + block_scan_exclusive(c, &total);
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) {
        if (occ[e]) {
            rank[base + e] = r;
            unique[r] = tkeys[base + e];
            if (occ_out) occ_out[r] = tocc[base + e];
            r++;
        }
    }
}

__global__ void dedup_inverse_kernel(long long n, const int* __restrict__ pos, const int* __restrict__ rank,
                                     int* __restrict__ inverse) {
    for (long long i = thread_id(); i < n; i += grid_threads()) inverse[i] = rank[pos[i]];
}

// ------------------------------------------------------------------------ lookup / insert
// Phase 1: find each ID's slot, or (insert) claim one: the first DELETED slot met on the probe
// path if the path ends at an EMPTY slot without the ID, else that EMPTY slot.  lpos = slot or
// -1 (absent, or no free slot: overflow bit 1), lfresh = 1 when claimed here.
__global__ void lookup_probe_kernel(EmbArgs t, long long n_max, const uint64_t* __restrict__ unique,
                                    const long long* __restrict__ num_unique, int insert,
                                    int* __restrict__ lpos, int* __restrict__ lfresh) {
    const long long nu = min(*num_unique, n_max);
    const long long mask = t.key_capacity - 1;
    for (long long u = thread_id(); u < nu; u += grid_threads()) {
        const uint64_t key = unique[u];
        long long p = (long long)(mix64(key) & (uint64_t)mask);
        long long tomb = -1, slot = -1;
        int fresh = 0;
        bool done = false;
        for (long long step = 0; step < 2 * t.key_capacity && !done; step++) {
            const uint64_t k = load_key(t.keys + p);
            if (k == key) {
                slot = p;
                done = true;
            } else if (k == KEY_DELETED) {
                if (tomb < 0) tomb = p;
                p = (p + 1) & mask;
            } else if (k == KEY_EMPTY) {
                if (!insert) {
                    done = true;   // absent
                } else {
                    const long long tgt = tomb >= 0 ? tomb : p;
                    const uint64_t expect = tomb >= 0 ? KEY_DELETED : KEY_EMPTY;
                    if (cas_key(t.keys + tgt, expect, key) == expect) {
                        slot = tgt;
                        fresh = 1;
                        done = true;
                    } else if (tomb >= 0) {
                        tomb = -1;           // another ID took the deleted slot: look at p again
                    } else {
                        p = (p + 1) & mask;  // another ID took this empty slot
                    }
                }
            } else {
                p = (p + 1) & mask;
            }
        }
        if (!done && insert && tomb >= 0 && cas_key(t.keys + tomb, KEY_DELETED, key) == KEY_DELETED) {
            slot = tomb;   // the whole store was walked: no EMPTY slot, but a DELETED one
            fresh = 1;
            done = true;
        }
        if (fresh) atomicAdd(t.state + MTGR_EMB_STATE_NUM_KEYS, 1);
        if (!done && insert) atomicOr(t.state + MTGR_EMB_STATE_OVERFLOW, 2);
        lpos[u] = (int)slot;
        lfresh[u] = fresh;
    }
}

// A free row: the top of the free-row stack, else the next never-used row, else -1.  The
// stack top may go negative and the row counter past the capacity; fixup_kernel clamps both.
__device__ __forceinline__ int alloc_row(const EmbArgs& t) {
    const int i = atomicSub(t.state + MTGR_EMB_STATE_FREE_TOP, 1) - 1;
    if (i >= 0) return t.free_rows[i];
    const int r = atomicAdd(t.state + MTGR_EMB_STATE_NEXT_ROW, 1);
    return r < t.row_capacity ? r : -1;
}

__device__ __forceinline__ void zero_row(const EmbArgs& t, int row) {
    uint4* v = (uint4*)((char*)t.values + (long long)row * t.dim * t.esize);
    const int chunks = t.dim * t.esize / 16;
    for (int c = 0; c < chunks; c++) v[c] = make_uint4(0, 0, 0, 0);
}

// Phase 2: rows for the claimed slots, then counters and timestamps.
__global__ void lookup_finish_kernel(EmbArgs t, long long n_max, const int* __restrict__ occurrences,
                                     const long long* __restrict__ num_unique, int now,
                                     const int* __restrict__ lpos, const int* __restrict__ lfresh,
                                     int* __restrict__ rows) {
    const long long nu = min(*num_unique, n_max);
    for (long long u = thread_id(); u < nu; u += grid_threads()) {
        const int p = lpos[u];
        if (p < 0) {
            rows[u] = -1;
            continue;
        }
        int row;
        if (lfresh[u]) {
            row = alloc_row(t);
            if (row < 0) {
                // No row: release the slot as DELETED (IDs inserted meanwhile may have probed
                // past it, so it must not become EMPTY).
                __hip_atomic_store(t.keys + p, KEY_DELETED, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                atomicSub(t.state + MTGR_EMB_STATE_NUM_KEYS, 1);
                atomicOr(t.state + MTGR_EMB_STATE_OVERFLOW, 1);
                rows[u] = -1;
                continue;
            }
            t.key_rows[p] = row;
            zero_row(t, row);
            t.counts[row] = 0u;
        } else {
            row = t.key_rows[p];
        }
        t.counts[row] += occurrences ? (uint32_t)occurrences[u] : 1u;
        t.last_ts[row] = now;
        rows[u] = row;
    }
}

__global__ void fixup_kernel(EmbArgs t) {
    int* s = t.state;
    s[MTGR_EMB_STATE_FREE_TOP] = max(s[MTGR_EMB_STATE_FREE_TOP], 0);
    s[MTGR_EMB_STATE_NEXT_ROW] = min(s[MTGR_EMB_STATE_NEXT_ROW], t.row_capacity);
}

// ------------------------------------------------------------------------ gather / sgd
// One thread per 16-byte chunk of an output row.
__global__ void gather_kernel(EmbArgs t, long long n, const int* __restrict__ inverse,
                              const int* __restrict__ rows, void* __restrict__ out, long long ld_out) {
    const int cpr = t.dim * t.esize / 16;
    const long long total = n * cpr;
    for (long long c = thread_id(); c < total; c += grid_threads()) {
        const long long i = c / cpr;
        const int j = (int)(c - i * cpr);
        const int row = rows[inverse[i]];
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row >= 0) v = ((const uint4*)((const char*)t.values + (long long)row * t.dim * t.esize))[j];
        ((uint4*)((char*)out + i * ld_out * t.esize))[j] = v;
    }
}

__device__ __forceinline__ void load_chunk(const void* base, int esize, float* f) {
    const uint4 v = *(const uint4*)base;
    if (esize == 2) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; e++) {
            f[2 * e] = __uint_as_float(w[e] << 16);
            f[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
        }
    } else {
        f[0] = __uint_as_float(v.x);
        f[1] = __uint_as_float(v.y);
        f[2] = __uint_as_float(v.z);
        f[3] = __uint_as_float(v.w);
    }
}

// Grouping of a batch's positions by unique ID (a counting sort): start = exclusive scan of
// the occurrences, then each position takes the next free place of its ID's range.
__global__ __launch_bounds__(THREADS) void iscan_count_kernel(const int* __restrict__ in,
                                                              const long long* __restrict__ num, long long n_max,
                                                              int* __restrict__ bsum) {
    const long long nv = min(*num, n_max);
    const long long base = (long long)blockIdx.x * SCAN_BLOCK + threadIdx.x * SCAN_PER_THREAD;
    int c = 0;
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) c += base + e < nv ? in[base + e] : 0;
    int total;
    block_scan_exclusive(c, &total);
    if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

__global__ __launch_bounds__(THREADS) void iscan_apply_kernel(const int* __restrict__ in,
                                                              const long long* __restrict__ num, long long n_max,
                                                              const int* __restrict__ bsum, int* __restrict__ out) {
    const long long nv = min(*num, n_max);
    const long long base = (long long)blockIdx.x * SCAN_BLOCK + threadIdx.x * SCAN_PER_THREAD;
    int v[SCAN_PER_THREAD], c = 0;
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) {
        v[e] = base + e < nv ? in[base + e] : 0;
        c += v[e];
    }
    int total;
    int r = bsum[blockIdx.x] + block_scan_exclusive(c, &total);
#pragma unroll
    for (int e = 0; e < SCAN_PER_THREAD; e++) {
        if (base + e < nv) out[base + e] = r;
        r += v[e];
    }
}

// Counting-sort scatter of the positions: list[start[u] + r] = i for the r-th position of ID u
// (lu = u alongside).  A workgroup takes DEDUP_CHUNK positions and counts its IDs in an LDS hash
// first, so a hot ID costs one global atomic per workgroup; its positions then take
// consecutive places from the range reserved there.
__global__ __launch_bounds__(THREADS) void group_scatter_kernel(long long n, const int* __restrict__ inverse,
                                                                const int* __restrict__ start, int* cursor,
                                                                int* __restrict__ list, int* __restrict__ lu) {
    __shared__ int lkey[DEDUP_LCAP];
    __shared__ int lcount[DEDUP_LCAP];
    __shared__ int lbase[DEDUP_LCAP];
    const long long i0 = (long long)blockIdx.x * DEDUP_CHUNK;
    for (int e = threadIdx.x; e < DEDUP_LCAP; e += THREADS) {
        lkey[e] = -1;
        lcount[e] = 0;
    }
    __syncthreads();
    int slot[DEDUP_PER_THREAD], rank[DEDUP_PER_THREAD];
#pragma unroll
    for (int k = 0; k < DEDUP_PER_THREAD; k++) {
        const long long i = i0 + threadIdx.x + (long long)k * THREADS;
        slot[k] = -1;
        rank[k] = 0;
        if (i >= n) continue;
        const int u = inverse[i];
        int p = (int)(mix64((uint64_t)u) & (DEDUP_LCAP - 1));
        for (int step = 0; step < DEDUP_LCAP; step++) {
            const int old = atomicCAS(&lkey[p], -1, u);
            if (old == -1 || old == u) break;
            p = (p + 1) & (DEDUP_LCAP - 1);
        }
        rank[k] = atomicAdd(&lcount[p], 1);
        slot[k] = p;
    }
    __syncthreads();
    for (int e = threadIdx.x; e < DEDUP_LCAP; e += THREADS) {
        const int u = lkey[e];
        if (u >= 0) lbase[e] = start[u] + atomicAdd(cursor + u, lcount[e]);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < DEDUP_PER_THREAD; k++) {
        const long long i = i0 + threadIdx.x + (long long)k * THREADS;
        if (i >= n) continue;
        const int p = lbase[slot[k]] + rank[k];
        if (p < n) {   // always, for occurrences consistent with inverse
            list[p] = (int)i;
            lu[p] = lkey[slot[k]];
        }
    }
}

// Sum of each ID's gradient rows.  The grouped positions are cut into chunks of GROUP_CHUNK;
// a workgroup of THREADS threads takes CPB = THREADS / cpr consecutive chunks, one thread per
// (chunk, 16-byte column block).  A thread walks its chunk and sums runs of one ID in
// registers: runs strictly inside the chunk are complete IDs and are stored; the first and last
// run go to LDS, where one thread per column then merges equal IDs across the workgroup's chunks
// and stores each merged run, or adds it with a float atomic when the ID continues beyond the
// workgroup.  A hot ID with thousands of positions thus costs one atomic per workgroup and
// column element instead of one per chunk.
constexpr int GROUP_CHUNK = 32;

template <int ESIZE>
__global__ __launch_bounds__(THREADS) void group_sum_kernel(EmbArgs t, long long n, const int* __restrict__ list,
                                                            const int* __restrict__ lu,
                                                            const int* __restrict__ start,
                                                            const int* __restrict__ occ,
                                                            const void* __restrict__ grad, long long ld_grad,
                                                            float* acc) {
    constexpr int epc = 16 / ESIZE, UNR = 8;
    static_assert(GROUP_CHUNK % UNR == 0, "whole unrolled steps");
    __shared__ float first_part[THREADS][epc];
    __shared__ float last_part[THREADS][epc];
    __shared__ int first_u[THREADS];
    __shared__ int last_u[THREADS];
    const int cpr = t.dim / epc;                       // column blocks per row (<= THREADS here)
    const int cpb = THREADS / cpr;                     // chunks per workgroup
    const long long P0 = (long long)blockIdx.x * cpb * GROUP_CHUNK, P1 = min(n, P0 + (long long)cpb * GROUP_CHUNK);
    const int c = threadIdx.x / cpr, j = threadIdx.x - c * cpr;
    const long long p0 = P0 + (long long)c * GROUP_CHUNK, p1 = min(P1, p0 + GROUP_CHUNK);
    auto store_or_add = [&](int u, const float* f, long long lo, long long hi) {
        float* dst = acc + (long long)u * t.dim + j * epc;
        const long long s0 = start[u], s1 = s0 + occ[u];
        if (s0 >= lo && s1 <= hi) {
#pragma unroll
            for (int e = 0; e < epc; e++) dst[e] = f[e];
        } else {
#pragma unroll
            for (int e = 0; e < epc; e++) atomicAdd(dst + e, f[e]);
        }
    };
    float f[epc];
#pragma unroll
    for (int e = 0; e < epc; e++) f[e] = 0.f;
    int cur = -1, runs = 0;
    if (c < cpb) {
        for (long long pb = p0; pb < p1; pb += UNR) {
            int ii[UNR], uu[UNR];
#pragma unroll
            for (int k = 0; k < UNR; k++) {
                const bool in = pb + k < p1;
                ii[k] = in ? list[pb + k] : -1;
                uu[k] = in ? lu[pb + k] : -1;
            }
            float g[UNR][8];
#pragma unroll
            for (int k = 0; k < UNR; k++) {
                if (ii[k] >= 0 && ii[k] < n)
                    load_chunk((const char*)grad + ((long long)ii[k] * ld_grad + (long long)j * epc) * ESIZE, ESIZE,
                               g[k]);
                else
                    uu[k] = -1;   // past the chunk (or, for inconsistent occurrences, a hole)
            }
#pragma unroll
            for (int k = 0; k < UNR; k++) {
                if (uu[k] < 0) continue;
                if (uu[k] != cur) {
                    if (cur >= 0) {
                        if (runs == 1) {   // the first run of the chunk: to LDS
                            first_u[threadIdx.x] = cur;
#pragma unroll
                            for (int e = 0; e < epc; e++) first_part[threadIdx.x][e] = f[e];
                        } else {           // a run strictly inside the chunk: a whole ID
                            store_or_add(cur, f, p0, p1);
                        }
                    }
                    cur = uu[k];
                    runs++;
#pragma unroll
                    for (int e = 0; e < epc; e++) f[e] = 0.f;
                }
#pragma unroll
                for (int e = 0; e < epc; e++) f[e] += g[k][e];
            }
        }
    }
    // the last run (the first as well when the chunk holds one ID; none for an empty chunk)
    if (runs == 1) first_u[threadIdx.x] = -1;
    if (runs == 0) first_u[threadIdx.x] = -1;
    last_u[threadIdx.x] = cur;
#pragma unroll
    for (int e = 0; e < epc; e++) last_part[threadIdx.x][e] = f[e];
    __syncthreads();
    if (threadIdx.x < cpr) {
        int run_u = -1;
        float r[epc];
#pragma unroll
        for (int e = 0; e < epc; e++) r[e] = 0.f;
        for (int cc = 0; cc < cpb; cc++) {
            const int pair = cc * cpr + j;
#pragma unroll
            for (int half = 0; half < 2; half++) {
                const int u = half == 0 ? first_u[pair] : last_u[pair];
                if (u < 0) continue;
                const float* part = half == 0 ? first_part[pair] : last_part[pair];
                if (u != run_u) {
                    if (run_u >= 0) store_or_add(run_u, r, P0, P1);
                    run_u = u;
#pragma unroll
                    for (int e = 0; e < epc; e++) r[e] = 0.f;
                }
#pragma unroll
                for (int e = 0; e < epc; e++) r[e] += part[e];
            }
        }
        if (run_u >= 0) store_or_add(run_u, r, P0, P1);
    }
}

// values[rows[u], :] -= lr * acc[u, :], rounded to the table's dtype.
template <int ESIZE>
__global__ void sgd_apply_kernel(EmbArgs t, long long n_max, const int* __restrict__ rows,
                                 const long long* __restrict__ num_unique, const float* __restrict__ acc,
                                 float lr) {
    constexpr int epc = 16 / ESIZE;
    const long long nu = min(*num_unique, n_max);
    const int cpr = t.dim / epc;
    const long long total = nu * cpr;
    for (long long c = thread_id(); c < total; c += grid_threads()) {
        const long long u = c / cpr;
        const int j = (int)(c - u * cpr);
        const int row = rows[u];
        if (row < 0) continue;
        char* vp = (char*)t.values + ((long long)row * t.dim + (long long)j * epc) * ESIZE;
        float f[8];
        load_chunk(vp, ESIZE, f);
        const float* g = acc + u * t.dim + j * epc;
#pragma unroll
        for (int e = 0; e < epc; e++) f[e] = __builtin_fmaf(-lr, g[e], f[e]);
        uint4 v;
        if constexpr (ESIZE == 2) {
            v = make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                           pack_bf16x2(f[6], f[7]));
        } else {
            v = make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                           __float_as_uint(f[3]));
        }
        *(uint4*)vp = v;
    }
}

// ------------------------------------------------------------------------ evict / rehash
__global__ void evict_kernel(EmbArgs t, int threshold, uint32_t min_count, long long* num_evicted) {
    for (long long p = thread_id(); p < t.key_capacity; p += grid_threads()) {
        const uint64_t k = t.keys[p];
        if (k >= KEY_DELETED) continue;
        const int row = t.key_rows[p];
        if (row < 0 || (t.last_ts[row] >= threshold && t.counts[row] >= min_count)) continue;
        t.keys[p] = KEY_DELETED;
        t.key_rows[p] = -1;
        const int i = atomicAdd(t.state + MTGR_EMB_STATE_FREE_TOP, 1);
        t.free_rows[i] = row;
        atomicSub(t.state + MTGR_EMB_STATE_NUM_KEYS, 1);
        atomicAdd((unsigned long long*)num_evicted, 1ull);
    }
}

__global__ void rehash_kernel(EmbArgs from, EmbArgs to) {
    const long long mask = to.key_capacity - 1;
    for (long long p = thread_id(); p < from.key_capacity; p += grid_threads()) {
        const uint64_t key = from.keys[p];
        if (key >= KEY_DELETED) continue;
        long long q = (long long)(mix64(key) & (uint64_t)mask);
        bool placed = false;
        for (long long step = 0; step < to.key_capacity && !placed; step++) {
            if (cas_key(to.keys + q, KEY_EMPTY, key) == KEY_EMPTY) {
                to.key_rows[q] = from.key_rows[p];
                placed = true;
            } else {
                q = (q + 1) & mask;
            }
        }
        if (!placed) atomicOr(to.state + MTGR_EMB_STATE_OVERFLOW, 2);
    }
}

int grid_for(long long work) {
    const long long blocks = (work + THREADS - 1) / THREADS;
    return (int)max(1ll, min(blocks, 8192ll));
}

}  // namespace

size_t dedup_set_capacity(long long n) {
    size_t c = 64;
    while ((long long)c < 2 * n) c <<= 1;
    return c;
}

size_t dedup_workspace_bytes(long long n) {
    const size_t tcap = dedup_set_capacity(n);
    const size_t nblk = (tcap + SCAN_BLOCK - 1) / SCAN_BLOCK;
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    return a(tcap * 8) + a(tcap * 4) * 2 + a((size_t)n * 4) + a((nblk + 1) * 4);
}

hipError_t launch_emb_init(const EmbArgs& t, hipStream_t s) {
    fill_u64_kernel<<<grid_for(t.key_capacity), THREADS, 0, s>>>(t.keys, t.key_capacity, KEY_EMPTY);
    fill_i32_kernel<<<grid_for(t.key_capacity), THREADS, 0, s>>>(t.key_rows, t.key_capacity, -1);
    fill_i32_kernel<<<1, THREADS, 0, s>>>(t.state, MTGR_EMB_STATE_WORDS, 0);
    return hipGetLastError();
}

hipError_t launch_emb_dedup(long long n, const uint64_t* ids, uint64_t* unique, int* occ, int* inverse,
                            long long* num_unique, void* ws, hipStream_t s) {
    const size_t tcap = dedup_set_capacity(n);
    const size_t nblk = (tcap + SCAN_BLOCK - 1) / SCAN_BLOCK;
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    char* w = (char*)ws;
    uint64_t* tkeys = (uint64_t*)w;
    w += a(tcap * 8);
    int* tocc = (int*)w;
    w += a(tcap * 4);
    int* rank = (int*)w;
    w += a(tcap * 4);
    int* pos = (int*)w;
    w += a((size_t)n * 4);
    int* bsum = (int*)w;
    fill_u64_kernel<<<grid_for(tcap), THREADS, 0, s>>>(tkeys, (long long)tcap, KEY_EMPTY);
    fill_i32_kernel<<<grid_for(tcap), THREADS, 0, s>>>(tocc, (long long)tcap, 0);
    if (n > 0)
        dedup_insert_kernel<<<(int)((n + DEDUP_CHUNK - 1) / DEDUP_CHUNK), THREADS, 0, s>>>(n, ids, tkeys, tocc, pos,
                                                                                         (long long)tcap - 1);
    scan_count_kernel<<<(int)nblk, THREADS, 0, s>>>(tkeys, (long long)tcap, bsum);
    scan_top_kernel<<<1, THREADS, 0, s>>>(bsum, (long long)nblk, num_unique);
    scan_emit_kernel<<<(int)nblk, THREADS, 0, s>>>(tkeys, tocc, (long long)tcap, bsum, rank, unique, occ);
    if (n > 0) dedup_inverse_kernel<<<grid_for(n), THREADS, 0, s>>>(n, pos, rank, inverse);
    return hipGetLastError();
}

hipError_t launch_emb_lookup(const EmbArgs& t, long long n_max, const uint64_t* unique, const int* occ,
                             const long long* num_unique, int now, int insert, int* rows, void* ws,
                             hipStream_t s) {
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    int* lpos = (int*)ws;
    int* lfresh = (int*)((char*)ws + a((size_t)n_max * 4));
    lookup_probe_kernel<<<grid_for(n_max), THREADS, 0, s>>>(t, n_max, unique, num_unique, insert, lpos, lfresh);
    lookup_finish_kernel<<<grid_for(n_max), THREADS, 0, s>>>(t, n_max, occ, num_unique, now, lpos, lfresh, rows);
    fixup_kernel<<<1, 1, 0, s>>>(t);
    return hipGetLastError();
}

size_t lookup_workspace_bytes(long long n_max) {
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    return 2 * a((size_t)n_max * 4);
}

hipError_t launch_emb_gather(const EmbArgs& t, long long n, const int* inverse, const int* rows, void* out,
                             long long ld_out, hipStream_t s) {
    const long long chunks = n * (t.dim * t.esize / 16);
    gather_kernel<<<grid_for(chunks), THREADS, 0, s>>>(t, n, inverse, rows, out, ld_out);
    return hipGetLastError();
}

namespace {
struct SgdLayout {
    size_t acc, start, cursor, list, lu, bsum, count, total;
};
SgdLayout sgd_layout(long long n, long long n_max, int dim) {
    auto a = [](size_t b) { return (b + 255) & ~(size_t)255; };
    const size_t nblk = ((size_t)n_max + SCAN_BLOCK - 1) / SCAN_BLOCK;
    SgdLayout L;
    L.acc = 0;
    L.start = L.acc + a((size_t)n_max * dim * sizeof(float));
    L.cursor = L.start + a(((size_t)n_max + 1) * 4);
    L.list = L.cursor + a((size_t)n_max * 4);
    L.lu = L.list + a((size_t)n * 4);
    L.bsum = L.lu + a((size_t)n * 4);
    L.count = L.bsum + a((nblk + 1) * 4);
    L.total = L.count + 256;
    return L;
}
}  // namespace

size_t sgd_workspace_bytes(long long n, long long n_max, int dim) { return sgd_layout(n, n_max, dim).total; }

hipError_t launch_emb_sgd(const EmbArgs& t, long long n, const int* inverse, const int* occ, const void* grad,
                          long long ld_grad, long long n_max, const int* rows, const long long* num_unique,
                          float lr, void* ws, hipStream_t s) {
    const SgdLayout L = sgd_layout(n, n_max, t.dim);
    char* w = (char*)ws;
    float* acc = (float*)(w + L.acc);
    int* start = (int*)(w + L.start);
    int* cursor = (int*)(w + L.cursor);
    int* list = (int*)(w + L.list);
    int* lu = (int*)(w + L.lu);
    int* bsum = (int*)(w + L.bsum);
    long long* count = (long long*)(w + L.count);
    const long long nblk = (n_max + SCAN_BLOCK - 1) / SCAN_BLOCK;
    const long long cells = n_max * t.dim;
    fill_f32_kernel<<<grid_for(cells), THREADS, 0, s>>>(acc, cells, 0.f);
    if (n > 0) {
        fill_i32_kernel<<<grid_for(n_max), THREADS, 0, s>>>(cursor, n_max, 0);
        iscan_count_kernel<<<(int)nblk, THREADS, 0, s>>>(occ, num_unique, n_max, bsum);
        scan_top_kernel<<<1, THREADS, 0, s>>>(bsum, nblk, count);
        iscan_apply_kernel<<<(int)nblk, THREADS, 0, s>>>(occ, num_unique, n_max, bsum, start);
        group_scatter_kernel<<<(int)((n + DEDUP_CHUNK - 1) / DEDUP_CHUNK), THREADS, 0, s>>>(n, inverse, start, cursor,
                                                                                          list, lu);
        const int cpr = t.dim * t.esize / 16, cpb = THREADS / cpr;
        const long long nchunk = (n + GROUP_CHUNK - 1) / GROUP_CHUNK;
        const int blocks = (int)((nchunk + cpb - 1) / cpb);
        if (t.esize == 2)
            group_sum_kernel<2><<<blocks, THREADS, 0, s>>>(t, n, list, lu, start, occ, grad, ld_grad, acc);
        else
            group_sum_kernel<4><<<blocks, THREADS, 0, s>>>(t, n, list, lu, start, occ, grad, ld_grad, acc);
    }
    const int epc = 16 / t.esize;
    if (t.esize == 2)
        sgd_apply_kernel<2><<<grid_for(n_max * (t.dim / epc)), THREADS, 0, s>>>(t, n_max, rows, num_unique, acc, lr);
    else
        sgd_apply_kernel<4><<<grid_for(n_max * (t.dim / epc)), THREADS, 0, s>>>(t, n_max, rows, num_unique, acc, lr);
    return hipGetLastError();
}

hipError_t launch_emb_evict(const EmbArgs& t, int threshold, uint32_t min_count, long long* num_evicted,
                            hipStream_t s) {
    zero_i64_kernel<<<1, 1, 0, s>>>(num_evicted);
    evict_kernel<<<grid_for(t.key_capacity), THREADS, 0, s>>>(t, threshold, min_count, num_evicted);
    return hipGetLastError();
}

hipError_t launch_emb_rehash(const EmbArgs& from, const EmbArgs& to, hipStream_t s) {
    fill_u64_kernel<<<grid_for(to.key_capacity), THREADS, 0, s>>>(to.keys, to.key_capacity, KEY_EMPTY);
    fill_i32_kernel<<<grid_for(to.key_capacity), THREADS, 0, s>>>(to.key_rows, to.key_capacity, -1);
    rehash_kernel<<<grid_for(from.key_capacity), THREADS, 0, s>>>(from, to);
    return hipGetLastError();
}

}  // namespace mtgr
