// Internal device-side helpers for the gfx950 kernels (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define MTGR_RAB_LDS 64   // relative-bias buckets held in LDS (the ABI maximum)

namespace mtgr {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;

constexpr int SEG_USER = 0, SEG_HIST = 1, SEG_RT = 2, SEG_CAND = 3;

// Per-64-token tile summary flags (relative to one user's tokens).
constexpr int TS_ANY_STATIC = 1;   // some valid token is USER/HIST
constexpr int TS_ALL_STATIC = 2;   // all 64 slots are valid USER/HIST tokens
constexpr int TS_ANY_RT = 4;       // some valid token is RT
constexpr int TS_ANY_DYN = 8;      // some valid token is RT or CAND
constexpr int TS_ANY_CAND = 16;    // some valid token is CAND
constexpr int SUMMARY_TILE = 64;

// Tile classes of a (query range, key range) pair.
constexpr int TILE_MASKED = 0, TILE_PARTIAL = 1, TILE_FULL = 2;

struct TileSummary {
    int flags;
    int min_rt_ts;    // min ts over RT tokens (INT_MAX if none)
    int max_dyn_ts;   // max ts over RT/CAND tokens (INT_MIN if none)
    int pad;
};

__device__ __forceinline__ TileSummary combine(TileSummary a, TileSummary b) {
    TileSummary r;
    r.flags = ((a.flags | b.flags) & ~TS_ALL_STATIC) | (a.flags & b.flags & TS_ALL_STATIC);
    r.min_rt_ts = min(a.min_rt_ts, b.min_rt_ts);
    r.max_dyn_ts = max(a.max_dyn_ts, b.max_dyn_ts);
    r.pad = 0;
    return r;
}

__device__ __forceinline__ TileSummary empty_summary() {
    TileSummary r;
    r.flags = TS_ALL_STATIC;  // neutral for combine()
    r.min_rt_ts = 0x7fffffff;
    r.max_dyn_ts = (int)0x80000000;
    r.pad = 0;
    return r;
}

__device__ __forceinline__ TileSummary load_summary(const int4* s, int idx) {
    int4 v = s[idx];
    TileSummary r;
    r.flags = v.x;
    r.min_rt_ts = v.y;
    r.max_dyn_ts = v.z;
    r.pad = 0;
    return r;
}

// Class of the pair (queries summarised by sq, keys summarised by sk).  `overlap`
// says whether the two token ranges intersect (the diagonal i == j is always seen).
__device__ __forceinline__ int tile_class(TileSummary sq, TileSummary sk, bool overlap) {
    if (sk.flags & TS_ALL_STATIC) return TILE_FULL;
    if (sk.flags & TS_ANY_STATIC) return TILE_PARTIAL;
    if ((sk.flags & TS_ANY_RT) && (sq.flags & TS_ANY_DYN) && sk.min_rt_ts < sq.max_dyn_ts)
        return TILE_PARTIAL;
    return overlap ? TILE_PARTIAL : TILE_MASKED;
}

// Walks, in increasing order, the 64-token tiles of one user whose class against a fixed
// tile range is not MASKED.  The classes of 64 consecutive tiles are evaluated at once, one tile
// per lane, and kept as two wave-uniform bit masks, so stepping to the next visible tile costs a
// few scalar bit operations and one summary load per 64 tiles instead of a dependent global load
// per tile.  `ClassFn(t)` returns the class of tile t (t < ntile); all lanes must call next().
template <class ClassFn>
struct TileWalker {
    ClassFn class_of;
    int ntile;
    int base;                  // first tile of the current window (multiple of 64)
    unsigned long long vis;    // bit j: tile base + j is not MASKED
    unsigned long long part;   // bit j: tile base + j is PARTIAL

    __device__ TileWalker(ClassFn f, int n) : class_of(f), ntile(n), base(-64), vis(0), part(0) {}

    __device__ void load(int b) {
        base = b;
        const int t = b + (int)(threadIdx.x & 63);
        const int c = t < ntile ? class_of(t) : TILE_MASKED;
        vis = __ballot(c != TILE_MASKED);
        part = __ballot(c == TILE_PARTIAL);
    }

    // First visible tile >= t (ntile if none); its class in *cls.
    __device__ int next(int t, int* cls) {
        while (t < ntile) {
            if (t >= base + 64) load(t & ~63);
            const unsigned long long m = vis >> (t - base);
            if (m) {
                t += __builtin_ctzll(m);
                *cls = ((part >> (t - base)) & 1ull) ? TILE_PARTIAL : TILE_FULL;
                return t;
            }
            t = base + 64;
        }
        *cls = TILE_MASKED;
        return ntile;
    }
};

// Per-token mask code: bit0 static, bit1 real-time, bit2 dynamic (RT or CAND), bit3 valid.
constexpr int KC_STATIC = 1, KC_RT = 2, KC_DYN = 4, KC_VALID = 8;

__device__ __forceinline__ int token_code(int seg) {
    int c = KC_VALID;
    if (seg <= SEG_HIST) c |= KC_STATIC;
    if (seg == SEG_RT) c |= KC_RT;
    if (seg >= SEG_RT) c |= KC_DYN;
    return c;
}

// Dynamic mask of Sec. 4.2 from token codes: i == j, static key (rule 1), or an RT key
// strictly earlier than a dynamic query (rule 2); candidates only see themselves (rule 3).
// Evaluated with bitwise logic so that it compiles to compares and selects, not branches.
__device__ __forceinline__ bool visible(int qcode, int qts, int qidx, int kcode, int kts,
                                        int kidx) {
    const int both_valid = kcode & qcode & KC_VALID;
    const int rule2 = (kcode & KC_RT) & ((qcode & KC_DYN) >> 1) & (kts < qts ? KC_RT : 0);
    const int seen = (kcode & KC_STATIC) | (qidx == kidx ? 1 : 0) | (rule2 >> 1);
    return (seen != 0) & (both_valid != 0);
}

// The mask as one 64-bit comparison: key j is visible to query i (i != j) iff
// query_value(i) >= key_threshold(j).  A static key is seen by every query (threshold -2^63); an
// RT key by the RT and candidate queries later than it (threshold ts_j + 1 against the query's
// ts); a candidate key, and a padded key (code 0), by nobody but itself (threshold 2^63 - 1);
// a static query has the value -2^63, so it sees static keys only.  Equal to visible() for every
// valid query row and every int32 timestamp.
__device__ __forceinline__ long long key_threshold(int kcode, int kts) {
    if (kcode & KC_STATIC) return (long long)0x8000000000000000ull;
    if (kcode & KC_RT) return (long long)kts + 1;
    return 0x7fffffffffffffffll;
}
__device__ __forceinline__ long long query_value(int qcode, int qts) {
    return (qcode & KC_DYN) ? (long long)qts : (long long)0x8000000000000000ull;
}

// visible() with the diagonal test i == j already evaluated by the caller.
__device__ __forceinline__ bool visible_diag(int qcode, int qts, int kcode, int kts, bool diag) {
    const int both_valid = kcode & qcode & KC_VALID;
    const int rule2 = (kcode & KC_RT) & ((qcode & KC_DYN) >> 1) & (kts < qts ? KC_RT : 0);
    const int seen = (kcode & KC_STATIC) | (diag ? 1 : 0) | (rule2 >> 1);
    return (seen != 0) & (both_valid != 0);
}

// Half-octave log-time bucket of |a - b| (gap as uint32), clamped to nb - 1.
__device__ __forceinline__ int rab_bucket(int a, int b, int nb) {
    uint32_t g = a >= b ? (uint32_t)a - (uint32_t)b : (uint32_t)b - (uint32_t)a;
    int bk;
    if (g < 2u) {
        bk = (int)g;
    } else {
        int e = 31 - __clz(g);
        bk = 2 * e + (int)((g >> (e - 1)) & 1u);
    }
    return min(bk, nb - 1);
}

// With a relative bias the forward and the recomputing dQ kernel keep the bias table in LDS
// multiplied by -log2(e), so that the sigmoid's exponent y = -log2(e) (alpha s + rab) is one fma
// of the score (c_exp = -log2(e) alpha).  They work with P'' = y sigmoid = -log2(e) silu(x); the
// factor -ln 2 that turns P'' back into silu(x) is applied once to the output, and silu'(x) =
// sigmoid + x sigmoid (1 - sigmoid) = sigmoid - ln 2 P'' (1 - sigmoid).
constexpr float NEG_LOG2E = -1.4426950408889634f;
constexpr float NEG_LN2 = -0.6931471805599453f;

// P'' and the sigmoid for the scaled exponent y.
__device__ __forceinline__ float silu_scaled(float y, float& sg) {
    sg = __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(y));
    return y * sg;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
    return __uint_as_float(((uint32_t)h) << 16);
}

// Stores with the non-temporal hint, for results written once and not read again by the kernel
// (output rows, the stored dS blocks): measured faster than plain stores for these full-line
// writes.
typedef unsigned int u32x4_nt __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_nt __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_nt16(void* dst, const void* src) {
    __builtin_nontemporal_store(*(const u32x4_nt*)src, (u32x4_nt*)dst);
}
__device__ __forceinline__ void store_nt8(void* dst, uint32_t lo, uint32_t hi) {
    const u32x2_nt v = {lo, hi};
    __builtin_nontemporal_store(v, (u32x2_nt*)dst);
}

// Element access of the vector-ALU kernels, which store either fp32 or bf16 and compute in fp32.
__device__ __forceinline__ float ld_elem(const float* p, long long i) { return p[i]; }
__device__ __forceinline__ float ld_elem(const uint16_t* p, long long i) { return bf16_to_f32(p[i]); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));

// fp32 pair -> packed bf16 pair, round to nearest even (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const float2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}

__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return pack_bf16x2(f, 0.f) & 0xffffu; }

__device__ __forceinline__ void st_elem(float* p, long long i, float v) { p[i] = v; }
__device__ __forceinline__ void st_elem(uint16_t* p, long long i, float v) { p[i] = (uint16_t)f32_to_bf16_bits(v); }

// v + (v of another lane of the same 16-lane row), the partner chosen by a DPP control.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
    return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the wave, equal in every lane: four DPP steps give each lane its 16-lane row sum
// (quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror, row_mirror), then the four row
// sums are read with v_readlane and added in a fixed order.
__device__ __forceinline__ float wave_sum(float v) {
    v = dpp_add<0xB1>(v);
    v = dpp_add<0x4E>(v);
    v = dpp_add<0x141>(v);
    v = dpp_add<0x140>(v);
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ int wave_min(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = min(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ int wave_max(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = max(v, __shfl_xor(v, off, 64));
    return v;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) short4_t lds_short4;
typedef __attribute__((address_space(3))) void lds_void;

// ---------------------------------------------------------------- swizzled LDS tiles
// A tile holds 64 rows of DH bf16 without padding; row r's 16-byte chunk c is stored at chunk
// position  r * CPR + (c ^ swz(r)),  CPR = DH / 8.  LDS has 64 banks of 4 bytes; a 16-byte
// read (ds_read_b128) is served 16 lanes at a time and an 8-byte read (ds_read_b64_tr_b16)
// 32 lanes at a time.  swz depends on r mod 16 only and is chosen (per CPR, by exhaustive
// search over linear maps of the row bits) so that both operand patterns are conflict-free:
// 16 consecutive rows at one chunk (MFMA operand rows) and 4 consecutive rows x 4 adjacent
// chunks x 2 halves (the suppliers of one transposing read).
template <int CPR>
__device__ __forceinline__ int swz(int row) {
    if constexpr (CPR == 16 || CPR == 32) return ((row & 3) << 2) | ((row >> 2) & 3);
    else if constexpr (CPR == 8)
        return ((row >> 1) & 1) | (((row >> 2) & 1) << 1) | ((((row >> 1) ^ (row >> 3)) & 1) << 2);
    else return (row >> 2) & (CPR - 1);
}

template <int CPR>
__device__ __forceinline__ int tile_chunk(int row, int chunk) {
    return row * CPR + (chunk ^ swz<CPR>(row));
}

// 8 bf16 (16 bytes) of row `row`, logical chunk `chunk`.
template <int CPR>
__device__ __forceinline__ bf16x8 tile_read8(const uint16_t* tile, int row, int chunk) {
    return *(const bf16x8*)(tile + 8 * tile_chunk<CPR>(row, chunk));
}

// MFMA 32x32x16 operand read "down the columns" of a swizzled row-major bf16 tile with the
// transposing load ds_read_b64_tr_b16.  Lane l receives column c0 + (l % 32) and, in its 8
// k-slots, rows r0 + 4 (l / 32) + {0,1,2,3} (slots 0..3) and r0 + 8 + 4 (l / 32) + {0,1,2,3}
// (slots 4..7): the row order of the 32x32 accumulator layout, so P^T / dS^T taken from an
// accumulator pair with it slot for slot.  Within each 16-lane group, lane j = 4 s + q
// supplies row (.. + s), columns (.. + 4 q .. 4 q + 3); the hardware hands lane i of the group
// element i % 4 of supplier 4 s + i / 4 in slot s.  r0 is a multiple of 16, c0 of 32.
template <int CPR>
__device__ __forceinline__ bf16x8 tile_read_tr(const uint16_t* tile, int r0, int c0, int lane) {
    const int j = lane & 15;
    const int row = r0 + 4 * (lane >> 5) + (j >> 2);
    const int colx = c0 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const uint16_t* p0 = tile + 8 * tile_chunk<CPR>(row, colx >> 3) + (colx & 7);
    const uint16_t* p1 = tile + 8 * tile_chunk<CPR>(row + 8, colx >> 3) + (colx & 7);
    const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p0);
    const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)p1);
    const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// ---------------------------------------------------------------- global -> LDS copies
// global_load_lds_dwordx4 / _dword (lane l of one instruction lands at the LDS address in M0
// plus 16 l, resp. 4 l) are issued through inline asm: the compiler then neither inserts
// conservative "wait for every copy" counters before unrelated LDS reads nor sees the LDS
// writes, and the kernels order the copies themselves with wait_vmcnt + lds_barrier.  M0 is
// written only here (the kernels use no other M0 consumer).
__device__ __forceinline__ uint32_t lds_address(const void* p) {
    return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_void*)p);
}

// Pointer known to be equal in all lanes, moved to scalar registers.
template <class T>
__device__ __forceinline__ const T* uniform_ptr(const T* p) {
    const unsigned long long v = (unsigned long long)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const T*)(uintptr_t)(((unsigned long long)hi << 32) | lo);
}

// One copy instruction: source address = sbase (wave-uniform) + voff (per lane, bytes).
__device__ __forceinline__ void lds_dma16(uint32_t lds_base, const void* sbase, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :: "s"(lds_base), "v"(voff), "s"(sbase) : "memory");
}

// The same copy with the non-temporal hint: for data read once (the stored dS blocks), so that it
// does not displace reused tiles from the caches.
__device__ __forceinline__ void lds_dma16_nt(uint32_t lds_base, const void* sbase, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 nt"
                 :: "s"(lds_base), "v"(voff), "s"(sbase) : "memory");
}

__device__ __forceinline__ void lds_dma4(uint32_t lds_base, const void* sbase, uint32_t voff) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2"
                 :: "s"(lds_base), "v"(voff), "s"(sbase) : "memory");
}

// Wait until at most N vector-memory operations of this wave are outstanding; they complete
// in issue order, so everything issued before the last N has landed (copies included).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

__device__ __forceinline__ void wait_vmem() { wait_vmcnt<0>(); }

// The same wait as a real s_waitcnt instruction (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left at their maxima).  The compiler's own counter bookkeeping sees it, so
// loads it issued earlier (e.g. before a loop) are known complete afterwards and get no extra
// wait inside the loop, where such a wait would also cover the copies in flight.
template <int N>
__device__ __forceinline__ void wait_vmcnt_seen() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
    asm volatile("" ::: "memory");
}

// This wave's LDS operations (and scalar loads) have completed, as a real s_waitcnt that the
// compiler's counter bookkeeping sees: reads issued before it need no further wait.
__device__ __forceinline__ void wait_lgkm_seen() {
    __builtin_amdgcn_s_waitcnt(0xC07F);      // lgkmcnt(0); vmcnt and expcnt at their maxima
    asm volatile("" ::: "memory");
}

// lds_barrier with the LDS wait visible to the compiler (see wait_lgkm_seen).
__device__ __forceinline__ void lds_barrier_seen() {
    wait_lgkm_seen();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Workgroup barrier for LDS hand-offs: this wave's LDS reads and writes have completed, and
// no other wave passes until all waves arrive.  Copies into LDS must be waited for first.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Byte offset, within a swizzled tile, of 16-byte chunk `chunk` of row `row`.
template <int CPR>
__device__ __forceinline__ uint32_t tile_ofs(int row, int chunk) {
    return 16u * (uint32_t)tile_chunk<CPR>(row, chunk);
}

// Byte offsets of this lane's two ds_read_b64_tr_b16 supplier addresses for tile_read_tr with
// r0 = 0 and column block c0 (a multiple of 32).  Since the swizzle depends on the row modulo
// 16 only, the reads for row block r0 (a multiple of 16) are at these offsets plus
// r0 * CPR * 16 bytes.
template <int CPR>
__device__ __forceinline__ void tile_ofs_tr(int c0, int lane, uint32_t& o0, uint32_t& o1) {
    const int j = lane & 15;
    const int row = 4 * (lane >> 5) + (j >> 2);
    const int colx = c0 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    o0 = tile_ofs<CPR>(row, colx >> 3) + 2u * (uint32_t)(colx & 7);
    o1 = tile_ofs<CPR>(row + 8, colx >> 3) + 2u * (uint32_t)(colx & 7);
}

// 16 bytes at byte offset `off` of an LDS tile.
__device__ __forceinline__ bf16x8 lds_read16(const uint16_t* tile, uint32_t off) {
    return *(const bf16x8*)((const char*)tile + off);
}

// tile_read_tr from precomputed supplier offsets (o0, o1) plus a constant byte offset.
__device__ __forceinline__ bf16x8 lds_read_tr(const uint16_t* tile, uint32_t o0, uint32_t o1) {
    const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)((const char*)tile + o0));
    const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_short4*)((const char*)tile + o1));
    const short __attribute__((ext_vector_type(8))) v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Asynchronous copy of rows [row0, row0 + ROWS) of a [.., ld] bf16 matrix (columns col0 ..
// col0 + DH) into a swizzled tile.  Rows at or past `nrows` are replaced by row nrows - 1, a
// valid row whose values the mask or a zero multiplier neutralises; the caller guarantees
// row0 < nrows.  Instruction i of wave w of the 256-thread workgroup fills the 64 chunks
// (16 bytes each) of LDS block 4 i + w, i.e. tile rows RPI i + (64 / CPR) w + lane / CPR with
// RPI = 256 / CPR; when the tile has fewer than 256 chunks only the first waves issue.  A
// lane's row within the block is the same for every instruction, and so is its chunk when RPI
// is a multiple of 16 (the swizzle depends on row mod 16 only); with 32 chunks per row (RPI 8)
// the source chunk alternates between even and odd instructions.  Each instruction needs one
// wave-uniform base address and one per-lane 32-bit offset.  The caller guarantees
// ROWS * ld * 2 < 2^31.
//
// With CLAMP_COLS, columns at or past `ncols` (a multiple of 8, > col0) are replaced by the
// last valid 16-byte chunk of the row: the copy stays inside the matrix, and the tile columns
// past the edge hold values that the caller never stores.
template <int DH, int ROWS = 64, bool CLAMP_COLS = false, bool KEEP_OFFSETS = false>
__device__ __forceinline__ void tile_dma(uint16_t* tile, const uint16_t* base, long long ld, int row0,
                                         int nrows, int col0, int tid, int ncols = 0) {
    constexpr int CPR = DH / 8, RPI = 256 / CPR, NCH = ROWS * CPR;
    static_assert(NCH % 64 == 0, "whole LDS blocks");
    // The per-lane offsets are recomputed at every call (a few VALU instructions) rather than
    // hoisted out of the caller's loop, where they would hold VGPRs for the whole loop; with
    // KEEP_OFFSETS (a caller with registers to spare) the compiler may keep them.
    int lane = tid & 63;
    if constexpr (!KEEP_OFFSETS) asm volatile("" : "+v"(lane));
    const int w = tid >> 6;
    const int rl = w * (64 / CPR) + lane / CPR;             // row within block 0 of this wave
    // source chunk of the lane in instruction i (tile row i * RPI + rl)
    auto src_chunk = [&](int i) {
        const int c = (lane % CPR) ^ swz<CPR>(RPI % 16 == 0 ? rl : i * RPI + rl);
        if constexpr (CLAMP_COLS) return min(c, ((ncols - col0) >> 3) - 1);
        else return c;
    };
    const uint16_t* tbase = base + (long long)row0 * ld + col0;
    const uint32_t ltile = __builtin_amdgcn_readfirstlane(lds_address(tile) + (uint32_t)w * 1024u);
    if (NCH < 256 && w * 64 >= NCH) return;
    if (row0 + ROWS <= nrows) {
#pragma unroll
        for (int i = 0; i < (NCH + 255) / 256; i++) {
            const uint32_t voff = (uint32_t)(rl * ld + src_chunk(i) * 8) * 2u;
            lds_dma16(ltile + (uint32_t)i * 4096u, uniform_ptr(tbase + (long long)i * RPI * ld), voff);
        }
    } else {
        const int last = nrows - 1 - row0;                  // >= 0: the tile holds a valid row
#pragma unroll
        for (int i = 0; i < (NCH + 255) / 256; i++) {
            const uint32_t voff = (uint32_t)(min(i * RPI + rl, last) * ld + src_chunk(i) * 8) * 2u;
            lds_dma16(ltile + (uint32_t)i * 4096u, uniform_ptr(tbase), voff);
        }
    }
}

// tile_dma of the same rows and columns of two matrices into two tiles (the query unit's Q and
// dO): the per-lane row and chunk are derived once for both copies.
template <int DH, int ROWS>
__device__ __forceinline__ void tile_dma_pair(uint16_t* tile_a, const uint16_t* base_a, long long ld_a,
                                              uint16_t* tile_b, const uint16_t* base_b, long long ld_b,
                                              int row0, int nrows, int col0, int tid) {
    constexpr int CPR = DH / 8, RPI = 256 / CPR, NCH = ROWS * CPR;
    static_assert(NCH % 64 == 0, "whole LDS blocks");
    int lane = tid & 63;
    asm volatile("" : "+v"(lane));
    const int w = tid >> 6;
    const int rl = w * (64 / CPR) + lane / CPR;
    auto src_chunk = [&](int i) { return (lane % CPR) ^ swz<CPR>(RPI % 16 == 0 ? rl : i * RPI + rl); };
    const uint16_t* ta = base_a + (long long)row0 * ld_a + col0;
    const uint16_t* tb = base_b + (long long)row0 * ld_b + col0;
    const uint32_t la = __builtin_amdgcn_readfirstlane(lds_address(tile_a) + (uint32_t)w * 1024u);
    const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_address(tile_b) + (uint32_t)w * 1024u);
    if (NCH < 256 && w * 64 >= NCH) return;
    if (row0 + ROWS <= nrows) {
#pragma unroll
        for (int i = 0; i < (NCH + 255) / 256; i++) {
            const int c8 = src_chunk(i) * 8;
            lds_dma16(la + (uint32_t)i * 4096u, uniform_ptr(ta + (long long)i * RPI * ld_a),
                      (uint32_t)(rl * ld_a + c8) * 2u);
            lds_dma16(lb + (uint32_t)i * 4096u, uniform_ptr(tb + (long long)i * RPI * ld_b),
                      (uint32_t)(rl * ld_b + c8) * 2u);
        }
    } else {
        const int last = nrows - 1 - row0;                  // >= 0: the tile holds a valid row
#pragma unroll
        for (int i = 0; i < (NCH + 255) / 256; i++) {
            const int c8 = src_chunk(i) * 8, r = min(i * RPI + rl, last);
            lds_dma16(la + (uint32_t)i * 4096u, uniform_ptr(ta), (uint32_t)(r * ld_a + c8) * 2u);
            lds_dma16(lb + (uint32_t)i * 4096u, uniform_ptr(tb), (uint32_t)(r * ld_b + c8) * 2u);
        }
    }
}

// Timestamps and mask codes of N (at most 64) consecutive tokens into LDS (two 4-byte-per-lane
// copies issued by wave 0).  Tokens at or past `ntok` are copied from token ntok - 1
// (tok0 < ntok); the caller zeroes their codes once the copy has landed.
template <int N = 64>
__device__ __forceinline__ void codes_dma(int* dst_ts, int* dst_code, const int* ts, const int* code,
                                          int tok0, int ntok, int tid) {
    static_assert(N <= 64, "one wave");
    if (tid < N) {
        const uint32_t voff = (uint32_t)min(tid, ntok - 1 - tok0) * 4u;
        lds_dma4(lds_address(dst_ts), uniform_ptr(ts + tok0), voff);
        lds_dma4(lds_address(dst_code), uniform_ptr(code + tok0), voff);
    }
}

}  // namespace mtgr
