// Host-side internal declarations shared by the C-ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace mtgr {

// Arguments of every attention kernel (one struct, passed by value).
struct AttnArgs {
    const int* offsets;
    const int8_t* seg;
    const int* ts;
    const void* q;
    const void* k;
    const void* v;
    const float* rab;
    const void* dout;
    void* out;
    void* dq;
    void* dk;
    void* dv;
    float* drab;
    long long ld_q, ld_k, ld_v, ld_o;
    const int4* summ;     // [B][ntile] per-64-token tile summaries
    const int* tok_code;  // [T] per-token mask code (token_code of seg)
    const int2* items;    // work list: {user, (tile << 8) | head}, user < 0 = empty slot
    const long long* ds_off;  // [B+1] first stored-dS block of each user (H ceil(n_b/64)^2 blocks each)
    uint16_t* ds;             // stored dS: 64 x 64 bf16 blocks in the dK/dV kernel's fragment order
    int ntile;
    int heads;
    float alpha;
    int nbuckets;
    int cand_rows;            // forward: write candidate rows only
    // Cached forward (the query side above holds a request's candidates): the key side is a
    // caller-held cache of the users' user-side tokens, with its own layout and plan.
    const void* kc;
    const void* vc;
    long long ld_kc, ld_vc;
    const int* offsets_k;     // [B+1] cache offsets
    const int* ts_k;          // [Tc] cache timestamps
    const int* tok_code_k;    // [Tc] cache token codes (from the cache's plan)
    const int4* summ_k;       // [B][ntile_k] cache tile summaries (from the cache's plan)
    int ntile_k;
};

// Number of physical work-list slots for tiles of `bm` rows (see build_schedule).
long long schedule_slots(long long total_tokens, int num_users, int max_seqlen, int heads, int bm);

// Launchers; each returns the hipError_t of its launch.
hipError_t launch_tile_summaries(const int* offsets, const int8_t* seg, const int* ts, int num_users,
                                 int ntile, int4* summ, int* tok_code, hipStream_t s);
hipError_t launch_build_schedule(const int* offsets, int num_users, int heads, int bm, int2* items,
                                 int slots, int* sorted_users, hipStream_t s);
hipError_t launch_fill_f32(float* p, long long n, float value, hipStream_t s);

hipError_t launch_attn_fwd_bf16(const AttnArgs& a, int head_dim, int slots, hipStream_t s);
// Candidates of a request against the users' cached user-side keys (bf16, head_dim 32..128).
hipError_t launch_attn_fwd_cached_bf16(const AttnArgs& a, int head_dim, int slots, hipStream_t s);
hipError_t launch_attn_fwd_f32(const AttnArgs& a, int head_dim, int slots, hipStream_t s);
// Which backward kernels run (bf16).
struct BwdPlan {
    bool dkdv;          // dk/dv kernel (forms drab when a.drab is set)
    bool store_ds;      // ... also writes dS blocks to a.ds
    bool dq_from_ds;    // dq = alpha dS k from the stored blocks
    bool dq_recompute;  // dq kernel recomputing S, dP, dS (forms drab when a.drab is set)
};
constexpr size_t DS_BLOCK_BYTES = 64 * 64 * 2;   // one stored-dS block (64 keys x 64 queries bf16)

hipError_t launch_attn_bwd_bf16(const AttnArgs& a, int head_dim, int slots, const BwdPlan& plan,
                                hipStream_t s);
hipError_t launch_ds_offsets(const int* offsets, int num_users, int heads, long long* ds_off,
                             hipStream_t s);
// Vector-ALU backward: fp32 storage at any supported head_dim, or bf16 storage at head_dim 16.
hipError_t launch_attn_bwd_vec(const AttnArgs& a, bool bf16, int head_dim, int slots, bool dq, bool dkdv,
                               hipStream_t s);

struct GlnArgs {
    long long T;
    int d;
    int G;
    float eps;
    long long ld_x, ld_u, ld_y;
    const void* x;
    const void* u;
    const int8_t* gid;
    const float* gamma;
    const float* beta;
    void* y;
    float* mean;
    float* rstd;
    const void* dy;
    void* dx;
    void* du;
    float* dgamma;
    float* dbeta;
    float* workspace;   // backward: per-workgroup dgamma/dbeta partials
};

constexpr int GLN_BWD_SLOTS = 256;            // target workgroups of the backward (one per CU)
constexpr int GLN_LDS_ACC_BYTES = 64 * 1024;  // largest per-workgroup accumulator kept in LDS
void gln_bwd_partition(long long T, int* nslots, int* tokens_per_wave);
size_t gln_bwd_workspace_bytes(long long T, int d, int G);

hipError_t launch_gln_fwd(const GlnArgs& a, bool bf16, hipStream_t s);
hipError_t launch_gln_bwd(const GlnArgs& a, bool bf16, hipStream_t s);

constexpr int ATTN_TILE_BF16 = 128;   // query / key rows per work item, bf16 kernels
constexpr int ATTN_TILE_F32 = 64;     // rows per work item, vector-ALU kernels (fp32, bf16 at dh 16)
constexpr int SCHED_BUCKETS = 4096;   // length buckets of the heavy-first sort
constexpr int XCDS = 8;               // accelerator complex dies of an MI355X

// Bias + SiLU of the encoder layer's projection: out = silu(h + bias), or with `backward`
// out = g * silu'(h + bias).  [rows, cols] with row strides; bias [cols] fp32 or NULL.
hipError_t launch_bias_silu(long long rows, int cols, bool bf16, bool backward, const void* h, long long ld_h,
                            const float* bias, const void* g, long long ld_g, void* out, long long ld_out,
                            hipStream_t s);

// Dense bf16 products of the encoder layer (gemm.hip).
constexpr int GEMM_NN = 0, GEMM_NT = 1, GEMM_TN = 2;
constexpr int GEMM_EPI_NONE = 0, GEMM_EPI_BIAS_SILU = 1, GEMM_EPI_BIAS_RESIDUAL = 2;
struct GemmArgs {
    int layout, epilogue;
    long long M, N, K;
    const void* A;
    long long lda;
    const void* B;
    long long ldb;
    void* C;
    long long ldc;
    void* C2;                 // BIAS_SILU: the activation
    long long ldc2;
    const void* R;            // BIAS_RESIDUAL: the residual
    long long ldr;
    const float* bias;        // [N] fp32
    float* colsum;            // TN: [N] column sums of B, or NULL
    float* partial;           // TN: [splits][M][N] fp32 workspace
    float* colsum_partial;    // TN: [splits][N] fp32 workspace
    int mblocks, nblocks, splits, ks_per_split;
};
hipError_t launch_clock_probe(int iters, int blocks, long long* out, hipStream_t s);
void gemm_plan(int layout, long long M, long long N, long long K, int* mblocks, int* nblocks, int* splits,
               int* ks_per_split);
size_t gemm_workspace_bytes(int layout, long long M, long long N, long long K);
hipError_t launch_gemm_bf16(const GemmArgs& g, hipStream_t s);

// Elementwise out = a + b (bf16 or fp32) on [rows, cols] with row strides.
hipError_t launch_add(long long rows, int cols, bool bf16, const void* a, long long lda, const void* b,
                      long long ldb, void* out, long long ldo, hipStream_t s);

// Debug validation of a jagged batch: `first` (VALIDATE_CONDITIONS 64-bit slots of device
// memory) receives per condition the smallest failing index, ~0 if none.
constexpr int VALIDATE_CONDITIONS = 6;
hipError_t launch_validate(const int* offsets, int num_users, long long total, int max_seqlen,
                           const int8_t* seg, const int8_t* group_ids, int groups,
                           unsigned long long* first, hipStream_t s);

// Dynamic embedding table (see include/mtgr_embedding.h): the table descriptor as the
// kernels take it.
struct EmbArgs {
    long long key_capacity;   // power of two
    int row_capacity;
    int dim;
    int esize;                // bytes per value element: 2 (bf16) or 4 (fp32)
    uint64_t* keys;
    int* key_rows;
    void* values;
    uint32_t* counts;
    int* last_ts;
    int* free_rows;
    int* state;
};
size_t dedup_set_capacity(long long n);
size_t dedup_workspace_bytes(long long n);
size_t lookup_workspace_bytes(long long n_max);
hipError_t launch_emb_init(const EmbArgs& t, hipStream_t s);
hipError_t launch_emb_dedup(long long n, const uint64_t* ids, uint64_t* unique, int* occ, int* inverse,
                            long long* num_unique, void* ws, hipStream_t s);
hipError_t launch_emb_lookup(const EmbArgs& t, long long n_max, const uint64_t* unique, const int* occ,
                             const long long* num_unique, int now, int insert, int* rows, void* ws,
                             hipStream_t s);
hipError_t launch_emb_gather(const EmbArgs& t, long long n, const int* inverse, const int* rows, void* out,
                             long long ld_out, hipStream_t s);
size_t sgd_workspace_bytes(long long n, long long n_max, int dim);
hipError_t launch_emb_sgd(const EmbArgs& t, long long n, const int* inverse, const int* occ, const void* grad,
                          long long ld_grad, long long n_max, const int* rows, const long long* num_unique,
                          float lr, void* ws, hipStream_t s);
hipError_t launch_emb_evict(const EmbArgs& t, int threshold, uint32_t min_count, long long* num_evicted,
                            hipStream_t s);
hipError_t launch_emb_rehash(const EmbArgs& from, const EmbArgs& to, hipStream_t s);

}  // namespace mtgr
