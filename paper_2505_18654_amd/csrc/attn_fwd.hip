// Forward of the jagged dynamic-mask SiLU attention (Eq. 5, Sec. 4.2).
//
// bf16 kernel: one workgroup = 4 waves = 128 query rows of one (user, head); each wave owns
// 32 query rows and walks the user's 64-key tiles that are not fully masked, 32 keys (one
// "half") at a time.  Per half each wave computes
//     S^T (32 keys x 32 queries) = K Q^T          v_mfma_f32_32x32x16_bf16, Q held in VGPRs
//     P' = silu(alpha S + rab) * (alpha or 1)^-1, masked     in registers
//     O^T (dh x 32 queries)     += V^T P'^T        V^T read with ds_read_b64_tr_b16
// and O is scaled once by alpha / n_b (1 / n_b with a relative bias) at the end.  Computing
// the transposed products lets the accumulator layout of S^T (lane = query column, registers
// = keys) serve directly as the B operand of the second product, so P never goes through LDS,
// and the transposing LDS read gives V^T without a transposed copy.  The mask is evaluated
// only on PARTIAL tiles.
//
// Software pipeline: while a wave turns S of one half into P' (VALU and transcendental work)
// it issues, one by one in between, the MFMAs of the NEXT half's S and of the current half's
// P'V product, so the matrix cores and the vector ALUs of a wave run side by side (a wave's
// MFMA and VALU instructions overlap; separate waves doing one each barely do on gfx950).
// K runs one tile ahead of V in two LDS buffers each, filled straight from global memory
// (global_load_lds) about one tile before use; two barriers per tile.
#include <type_traits>

#include "mtgr_device.h"
#include "mtgr_internal.h"

#ifndef MTGR_FWD_PF
#define MTGR_FWD_PF 3
#endif
#ifndef MTGR_FWD_SB
#define MTGR_FWD_SB 4
#endif
#ifndef MTGR_FWD_SGB
#define MTGR_FWD_SGB 0
#endif
#ifndef MTGR_FWD_SGB_DS
#define MTGR_FWD_SGB_DS 2
#endif

namespace mtgr {

namespace {

constexpr int BM = 128;   // query rows per workgroup
constexpr int BN = 64;    // keys per tile

__device__ __forceinline__ uint4 ldg16(const uint16_t* p) { return *(const uint4*)p; }

}  // namespace

// CACHED: the query rows are a request's candidates (a.q, a.offsets, a.seg, a.ts, a.summ) and the
// keys are the users' cached user-side tokens (a.kc, a.vc, a.offsets_k, a.ts_k, a.tok_code_k,
// a.summ_k).  Candidates see only user-side keys and themselves (Sec. 4.2), so no key tile holds
// a candidate; each candidate's own term p_ii v_i is added after the tiles, and n_b counts both
// sides.
//
// Masking.  Masked scores are replaced before the SiLU by a value whose P' is exactly zero, in
// a pass of their own on PARTIAL tiles, so that one epilogue serves every tile: 0 without a
// relative bias (silu(0) = 0); with a bias, -1e30 / alpha, so that alpha s + rab is about -1e30,
// the sigmoid 0 and P'' = y * 0 (the host requires |alpha| >= 1e-7 and finite bias values
// far below 1e29 for it).  RSEL instead selects P' = 0 element by element in the epilogue (a
// second epilogue path): the host picks it for a bias with |alpha| < 1e-7.
template <int DH, bool RAB, bool CACHED, bool RSEL>
__global__ __launch_bounds__(256, 2) void attn_fwd_bf16_kernel(AttnArgs a) {
    constexpr int CPR = DH / 8;          // 16-byte chunks per row
    constexpr int KSTEPS = DH / 16;      // k-steps of S^T = K Q^T per 32-key half
    constexpr int DBLK = DH / 32;        // 32-row blocks of O^T (MFMAs per 16-key PV step)
    constexpr int TILE = BN * DH;        // elements of one 64-row tile
    constexpr int NM = 2 * DBLK + KSTEPS;   // MFMA slots of one half-step
    constexpr int EPM = 16 / NM;         // P' elements computed per slot
    static_assert(NM * EPM == 16, "slot plan");
    constexpr int NK = DH / 32;          // LDS-DMA instructions per wave for one tile
    constexpr int PF = MTGR_FWD_PF;      // operand prefetch distance in MFMA slots
    constexpr int SB = MTGR_FWD_SB;      // MFMA slots per scheduling region

    __shared__ __align__(16) uint16_t sK[2][TILE];
    __shared__ __align__(16) uint16_t sV[2][TILE];
    __shared__ int sVts[2][BN];          // timestamps / mask codes travel with the V tile
    __shared__ int sVcode[2][BN];
    __shared__ __align__(16) long long sVthr[2][BN];   // key_threshold of each key of the tile
    __shared__ float sRab[MTGR_RAB_LDS];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;        // query rows of the user
    int okb = ob, nkb = nb;                                          // key rows of the user
    if constexpr (CACHED) {
        okb = a.offsets_k[b];
        nkb = a.offsets_k[b + 1] - okb;
    }
    const int q0 = qt * BM;
    const int ntq = (nb + BN - 1) / BN;
    const int ntk = (nkb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)(CACHED ? nb + nkb : nb);
    const float alpha = a.alpha;
    const int4* summ = a.summ + (long long)b * a.ntile;
    const int4* summk = CACHED ? a.summ_k + (long long)b * a.ntile_k : summ;

    TileSummary sq = load_summary(summ, 2 * qt);
    if (2 * qt + 1 < ntq) sq = combine(sq, load_summary(summ, 2 * qt + 1));
    if (a.cand_rows && !(sq.flags & TS_ANY_CAND)) return;   // no candidate row to form

    const int col = lane & 31, hh = lane >> 5;
    const int qi = q0 + w * 32 + col;
    const bool qvalid = qi < nb;
    int qcode = 0, qts = 0;
    if (qvalid) {
        qcode = token_code(a.seg[ob + qi]);
        qts = a.ts[ob + qi];
    }
    const long long ldk = CACHED ? a.ld_kc : a.ld_k, ldv = CACHED ? a.ld_vc : a.ld_v;
    const uint16_t* Kb = (const uint16_t*)(CACHED ? a.kc : a.k) + (long long)okb * ldk;
    const uint16_t* Vb = (const uint16_t*)(CACHED ? a.vc : a.v) + (long long)okb * ldv;
    const int* kts_g = (CACHED ? a.ts_k : a.ts) + okb;
    const int* kcode_g = (CACHED ? a.tok_code_k : a.tok_code) + okb;
    const uint16_t* Qb = (const uint16_t*)a.q + (long long)ob * a.ld_q;
    bf16x8 qreg[KSTEPS];
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? NEG_LOG2E * a.rab[h * a.nbuckets + tid] : 0.f;

    // Per-lane LDS byte offsets of the MFMA operands, shared by every tile and buffer: the
    // K operand of k-step kk (row col, chunk 2 kk + hh; rows 32..63 add 32 * CPR * 16 bytes)
    // and the two transposing-read supplier addresses of V^T column block db (row blocks of
    // 16 keys add 16 * CPR * 16 bytes).  The swizzle XORs the chunk index with a per-row
    // constant, and a row's chunks fill an aligned block of CPR * 16 bytes, so the offset of
    // k-step kk is that of k-step 0 XOR 32 kk, and that of column block db the one of block 0
    // XOR 64 db: three live registers instead of KSTEPS + 2 DBLK.
    uint32_t kofs0 = tile_ofs<CPR>(col, hh), vofs0 = 0, vofs1 = 0;
    tile_ofs_tr<CPR>(0, lane, vofs0, vofs1);
    constexpr uint32_t ROW16 = 16u * CPR * 16u;   // bytes of 16 tile rows

    floatx16 oacc[DBLK];
#pragma unroll
    for (int i = 0; i < DBLK; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) oacc[i][r] = 0.f;

    auto class_of = [&](int t) {
        const bool overlap = !CACHED && (t * BN < q0 + BM) && (q0 < t * BN + BN);
        return tile_class(sq, load_summary(summk, t), overlap);
    };
    TileWalker<decltype(class_of)> walk(class_of, ntk);

    // The copies' per-lane offsets are loop invariants kept in registers, except in the
    // select-masked bias instantiation (256 VGPRs).
    auto issue_k = [&](int t, int buf) { tile_dma<DH, 64, false, !RSEL>(sK[buf], Kb, ldk, t * BN, nkb, h * DH, tid); };
    auto issue_v = [&](int t, int buf) {
        tile_dma<DH, 64, false, !RSEL>(sV[buf], Vb, ldv, t * BN, nkb, h * DH, tid);
        codes_dma(sVts[buf], sVcode[buf], kts_g, kcode_g, t * BN, nkb, tid);
    };

    // p' for the accumulator value sv of key kl (relative to the tile):
    // silu(alpha s) / alpha = s / (1 + 2^(-alpha s log2 e)), or with a relative bias
    // -log2(e) silu(alpha s + rab) = y / (1 + 2^y), y = -log2(e) (alpha s + rab) (the table in LDS
    // holds -log2(e) rab).
    const float c_exp = -1.4426950408889634f * alpha;
    // qrel = qi - (first key of the tile) - 4 hh; the key of element e of half HC is the
    // tile's key 32 HC + 8 (e / 4) + 4 hh + e % 4, so the diagonal test compares qrel with a
    // compile-time constant.
    auto p_of = [&](auto masked_tag, float sv, int kl, int kc, const int* kts, const int* kcode, int qrel) {
        constexpr bool MASKED = decltype(masked_tag)::value;
        float p;
        if (RAB) {
            float sg;
            p = silu_scaled(__builtin_fmaf(sv, c_exp, sRab[rab_bucket(qts, kts[kl], a.nbuckets)]), sg);
        } else {
            p = sv * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(sv * c_exp));
        }
        if (MASKED) p = visible_diag(qcode, qts, kcode[kl], kts[kl], qrel == kc) ? p : 0.f;
        return p;
    };

    // One half-step.  Consumes S of the current half (`cur`, keys 32 HC .. 32 HC + 31 of the
    // tile in V buffer VB), adds its first 16 keys' P'V to O, and leaves the packed P' of its
    // last 16 keys in pk_out (their PV MFMAs are issued by the caller: carried into the next
    // half-step or flushed).  With CARRY it first issues the carried PV MFMAs of keys 16 .. 31
    // (pk_in) of the same tile; with HAS_NEXT it computes the next half's S into `nxt` from
    // rows 32 HN .. 32 HN + 31 of K buffer KB.  Buffer indices and halves are compile-time
    // constants, so every LDS address is a per-lane base plus an immediate offset.  MFMA slot
    // m (in issue order):
    //   [0, DBLK)                       carried PV (k-step 1 of half 0)
    //   [DBLK, DBLK + KSTEPS/2)         next S, k-steps 0 .. KSTEPS/2 - 1
    //   [DBLK + KSTEPS/2, 2 DBLK + ...) PV of keys 32 HC .. 32 HC + 15
    //   [2 DBLK + KSTEPS/2, NM)         next S, remaining k-steps
    // and slot m first computes P' elements m EPM .. m EPM + EPM - 1 (registers of `cur`).
    auto half_step = [&](auto carry_tag, auto next_tag, auto masked_tag, auto vb_tag, auto hc_tag,
                         auto kb_tag, auto hn_tag, const floatx16& cur, floatx16& nxt,
                         const uint32_t* pk_in, uint32_t* pk_out, int qrel) {
        constexpr bool CARRY = decltype(carry_tag)::value;
        constexpr bool HAS_NEXT = decltype(next_tag)::value;
        constexpr int VB = decltype(vb_tag)::value, HC = decltype(hc_tag)::value;
        constexpr int KB = decltype(kb_tag)::value, HN = decltype(hn_tag)::value;
        const uint16_t* Vc = sV[VB];
        const uint16_t* Kn = sK[KB];
        // The XOR-derived operand offsets are loop invariants that the compiler keeps in registers
        // (16 reads' worth for 3 more VGPRs: 64 VALU instructions fewer per two tiles).  The
        // select-masked bias instantiation, at 256 VGPRs, derives them afresh in every half-step
        // (one XOR per read) instead: kept live there, they spill.
        uint32_t kb0 = kofs0, vb0 = vofs0, vb1 = vofs1;
        if constexpr (RSEL) asm volatile("" : "+v"(kb0), "+v"(vb0), "+v"(vb1));
        auto kofs = [&](int kk) { return kb0 ^ (32u * (uint32_t)kk); };
        const int* kts = sVts[VB];
        const int* kcode = sVcode[VB];
        uint32_t pk0[4];
        float pv[16];
        auto active = [&](int m) {
            if (m < DBLK) return CARRY;
            if (m < DBLK + KSTEPS / 2) return HAS_NEXT;
            if (m < 2 * DBLK + KSTEPS / 2) return true;
            return HAS_NEXT;
        };
        auto operand = [&](int m) {
            if (m < DBLK) return lds_read_tr(Vc, (vb0 ^ (64u * m)) + ROW16, (vb1 ^ (64u * m)) + ROW16);
            if (m < DBLK + KSTEPS / 2) return lds_read16(Kn, kofs(m - DBLK) + 2 * HN * ROW16);
            if (m < 2 * DBLK + KSTEPS / 2) {
                const uint32_t db = m - DBLK - KSTEPS / 2;
                return lds_read_tr(Vc, (vb0 ^ (64u * db)) + 2 * HC * ROW16, (vb1 ^ (64u * db)) + 2 * HC * ROW16);
            }
            return lds_read16(Kn, kofs(m - 2 * DBLK) + 2 * HN * ROW16);
        };
        bf16x8 op[NM];
#pragma unroll
        for (int m = 0; m < PF && m < NM; m++)
            if (active(m)) op[m] = operand(m);
#pragma unroll
        for (int m = 0; m < NM; m++) {
            if (m + PF < NM && active(m + PF)) op[m + PF] = operand(m + PF);   // PF slots ahead
#pragma unroll
            for (int e = m * EPM; e < m * EPM + EPM; e++) {
                const int kc = 32 * HC + 8 * (e >> 2) + (e & 3);
                pv[e] = p_of(masked_tag, cur[e], kc + 4 * hh, kc, kts, kcode, qrel);
                if (e & 1) {
                    const uint32_t pp = pack_bf16x2(pv[e - 1], pv[e]);
                    if (e < 8) pk0[e >> 1] = pp; else pk_out[(e - 8) >> 1] = pp;
                }
            }
            if (m < DBLK) {
                if (CARRY) {
                    const bf16x8 pb = as_bf16x8(make_uint4(pk_in[0], pk_in[1], pk_in[2], pk_in[3]));
                    oacc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[m], pb, oacc[m], 0, 0, 0);
                }
            } else if (m < DBLK + KSTEPS / 2) {
                if (HAS_NEXT) {
                    const int kk = m - DBLK;
                    nxt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[m], qreg[kk], kk == 0 ? floatx16{} : nxt, 0, 0, 0);
                }
            } else if (m < 2 * DBLK + KSTEPS / 2) {
                const int db = m - DBLK - KSTEPS / 2;
                const bf16x8 pb = as_bf16x8(make_uint4(pk0[0], pk0[1], pk0[2], pk0[3]));
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[m], pb, oacc[db], 0, 0, 0);
            } else {
                if (HAS_NEXT) {
                    const int kk = m - 2 * DBLK;
                    nxt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(op[m], qreg[kk], nxt, 0, 0, 0);
                }
            }
            if constexpr (MTGR_FWD_SGB == 0) {
                if ((m + 1) % SB == 0) __builtin_amdgcn_sched_barrier(0);   // scheduling region
            }
        }
        if constexpr (MTGR_FWD_SGB > 0) {
            // one scheduling region per half-step, laid out as NM groups of
            // {1 MFMA, SGB VALU, SGB_DS LDS reads}
#pragma unroll
            for (int m = 0; m < NM; m++) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, MTGR_FWD_SGB, 0);
                __builtin_amdgcn_sched_group_barrier(0x100, MTGR_FWD_SGB_DS, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // Masked scores replaced by s_masked before the SiLU (see the kernel's comment).
    constexpr bool SMASK = !RAB || !RSEL;
    const float s_masked = RAB ? -1e30f / alpha : 0.f;
    const long long qv = query_value(qcode, qts);
    auto premask = [&](floatx16& cur, auto hc_tag, const long long* thr, int qrel) {
        constexpr int HC = decltype(hc_tag)::value;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int kc = 32 * HC + 8 * (e >> 2) + (e & 3);
            const int kl = kc + 4 * hh;
            cur[e] = (qv >= thr[kl] || qrel == kc) ? cur[e] : s_masked;
        }
    };
    using C0 = std::integral_constant<int, 0>;
    using C1 = std::integral_constant<int, 1>;
    using T = std::true_type;
    using F = std::false_type;

    int cls0, cls1 = TILE_MASKED;
    int t0 = walk.next(0, &cls0);                                // t_i
    int t1 = t0 < ntk ? walk.next(t0 + 1, &cls1) : ntk;          // t_{i+1}
    // The workgroup's 128 query rows come in as two tiles, through the buffers of K(t_{i+1}) and
    // V(t_{i+1}) (copied later): whole rows per copy instruction, where per-lane loads of each
    // lane's operand chunks touched 32 rows per instruction (the forward took 12 % longer).
    // Rows past the user's end are copies of its last row; their lanes use zeros.
    tile_dma<DH>(sK[1], Qb, a.ld_q, q0, nb, h * DH, tid);
    if (q0 + BN < nb) tile_dma<DH>(sV[1], Qb, a.ld_q, q0 + BN, nb, h * DH, tid);
    if (t0 < ntk) {
        issue_k(t0, 0);
        issue_v(t0, 0);
    }
    wait_vmcnt_seen<0>();                                        // Q, K, V, codes
    lds_barrier();
    {
        const uint16_t* sQ = w < 2 ? sK[1] : sV[1];
#pragma unroll
        for (int kk = 0; kk < KSTEPS; kk++) {
            const bf16x8 v = tile_read8<CPR>(sQ, 32 * (w & 1) + col, 2 * kk + hh);
            qreg[kk] = qvalid ? v : bf16x8{};
        }
    }
    wait_lgkm_seen();
    lds_barrier();                                               // every wave holds its Q
    if (t0 < ntk) {
        if (t1 < ntk) issue_k(t1, 1);
        floatx16 sA, sB;                                         // S(t_i, keys 0..31) in sA
#pragma unroll
        for (int kk = 0; kk < KSTEPS; kk++)
            sA = __builtin_amdgcn_mfma_f32_32x32x16_bf16(lds_read16(sK[0], kofs0 ^ (32u * kk)), qreg[kk],
                                                        kk == 0 ? floatx16{} : sA, 0, 0, 0);
        // Tile t_i, whose K and V sit in buffers P (the tile loop is unrolled by two so that P
        // is a compile-time constant).  Returns false after the last tile.
        auto tile = [&](auto par) {
            constexpr int P = decltype(par)::value;
            using CP = std::integral_constant<int, P>;
            using CQ = std::integral_constant<int, P ^ 1>;
            // top: V(t_i) (and its codes) landed; K(t_{i+1}) may still be in flight
            if (t1 < ntk) wait_vmcnt<NK>(); else wait_vmem();
            if (tid < BN) {
                // padded keys get code 0; every key gets its visibility threshold
                int c = sVcode[P][tid];
                if (t0 * BN + tid >= nkb) sVcode[P][tid] = c = 0;
                sVthr[P][tid] = key_threshold(c, sVts[P][tid]);
            }
            lds_barrier();
            if (t1 < ntk) issue_v(t1, P ^ 1);                      // V(t_{i-1})'s buffer
            const bool partial = cls0 == TILE_PARTIAL;
            // (cached: no key is the query itself, so the diagonal test never holds)
            const int qrel = CACHED ? -(1 << 20) : qi - t0 * BN - 4 * hh;
            uint32_t pkA[4], pkB[4];
            // half 0 of t_i; next S = half 1 of t_i (same K buffer)
            if (SMASK && partial) premask(sA, C0{}, sVthr[P], qrel);
            if (!SMASK && partial)
                half_step(F{}, T{}, T{}, CP{}, C0{}, CP{}, C1{}, sA, sB, pkA, pkA, qrel);
            else
                half_step(F{}, T{}, F{}, CP{}, C0{}, CP{}, C1{}, sA, sB, pkA, pkA, qrel);
            int cls2 = TILE_MASKED;
            int t2 = ntk;
            if (t1 < ntk) {
                // middle: K(t_{i+1}) landed everywhere and K(t_i) is no longer read -> K(t_{i+2})
                if (w == 0) wait_vmcnt<NK + 2>(); else wait_vmcnt<NK>();
                lds_barrier();
                t2 = walk.next(t1 + 1, &cls2);
                if (t2 < ntk) issue_k(t2, P);
            }
            // half 1 of t_i; next S = half 0 of t_{i+1}.  After the last tile that S is formed
            // from the idle K buffer (no copy is in flight into it) and never used: one code
            // path for every tile keeps the O accumulators in one set of registers.
            if (SMASK && partial) premask(sB, C1{}, sVthr[P], qrel);
            if (!SMASK && partial)
                half_step(T{}, T{}, T{}, CP{}, C1{}, CQ{}, C0{}, sB, sA, pkA, pkB, qrel);
            else
                half_step(T{}, T{}, F{}, CP{}, C1{}, CQ{}, C0{}, sB, sA, pkA, pkB, qrel);
            // PV of keys 48 .. 63
            const bf16x8 pb = as_bf16x8(make_uint4(pkB[0], pkB[1], pkB[2], pkB[3]));
#pragma unroll
            for (int db = 0; db < DBLK; db++)
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    lds_read_tr(sV[P], (vofs0 ^ (64u * db)) + 3 * ROW16, (vofs1 ^ (64u * db)) + 3 * ROW16), pb,
                    oacc[db], 0, 0, 0);
            const bool more = t1 < ntk;
            t0 = t1;
            cls0 = cls1;
            t1 = t2;
            cls1 = cls2;
            return more;
        };
        while (tile(C0{}) && tile(C1{})) {
        }
        __syncthreads();                                         // K buffers are reused below
    }

    if constexpr (CACHED) {
        // The candidate's own term: p_ii v_i with s_ii = q_i . k_i (bias bucket 0), p rounded
        // to bf16 as the tiles round P.  Lane (col, hh) holds features 16 kk + 8 hh .. + 7 of q
        // in qreg, and O^T rows 32 db + 8 g + 4 hh + 0..3.
        float dot = 0.f;
        if (qvalid) {
            const uint16_t* Kq = (const uint16_t*)a.k + (long long)(ob + qi) * a.ld_k + h * DH + 8 * hh;
#pragma unroll
            for (int kk = 0; kk < KSTEPS; kk++) {
                const uint4 kv = ldg16(Kq + 16 * kk);
                const uint4 qv = __builtin_bit_cast(uint4, qreg[kk]);
                const uint32_t kw[4] = {kv.x, kv.y, kv.z, kv.w}, qw[4] = {qv.x, qv.y, qv.z, qv.w};
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    dot = __builtin_fmaf(__uint_as_float(qw[i] << 16), __uint_as_float(kw[i] << 16), dot);
                    dot = __builtin_fmaf(__uint_as_float(qw[i] & 0xffff0000u), __uint_as_float(kw[i] & 0xffff0000u), dot);
                }
            }
        }
        dot += __shfl_xor(dot, 32, 64);   // the other 8 features of every k-step
        float p;
        if (RAB) {
            float sg;
            p = silu_scaled(__builtin_fmaf(dot, c_exp, sRab[0]), sg);
        } else {
            p = dot * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(dot * c_exp));
        }
        p = __uint_as_float(f32_to_bf16_bits(p) << 16);
        if (qvalid) {
            const uint16_t* Vq = (const uint16_t*)a.v + (long long)(ob + qi) * a.ld_v + h * DH + 4 * hh;
#pragma unroll
            for (int db = 0; db < DBLK; db++)
#pragma unroll
                for (int g = 0; g < 4; g++) {
                    const uint2 vv = *(const uint2*)(Vq + 32 * db + 8 * g);
                    oacc[db][4 * g + 0] = __builtin_fmaf(p, __uint_as_float(vv.x << 16), oacc[db][4 * g + 0]);
                    oacc[db][4 * g + 1] = __builtin_fmaf(p, __uint_as_float(vv.x & 0xffff0000u), oacc[db][4 * g + 1]);
                    oacc[db][4 * g + 2] = __builtin_fmaf(p, __uint_as_float(vv.y << 16), oacc[db][4 * g + 2]);
                    oacc[db][4 * g + 3] = __builtin_fmaf(p, __uint_as_float(vv.y & 0xffff0000u), oacc[db][4 * g + 3]);
                }
        }
    }

    // Output: O^T accumulators scaled by alpha / n_b (-ln 2 / n_b with a relative bias) -> bf16
    // rows of this wave staged in LDS (swizzled 32-row tile inside the K buffers) -> 16-byte
    // coalesced stores.
    const float oscale = RAB ? NEG_LN2 * inv_n : alpha * inv_n;
    uint16_t* sO = sK[w >> 1] + (w & 1) * 32 * DH;
#pragma unroll
    for (int db = 0; db < DBLK; db++) {
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int d = 32 * db + 8 * g + 4 * hh;
            *(uint2*)&sO[8 * tile_chunk<CPR>(col, d >> 3) + (d & 7)] =
                make_uint2(pack_bf16x2(oacc[db][4 * g + 0] * oscale, oacc[db][4 * g + 1] * oscale),
                           pack_bf16x2(oacc[db][4 * g + 2] * oscale, oacc[db][4 * g + 3] * oscale));
        }
    }
    __syncthreads();
    uint16_t* O = (uint16_t*)a.out;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; i++) {
        const int c = lane + 64 * i, row = c / CPR, cc = c % CPR;
        const int qr = q0 + w * 32 + row;
        if (qr < nb && (!a.cand_rows || a.seg[ob + qr] == SEG_CAND))
            store_nt16(O + (long long)(ob + qr) * a.ld_o + h * DH + cc * 8, &sO[8 * tile_chunk<CPR>(row, cc)]);
    }
}

// Vector-ALU kernel (fp32 storage, the parity mode; or bf16 storage at head_dim 16, where a
// pair holds 64 flop of products against the SiLU's transcendental work, so matrix cores would
// not pay): 64 query rows per workgroup, 4 threads per row each owning dh/4 features; keys
// staged 32 at a time in LDS as fp32; plain FMA loops in fp32.
template <int DH, bool RAB, class E>
__global__ __launch_bounds__(256) void attn_fwd_vec_kernel(AttnArgs a) {
    constexpr int BMF = 64, SUB = 32, Q4 = DH / 4, KP = DH + 1;
    __shared__ float sK[SUB * KP];
    __shared__ float sV[SUB * KP];
    __shared__ int sKcode[SUB];
    __shared__ int sKts[SUB];
    __shared__ float sRab[MTGR_RAB_LDS];
    const int tid = threadIdx.x;
    const int2 item = a.items[blockIdx.x];
    if (item.x < 0) return;
    const int b = item.x, qt = item.y >> 8, h = item.y & 255;
    const int ob = a.offsets[b], nb = a.offsets[b + 1] - ob;
    const int q0 = qt * BMF;
    const int ntk = (nb + BN - 1) / BN;
    const float inv_n = 1.0f / (float)nb;
    const int4* summ = a.summ + (long long)b * a.ntile;
    const TileSummary sq = load_summary(summ, qt);
    if (a.cand_rows && !(sq.flags & TS_ANY_CAND)) return;   // no candidate row to form

    const int qi = q0 + (tid >> 2), part = tid & 3;
    const bool qvalid = qi < nb;
    int qcode = 0, qts = 0;
    const E* Q = (const E*)a.q;
    const E* K = (const E*)a.k;
    const E* V = (const E*)a.v;
    float qv[Q4], ov[Q4];
#pragma unroll
    for (int c = 0; c < Q4; c++) {
        qv[c] = qvalid ? ld_elem(Q, (long long)(ob + qi) * a.ld_q + h * DH + part * Q4 + c) : 0.f;
        ov[c] = 0.f;
    }
    if (qvalid) {
        qcode = token_code(a.seg[ob + qi]);
        qts = a.ts[ob + qi];
    }
    if (RAB && tid < MTGR_RAB_LDS) sRab[tid] = tid < a.nbuckets ? a.rab[h * a.nbuckets + tid] : 0.f;

    for (int t = 0; t < ntk; t++) {
        const bool overlap = (t * BN < q0 + BMF) && (q0 < t * BN + BN);
        const int cls = tile_class(sq, load_summary(summ, t), overlap);
        if (cls == TILE_MASKED) continue;
        for (int sub = 0; sub < BN / SUB; sub++) {
            const int kb = t * BN + sub * SUB;
            __syncthreads();
            for (int i = tid; i < SUB * DH; i += 256) {
                const int row = i / DH, c = i % DH, key = kb + row;
                sK[row * KP + c] = key < nb ? ld_elem(K, (long long)(ob + key) * a.ld_k + h * DH + c) : 0.f;
                sV[row * KP + c] = key < nb ? ld_elem(V, (long long)(ob + key) * a.ld_v + h * DH + c) : 0.f;
            }
            if (tid < SUB) {
                const int key = kb + tid;
                sKcode[tid] = key < nb ? token_code(a.seg[ob + key]) : 0;
                sKts[tid] = key < nb ? a.ts[ob + key] : 0;
            }
            __syncthreads();
            for (int j = 0; j < SUB; j++) {
                float s = 0.f;
#pragma unroll
                for (int c = 0; c < Q4; c++) s = fmaf(qv[c], sK[j * KP + part * Q4 + c], s);
                s += __shfl_xor(s, 1, 64);
                s += __shfl_xor(s, 2, 64);
                float x = s * a.alpha;
                if (RAB) x += sRab[rab_bucket(qts, sKts[j], a.nbuckets)];
                const float p = x / (1.0f + expf(-x)) * inv_n;
                const bool vis = visible(qcode, qts, qi, sKcode[j], sKts[j], kb + j);
                if (vis) {
#pragma unroll
                    for (int c = 0; c < Q4; c++) ov[c] = fmaf(p, sV[j * KP + part * Q4 + c], ov[c]);
                }
            }
        }
    }
    if (qvalid && (!a.cand_rows || a.seg[ob + qi] == SEG_CAND)) {
        E* O = (E*)a.out;
#pragma unroll
        for (int c = 0; c < Q4; c++) st_elem(O, (long long)(ob + qi) * a.ld_o + h * DH + part * Q4 + c, ov[c]);
    }
}

template <int DH, bool CACHED>
static hipError_t fwd_bf16_dh(const AttnArgs& a, int slots, hipStream_t s) {
    if (a.rab && fabsf(a.alpha) >= 1e-7f)
        attn_fwd_bf16_kernel<DH, true, CACHED, false><<<slots, 256, 0, s>>>(a);
    else if (a.rab)
        attn_fwd_bf16_kernel<DH, true, CACHED, true><<<slots, 256, 0, s>>>(a);
    else
        attn_fwd_bf16_kernel<DH, false, CACHED, false><<<slots, 256, 0, s>>>(a);
    return hipGetLastError();
}

template <int DH, class E>
static hipError_t fwd_vec_dh(const AttnArgs& a, int slots, hipStream_t s) {
    if (a.rab)
        attn_fwd_vec_kernel<DH, true, E><<<slots, 256, 0, s>>>(a);
    else
        attn_fwd_vec_kernel<DH, false, E><<<slots, 256, 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_attn_fwd_bf16(const AttnArgs& a, int head_dim, int slots, hipStream_t s) {
    switch (head_dim) {
        case 16: return fwd_vec_dh<16, uint16_t>(a, slots, s);
        case 32: return fwd_bf16_dh<32, false>(a, slots, s);
        case 64: return fwd_bf16_dh<64, false>(a, slots, s);
        case 128: return fwd_bf16_dh<128, false>(a, slots, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_fwd_cached_bf16(const AttnArgs& a, int head_dim, int slots, hipStream_t s) {
    switch (head_dim) {
        case 32: return fwd_bf16_dh<32, true>(a, slots, s);
        case 64: return fwd_bf16_dh<64, true>(a, slots, s);
        case 128: return fwd_bf16_dh<128, true>(a, slots, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_fwd_f32(const AttnArgs& a, int head_dim, int slots, hipStream_t s) {
    switch (head_dim) {
        case 16: return fwd_vec_dh<16, float>(a, slots, s);
        case 32: return fwd_vec_dh<32, float>(a, slots, s);
        case 64: return fwd_vec_dh<64, float>(a, slots, s);
        case 128: return fwd_vec_dh<128, float>(a, slots, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace mtgr
