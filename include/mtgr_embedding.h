/*
 * mtgr_embedding.h — C ABI of the dynamic embedding table of MTGR's training framework
 * (arXiv 2505.18654, Sec. 5: "Dynamic Hash Table" and "Embedding Lookup") on one MI355X.
 *
 * The table is decoupled as the paper describes: a compact KEY STORE maps 64-bit sparse IDs
 * to row indices (open addressing, linear probing), and a VALUE STORE holds the embedding
 * rows together with per-row metadata (an occurrence counter and the time of the last
 * lookup) that drive eviction.  The key store can be rebuilt at another capacity without
 * moving any embedding row (mtgr_embedding_rehash).  A lookup first de-duplicates the IDs of
 * a batch (mtgr_embedding_dedup), so that every ID is probed, inserted and updated once.
 *
 * Conventions: those of mtgr_hstu.h (caller-owned device memory, asynchronous calls on
 * `stream`, status codes, mtgr_last_error_message).  In addition:
 *   - IDs are uint64; the two largest values (MTGR_EMB_KEY_EMPTY, MTGR_EMB_KEY_DELETED) mark
 *     free and deleted key slots and must not be used as IDs (undefined if they are).
 *   - Counts produced on the device (number of unique IDs, of evicted keys) are written to
 *     device memory; the calls that consume them read them there, so a dedup -> lookup ->
 *     gather -> sgd sequence needs no host synchronisation.  Such calls take an upper bound
 *     (n_max) on the host to size their launches and workspaces.
 *   - Calls on one table must not overlap in time (they update it in place without locks);
 *     any number of tables may be used concurrently.
 *   - Row indices, unique positions and the order of the unique IDs depend on the order in
 *     which concurrent threads won their atomic operations: they are valid but not
 *     reproducible.  What is reproducible: the set of unique IDs, ids[n] ==
 *     unique[inverse[n]], the ID -> embedding mapping and every gathered value; the sgd
 *     update sums each ID's gradients in an order that varies (last bits only).
 */
#ifndef MTGR_EMBEDDING_H
#define MTGR_EMBEDDING_H

#include "mtgr_hstu.h"

#ifdef __cplusplus
extern "C" {
#endif

#define MTGR_EMB_KEY_EMPTY 0xFFFFFFFFFFFFFFFFull     /* free key slot */
#define MTGR_EMB_KEY_DELETED 0xFFFFFFFFFFFFFFFEull   /* slot of an evicted key (reusable) */
#define MTGR_EMB_STATE_WORDS 8                         /* int32 words of table state */

/* State words (device, int32): rows handed out from the never-used tail of the value store,
 * entries of the free-row stack, live keys, and overflow flags (bit 0: a lookup found no free
 * row, bit 1: no free key slot). */
enum {
    MTGR_EMB_STATE_NEXT_ROW = 0,
    MTGR_EMB_STATE_FREE_TOP = 1,
    MTGR_EMB_STATE_NUM_KEYS = 2,
    MTGR_EMB_STATE_OVERFLOW = 3
};

/* One table.  All pointers are caller-owned device memory, 16-byte aligned.
 *   keys      [key_capacity] uint64      key store: ID of each slot, or EMPTY / DELETED
 *   key_rows  [key_capacity] int32       value-store row of each live slot (-1 otherwise)
 *   values    [row_capacity, dim]        embedding rows, dtype bf16 or fp32, row stride dim
 *   counts    [row_capacity] uint32      occurrences of the row's ID over all lookups
 *   last_ts   [row_capacity] int32       `now` of the row's last lookup
 *   free_rows [row_capacity] int32       stack of rows released by eviction
 *   state     [MTGR_EMB_STATE_WORDS] int32
 * key_capacity is a power of two >= 2 and at least row_capacity + 1 (so that a probe always
 * meets a non-live slot); row_capacity in 1 .. 2^31 - 1; dim a multiple of 8 in 8 .. 1024. */
typedef struct {
    int64_t key_capacity;
    int64_t row_capacity;
    int32_t dim;
    mtgr_dtype_t dtype;
    uint64_t* keys;
    int32_t* key_rows;
    void* values;
    uint32_t* counts;
    int32_t* last_ts;
    int32_t* free_rows;
    int32_t* state;
} mtgr_embedding_table_t;

/* Empty table: every key slot EMPTY, key_rows -1, state zero.  Value rows, counts and
 * timestamps are left as they are (a row is zero-filled when an ID first takes it). */
mtgr_status_t mtgr_embedding_init(const mtgr_embedding_table_t* t, mtgr_stream_t stream);

/* Workspace bytes of mtgr_embedding_dedup for n IDs (n in 0 .. 2^30). */
mtgr_status_t mtgr_embedding_dedup_workspace_size(int64_t n, size_t* bytes);

/* De-duplication of a batch of IDs (the "IDs remain unique" step of the embedding lookup):
 *   unique      [n] uint64   the distinct IDs, first *num_unique entries valid
 *   occurrences [n] int32    occurrences[u] = #{i : ids[i] == unique[u]}
 *   inverse     [n] int32    unique[inverse[i]] == ids[i]
 *   num_unique  [1] int64    (device)
 * ids [n] uint64.  A temporary hash set in the workspace (power-of-two capacity >= 2n) holds
 * each ID once; the unique list is that set compacted. */
mtgr_status_t mtgr_embedding_dedup(int64_t n, const uint64_t* ids, uint64_t* unique,
                                   int32_t* occurrences, int32_t* inverse, int64_t* num_unique,
                                   void* workspace, size_t workspace_bytes, mtgr_stream_t stream);

/* Workspace bytes of mtgr_embedding_lookup for up to n_max unique IDs. */
mtgr_status_t mtgr_embedding_lookup_workspace_size(int64_t n_max, size_t* bytes);

/* Lookup (and, with insert != 0, insertion) of *num_unique distinct IDs (<= n_max):
 *   rows[u] = value-store row of unique[u], or -1 when the ID is absent and insert == 0, or
 *   when the table is full (then the overflow bits of state are set; the caller grows the
 *   table with mtgr_embedding_rehash and retries).
 * A new ID takes a row from the free-row stack, else the next never-used row; the row is
 * zero-filled and its counter zeroed.  For every ID found or inserted: counts[row] +=
 * occurrences[u] (1 if occurrences is NULL) and last_ts[row] = now.  unique must hold
 * distinct IDs (as produced by mtgr_embedding_dedup); duplicates are undefined. */
mtgr_status_t mtgr_embedding_lookup(const mtgr_embedding_table_t* t, int64_t n_max,
                                    const uint64_t* unique, const int32_t* occurrences,
                                    const int64_t* num_unique, int32_t now, int32_t insert,
                                    int32_t* rows, void* workspace, size_t workspace_bytes,
                                    mtgr_stream_t stream);

/* Embedding output of a batch: out[i, :] = values[rows[inverse[i]], :] (zeros where the row
 * is -1).  out [n, dim] of the table's dtype with row stride ld_out (>= dim, a multiple of 8),
 * 16-byte aligned.  inverse[i] must index a valid entry of rows. */
mtgr_status_t mtgr_embedding_gather(const mtgr_embedding_table_t* t, int64_t n,
                                    const int32_t* inverse, const int32_t* rows, void* out,
                                    int64_t ld_out, mtgr_stream_t stream);

/* Workspace bytes of mtgr_embedding_sgd for n IDs and up to n_max unique IDs. */
mtgr_status_t mtgr_embedding_sgd_workspace_size(int64_t n, int64_t n_max, int32_t dim, size_t* bytes);

/* Sparse SGD step of the embedding rows of a batch:
 *   g[u, :] = sum over i with inverse[i] == u of grad_out[i, :]          (fp32)
 *   values[rows[u], :] -= lr * g[u, :]      for u < *num_unique with rows[u] >= 0
 * grad_out [n, dim] of the table's dtype, row stride ld_grad; inverse, occurrences and
 * num_unique as produced by mtgr_embedding_dedup and rows by mtgr_embedding_lookup for the same
 * batch.  The positions are grouped by ID first (a counting sort driven by occurrences), so
 * each ID's gradient rows are summed in registers; only groups that straddle a 64-position
 * chunk are combined with float atomics (their order, and the last bits, vary). */
mtgr_status_t mtgr_embedding_sgd(const mtgr_embedding_table_t* t, int64_t n, const int32_t* inverse,
                                 const int32_t* occurrences, const void* grad_out, int64_t ld_grad,
                                 int64_t n_max, const int32_t* rows, const int64_t* num_unique, float lr,
                                 void* workspace, size_t workspace_bytes, mtgr_stream_t stream);

/* Eviction by time and frequency: every live key whose row has last_ts < threshold or
 * counts < min_count is deleted (its slot becomes DELETED, its row goes onto the free-row
 * stack).  min_count = 0 evicts by time only.  *num_evicted (device int64) receives the number
 * of deleted keys. */
mtgr_status_t mtgr_embedding_evict(const mtgr_embedding_table_t* t, int32_t threshold, uint32_t min_count,
                                   int64_t* num_evicted, mtgr_stream_t stream);

/* Rebuilds the key store of `from` into the key store of `to` (its keys / key_rows, of
 * to->key_capacity slots): every live key is re-inserted, deleted slots are dropped.  The two
 * descriptors must share values, counts, last_ts, free_rows and state and agree on
 * row_capacity, dim and dtype; to->key_capacity must exceed the live key count (and
 * row_capacity, as always).  Afterwards `to` is the table; `from`'s key store is unchanged. */
mtgr_status_t mtgr_embedding_rehash(const mtgr_embedding_table_t* from,
                                    const mtgr_embedding_table_t* to, mtgr_stream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* MTGR_EMBEDDING_H */
