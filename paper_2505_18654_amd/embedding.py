"""Dynamic embedding table on the device (MTGR Sec. 5, "Dynamic Hash Table" and "Embedding
Lookup"), driven through the C ABI of include/mtgr_embedding.h.

Torch provides the device buffers and the stream; every step (de-duplication, probing,
insertion, gather, the sparse SGD step, eviction, rebuilding the key store) runs in the
library's HIP kernels.  IDs are int64 tensors holding the bit patterns of uint64 IDs.

    table = DynamicEmbedding(row_capacity=1 << 20, dim=64)
    out, batch = table.lookup(ids, now=t)        # dedup + lookup/insert + gather
    ...
    table.sgd(batch, grad_out, lr=0.05)          # sparse update of the batch's rows
    table.evict(threshold=t - window)            # drop IDs not seen since the threshold
    table.evict(threshold=0, min_count=3)        # drop IDs seen fewer than 3 times
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import hstu


def _next_pow2(n: int) -> int:
    c = 2
    while c < n:
        c <<= 1
    return c


@dataclass
class Batch:
    """What a lookup leaves for the backward of the same batch."""
    n: int
    n_max: int
    inverse: torch.Tensor       # [n] int32
    rows: torch.Tensor          # [n_max] int32, first num_unique valid
    num_unique: torch.Tensor    # [1] int64 (device)
    unique: torch.Tensor        # [n_max] int64
    occurrences: torch.Tensor   # [n_max] int32


class DynamicEmbedding:
    def __init__(self, row_capacity: int, dim: int, key_capacity: int | None = None,
                 dtype: torch.dtype = torch.bfloat16, device="cuda"):
        if dtype not in (torch.bfloat16, torch.float32):
            raise ValueError("dtype must be bfloat16 or float32")
        self.row_capacity = int(row_capacity)
        self.dim = int(dim)
        self.dtype = dtype
        self.device = torch.device(device)
        key_capacity = key_capacity or _next_pow2(2 * self.row_capacity)
        kw = dict(device=self.device)
        self.values = torch.empty(self.row_capacity, self.dim, dtype=dtype, **kw)
        self.counts = torch.zeros(self.row_capacity, dtype=torch.int32, **kw)
        self.last_ts = torch.zeros(self.row_capacity, dtype=torch.int32, **kw)
        self.free_rows = torch.empty(self.row_capacity, dtype=torch.int32, **kw)
        self.state = torch.zeros(hstu.MTGR_EMB_STATE_WORDS, dtype=torch.int32, **kw)
        self._alloc_keys(key_capacity)
        self.table = self._descriptor()
        hstu.mtgr_embedding_init(self.table)

    # -------------------------------------------------------------- storage
    def _alloc_keys(self, key_capacity: int) -> None:
        self.key_capacity = int(key_capacity)
        self.keys = torch.empty(self.key_capacity, dtype=torch.int64, device=self.device)
        self.key_rows = torch.empty(self.key_capacity, dtype=torch.int32, device=self.device)

    def _descriptor(self, keys=None, key_rows=None, key_capacity=None) -> hstu.EmbeddingTable:
        keys = self.keys if keys is None else keys
        key_rows = self.key_rows if key_rows is None else key_rows
        return hstu.EmbeddingTable(
            key_capacity=self.key_capacity if key_capacity is None else key_capacity,
            row_capacity=self.row_capacity, dim=self.dim,
            dtype=hstu.MTGR_DTYPE_BF16 if self.dtype == torch.bfloat16 else hstu.MTGR_DTYPE_FP32,
            keys=keys.data_ptr(), key_rows=key_rows.data_ptr(), values=self.values.data_ptr(),
            counts=self.counts.data_ptr(), last_ts=self.last_ts.data_ptr(),
            free_rows=self.free_rows.data_ptr(), state=self.state.data_ptr())

    # -------------------------------------------------------------- steps
    def dedup(self, ids: torch.Tensor):
        """(unique [n], occurrences [n], inverse [n], num_unique [1] on the device)."""
        n = ids.numel()
        unique = torch.empty(max(n, 1), dtype=torch.int64, device=self.device)
        occ = torch.empty(max(n, 1), dtype=torch.int32, device=self.device)
        inverse = torch.empty(max(n, 1), dtype=torch.int32, device=self.device)
        num = torch.empty(1, dtype=torch.int64, device=self.device)
        wsb = hstu.mtgr_embedding_dedup_workspace_size(n)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
        hstu.mtgr_embedding_dedup(n, ids.contiguous(), unique, occ, inverse, num, ws, wsb)
        return unique, occ, inverse, num

    def lookup(self, ids: torch.Tensor, now: int, insert: bool = True, gather: bool = True):
        """De-duplicate, look up (inserting new IDs) and gather a batch of IDs.
        Returns (out [n, dim] or None, Batch)."""
        n = ids.numel()
        unique, occ, inverse, num = self.dedup(ids)
        n_max = max(n, 1)
        rows = torch.empty(n_max, dtype=torch.int32, device=self.device)
        wsb = hstu.mtgr_embedding_lookup_workspace_size(n_max)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
        hstu.mtgr_embedding_lookup(self.table, n_max, unique, occ, num, int(now), insert, rows, ws, wsb)
        batch = Batch(n, n_max, inverse, rows, num, unique, occ)
        out = self.gather(batch) if gather else None
        return out, batch

    def gather(self, batch: Batch, out: torch.Tensor | None = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(batch.n, self.dim, dtype=self.dtype, device=self.device)
        hstu.mtgr_embedding_gather(self.table, batch.n, batch.inverse, batch.rows, out, out.stride(0))
        return out

    def sgd(self, batch: Batch, grad_out: torch.Tensor, lr: float) -> None:
        grad_out = grad_out.to(self.dtype)
        wsb = hstu.mtgr_embedding_sgd_workspace_size(batch.n, batch.n_max, self.dim)
        ws = torch.empty(wsb, dtype=torch.uint8, device=self.device)
        hstu.mtgr_embedding_sgd(self.table, batch.n, batch.inverse, batch.occurrences, grad_out,
                                grad_out.stride(0), batch.n_max, batch.rows, batch.num_unique, float(lr), ws, wsb)

    def evict(self, threshold: int, min_count: int = 0) -> int:
        """Deletes every ID whose last lookup was before `threshold` or whose occurrence count
        is below `min_count`; returns how many (synchronises to read the count)."""
        num = torch.empty(1, dtype=torch.int64, device=self.device)
        hstu.mtgr_embedding_evict(self.table, int(threshold), int(min_count), num)
        return int(num.item())

    def grow(self, key_capacity: int) -> None:
        """Rebuilds the key store at `key_capacity` slots (deleted slots dropped); the value
        store does not move."""
        old = self.table
        keys = torch.empty(int(key_capacity), dtype=torch.int64, device=self.device)
        key_rows = torch.empty(int(key_capacity), dtype=torch.int32, device=self.device)
        new = self._descriptor(keys, key_rows, int(key_capacity))
        hstu.mtgr_embedding_rehash(old, new)
        self.keys, self.key_rows, self.key_capacity, self.table = keys, key_rows, int(key_capacity), new

    # -------------------------------------------------------------- state (synchronising)
    def stats(self) -> dict:
        s = self.state.tolist()
        return {"next_row": s[hstu.MTGR_EMB_STATE_NEXT_ROW], "free_top": s[hstu.MTGR_EMB_STATE_FREE_TOP],
                "num_keys": s[hstu.MTGR_EMB_STATE_NUM_KEYS], "overflow": s[hstu.MTGR_EMB_STATE_OVERFLOW]}
