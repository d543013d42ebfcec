"""Plain reference of the dynamic embedding table (MTGR Sec. 5, "Dynamic Hash Table" and
"Embedding Lookup"): a Python dict from ID to embedding row and metadata.

TEST INFRASTRUCTURE ONLY: used by tests/ and the benchmark's cpu_baseline leg; the product
package never imports it.  Values are float64; the device table stores bf16 or fp32.

What the device table computes, written as plainly as possible:
  dedup(ids)            -> distinct IDs, their occurrence counts, and for every position the
                           index of its ID among the distinct ones (first-occurrence order here;
                           the device order is arbitrary);
  lookup(unique, occ, now, insert)
                        -> for each ID: found, or (insert and a row is free) a new all-zero row;
                           every found / inserted ID gets count += occ and last_ts = now;
  gather(ids)           -> the rows of the IDs (zeros for absent IDs);
  sgd(ids, grad, lr)    -> row(id) -= lr * (sum of grad rows at the positions holding id);
  evict(threshold, min_count)
                        -> every ID whose last_ts < threshold or whose count < min_count is
                           removed; returns how many.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np


class Row:
    __slots__ = ("value", "count", "last_ts")

    def __init__(self, dim: int):
        self.value = np.zeros(dim, np.float64)
        self.count = 0
        self.last_ts = 0


class DictTable:
    def __init__(self, row_capacity: int, dim: int):
        self.row_capacity = int(row_capacity)
        self.dim = int(dim)
        self.rows: Dict[int, Row] = {}

    @staticmethod
    def dedup(ids) -> Tuple[List[int], List[int], List[int]]:
        """(unique in first-occurrence order, occurrences, inverse)."""
        index: Dict[int, int] = {}
        unique: List[int] = []
        occ: List[int] = []
        inverse: List[int] = []
        for x in (int(v) for v in ids):
            if x not in index:
                index[x] = len(unique)
                unique.append(x)
                occ.append(0)
            occ[index[x]] += 1
            inverse.append(index[x])
        return unique, occ, inverse

    def lookup(self, unique, occurrences, now: int, insert: bool) -> List[bool]:
        """Per ID whether it has a row afterwards.  Raises if inserting would need more rows
        than the capacity (which IDs the device leaves out then is not defined)."""
        unique = [int(u) for u in unique]
        new = [u for u in unique if u not in self.rows]
        if insert and len(self.rows) + len(new) > self.row_capacity:
            raise OverflowError("more distinct IDs than free rows")
        has = []
        for u, o in zip(unique, occurrences):
            if u not in self.rows:
                if not insert:
                    has.append(False)
                    continue
                self.rows[u] = Row(self.dim)
            r = self.rows[u]
            r.count += int(o)
            r.last_ts = int(now)
            has.append(True)
        return has

    def gather(self, ids) -> np.ndarray:
        out = np.zeros((len(ids), self.dim), np.float64)
        for i, x in enumerate(ids):
            r = self.rows.get(int(x))
            if r is not None:
                out[i] = r.value
        return out

    def sgd(self, ids, grad, lr: float) -> None:
        grad = np.asarray(grad, np.float64)
        total: Dict[int, np.ndarray] = {}
        for i, x in enumerate(ids):
            x = int(x)
            if x in total:
                total[x] = total[x] + grad[i]
            else:
                total[x] = grad[i].copy()
        for x, g in total.items():
            r = self.rows.get(x)
            if r is not None:
                r.value = r.value - lr * g

    def evict(self, threshold: int, min_count: int = 0) -> int:
        gone = [k for k, r in self.rows.items() if r.last_ts < threshold or r.count < min_count]
        for k in gone:
            del self.rows[k]
        return len(gone)
