"""Synthetic MTGR batches: jagged per-user token sequences [U | S | R | I].

The paper's training data is proprietary; these generators stand in for it
with the shapes of the five benchmark workloads (tiny, small, mtgr_small,
mtgr_large, serving).  Sequence layout follows the token concatenation of
Eq. 4 (user-feature tokens, history items, real-time items, candidates), the
real-time segment is chronological (Sec. 4.1), candidates of a training sample
are aggregated over one window and candidates of a serving request share the
request time (Sec. 4.1).

Everything here is a random draw; no quantity of the method is computed.
Values are drawn per user from their own seeded stream, so any subset of users
can be regenerated bit-identically without drawing the whole batch.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Iterable, Optional

import numpy as np

SEG_USER, SEG_HIST, SEG_RT, SEG_CAND = 0, 1, 2, 3
WINDOW = 86400                 # one day, in seconds; window start is t = 0
HISTORY_SPAN = 180 * 86400     # history predates the window by up to 180 days
NUM_GROUPS = 4                 # Group-LN groups = the four token domains


@dataclass(frozen=True)
class ConfigSpec:
    name: str
    seed: int
    num_users: int
    n_user_tokens: int
    heads: int
    head_dim: int
    dtype: str                      # "fp32" or "bf16"
    rab_buckets: int = 0            # 0 = no relative bias
    fwd_only: bool = False
    serving: bool = False           # candidates stamped at the request time


CONFIGS: Dict[str, ConfigSpec] = {
    "tiny": ConfigSpec("tiny", 0, 4, 2, 2, 16, "fp32"),
    "small": ConfigSpec("small", 1, 32, 4, 4, 64, "bf16"),
    "mtgr_small": ConfigSpec("mtgr_small", 2, 128, 8, 4, 128, "bf16", rab_buckets=64),
    "mtgr_large": ConfigSpec("mtgr_large", 3, 64, 16, 8, 128, "bf16"),
    "serving": ConfigSpec("serving", 4, 1024, 8, 6, 128, "bf16", fwd_only=True, serving=True),
}


def _draw_counts(spec: ConfigSpec, rng: np.random.Generator):
    """Per-user (history, real-time, candidate) counts, drawn in that order."""
    name = spec.name
    if name == "tiny":
        return int(rng.integers(8, 25)), int(rng.integers(2, 7)), int(rng.integers(1, 5))
    if name == "small":
        return int(rng.integers(50, 301)), int(rng.integers(5, 31)), int(rng.integers(1, 17))
    if name == "mtgr_small":
        h = int(rng.integers(100, 901))
        r = int(rng.integers(10, 65))
        c = int(rng.integers(8, 65))
        h = min(h, 1024 - spec.n_user_tokens - r - c)   # total length <= 1024
        return h, r, c
    if name == "mtgr_large":
        h = int(np.clip(np.rint(rng.lognormal(np.log(600.0), 1.0)), 1, 3000))
        r = int(rng.integers(32, 129))
        c = int(rng.integers(16, 129))
        if rng.random() < 0.05:                          # near-empty tail user
            h, r, c = 0, 0, int(rng.integers(1, 4))
        return h, r, c
    if name == "serving":
        return int(rng.integers(200, 2001)), int(rng.integers(1, 129)), int(rng.integers(100, 501))
    raise KeyError(name)


@dataclass
class Layout:
    """Jagged batch metadata (no tensor values)."""
    spec: ConfigSpec
    offsets: np.ndarray            # int64 [B+1]
    seg: np.ndarray                # int8  [T]
    ts: np.ndarray                 # int32 [T]
    counts: np.ndarray             # int64 [B, 4]: user, history, real-time, candidate
    extra: dict = field(default_factory=dict)

    @property
    def num_users(self) -> int:
        return len(self.offsets) - 1

    @property
    def total_tokens(self) -> int:
        return int(self.offsets[-1])

    @property
    def max_seqlen(self) -> int:
        return int(np.max(np.diff(self.offsets))) if self.num_users else 0

    @property
    def d(self) -> int:
        return self.spec.heads * self.spec.head_dim

    def user_slice(self, b: int) -> slice:
        return slice(int(self.offsets[b]), int(self.offsets[b + 1]))

    def subset(self, users: Iterable[int]) -> "Layout":
        """Layout of the given users only, re-packed contiguously."""
        users = list(users)
        segs, tss, lens = [], [], []
        for b in users:
            sl = self.user_slice(b)
            segs.append(self.seg[sl])
            tss.append(self.ts[sl])
            lens.append(sl.stop - sl.start)
        off = np.zeros(len(users) + 1, np.int64)
        off[1:] = np.cumsum(lens)
        base = self.extra.get("users")           # compose with an earlier subset
        orig = [base[u] for u in users] if base is not None else users
        return Layout(self.spec, off,
                      np.concatenate(segs) if segs else np.zeros(0, np.int8),
                      np.concatenate(tss) if tss else np.zeros(0, np.int32),
                      self.counts[users], dict(self.extra, users=orig))


def make_layout(config: str, seed: Optional[int] = None) -> Layout:
    """Draw the jagged layout of one batch of `config`."""
    spec = CONFIGS[config]
    seed = spec.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    counts = np.zeros((spec.num_users, 4), np.int64)
    for b in range(spec.num_users):
        h, r, c = _draw_counts(spec, rng)
        counts[b] = (spec.n_user_tokens, h, r, c)
    segs, tss = [], []
    for b in range(spec.num_users):
        nu, h, r, c = (int(x) for x in counts[b])
        trng = np.random.default_rng([seed, 1, b])
        ts_hist = np.sort(trng.integers(-HISTORY_SPAN, 0, size=h)).astype(np.int32)
        ts_rt = np.sort(trng.choice(WINDOW, size=r, replace=False)).astype(np.int32)
        if spec.serving:
            ts_cand = np.full(c, WINDOW, np.int32)
        else:
            ts_cand = trng.integers(0, WINDOW, size=c).astype(np.int32)
        segs.append(np.concatenate([np.full(nu, SEG_USER, np.int8), np.full(h, SEG_HIST, np.int8),
                                    np.full(r, SEG_RT, np.int8), np.full(c, SEG_CAND, np.int8)]))
        tss.append(np.concatenate([np.zeros(nu, np.int32), ts_hist, ts_rt, ts_cand]))
    offsets = np.zeros(spec.num_users + 1, np.int64)
    offsets[1:] = np.cumsum(counts.sum(axis=1))
    return Layout(spec, offsets, np.concatenate(segs), np.concatenate(tss), counts, {"seed": seed})


# ---------------------------------------------------------------- bf16 storage

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest even) and return the uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(x: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


# ---------------------------------------------------------------- tensor values

TOKEN_TENSORS = ("q", "k", "v", "u", "do", "dy")


def make_values(layout: Layout, users: Optional[Iterable[int]] = None,
                tensors: Iterable[str] = TOKEN_TENSORS, bf16_bits: bool = False) -> dict:
    """Draw per-token tensors for `users` (default all) plus the global params.

    Per-token tensors have shape [T_sel, H, dh] (q, k, v, do) or [T_sel, d]
    (u, dy), concatenated over the selected users in the given order.
    q, k, v, u ~ N(0, 1/dh) (variance 1/dh); do, dy ~ N(0, 1).  In bf16
    configs the values are rounded to bf16; with `bf16_bits=True` the uint16
    bit patterns are returned instead of float32.
    gamma = 1 + 0.1 N(0,1), beta = 0.1 N(0,1), both [G, d] fp32;
    rab ~ 0.02 N(0,1), [H, buckets] fp32, when the config has a bias.
    """
    spec = layout.spec
    H, dh = spec.heads, spec.head_dim
    d = H * dh
    seed = layout.extra.get("seed", spec.seed)
    base_users = layout.extra.get("users")     # a subset layout maps back to original ids
    sel = list(range(layout.num_users)) if users is None else list(users)
    is_bf16 = spec.dtype == "bf16"
    out = {}
    for ti, name in enumerate(TOKEN_TENSORS):
        if name not in tensors:
            continue
        parts = []
        for b in sel:
            n = int(layout.offsets[b + 1] - layout.offsets[b])
            ob = base_users[b] if base_users is not None else b
            rng = np.random.default_rng([seed, 100 + ti, ob])
            shape = (n, H, dh) if name in ("q", "k", "v", "do") else (n, d)
            x = rng.standard_normal(shape, dtype=np.float32)
            if name in ("q", "k", "v", "u"):
                x *= np.float32(1.0 / np.sqrt(dh))
            if is_bf16:
                x = f32_to_bf16_bits(x) if bf16_bits else round_bf16(x)
            parts.append(x)
        if parts:
            out[name] = np.concatenate(parts, axis=0)
        else:
            shape = (0, H, dh) if name in ("q", "k", "v", "do") else (0, d)
            out[name] = np.zeros(shape, np.uint16 if (is_bf16 and bf16_bits) else np.float32)
    prng = np.random.default_rng([seed, 7])
    out["gamma"] = (1.0 + 0.1 * prng.standard_normal((NUM_GROUPS, d))).astype(np.float32)
    out["beta"] = (0.1 * prng.standard_normal((NUM_GROUPS, d))).astype(np.float32)
    if spec.rab_buckets:
        out["rab"] = (0.02 * np.random.default_rng([seed, 8]).standard_normal(
            (H, spec.rab_buckets))).astype(np.float32)
    else:
        out["rab"] = None
    return out
