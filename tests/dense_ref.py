"""Dense, padded torch (fp64) formulation of Eq. 5 used only to pin the oracle.

It builds the whole [B, L, L] visibility matrix from the three mask rules with
tensor comparisons, pads users to a common length with tokens that nobody sees,
runs the attention as batched matmuls and takes every gradient with autograd.
It is a different route from the oracle's per-pair loops and hand-derived
backward, so agreement between the two pins both.
"""
from __future__ import annotations

import numpy as np
import torch


def rule_mask(seg: torch.Tensor, ts: torch.Tensor, valid: torch.Tensor) -> torch.Tensor:
    """[B, L] segment/time/validity -> [B, L, L] bool visibility (query row, key col)."""
    seg_q, seg_k = seg[:, :, None], seg[:, None, :]
    ts_q, ts_k = ts[:, :, None].long(), ts[:, None, :].long()
    L = seg.shape[1]
    eye = torch.eye(L, dtype=torch.bool)[None]
    static_key = (seg_k == 0) | (seg_k == 1)                       # rule 1
    rt_key_seen = (seg_k == 2) & ((seg_q == 2) | (seg_q == 3)) & (ts_k < ts_q)   # rule 2
    # rule 3: candidates are seen only on the diagonal
    m = eye | static_key | rt_key_seen
    both_valid = valid[:, :, None] & valid[:, None, :]
    return m & both_valid


def bucket_torch(delta: torch.Tensor) -> torch.Tensor:
    """Half-octave bucket through float log2 (exact for gaps < 2**24 here)."""
    d = delta.double()
    e = torch.floor(torch.log2(torch.clamp(d, min=1.0)))
    hi = (d >= 1.5 * torch.pow(2.0, e)).long()
    out = 2 * e.long() + hi
    return torch.where(delta < 2, delta, out)


def pad(offsets, *arrays, fill=0):
    offsets = np.asarray(offsets)
    B = len(offsets) - 1
    L = int(np.max(np.diff(offsets))) if B else 0
    out = []
    for a in arrays:
        a = np.asarray(a)
        p = np.full((B, L) + a.shape[1:], fill, dtype=a.dtype)
        for b in range(B):
            n = offsets[b + 1] - offsets[b]
            p[b, :n] = a[offsets[b]:offsets[b + 1]]
        out.append(p)
    valid = np.zeros((B, L), bool)
    for b in range(B):
        valid[b, :offsets[b + 1] - offsets[b]] = True
    return out, valid


def unpad(offsets, x):
    parts = [x[b, :offsets[b + 1] - offsets[b]] for b in range(len(offsets) - 1)]
    return torch.cat(parts, 0)


def dense_attention(offsets, seg, ts, q, k, v, rab=None, alpha=1.0):
    """q, k, v torch fp64 [T, H, dh] (may require grad); returns [T, H, dh]."""
    offsets = np.asarray(offsets)
    (seg_p, ts_p), valid = pad(offsets, seg, ts)
    seg_p, ts_p, valid = torch.from_numpy(seg_p).long(), torch.from_numpy(ts_p), torch.from_numpy(valid)
    M = rule_mask(seg_p, ts_p, valid)                               # [B, L, L]
    B, L = seg_p.shape
    n = torch.tensor(np.diff(offsets), dtype=torch.float64).clamp(min=1.0)

    def to_pad(x):
        parts = []
        for b in range(B):
            xb = x[int(offsets[b]):int(offsets[b + 1])]
            parts.append(torch.nn.functional.pad(xb, (0, 0, 0, 0, 0, L - xb.shape[0])))
        return torch.stack(parts, 0)                                # [B, L, H, dh]

    qp, kp, vp = to_pad(q), to_pad(k), to_pad(v)
    S = alpha * torch.einsum("bihd,bjhd->bhij", qp, kp)
    if rab is not None:
        gap = (ts_p[:, :, None].long() - ts_p[:, None, :].long()).abs()
        bk = bucket_torch(gap).clamp(max=rab.shape[1] - 1)          # [B, L, L]
        S = S + rab[:, bk].permute(1, 0, 2, 3)                      # [B, H, L, L]
    P = torch.where(M[:, None], torch.nn.functional.silu(S), torch.zeros_like(S)) / n[:, None, None, None]
    O = torch.einsum("bhij,bjhd->bihd", P, vp)
    return unpad(offsets, O)


def dense_gln(x, u, gid, gamma, beta, eps=1e-5):
    """torch fp64: layer_norm(x*u) without affine, then the token's group affine."""
    z = x * u if u is not None else x
    zn = torch.nn.functional.layer_norm(z, (z.shape[1],), eps=eps)
    g = torch.as_tensor(np.asarray(gid), dtype=torch.long)
    return zn * gamma[g] + beta[g]
