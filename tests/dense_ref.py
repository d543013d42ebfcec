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


def bf16_half_ulp(x):
    """Half the spacing of bf16 numbers (8 significant bits) at |x|: the largest rounding error
    of x, 2^(e - 9) for |x| in [2^(e-1), 2^e); 0 at 0."""
    a = np.abs(x)
    return np.where(a > 0, np.ldexp(1.0, np.frexp(a)[1] - 9), 0.0)


def operand_rounding_bounds(offsets, seg, ts, q, k, v, dout, rab=None, alpha=1.0):
    """Per-element bound of the error that rounding the MFMA operands P and dS to bf16 (round to
    nearest: at most half an ulp of each value, h(x)) adds to the attention outputs, for inputs
    whose sums cancel (activations with a non-zero mean) or hold a single term (a candidate
    that sees only itself): rounding every P or dS factor moves a sum by at most
        o_i: sum_j h(p_ij) |v_j|           dv_j: sum_i h(p_ij) |dout_i|
        dq_i: alpha sum_j h(dS_ij) |k_j|    dk_j: alpha sum_i h(dS_ij) |q_i|
    with p, dS rounded before their factor 1/n_b, as the kernels do (alpha = 1: p = silu(s)).
    numpy fp64 [T, H, dh] in,
    dict of [T, H, dh] bounds out; dense per user (small batches only)."""
    offsets = np.asarray(offsets)
    q, k, v, dout = (np.asarray(x, np.float64) for x in (q, k, v, dout))
    out = {name: np.zeros_like(q) for name in ("o", "dq", "dk", "dv")}
    for b in range(len(offsets) - 1):
        s0, s1 = int(offsets[b]), int(offsets[b + 1])
        n = s1 - s0
        if n == 0:
            continue
        sg_t = torch.from_numpy(np.asarray(seg[s0:s1], np.int64))[None]
        ts_t = torch.from_numpy(np.asarray(ts[s0:s1]))[None]
        M = rule_mask(sg_t, ts_t, torch.ones(1, n, dtype=torch.bool))[0].numpy()
        for h in range(q.shape[1]):
            Q, K, V, G = q[s0:s1, h], k[s0:s1, h], v[s0:s1, h], dout[s0:s1, h]
            S = alpha * (Q @ K.T)
            if rab is not None:
                gap = np.abs(np.asarray(ts[s0:s1], np.int64)[:, None] - np.asarray(ts[s0:s1], np.int64)[None, :])
                bk = bucket_torch(torch.from_numpy(gap)).clamp(max=rab.shape[1] - 1).numpy()
                S = S + np.asarray(rab)[h][bk]
            sg = 1.0 / (1.0 + np.exp(-S))
            # the kernels round p and dS before the factor 1/n_b (applied once per output)
            P = np.where(M, S * sg, 0.0)
            dS = np.where(M, (G @ V.T) * sg * (1.0 + S * (1.0 - sg)), 0.0)
            hP, hdS = bf16_half_ulp(P) / n, bf16_half_ulp(dS) / n
            out["o"][s0:s1, h] = hP @ np.abs(V)
            out["dv"][s0:s1, h] = hP.T @ np.abs(G)
            out["dq"][s0:s1, h] = abs(alpha) * hdS @ np.abs(K)
            out["dk"][s0:s1, h] = abs(alpha) * hdS.T @ np.abs(Q)
    return out
