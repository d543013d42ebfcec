"""torch-facing wrappers of the C ABI (buffers from torch, compute in the library).

`Jagged` holds the per-batch metadata on the device; the functions below
allocate outputs and workspace with torch and call the C entry points on the
current stream.  Nothing here computes any part of the method.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import torch

from . import hstu


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return hstu.MTGR_DTYPE_BF16
    if t.dtype == torch.float32:
        return hstu.MTGR_DTYPE_FP32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _token_stride(t: torch.Tensor, inner: int) -> int:
    """Token stride of a [T, H, dh] or [T, d] view whose inner dims are dense."""
    if t.dim() == 3:
        if t.stride(2) != 1 or t.stride(1) != t.shape[2]:
            raise ValueError("head and feature dims must be dense")
    elif t.dim() == 2:
        if t.stride(1) != 1:
            raise ValueError("feature dim must be dense")
    if t.shape[0] <= 1:
        return inner
    return t.stride(0)


def _like_layout(t: torch.Tensor) -> torch.Tensor:
    """Uninitialised tensor with the same shape and strides as `t` (gradients share the
    token stride of their primal, e.g. column slices of one fused projection)."""
    return torch.empty_strided(t.shape, t.stride(), dtype=t.dtype, device=t.device)


@dataclass
class Jagged:
    """Device metadata of a jagged batch of users: offsets [B+1] int32, seg [T] int8, ts [T] int32."""
    offsets: torch.Tensor
    seg: torch.Tensor
    ts: torch.Tensor
    max_seqlen: int

    @property
    def num_users(self) -> int:
        return self.offsets.numel() - 1

    @property
    def total_tokens(self) -> int:
        return self.seg.numel()

    @staticmethod
    def from_host(offsets, seg, ts, device="cuda") -> "Jagged":
        off = torch.as_tensor(offsets).to(torch.int32)
        lens = off[1:] - off[:-1]
        max_len = int(lens.max()) if lens.numel() else 0
        return Jagged(off.to(device), torch.as_tensor(seg).to(torch.int8).to(device),
                      torch.as_tensor(ts).to(torch.int32).to(device), max_len)


def attn_problem(jag: Jagged, q, k, v, out, rab=None, alpha: float = 1.0,
                 flags: int = 0) -> hstu.HstuProblem:
    T, H, dh = q.shape
    row = H * dh
    nb = 0 if rab is None else rab.shape[1]
    return hstu.attn_problem(jag.num_users, T, jag.max_seqlen, H, dh, _dtype_code(q), alpha, nb,
                             _token_stride(q, row), _token_stride(k, row), _token_stride(v, row),
                             _token_stride(out, row), flags)


def validate_batch(jag: Jagged, group_ids=None, num_groups: int = 0, scratch=None) -> None:
    """Debugging aid (synchronises): checks offsets, seg and optional group ids on the device
    through mtgr_debug_validate_inputs; raises hstu.MtgrError naming the first bad index."""
    p = hstu.attn_problem(jag.num_users, jag.total_tokens, jag.max_seqlen, 1, 16)
    if scratch is None:
        scratch = torch.empty(hstu.MTGR_VALIDATE_SCRATCH_BYTES, dtype=torch.uint8, device=jag.offsets.device)
    hstu.mtgr_debug_validate_inputs(p, jag.offsets, jag.seg, group_ids, num_groups, scratch, scratch.numel())


def attn_plan(q, jag: Jagged, workspace=None, rab=None, backward: bool = False):
    """Builds the batch plan (tile summaries + work list) once; pass the returned workspace
    with planned=True to attn_fwd / attn_bwd for every layer on the same batch.  backward=True
    allocates the larger workspace with which the backward stores dS instead of recomputing."""
    p = attn_problem(jag, q, q, q, q, rab)
    if workspace is None:
        workspace = workspace_for(p, q.device, backward)
    hstu.mtgr_hstu_attn_plan(p, jag.offsets, jag.seg, jag.ts, workspace, workspace.numel())
    return workspace


def workspace_for(problem: hstu.HstuProblem, device, backward: bool = False) -> torch.Tensor:
    n = hstu.mtgr_hstu_attn_workspace_size(problem, backward)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def attn_fwd(q, k, v, jag: Jagged, rab=None, alpha: float = 1.0, out=None, workspace=None,
             planned: bool = False, cand_rows: bool = False):
    """Eq. 5 forward: returns out [T, H, dh] (same dtype as q).  cand_rows=True forms only the
    candidate tokens' rows (the other rows of `out` are left as they were)."""
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    flags = (hstu.MTGR_ATTN_PLANNED if planned else 0) | (hstu.MTGR_FWD_CAND_ROWS if cand_rows else 0)
    p = attn_problem(jag, q, k, v, out, rab, alpha, flags)
    if workspace is None:
        workspace = workspace_for(p, q.device)
    hstu.mtgr_hstu_attn_fwd(p, jag.offsets, jag.seg, jag.ts, q, k, v, rab, out, workspace,
                            workspace.numel())
    return out


@dataclass
class UserCache:
    """The user-side tokens (U | S | R) of a batch of users held across serving requests: their
    layout, this layer's keys and values [Tc, H, dh], and the cache's plan (tile summaries and
    token codes, built once by user_cache())."""
    jag: Jagged
    k: torch.Tensor
    v: torch.Tensor
    plan: torch.Tensor


def user_cache(k, v, jag: Jagged) -> UserCache:
    """Plans a user-side cache (mtgr_hstu_attn_plan on its layout) for attn_fwd_cached."""
    return UserCache(jag, k, v, attn_plan(k, jag))


def attn_fwd_cached(q, k, v, jag: Jagged, cache: UserCache, rab=None, alpha: float = 1.0, out=None,
                    workspace=None, planned: bool = False):
    """Candidate rows of a request (q, k, v, jag: the candidates) against the users' cached
    user-side keys and values (mtgr_hstu_attn_fwd_cached).  Returns out [Tq, H, dh]."""
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    p = attn_problem(jag, q, k, v, out, rab, alpha, hstu.MTGR_ATTN_PLANNED if planned else 0)
    pc = attn_problem(cache.jag, cache.k, cache.k, cache.v, cache.k)
    if workspace is None:
        workspace = workspace_for(p, q.device)
    hstu.mtgr_hstu_attn_fwd_cached(p, jag.offsets, jag.seg, jag.ts, q, k, v, rab, out, pc, cache.jag.offsets,
                                   cache.jag.ts, cache.k, cache.v, cache.plan, cache.plan.numel(), workspace,
                                   workspace.numel())
    return out


def attn_bwd(q, k, v, dout, jag: Jagged, rab=None, alpha: float = 1.0, need_drab: bool = True,
             grads=None, workspace=None, planned: bool = False, parts: str = "all"):
    """Backward of Eq. 5: returns (dq, dk, dv, drab-or-None).

    parts: "all"; "dq" or "dkdv" (one side only); or the two halves of the stored-dS path as
    two calls on one backward-size workspace: "dkdv_keep_ds" (dk, dv, drab and the dS blocks)
    then "dq_from_ds" (dq from them; drab is not formed again)."""
    flags = (hstu.MTGR_ATTN_PLANNED if planned else 0) | {
        "all": 0, "dq": hstu.MTGR_BWD_SKIP_DKDV, "dkdv": hstu.MTGR_BWD_SKIP_DQ,
        "dkdv_keep_ds": hstu.MTGR_BWD_SKIP_DQ | hstu.MTGR_BWD_KEEP_DS,
        "dq_from_ds": hstu.MTGR_BWD_SKIP_DKDV | hstu.MTGR_BWD_DS_READY}[parts]
    if parts == "dq_from_ds":
        need_drab = False
    if grads is None:
        dq, dk, dv = (_like_layout(x) for x in (q, k, v))
        drab = torch.empty_like(rab) if (rab is not None and need_drab) else None
    else:
        dq, dk, dv, drab = grads
        if not need_drab:
            drab = None
    p = attn_problem(jag, q, k, v, dout, rab, alpha, flags)
    if _token_stride(dq, q.shape[1] * q.shape[2]) != p.ld_q or \
            _token_stride(dk, q.shape[1] * q.shape[2]) != p.ld_k or \
            _token_stride(dv, q.shape[1] * q.shape[2]) != p.ld_v:
        raise ValueError("gradients must share the layout of q, k, v")
    if workspace is None:
        workspace = workspace_for(p, q.device, backward=True)
    hstu.mtgr_hstu_attn_bwd(p, jag.offsets, jag.seg, jag.ts, q, k, v, rab, dout, dq, dk, dv, drab,
                            workspace, workspace.numel())
    return dq, dk, dv, drab


def gln_fwd(x, u, group_ids, gamma, beta, eps: float = 1e-5, y=None, stats=None):
    """Gate + Group-LN forward: returns (y, mean, rstd)."""
    T, d = x.shape
    if y is None:
        y = torch.empty((T, d), dtype=x.dtype, device=x.device)
    if stats is None:
        mean = torch.empty(T, dtype=torch.float32, device=x.device)
        rstd = torch.empty(T, dtype=torch.float32, device=x.device)
    else:
        mean, rstd = stats
    p = hstu.gln_problem(T, d, gamma.shape[0], _dtype_code(x), eps, _token_stride(x, d),
                         _token_stride(u, d) if u is not None else d, _token_stride(y, d))
    hstu.mtgr_group_layernorm_fwd(p, x, u, group_ids, gamma, beta, y, mean, rstd)
    return y, mean, rstd


def gln_bwd(dy, x, u, group_ids, gamma, mean, rstd, eps: float = 1e-5, grads=None, workspace=None):
    """Gate + Group-LN backward: returns (dx, du-or-None, dgamma, dbeta)."""
    T, d = x.shape
    if grads is None:
        dx = _like_layout(x)
        du = _like_layout(u) if u is not None else None
        dgamma = torch.empty_like(gamma)
        dbeta = torch.empty_like(gamma)
    else:
        dx, du, dgamma, dbeta = grads
    p = hstu.gln_problem(T, d, gamma.shape[0], _dtype_code(x), eps, _token_stride(x, d),
                         _token_stride(u, d) if u is not None else d, _token_stride(dy, d))
    if _token_stride(dx, d) != p.ld_x or (du is not None and _token_stride(du, d) != p.ld_u):
        raise ValueError("gradients must share the layout of x, u")
    if workspace is None:
        n = hstu.mtgr_group_layernorm_workspace_size(p, True)
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=x.device)
    hstu.mtgr_group_layernorm_bwd(p, dy, x, u, group_ids, gamma, mean, rstd, dx, du, dgamma, dbeta,
                                  workspace, workspace.numel())
    return dx, du, dgamma, dbeta


def gln_workspace(x, groups: int) -> torch.Tensor:
    T, d = x.shape
    p = hstu.gln_problem(T, d, groups, _dtype_code(x))
    n = hstu.mtgr_group_layernorm_workspace_size(p, True)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=x.device)


_GEMM_LAYOUTS = {"nn": hstu.MTGR_GEMM_NN, "nt": hstu.MTGR_GEMM_NT, "tn": hstu.MTGR_GEMM_TN}


def _row_ld(t: torch.Tensor) -> int:
    if t.dim() != 2 or t.dtype != torch.bfloat16 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError("GEMM operands are 2-D bf16 with a dense inner dim")
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def gemm(a, b, layout: str = "nn", out=None, bias=None, residual=None, silu_out=None, colsum=None,
         workspace=None):
    """bf16 product through mtgr_gemm_bf16: 'nn' a @ b, 'nt' a @ b.T, 'tn' a.T @ b, with the
    encoder layer's fused epilogues (bias + SiLU into `silu_out`, or bias + residual) and, for
    'tn', the fp32 column sums of b into `colsum`.  Returns `out`."""
    lay = _GEMM_LAYOUTS[layout]
    if layout == "nn":
        (M, K), N = a.shape, b.shape[1]
    elif layout == "nt":
        (M, K), N = a.shape, b.shape[0]
    else:
        (K, M), N = a.shape, b.shape[1]
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    epi = hstu.MTGR_GEMM_EPI_NONE
    if silu_out is not None:
        epi = hstu.MTGR_GEMM_EPI_BIAS_SILU
    elif residual is not None:
        epi = hstu.MTGR_GEMM_EPI_BIAS_RESIDUAL
    ws_bytes = 0
    if layout == "tn":
        ws_bytes = hstu.mtgr_gemm_workspace_size(lay, M, N, K)
        if workspace is None or workspace.numel() < ws_bytes:
            workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=a.device)
        ws_bytes = workspace.numel()
    hstu.mtgr_gemm_bf16(lay, M, N, K, a, _row_ld(a), b, _row_ld(b), out, _row_ld(out), epi, bias,
                        residual, _row_ld(residual) if residual is not None else 0, silu_out,
                        _row_ld(silu_out) if silu_out is not None else 0, colsum, workspace, ws_bytes)
    return out


def add(a, b, out=None):
    """out = a + b through mtgr_add (2-D, dense inner dim)."""
    if out is None:
        out = torch.empty_like(a)
    rows, cols = a.shape
    hstu.mtgr_add(rows, cols, _dtype_code(a), a, _token_stride(a, cols), b, _token_stride(b, cols), out,
                  _token_stride(out, cols))
    return out
