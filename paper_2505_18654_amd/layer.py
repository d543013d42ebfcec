"""One MTGR encoder layer (Sec. 4.2) built around the attention path, forward and backward.

    Xt = GroupLN_in(X)                                   input Group-LN (u = NULL)
    [Q | K | V | U] = silu(Xt W_in + b_in)               the projection MLPs, one fused GEMM
    Vt = Eq. 5 attention (dynamic mask, 1 / n_b)
    X' = GroupLN(Vt (*) U) W_out + b_out + X             Eq. 6; the top MLP as one linear map

Every step runs in this package's HIP kernels through the C ABI: the projection product with
bias + SiLU in its epilogue (it keeps the pre-activation for the backward), the output product
with bias + residual in its epilogue, the input-gradient products (A B^T), the weight-gradient
products (A^T B, split over tokens) with the bias gradients as fused column sums, Group-LN,
the attention and the residual add of the input gradient.  Q, K, V, U are column views of the
one [T, 4d] activation, which the kernels take with their token stride, and their gradients are
written into the same layout, so the backward's input-projection products read one [T, 4d]
gradient.  torch only allocates.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import torch

from . import hstu, ops


@dataclass
class LayerParams:
    gamma_in: torch.Tensor   # [G, d] fp32
    beta_in: torch.Tensor    # [G, d] fp32
    w_in: torch.Tensor       # [d, 4d] (activation dtype): columns Q | K | V | U
    b_in: torch.Tensor       # [4d] fp32
    gamma: torch.Tensor      # [G, d] fp32
    beta: torch.Tensor       # [G, d] fp32
    w_out: torch.Tensor      # [d, d]
    b_out: torch.Tensor      # [d] fp32


def _split(a: torch.Tensor, d: int, heads: int):
    T = a.shape[0]
    cols = [a[:, i * d:(i + 1) * d] for i in range(4)]
    return [c.view(T, heads, d // heads) for c in cols[:3]] + [cols[3]]


def layer_fwd(x: torch.Tensor, jag: ops.Jagged, P: LayerParams, heads: int, rab=None, alpha: float = 1.0,
              eps: float = 1e-5, workspace=None, planned: bool = False):
    """Returns (x_out [T, d], ctx for layer_bwd)."""
    T, d = x.shape
    xt, m0, r0 = ops.gln_fwd(x, None, jag.seg, P.gamma_in, P.beta_in, eps)
    h = torch.empty((T, 4 * d), dtype=x.dtype, device=x.device)    # pre-activation
    a = torch.empty_like(h)
    ops.gemm(xt, P.w_in, "nn", out=h, bias=P.b_in, silu_out=a)
    q, k, v, u = _split(a, d, heads)
    o = ops.attn_fwd(q, k, v, jag, rab, alpha, workspace=workspace, planned=planned)
    y, m1, r1 = ops.gln_fwd(o.view(T, d), u, jag.seg, P.gamma, P.beta, eps)
    x_out = ops.gemm(y, P.w_out, "nn", bias=P.b_out, residual=x)
    ctx = dict(x=x, xt=xt, m0=m0, r0=r0, h=h, a=a, o=o, y=y, m1=m1, r1=r1)
    return x_out, ctx


def layer_bwd(dx_out: torch.Tensor, ctx: dict, jag: ops.Jagged, P: LayerParams, heads: int, rab=None,
              alpha: float = 1.0, eps: float = 1e-5, workspace=None, planned: bool = False,
              need_drab: bool = True, keep: Optional[dict] = None) -> dict:
    """Gradients of layer_fwd: dict with x, every LayerParams field and (with rab) rab.
    `workspace` should be a backward-size attention workspace (ops.attn_plan(backward=True)).
    `keep`, if given, receives the intermediate gradients (dy, do, da, dh, dxt, dx_gln) for
    stage-by-stage checks."""
    x, xt, h, a, o, y = (ctx[n] for n in ("x", "xt", "h", "a", "o", "y"))
    T, d = x.shape
    g = {"b_out": torch.empty(d, dtype=torch.float32, device=x.device)}
    g["w_out"] = ops.gemm(y, dx_out, "tn", colsum=g["b_out"])
    dy = ops.gemm(dx_out, P.w_out, "nt")
    da = torch.empty_like(a)
    dq, dk, dv, du = _split(da, d, heads)
    q, k, v, u = _split(a, d, heads)
    do = torch.empty_like(o)
    dgam, dbet = torch.empty_like(P.gamma), torch.empty_like(P.beta)
    ops.gln_bwd(dy, o.view(T, d), u, jag.seg, P.gamma, ctx["m1"], ctx["r1"], eps,
                grads=(do.view(T, d), du, dgam, dbet))
    g["gamma"], g["beta"] = dgam, dbet
    drab = torch.empty_like(rab) if (rab is not None and need_drab) else None
    ops.attn_bwd(q, k, v, do, jag, rab, alpha, need_drab=drab is not None, grads=(dq, dk, dv, drab),
                 workspace=workspace, planned=planned)
    if drab is not None:
        g["rab"] = drab
    if keep is not None:
        keep.update(dy=dy, do=do, da=da.clone())
    hstu.mtgr_bias_silu_bwd(T, 4 * d, ops._dtype_code(h), h, 4 * d, P.b_in, da, 4 * d, da, 4 * d)
    g["b_in"] = torch.empty(4 * d, dtype=torch.float32, device=x.device)
    g["w_in"] = ops.gemm(xt, da, "tn", colsum=g["b_in"])
    dxt = ops.gemm(da, P.w_in, "nt")
    dx, _, g["gamma_in"], g["beta_in"] = ops.gln_bwd(dxt, x, None, jag.seg, P.gamma_in, ctx["m0"], ctx["r0"], eps)
    g["x"] = ops.add(dx, dx_out)
    if keep is not None:
        keep.update(dh=da, dxt=dxt, dx_gln=dx)
    return g
