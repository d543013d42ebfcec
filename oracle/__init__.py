"""Python access to the CPU oracle (plain C, fp64, OpenMP).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the benchmark's cpu_baseline
leg and by the smoke check.  The product package never imports it.

`build()` compiles mtgr_oracle.c with gcc (-O2 -fopenmp, no fast-math) into
oracle/libmtgr_oracle.so; the wrappers below take numpy arrays, upcast every
floating-point input to float64 and return float64 results.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mtgr_oracle.c")
LIB_PATH = os.path.join(_HERE, "libmtgr_oracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle shared library (always recompiles when force=True)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-std=c99", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True, cwd=_HERE)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, dbl, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
        L.mtgr_oracle_visible.argtypes = [ctypes.c_int, i32, ctypes.c_int, i32, ctypes.c_int]
        L.mtgr_oracle_visible.restype = ctypes.c_int
        L.mtgr_oracle_rab_bucket.argtypes = [ctypes.c_uint32]
        L.mtgr_oracle_rab_bucket.restype = ctypes.c_int
        L.mtgr_oracle_count_visible.argtypes = [i32, vp, vp, vp]
        L.mtgr_oracle_count_visible.restype = i64
        L.mtgr_oracle_attn_fwd.argtypes = [i32, vp, vp, vp, i32, i32, dbl, vp, vp, vp, vp, i32, vp]
        L.mtgr_oracle_attn_fwd.restype = None
        L.mtgr_oracle_attn_bwd.argtypes = [i32, vp, vp, vp, i32, i32, dbl, vp, vp, vp, vp, i32, vp,
                                           vp, vp, vp, vp]
        L.mtgr_oracle_attn_bwd.restype = None
        L.mtgr_oracle_gln_fwd.argtypes = [i64, i32, i32, dbl, vp, vp, vp, vp, vp, vp, vp, vp]
        L.mtgr_oracle_gln_fwd.restype = None
        L.mtgr_oracle_gln_bwd.argtypes = [i64, i32, i32, dbl, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.mtgr_oracle_gln_bwd.restype = None
        _lib = L
    return _lib


def _f64(x):
    return None if x is None else np.ascontiguousarray(x, dtype=np.float64)


def _p(x):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def _meta(offsets, seg, ts):
    return (np.ascontiguousarray(offsets, dtype=np.int64), np.ascontiguousarray(seg, dtype=np.int8),
            np.ascontiguousarray(ts, dtype=np.int32))


def visible(seg_i: int, ts_i: int, seg_j: int, ts_j: int, same: bool) -> bool:
    return bool(lib().mtgr_oracle_visible(int(seg_i), int(ts_i), int(seg_j), int(ts_j), int(same)))


def rab_bucket(delta: int) -> int:
    return int(lib().mtgr_oracle_rab_bucket(int(delta) & 0xFFFFFFFF))


def count_visible(offsets, seg, ts) -> int:
    off, sg, t = _meta(offsets, seg, ts)
    return int(lib().mtgr_oracle_count_visible(len(off) - 1, _p(off), _p(sg), _p(t)))


def mask_matrix(seg, ts) -> np.ndarray:
    """Dense visibility matrix of one user's tokens (row = query, col = key)."""
    n = len(seg)
    m = np.zeros((n, n), dtype=bool)
    for i in range(n):
        for j in range(n):
            m[i, j] = visible(seg[i], ts[i], seg[j], ts[j], i == j)
    return m


def attn_fwd(offsets, seg, ts, q, k, v, rab: Optional[np.ndarray] = None, alpha: float = 1.0):
    """Eq. 5 forward.  q, k, v: [T, H, dh].  Returns out [T, H, dh] float64."""
    off, sg, t = _meta(offsets, seg, ts)
    q, k, v, rab = _f64(q), _f64(k), _f64(v), _f64(rab)
    T, H, dh = q.shape
    out = np.empty((T, H, dh), np.float64)
    nb = 0 if rab is None else rab.shape[1]
    lib().mtgr_oracle_attn_fwd(len(off) - 1, _p(off), _p(sg), _p(t), H, dh, float(alpha),
                               _p(q), _p(k), _p(v), _p(rab), nb, _p(out))
    return out


def attn_bwd(offsets, seg, ts, q, k, v, dout, rab: Optional[np.ndarray] = None,
             alpha: float = 1.0):
    """Backward of Eq. 5.  Returns (dq, dk, dv, drab-or-None), float64."""
    off, sg, t = _meta(offsets, seg, ts)
    q, k, v, dout, rab = _f64(q), _f64(k), _f64(v), _f64(dout), _f64(rab)
    T, H, dh = q.shape
    dq, dk, dv = (np.empty((T, H, dh), np.float64) for _ in range(3))
    nb = 0 if rab is None else rab.shape[1]
    drab = None if rab is None else np.empty((H, nb), np.float64)
    lib().mtgr_oracle_attn_bwd(len(off) - 1, _p(off), _p(sg), _p(t), H, dh, float(alpha),
                               _p(q), _p(k), _p(v), _p(rab), nb, _p(dout),
                               _p(dq), _p(dk), _p(dv), _p(drab))
    return dq, dk, dv, drab


def gln_fwd(x, u, gid, gamma, beta, eps: float = 1e-5):
    """Eq. 6 gate + Group-LN.  x, u: [T, d] (u may be None).  Returns (y, mean, rstd)."""
    x, u, gamma, beta = _f64(x), _f64(u), _f64(gamma), _f64(beta)
    gid = np.ascontiguousarray(gid, dtype=np.int8)
    T, d = x.shape
    G = gamma.shape[0]
    y = np.empty((T, d), np.float64)
    mean = np.empty(T, np.float64)
    rstd = np.empty(T, np.float64)
    lib().mtgr_oracle_gln_fwd(T, d, G, float(eps), _p(x), _p(u), _p(gid), _p(gamma), _p(beta),
                              _p(y), _p(mean), _p(rstd))
    return y, mean, rstd


def gln_bwd(x, u, gid, gamma, dy, eps: float = 1e-5):
    """Backward of gate + Group-LN.  Returns (dx, du-or-None, dgamma, dbeta)."""
    x, u, gamma, dy = _f64(x), _f64(u), _f64(gamma), _f64(dy)
    gid = np.ascontiguousarray(gid, dtype=np.int8)
    T, d = x.shape
    G = gamma.shape[0]
    dx = np.empty((T, d), np.float64)
    du = None if u is None else np.empty((T, d), np.float64)
    dgamma = np.empty((G, d), np.float64)
    dbeta = np.empty((G, d), np.float64)
    lib().mtgr_oracle_gln_bwd(T, d, G, float(eps), _p(x), _p(u), _p(gid), _p(gamma), _p(dy),
                              _p(dx), _p(du), _p(dgamma), _p(dbeta))
    return dx, du, dgamma, dbeta


# ------------------------------------------------------------------ encoder layer (Sec. 4.2)
# The layer around the attention, read as (Sec. 4.2): Xt = GroupLN_in(X);
# [Q | K | V | U] = silu(Xt W_in + b_in) (the four projection MLPs as one fused linear map
# with SiLU, as in HSTU); Vt = Eq. 5 attention; X' = GroupLN(Vt (*) U) W_out + b_out + X
# (Eq. 6 with the top MLP read as one linear map).  Plain fp64 composition of the functions
# above and numpy matmuls; params: dict of gamma_in, beta_in [G, d], w_in [d, 4d], b_in [4d],
# gamma, beta [G, d], w_out [d, d], b_out [d].

def _silu(z):
    return z / (1.0 + np.exp(-z))


def _keep(x):
    return x


def layer_fwd(offsets, seg, ts, x, params, heads: int, rab=None, alpha: float = 1.0, eps: float = 1e-5,
              store=_keep):
    """One encoder layer forward.  x [T, d].  Returns (x_out, cache).

    `store` is applied to every intermediate that the layer keeps in memory between its steps
    (the identity by default).  Training runs in bf16 mixed precision (Sec. 5, other
    optimisations), so passing a rounding to bf16 gives the exact layer evaluated with
    bf16-stored intermediates: each step's input is the stored value, each step computes
    exactly.  The bias is added to the unrounded product, and the pre-activation kept for the
    backward is the stored product plus the bias."""
    x = _f64(x)
    T, d = x.shape
    dh = d // heads
    P = {k: _f64(v) for k, v in params.items()}
    xt, m0, r0 = gln_fwd(x, None, seg, P["gamma_in"], P["beta_in"], eps)
    xt = store(xt)
    z = xt @ P["w_in"]
    a = store(_silu(z + P["b_in"]))
    h = store(z) + P["b_in"]
    q, k, v, u = (a[:, i * d:(i + 1) * d] for i in range(4))
    o = attn_fwd(offsets, seg, ts, q.reshape(T, heads, dh), k.reshape(T, heads, dh),
                 v.reshape(T, heads, dh), rab, alpha).reshape(T, d)
    o = store(o)
    y, m1, r1 = gln_fwd(o, u, seg, P["gamma"], P["beta"], eps)
    y = store(y)
    x_out = store(y @ P["w_out"] + P["b_out"] + x)
    cache = dict(x=x, xt=xt, h=h, a=a, o=o, y=y)
    return x_out, cache


def layer_bwd(offsets, seg, ts, dx_out, cache, params, heads: int, rab=None, alpha: float = 1.0,
              eps: float = 1e-5, store=_keep):
    """Backward of layer_fwd: returns dict of dx and every parameter gradient (drab if rab).
    `store` as in layer_fwd, applied to every gradient kept between steps and to the weight
    gradients (the bias, Group-LN and relative-bias gradients stay in full precision)."""
    dx_out = _f64(dx_out)
    P = {k: _f64(v) for k, v in params.items()}
    x, xt, h, a, o, y = (cache[n] for n in ("x", "xt", "h", "a", "o", "y"))
    T, d = x.shape
    dh = d // heads
    g = {"w_out": store(y.T @ dx_out), "b_out": dx_out.sum(0)}
    dy = store(dx_out @ P["w_out"].T)
    u = a[:, 3 * d:]
    do, du, g["gamma"], g["beta"] = gln_bwd(o, u, seg, P["gamma"], dy, eps)
    do, du = store(do), store(du)
    q, k, v = (a[:, i * d:(i + 1) * d].reshape(T, heads, dh) for i in range(3))
    dq, dk, dv, drab = attn_bwd(offsets, seg, ts, q, k, v, do.reshape(T, heads, dh), rab, alpha)
    da = store(np.concatenate([dq.reshape(T, d), dk.reshape(T, d), dv.reshape(T, d), du], axis=1))
    s = 1.0 / (1.0 + np.exp(-h))
    dhh = store(da * s * (1.0 + h * (1.0 - s)))
    g["w_in"] = store(xt.T @ dhh)
    g["b_in"] = dhh.sum(0)
    dxt = store(dhh @ P["w_in"].T)
    dx, _, g["gamma_in"], g["beta_in"] = gln_bwd(x, None, seg, P["gamma_in"], dxt, eps)
    g["x"] = store(store(dx) + dx_out)
    if rab is not None:
        g["rab"] = drab
    return g
