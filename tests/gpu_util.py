"""Helpers for the GPU parity tests: run the library, run the oracle on the same
inputs, compare with the max-abs / RMS criterion."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2505_18654_amd import ops
from synth import CONFIGS, Layout, make_values
from synth.batches import ConfigSpec
from synth.torch_inputs import device_inputs

TOL = {"bf16": 2e-2, "fp32": 1e-4}
# Elementwise allowance for bf16 results: one half-ulp (2^-9) for storing the output in bf16
# plus one for the bf16 rounding of the MFMA operand (P or dS) that produced it.
STORAGE_ULP = {"bf16": 2.0 ** -8, "fp32": 0.0}


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def rel_err(got, want) -> float:
    """max |got - want| / rms(want) (0 when both are all-zero)."""
    want = np.asarray(want, np.float64)
    got = np.asarray(got, np.float64)
    if want.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(want ** 2)))
    err = float(np.max(np.abs(got - want)))
    if rms == 0.0:
        return 0.0 if err == 0.0 else float("inf")
    return err / rms


def to_np(t) -> np.ndarray:
    return None if t is None else t.float().cpu().numpy().astype(np.float64)


def rows_of(layout, users):
    if not len(users):
        return np.zeros(0, np.int64)
    return np.concatenate([np.arange(layout.offsets[b], layout.offsets[b + 1]) for b in users])


def custom_layout(seg_per_user, ts_per_user, heads=2, head_dim=64, dtype="bf16", rab_buckets=0,
                  seed=77) -> Layout:
    spec = ConfigSpec("custom", seed, len(seg_per_user), 0, heads, head_dim, dtype,
                      rab_buckets=rab_buckets)
    lens = [len(s) for s in seg_per_user]
    off = np.zeros(len(lens) + 1, np.int64)
    off[1:] = np.cumsum(lens)
    seg = np.concatenate([np.asarray(s, np.int8) for s in seg_per_user]) if lens else np.zeros(0, np.int8)
    ts = np.concatenate([np.asarray(t, np.int32) for t in ts_per_user]) if lens else np.zeros(0, np.int32)
    counts = np.array([[np.sum(np.asarray(s) == g) for g in range(4)] for s in seg_per_user], np.int64)
    return Layout(spec, off, seg, ts, counts.reshape(-1, 4), {"seed": seed})


def jagged(inp) -> ops.Jagged:
    return ops.Jagged(inp["offsets"], inp["seg"], inp["ts"], inp["max_seqlen"])


def gpu_step(inp, fwd_only=False, eps=1e-5):
    """The hot path on the device: attention fwd -> gate + Group-LN fwd -> their backward."""
    jag = jagged(inp)
    q, k, v, u = inp["q"], inp["k"], inp["v"], inp["u"]
    T, H, dh = q.shape
    o = ops.attn_fwd(q, k, v, jag, inp["rab"])
    y, mean, rstd = ops.gln_fwd(o.view(T, H * dh), u, inp["seg"], inp["gamma"], inp["beta"], eps)
    res = {"o": o, "y": y, "mean": mean, "rstd": rstd}
    if fwd_only:
        return res
    dx, du, dg, db = ops.gln_bwd(inp["dy"], o.view(T, H * dh), u, inp["seg"], inp["gamma"], mean,
                                 rstd, eps)
    dq, dk, dv, drab = ops.attn_bwd(q, k, v, dx.view(T, H, dh), jag, inp["rab"])
    res.update(dict(do=dx, du=du, dgamma=dg, dbeta=db, dq=dq, dk=dk, dv=dv, drab=drab))
    return res


def oracle_stages(layout, users, inp, gpu, fwd_only=False, eps=1e-5):
    """Oracle of every stage on `users`, each stage fed with the device's stored input.

    Attention forward takes the generated q, k, v; Group-LN takes the device's attention
    output rows; the attention backward takes the device's Group-LN input gradient as
    dout.  Each comparison therefore isolates one kernel."""
    sub = layout.subset(users)
    vals = make_values(sub)
    H, dh = layout.spec.heads, layout.spec.head_dim
    rows = rows_of(layout, users)
    T = len(rows)
    rab = inp["rab_np"]
    ref = {"o": oracle.attn_fwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"], vals["v"], rab)}
    x = to_np(gpu["o"])[rows].reshape(T, H * dh)
    ref["y"], ref["mean"], ref["rstd"] = oracle.gln_fwd(x, vals["u"], sub.seg, inp["gamma_np"],
                                                        inp["beta_np"], eps)
    if fwd_only:
        return ref
    dx, du, dg, db = oracle.gln_bwd(x, vals["u"], sub.seg, inp["gamma_np"], vals["dy"], eps)
    ref.update(do=dx, du=du, dgamma=dg, dbeta=db)
    dout = to_np(gpu["do"])[rows].reshape(T, H, dh)
    dq, dk, dv, drab = oracle.attn_bwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"], vals["v"],
                                       dout, rab)
    ref.update(dq=dq, dk=dk, dv=dv, drab=drab)
    return ref


PER_TOKEN = ("o", "y", "mean", "rstd", "do", "du", "dq", "dk", "dv")
PER_BATCH = ("dgamma", "dbeta", "drab")


def per_user_err(layout, users, got, want, ulp):
    """max over users of  max_i (|got_i - want_i| - ulp |want_i|)_+ / rms_user(want)."""
    worst = 0.0
    row = 0
    got = got.reshape(len(got), -1)
    want = want.reshape(len(want), -1)
    for b in users:
        n = int(layout.offsets[b + 1] - layout.offsets[b])
        if n == 0:
            continue
        g, w = got[row:row + n], want[row:row + n]
        row += n
        rms = float(np.sqrt(np.mean(w ** 2)))
        excess = float(np.max(np.maximum(np.abs(g - w) - ulp * np.abs(w), 0.0)))
        if rms == 0.0:
            e = 0.0 if excess == 0.0 else float("inf")
        else:
            e = excess / rms
        worst = max(worst, e)
    return worst


def compare(layout, users, gpu, ref, tol, whole_batch: bool):
    """Per-tensor errors.  Per-token outputs: per-user max-abs / RMS after the storage
    allowance; batch-summed gradients (only when every user is compared): whole-tensor
    max-abs / RMS.  Returns (errors, raw whole-batch errors, failures)."""
    rows = rows_of(layout, users)
    ulp = STORAGE_ULP[layout.spec.dtype]
    errs, raw = {}, {}
    for name in PER_TOKEN:
        if name not in ref or ref[name] is None or name not in gpu or gpu[name] is None:
            continue
        g = to_np(gpu[name])[rows].reshape(ref[name].shape)
        raw[name] = rel_err(g, ref[name])
        errs[name] = per_user_err(layout, users, g, ref[name], ulp)
    if whole_batch:
        for name in PER_BATCH:
            if ref.get(name) is not None and gpu.get(name) is not None:
                g = to_np(gpu[name])
                raw[name] = rel_err(g, ref[name])
                errs[name] = raw[name]
    bad = {k: v for k, v in errs.items() if not v <= tol}
    return errs, raw, bad


def make_inputs(layout, users=None, all_exact=False):
    return device_inputs(layout, "cuda", exact_users=users, all_exact=all_exact)


def config(name):
    return CONFIGS[name]
