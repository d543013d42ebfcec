"""The backward's ways to form dq, dk, dv through the C ABI.

1. one call on a backward-size workspace: the dK/dV kernel stores dS, dq is formed from it;
2. the same as two calls (MTGR_BWD_KEEP_DS, then MTGR_BWD_DS_READY);
3. one call on the forward-size workspace: the dq kernel recomputes S, dP and dS;
4. one side per call (recomputing).

dk and dv come from the same kernel in every case and must agree bit for bit; dq of the
stored paths agree bit for bit with each other (drab, summed with float atomics across
workgroups, to 1e-4); every dq and drab is checked against the oracle (bf16 bar of
test_gpu_parity.py), and drab must be formed exactly once.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import hstu, ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout, make_values
from tests.gpu_util import (TOL, custom_layout, jagged, make_inputs, per_user_err, record, rel_err,
                            rows_of, say, to_np)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def all_paths(inp):
    jag = jagged(inp)
    q, k, v, do, rab = inp["q"], inp["k"], inp["v"], inp["do"], inp["rab"]
    p = ops.attn_problem(jag, q, k, v, do, rab)
    ws_fwd = ops.workspace_for(p, q.device, backward=False)
    ws_bwd = ops.workspace_for(p, q.device, backward=True)
    assert ws_bwd.numel() > ws_fwd.numel()
    out = {"stored": ops.attn_bwd(q, k, v, do, jag, rab, workspace=ws_bwd),
           "recompute": ops.attn_bwd(q, k, v, do, jag, rab, workspace=ws_fwd)}
    ops.attn_plan(q, jag, workspace=ws_bwd, rab=rab, backward=True)
    g = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
         None if rab is None else torch.empty_like(rab))
    ops.attn_bwd(q, k, v, do, jag, rab, grads=g, workspace=ws_bwd, planned=True, parts="dkdv_keep_ds")
    ops.attn_bwd(q, k, v, do, jag, rab, grads=g, workspace=ws_bwd, planned=True, parts="dq_from_ds")
    out["two_calls"] = g
    dq1, _, _, drab1 = ops.attn_bwd(q, k, v, do, jag, rab, workspace=ws_fwd, parts="dq")
    _, dk1, dv1, _ = ops.attn_bwd(q, k, v, do, jag, rab, workspace=ws_fwd, parts="dkdv", need_drab=False)
    out["one_side"] = (dq1, dk1, dv1, drab1)
    torch.cuda.synchronize()
    return out


def check_consistency(out, rab):
    ref = out["stored"]
    for name in ("recompute", "two_calls", "one_side"):
        assert torch.equal(out[name][1], ref[1]), f"dk {name}"
        assert torch.equal(out[name][2], ref[2]), f"dv {name}"
    assert torch.equal(out["two_calls"][0], ref[0]), "dq two_calls"
    assert torch.equal(out["one_side"][0], out["recompute"][0]), "dq one_side"
    if rab is not None:   # drab is summed with float atomics across workgroups: order varies
        e = rel_err(to_np(out["two_calls"][3]), to_np(ref[3]))
        assert e <= 1e-4, ("drab two_calls", e)


@pytest.mark.parametrize("config,users", [("mtgr_small", [0, 5, 9]), ("mtgr_large", [1, 7, 33])])
def test_paths_agree_and_match_oracle(config, users):
    L = make_layout(config)
    inp = make_inputs(L, users=users)
    say(f"[bwd paths] {config} users={users}")
    out = all_paths(inp)
    check_consistency(out, inp["rab"])
    sub = L.subset(users)
    vals = make_values(sub)
    rows = rows_of(L, users)
    dq_ref, dk_ref, dv_ref, _ = oracle.attn_bwd(sub.offsets, sub.seg, sub.ts, vals["q"], vals["k"],
                                                vals["v"], to_np(inp["do"])[rows], inp["rab_np"])
    tol = TOL["bf16"]
    for name in ("stored", "recompute"):
        dq, dk, dv, _ = out[name]
        figs = {t: per_user_err(L, users, to_np(x)[rows], r, "bf16", tol)
                for t, x, r in (("dq", dq, dq_ref), ("dk", dk, dk_ref), ("dv", dv, dv_ref))}
        record(f"bwd-paths-{config}-{name}", figs)
        errs = {t: e["checked"] for t, e in figs.items()}
        say(f"[bwd paths] {config} {name} " + " ".join(f"{t}={e:.2e}" for t, e in errs.items()))
        assert max(errs.values()) <= tol, (name, errs)


def test_drab_formed_once():
    """Whole-batch drab against the oracle for the stored path (formed by the dK/dV kernel),
    the recomputing path (the dK/dV kernel again, the dq kernel not) and the dq-only call
    (formed by the recomputing dq kernel)."""
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(11)
    segs, tss = [], []
    for n_s, n_r, n_c in ((150, 40, 20), (60, 3, 2), (300, 90, 50)):
        segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 4 + sorted(rng.integers(-10**6, 0, n_s).tolist()) +
                   sorted(rng.choice(86400, n_r, replace=False).tolist()) + rng.integers(0, 86400, n_c).tolist())
    L = custom_layout(segs, tss, heads=2, head_dim=128, dtype="bf16", rab_buckets=64)
    inp = make_inputs(L, all_exact=True)
    say("[bwd paths] drab")
    out = all_paths(inp)
    check_consistency(out, inp["rab"])
    vals = make_values(L)
    ref = oracle.attn_bwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], to_np(inp["do"]),
                          inp["rab_np"])[3]
    for name in ("stored", "recompute", "one_side"):
        e = rel_err(to_np(out[name][3]), ref)
        say(f"[bwd paths] drab {name} {e:.2e}")
        assert e <= TOL["bf16"], (name, e)


def test_stored_path_flag_errors():
    L = make_layout("small")
    inp = make_inputs(L, users=[0])
    jag = jagged(inp)
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
    p = ops.attn_problem(jag, q, k, v, do)
    ws_fwd = ops.workspace_for(p, q.device, backward=False)
    with pytest.raises(hstu.MtgrError) as e:   # needs the backward-size workspace
        ops.attn_bwd(q, k, v, do, jag, workspace=ws_fwd, parts="dkdv_keep_ds")
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL
    with pytest.raises(hstu.MtgrError) as e:
        ops.attn_bwd(q, k, v, do, jag, workspace=ws_fwd, parts="dq_from_ds")
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL


@pytest.mark.parametrize("alpha", [0.0883883, -0.7, 3.0, 1e-25, 0.0])
def test_alpha_values(alpha):
    """Score scales of either sign, a tiny one and zero (every other test uses alpha = 1):
    both backward forms against the oracle on users with every mask case."""
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(23)
    segs, tss = [], []
    for n_s, n_r, n_c in ((150, 40, 20), (60, 3, 2), (200, 70, 45)):
        segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 4 + sorted(rng.integers(-10**6, 0, n_s).tolist()) +
                   sorted(rng.choice(86400, n_r, replace=False).tolist()) + rng.integers(0, 86400, n_c).tolist())
    L = custom_layout(segs, tss, heads=2, head_dim=128, dtype="bf16", rab_buckets=0)
    inp = make_inputs(L, all_exact=True)
    jag = jagged(inp)
    q, k, v, do = inp["q"], inp["k"], inp["v"], inp["do"]
    say(f"[bwd paths] alpha={alpha}")
    p = ops.attn_problem(jag, q, k, v, do, None, alpha)
    outs = {"stored": ops.attn_bwd(q, k, v, do, jag, alpha=alpha,
                                   workspace=ops.workspace_for(p, q.device, backward=True)),
            "recompute": ops.attn_bwd(q, k, v, do, jag, alpha=alpha,
                                      workspace=ops.workspace_for(p, q.device, backward=False))}
    torch.cuda.synchronize()
    vals = make_values(L)
    ref = oracle.attn_bwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], to_np(do), None,
                          alpha=alpha)
    users = list(range(L.num_users))
    errs = {}
    for name, (dq, dk, dv, _) in outs.items():
        for t, x, r in (("dq", dq, ref[0]), ("dk", dk, ref[1]), ("dv", dv, ref[2])):
            g = to_np(x)
            if alpha == 0.0:
                assert np.all(g == 0), (name, t)
                continue
            errs[(name, t)] = per_user_err(L, users, g, r, "bf16", TOL["bf16"])["checked"]
    say(f"[bwd paths] alpha={alpha} " + " ".join(f"{n}.{t}={e:.2e}" for (n, t), e in errs.items()))
    assert all(e <= TOL["bf16"] for e in errs.values()), errs


@pytest.mark.parametrize("alpha", [1.0, -0.7, 3.0, 2e-7, 5e-8, 1e-25, 0.0])
def test_forward_with_bias_alpha_values(alpha):
    """The forward with a relative bias masks through the score (alpha s + rab about -1e30)
    when |alpha| >= 1e-7 and selects zero element by element below that: both against the
    oracle, on users with every mask case (partial tiles on and off the diagonal)."""
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(29)
    segs, tss = [], []
    for n_s, n_r, n_c in ((150, 40, 20), (60, 3, 2), (200, 70, 45)):
        segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 4 + sorted(rng.integers(-10**6, 0, n_s).tolist()) +
                   sorted(rng.choice(86400, n_r, replace=False).tolist()) + rng.integers(0, 86400, n_c).tolist())
    L = custom_layout(segs, tss, heads=2, head_dim=128, dtype="bf16", rab_buckets=64)
    inp = make_inputs(L, all_exact=True)
    jag = jagged(inp)
    q, k, v, rab = inp["q"], inp["k"], inp["v"], inp["rab"]
    say(f"[bwd paths] forward with bias, alpha={alpha}")
    o = ops.attn_fwd(q, k, v, jag, rab, alpha)
    torch.cuda.synchronize()
    vals = make_values(L)
    ref = oracle.attn_fwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], vals["rab"], alpha)
    e = per_user_err(L, list(range(L.num_users)), to_np(o), ref, "bf16", TOL["bf16"])
    say(f"[bwd paths] forward with bias, alpha={alpha}: {e['checked']:.2e} (literal {e['literal']:.2e})")
    assert e["checked"] <= TOL["bf16"], e
