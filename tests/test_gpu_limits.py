"""GPU parity at the limits: head counts 1 and MTGR_MAX_HEADS = 255, and users longer than one
window of the tile walker.

The work list packs the head into the low 8 bits of an item, the relative-bias table and its
gradient are indexed per head, and the tile summaries and token codes are per user: the
largest head count exercises every head index the packing allows, a single head the smallest
grid.  Forward and both backward forms against the oracle (Eq. 5 and its backward), with and
without the relative bias, on users that hold every mask case.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import hstu, ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_values
from tests.gpu_util import TOL, custom_layout, jagged, make_inputs, per_user_err, rel_err, say, to_np

pytestmark = pytest.mark.gpu

MAX_HEADS = hstu.MTGR_MAX_HEADS


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def users():
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(41)
    segs, tss = [], []
    for n_s, n_r, n_c in ((90, 25, 14), (20, 2, 1), (0, 0, 3), (140, 33, 20)):
        segs.append([U] * 2 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 2 + sorted(rng.integers(-10**6, 0, n_s).tolist()) +
                   sorted(rng.choice(86400, n_r, replace=False).tolist()) + rng.integers(0, 86400, n_c).tolist())
    return segs, tss


def check_attention(L, label):
    """Forward and both backward forms of the layout's batch against the oracle."""
    dtype, dh, rab = L.spec.dtype, L.spec.head_dim, L.spec.rab_buckets
    inp = make_inputs(L, all_exact=True)
    jag = jagged(inp)
    q, k, v, do, rb = inp["q"], inp["k"], inp["v"], inp["do"], inp["rab"]
    say(f"[limits] {label}: T={L.total_tokens} users={L.num_users}")
    o = ops.attn_fwd(q, k, v, jag, rb)
    p = ops.attn_problem(jag, q, k, v, do, rb)
    outs = {"stored": ops.attn_bwd(q, k, v, do, jag, rb, workspace=ops.workspace_for(p, q.device, backward=True))}
    if dtype == "bf16" and dh >= 32:
        outs["recompute"] = ops.attn_bwd(q, k, v, do, jag, rb,
                                         workspace=ops.workspace_for(p, q.device, backward=False))
    torch.cuda.synchronize()

    vals = make_values(L)
    rab_np = inp["rab_np"] if rab else None
    tol = TOL[dtype]
    ev = list(range(L.num_users))
    o_ref = oracle.attn_fwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], rab_np)
    errs = {"o": per_user_err(L, ev, to_np(o), o_ref, dtype, tol)["checked"]}
    ref = oracle.attn_bwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], to_np(do), rab_np)
    for name, (dq, dk, dv, drab) in outs.items():
        for t, x, r in (("dq", dq, ref[0]), ("dk", dk, ref[1]), ("dv", dv, ref[2])):
            errs[f"{name}.{t}"] = per_user_err(L, ev, to_np(x), r, dtype, tol)["checked"]
        if rab:
            errs[f"{name}.drab"] = rel_err(to_np(drab), ref[3])
    say(f"[limits] {label}: " + " ".join(f"{n}={e:.2e}" for n, e in errs.items()))
    assert all(e <= tol for e in errs.values()), (label, errs)
    if len(outs) == 2:   # dK, dV come from the same kernel in both forms; dQ sums in another order
        for i, t in ((1, "dk"), (2, "dv")):
            assert torch.equal(outs["stored"][i], outs["recompute"][i]), (label, t)


@pytest.mark.parametrize("heads", [1, MAX_HEADS])
@pytest.mark.parametrize("dtype,dh,rab", [("bf16", 32, 64), ("bf16", 32, 0), ("bf16", 16, 64), ("fp32", 16, 64)])
def test_head_count_limits(heads, dtype, dh, rab):
    segs, tss = users()
    L = custom_layout(segs, tss, heads=heads, head_dim=dh, dtype=dtype, rab_buckets=rab)
    check_attention(L, f"H={heads} {dtype} dh={dh} rab={rab}")


def long_users():
    """Users longer than 64 tiles of 64 tokens, so the tile walker reloads its window of tile
    classes (every other test user fits one window): real-time tokens in time order (causal)
    followed by candidates, whose tiles against each other are MASKED off the diagonal, so the
    last window of the first user holds candidate tiles only and is skipped whole; a short user
    between them.  (A user made almost only of candidates, each key seen by itself alone, has
    per-user gradient RMS diluted several times by those near-zero keys; the bar is per user.)"""
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(43)
    segs, tss = [], []
    for n_u, n_s, n_r, n_c in ((4, 60, 4800, 3436), (3, 40, 10, 5), (12, 100, 4500, 200)):
        segs.append([U] * n_u + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * n_u + sorted(rng.integers(-10**7, 0, n_s).tolist()) +
                   sorted(rng.choice(10**6, n_r, replace=False).tolist()) + rng.integers(0, 10**6, n_c).tolist())
    return segs, tss


@pytest.mark.parametrize("dtype,dh,rab", [("bf16", 128, 0), ("bf16", 64, 64), ("fp32", 32, 64)])
def test_long_users_across_walker_windows(dtype, dh, rab):
    segs, tss = long_users()
    L = custom_layout(segs, tss, heads=2, head_dim=dh, dtype=dtype, rab_buckets=rab)
    assert max(len(x) for x in segs) > 64 * 64
    check_attention(L, f"long users {dtype} dh={dh} rab={rab}")
