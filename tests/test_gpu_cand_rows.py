"""Candidate-rows forward (MTGR_FWD_CAND_ROWS): the one pass per user that scores all of its
candidates (user sample aggregation, Sec. 4.1, Eq. 3).  Through the C ABI:
  - every candidate row equals the full forward's row bit for bit (same tiles, same order);
  - every other row of the output is left untouched (a sentinel survives);
  - the candidate rows meet the oracle bar of test_gpu_parity.py.
Covered: serving users (candidates at the end, all seeing every RT token), candidates placed
between history and RT tokens (the mask depends on seg and ts only), users without
candidates, only candidates, ragged tails, the fp32 path and a relative bias."""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout, make_values
from tests.gpu_util import TOL, custom_layout, jagged, make_inputs, per_user_err, say, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def layouts():
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(21)
    segs, tss = [], []
    # candidates at the end, before the RT block, none, only candidates, a ragged short user
    for n_s, n_r, n_c, where in ((300, 40, 150, "end"), (200, 30, 90, "mid"), (130, 10, 0, "end"),
                                (0, 0, 70, "end"), (5, 3, 2, "end"), (60, 70, 140, "mid")):
        hist = sorted(rng.integers(-10**6, 0, n_s).tolist())
        rt = sorted(rng.choice(86400, n_r, replace=False).tolist())
        cand = rng.integers(0, 86400, n_c).tolist()
        if where == "end":
            segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
            tss.append([0] * 4 + hist + rt + cand)
        else:
            segs.append([U] * 4 + [S] * n_s + [C] * n_c + [R] * n_r)
            tss.append([0] * 4 + hist + cand + rt)
    return segs, tss


def run_case(L, inp, label):
    jag = jagged(inp)
    q, k, v, rab = inp["q"], inp["k"], inp["v"], inp["rab"]
    full = ops.attn_fwd(q, k, v, jag, rab)
    sentinel = torch.full_like(q, 1234.0)
    got = ops.attn_fwd(q, k, v, jag, rab, out=sentinel.clone(), cand_rows=True)
    torch.cuda.synchronize()
    cand = torch.as_tensor(L.seg == SEG_CAND, device=q.device)
    assert torch.equal(got[cand], full[cand]), f"{label}: candidate rows differ from the full forward"
    assert torch.equal(got[~cand], sentinel[~cand]), f"{label}: a non-candidate row was written"
    users = list(range(L.num_users))
    vals = make_values(L)
    ref = oracle.attn_fwd(L.offsets, L.seg, L.ts, vals["q"], vals["k"], vals["v"], inp["rab_np"])
    g = to_np(got)
    c = (L.seg == SEG_CAND)
    g_c, r_c = np.where(c[:, None, None], g, ref), ref   # non-candidate rows compare equal
    err = per_user_err(L, users, g_c, r_c, L.spec.dtype, TOL[L.spec.dtype])["checked"]
    say(f"[cand_rows] {label} candidates={int(c.sum())} err={err:.2e}")
    assert err <= TOL[L.spec.dtype], (label, err)


@pytest.mark.parametrize("dtype,dh,rab", [("bf16", 128, 0), ("bf16", 64, 64), ("bf16", 32, 0), ("fp32", 64, 0)])
def test_custom_layouts(dtype, dh, rab):
    segs, tss = layouts()
    L = custom_layout(segs, tss, heads=2, head_dim=dh, dtype=dtype, rab_buckets=rab)
    run_case(L, make_inputs(L, all_exact=True), f"custom-{dtype}-{dh}-rab{rab}")


def test_serving_subset():
    L = make_layout("serving")
    users = [0, 1, int(np.argmax(np.diff(L.offsets))), L.num_users - 1]
    sub = L.subset(sorted(set(users)))
    run_case(sub, make_inputs(sub, all_exact=True), "serving-subset")


def test_long_users():
    """Users longer than one 64-tile window of the tile walker (8,300 and 4,812 tokens), with
    3,436 and 200 candidates."""
    from tests.test_gpu_limits import long_users
    segs, tss = long_users()
    L = custom_layout(segs, tss, heads=2, head_dim=128, dtype="bf16", rab_buckets=64)
    run_case(L, make_inputs(L, all_exact=True), "long-bf16-128-rab64")
