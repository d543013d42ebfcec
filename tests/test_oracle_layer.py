"""Pins of the encoder-layer oracle (oracle.layer_fwd / layer_bwd, Sec. 4.2 read as
GroupLN -> fused linear + SiLU -> Eq. 5 attention -> gate + GroupLN -> linear + residual):
the forward against a dense torch fp64 formulation written independently (tests/dense_ref.py
for the attention and the Group-LN), and every gradient of the hand-chained backward against
torch autograd of that formulation."""
import numpy as np
import pytest
import torch

import oracle
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER
from tests.dense_ref import dense_attention, dense_gln


def tiny_batch(seed=0, heads=2, dh=8, G=4, rab=True):
    rng = np.random.default_rng(seed)
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    segs = [[U, U, S, S, S, R, R, C, C], [U, S, S, R, C, C, C], [S, S, S, S]]
    seg = np.concatenate([np.array(s, np.int8) for s in segs])
    ts = np.concatenate([np.array([0, 0, -50, -30, -10, 5, 9, 7, 12]), np.array([0, -4, -2, 3, 1, 8, 9]),
                         np.array([-9, -7, -5, -3])]).astype(np.int32)
    offsets = np.array([0, 9, 16, 20])
    T, d = len(seg), heads * dh
    x = rng.standard_normal((T, d))
    params = dict(gamma_in=1 + 0.1 * rng.standard_normal((G, d)), beta_in=0.1 * rng.standard_normal((G, d)),
                  w_in=rng.standard_normal((d, 4 * d)) / np.sqrt(d), b_in=0.1 * rng.standard_normal(4 * d),
                  gamma=1 + 0.1 * rng.standard_normal((G, d)), beta=0.1 * rng.standard_normal((G, d)),
                  w_out=rng.standard_normal((d, d)) / np.sqrt(d), b_out=0.1 * rng.standard_normal(d))
    rab_v = 0.3 * rng.standard_normal((heads, 64)) if rab else None
    return offsets, seg, ts, x, params, rab_v


def dense_layer(offsets, seg, ts, x, P, heads, rab, alpha=1.0, eps=1e-5):
    T, d = x.shape
    dh = d // heads
    xt = dense_gln(x, None, seg, P["gamma_in"], P["beta_in"], eps)
    a = torch.nn.functional.silu(xt @ P["w_in"] + P["b_in"])
    q, k, v, u = (a[:, i * d:(i + 1) * d] for i in range(4))
    o = dense_attention(offsets, seg, ts, q.reshape(T, heads, dh), k.reshape(T, heads, dh),
                        v.reshape(T, heads, dh), rab, alpha).reshape(T, d)
    y = dense_gln(o, u, seg, P["gamma"], P["beta"], eps)
    return y @ P["w_out"] + P["b_out"] + x


@pytest.mark.parametrize("with_rab", [False, True])
def test_layer_forward_and_gradients_match_autograd(with_rab):
    heads = 2
    offsets, seg, ts, x, params, rab = tiny_batch(rab=with_rab, heads=heads)
    out, cache = oracle.layer_fwd(offsets, seg, ts, x, params, heads, rab)
    tx = torch.tensor(x, dtype=torch.float64, requires_grad=True)
    tP = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in params.items()}
    trab = None if rab is None else torch.tensor(rab, dtype=torch.float64, requires_grad=True)
    ref = dense_layer(offsets, seg, ts, tx, tP, heads, trab)
    np.testing.assert_allclose(out, ref.detach().numpy(), rtol=1e-10, atol=1e-12)
    dout = np.random.default_rng(5).standard_normal(out.shape)
    ref.backward(torch.tensor(dout))
    g = oracle.layer_bwd(offsets, seg, ts, dout, cache, params, heads, rab)
    np.testing.assert_allclose(g["x"], tx.grad.numpy(), rtol=1e-9, atol=1e-11)
    for name, t in tP.items():
        np.testing.assert_allclose(g[name], t.grad.numpy(), rtol=1e-9, atol=1e-11, err_msg=name)
    if with_rab:
        np.testing.assert_allclose(g["rab"], trab.grad.numpy(), rtol=1e-9, atol=1e-11)


def test_storage_hook_sees_each_kept_intermediate_once():
    """The store hook (bf16-stored intermediates, Sec. 5's mixed precision) is applied exactly to
    the values the layer keeps between steps: recorded with an identity hook, they are the exact
    layer's intermediates, in order, and the results are unchanged."""
    heads = 2
    offsets, seg, ts, x, params, rab = tiny_batch(heads=heads)
    out, cache = oracle.layer_fwd(offsets, seg, ts, x, params, heads, rab)
    dout = np.random.default_rng(6).standard_normal(out.shape)
    g = oracle.layer_bwd(offsets, seg, ts, dout, cache, params, heads, rab)
    seen = []

    def rec(a):
        seen.append(np.array(a))
        return a
    out2, cache2 = oracle.layer_fwd(offsets, seg, ts, x, params, heads, rab, store=rec)
    np.testing.assert_array_equal(out2, out)
    fwd = [cache["xt"], cache["a"], cache["h"] - params["b_in"], cache["o"], cache["y"], out]
    assert len(seen) == len(fwd)
    for s, want in zip(seen, fwd):
        np.testing.assert_allclose(s, want, rtol=0, atol=1e-12)
    seen.clear()
    g2 = oracle.layer_bwd(offsets, seg, ts, dout, cache2, params, heads, rab, store=rec)
    for k in g:
        np.testing.assert_array_equal(g2[k], g[k])
    # w_out grad, dy, do, du, [dq|dk|dv|du], dh, w_in grad, dxt, dx of the input Group-LN, dx
    assert len(seen) == 10
    np.testing.assert_array_equal(seen[0], g["w_out"])
    np.testing.assert_array_equal(seen[6], g["w_in"])
    np.testing.assert_array_equal(seen[-1], g["x"])
    np.testing.assert_allclose(seen[-2] + dout, g["x"], rtol=0, atol=1e-12)


def test_storage_hook_rounds_to_bf16():
    from synth.batches import round_bf16
    heads = 2
    offsets, seg, ts, x, params, rab = tiny_batch(heads=heads)
    rb = lambda a: round_bf16(np.asarray(a)).astype(np.float64)
    out, cache = oracle.layer_fwd(offsets, seg, ts, x, params, heads, rab, store=rb)
    for name in ("xt", "a", "o", "y"):
        np.testing.assert_array_equal(rb(cache[name]), cache[name], err_msg=name)
    np.testing.assert_array_equal(rb(out), out)
    exact, _ = oracle.layer_fwd(offsets, seg, ts, x, params, heads, rab)
    rel = np.max(np.abs(out - exact)) / np.sqrt(np.mean(exact ** 2))
    assert 0 < rel < 0.05
    g = oracle.layer_bwd(offsets, seg, ts, np.ones_like(out), cache, params, heads, rab, store=rb)
    for name in ("x", "w_in", "w_out"):
        np.testing.assert_array_equal(rb(g[name]), g[name], err_msg=name)
