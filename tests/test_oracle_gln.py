"""Pins of the oracle's gate + Group-LayerNorm (Eq. 6 without the MLP), CPU only."""
import numpy as np
import pytest
import torch

import oracle
from tests.dense_ref import dense_gln


def case(seed, T=37, d=24, G=4, gate=True):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, d))
    u = rng.standard_normal((T, d)) if gate else None
    gid = rng.integers(0, G, T).astype(np.int8)
    gamma = 1.0 + 0.3 * rng.standard_normal((G, d))
    beta = 0.3 * rng.standard_normal((G, d))
    dy = rng.standard_normal((T, d))
    return x, u, gid, gamma, beta, dy


def test_single_group_is_library_layer_norm():
    x, u, gid, gamma, beta, _ = case(0, G=1)
    y, mean, rstd = oracle.gln_fwd(x, u, gid, gamma, beta, eps=1e-5)
    z = torch.tensor(x * u)
    want = torch.nn.functional.layer_norm(z, (z.shape[1],), torch.tensor(gamma[0]),
                                          torch.tensor(beta[0]), eps=1e-5)
    np.testing.assert_allclose(y, want.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(mean, (x * u).mean(1), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(rstd, 1 / np.sqrt((x * u).var(1) + 1e-5), rtol=1e-12)


@pytest.mark.parametrize("gate", [True, False])
def test_groups_gather_affine(gate):
    x, u, gid, gamma, beta, _ = case(1, gate=gate)
    y, _, _ = oracle.gln_fwd(x, u, gid, gamma, beta)
    z = torch.tensor(x * u if gate else x)
    zn = torch.nn.functional.layer_norm(z, (z.shape[1],), eps=1e-5).numpy()
    for t in range(len(gid)):
        np.testing.assert_allclose(y[t], zn[t] * gamma[gid[t]] + beta[gid[t]], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("gate", [True, False])
def test_bwd_matches_autograd(gate):
    x, u, gid, gamma, beta, dy = case(2, gate=gate)
    dx, du, dg, db = oracle.gln_bwd(x, u, gid, gamma, dy)
    tx = torch.tensor(x, requires_grad=True)
    tu = torch.tensor(u, requires_grad=True) if gate else None
    tg = torch.tensor(gamma, requires_grad=True)
    tb = torch.tensor(beta, requires_grad=True)
    dense_gln(tx, tu, gid, tg, tb).backward(torch.tensor(dy))
    np.testing.assert_allclose(dx, tx.grad.numpy(), rtol=1e-10, atol=1e-11)
    if gate:
        np.testing.assert_allclose(du, tu.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_bwd_finite_differences():
    x, u, gid, gamma, beta, dy = case(3, T=9, d=16)
    dx, du, dg, db = oracle.gln_bwd(x, u, gid, gamma, dy)
    h = 1e-6
    rng = np.random.default_rng(0)
    args = {"x": x, "u": u, "gamma": gamma, "beta": beta}
    grads = {"x": dx, "u": du, "gamma": dg, "beta": db}
    for name in args:
        delta = rng.standard_normal(args[name].shape)
        p, m = dict(args), dict(args)
        p[name] = args[name] + h * delta
        m[name] = args[name] - h * delta
        yp = oracle.gln_fwd(p["x"], p["u"], gid, p["gamma"], p["beta"])[0]
        ym = oracle.gln_fwd(m["x"], m["u"], gid, m["gamma"], m["beta"])[0]
        numeric = np.sum(dy * (yp - ym)) / (2 * h)
        analytic = np.sum(grads[name] * delta)
        assert abs(numeric - analytic) <= 1e-6 * max(1.0, abs(analytic)), name


def test_token_independence():
    """Each token is normalised over its own features only (no pooling across tokens)."""
    x, u, gid, gamma, beta, _ = case(4)
    y1 = oracle.gln_fwd(x, u, gid, gamma, beta)[0]
    x2 = x.copy()
    x2[5] *= 10.0
    y2 = oracle.gln_fwd(x2, u, gid, gamma, beta)[0]
    others = np.arange(len(gid)) != 5
    np.testing.assert_array_equal(y1[others], y2[others])


def test_constant_row_gives_beta():
    x, u, gid, gamma, beta, _ = case(5, gate=False)
    x[3] = 2.5
    y = oracle.gln_fwd(x, None, gid, gamma, beta)[0]
    np.testing.assert_allclose(y[3], beta[gid[3]], rtol=0, atol=1e-12)
