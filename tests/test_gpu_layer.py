"""The encoder layer around the path (paper_2505_18654_amd/layer.py, Sec. 4.2) against the
oracle.  As in test_gpu_parity.py every stage is checked on the device's stored input (the
Group-LNs, the projection GEMM, bias + SiLU, the attention, the output GEMM and residual, and
each backward step), at the bf16 bar of test_gpu_parity.py: per user for token tensors,
max/rms for the fp32 parameter gradients and, for the bf16 weight gradients of the GEMMs, the
bar of token tensors over the whole tensor (they are heavy-tailed: max/rms of dW_in is about
12, so their bf16 storage rounding is subtracted first).  The whole layer is also compared end
to end with the fp64 oracle layer
(oracle.layer_fwd / layer_bwd, pinned to torch autograd in test_oracle_layer.py); there the
bf16 rounding of every stored intermediate compounds; that comparison is held to a tolerance
derived from the oracle run with bf16-stored intermediates (see the end of run()).
Every stage, the products included, runs in the library's kernels."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import layer, ops
from synth import SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, make_layout
from synth.batches import round_bf16
from tests.dense_ref import operand_rounding_bounds
from tests.gpu_util import TOL, custom_layout, per_user_err, rel_err, say, tensor_err, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def params_for(d, G=4, seed=0):
    rng = np.random.default_rng(seed)
    bf = lambda a: torch.tensor(a, dtype=torch.float32).bfloat16().float().numpy().astype(np.float64)
    return dict(gamma_in=1 + 0.1 * rng.standard_normal((G, d)), beta_in=0.1 * rng.standard_normal((G, d)),
                w_in=bf(rng.standard_normal((d, 4 * d)) / np.sqrt(d)), b_in=0.1 * rng.standard_normal(4 * d),
                gamma=1 + 0.1 * rng.standard_normal((G, d)), beta=0.1 * rng.standard_normal((G, d)),
                w_out=bf(rng.standard_normal((d, d)) / np.sqrt(d)), b_out=0.1 * rng.standard_normal(d))


def to_dev(P):
    f32 = lambda a: torch.tensor(a, dtype=torch.float32, device="cuda")
    bf = lambda a: torch.tensor(a, dtype=torch.float32, device="cuda").bfloat16()
    return layer.LayerParams(f32(P["gamma_in"]), f32(P["beta_in"]), bf(P["w_in"]), f32(P["b_in"]),
                             f32(P["gamma"]), f32(P["beta"]), bf(P["w_out"]), f32(P["b_out"]))


def run(L, heads, rab_buckets, label):
    T, d = L.total_tokens, heads * L.spec.head_dim
    dh_ = d // heads
    rng = np.random.default_rng(3)
    x = torch.tensor(rng.standard_normal((T, d)), dtype=torch.float32, device="cuda").bfloat16()
    dxo = torch.tensor(rng.standard_normal((T, d)), dtype=torch.float32, device="cuda").bfloat16()
    P = params_for(d)
    rab_np = None if not rab_buckets else 0.05 * rng.standard_normal((heads, rab_buckets))
    rab = None if rab_np is None else torch.tensor(rab_np, dtype=torch.float32, device="cuda")
    jag = ops.Jagged.from_host(L.offsets, L.seg, L.ts)
    Pd = to_dev(P)
    out, ctx = layer.layer_fwd(x, jag, Pd, heads, rab)
    keep = {}
    g = layer.layer_bwd(dxo, ctx, jag, Pd, heads, rab, keep=keep)
    torch.cuda.synchronize()
    users = list(range(L.num_users))
    tol = TOL["bf16"]
    figs = {}

    def tok(got, want, extra=None):
        r = per_user_err(L, users, to_np(got).reshape(T, -1), np.asarray(want).reshape(T, -1), "bf16", tol,
                         extra)
        figs[len(figs)] = r
        if r["checked"] > tol:
            say(f"[layer] {label} above the bar: {r}")
            dump = os.environ.get("MTGR_PARITY_DUMP")
            if dump:   # the worst user's stage inputs and outputs, for offline analysis
                b = r["worst_user"]["user"]
                sl = slice(int(L.offsets[b]), int(L.offsets[b + 1]))
                np.savez(os.path.join(dump, f"layer_{label}_{len(figs)}.npz"), user=b,
                         seg=L.seg[sl], ts=L.ts[sl], got=to_np(got).reshape(T, -1)[sl],
                         want=np.asarray(want).reshape(T, -1)[sl],
                         **{k: v[sl] for k, v in D.items()}, **{"keep_" + k: v[sl] for k, v in K.items()})
        return r["checked"]
    D = {k: to_np(v) for k, v in ctx.items()}
    K = {k: to_np(v) for k, v in keep.items()}
    xn, dxn = to_np(x), to_np(dxo)
    silu = lambda z: z / (1.0 + np.exp(-z))

    def wgrad(got, want):   # bf16-stored weight gradient: the bar of token tensors, one RMS
        return tensor_err(to_np(got), np.asarray(want), "bf16", tol)["checked"]
    e = {}
    # forward, each stage on the device's stored input
    xt_r, _, _ = oracle.gln_fwd(xn, None, L.seg, P["gamma_in"], P["beta_in"])
    e["xt"] = tok(ctx["xt"], xt_r)
    e["h"] = tok(ctx["h"], D["xt"] @ P["w_in"])
    # the activation is formed in the product's epilogue from the fp32 accumulator (not from the
    # stored pre-activation h): its input is the stored xt
    e["a"] = tok(ctx["a"], silu(D["xt"] @ P["w_in"] + P["b_in"]))
    q, k, v, u = (D["a"][:, i * d:(i + 1) * d] for i in range(4))
    # The attention stage takes the layer's own activations (SiLU outputs, non-zero mean), so its
    # sums cancel: each output also gets the bound of its bf16 P / dS operand rounding.
    ob = operand_rounding_bounds(L.offsets, L.seg, L.ts, q.reshape(T, heads, dh_), k.reshape(T, heads, dh_),
                                 v.reshape(T, heads, dh_), K["do"].reshape(T, heads, dh_), rab_np)
    e["o"] = tok(ctx["o"], oracle.attn_fwd(L.offsets, L.seg, L.ts, q.reshape(T, heads, dh_), k.reshape(T, heads, dh_),
                                          v.reshape(T, heads, dh_), rab_np), ob["o"])
    o = D["o"].reshape(T, d)
    y_r, _, _ = oracle.gln_fwd(o, u, L.seg, P["gamma"], P["beta"])
    e["y"] = tok(ctx["y"], y_r)
    e["x_out"] = tok(out, D["y"] @ P["w_out"] + P["b_out"] + xn)
    # backward
    e["dy"] = tok(keep["dy"], dxn @ P["w_out"].T)
    e["w_out"] = wgrad(g["w_out"], D["y"].T @ dxn)
    e["b_out"] = rel_err(to_np(g["b_out"]), dxn.sum(0))
    do_r, du_r, dg_r, db_r = oracle.gln_bwd(o, u, L.seg, P["gamma"], K["dy"])
    e["do"] = tok(keep["do"], do_r)
    e["du"] = tok(keep["da"][:, 3 * d:], du_r)
    e["gamma"], e["beta"] = rel_err(to_np(g["gamma"]), dg_r), rel_err(to_np(g["beta"]), db_r)
    dq_r, dk_r, dv_r, drab_r = oracle.attn_bwd(L.offsets, L.seg, L.ts, q.reshape(T, heads, dh_), k.reshape(T, heads, dh_),
                                               v.reshape(T, heads, dh_), K["do"].reshape(T, heads, dh_), rab_np)
    for n, r, c in (("dq", dq_r, 0), ("dk", dk_r, 1), ("dv", dv_r, 2)):
        e[n] = tok(keep["da"][:, c * d:(c + 1) * d], r, ob[n])
    if rab is not None:
        e["rab"] = rel_err(to_np(g["rab"]), drab_r)
    z = D["h"] + P["b_in"]
    s_ = 1.0 / (1.0 + np.exp(-z))
    e["dh"] = tok(keep["dh"], K["da"] * s_ * (1.0 + z * (1.0 - s_)))
    e["w_in"] = wgrad(g["w_in"], D["xt"].T @ K["dh"])
    e["b_in"] = rel_err(to_np(g["b_in"]), K["dh"].sum(0))
    e["dxt"] = tok(keep["dxt"], K["dh"] @ P["w_in"].T)
    dxg_r, _, dgi_r, dbi_r = oracle.gln_bwd(xn, None, L.seg, P["gamma_in"], K["dxt"])
    e["dx_gln"] = tok(keep["dx_gln"], dxg_r)
    e["gamma_in"], e["beta_in"] = rel_err(to_np(g["gamma_in"]), dgi_r), rel_err(to_np(g["beta_in"]), dbi_r)
    e["dx"] = tok(g["x"], K["dx_gln"] + dxn)
    say(f"[layer] {label} stages " + " ".join(f"{k}={v:.1e}" for k, v in e.items()))
    bad = {k: v for k, v in e.items() if not v <= TOL["bf16"]}
    assert not bad, (label, bad)
    # End to end against the exact fp64 layer.  Every intermediate the device keeps is bf16, so
    # the device's outputs carry the compounded storage rounding of the whole chain.  The
    # tolerance is derived from the oracle itself: the same exact layer evaluated with
    # bf16-stored intermediates (oracle store hook) shows how far storage rounding alone moves
    # each output; the device, which rounds at the same points (plus its bf16 attention
    # operands and fp32 sums), is held to twice that plus the stage bar.
    ref, cache = oracle.layer_fwd(L.offsets, L.seg, L.ts, xn, P, heads, rab_np)
    gr = oracle.layer_bwd(L.offsets, L.seg, L.ts, dxn, cache, P, heads, rab_np)
    rb = lambda a: round_bf16(np.asarray(a)).astype(np.float64)
    ref_s, cache_s = oracle.layer_fwd(L.offsets, L.seg, L.ts, xn, P, heads, rab_np, store=rb)
    gr_s = oracle.layer_bwd(L.offsets, L.seg, L.ts, dxn, cache_s, P, heads, rab_np, store=rb)

    def lit(got, want):
        return per_user_err(L, users, np.asarray(got).reshape(T, -1), np.asarray(want).reshape(T, -1), "bf16",
                            tol)["literal"]
    ee, es, ed = {}, {}, {}
    for name, got, want, want_s in (("x_out", to_np(out), ref, ref_s), ("dx", to_np(g["x"]), gr["x"], gr_s["x"])):
        ee[name], es[name], ed[name] = lit(got, want), lit(want_s, want), lit(got, want_s)
    for name in ("w_in", "b_in", "w_out", "b_out", "gamma_in", "beta_in", "gamma", "beta") + (
            ("rab",) if rab is not None else ()):
        got = to_np(g[name])
        ee[name], es[name], ed[name] = rel_err(got, gr[name]), rel_err(gr_s[name], gr[name]), rel_err(got, gr_s[name])
    say(f"[layer] {label} end-to-end vs exact " + " ".join(f"{k}={v:.1e}" for k, v in ee.items()))
    say(f"[layer] {label} storage rounding alone " + " ".join(f"{k}={v:.1e}" for k, v in es.items()))
    say(f"[layer] {label} vs bf16-stored oracle " + " ".join(f"{k}={v:.1e}" for k, v in ed.items()))
    over = {k: (ee[k], 2 * es[k] + tol) for k in ee if not ee[k] <= 2 * es[k] + tol}
    assert not over, (label, over)


def test_layer_small_config():
    L = make_layout("small")
    run(L, L.spec.heads, 0, "small")


def test_layer_with_rab():
    U, S, R, C = SEG_USER, SEG_HIST, SEG_RT, SEG_CAND
    rng = np.random.default_rng(9)
    segs, tss = [], []
    for n_s, n_r, n_c in ((200, 30, 40), (90, 8, 5), (400, 60, 120)):
        segs.append([U] * 4 + [S] * n_s + [R] * n_r + [C] * n_c)
        tss.append([0] * 4 + sorted(rng.integers(-10**6, 0, n_s).tolist()) +
                   sorted(rng.choice(86400, n_r, replace=False).tolist()) + rng.integers(0, 86400, n_c).tolist())
    L = custom_layout(segs, tss, heads=2, head_dim=128, dtype="bf16", rab_buckets=64)
    run(L, 2, 64, "rab")
