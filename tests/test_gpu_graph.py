"""The whole attention step captured in a HIP graph and replayed (GPU).

The library allocates nothing, synchronises nothing and issues no memset or copy on the step's
path, so plan, forward, gate + Group-LN forward and backward and the backward (dK/dV storing dS,
then dQ from it; on the fp32 path the two recomputing kernels) can be recorded on a capture
stream (torch.cuda.CUDAGraph drives hipStreamBeginCapture; every call launches on the current
stream).  Each replay runs after eager work that overwrites every output with NaN and after a
synchronisation, and must reproduce the eager step: bit for bit for every output that no float
atomic forms, and to 1e-5 of their RMS the batch sums that float atomics form in a varying
order (dgamma and dbeta: LDS atomics among a workgroup's waves; drab: atomics across
workgroups).
"""
import math

import pytest
import torch

from paper_2505_18654_amd import ops
from synth import make_layout
from synth.torch_inputs import device_inputs
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def make_step(workload):
    L = make_layout(workload)
    spec = L.spec
    H, dh = spec.heads, spec.head_dim
    T, d = L.total_tokens, spec.heads * spec.head_dim
    inp = device_inputs(L, "cuda", tensors=("q", "k", "v", "u", "dy"))
    jag = ops.Jagged(inp["offsets"], inp["seg"], inp["ts"], inp["max_seqlen"])
    q, k, v, u, dy = inp["q"], inp["k"], inp["v"], inp["u"], inp["dy"]
    rab, gamma, beta, seg = inp["rab"], inp["gamma"], inp["beta"], inp["seg"]
    out = {
        "o": torch.empty_like(q), "y": torch.empty((T, d), dtype=q.dtype, device="cuda"),
        "mean": torch.empty(T, dtype=torch.float32, device="cuda"),
        "rstd": torch.empty(T, dtype=torch.float32, device="cuda"),
        "dx": torch.empty((T, d), dtype=q.dtype, device="cuda"),
        "du": torch.empty((T, d), dtype=q.dtype, device="cuda"),
        "dgamma": torch.empty_like(gamma), "dbeta": torch.empty_like(gamma),
        "dq": torch.empty_like(q), "dk": torch.empty_like(k), "dv": torch.empty_like(v),
    }
    if rab is not None:
        out["drab"] = torch.empty_like(rab)
    ws = ops.workspace_for(ops.attn_problem(jag, q, k, v, out["o"], rab), "cuda", backward=True)
    gws = ops.gln_workspace(out["y"], gamma.shape[0])
    mfma = spec.dtype == "bf16" and dh in (32, 64, 128)
    parts = ("dkdv_keep_ds", "dq_from_ds") if mfma else ("dkdv", "dq")
    grads = (out["dq"], out["dk"], out["dv"], out.get("drab"))

    def step():
        ops.attn_plan(q, jag, workspace=ws, rab=rab)
        ops.attn_fwd(q, k, v, jag, rab, out=out["o"], workspace=ws, planned=True)
        ops.gln_fwd(out["o"].view(T, d), u, seg, gamma, beta, y=out["y"], stats=(out["mean"], out["rstd"]))
        ops.gln_bwd(dy, out["o"].view(T, d), u, seg, gamma, out["mean"], out["rstd"],
                    grads=(out["dx"], out["du"], out["dgamma"], out["dbeta"]), workspace=gws)
        for part in parts:
            ops.attn_bwd(q, k, v, out["dx"].view(T, H, dh), jag, rab, grads=grads, workspace=ws,
                         planned=True, parts=part)
    return step, out


@pytest.mark.parametrize("workload", ["tiny", "small", "mtgr_small"])
def test_graph_replay_equals_eager(workload):
    say(f"[graph] {workload}: eager step")
    step, out = make_step(workload)
    step()
    torch.cuda.synchronize()
    ref = {n: t.clone() for n, t in out.items()}
    for n, t in ref.items():
        assert torch.isfinite(t.float()).all(), n

    # warm-up on a side stream, then capture
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    say(f"[graph] {workload}: capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(3):
        for t in out.values():
            t.fill_(math.nan)
        torch.cuda.synchronize()
        say(f"[graph] {workload}: replay {r}")
        g.replay()
        torch.cuda.synchronize()
        for n, t in out.items():
            if n in ("drab", "dgamma", "dbeta"):
                want = ref[n].double()
                err = (t.double() - want).abs().max().item() / max(want.pow(2).mean().sqrt().item(), 1e-30)
                assert err <= 1e-5, (workload, r, n, err)
            else:
                assert torch.equal(t, ref[n]), (workload, r, n)
    del g
