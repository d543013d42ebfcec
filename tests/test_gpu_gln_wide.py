"""Gate + Group-LN (Eq. 6) at widths above the workloads' (d = 2048 and 4096): the backward
kernel then runs half as many waves per workgroup (and, at 8 chunks per lane, without the
next-row prefetch); and at widths that leave lanes past a row's last 16-byte chunk (d = 768 and
1000), where those lanes load the last chunk again and ignore it.  Forward and backward against
the oracle (GPU)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import ops
from tests.gpu_util import TOL, rel_err, say, tensor_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("d,dtype,groups,gate", [(2048, torch.bfloat16, 4, True), (4096, torch.bfloat16, 4, True),
                                                 (4096, torch.bfloat16, 2, False), (1024, torch.float32, 4, True),
                                                 (2048, torch.float32, 3, True), (768, torch.bfloat16, 4, True),
                                                 (1000, torch.bfloat16, 3, False), (200, torch.float32, 2, True)])
def test_wide_rows(d, dtype, groups, gate):
    rng = np.random.default_rng(d + groups)
    T = 700
    key = "bf16" if dtype == torch.bfloat16 else "fp32"
    x = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(dtype).cuda()
    u = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(dtype).cuda() if gate else None
    dy = torch.from_numpy(rng.standard_normal((T, d)).astype(np.float32)).to(dtype).cuda()
    gid_np = np.sort(rng.integers(0, groups, T)).astype(np.int8)
    gid = torch.from_numpy(gid_np).cuda()
    gamma = torch.from_numpy(1 + 0.1 * rng.standard_normal((groups, d)).astype(np.float32)).cuda()
    beta = torch.from_numpy(0.1 * rng.standard_normal((groups, d)).astype(np.float32)).cuda()
    say(f"[gln wide] d={d} {key} G={groups} gate={gate}")
    y, mean, rstd = ops.gln_fwd(x, u, gid, gamma, beta)
    ws = ops.gln_workspace(x, groups)
    dx, du, dgamma, dbeta = ops.gln_bwd(dy, x, u, gid, gamma, mean, rstd, workspace=ws)
    torch.cuda.synchronize()
    f = lambda t: None if t is None else t.float().cpu().numpy()
    ry, _, _ = oracle.gln_fwd(f(x), f(u), gid_np, f(gamma), f(beta))
    rdx, rdu, rdg, rdb = oracle.gln_bwd(f(x), f(u), gid_np, f(gamma), f(dy))
    tok = lambda got, want: tensor_err(got, want, key, TOL[key])["checked"]
    errs = {"y": tok(f(y), ry), "dx": tok(f(dx), rdx),
            "dgamma": rel_err(f(dgamma), rdg), "dbeta": rel_err(f(dbeta), rdb)}
    if gate:
        errs["du"] = tok(f(du), rdu)
    say("[gln wide] " + " ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    assert all(v <= TOL[key] for v in errs.values()), errs
