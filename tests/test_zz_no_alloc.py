"""The allocation-free forward (mtgr_hstu_attn_fwd_noalloc), through the C ABI, against the
forward with a caller-owned workspace (mtgr_hstu_attn_fwd) on the same inputs: the same kernels
and the same plan, so the outputs must agree bit for bit.  Two calls in a row share the
library's scratch array; the second takes a smaller batch (fewer users and tokens, another head
dim, no relative bias) and must not see the first call's plan.  The second is also checked
against the oracle at the bf16 bar."""
import numpy as np
import pytest
import torch

import oracle
from paper_2505_18654_amd import hstu, ops
from synth import make_layout, make_values
from tests.gpu_util import TOL, jagged, make_inputs, per_user_err, say, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def both(inp, cand_rows=False):
    jag = jagged(inp)
    q, k, v, rab = inp["q"], inp["k"], inp["v"], inp["rab"]
    ref = ops.attn_fwd(q, k, v, jag, rab, cand_rows=cand_rows,
                       out=torch.zeros_like(q) if cand_rows else None)
    p = ops.attn_problem(jag, q, k, v, q, rab)
    if cand_rows:
        p.flags |= hstu.MTGR_FWD_CAND_ROWS
    got = torch.zeros_like(q) if cand_rows else torch.full_like(q, 777.0)
    hstu.mtgr_hstu_attn_fwd_noalloc(p, jag.offsets, jag.seg, jag.ts, q, k, v, rab, got)
    return ref, got


def test_noalloc_matches_workspace_forward_twice():
    big = make_layout("mtgr_small").subset(list(range(40)))     # 40 users, relative bias, dh 128
    small = make_layout("small").subset([0, 3, 7, 11, 30])      # 5 users, no bias, dh 64
    say(f"[noalloc] first call T={big.total_tokens}, second T={small.total_tokens}")
    a_in = make_inputs(big, all_exact=True)
    b_in = make_inputs(small, all_exact=True)
    ref_a, got_a = both(a_in)
    ref_b, got_b = both(b_in)
    torch.cuda.synchronize()
    assert torch.equal(got_a, ref_a), "first call differs from mtgr_hstu_attn_fwd"
    assert torch.equal(got_b, ref_b), "second (smaller) call differs from mtgr_hstu_attn_fwd"
    vals = make_values(small, tensors=("q", "k", "v"))
    want = oracle.attn_fwd(small.offsets, small.seg, small.ts, vals["q"], vals["k"], vals["v"])
    e = per_user_err(small, list(range(small.num_users)), to_np(got_b), want, "bf16", TOL["bf16"])
    say(f"[noalloc] second call vs oracle: checked {e['checked']:.2e} literal {e['literal']:.2e}")
    assert e["checked"] <= TOL["bf16"]
    # a third call with candidate rows only, on the larger batch again
    ref_c, got_c = both(a_in, cand_rows=True)
    torch.cuda.synchronize()
    assert torch.equal(got_c, ref_c), "candidate-rows call differs"
