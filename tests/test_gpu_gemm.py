"""The encoder layer's dense products (mtgr_gemm_bf16) and residual add (mtgr_add) against
their plain definitions, element by element.

The reference of a product is the fp64 product of the same bf16 inputs (numpy on the CPU).
Each element is held to a bound that follows from the arithmetic, not a tuned tolerance:
the kernel forms exact bf16 x bf16 products, adds them in fp32 (K terms, then at most
`splits` partial sums), applies the epilogue in fp32 and rounds once to bf16, so

    |got - ref| <= h(got) + g * S,   g = (K + splits + 4) 2^-24,   S = |A| |B|  (fp64)

with h(x) the half-ulp of bf16 at x (the storage rounding).  The epilogues add their own
roundings: bias + residual two fp32 additions; bias + SiLU the fp32 rounding of z = AB + b, the
SiLU's sensitivity to z (|silu'| < 1.1) and the hardware exp2 / reciprocal (relative error a
few fp32 ulps of |z| + 1).  The column sums (the bias gradient) are fp32 sums over K held to
g * sum |B|.  The residual add is bit-exact against the fp32 sum rounded to bf16."""
import numpy as np
import pytest
import torch

from paper_2505_18654_amd import hstu, ops
from tests.dense_ref import bf16_half_ulp
from tests.gpu_util import say

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def rand_bf16(shape, seed, scale=1.0, cols=None):
    """Seeded bf16 matrix on the device; with `cols` wider than shape[1] the result is a column
    slice of a wider matrix (a strided operand)."""
    g = torch.Generator().manual_seed(seed)
    w = cols or shape[1]
    full = (torch.randn((shape[0], w), generator=g) * scale).bfloat16()
    return full.cuda()[:, :shape[1]]


def f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def splits_of(layout, M, N, K):
    if layout != hstu.MTGR_GEMM_TN:
        return 1
    ws = hstu.mtgr_gemm_workspace_size(layout, M, N, K)
    return max(1, round(ws / ((M * N + N) * 4)))


def assert_within(name, got, ref, bound):
    err = np.abs(got - ref)
    ratio = float(np.max(err / bound)) if err.size else 0.0
    say(f"[gemm] {name}: max |got - ref| / bound = {ratio:.3f} (max err {float(err.max()) if err.size else 0:.2e})")
    assert np.isfinite(got).all(), name
    assert ratio <= 1.0, (name, ratio)


def product_ref(layout, A, B):
    a, b = f64(A), f64(B)
    if layout == "nn":
        return a @ b, np.abs(a) @ np.abs(b)
    if layout == "nt":
        return a @ b.T, np.abs(a) @ np.abs(b).T
    return a.T @ b, np.abs(a).T @ np.abs(b)


@pytest.mark.parametrize("layout, M, N, K", [
    ("nn", 1, 128, 32), ("nn", 256, 128, 32), ("nn", 1000, 384, 96), ("nn", 4099, 2048, 512),
    ("nt", 999, 256, 1024), ("nt", 37, 512, 2048), ("nt", 4096, 1024, 4096),
    ("tn", 256, 1024, 1000), ("tn", 512, 128, 17), ("tn", 256, 128, 40000), ("tn", 768, 3072, 4099),
    ("tn", 1024, 4096, 1),
    # edges that are not whole 256 x 256 tiles: N, and M of A^T B, only multiples of 8
    ("nn", 300, 136, 64), ("nt", 513, 264, 96), ("tn", 264, 1000, 777), ("tn", 8, 8, 5),
])
def test_gemm_plain(layout, M, N, K):
    say(f"[gemm] plain {layout} M={M} N={N} K={K}")
    if layout == "nn":
        A, B = rand_bf16((M, K), 1), rand_bf16((K, N), 2)
    elif layout == "nt":
        A, B = rand_bf16((M, K), 1), rand_bf16((N, K), 2)
    else:
        A, B = rand_bf16((K, M), 1), rand_bf16((K, N), 2)
    colsum = torch.full((N,), float("nan"), device="cuda") if layout == "tn" else None
    C = ops.gemm(A, B, layout, colsum=colsum)
    torch.cuda.synchronize()
    ref, S = product_ref(layout, A, B)
    got = f64(C)
    g = (K + splits_of(ops._GEMM_LAYOUTS[layout], M, N, K) + 4) * U
    assert_within(f"{layout} {M}x{N}x{K}", got, ref, bf16_half_ulp(got) + g * S + 1e-30)
    if colsum is not None:
        b = f64(B)
        assert_within(f"{layout} colsum", colsum.cpu().numpy().astype(np.float64), b.sum(0),
                      g * np.abs(b).sum(0) + 1e-30)


def test_gemm_split_sums_are_deterministic():
    A, B = rand_bf16((30000, 512), 3), rand_bf16((30000, 2048), 4)
    cs1, cs2 = torch.empty(2048, device="cuda"), torch.empty(2048, device="cuda")
    C1 = ops.gemm(A, B, "tn", colsum=cs1)
    C2 = ops.gemm(A, B, "tn", colsum=cs2)
    torch.cuda.synchronize()
    assert torch.equal(C1, C2) and torch.equal(cs1, cs2)


@pytest.mark.parametrize("M, N, K", [(777, 1024, 256), (8192, 2048, 512), (3, 128, 64)])
def test_gemm_bias_silu(M, N, K):
    say(f"[gemm] bias+silu M={M} N={N} K={K}")
    A, B = rand_bf16((M, K), 5), rand_bf16((K, N), 6, scale=K ** -0.5 * 2)
    bias = torch.randn(N, generator=torch.Generator().manual_seed(7)).cuda() * 0.5
    h = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    a = torch.empty_like(h)
    ops.gemm(A, B, "nn", out=h, bias=bias, silu_out=a)
    torch.cuda.synchronize()
    ref, S = product_ref("nn", A, B)
    g = (K + 5) * U
    got_h = f64(h)
    assert_within("pre-activation", got_h, ref, bf16_half_ulp(got_h) + g * S + 1e-30)
    z = ref + f64(bias[None, :])
    silu = z / (1.0 + np.exp(-z))
    got_a = f64(a)
    bound = bf16_half_ulp(got_a) + 1.1 * (g * S + 2 * U * np.abs(z)) + 16 * U * (np.abs(z) + 1) * np.abs(silu)
    assert_within("silu", got_a, silu, bound + 1e-30)


@pytest.mark.parametrize("M, N, K", [(555, 256, 256), (4096, 1024, 1024)])
def test_gemm_bias_residual(M, N, K):
    say(f"[gemm] bias+residual M={M} N={N} K={K}")
    A, B = rand_bf16((M, K), 8), rand_bf16((K, N), 9, scale=K ** -0.5)
    R = rand_bf16((M, N), 10)
    bias = torch.randn(N, generator=torch.Generator().manual_seed(11)).cuda() * 0.1
    C = ops.gemm(A, B, "nn", bias=bias, residual=R)
    torch.cuda.synchronize()
    ref, S = product_ref("nn", A, B)
    br = f64(bias[None, :]) + f64(R)
    want = ref + br
    got = f64(C)
    bound = bf16_half_ulp(got) + (K + 5) * U * S + 2 * U * (np.abs(br) + np.abs(want))
    assert_within("bias+residual", got, want, bound + 1e-30)


def test_gemm_strided_operands():
    """Operands and results as column slices of wider matrices, as in the layer (Q | K | V | U
    views of one activation)."""
    M, N, K = 600, 256, 512
    A = rand_bf16((M, K), 12, cols=K + 64)
    B = rand_bf16((K, N), 13, cols=N + 256)
    Cfull = torch.full((M, N + 128), 7.0, dtype=torch.bfloat16, device="cuda")
    C = Cfull[:, 64:64 + N]
    ops.gemm(A, B, "nn", out=C)
    Bt = rand_bf16((N, K), 14, cols=K + 32)
    D = ops.gemm(A, Bt, "nt")
    At = rand_bf16((K, M - 88), 15, cols=M + 40)
    G = rand_bf16((K, N), 16, cols=4 * N)
    cs = torch.empty(N, device="cuda")
    E = ops.gemm(At, G, "tn", colsum=cs)
    torch.cuda.synchronize()
    for name, lay, a, b, got in (("nn", "nn", A, B, C), ("nt", "nt", A, Bt, D), ("tn", "tn", At, G, E)):
        ref, S = product_ref(lay, a, b)
        g = f64(got)
        assert_within(f"strided {name}", g, ref, bf16_half_ulp(g) + (a.shape[0 if lay == "tn" else 1] + 70) * U * S
                      + 1e-30)
    untouched = torch.cat([Cfull[:, :64], Cfull[:, 64 + N:]], 1)
    assert bool((untouched == 7.0).all())


def test_add_is_exact():
    a, b = rand_bf16((1001, 512), 17), rand_bf16((1001, 512), 18, cols=640)
    out = ops.add(a, b)
    torch.cuda.synchronize()
    want = (a.cpu().float() + b.cpu().float()).bfloat16()
    assert torch.equal(out.cpu(), want)
