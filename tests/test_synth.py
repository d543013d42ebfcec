"""The synthetic generator: determinism, segment order, length bounds (CPU only)."""
import numpy as np
import pytest

from synth import (CONFIGS, SEG_CAND, SEG_HIST, SEG_RT, SEG_USER, WINDOW, bf16_bits_to_f32,
                   f32_to_bf16_bits, make_layout, make_values)

BOUNDS = {  # (user tokens, history lo/hi, real-time lo/hi, candidates lo/hi)
    "tiny": (2, 8, 24, 2, 6, 1, 4),
    "small": (4, 50, 300, 5, 30, 1, 16),
    "mtgr_small": (8, 0, 900, 10, 64, 8, 64),
    "mtgr_large": (16, 0, 3000, 0, 128, 1, 128),
    "serving": (8, 200, 2000, 1, 128, 100, 500),
}


@pytest.mark.parametrize("config", list(CONFIGS))
def test_layout_shape_and_order(config):
    L = make_layout(config)
    L2 = make_layout(config)
    np.testing.assert_array_equal(L.offsets, L2.offsets)
    np.testing.assert_array_equal(L.ts, L2.ts)
    nu, hlo, hhi, rlo, rhi, clo, chi = BOUNDS[config]
    assert L.num_users == CONFIGS[config].num_users
    for b in range(L.num_users):
        s, t = L.seg[L.user_slice(b)], L.ts[L.user_slice(b)]
        assert np.all(np.diff(s) >= 0)                       # [U | S | R | I]
        c = [int(np.sum(s == g)) for g in range(4)]
        assert c[0] == nu and hlo <= c[1] <= hhi and rlo <= c[2] <= rhi and clo <= c[3] <= chi
        assert np.all(t[s == SEG_USER] == 0)
        assert np.all(t[s == SEG_HIST] < 0)
        rt = t[s == SEG_RT]
        assert np.all(np.diff(rt) > 0) and np.all((rt >= 0) & (rt < WINDOW))
        cand = t[s == SEG_CAND]
        if CONFIGS[config].serving:
            assert np.all(cand == WINDOW)
        else:
            assert np.all((cand >= 0) & (cand < WINDOW))
    if config == "mtgr_small":
        assert L.max_seqlen <= 1024
    if config == "mtgr_large":
        n = np.diff(L.offsets)
        assert n.min() < 20 and n.max() > 2000


def test_subset_values_match_full_draw():
    L = make_layout("small")
    full = make_values(L)
    users = [5, 1, 17]
    sub = L.subset(users)
    part = make_values(sub)
    idx = np.concatenate([np.arange(L.offsets[b], L.offsets[b + 1]) for b in users])
    for name in ("q", "k", "v", "u", "do", "dy"):
        np.testing.assert_array_equal(full[name][idx], part[name])
    np.testing.assert_array_equal(full["gamma"], part["gamma"])


def test_bf16_rounding():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -3.14159, 0.0, 65504.0], np.float32)
    r = bf16_bits_to_f32(f32_to_bf16_bits(x))
    assert r[0] == 1.0 and r[1] == 1.0                # tie rounds to even
    assert r[2] == 1.0 + 4 * 2**-8
    assert abs(r[3] - x[3]) <= 2**-7 * 4
    vals = make_values(make_layout("small"), users=[0], tensors=("q",))
    assert np.array_equal(vals["q"], bf16_bits_to_f32(f32_to_bf16_bits(vals["q"])))


def test_subset_of_subset_keeps_original_users():
    L = make_layout("small")
    a = L.subset([7, 3, 20])
    b = a.subset([2, 0])
    np.testing.assert_array_equal(make_values(b)["q"], make_values(L.subset([20, 7]))["q"])
