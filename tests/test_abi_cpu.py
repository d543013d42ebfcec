"""The C ABI on the CPU: the library loads, exports every declared symbol, and rejects
bad arguments with a status before touching the device (CPU only, no GPU calls)."""
import ctypes
import os
import re

import pytest

from paper_2505_18654_amd import hstu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]

BF16, FP32 = hstu.MTGR_DTYPE_BF16, hstu.MTGR_DTYPE_FP32
FAKE = 0x7f0000000000           # 256-byte aligned non-NULL address, never dereferenced


def declared_functions():
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mtgr_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert "mtgr_hstu_attn_fwd" in names and "mtgr_group_layernorm_bwd" in names
    assert "mtgr_embedding_lookup" in names
    L = hstu.lib()
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(hstu.EXPORTED)


def test_version_and_status_strings():
    assert hstu.mtgr_version() == 100
    for s in range(6):
        assert hstu.mtgr_status_string(s)
    assert hstu.mtgr_status_string(99) == "unknown status"


def test_struct_layout_matches_header():
    assert ctypes.sizeof(hstu.HstuProblem) == 72
    assert ctypes.sizeof(hstu.GlnProblem) == 48
    assert hstu.HstuProblem.ld_q.offset == 40


def prob(**kw):
    base = dict(num_users=4, total_tokens=100, max_seqlen=40, heads=2, head_dim=64, dtype=BF16)
    base.update(kw)
    return hstu.attn_problem(**base)


@pytest.mark.parametrize("mutate,status", [
    (dict(head_dim=48), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(head_dim=8), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(num_users=2**20, total_tokens=2**30, max_seqlen=1000, heads=200),
     hstu.MTGR_ERROR_UNSUPPORTED),                               # 2^24 or more work items
    (dict(dtype=7), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(heads=0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(heads=256), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(num_users=-1), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(total_tokens=-5), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(total_tokens=2**31), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(max_seqlen=0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(max_seqlen=300000), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(rab_buckets=65), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(ld_q=100), hstu.MTGR_ERROR_INVALID_ARGUMENT),        # below H*dh = 128
    (dict(ld_k=132), hstu.MTGR_ERROR_INVALID_ARGUMENT),        # 264 bytes: not 16-byte multiple
    (dict(ld_v=(1 << 24) + 8), hstu.MTGR_ERROR_UNSUPPORTED),   # above MTGR_MAX_LD
    (dict(alpha=float("nan")), hstu.MTGR_ERROR_INVALID_ARGUMENT),
])
def test_problem_validation(mutate, status):
    p = prob(**mutate)
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_hstu_attn_workspace_size(p)
    assert e.value.status == status
    assert hstu.mtgr_last_error_message()


def test_unknown_flags_rejected():
    p = prob()
    p.flags = 64
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_hstu_attn_workspace_size(p)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT


def test_head_dim_16_supported_in_both_dtypes():
    """head_dim 16 runs on the vector-ALU kernels (fp32, and bf16 storage with fp32
    arithmetic): no stored-dS region, so both workspace sizes are equal."""
    for dt in (FP32, BF16):
        p = prob(dtype=dt, head_dim=16)
        fwd_bytes = hstu.mtgr_hstu_attn_workspace_size(p)
        assert fwd_bytes > 0
        assert hstu.mtgr_hstu_attn_workspace_size(p, backward=True) == fwd_bytes
    assert (hstu.mtgr_hstu_attn_workspace_size(prob(head_dim=32), backward=True) >
            hstu.mtgr_hstu_attn_workspace_size(prob(head_dim=32)))


def test_largest_accepted_work_list():
    """Just below 2^24 workgroups is accepted; the launch bound is checked on the host."""
    ok = prob(num_users=1000, total_tokens=2**24, max_seqlen=2000, heads=64)
    assert hstu.mtgr_hstu_attn_workspace_size(ok) > 0


def test_workspace_grows_with_problem():
    a = hstu.mtgr_hstu_attn_workspace_size(prob())
    b = hstu.mtgr_hstu_attn_workspace_size(prob(num_users=40, total_tokens=1000))
    assert 0 < a < b
    assert a % 256 == 0
    assert hstu.mtgr_hstu_attn_workspace_size(prob(num_users=0, total_tokens=0)) == 0


def fwd(p, **over):
    args = dict(offsets=FAKE, seg=FAKE, ts=FAKE, q=FAKE, k=FAKE, v=FAKE, rab=None, out=FAKE,
                workspace=FAKE, workspace_bytes=1 << 30)
    args.update(over)
    hstu.mtgr_hstu_attn_fwd(p, args["offsets"], args["seg"], args["ts"], args["q"], args["k"],
                            args["v"], args["rab"], args["out"], args["workspace"],
                            args["workspace_bytes"], 0)


@pytest.mark.parametrize("name", ["offsets", "seg", "ts", "q", "k", "v", "out", "workspace"])
def test_fwd_null_pointers(name):
    with pytest.raises(hstu.MtgrError) as e:
        fwd(prob(), **{name: None})
    assert e.value.status == hstu.MTGR_ERROR_NULL_POINTER
    assert name in hstu.mtgr_last_error_message()


@pytest.mark.parametrize("name", ["q", "k", "v", "out"])
def test_fwd_misaligned_tensors(name):
    with pytest.raises(hstu.MtgrError) as e:
        fwd(prob(), **{name: FAKE + 2})
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT


def test_fwd_workspace_checks():
    p = prob()
    need = hstu.mtgr_hstu_attn_workspace_size(p)
    with pytest.raises(hstu.MtgrError) as e:
        fwd(p, workspace_bytes=need - 1)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL
    with pytest.raises(hstu.MtgrError) as e:
        fwd(p, workspace=FAKE + 16)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT


def test_fwd_rab_without_buckets():
    with pytest.raises(hstu.MtgrError) as e:
        fwd(prob(), rab=FAKE)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT


def test_empty_batches_are_noops():
    for p in (prob(num_users=0, total_tokens=0), prob(num_users=3, total_tokens=0)):
        fwd(p, offsets=FAKE, seg=None, ts=None, q=None, k=None, v=None, out=None, workspace=None,
            workspace_bytes=0)
        hstu.mtgr_hstu_attn_bwd(p, FAKE, None, None, None, None, None, None, None, None, None, None,
                                None, None, 0, 0)


def test_bwd_argument_checks():
    p = prob(rab_buckets=64)
    args = [FAKE] * 12
    with pytest.raises(hstu.MtgrError) as e:       # drab without rab
        hstu.mtgr_hstu_attn_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE,
                                FAKE, FAKE, 1 << 30, 0)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    with pytest.raises(hstu.MtgrError) as e:       # missing dout
        hstu.mtgr_hstu_attn_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE,
                                FAKE, FAKE, 1 << 30, 0)
    assert e.value.status == hstu.MTGR_ERROR_NULL_POINTER
    assert len(args) == 12


def test_backward_workspace_sizes():
    """backward = 1 adds the stored-dS blocks for bf16: H * ntile * (T/64 + B) blocks of 8 KB
    on top of the plan; fp32 always recomputes, so its size does not grow."""
    p = prob(num_users=4, total_tokens=100, max_seqlen=40, heads=2, head_dim=64)
    base = hstu.mtgr_hstu_attn_workspace_size(p, False)
    big = hstu.mtgr_hstu_attn_workspace_size(p, True)
    ntile = (40 + 63) // 64
    assert big - base == 2 * ntile * ((100 + 63) // 64 + 4) * 64 * 64 * 2
    pf = prob(dtype=FP32, head_dim=64)
    assert hstu.mtgr_hstu_attn_workspace_size(pf, True) == hstu.mtgr_hstu_attn_workspace_size(pf, False)


def bwd_call(p, drab=None, workspace_bytes=1 << 30):
    hstu.mtgr_hstu_attn_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE if p.num_rab_buckets else None,
                            FAKE, FAKE, FAKE, FAKE, drab, FAKE, workspace_bytes, 0)


@pytest.mark.parametrize("flags,drab,status", [
    (hstu.MTGR_BWD_KEEP_DS, None, hstu.MTGR_ERROR_INVALID_ARGUMENT),            # needs SKIP_DQ
    (hstu.MTGR_BWD_DS_READY, None, hstu.MTGR_ERROR_INVALID_ARGUMENT),           # needs SKIP_DKDV
    (hstu.MTGR_BWD_DS_READY | hstu.MTGR_BWD_SKIP_DKDV, FAKE, hstu.MTGR_ERROR_INVALID_ARGUMENT),
])
def test_stored_ds_flag_checks(flags, drab, status):
    p = prob(rab_buckets=64 if drab else 0)
    p.flags = flags
    with pytest.raises(hstu.MtgrError) as e:
        bwd_call(p, drab=drab)
    assert e.value.status == status


@pytest.mark.parametrize("flags", [hstu.MTGR_BWD_KEEP_DS | hstu.MTGR_BWD_SKIP_DQ,
                                   hstu.MTGR_BWD_DS_READY | hstu.MTGR_BWD_SKIP_DKDV])
def test_stored_ds_flags_need_backward_workspace(flags):
    p = prob()
    base = hstu.mtgr_hstu_attn_workspace_size(p, False)
    p.flags = flags
    with pytest.raises(hstu.MtgrError) as e:
        bwd_call(p, workspace_bytes=base)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL
    pf = prob(dtype=FP32)
    pf.flags = flags
    with pytest.raises(hstu.MtgrError) as e:                    # fp32 has no stored-dS path
        bwd_call(pf)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL


@pytest.mark.parametrize("mutate,status", [
    (dict(dim=12), hstu.MTGR_ERROR_INVALID_ARGUMENT),          # bf16 needs multiples of 8
    (dict(dim=8192), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(groups=0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(groups=128), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(eps=0.0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(ld_x=8), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(dtype=3), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(num_tokens=-1), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(num_tokens=2**28), hstu.MTGR_ERROR_UNSUPPORTED),      # grid bound of the forward
])
def test_gln_validation(mutate, status):
    base = dict(num_tokens=10, dim=64, groups=4, dtype=BF16)
    base.update(mutate)
    p = hstu.gln_problem(**base)
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_group_layernorm_workspace_size(p)
    assert e.value.status == status


def test_gln_pointer_checks():
    p = hstu.gln_problem(10, 64, 4, BF16)
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_group_layernorm_fwd(p, FAKE, None, FAKE, FAKE, FAKE, None, None, None, 0)
    assert e.value.status == hstu.MTGR_ERROR_NULL_POINTER
    with pytest.raises(hstu.MtgrError) as e:       # du given without u
        hstu.mtgr_group_layernorm_bwd(p, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                      FAKE, None, 0, 0)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    assert hstu.mtgr_group_layernorm_workspace_size(p) == 0
    need = hstu.mtgr_group_layernorm_workspace_size(p, True)
    assert need >= 2 * 4 * 64 * 4
    with pytest.raises(hstu.MtgrError) as e:       # backward workspace too small
        hstu.mtgr_group_layernorm_bwd(p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                      FAKE, FAKE, need - 1, 0)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(hstu, "_lib", None)
    monkeypatch.setattr(hstu, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(hstu.MtgrLibraryMissing):
        hstu.lib()


def validate(p, **over):
    args = dict(offsets=FAKE, seg=FAKE, group_ids=None, num_groups=0, scratch=FAKE,
                scratch_bytes=hstu.MTGR_VALIDATE_SCRATCH_BYTES)
    args.update(over)
    hstu.mtgr_debug_validate_inputs(p, args["offsets"], args["seg"], args["group_ids"], args["num_groups"],
                                    args["scratch"], args["scratch_bytes"], 0)


@pytest.mark.parametrize("over,status", [
    (dict(offsets=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(seg=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(scratch=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(scratch_bytes=hstu.MTGR_VALIDATE_SCRATCH_BYTES - 1), hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL),
    (dict(scratch=FAKE + 4), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(group_ids=FAKE, num_groups=0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(group_ids=FAKE, num_groups=128), hstu.MTGR_ERROR_INVALID_ARGUMENT),
])
def test_validate_inputs_host_checks(over, status):
    """Host-side argument checks of the debug validator (before any device work)."""
    with pytest.raises(hstu.MtgrError) as e:
        validate(prob(), **over)
    assert e.value.status == status
    with pytest.raises(hstu.MtgrError) as e:
        validate(prob(num_users=-1))
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT


def test_cand_rows_flag_is_forward_only():
    p = prob()
    p.flags = hstu.MTGR_FWD_CAND_ROWS
    assert hstu.mtgr_hstu_attn_workspace_size(p) > 0
    with pytest.raises(hstu.MtgrError) as e:
        bwd_call(p)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    assert "forward only" in hstu.mtgr_last_error_message()


# ------------------------------------------------------------------ embedding table

def emb_table(**kw):
    base = dict(key_capacity=1024, row_capacity=500, dim=64, dtype=BF16, keys=FAKE, key_rows=FAKE,
                values=FAKE, counts=FAKE, last_ts=FAKE, free_rows=FAKE, state=FAKE)
    base.update(kw)
    return hstu.EmbeddingTable(**base)


def test_embedding_struct_layout():
    assert ctypes.sizeof(hstu.EmbeddingTable) == 80
    assert hstu.EmbeddingTable.keys.offset == 24


@pytest.mark.parametrize("mutate,status", [
    (dict(key_capacity=1000), hstu.MTGR_ERROR_INVALID_ARGUMENT),     # not a power of two
    (dict(key_capacity=256), hstu.MTGR_ERROR_INVALID_ARGUMENT),      # below row_capacity + 1
    (dict(row_capacity=0), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(row_capacity=2 ** 31), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(dim=12), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(dim=2048), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(dtype=5), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(values=0), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(state=FAKE + 4), hstu.MTGR_ERROR_INVALID_ARGUMENT),        # misaligned
])
def test_embedding_table_checks(mutate, status):
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_init(emb_table(**mutate), stream=0)
    assert e.value.status == status


def test_embedding_call_checks():
    t = emb_table()
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_dedup_workspace_size(2 ** 31)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    need = hstu.mtgr_embedding_dedup_workspace_size(1000)
    assert need >= 1000 * 4 + 2048 * 16
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_dedup(1000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, stream=0)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_gather(t, 10, FAKE, FAKE, FAKE, 60, stream=0)   # ld_out < dim
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_sgd(t, 10, FAKE, FAKE, FAKE, 64, 10, FAKE, FAKE, float("nan"), FAKE, 1 << 20, stream=0)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    wsb = hstu.mtgr_embedding_lookup_workspace_size(100)
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_lookup(t, 100, FAKE, None, FAKE, 0, 1, FAKE, FAKE, wsb - 1, stream=0)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL
    other = emb_table(keys=FAKE + 4096, key_rows=FAKE + 8192, key_capacity=2048)
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_rehash(t, emb_table(key_capacity=2048, values=FAKE + 256), stream=0)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT      # different value store
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_embedding_rehash(t, emb_table(key_capacity=2048), stream=0)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT      # same key store
    assert other.key_capacity == 2048


def noalloc(p, **over):
    args = dict(offsets=FAKE, seg=FAKE, ts=FAKE, q=FAKE, k=FAKE, v=FAKE, rab=None, out=FAKE)
    args.update(over)
    hstu.mtgr_hstu_attn_fwd_noalloc(p, args["offsets"], args["seg"], args["ts"], args["q"], args["k"],
                                    args["v"], args["rab"], args["out"], 0)


def test_noalloc_refusals_before_any_device_call():
    """The allocation-free forward rejects, on the host and before touching the device, a plan
    larger than its scratch array, the MTGR_ATTN_PLANNED flag and invalid problems."""
    big = prob(num_users=4096, total_tokens=6_000_000, max_seqlen=3000, heads=8)
    assert hstu.mtgr_hstu_attn_workspace_size(big) > hstu.MTGR_NOALLOC_SCRATCH_BYTES
    with pytest.raises(hstu.MtgrError) as e:
        noalloc(big)
    assert e.value.status == hstu.MTGR_ERROR_UNSUPPORTED
    assert "scratch" in hstu.mtgr_last_error_message()
    p = prob()
    p.flags = hstu.MTGR_ATTN_PLANNED
    with pytest.raises(hstu.MtgrError) as e:
        noalloc(p)
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    with pytest.raises(hstu.MtgrError) as e:
        noalloc(prob(head_dim=48))
    assert e.value.status == hstu.MTGR_ERROR_UNSUPPORTED
    noalloc(prob(num_users=0, total_tokens=0))     # empty batch: a successful no-op


def test_noalloc_scratch_covers_the_workloads():
    """The five benchmark workloads fit the scratch (serving: 1024 users, 1.5M tokens)."""
    from synth import make_layout
    for name in ("tiny", "small", "mtgr_small", "mtgr_large", "serving"):
        L = make_layout(name)
        p = prob(num_users=L.num_users, total_tokens=L.total_tokens, max_seqlen=L.max_seqlen,
                 heads=L.spec.heads, head_dim=L.spec.head_dim,
                 dtype=BF16 if L.spec.dtype == "bf16" else FP32)
        assert hstu.mtgr_hstu_attn_workspace_size(p) <= hstu.MTGR_NOALLOC_SCRATCH_BYTES, name


def cached(p, pc, **over):
    args = dict(offsets=FAKE, seg=FAKE, ts=FAKE, q=FAKE, k=FAKE, v=FAKE, rab=None, out=FAKE, offsets_c=FAKE,
                ts_c=FAKE, kc=FAKE, vc=FAKE, cache_plan=FAKE, cache_plan_bytes=1 << 30, workspace=FAKE,
                workspace_bytes=1 << 30)
    args.update(over)
    hstu.mtgr_hstu_attn_fwd_cached(p, args["offsets"], args["seg"], args["ts"], args["q"], args["k"], args["v"],
                                   args["rab"], args["out"], pc, args["offsets_c"], args["ts_c"], args["kc"],
                                   args["vc"], args["cache_plan"], args["cache_plan_bytes"], args["workspace"],
                                   args["workspace_bytes"], 0)


@pytest.mark.parametrize("request_kw,cache_kw,over,status", [
    (dict(), dict(heads=4), {}, hstu.MTGR_ERROR_INVALID_ARGUMENT),          # heads differ
    (dict(), dict(num_users=5), {}, hstu.MTGR_ERROR_INVALID_ARGUMENT),      # users differ
    (dict(dtype=FP32), dict(dtype=FP32), {}, hstu.MTGR_ERROR_UNSUPPORTED),  # matrix cores only
    (dict(head_dim=16), dict(head_dim=16), {}, hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(), dict(), dict(kc=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(), dict(), dict(offsets_c=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(), dict(), dict(cache_plan=FAKE + 16), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(), dict(), dict(cache_plan_bytes=256), hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL),
])
def test_cached_forward_validation(request_kw, cache_kw, over, status):
    """Host-side checks of the cached forward: request and cache must agree in users, heads,
    head_dim and dtype; the matrix-core shapes only; the cache's plan must be large enough."""
    p = prob(**request_kw)
    pc = prob(**dict(dict(total_tokens=300, max_seqlen=120), **cache_kw))
    with pytest.raises(hstu.MtgrError) as e:
        cached(p, pc, **over)
    assert e.value.status == status


def test_cached_forward_flags():
    p = prob()
    p.flags = hstu.MTGR_FWD_CAND_ROWS
    with pytest.raises(hstu.MtgrError) as e:
        cached(p, prob())
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_hstu_attn_fwd_cached(prob(), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, None, FAKE, FAKE,
                                       FAKE, FAKE, FAKE, 1 << 30, FAKE, 1 << 30, 0)
    assert e.value.status == hstu.MTGR_ERROR_NULL_POINTER


# ------------------------------------------------------------------ dense products
NN, NT, TN = hstu.MTGR_GEMM_NN, hstu.MTGR_GEMM_NT, hstu.MTGR_GEMM_TN
EPI_SILU, EPI_RES = hstu.MTGR_GEMM_EPI_BIAS_SILU, hstu.MTGR_GEMM_EPI_BIAS_RESIDUAL


def gemm(layout=NN, M=512, N=256, K=256, A=FAKE, lda=None, B=FAKE, ldb=None, C=FAKE, ldc=None, epilogue=0,
         bias=None, R=None, ldr=0, C2=None, ldc2=0, colsum=None, workspace=FAKE, workspace_bytes=1 << 30):
    lda = lda if lda is not None else (M if layout == TN else K)
    ldb = ldb if ldb is not None else (K if layout == NT else N)
    ldc = ldc if ldc is not None else N
    hstu.mtgr_gemm_bf16(layout, M, N, K, A, lda, B, ldb, C, ldc, epilogue, bias, R, ldr, C2, ldc2, colsum,
                        workspace, workspace_bytes, 0)


@pytest.mark.parametrize("kw, status", [
    (dict(layout=3), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(epilogue=3), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(N=204), hstu.MTGR_ERROR_UNSUPPORTED),                        # N % 8
    (dict(K=100), hstu.MTGR_ERROR_UNSUPPORTED),                        # NN: K % 32
    (dict(layout=NT, K=48), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(layout=TN, M=300), hstu.MTGR_ERROR_UNSUPPORTED),             # TN: M % 8
    (dict(layout=TN, epilogue=EPI_SILU, bias=FAKE, C2=FAKE, ldc2=256), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(K=0), hstu.MTGR_ERROR_UNSUPPORTED),
    (dict(M=-1), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(A=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(C=FAKE + 8), hstu.MTGR_ERROR_INVALID_ARGUMENT),              # misaligned
    (dict(lda=100), hstu.MTGR_ERROR_INVALID_ARGUMENT),                 # ld < K
    (dict(ldb=260), hstu.MTGR_ERROR_INVALID_ARGUMENT),                 # ld % 8
    (dict(ldc=1 << 22), hstu.MTGR_ERROR_UNSUPPORTED),                  # ld too large
    (dict(epilogue=EPI_SILU, C2=FAKE, ldc2=256), hstu.MTGR_ERROR_NULL_POINTER),       # no bias
    (dict(epilogue=EPI_SILU, bias=FAKE + 4, C2=FAKE, ldc2=256), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(epilogue=EPI_SILU, bias=FAKE), hstu.MTGR_ERROR_NULL_POINTER),               # no C2
    (dict(epilogue=EPI_RES, bias=FAKE, R=FAKE, ldr=128), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(colsum=FAKE), hstu.MTGR_ERROR_INVALID_ARGUMENT),             # colsum needs TN
    (dict(layout=TN, colsum=FAKE + 2), hstu.MTGR_ERROR_INVALID_ARGUMENT),
    (dict(layout=TN, workspace=None), hstu.MTGR_ERROR_NULL_POINTER),
    (dict(layout=TN, workspace_bytes=1024), hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL),
])
def test_gemm_argument_checks(kw, status):
    with pytest.raises(hstu.MtgrError) as e:
        gemm(**kw)
    assert e.value.status == status, str(e.value)


def test_gemm_empty_output_is_a_noop():
    gemm(M=0, A=None, B=None, C=None)
    gemm(layout=TN, N=0, A=None, B=None, C=None, workspace=None, workspace_bytes=0)


def test_gemm_workspace_sizes():
    assert hstu.mtgr_gemm_workspace_size(NN, 4096, 2048, 512) == 0
    assert hstu.mtgr_gemm_workspace_size(NT, 4096, 512, 2048) == 0
    # weight gradient of the projection at 2^20 tokens, d = 512: one 256 x 256 tile per
    # (m, n) block, enough K splits for one workgroup per CU, fp32 partials plus column sums
    ws = hstu.mtgr_gemm_workspace_size(TN, 512, 2048, 1 << 20)
    tiles = 2 * 8
    splits = -(-256 // tiles)
    assert ws >= splits * (512 * 2048 + 2048) * 4
    # a short K is not split
    assert hstu.mtgr_gemm_workspace_size(TN, 256, 128, 40) == (256 * 128 + 128) * 4
    # the exact size is accepted, one byte less is refused
    need = hstu.mtgr_gemm_workspace_size(TN, 256, 128, 1000)
    with pytest.raises(hstu.MtgrError) as e:
        gemm(layout=TN, M=256, N=128, K=1000, workspace_bytes=need - 1)
    assert e.value.status == hstu.MTGR_ERROR_WORKSPACE_TOO_SMALL


def test_add_argument_checks():
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_add(10, 60, BF16, FAKE, 64, FAKE, 64, FAKE, 64, 0)          # cols % 8
    assert e.value.status == hstu.MTGR_ERROR_INVALID_ARGUMENT
    with pytest.raises(hstu.MtgrError) as e:
        hstu.mtgr_add(10, 64, BF16, FAKE, 64, None, 64, FAKE, 64, 0)
    assert e.value.status == hstu.MTGR_ERROR_NULL_POINTER
    hstu.mtgr_add(0, 64, BF16, None, 64, None, 64, None, 64, 0)


def test_clock_probe_argument_checks():
    for args, status in (((0, 4, FAKE), hstu.MTGR_ERROR_INVALID_ARGUMENT),
                         ((10, 0, FAKE), hstu.MTGR_ERROR_INVALID_ARGUMENT),
                         ((10, 70000, FAKE), hstu.MTGR_ERROR_INVALID_ARGUMENT),
                         ((10, 4, None), hstu.MTGR_ERROR_NULL_POINTER),
                         ((10, 4, FAKE + 4), hstu.MTGR_ERROR_INVALID_ARGUMENT)):
        with pytest.raises(hstu.MtgrError) as e:
            hstu.mtgr_debug_clock_probe(*args, stream=0)
        assert e.value.status == status


def test_binding_constants_match_the_headers():
    """Every integer #define of include/*.h that the Python binding mirrors has the header's value."""
    checked = []
    for name in sorted(os.listdir(os.path.join(ROOT, "include"))):
        if not name.endswith(".h"):
            continue
        text = open(os.path.join(ROOT, "include", name)).read()
        for m in re.finditer(r"^#define\s+(MTGR_\w+)\s+([^\n]*?)\s*(?:/\*.*)?$", text, re.M):
            macro, expr = m.group(1), m.group(2)
            if not expr or not hasattr(hstu, macro):
                continue
            value = eval(re.sub(r"\b(0x[0-9A-Fa-f]+|\d+)(?:ull|ll|u)\b", r"\1", expr), {"__builtins__": {}})
            assert getattr(hstu, macro) == value, (name, macro, expr, getattr(hstu, macro))
            checked.append(macro)
    assert {"MTGR_MAX_HEADS", "MTGR_MAX_GROUPS", "MTGR_MAX_RAB_BUCKETS", "MTGR_MAX_LD"} <= set(checked), checked
