"""The device embedding table against the dict oracle (GPU).

IDs, row indices and the order of the unique list depend on atomic races, so the checks
compare what is unique: the set of distinct IDs, unique[inverse] == ids, per-ID occurrence
counts, the ID -> embedding mapping (through gathers), counters, timestamps, eviction counts
and capacity accounting.  Gathers are bit-exact; SGD updates are compared to the fp64 oracle
within one rounding of the table's dtype per step (their summation order varies)."""
import collections

import numpy as np
import pytest
import torch

from oracle.embedding import DictTable
from paper_2505_18654_amd.embedding import DynamicEmbedding
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def zipf_ids(rng, n, universe, a=1.15):
    """Skewed IDs spread over the whole 64-bit range (including the sign bit)."""
    base = rng.zipf(a, n) % universe
    return (base.astype(np.uint64) * np.uint64(0x9E3779B97F4A7C15)) ^ np.uint64(0x5555)


def to_dev(ids_u64):
    return torch.from_numpy(ids_u64.view(np.int64).copy()).cuda()


def u64(t):
    return t.cpu().numpy().view(np.uint64)


@pytest.mark.parametrize("n,universe", [(0, 1), (1, 1), (1000, 50), (100_000, 5_000), (300_000, 10**9)])
def test_dedup(n, universe):
    rng = np.random.default_rng(n)
    ids = zipf_ids(rng, n, universe)
    t = DynamicEmbedding(16, 8)
    unique, occ, inverse, num = t.dedup(to_dev(ids))
    torch.cuda.synchronize()
    nu = int(num.item())
    ref_u, ref_occ, _ = DictTable.dedup(ids)
    say(f"[embedding] dedup n={n} unique={nu}")
    assert nu == len(ref_u)
    got_u = u64(unique)[:nu]
    assert set(got_u.tolist()) == set(ref_u)
    if n:
        np.testing.assert_array_equal(got_u[inverse.cpu().numpy()[:n]], ids)
        cnt = collections.Counter(ids.tolist())
        assert [cnt[x] for x in got_u.tolist()] == occ.cpu().numpy()[:nu].tolist()


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_training_sequence_matches_oracle(dtype):
    """Batches of skewed IDs: lookup with insertion, gather, SGD; then eviction and reuse."""
    rng = np.random.default_rng(7)
    dim, cap = 64, 4096
    t = DynamicEmbedding(cap, dim, dtype=dtype)
    ref = DictTable(cap, dim)
    lr = 0.5
    tol = 1e-5 if dtype == torch.float32 else 2.0 ** -7
    for step in range(6):
        ids = zipf_ids(rng, 3000, 1500)
        out, b = t.lookup(to_dev(ids), now=10 + step)
        u, occ, _ = ref.dedup(ids)
        ref.lookup(u, occ, now=10 + step, insert=True)
        want = ref.gather(ids)
        got = out.float().cpu().numpy()
        err = np.max(np.abs(got - want)) / max(1e-30, float(np.sqrt(np.mean(want ** 2))) if want.any() else 1.0)
        say(f"[embedding] {dtype} step {step} gather err {err:.2e}")
        assert err <= tol * 4, (step, err)
        grad = rng.standard_normal((len(ids), dim)).astype(np.float32)
        t.sgd(b, torch.from_numpy(grad).cuda(), lr)
        ref.sgd(ids, grad.astype(np.float64) if dtype == torch.float32 else
                torch.from_numpy(grad).to(torch.bfloat16).float().numpy().astype(np.float64), lr)
    torch.cuda.synchronize()
    st = t.stats()
    assert st["num_keys"] == len(ref.rows) == st["next_row"] and st["overflow"] == 0
    # counters and timestamps of every live ID, through its row
    keys = np.array(sorted(ref.rows), np.uint64)
    _, ub = t.lookup(to_dev(keys), now=999, insert=False, gather=False)
    torch.cuda.synchronize()
    # that lookup added one occurrence and stamped 999: undo in the comparison
    got_u = u64(ub.unique)[:len(keys)]
    rows = ub.rows.cpu().numpy()[:len(keys)]
    assert (rows >= 0).all()
    counts = t.counts.cpu().numpy().view(np.uint32)[rows]
    stamp = t.last_ts.cpu().numpy()[rows]
    assert (stamp == 999).all()
    assert [ref.rows[int(k)].count + 1 for k in got_u] == counts.tolist()
    # eviction: everything stamped before 999 goes except nothing; evict at 1000 removes all
    n_ev = t.evict(1000)
    assert n_ev == len(ref.rows)
    assert t.stats()["num_keys"] == 0 and t.stats()["free_top"] == n_ev
    # re-insertion reuses freed rows and starts from zero rows and counters
    ids = zipf_ids(rng, 500, 300)
    out, b = t.lookup(to_dev(ids), now=2000)
    torch.cuda.synchronize()
    assert not out.float().abs().sum().item()
    st = t.stats()
    nu = int(b.num_unique.item())
    assert st["next_row"] == len(ref.rows) and st["free_top"] == n_ev - nu and st["num_keys"] == nu


def test_evict_by_time_and_lookup_without_insert():
    rng = np.random.default_rng(3)
    t = DynamicEmbedding(2000, 16)
    ref = DictTable(2000, 16)
    for step in range(8):
        ids = zipf_ids(rng, 400, 900)
        t.lookup(to_dev(ids), now=step, gather=False)
        u, occ, _ = ref.dedup(ids)
        ref.lookup(u, occ, now=step, insert=True)
    for thr in (2, 5):
        assert t.evict(thr) == ref.evict(thr)
    assert t.evict(0, min_count=4) == ref.evict(0, min_count=4)   # by frequency
    live = np.array(sorted(ref.rows), np.uint64)
    probe = np.concatenate([live, np.array([1, 2, 3], np.uint64)])   # three IDs never inserted
    _, b = t.lookup(to_dev(probe), now=50, insert=False, gather=False)
    torch.cuda.synchronize()
    nu = int(b.num_unique.item())
    got = dict(zip(u64(b.unique)[:nu].tolist(), b.rows.cpu().numpy()[:nu].tolist()))
    assert all(got[int(k)] >= 0 for k in live)
    assert all(got[k] == -1 for k in (1, 2, 3) if k not in ref.rows)
    assert len(set(got[int(k)] for k in live)) == len(live)    # distinct rows


def test_row_capacity_overflow():
    t = DynamicEmbedding(100, 8, key_capacity=256)
    ids = np.arange(1, 161, dtype=np.uint64) * np.uint64(977)
    out, b = t.lookup(to_dev(ids), now=1)
    torch.cuda.synchronize()
    rows = b.rows.cpu().numpy()[:int(b.num_unique.item())]
    st = t.stats()
    say(f"[embedding] overflow stats {st}")
    assert (rows >= 0).sum() == 100 and (rows == -1).sum() == 60
    assert len(set(rows[rows >= 0].tolist())) == 100
    assert st["overflow"] & 1 and st["num_keys"] == 100 and st["next_row"] == 100 and st["free_top"] == 0
    # the 60 released slots are DELETED; looking the inserted IDs up again still finds them
    _, b2 = t.lookup(to_dev(ids), now=2, insert=False, gather=False)
    torch.cuda.synchronize()
    got = dict(zip(u64(b.unique)[:160].tolist(), rows.tolist()))
    got2 = dict(zip(u64(b2.unique)[:160].tolist(), b2.rows.cpu().numpy()[:160].tolist()))
    assert got == got2


def test_grow_keeps_the_mapping():
    rng = np.random.default_rng(5)
    t = DynamicEmbedding(3000, 32, key_capacity=4096)
    ids = zipf_ids(rng, 5000, 2500)
    t.lookup(to_dev(ids), now=1, gather=False)
    t.evict(1)   # nothing (all stamped 1)
    grad = torch.randn(len(ids), 32, device="cuda")
    _, b = t.lookup(to_dev(ids), now=2, gather=False)
    t.sgd(b, grad, 0.1)
    before = t.lookup(to_dev(ids), now=3)[0].clone()
    _, b = t.lookup(to_dev(ids[:700]), now=4, gather=False)
    t.evict(4)   # drops the IDs not in the first 700 positions
    t.grow(1 << 14)
    after, _ = t.lookup(to_dev(ids[:700]), now=5)
    torch.cuda.synchronize()
    assert torch.equal(after, before[:700])
    assert t.stats()["num_keys"] == len(set(ids[:700].tolist()))


@pytest.mark.parametrize("dim,dtype", [(8, torch.float32), (8, torch.bfloat16), (1024, torch.float32),
                                       (1024, torch.bfloat16), (200, torch.bfloat16)])
def test_dims(dim, dtype):
    """Smallest and largest widths (at 1024 fp32 a workgroup holds one 32-position chunk per
    column block), and a width that does not divide the workgroup evenly."""
    rng = np.random.default_rng(dim)
    t = DynamicEmbedding(600, dim, dtype=dtype)
    ref = DictTable(600, dim)
    lr = 0.25
    for step in range(3):
        ids = zipf_ids(rng, 2000, 500)
        out, b = t.lookup(to_dev(ids), now=step)
        u, occ, _ = ref.dedup(ids)
        ref.lookup(u, occ, now=step, insert=True)
        want = ref.gather(ids)
        got = out.float().cpu().numpy()
        scale = float(np.sqrt(np.mean(want ** 2))) if want.any() else 1.0
        tol = 1e-5 if dtype == torch.float32 else 2.0 ** -4
        assert np.max(np.abs(got - want)) <= tol * scale, (step, np.max(np.abs(got - want)) / scale)
        grad = torch.randn(len(ids), dim, device="cuda", dtype=dtype)
        t.sgd(b, grad, lr)
        ref.sgd(ids, grad.float().cpu().numpy().astype(np.float64), lr)
