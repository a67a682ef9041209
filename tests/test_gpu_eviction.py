"""Feature eviction on the GPU (through the C ABI) against the CPU oracle.

Integer results are bit-exact: the evicted count, the surviving key set, the
row of every key (reused rows come off the free stack in the same order) and
the rows' initial values.  Steps with evictions between them keep the whole
step's parity (stage-wise, as in the other parity tests).
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import recis as R
from paper_2509_20883_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _same_table(gt, ot):
    ek, er = gt.export()
    rk, rr = ot.export()
    ek, er = ek.cpu().numpy(), er.cpu().numpy()
    o1, o2 = np.argsort(ek), np.argsort(rk)
    assert np.array_equal(ek[o1], rk[o2]), "key sets differ"
    assert np.array_equal(er[o1], rr[o2]), "rows differ"
    assert gt.size() == ot.size()


@pytest.mark.parametrize("k,opt", [(0, O.ADAGRAD), (2, O.ADAGRAD), (1, O.ADAM_RW)])
def test_steps_with_evictions_match_oracle(k, opt):
    w = W.workload(k, mini=(k != 0))
    w.opt = opt
    _log("eviction steps", w.name)
    gt, ot = P.gpu_table(w, evictable=True), P.oracle_table(w)
    P.prepopulate(w, gt, ot)
    for step in range(6):
        b = W.make_batch(w, step)
        grad = W.make_grad(w, b, step)
        U, nn = P.run_step_parity(w, gt, ot, b, grad, step)
        if step in (1, 3, 4):
            age = {1: 0, 3: 1, 4: 0}[step]
            ne, no = gt.evict(age), ot.evict(age)
            _log(f"  step {step}: U={U} new={nn} evicted {ne} (oracle {no})")
            assert ne == no
            _same_table(gt, ot)
    gt.check()
    gt.close()


def test_eviction_churn_purges_tombstones():
    """A small IDMap that keeps taking new keys while old ones are evicted:
    tombstones pile up until a rehash drops them; rows are reused."""
    _log("eviction churn")
    gt = R.Table(8, O.F32, O.ADAGRAD, capacity_slots=1024, max_load=0.75, block_rows=256, seed=3,
                 evictable=True)
    ot = O.Table(8, opt=O.ADAGRAD, seed=3)
    g = np.random.default_rng(5)
    for it in range(30):
        keys = (g.integers(0, 300, size=200) + 300 * it).astype(np.int64)   # mostly new keys each call
        if it % 4 == 3:
            keys = np.concatenate([keys, np.arange(0, 50, dtype=np.int64)])  # a few old ones come back
        rows, nins = gt.find_or_insert(torch.from_numpy(keys).cuda())
        st, rref, nref = ot.find_or_insert(keys)
        assert st == O.OK
        assert np.array_equal(rows.cpu().numpy(), rref), f"call {it}: rows"
        assert int(nins.item()) == nref
        if it % 2 == 1:
            assert gt.evict(1) == ot.evict(1)
            _same_table(gt, ot)
    # rows are reused: far fewer rows than keys ever inserted
    assert ot.rows_allocated() < 2000
    _, wg, sg = (None, *gt.read_rows(gt.find(torch.from_numpy(ot.export()[0]).cuda())))
    _, wr, sr = ot.read_rows(ot.export()[0])
    assert np.array_equal(wg.cpu().numpy(), wr) and np.array_equal(sg.cpu().numpy(), sr)
    assert gt.capacity() <= 4096
    gt.check()
    gt.close()


def test_evict_errors_and_empty():
    t = R.Table(16, O.F32, O.ADAGRAD, capacity_slots=256, seed=1)
    with pytest.raises(R.RecisError):
        t.evict(0)
    t.close()
    t = R.Table(16, O.F32, O.ADAM, capacity_slots=256, seed=1, evictable=True)
    assert t.evict(0) == 0 and t.size() == 0
    t.find_or_insert(torch.arange(10, dtype=torch.int64, device="cuda"))
    assert t.evict(5) == 0 and t.size() == 10
    t.find_or_insert(torch.arange(3, dtype=torch.int64, device="cuda"))
    assert t.evict(0) == 7 and t.size() == 3
    rows = t.find(torch.arange(10, dtype=torch.int64, device="cuda")).cpu().numpy()
    assert rows[:3].tolist() == [0, 1, 2] and np.all(rows[3:] == -1)
    t.check()
    t.close()


def _same_contents(gt, ot):
    rk, _ = ot.export()
    wg, sg = gt.read_rows(gt.find(torch.from_numpy(rk).cuda()))
    _, wr, sr = ot.read_rows(rk)
    assert np.array_equal(wg.cpu().numpy(), wr) and np.array_equal(sg.cpu().numpy(), sr), "row contents differ"


@pytest.mark.parametrize("k,opt,alloc", [(0, O.ADAGRAD, False), (2, O.ADAGRAD, False), (1, O.ADAM_RW, False),
                                         (2, O.ADAGRAD, True)])
def test_compaction_after_evictions_matches_oracle(k, opt, alloc):
    """Steps, evictions, then compaction on both sides: the key -> row map is
    bit-exact (the k-th row at or above the live count into the k-th free row
    below it), every key's row contents are unchanged (the oracle holds the
    GPU's rows: stage-wise parity resynchronises it), Blocks memory past the
    live rows is released, and later steps (new keys at rows L, L+1, ...)
    keep the step parity."""
    w = W.workload(k, mini=(k != 0))
    w.opt = opt
    _log("compaction", w.name, "allocator" if alloc else "")
    kw = dict(evictable=True, block_rows=1024)
    if alloc:
        kw["allocator"] = R.TorchAllocator()
    gt, ot = P.gpu_table(w, **kw), P.oracle_table(w)
    P.prepopulate(w, gt, ot)
    for step in range(4):
        b = W.make_batch(w, step)
        P.run_step_parity(w, gt, ot, b, W.make_grad(w, b, step), step)
        if step in (1, 2):
            assert gt.evict(0) == ot.evict(0)
    live = ot.size()
    allocated = ot.rows_allocated()
    moved, released = gt.compact()
    assert moved == ot.compact()
    _log(f"  live {live} rows {allocated}: moved {moved}, released {released} bytes")
    _same_table(gt, ot)
    _same_contents(gt, ot)
    assert ot.rows_allocated() == live and released >= 0
    for step in range(4, 6):
        b = W.make_batch(w, step)
        P.run_step_parity(w, gt, ot, b, W.make_grad(w, b, step), step)
    _same_table(gt, ot)
    assert gt.compact()[0] == ot.compact() == 0  # compact again: nothing free, nothing moves
    gt.check()
    gt.close()


def test_compact_errors_and_trivial_cases():
    t = R.Table(16, O.F32, O.ADAGRAD, capacity_slots=256, seed=1)
    with pytest.raises(R.RecisError):
        t.compact()                               # not evictable
    t.close()
    t = R.Table(16, O.F32, O.ADAM, capacity_slots=256, seed=1, evictable=True, block_rows=64)
    assert t.compact() == (0, 0)                  # empty table
    t.find_or_insert(torch.arange(200, dtype=torch.int64, device="cuda"))
    assert t.compact()[0] == 0                    # nothing free: nothing moves
    t.find_or_insert(torch.arange(100, 110, dtype=torch.int64, device="cuda"))
    assert t.evict(0) == 190 and t.size() == 10   # keys 100..109 stay, at rows 100..109
    moved, released = t.compact()
    assert moved == 10 and released >= 0
    rows = t.find(torch.arange(100, 110, dtype=torch.int64, device="cuda")).cpu().numpy()
    assert rows.tolist() == list(range(10))       # row 100 + j -> hole j
    t.find_or_insert(torch.arange(110, dtype=torch.int64, device="cuda"))
    assert t.size() == 110
    t.check()
    t.close()
