"""The largest batch the C ABI accepts (2^28 ids): the dedup passes at their
limits (512 dedup blocks of 128 tiles, 4096 partitions, 19-bit record
indices).  The oracle cannot run at this size in a test, so the checks are
the ones that hold at any size: the distinct keys in first-occurrence order
(from numpy.unique), the new rows numbered in that order, every id's row or
slot against a plain IDMap find / a gather, and the owner grouping of the ids
partition against the oracle applied to the distinct keys.
"""
import gc
import time

import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import recis as R

pytestmark = pytest.mark.gpu

N_MAX = 1 << 28
T0 = time.time()


def _log(*a):
    print(f"[{time.time() - T0:6.1f}s]", *a, flush=True)


@pytest.fixture(scope="module")
def big():
    _log("max size: generating 2^28 ids over 2^20 keys")
    g = np.random.default_rng(28)
    vals = (g.integers(0, 1 << 20, size=N_MAX, dtype=np.int64) * 0x9E3779B1 + 12345) ^ (1 << 40)
    _log("max size: numpy.unique")
    uk, first = np.unique(vals, return_index=True)
    order = np.argsort(first, kind="stable")
    keys_first = uk[order]
    del uk, first, order
    _log(f"max size: {keys_first.size} distinct keys")
    yield vals, keys_first
    gc.collect()
    torch.cuda.empty_cache()


def test_find_or_insert_at_max_size(big):
    vals, keys_first = big
    U = keys_first.size
    t = R.Table(8, O.F32, O.ADAGRAD, capacity_slots=1 << 22, seed=5)
    try:
        v = torch.from_numpy(vals).cuda()
        _log("max size: find_or_insert of 2^28 ids")
        rows, nins = t.find_or_insert(v)
        torch.cuda.synchronize()
        assert int(nins.item()) == U and t.size() == U
        # new rows are numbered in first-occurrence order
        kf = torch.from_numpy(keys_first).cuda()
        assert torch.equal(t.find(kf), torch.arange(U, dtype=torch.int64, device="cuda"))
        # every id's row is its key's row (a plain IDMap lookup of every id)
        assert torch.equal(rows, t.find(v))
        # initial values of a sample of rows
        sel = np.random.default_rng(1).choice(U, size=2000, replace=False)
        wg, _ = t.read_rows(torch.from_numpy(sel.astype(np.int64)).cuda())
        wg = wg.cpu().numpy()
        for i, r in enumerate(sel[:200]):
            assert np.array_equal(wg[i], O.init_row(5, int(keys_first[r]), 8, -0.01, 0.01))
        t.check()
        del v, rows, kf
    finally:
        t.close()
        gc.collect()
        torch.cuda.empty_cache()


def test_ids_partition_at_max_size(big):
    vals, keys_first = big
    U = keys_first.size
    G, seed = 8, 77
    v = torch.from_numpy(vals).cuda()
    _log("max size: ids partition of 2^28 ids")
    keys, offs, inv, info = R.IdsPartition()(v, G, seed)
    torch.cuda.synchronize()
    assert int(info[0].item()) == U and int(info[1].item()) == 0
    ek, eo, _, _ = O.ids_partition(keys_first, G, seed)
    assert np.array_equal(keys[:U].cpu().numpy(), ek), "keys grouped by owner"
    assert np.array_equal(offs.cpu().numpy(), eo), "shard offsets"
    assert torch.equal(keys[inv.long()], v), "keys_out[inverse] == values"
    del v, keys, inv
    gc.collect()
    torch.cuda.empty_cache()
