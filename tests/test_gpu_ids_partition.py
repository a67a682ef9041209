"""Ids partition on the GPU (through the C ABI) against the CPU oracle.

Integer work: keys, shard offsets, inverse and the distinct-key count must be
bit-exact.  Cases span one rank tile to the full one-million-id input, ragged
tails, one shard, power-of-two and other shard counts up to the maximum, the
two-level count scan, blocks of several rank tiles, reserved keys, an empty
batch and workspace reuse with a smaller second call.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import recis as R
from paper_2509_20883_amd import workloads as W

pytestmark = pytest.mark.gpu

I64_MIN = np.iinfo(np.int64).min


def _log(*a):
    print(*a, flush=True)


def _run(part, values, G, seed):
    v = torch.from_numpy(values).cuda()
    keys, offs, inv, info = part(v, G, seed)
    torch.cuda.synchronize()
    info = info.cpu().numpy()
    U = int(info[0])
    return keys[:U].cpu().numpy(), offs.cpu().numpy(), inv.cpu().numpy(), info


def _check(part, values, G, seed):
    keys, offs, inv, info = _run(part, values, G, seed)
    ek, eo, ei, erej = O.ids_partition(values, G, seed)
    assert int(info[0]) == len(ek)
    assert np.array_equal(keys, ek), "keys"
    assert np.array_equal(offs, eo), "shard offsets"
    assert np.array_equal(inv, ei), "inverse"
    assert (int(info[1]) & 1) == (1 if erej else 0)
    assert (int(info[1]) & ~1) == 0
    return len(ek)


def _zipf_ids(n, V, s, seed):
    g = np.random.default_rng(seed)
    r = g.zipf(s, size=4 * n)
    r = r[r <= V][:n]
    return (r.astype(np.int64) * 0x9E3779B1) ^ 0x1234567


@pytest.mark.parametrize("n,G", [(1, 1), (1, 8), (100, 3), (1024, 2), (1025, 8), (4097, 5), (70001, 8),
                                 (70001, 1), (131072, 64), (250003, 1000), (250003, 1024), (40000, 7),
                                 # owner-count tables of 8256 and 12800 entries: past the histogram's
                                 # own scan (at most 8192), scanned by one block of their own
                                 (131073, 64), (131072, 100)])
def test_ids_partition_matches_oracle(n, G):
    _log(f"ids_partition n={n} G={G}")
    part = R.IdsPartition()
    vals = _zipf_ids(n, max(n // 3, 1), 1.1, n + G)
    _check(part, vals, G, 0xC0FFEE ^ G)


def test_ids_partition_all_distinct_and_all_equal():
    part = R.IdsPartition()
    g = np.random.default_rng(3)
    _log("ids_partition all distinct 300000")
    vals = g.permutation(np.arange(300000, dtype=np.int64)) * 1000003 - (1 << 50)
    assert _check(part, vals, 16, 5) == 300000
    _log("ids_partition all equal 200000")
    assert _check(part, np.full(200000, -42, dtype=np.int64), 6, 5) == 1
    _log("ids_partition extreme keys")
    vals = np.array([np.iinfo(np.int64).max, I64_MIN + 2, 0, -1, 1, np.iinfo(np.int64).max] * 999, dtype=np.int64)
    assert _check(part, vals, 3, 0xFFFFFFFFFFFFFFFF) == 5


def test_ids_partition_reserved_keys_are_skipped():
    _log("ids_partition reserved keys")
    part = R.IdsPartition()
    vals = _zipf_ids(50000, 20000, 1.2, 9)
    vals[::97] = I64_MIN
    vals[5::131] = I64_MIN + 1
    _check(part, vals, 8, 1)


def test_ids_partition_empty_and_reuse():
    _log("ids_partition empty + workspace reuse")
    part = R.IdsPartition()
    keys, offs, inv, info = _run(part, np.zeros(0, dtype=np.int64), 4, 0)
    assert offs.tolist() == [0] * 5 and info.tolist() == [0, 0] and inv.size == 0
    big = W.ids_partition_values(step=1)
    _check(part, big, W.IDS_PARTITION_SHARDS, W.IDS_PARTITION_SEED)
    small = _zipf_ids(3000, 500, 1.1, 4)
    _check(part, small, W.IDS_PARTITION_SHARDS, W.IDS_PARTITION_SEED)
    _check(part, big[:777777], 13, 77)


def test_ids_partition_full_size_input():
    # the one-million-id input of the benchmark, in the configuration it times
    _log("ids_partition full size")
    part = R.IdsPartition()
    vals = W.ids_partition_values(step=0)
    U = _check(part, vals, W.IDS_PARTITION_SHARDS, W.IDS_PARTITION_SEED)
    assert U > 100000
    # repeated calls on one workspace give the same result
    k1, o1, i1, _ = _run(part, vals, W.IDS_PARTITION_SHARDS, W.IDS_PARTITION_SEED)
    k2, o2, i2, _ = _run(part, vals, W.IDS_PARTITION_SHARDS, W.IDS_PARTITION_SEED)
    assert np.array_equal(k1, k2) and np.array_equal(o1, o2) and np.array_equal(i1, i2)


def test_ids_partition_rejects_bad_arguments():
    v = torch.zeros(10, dtype=torch.int64, device="cuda")
    with pytest.raises(R.RecisError):
        R.ids_partition(v, 0)
    with pytest.raises(R.RecisError):
        R.ids_partition(v, 1025)
    assert R.ids_partition_workspace_bytes(10, 0) == 0
    assert R.ids_partition_workspace_bytes(-1, 4) == 0
    assert R.ids_partition_workspace_bytes((1 << 28) + 1, 4) == 0
