"""The dedup passes where a dedup block's record count crosses the limits of
the tile pass's partition-order copy.

The tile pass assembles that copy in LDS, 8192 records (one chunk) at a time,
for a block of at most four chunks, and scatters the records of a larger
block.  With all-distinct ids every tile of 4096 ids yields 4096 records, so
the batch size alone fixes the records per block (R tiles per block, R =
ceil(tiles / 256)):
  - 767 full tiles + 1 id: R = 3, blocks of 12288 records (two chunks) and a
    last block of 8193 (a second chunk holding one record);
  - 2048 tiles: R = 8, every block exactly four chunks (32768 records);
  - 2049 tiles: R = 9, blocks of 36864 records (scattered) beside a last
    block of six tiles (three chunks) in the same launch.
Checked against what the definitions fix: a fresh table numbers new keys in
first-occurrence order, so find_or_insert of distinct ids returns 0..n-1 and,
with repeats, each id's first-occurrence rank (numpy.unique); the ids
partition groups the distinct keys by owner as the oracle does.
"""
import gc

import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import recis as R

pytestmark = pytest.mark.gpu

TILE = 4096
MIX = np.uint64(0x9E3779B97F4A7C15)  # odd: i -> i * MIX mod 2^62 is a bijection
MASK62 = np.uint64((1 << 62) - 1)

CASES = {
    "two-chunks-one-record-tail": 767 * TILE + 1,
    "four-chunks-exactly": 2048 * TILE,
    "scatter-beside-staged": 2049 * TILE,
}


def distinct_ids(n: int, salt: int) -> np.ndarray:
    i = np.arange(n, dtype=np.uint64) + np.uint64(salt)
    return ((i * MIX) & MASK62).astype(np.int64)


def first_ranks(vals: np.ndarray) -> np.ndarray:
    """Rank of each id's key in first-occurrence order."""
    _, first, inv = np.unique(vals, return_index=True, return_inverse=True)
    rank_of_sorted = np.empty(first.size, dtype=np.int64)
    rank_of_sorted[np.argsort(first, kind="stable")] = np.arange(first.size, dtype=np.int64)
    return rank_of_sorted[inv]


def _table(n: int) -> R.Table:
    cap = 1 << max(17, int(np.ceil(np.log2(n / 0.7))))
    return R.Table(8, O.F32, O.ADAGRAD, capacity_slots=cap, seed=3)


def _cleanup():
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("case", list(CASES))
def test_find_or_insert_distinct(case):
    n = CASES[case]
    print(f"dedup chunks: {case}, n={n}", flush=True)
    v = torch.from_numpy(distinct_ids(n, 11)).cuda()
    t = _table(n)
    try:
        rows, nins = t.find_or_insert(v)
        torch.cuda.synchronize()
        assert int(nins.item()) == n and t.size() == n
        assert torch.equal(rows, torch.arange(n, dtype=torch.int64, device="cuda")), "rows of distinct ids"
        # a second call finds every key where it was put
        rows2, nins2 = t.find_or_insert(v.flip(0))
        assert int(nins2.item()) == 0
        assert torch.equal(rows2, torch.arange(n - 1, -1, -1, dtype=torch.int64, device="cuda"))
        t.check()
    finally:
        t.close()
        del v
        _cleanup()


def test_find_or_insert_repeats_multi_chunk():
    """Repeated keys (a record's count and ranks above one) through staged
    blocks of three to four chunks and scattered ones."""
    n = 2049 * TILE
    g = np.random.default_rng(2049)
    base = distinct_ids(int(n * 0.9), 5)
    vals = base[g.integers(0, base.size, size=n)]
    print(f"dedup chunks: repeats, n={n}", flush=True)
    v = torch.from_numpy(vals).cuda()
    t = _table(n)
    try:
        rows, nins = t.find_or_insert(v)
        torch.cuda.synchronize()
        want = first_ranks(vals)
        assert int(nins.item()) == int(want.max()) + 1
        assert np.array_equal(rows.cpu().numpy(), want), "rows in first-occurrence order"
        t.check()
    finally:
        t.close()
        del v
        _cleanup()


def test_ids_partition_scatter_beside_staged():
    n = CASES["scatter-beside-staged"]
    G, seed = 8, 1234
    vals = distinct_ids(n, 99)
    print(f"dedup chunks: ids partition, n={n}", flush=True)
    v = torch.from_numpy(vals).cuda()
    keys, offs, inv, info = R.IdsPartition()(v, G, seed)
    torch.cuda.synchronize()
    assert int(info[0].item()) == n and int(info[1].item()) == 0
    ek, eo, _, _ = O.ids_partition(vals, G, seed)
    assert np.array_equal(keys[:n].cpu().numpy(), ek), "keys grouped by owner"
    assert np.array_equal(offs.cpu().numpy(), eo), "shard offsets"
    assert torch.equal(keys[inv.long()], v), "keys_out[inverse] == values"
    del v, keys, inv
    _cleanup()
