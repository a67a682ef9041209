"""Host logic on the CPU: the seeded input generators and bench.py's byte
accounting.

The generators hold none of the method's arithmetic; these checks tie them to
the workload recipes they stand for (shapes, length distributions, Zipf
exponents, vocabularies, key namespaces) and to determinism by seed.  The
accounting helpers are checked on hand-sized batches.
"""
import importlib.util
import os

import numpy as np
import pytest

from paper_2509_20883_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


# --------------------------------------------------------------------------- generators


def test_batches_are_deterministic_and_feature_major():
    for k in (0, 1, 2, 5):
        w = W.workload(k, mini=True)
        a, b = W.make_batch(w, 3), W.make_batch(w, 3)
        assert np.array_equal(a.values, b.values) and np.array_equal(a.offsets, b.offsets)
        c = W.make_batch(w, 4)
        assert not np.array_equal(a.values, c.values) or a.n == 0
        assert a.offsets[0] == 0 and a.offsets[-1] == a.n and np.all(np.diff(a.offsets) >= 0)
        assert a.bags == w.batch * w.n_features


@pytest.mark.parametrize("k,lo,hi", [(0, 1, 8), (5, 16, 234)])
def test_uniform_bag_lengths(k, lo, hi):
    w = W.workload(k)
    lens = np.diff(W.make_batch(w, 0).offsets)
    assert lens.min() >= lo and lens.max() <= hi
    assert abs(lens.mean() - (lo + hi) / 2) < 0.05 * (lo + hi)


def test_multi_hot_poisson_lengths_and_namespaced_keys():
    w = W.workload(2, mini=True)
    b = W.make_batch(w, 0)
    lens = np.diff(b.offsets)
    assert lens.min() >= 1 and lens.max() <= 200
    assert abs(lens.mean() - 20) < 1.0
    fid = b.values >> W.ID_BITS
    # feature f's ids carry f in the high bits, feature-major
    bags_per_f = w.batch
    for f in (0, 7, w.n_features - 1):
        seg = b.values[b.offsets[f * bags_per_f]:b.offsets[(f + 1) * bags_per_f]]
        assert np.all((seg >> W.ID_BITS) == f)
    assert fid.min() == 0 and fid.max() == w.n_features - 1


def test_single_hot_workload_shape():
    w = W.workload(1)
    assert (w.batch, w.n_features, w.dim, w.zipf_s) == (65536, 26, 64, 1.05)
    assert all(10 ** 2 - 1 <= v <= 10 ** 7 + 1 for v in w.vocab)
    b = W.make_batch(w, 0, batch=512)
    assert np.all(np.diff(b.offsets) == 1)


def test_zipf_ranks_follow_the_exponent():
    g = np.random.default_rng(0)
    for s in (1.05, 1.2):
        r = W.zipf_ranks(400000, 10 ** 6, s, g)
        assert r.min() >= 1 and r.max() <= 10 ** 6
        c = np.bincount(r, minlength=11)
        # P(1) / P(2) = 2^s and P(1) / P(4) = 4^s within sampling error
        assert abs(c[1] / c[2] - 2 ** s) < 0.1 * 2 ** s
        assert abs(c[1] / c[4] - 4 ** s) < 0.15 * 4 ** s
    # the rejection-inversion sampler (vocabularies above 1e7) agrees
    r = W.zipf_ranks(300000, 10 ** 8, 1.2, g)
    c = np.bincount(r[r <= 4], minlength=5)
    assert abs(c[1] / c[2] - 2 ** 1.2) < 0.15 * 2 ** 1.2 and r.max() <= 10 ** 8


def test_rank_to_id_is_a_bijection_on_40_bits():
    r = np.arange(200000, dtype=np.int64)
    ids = W.rank_to_id(r, 12345)
    assert len(np.unique(ids)) == r.size
    assert ids.min() >= 0 and ids.max() < (1 << W.ID_BITS)


def test_prepopulation_subset_is_about_ninety_percent():
    w = W.workload(1)
    ids = W.rank_to_id(np.arange(1, 100001, dtype=np.int64), w.salt(3))
    frac = W.prepop_member(w, 3, ids).mean()
    assert 0.88 < frac < 0.92


def test_ids_partition_and_feature_inputs():
    v = W.ids_partition_values(0, batch=100)
    assert v.size == 26 * 100
    vals, co, bnd, bo = W.bucketize_columns(5, 1000, 7, step=1)
    assert co.tolist() == [0, 1000, 2000, 3000, 4000, 5000] and bo[-1] == 35
    for c in range(5):
        assert np.all(np.diff(bnd[bo[c]:bo[c + 1]]) >= 0)       # sorted boundaries
    ids, co, m = W.mod_columns(4, [10, 0, 5, 3], step=2)
    assert co.tolist() == [0, 10, 10, 15, 18] and np.all(m >= 100) and np.all(m <= 10 ** 7)


# --------------------------------------------------------------------------- bench accounting


def test_window_mask_head_and_tail():
    B = _bench()
    w = W.workload(5)
    w.pad_len = 3
    off = np.array([0, 2, 7, 7, 10], dtype=np.int64)          # lengths 2, 5, 0, 3
    tail = B.window_mask(w, off, 10)
    assert tail.tolist() == [1, 1, 0, 0, 1, 1, 1, 1, 1, 1]
    w.mode = W.NONE
    head = B.window_mask(w, off, 10)
    assert head.tolist() == [1, 1, 1, 1, 1, 0, 0, 1, 1, 1]
    w.mode = W.SUM
    assert B.window_mask(w, off, 10) is None


def test_key_stats_and_kernel_bytes_by_hand():
    B = _bench()
    vals = np.array([7] * 40 + [1, 2, 2, 3], dtype=np.int64)    # one hot key (40 ids), three short keys
    # bags 0-3: ten 7s each; bag 4: [1]; bag 5: [2]; bag 6: [2, 3]; bags 7-9 empty
    offs = np.array([0, 10, 20, 30, 40, 41, 42, 44, 44, 44, 44], dtype=np.int64)
    G = offs.size - 1
    ks = B.key_stats(vals, offs)
    assert (ks["U"], ks["U_long"], ks["N_long"], ks["U_short"], ks["N_short"]) == (4, 1, 40, 3, 4)
    assert ks["units"] == 2                                      # 40 ids in units of 32
    assert (ks["Gb_long"], ks["Gb_short"]) == (4, 3)             # distinct bags of each kind of key
    w = W.workload(0)                                            # dim 16 fp32, Adagrad, sum
    R, S = B.row_bytes(w)
    assert (R, S) == (64, 64)
    N, U = vals.size, 4
    # short keys: each of their 3 bags' gradient rows once, 4 inverse reads, 3 row+state updates;
    # the implementation also reads every key's segment descriptor and one gradient row per id
    assert B.kernel_bytes(w, "bwd_short", N, G, ks) == (64 * 3 + 4 * 4 + 2 * (R + S) * 3,
                                                        16 * 4 + 4 * 4 + 64 * 4 + 2 * (R + S) * 3)
    # hot key: its 4 bags' gradient rows, 40 inverse reads, one update; the implementation reads
    # 2 unit descriptors, 40 gradient rows, and writes and reads 2 partial rows
    assert B.kernel_bytes(w, "bwd_long", N, G, ks) == (64 * 4 + 4 * 40 + 2 * (R + S),
                                                       16 * 2 + 4 * 40 + 64 * 40 + 2 * 4 * 16 * 2 + 2 * (R + S))
    # pool: offsets, inverse, row ids, unique rows, output; the implementation reads a row id per
    # id and writes each id's gradient row
    out = G * 16 * 4
    assert B.kernel_bytes(w, "pool", N, G, ks) == (8 * (G + 1) + 4 * N + 8 * U + R * U + out,
                                                   8 * (G + 1) + 8 * N + R * U + out + 4 * N)
    w.opt = 5                                                    # row-wise Adam: m per element + v per row
    assert B.row_bytes(w) == (64, 4 * 17)


def test_ids_partition_bytes():
    B = _bench()
    assert B.ids_partition_bytes(100, 10, 8) == 800 + 80 + 72 + 400 + 16


def test_b_occ_counts_every_gathered_row():
    B = _bench()
    w = W.workload(0)                                            # dim 16 fp32: 64-byte rows
    R, _ = B.row_bytes(w)
    # 100 ids over 30 unique keys: 70 re-read rows more than the algorithmic count
    assert B.b_occ(w, 100, 10, 30, 5) - B.b_alg(w, 100, 10, 30, 5) == R * 70
    w.mode, w.pad_len = W.NONE, 4                                # padded: only the copied window's rows
    assert B.b_occ(w, 100, 10, 30, 5, V=40) - B.b_alg(w, 100, 10, 30, 5, V=40) == R * 10
