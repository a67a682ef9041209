"""Fused bucketize and mod on the GPU (through the C ABI) against the CPU oracle.

Integer outputs, so bit-exact.  Cases: the benchmark shape (100 columns of
10,000 values), columns shorter than a block (blocks spanning many columns,
the global-memory search), more columns than the LDS stage holds, empty columns, more boundaries than the LDS stage
holds, no boundaries, NaN / -0.0 / exact boundary hits, extreme ids, moduli 1
and near 2^62, a single element, and the host-side validation.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import recis as R
from paper_2509_20883_amd import workloads as W

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _bucketize_gpu(v, co, b, bo, validate=True):
    out = R.fused_bucketize(_dev(v), _dev(co), _dev(b if b.size else np.zeros(1, np.float32)), _dev(bo),
                            validate=validate)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def _mod_gpu(v, co, m, validate=True):
    out = R.fused_mod(_dev(v), _dev(co), _dev(m), validate=validate)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_bucketize_benchmark_shape():
    _log("bucketize 100 x 10000")
    args = W.bucketize_columns()
    assert np.array_equal(_bucketize_gpu(*args), O.bucketize(*args))


def test_bucketize_ragged_small_empty_and_wide_columns():
    g = np.random.default_rng(7)
    sizes = g.integers(0, 700, size=300)
    sizes[::7] = 0
    nb = g.integers(0, 40, size=300)
    nb[3], nb[10], nb[11] = 5000, 0, 9000           # wider than the LDS stage; none
    _log("bucketize 300 ragged columns")
    v, co, b, bo = W.bucketize_columns(300, sizes, nb, step=3)
    v[::13] = np.nan
    v[5::29] = -0.0
    hits = np.flatnonzero(np.diff(co) > 0)
    for c in hits[:50]:                              # exact boundary hits
        if bo[c + 1] > bo[c]:
            v[co[c]] = b[bo[c] + (bo[c + 1] - bo[c]) // 2]
    assert np.array_equal(_bucketize_gpu(v, co, b, bo), O.bucketize(v, co, b, bo))
    _log("bucketize one long column with 9000 boundaries")
    v, co, b, bo = W.bucketize_columns(2, [50000, 3], [9000, 1], step=4)
    assert np.array_equal(_bucketize_gpu(v, co, b, bo), O.bucketize(v, co, b, bo))
    _log("bucketize single element")
    v, co, b, bo = W.bucketize_columns(1, 1, 3, step=5)
    assert np.array_equal(_bucketize_gpu(v, co, b, bo), O.bucketize(v, co, b, bo))


def test_mod_benchmark_shape_and_ragged():
    _log("mod 100 x 10000")
    args = W.mod_columns()
    assert np.array_equal(_mod_gpu(*args), O.mod(*args))
    g = np.random.default_rng(8)
    sizes = g.integers(0, 900, size=500)
    sizes[::5] = 0
    _log("mod 500 ragged columns, extreme ids")
    v, co, m = W.mod_columns(500, sizes, step=2)
    v[:4] = [np.iinfo(np.int64).min, np.iinfo(np.int64).max, -1, 0]
    m[0], m[1], m[2] = 1, (1 << 62) + 7, 3
    assert np.array_equal(_mod_gpu(v, co, m), O.mod(v, co, m))


def test_more_columns_than_the_lds_stage():
    g = np.random.default_rng(10)
    sizes = g.integers(0, 300, size=1500)
    _log("bucketize 1500 columns")
    v, co, b, bo = W.bucketize_columns(1500, sizes, g.integers(0, 20, size=1500), step=6)
    assert np.array_equal(_bucketize_gpu(v, co, b, bo), O.bucketize(v, co, b, bo))
    _log("mod 1500 columns")
    v, co, m = W.mod_columns(1500, sizes, step=6)
    assert np.array_equal(_mod_gpu(v, co, m), O.mod(v, co, m))


def test_validation_and_nonpositive_modulus():
    v, co, m = W.mod_columns(4, 100, step=9)
    bad = m.copy()
    bad[2] = 0
    with pytest.raises(R.RecisError):
        _mod_gpu(v, co, bad, validate=True)
    out = _mod_gpu(v, co, bad, validate=False)      # documented: -1 for that column
    assert np.all(out[co[2]:co[3]] == -1)
    keep = np.r_[0:co[2], co[3]:co[4]]
    assert np.array_equal(out[keep], O.mod(v, co, np.where(bad > 0, bad, 1))[keep])
    vb, cb, b, bo = W.bucketize_columns(4, 100, 5, step=9)
    cbad = cb.copy()
    cbad[2] = cbad[3] + 1
    with pytest.raises(R.RecisError):
        _bucketize_gpu(vb, cbad, b, bo, validate=True)
    with pytest.raises(R.RecisError):
        R.fused_mod(_dev(v), _dev(np.zeros(1, np.int64)), _dev(m))   # ncols = 0
