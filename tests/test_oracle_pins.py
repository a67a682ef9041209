"""Pins of the CPU oracle against things other than itself (CPU only).

Each check ties one oracle function to a published value, an exact rational
computation, a library routine (numpy / torch on the CPU), a closed form or a
brute force over tiny inputs, so that a dropped term, wrong sign, wrong index
or transposed operand in the oracle fails here.
"""
import itertools
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


def _vectors():
    vals = []
    with open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("seed"):
                seed = int(line.split()[1])
                continue
            vals.append(int(line))
    return seed, vals


# --------------------------------------------------------------------------- mix64


def test_mix64_matches_published_splitmix64_vectors():
    seed, vals = _vectors()
    s = seed
    for v in vals:
        s = (s + GAMMA) & M64
        assert O.mix64(s) == v


def _unxorshift(y, k):
    x = y
    sh = k
    while sh < 64:
        x ^= y >> sh
        sh += k
    return x & M64


def mix64_inverse(z):
    """Inverse of the splitmix64 output function, step by step."""
    z = _unxorshift(z, 31)
    z = (z * pow(0x94D049BB133111EB, -1, 1 << 64)) & M64
    z = _unxorshift(z, 27)
    z = (z * pow(0xBF58476D1CE4E5B9, -1, 1 << 64)) & M64
    z = _unxorshift(z, 30)
    return z


def test_mix64_is_a_bijection():
    g = np.random.default_rng(1)
    for x in g.integers(0, 2**63, size=200, dtype=np.int64).tolist() + [0, 1, M64]:
        assert mix64_inverse(O.mix64(x)) == x


# --------------------------------------------------------------------------- row init


def _round_f32(fr: Fraction) -> np.float32:
    """Exact round-to-nearest-even of a rational to fp32."""
    f = np.float32(float(fr))
    cands = {f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))}
    best = None
    for c in cands:
        d = abs(Fraction(float(c)) - fr)
        key = (d, int(np.array(c, dtype=np.float32).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def _key_for_stream_state(seed, z):
    """The key whose per-row hash stream starts at splitmix64 state z."""
    k = mix64_inverse(z) ^ O.mix64(seed)
    return k - (1 << 64) if k >= (1 << 63) else k


@pytest.mark.parametrize("seed", [0, 2509, 0xDEADBEEFCAFEF00D])
def test_init_row_is_splitmix64_stream_on_unit_interval(seed):
    # With lo=0, hi=1 element j is exactly the top 24 bits of the (j+1)-th
    # splitmix64 output from the key's stream state, divided by 2^24.
    s0, vals = _vectors()
    key = _key_for_stream_state(seed, s0)
    w = O.init_row(seed, key, len(vals), 0.0, 1.0)
    expect = np.array([(v >> 40) / float(1 << 24) for v in vals], dtype=np.float32)
    assert np.array_equal(w, expect)


def test_init_row_single_rounding_on_symmetric_interval():
    s0, vals = _vectors()
    seed = 77
    key = _key_for_stream_state(seed, s0)
    lo, hi = np.float32(-0.01), np.float32(0.01)
    span = np.float32(hi - lo)
    w = O.init_row(seed, key, len(vals), float(lo), float(hi))
    for j, v in enumerate(vals):
        u = Fraction(v >> 40, 1 << 24)
        exact = u * Fraction(float(span)) + Fraction(float(lo))
        assert w[j] == _round_f32(exact), j


def test_init_row_distribution_and_sensitivity():
    D = 16
    keys = np.arange(-4000, 4000, 3, dtype=np.int64)
    W = np.stack([O.init_row(5, int(k), D, -0.01, 0.01) for k in keys])
    assert W.min() >= -0.01 and W.max() <= np.float32(0.01)
    # uniform on [-0.01, 0.01]: mean 0, variance 0.02^2/12, per element position
    assert abs(W.mean()) < 2e-4
    assert abs(W.var() / (0.02**2 / 12) - 1) < 0.05
    for j in range(D):
        assert abs(W[:, j].mean()) < 1.2e-3
    # adjacent elements uncorrelated; different seed / key give different rows
    c = np.corrcoef(W[:, :-1].ravel(), W[:, 1:].ravel())[0, 1]
    assert abs(c) < 0.05
    assert not np.array_equal(O.init_row(5, 10, D, -0.01, 0.01), O.init_row(6, 10, D, -0.01, 0.01))
    assert not np.array_equal(O.init_row(5, 10, D, -0.01, 0.01), O.init_row(5, 11, D, -0.01, 0.01))
    assert np.array_equal(O.init_row(5, 10, D, -0.01, 0.01), O.init_row(5, 10, D, -0.01, 0.01))


# --------------------------------------------------------------------------- bf16


def test_bf16_roundtrip_exhaustive():
    for h in range(1 << 16):
        x = O.bf16_to_f32(h)
        if np.isnan(x):
            assert O.bf16_rne(x) == 0x7FC0
        else:
            assert O.bf16_rne(x) == h


def test_bf16_rne_matches_torch_including_ties():
    g = np.random.default_rng(3)
    bits = g.integers(0, 1 << 32, size=20000, dtype=np.uint64).astype(np.uint32)
    # force exact ties (low 16 bits 0x8000) and near-ties on a third of them
    bits[::3] = (bits[::3] & 0xFFFF0000) | 0x8000
    bits[1::7] = (bits[1::7] & 0xFFFF0000) | 0x7FFF
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([O.bf16_rne(float(v)) for v in x], dtype=np.uint16)
    assert np.array_equal(got, ref)


# --------------------------------------------------------------------------- dedup


def _first_occurrence_unique(seq):
    _, idx = np.unique(seq, return_index=True)
    return seq[np.sort(idx)]


def test_dedup_brute_force_all_sequences_over_4_keys():
    alphabet = np.array([7, -3, 0, 2**62], dtype=np.int64)
    for n in range(0, 5):
        for combo in itertools.product(range(4), repeat=n):
            seq = alphabet[list(combo)] if n else np.zeros(0, dtype=np.int64)
            st, u, inv = O.dedup(seq)
            assert st == O.OK
            assert np.array_equal(u, _first_occurrence_unique(seq))
            assert np.array_equal(u[inv], seq)


def test_dedup_invariants_large():
    g = np.random.default_rng(11)
    seq = g.zipf(1.3, size=50000).astype(np.int64) * 1_000_003 - 7
    st, u, inv = O.dedup(seq)
    assert st == O.OK
    assert np.array_equal(u[inv], seq)                       # reconstruction
    assert len(np.unique(u)) == len(u)                       # distinct
    assert np.array_equal(np.sort(u), np.unique(seq))        # same set as numpy
    first = np.full(len(u), len(seq))
    np.minimum.at(first, inv, np.arange(len(seq)))
    assert np.all(np.diff(first) > 0)                        # first-occurrence order


def test_dedup_rejects_reserved_keys():
    for bad in (np.iinfo(np.int64).min, np.iinfo(np.int64).min + 1):
        st, _, _ = O.dedup(np.array([1, bad, 2], dtype=np.int64))
        assert st == O.EKEY
    st, u, _ = O.dedup(np.array([np.iinfo(np.int64).max, 0, -1], dtype=np.int64))
    assert st == O.OK and len(u) == 3


# --------------------------------------------------------------------------- ids partition


def _s64(x):
    x &= M64
    return x - (1 << 64) if x >= 1 << 63 else x


def _partition_brute(seq, G, seed):
    """Distinct keys sorted by (owner, first position): a sort, not the
    oracle's shard-by-shard scan; owners from the pinned mix64."""
    first = {}
    for i, k in enumerate(seq.tolist()):
        first.setdefault(k, i)
    own = {k: O.mix64((k & M64) ^ seed) % G for k in first}
    keys = sorted(first, key=lambda k: (own[k], first[k]))
    offs = [0] * (G + 1)
    for k in keys:
        offs[own[k] + 1] += 1
    offs = np.cumsum(offs)
    pos = {k: j for j, k in enumerate(keys)}
    return np.array(keys, dtype=np.int64), offs, np.array([pos[k] for k in seq.tolist()], dtype=np.int32)


def test_ids_partition_owner_pinned_to_published_vectors():
    # keys whose owner hash input is a splitmix64 state with a published
    # output: owner = that output mod G (G = 3 and 4 catch a mask for a mod
    # and a dropped seed)
    seed, vals = _vectors()
    oseed = 0xA5A5F00DCAFE1234
    states = [(seed + (j + 1) * GAMMA) & M64 for j in range(len(vals))]
    ks = [_s64(z ^ oseed) for z in states]
    order = [2, 0, 2, 4, 1, 3, 0, 1, 4, 4]
    seq = np.array([ks[j] for j in order], dtype=np.int64)
    for G in (3, 4):
        keys, offs, inv, rej = O.ids_partition(seq, G, oseed)
        own = {ks[j]: vals[j] % G for j in range(len(vals))}
        firstpos = {}
        for i, j in enumerate(order):
            firstpos.setdefault(ks[j], i)
        want = sorted(firstpos, key=lambda k: (own[k], firstpos[k]))
        assert keys.tolist() == want and rej == 0
        for s_ in range(G):
            seg = keys[offs[s_]:offs[s_ + 1]].tolist()
            assert all(own[k] == s_ for k in seg)
        assert offs[0] == 0 and offs[G] == len(want)
        assert np.array_equal(keys[inv], seq)


def test_ids_partition_brute_force_small():
    g = np.random.default_rng(21)
    for trial in range(60):
        n = int(g.integers(0, 40))
        alphabet = g.integers(-2**63 + 2, 2**63 - 1, size=int(g.integers(1, 12)), dtype=np.int64)
        seq = alphabet[g.integers(0, len(alphabet), size=n)] if n else np.zeros(0, dtype=np.int64)
        G = int(g.choice([1, 2, 3, 5, 8, 16]))
        seed = int(g.integers(0, 2**63)) * 2 + trial % 2
        keys, offs, inv, rej = O.ids_partition(seq, G, seed)
        ek, eo, ei = _partition_brute(seq, G, seed)
        assert np.array_equal(keys, ek) and np.array_equal(offs, eo) and np.array_equal(inv, ei) and rej == 0


def test_ids_partition_one_shard_is_dedup():
    g = np.random.default_rng(5)
    seq = g.zipf(1.2, size=20000).astype(np.int64) * 7919 - 3
    keys, offs, inv, _ = O.ids_partition(seq, 1, 123)
    st, u, uinv = O.dedup(seq)
    assert st == O.OK
    assert np.array_equal(keys, u) and np.array_equal(inv, uinv)
    assert offs.tolist() == [0, len(u)]


def test_ids_partition_invariants_large():
    g = np.random.default_rng(8)
    seq = (g.zipf(1.1, size=60000).astype(np.int64) * 1_000_003) ^ 0x5555
    G = 8
    keys, offs, inv, rej = O.ids_partition(seq, G, 99)
    assert rej == 0
    assert np.array_equal(keys[inv], seq)                          # reconstruction
    assert len(np.unique(keys)) == len(keys)                       # distinct
    assert np.array_equal(np.sort(keys), np.unique(seq))           # same set
    assert offs[0] == 0 and offs[-1] == len(keys) and np.all(np.diff(offs) >= 0)
    first = np.full(len(keys), len(seq))
    np.minimum.at(first, inv, np.arange(len(seq)))
    for s_ in range(G):
        lo, hi = offs[s_], offs[s_ + 1]
        assert all(O.mix64((int(k) & M64) ^ 99) % G == s_ for k in keys[lo:hi][:200])
        assert np.all(np.diff(first[lo:hi]) > 0)                   # first-occurrence order in a shard
    # a good owner hash spreads the distinct keys evenly (chi-square, 7 dof)
    cnt = np.diff(offs)
    exp = len(keys) / G
    assert ((cnt - exp) ** 2 / exp).sum() < 30


def test_ids_partition_reserved_keys_and_empty():
    lo = np.iinfo(np.int64).min
    seq = np.array([4, lo, 9, lo + 1, 4, lo], dtype=np.int64)
    keys, offs, inv, rej = O.ids_partition(seq, 2, 0)
    assert rej == 3
    assert sorted(keys.tolist()) == [4, 9]
    assert inv[1] == -1 and inv[3] == -1 and inv[5] == -1
    assert keys[inv[0]] == 4 and keys[inv[2]] == 9 and inv[4] == inv[0]
    keys, offs, inv, rej = O.ids_partition(np.zeros(0, dtype=np.int64), 5, 1)
    assert len(keys) == 0 and offs.tolist() == [0] * 6 and len(inv) == 0 and rej == 0
    with pytest.raises(ValueError):
        O.ids_partition(seq, 0, 0)


# --------------------------------------------------------------------------- bucketize / mod


def _columns(g, ncols, lo, hi):
    sizes = g.integers(lo, hi, size=ncols)
    off = np.zeros(ncols + 1, dtype=np.int64)
    np.cumsum(sizes, out=off[1:])
    return off


def test_bucketize_matches_searchsorted_right_and_tf_examples():
    # TensorFlow's documented example: boundaries [0, 10, 100],
    # input [[-5, 10000], [150, 10], [5, 100]] -> [[0, 3], [3, 2], [1, 3]]
    out = O.bucketize(np.array([-5, 10000, 150, 10, 5, 100], np.float32), np.array([0, 6]),
                      np.array([0, 10, 100], np.float32), np.array([0, 3]))
    assert out.tolist() == [0, 3, 3, 2, 1, 3]
    g = np.random.default_rng(31)
    coff = _columns(g, 40, 0, 300)
    nb = g.integers(0, 50, size=40)
    boff = np.zeros(41, dtype=np.int64)
    np.cumsum(nb, out=boff[1:])
    bnd = np.concatenate([np.sort(g.choice(np.linspace(-5, 5, 41), size=k).astype(np.float32)) for k in nb]
                         + [np.zeros(0, np.float32)])
    vals = g.choice(np.linspace(-6, 6, 121), size=int(coff[-1])).astype(np.float32)  # hits boundaries exactly
    vals[::17] = np.nan
    vals[5::23] = -0.0
    out = O.bucketize(vals, coff, bnd, boff)
    for c in range(40):
        v = vals[coff[c]:coff[c + 1]]
        b = bnd[boff[c]:boff[c + 1]]
        want = np.searchsorted(b, v, side="right")   # numpy orders NaN after every number
        assert np.array_equal(out[coff[c]:coff[c + 1]], want)


def test_mod_matches_numpy_floor_mod():
    g = np.random.default_rng(32)
    coff = _columns(g, 30, 0, 400)
    mods = g.integers(1, 10**6, size=30)
    mods[0], mods[1] = 1, (1 << 62) + 7
    vals = g.integers(-2**63, 2**63 - 1, size=int(coff[-1]), dtype=np.int64)
    vals[:3] = [np.iinfo(np.int64).min, -1, np.iinfo(np.int64).max]
    out = O.mod(vals, coff, mods)
    for c in range(30):
        v = vals[coff[c]:coff[c + 1]]
        assert np.array_equal(out[coff[c]:coff[c + 1]], np.mod(v, np.int64(mods[c])))
    # by hand: Python's % is the floor modulus
    out = O.mod(np.array([-7, 7, -1, 0, 12], np.int64), np.array([0, 5]), np.array([5]))
    assert out.tolist() == [-7 % 5, 7 % 5, -1 % 5, 0, 12 % 5]
    with pytest.raises(ValueError):
        O.mod(np.array([1], np.int64), np.array([0, 1]), np.array([0]))


# --------------------------------------------------------------------------- find-or-insert


def test_find_or_insert_invariants():
    T = O.Table(8, seed=9)
    g = np.random.default_rng(2)
    keys = g.integers(-50, 50, size=300).astype(np.int64)
    st, rows, nn = T.find_or_insert(keys)
    assert st == O.OK
    U = len(np.unique(keys))
    assert nn == U and T.size() == U
    # same key -> same row, distinct keys -> distinct rows, rows in [0, live)
    for k in np.unique(keys):
        assert len(set(rows[keys == k])) == 1
    assert len(set(rows.tolist())) == U and rows.min() == 0 and rows.max() == U - 1
    # new rows are numbered in first-occurrence order
    assert np.array_equal(rows[np.sort(np.unique(keys, return_index=True)[1])], np.arange(U))
    # re-inserting inserts nothing and returns the same rows
    st2, rows2, nn2 = T.find_or_insert(keys[::-1])
    assert nn2 == 0 and np.array_equal(rows2, rows[::-1])
    # present set equals the inserted set; rows hold their init values, state zero
    ek, er = T.export()
    assert np.array_equal(np.sort(ek), np.unique(keys))
    found, w, s = T.read_rows(np.unique(keys))
    assert found == U and np.all(s == 0)
    for k, wr in zip(np.unique(keys), w):
        assert np.array_equal(wr, O.init_row(9, int(k), 8, -0.01, 0.01))


def test_find_or_insert_bounded_table_efull_and_ekey():
    T = O.Table(4, max_live=3)
    st, rows, nn = T.find_or_insert(np.array([5, 6, 5, 7, 8, 9, 6], dtype=np.int64))
    assert st == O.EFULL and nn == 3
    assert rows.tolist() == [0, 1, 0, 2, -1, -1, 1]
    st, _, _ = T.find_or_insert(np.array([np.iinfo(np.int64).min], dtype=np.int64))
    assert st == O.EKEY


def test_bf16_table_rows_are_rounded_init():
    T = O.Table(8, row_dtype=O.BF16, seed=4)
    T.find_or_insert(np.array([1, 2, 3], dtype=np.int64))
    _, w, _ = T.read_rows(np.array([1, 2, 3], dtype=np.int64))
    for k, wr in zip([1, 2, 3], w):
        ref = torch.from_numpy(O.init_row(4, k, 8, -0.01, 0.01)).to(torch.bfloat16).float().numpy()
        assert np.array_equal(wr, ref)


# --------------------------------------------------------------------------- pooling


def _tiny_batch(g, n_bags, max_len, vocab, allow_empty=True):
    lens = g.integers(0 if allow_empty else 1, max_len + 1, size=n_bags)
    off = np.zeros(n_bags + 1, dtype=np.int64)
    np.cumsum(lens, out=off[1:])
    vals = (g.zipf(1.4, size=int(off[-1])) % vocab).astype(np.int64) * 31 + 5
    return vals, off


@pytest.mark.parametrize("row_dtype", [O.F32, O.BF16])
@pytest.mark.parametrize("mode", [O.SUM, O.MEAN])
def test_pooling_matches_torch_embedding_bag(mode, row_dtype):
    g = np.random.default_rng(5 + mode + 10 * row_dtype)
    vals, off = _tiny_batch(g, 60, 9, 40)
    D = 12
    T = O.Table(D, row_dtype=row_dtype, seed=3)
    r = T.forward(vals, off, mode)
    assert r["status"] == O.OK
    # dense weight from the rows the oracle holds, indexed by unique position
    _, W, _ = T.read_rows(r["unique"])
    idx = torch.from_numpy(r["inverse"].astype(np.int64))
    ref = torch.nn.functional.embedding_bag(idx, torch.from_numpy(W.astype(np.float64)),
                                            torch.from_numpy(off[:-1]), mode=["sum", "mean"][mode])
    np.testing.assert_allclose(r["out"], ref.numpy(), rtol=0, atol=1e-15)
    # a bag of length one is its row, bit-exact; total mass = sum_u count_u * w_u
    lens = np.diff(off)
    for gi in np.nonzero(lens == 1)[0][:5]:
        assert np.array_equal(r["out"][gi], W[r["inverse"][off[gi]]].astype(np.float64))
    if mode == O.SUM:
        cnt = np.bincount(r["inverse"], minlength=r["U"])
        np.testing.assert_allclose(r["out"].sum(0), (cnt[:, None] * W.astype(np.float64)).sum(0), atol=1e-12)
    assert np.all(r["out"][lens == 0] == 0)


def test_padded_gather_and_mask():
    g = np.random.default_rng(8)
    vals, off = _tiny_batch(g, 20, 12, 25)
    L, D = 8, 4
    T = O.Table(D, row_dtype=O.BF16, opt=O.ADAM, seed=1)
    r = T.forward(vals, off, O.NONE, pad_len=L)
    _, W, _ = T.read_rows(r["unique"])
    lens = np.diff(off)
    for gi in range(len(lens)):
        for t in range(L):
            if t < lens[gi]:
                assert r["mask"][gi, t] == 1
                assert np.array_equal(r["out"][gi, t], W[r["inverse"][off[gi] + t]])
            else:
                assert r["mask"][gi, t] == 0 and np.all(r["out"][gi, t] == 0)


def test_sequence_tile_tail_is_the_concat_of_the_last_rows():
    g = np.random.default_rng(12)
    vals, off = _tiny_batch(g, 25, 16, 30)
    L, D = 6, 4
    T = O.Table(D, seed=5)
    r = T.forward(vals, off, O.TAIL, pad_len=L)
    assert r["status"] == O.OK
    lens = np.diff(off)
    # definition: row g of the [B, L*D] tile is the concatenation of the rows
    # of the bag's last min(len, L) ids, zero-padded to L*D
    for gi in range(len(lens)):
        ids = vals[off[gi]:off[gi + 1]][-L:] if lens[gi] else vals[:0]
        _, Wg, _ = T.read_rows(ids) if ids.size else (0, np.zeros((0, D), np.float32), 0)
        want = np.zeros(L * D)
        want[:ids.size * D] = Wg.astype(np.float64).reshape(-1)
        assert np.array_equal(r["out"].reshape(len(lens), L * D)[gi], want)
        assert r["mask"][gi].tolist() == [1] * min(lens[gi], L) + [0] * (L - min(lens[gi], L))
    # the same as the head copy of a batch cut to each bag's last L ids
    cut = [vals[off[gi]:off[gi + 1]][-L:] for gi in range(len(lens))]
    off2 = np.zeros_like(off)
    np.cumsum([c.size for c in cut], out=off2[1:])
    r2 = O.Table(D, seed=5).forward(np.concatenate(cut), off2, O.NONE, pad_len=L)
    assert np.array_equal(r["out"], r2["out"]) and np.array_equal(r["mask"], r2["mask"])
    # ids cut off the front are still looked up (inserted)
    assert T.size() == len(np.unique(vals))


def test_backward_adjoint_identity_tail_tile():
    g = np.random.default_rng(14)
    vals, off = _tiny_batch(g, 30, 14, 20)
    L, D = 5, 3
    st, u, inv = O.dedup(vals)
    U = len(u)
    W = g.standard_normal((U, D))
    G = g.standard_normal((len(off) - 1, L, D)).astype(np.float32)
    lens = np.diff(off)
    fw = np.zeros((len(off) - 1, L, D))
    for gi in range(len(lens)):
        skip = max(lens[gi] - L, 0)
        for t in range(min(lens[gi], L)):
            fw[gi, t] = W[inv[off[gi] + skip + t]]
    Gn = G.copy()
    Gn[np.arange(L)[None, :] >= lens[:, None]] = np.nan
    gu = O.backward(off, inv, U, D, O.TAIL, L, Gn)
    assert np.all(np.isfinite(gu))
    lhs = float((fw * G.astype(np.float64)).sum())
    rhs = float((W * gu).sum())
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))
    # the ids cut off the front get no gradient
    front = np.zeros(U, bool)
    for gi in range(len(lens)):
        for i in range(off[gi], off[gi] + max(lens[gi] - L, 0)):
            front[inv[i]] = True
    kept = np.zeros(U, bool)
    for gi in range(len(lens)):
        for i in range(off[gi] + max(lens[gi] - L, 0), off[gi + 1]):
            kept[inv[i]] = True
    assert np.all(gu[front & ~kept] == 0)


# --------------------------------------------------------------------------- backward


@pytest.mark.parametrize("mode", [O.SUM, O.MEAN])
def test_backward_matches_torch_autograd(mode):
    g = np.random.default_rng(21 + mode)
    vals, off = _tiny_batch(g, 50, 10, 30)
    D = 6
    T = O.Table(D, seed=2)
    r = T.forward(vals, off, mode)
    _, W, _ = T.read_rows(r["unique"])
    G = g.standard_normal((len(off) - 1, D)).astype(np.float32)
    gu = O.backward(off, r["inverse"], r["U"], D, mode, 0, G)
    Wt = torch.from_numpy(W.astype(np.float64)).requires_grad_(True)
    out = torch.nn.functional.embedding_bag(torch.from_numpy(r["inverse"].astype(np.int64)), Wt,
                                            torch.from_numpy(off[:-1]), mode=["sum", "mean"][mode])
    out.backward(torch.from_numpy(G.astype(np.float64)))
    np.testing.assert_allclose(gu, Wt.grad.numpy(), rtol=1e-13, atol=1e-13)


def test_backward_adjoint_identity_padded_and_nan_masked():
    g = np.random.default_rng(4)
    vals, off = _tiny_batch(g, 30, 14, 20)
    L, D = 10, 3
    st, u, inv = O.dedup(vals)
    U = len(u)
    W = g.standard_normal((U, D))
    G = g.standard_normal((len(off) - 1, L, D)).astype(np.float32)
    # forward as a linear map of W (padded copy), then <fwd(W), G> = <W, bwd(G)>
    lens = np.diff(off)
    fw = np.zeros((len(off) - 1, L, D))
    for gi in range(len(lens)):
        for t in range(min(lens[gi], L)):
            fw[gi, t] = W[inv[off[gi] + t]]
    Gn = G.copy()
    Gn[np.arange(L)[None, :] >= lens[:, None]] = np.nan      # masked slots
    gu = O.backward(off, inv, U, D, O.NONE, L, Gn)
    assert np.all(np.isfinite(gu))
    lhs = float((fw * G.astype(np.float64)).sum())
    rhs = float((W * gu).sum())
    assert abs(lhs - rhs) <= 1e-12 * max(1.0, abs(lhs))


# --------------------------------------------------------------------------- optimizer


def test_first_step_closed_form_adagrad_and_adam():
    D = 5
    grads = np.array([[0.5, -2.0, 1e-3, 0.0, 7.0]], dtype=np.float32)
    for opt in (O.ADAGRAD, O.ADAM):
        T = O.Table(D, opt=opt, seed=1)
        _, rows, _ = T.find_or_insert(np.array([42], dtype=np.int64))
        _, w0, _ = T.read_rows(np.array([42], dtype=np.int64))
        lr, eps = 0.01, 1e-8
        T.optimizer(rows, grads, lr, eps)
        _, w1, s = T.read_rows(np.array([42], dtype=np.int64))
        gd = grads.astype(np.float64)
        expect = w0.astype(np.float64) - lr * gd / (np.abs(gd) + eps)
        np.testing.assert_allclose(w1, expect, rtol=0, atol=2e-9)
        if opt == O.ADAGRAD:
            np.testing.assert_array_equal(s[:, 0], (gd * gd).astype(np.float32))


def test_adagrad_matches_torch_multi_step_lazy():
    D, V = 4, 6
    g = np.random.default_rng(31)
    T = O.Table(D, opt=O.ADAGRAD, seed=7)
    keys = np.arange(V, dtype=np.int64) * 11
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    p = torch.nn.Parameter(torch.from_numpy(W0.astype(np.float64)))
    opt = torch.optim.Adagrad([p], lr=0.05, eps=1e-8, initial_accumulator_value=0.0)
    for step in range(5):
        touched = np.sort(g.choice(V, size=3, replace=False))
        G = g.standard_normal((3, D)).astype(np.float32)
        T.optimizer(rows[touched], G, 0.05, 1e-8)
        dense = torch.zeros(V, D, dtype=torch.float64)
        dense[touched] = torch.from_numpy(G.astype(np.float64))
        p.grad = dense
        opt.step()
    _, W, _ = T.read_rows(keys)
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-6, atol=1e-8)


def test_adam_matches_torch_sparse_adam_multi_step_lazy():
    D, V = 4, 7
    g = np.random.default_rng(32)
    T = O.Table(D, opt=O.ADAM, seed=8)
    keys = np.arange(V, dtype=np.int64) + 1000
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    p = torch.nn.Parameter(torch.from_numpy(W0.astype(np.float64)))
    opt = torch.optim.SparseAdam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    untouched_before = None
    for step in range(6):
        touched = np.sort(g.choice(V, size=3, replace=False))
        G = g.standard_normal((3, D)).astype(np.float32)
        if step == 2:
            G[0] = 0.0  # touched with a zero gradient still counts as touched
        _, before, sb = T.read_rows(keys)
        T.optimizer(rows[touched], G, 1e-3, 1e-8, 0.9, 0.999)
        _, after, sa = T.read_rows(keys)
        others = np.setdiff1d(np.arange(V), touched)
        assert np.array_equal(before[others], after[others]) and np.array_equal(sb[others], sa[others])
        idx = torch.from_numpy(touched.astype(np.int64))[None, :]
        p.grad = torch.sparse_coo_tensor(idx, torch.from_numpy(G.astype(np.float64)), (V, D))
        opt.step()
    _, W, _ = T.read_rows(keys)
    assert T.t == 6
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-5, atol=1e-9)


def test_adamw_matches_torch_adamw_multi_step():
    """AdamW (decoupled weight decay, the paper's SparseAdamW) against
    torch.optim.AdamW in fp64: every row is touched every step (then the lazy
    update equals the dense one); a partially touched step leaves the other
    rows, and their state, untouched (no decay either)."""
    D, V = 4, 6
    g = np.random.default_rng(33)
    T = O.Table(D, opt=O.ADAMW, seed=9)
    keys = np.arange(V, dtype=np.int64) + 2000
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    p = torch.nn.Parameter(torch.from_numpy(W0.astype(np.float64)))
    lr, wd = 0.1, 0.1  # steps of ~lr: decay before vs after the step differ by ~1e-3
    opt = torch.optim.AdamW([p], lr=lr, betas=(0.9, 0.999), eps=1e-8, weight_decay=wd)
    for step in range(5):
        G = g.standard_normal((V, D)).astype(np.float32)
        T.optimizer(rows, G, lr, 1e-8, 0.9, 0.999, weight_decay=wd)
        p.grad = torch.from_numpy(G.astype(np.float64))
        opt.step()
    _, W, _ = T.read_rows(keys)
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-5, atol=1e-9)
    # lazy: untouched rows keep their value (no decay) and state
    _, before, sb = T.read_rows(keys)
    T.optimizer(rows[:2], g.standard_normal((2, D)).astype(np.float32), lr, 1e-8, 0.9, 0.999, weight_decay=wd)
    _, after, sa = T.read_rows(keys)
    assert np.array_equal(before[2:], after[2:]) and np.array_equal(sb[2:], sa[2:])
    assert not np.array_equal(before[:2], after[:2])


def test_adam_eps_hat_form_identity_and_first_step():
    """Adam in the reordered form (lr_t = lr sqrt(1-b2^t) / (1-b1^t),
    w -= lr_t m / (sqrt(v) + eps_hat)) is Algorithm 1 with eps = eps_hat /
    sqrt(1-b2^t) (same moments); its first step from zero moments is
    w - lr sqrt(1-b2) g / (sqrt(1-b2) |g| + eps_hat)."""
    D, V = 8, 5
    g = np.random.default_rng(34)
    keys = np.arange(V, dtype=np.int64) + 3000
    lr, b1, b2, eps_hat = 2e-3, 0.9, 0.999, 1e-3
    # first step, closed form
    T = O.Table(D, opt=O.ADAM_TF, seed=10)
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    G = g.standard_normal((V, D)).astype(np.float32)
    T.optimizer(rows, G, lr, eps_hat, b1, b2)
    _, W1, S1 = T.read_rows(keys)
    Gd = G.astype(np.float64)
    ref = W0.astype(np.float64) - lr * np.sqrt(1 - b2) * Gd / (np.sqrt(1 - b2) * np.abs(Gd) + eps_hat)
    np.testing.assert_allclose(W1, ref, rtol=2e-7, atol=1e-12)
    np.testing.assert_allclose(S1[:, 0], (1 - b1) * Gd, rtol=1e-6)
    np.testing.assert_allclose(S1[:, 1], (1 - b2) * Gd * Gd, rtol=1e-6)
    # a later step from a random state: equal to Algorithm 1 with eps = eps_hat / sqrt(1 - b2^t)
    t = 7
    m = (0.1 * g.standard_normal((V, D))).astype(np.float32)
    v = (0.01 * np.abs(g.standard_normal((V, D)))).astype(np.float32)
    A = O.Table(D, opt=O.ADAM_TF, seed=10)
    B = O.Table(D, opt=O.ADAM, seed=10)
    for X in (A, B):
        X.find_or_insert(keys)
        X.write_rows(keys, W0, np.stack([m, v], axis=1))
        X.t = t - 1
    G = g.standard_normal((V, D)).astype(np.float32)
    A.optimizer(rows, G, lr, eps_hat, b1, b2)
    B.optimizer(rows, G, lr, eps_hat / np.sqrt(1 - b2 ** t), b1, b2)
    _, WA, SA = A.read_rows(keys)
    _, WB, SB = B.read_rows(keys)
    assert np.array_equal(SA, SB)
    ulp = np.spacing(np.abs(WB).astype(np.float32)).astype(np.float64)
    assert (np.abs(WA.astype(np.float64) - WB) <= ulp).all()
    assert not np.array_equal(WA, W0)


def test_step_is_forward_backward_optimizer():
    g = np.random.default_rng(41)
    vals, off = _tiny_batch(g, 40, 6, 25)
    D = 8
    G = g.standard_normal((len(off) - 1, D)).astype(np.float32)
    A = O.Table(D, opt=O.ADAM, seed=3)
    B = O.Table(D, opt=O.ADAM, seed=3)
    ra = A.step(vals, off, O.MEAN, G, 1e-3)
    rb = B.forward(vals, off, O.MEAN)
    gu = O.backward(off, rb["inverse"], rb["U"], D, O.MEAN, 0, G)
    B.optimizer(rb["rows"], gu.astype(np.float32), 1e-3)
    assert ra["U"] == rb["U"] and ra["n_new"] == rb["n_new"] == rb["U"]
    np.testing.assert_array_equal(ra["out"], rb["out"])
    _, wa, sa = A.read_rows(rb["unique"])
    _, wb, sb = B.read_rows(rb["unique"])
    assert np.array_equal(wa, wb) and np.array_equal(sa, sb)


# --------------------------------------------------------------------------- row-wise state


def test_rowwise_adagrad_dim1_matches_torch_adagrad():
    """With one element per row the row mean of g^2 is g^2: row-wise Adagrad
    is Adagrad (Duchi et al. 2011), here torch.optim.Adagrad over lazy steps."""
    V = 6
    g = np.random.default_rng(41)
    T = O.Table(1, opt=O.ADAGRAD_RW, seed=3)
    keys = np.arange(V, dtype=np.int64) * 7
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    p = torch.nn.Parameter(torch.from_numpy(W0.astype(np.float64)))
    opt = torch.optim.Adagrad([p], lr=0.05, eps=1e-8, initial_accumulator_value=0.0)
    for step in range(5):
        touched = np.sort(g.choice(V, size=3, replace=False))
        G = g.standard_normal((3, 1)).astype(np.float32)
        T.optimizer(rows[touched], G, 0.05, 1e-8)
        dense = torch.zeros(V, 1, dtype=torch.float64)
        dense[touched] = torch.from_numpy(G.astype(np.float64))
        p.grad = dense
        opt.step()
    _, W, S = T.read_rows(keys)
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(S[:, 0], opt.state[p]["sum"].numpy()[:, 0], rtol=1e-6)


def test_rowwise_adam_dim1_matches_torch_sparse_adam():
    V = 5
    g = np.random.default_rng(42)
    T = O.Table(1, opt=O.ADAM_RW, seed=4)
    keys = np.arange(V, dtype=np.int64) + 50
    _, rows, _ = T.find_or_insert(keys)
    _, W0, _ = T.read_rows(keys)
    p = torch.nn.Parameter(torch.from_numpy(W0.astype(np.float64)))
    opt = torch.optim.SparseAdam([p], lr=1e-2, betas=(0.9, 0.999), eps=1e-8)
    for step in range(6):
        touched = np.sort(g.choice(V, size=2, replace=False))
        G = g.standard_normal((2, 1)).astype(np.float32)
        T.optimizer(rows[touched], G, 1e-2, 1e-8, 0.9, 0.999)
        idx = torch.from_numpy(touched.astype(np.int64))[None, :]
        p.grad = torch.sparse_coo_tensor(idx, torch.from_numpy(G.astype(np.float64)), (V, 1))
        opt.step()
    _, W, _ = T.read_rows(keys)
    assert T.t == 6
    np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-5, atol=1e-9)


@pytest.mark.parametrize("rw,ew", [(O.ADAGRAD_RW, O.ADAGRAD), (O.ADAM_RW, O.ADAM)])
def test_rowwise_with_constant_row_gradients_equals_elementwise(rw, ew):
    """A gradient constant across each row has mean(g^2) = g_j^2 for every j,
    so the row-wise and the element-wise optimizers take the same steps (a
    dropped 1/dim or a per-element accumulator fails this at dim 8)."""
    D, V = 8, 6
    g = np.random.default_rng(43 + rw)
    keys = np.arange(V, dtype=np.int64) + 700
    A, B = O.Table(D, opt=rw, seed=5), O.Table(D, opt=ew, seed=5)
    _, rows, _ = A.find_or_insert(keys)
    B.find_or_insert(keys)
    for step in range(4):
        touched = np.sort(g.choice(V, size=4, replace=False))
        G = np.repeat(g.standard_normal((4, 1)), D, axis=1).astype(np.float32)
        A.optimizer(rows[touched], G, 0.02, 1e-8, 0.9, 0.999)
        B.optimizer(rows[touched], G, 0.02, 1e-8, 0.9, 0.999)
    _, WA, SA = A.read_rows(keys)
    _, WB, SB = B.read_rows(keys)
    np.testing.assert_allclose(WA, WB, rtol=1e-6, atol=1e-9)
    if rw == O.ADAGRAD_RW:
        np.testing.assert_allclose(SA[:, 0], SB[:, 0, 0], rtol=1e-6)
    else:
        np.testing.assert_allclose(SA[:, :D], SB[:, 0], rtol=1e-6)    # m per element
        np.testing.assert_allclose(SA[:, D], SB[:, 1, 0], rtol=1e-6)  # v per row


def test_rowwise_first_step_closed_form_and_layout():
    D = 4
    G = np.array([[3.0, -4.0, 0.0, 0.0]], dtype=np.float32)      # mean g^2 = 25 / 4
    T = O.Table(D, opt=O.ADAGRAD_RW, seed=6)
    _, rows, _ = T.find_or_insert(np.array([9], dtype=np.int64))
    _, w0, s0 = T.read_rows(np.array([9], dtype=np.int64))
    assert s0.shape == (1, 1) and s0[0, 0] == 0
    T.optimizer(rows, G, 0.1, 0.0)
    _, w1, s1 = T.read_rows(np.array([9], dtype=np.int64))
    assert s1[0, 0] == 6.25
    np.testing.assert_allclose(w1, w0.astype(np.float64) - 0.1 * G / 2.5, rtol=1.2e-7, atol=1e-12)  # fp32 storage
    # row-wise Adam keeps [m (dim) | v] and its first step is lr * g / sqrt(mean g^2)
    T = O.Table(D, opt=O.ADAM_RW, seed=6)
    _, rows, _ = T.find_or_insert(np.array([9], dtype=np.int64))
    _, w0, s0 = T.read_rows(np.array([9], dtype=np.int64))
    assert s0.shape == (1, D + 1)
    T.optimizer(rows, G, 0.1, 0.0, 0.9, 0.999)
    _, w1, s1 = T.read_rows(np.array([9], dtype=np.int64))
    np.testing.assert_allclose(s1[0, :D], 0.1 * G[0], rtol=1e-6)
    np.testing.assert_allclose(s1[0, D], 0.001 * 6.25, rtol=1e-6)
    np.testing.assert_allclose(w1, w0.astype(np.float64) - 0.1 * G / 2.5, rtol=1e-6, atol=1e-12)


# --------------------------------------------------------------------------- eviction


def test_eviction_removes_exactly_the_stale_keys():
    """Brute force: the test records, from its own inputs, the last call in
    which each key was looked up; evict(max_age) must keep exactly the keys
    with (calls so far - last call) <= max_age."""
    g = np.random.default_rng(51)
    T = O.Table(4, opt=O.ADAGRAD, seed=2)
    last = {}
    calls = 0
    for step in range(12):
        keys = g.integers(0, 60, size=int(g.integers(1, 25))).astype(np.int64)
        if step % 3 == 0:
            T.find_or_insert(keys)
        else:
            off = np.array([0, keys.size], dtype=np.int64)
            assert T.forward(keys, off, O.SUM)["status"] == O.OK
        calls += 1
        for k in keys.tolist():
            last[k] = calls
        if step in (5, 9, 11):
            max_age = int(g.integers(0, 4))
            n = T.evict(max_age)
            keep = {k for k, c in last.items() if calls - c <= max_age}
            assert n == len(last) - len(keep)
            last = {k: c for k, c in last.items() if k in keep}
            ek, er = T.export()
            assert set(ek.tolist()) == keep
            assert T.size() == len(keep)
            # rows of the live keys are distinct; live + free rows = rows allocated
            assert len(set(er.tolist())) == er.size
    assert T.clock == calls


def test_evicted_rows_are_reused_top_of_stack_first_and_reinitialised():
    D = 4
    T = O.Table(D, opt=O.ADAM, seed=9)
    st, rows, _ = T.find_or_insert(np.arange(10, dtype=np.int64))          # call 1: rows 0..9
    assert rows.tolist() == list(range(10))
    # update some rows so that stale values would show if a row leaked
    T.optimizer(rows, np.ones((10, D), np.float32), 0.1, 1e-8, 0.9, 0.999)
    keep = np.array([0, 1, 2, 4, 5, 6, 8], dtype=np.int64)
    T.find_or_insert(keep)                                                   # call 2
    assert T.evict(0) == 3                                                   # keys 3, 7, 9 age 1 > 0
    st, rows, nn = T.find_or_insert(np.array([100, 101, 102, 103, 3], dtype=np.int64))
    assert nn == 5
    # the free stack holds 3, 7, 9 (pushed in row order): 9 is taken first
    assert rows.tolist() == [9, 7, 3, 10, 11]
    assert T.rows_allocated() == 12
    _, w, s = T.read_rows(np.array([100, 101, 102, 103, 3], dtype=np.int64))
    for i, k in enumerate([100, 101, 102, 103, 3]):
        assert np.array_equal(w[i], O.init_row(9, k, D, -0.01, 0.01))       # fresh values, no leak
        assert np.all(s[i] == 0)


def test_eviction_max_age_zero_and_untouched_table():
    T = O.Table(2, seed=1)
    assert T.evict(5) == 0 and T.size() == 0
    T.find_or_insert(np.array([1, 2, 3], dtype=np.int64))
    T.find_or_insert(np.array([2], dtype=np.int64))
    assert T.evict(1) == 0                       # ages 1, 0, 1
    assert T.evict(0) == 2 and T.export()[0].tolist() == [2]
    st, rows, _ = T.find_or_insert(np.array([1], dtype=np.int64))
    assert rows.tolist() == [2]                  # rows 0 and 2 were freed (pushed 0, 2): 2 on top


# --------------------------------------------------------------------------- compaction


def test_compaction_moves_the_rows_above_the_live_count_into_the_holes_below():
    """Explicit case: rows 0..7, keys 10..17; evict the keys of rows 1, 3, 6.
    Live L = 5; holes below 5: rows 1, 3; rows holding keys at or above 5:
    5, 7.  Row 5 (key 15) moves to row 1, row 7 (key 17) to row 3."""
    D = 4
    T = O.Table(D, opt=O.ADAM, seed=3)
    keys = np.arange(10, 18, dtype=np.int64)
    _, rows, _ = T.find_or_insert(keys)                                    # call 1: rows 0..7
    assert rows.tolist() == list(range(8))
    T.optimizer(rows, np.arange(8 * D, dtype=np.float32).reshape(8, D) - 5, 0.1, 1e-8, 0.9, 0.999)
    T.find_or_insert(np.array([10, 12, 14, 15, 17], dtype=np.int64))      # call 2: 11, 13, 16 go stale
    assert T.evict(0) == 3
    _, w_before, s_before = T.read_rows(np.array([15, 17, 10, 12, 14], dtype=np.int64))
    assert T.compact() == 2
    ek, er = T.export()
    got = dict(zip(ek.tolist(), er.tolist()))
    assert got == {10: 0, 12: 2, 14: 4, 15: 1, 17: 3}
    assert T.rows_allocated() == 5
    _, w_after, s_after = T.read_rows(np.array([15, 17, 10, 12, 14], dtype=np.int64))
    assert np.array_equal(w_before, w_after) and np.array_equal(s_before, s_after)   # rows move whole
    # nothing is free any more: a new key takes row L
    _, rows, nn = T.find_or_insert(np.array([99], dtype=np.int64))
    assert rows.tolist() == [5] and nn == 1
    # a compact table stays put
    assert T.compact() == 0


@pytest.mark.parametrize("opt,dtype", [(O.ADAGRAD, O.F32), (O.ADAM, O.BF16), (O.ADAM_RW, O.F32)])
def test_compaction_brute_force(opt, dtype):
    """Random churn, then compaction: the key set and every key's row
    contents (values, state) are unchanged, the rows are exactly 0..L-1, the
    rows below L that held a key keep it, and the moved rows pair the holes
    and the rows at or above L in ascending order (checked against the
    pre-compaction key -> row map)."""
    g = np.random.default_rng(7)
    D = 8
    T = O.Table(D, row_dtype=dtype, opt=opt, seed=11)
    for step in range(10):
        keys = g.integers(0, 400, size=int(g.integers(20, 120))).astype(np.int64)
        _, rows, _ = T.find_or_insert(keys)
        T.optimizer(np.unique(rows), g.standard_normal((np.unique(rows).size, D)).astype(np.float32),
                    0.05, 1e-8, 0.9, 0.999)
        if step in (3, 6, 9):
            T.evict(int(g.integers(0, 2)))
    ek, er = T.export()
    before = dict(zip(ek.tolist(), er.tolist()))
    _, w0, s0 = T.read_rows(ek)
    L = len(before)
    holes = sorted(set(range(L)) - set(r for r in before.values() if r < L))
    movers = sorted(r for r in before.values() if r >= L)
    assert len(holes) == len(movers) and len(movers) > 0
    moved = T.compact()
    assert moved == len(movers)
    ek2, er2 = T.export()
    after = dict(zip(ek2.tolist(), er2.tolist()))
    assert set(after) == set(before) and sorted(after.values()) == list(range(L))
    dest = dict(zip(movers, holes))
    for k, r in before.items():
        assert after[k] == (dest[r] if r >= L else r)
    _, w1, s1 = T.read_rows(ek)
    assert np.array_equal(w0, w1) and np.array_equal(s0, s1)
    assert T.rows_allocated() == L
