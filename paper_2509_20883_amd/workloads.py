"""Seeded synthetic workloads for the sparse embedding step.

This module only draws inputs: ragged ID features in CSR form, upstream
gradients, and the key lists used to pre-populate a table.  It holds none of
the embedding method's arithmetic (no dedup, hashing into the table, pooling
or optimizer math), so both the HIP path and the CPU oracle may read what it
produces.

The paper measures on internal models and data (the MSE and LMA models of the
end-to-end section) that are not available; these generators stand in for
them with the shapes it describes: many single-hot categorical features,
multi-hot bags, long user-behaviour sequences on one shared item table, and a
table that keeps growing during continuous training (Embedding Engine, system
design section).

Conventions
-----------
* Keys are int64.  Features that live in separate logical tables but are
  fused into one physical table carry their feature id in the high bits:
  ``key = (fid << 40) | id`` with ``0 <= id < 2**40``.  Features sharing one
  logical table use the raw id.
* A batch is feature-major: bag ``g = f * B + b``.
* Zipf(s) over a vocabulary of V ranks is truncated: ``P(r) ~ r**-s``,
  ``r = 1..V``.  Rank r maps to an id through a salted bijection on 40 bits,
  so hot ids are not small consecutive integers.
* Every random stream comes from ``numpy.random.SeedSequence([2509, k, ...])``.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Iterator, List, Optional

import numpy as np

MASTER_SEED = 2509
ID_BITS = 40
ID_MASK = (1 << ID_BITS) - 1

# ---------------------------------------------------------------------------
# seeded streams and the rank -> id bijection (generator-only hashing)
# ---------------------------------------------------------------------------


def rng(*path: int) -> np.random.Generator:
    """A PCG64 stream identified by an integer path under the master seed."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([MASTER_SEED, *path])))


def seed64(*path: int) -> int:
    """A 64-bit integer seed (e.g. a table's init seed) for an integer path."""
    s = np.random.SeedSequence([MASTER_SEED, 0x7AB1E, *path]).generate_state(2, np.uint32)
    return int(s[0]) | (int(s[1]) << 32)


_ODD_A = np.uint64(0x9FB21C651E98DF25 & ID_MASK | 1)
_ODD_B = np.uint64(0xC2B2AE3D27D4EB4F & ID_MASK | 1)
_M40 = np.uint64(ID_MASK)


def rank_to_id(rank: np.ndarray, salt: int) -> np.ndarray:
    """Salted bijection of [0, 2**40): xorshift / odd-multiply rounds mod 2**40."""
    x = (rank.astype(np.uint64) + np.uint64(salt & ID_MASK)) & _M40
    x ^= x >> np.uint64(20)
    x = (x * _ODD_A) & _M40
    x ^= x >> np.uint64(17)
    x = (x * _ODD_B) & _M40
    x ^= x >> np.uint64(23)
    return x.astype(np.int64)


def _fmix(x: np.ndarray, salt: int) -> np.ndarray:
    """Generator-side 64-bit avalanche (murmur3 finaliser) used for subset picks."""
    with np.errstate(over="ignore"):
        z = x.astype(np.uint64) ^ np.uint64(salt & 0xFFFFFFFFFFFFFFFF)
        z ^= z >> np.uint64(33)
        z *= np.uint64(0xFF51AFD7ED558CCD)
        z ^= z >> np.uint64(33)
        z *= np.uint64(0xC4CEB9FE1A85EC53)
        z ^= z >> np.uint64(33)
    return z


# ---------------------------------------------------------------------------
# truncated Zipf sampling
# ---------------------------------------------------------------------------

_CDF_CACHE: dict = {}


def _zipf_cdf(V: int, s: float) -> np.ndarray:
    key = (V, s)
    c = _CDF_CACHE.get(key)
    if c is None:
        w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
        c = np.cumsum(w)
        c /= c[-1]
        if len(_CDF_CACHE) > 64:
            _CDF_CACHE.clear()
        _CDF_CACHE[key] = c
    return c


def _zipf_rejection_inversion(n: int, V: int, s: float, g: np.random.Generator) -> np.ndarray:
    """Truncated Zipf by rejection-inversion (Hoermann & Derflinger, 1996)."""
    one_m_s = 1.0 - s

    def H(x):
        return (np.power(x, one_m_s) - 1.0) / one_m_s

    def Hinv(u):
        return np.power(1.0 + one_m_s * u, 1.0 / one_m_s)

    h_x1 = H(1.5) - 1.0
    h_n = H(V + 0.5)
    thr = 2.0 - Hinv(H(2.5) - 2.0 ** (-s))
    out = np.empty(n, dtype=np.int64)
    todo = np.arange(n)
    while todo.size:
        u = h_n + g.random(todo.size) * (h_x1 - h_n)
        x = Hinv(u)
        k = np.clip(np.floor(x + 0.5), 1, V)
        ok = (k - x <= thr) | (u >= H(k + 0.5) - np.power(k, -s))
        out[todo[ok]] = k[ok].astype(np.int64)
        todo = todo[~ok]
    return out


def zipf_ranks(n: int, V: int, s: float, g: np.random.Generator) -> np.ndarray:
    """n ranks in [1, V] drawn from truncated Zipf(s)."""
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    if V <= 10_000_000:
        c = _zipf_cdf(V, s)
        r = np.searchsorted(c, g.random(n), side="right") + 1
        return np.minimum(r, V).astype(np.int64)
    return _zipf_rejection_inversion(n, V, s, g)


# ---------------------------------------------------------------------------
# configurations
# ---------------------------------------------------------------------------

SUM, MEAN, NONE, TAIL = 0, 1, 2, 3


def padded(mode: int) -> bool:
    """The padded copies: head (first L ids) and tail (last L ids, the sequence tile)."""
    return mode in (NONE, TAIL)

F32, BF16 = 0, 1
ADAGRAD, ADAM, ADAMW, ADAM_TF, ADAGRAD_RW, ADAM_RW = 0, 1, 2, 3, 4, 5


@dataclasses.dataclass
class Workload:
    """One synthetic workload: table descriptor, batch shape and hyper-parameters."""

    name: str
    index: int
    dim: int
    row_dtype: int
    opt: int
    mode: int
    batch: int
    n_features: int
    vocab: List[int]
    zipf_s: float
    lengths: str  # "one", "uniform:a:b", "poisson:m:lo:hi", "poisson:m", "mixed"
    namespaced: bool
    capacity_slots: int
    max_load: float = 0.75
    block_rows: int = 1 << 20
    pad_len: int = 0
    init_lo: float = -0.01
    init_hi: float = 0.01
    lr: float = 0.01
    eps: float = 1e-8
    beta1: float = 0.9
    beta2: float = 0.999
    weight_decay: float = 0.0
    prepop: str = "none"  # "none", "frac90", "all", "pool"
    grad_dtype: int = F32
    steps: int = 1
    # growing-table workload: pool sizes and fresh keys per step
    pool0: int = 0
    fresh_per_step: int = 0
    n_single: int = 0
    seed: int = 0
    mini: bool = False

    @property
    def table_seed(self) -> int:
        return self.seed

    def salt(self, f: int) -> int:
        return int(_fmix(np.array([self.index * 1000 + f], dtype=np.uint64), 0x5A17)[0]) & ID_MASK

    def feature_key(self, f: int, ids: np.ndarray) -> np.ndarray:
        if self.namespaced:
            return (np.int64(f) << np.int64(ID_BITS)) | ids
        return ids


def _vocab_logu(k: int, n: int, lo: float, hi: float) -> List[int]:
    g = rng(k, 0xC0CAB)
    return [int(round(10 ** x)) for x in g.uniform(lo, hi, size=n)]


def workload(k: int, mini: bool = False) -> Workload:
    """The k-th synthetic workload; ``mini`` shrinks batch and vocabulary for parity tests."""
    if k == 0:
        w = Workload("single-feature-d16-adagrad", 0, dim=16, row_dtype=F32, opt=ADAGRAD, mode=SUM,
                     batch=1024, n_features=1, vocab=[100_000], zipf_s=1.1, lengths="uniform:1:8",
                     namespaced=False, capacity_slots=1 << 17, lr=0.01, eps=1e-8, block_rows=1 << 12)
    elif k == 1:
        w = Workload("26-single-hot-d64-adam", 1, dim=64, row_dtype=F32, opt=ADAM, mode=SUM,
                     batch=65536, n_features=26, vocab=_vocab_logu(1, 26, 2.0, 7.0), zipf_s=1.05,
                     lengths="one", namespaced=True, capacity_slots=1 << 26, lr=1e-3, eps=1e-8,
                     prepop="frac90")
    elif k == 2:
        w = Workload("100-multi-hot-d32-bf16-mean-adagrad", 2, dim=32, row_dtype=BF16, opt=ADAGRAD,
                     mode=MEAN, batch=8192, n_features=100, vocab=[1_000_000] * 100, zipf_s=1.1,
                     lengths="poisson:20:1:200", namespaced=True, capacity_slots=1 << 24,
                     lr=0.01, eps=1e-8)
    elif k == 3:
        w = Workload("3-seq-1e8-d128-bf16-padded-adam", 3, dim=128, row_dtype=BF16, opt=ADAM,
                     mode=NONE, batch=512, n_features=3, vocab=[100_000_000], zipf_s=1.2,
                     lengths="uniform:100:1024", namespaced=False, capacity_slots=1 << 28,
                     pad_len=1024, lr=1e-3, eps=1e-8, prepop="all", grad_dtype=BF16)
    elif k == 4:
        w = Workload("200-feat-growing-d64-adam", 4, dim=64, row_dtype=F32, opt=ADAM, mode=SUM,
                     batch=32768, n_features=200, vocab=[], zipf_s=1.2, lengths="mixed",
                     namespaced=True, capacity_slots=1 << 25, lr=1e-3, eps=1e-8, prepop="pool",
                     pool0=20_000_000, fresh_per_step=300_000, n_single=150, steps=100)
    elif k == 5:
        # the sequence tile of the Reduction Operations benchmark (one million
        # ids of dim 16): 8000 behaviour sequences of U{16..234} ids (mean
        # 125), each tiled as the concatenation of its most recent 128 rows
        w = Workload("seq-tile-1M-d16-tail128-adagrad", 5, dim=16, row_dtype=F32, opt=ADAGRAD, mode=TAIL,
                     batch=8000, n_features=1, vocab=[1_000_000], zipf_s=1.2, lengths="uniform:16:234",
                     namespaced=False, capacity_slots=1 << 21, pad_len=128, lr=0.01, eps=1e-8)
    else:
        raise ValueError(f"no workload {k}")
    w.seed = seed64(k)
    if mini:
        w.mini = True
        w.batch = max(8, w.batch // 32)
        if w.vocab:
            w.vocab = [max(10, v // 100) for v in w.vocab]
        if k == 3:
            w.vocab = [1_000_000]
            w.pad_len = 256
            w.lengths = "uniform:20:300"
            w.capacity_slots = 1 << 21
        if k == 4:
            w.pool0 = 200_000
            w.fresh_per_step = 3_000
            w.capacity_slots = 1 << 18
            w.steps = 3
        if k in (1, 2):
            w.capacity_slots = 1 << 20
        if k == 5:
            w.pad_len = 48
            w.capacity_slots = 1 << 16
        w.block_rows = 1 << 14
    return w


def _bag_lengths(w: Workload, f: int, g: np.random.Generator) -> np.ndarray:
    B = w.batch
    spec = w.lengths
    if spec == "mixed":
        spec = "one" if f < w.n_single else "poisson:10"
    parts = spec.split(":")
    if parts[0] == "one":
        return np.ones(B, dtype=np.int64)
    if parts[0] == "uniform":
        lo, hi = int(parts[1]), int(parts[2])
        return g.integers(lo, hi + 1, size=B).astype(np.int64)
    if parts[0] == "poisson":
        m = float(parts[1])
        x = g.poisson(m, size=B).astype(np.int64)
        if len(parts) == 4:
            x = np.clip(x, int(parts[2]), int(parts[3]))
        return x
    raise ValueError(spec)


# ---------------------------------------------------------------------------
# growing-table pools
# ---------------------------------------------------------------------------


def pool_shares(w: Workload) -> np.ndarray:
    """Per-feature share of occurrences (expected), used to size each feature's live pool."""
    per = np.array([1.0 if f < w.n_single else 10.0 for f in range(w.n_features)])
    return per / per.sum()


def pool_sizes(w: Workload, step: int) -> np.ndarray:
    """Live pool size of each feature before ``step`` (0-based) of the growing workload."""
    sh = pool_shares(w)
    p0 = np.floor(w.pool0 * sh).astype(np.int64)
    fr = np.floor(w.fresh_per_step * sh).astype(np.int64)
    return p0 + fr * step


def fresh_counts(w: Workload) -> np.ndarray:
    return np.floor(w.fresh_per_step * pool_shares(w)).astype(np.int64)


# ---------------------------------------------------------------------------
# batches
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class Batch:
    values: np.ndarray   # int64[N]
    offsets: np.ndarray  # int64[G+1]
    n_features: int
    batch: int

    @property
    def n(self) -> int:
        return int(self.values.shape[0])

    @property
    def bags(self) -> int:
        return int(self.offsets.shape[0] - 1)


def make_batch(w: Workload, step: int = 0, batch: Optional[int] = None,
               features: Optional[List[int]] = None) -> Batch:
    """The ID batch of ``step``; ``batch``/``features`` select a bounded sample of it."""
    B = w.batch if batch is None else batch
    feats = list(range(w.n_features)) if features is None else list(features)
    vals, lens = [], []
    for f in feats:
        g = rng(w.index, 1 + int(w.mini), step, f)
        L = _bag_lengths(w, f, g)[:B]
        n = int(L.sum())
        if w.lengths == "mixed":
            P = int(pool_sizes(w, step)[f])
            nf = int(fresh_counts(w)[f])
            ranks = zipf_ranks(n, P, w.zipf_s, g)
            if nf > 0 and n > 0:
                nf = min(nf, n)
                pos = g.choice(n, size=nf, replace=False)
                ranks[pos] = P + 1 + np.arange(nf, dtype=np.int64)
            ids = rank_to_id(ranks, w.salt(f))
        else:
            V = w.vocab[min(f, len(w.vocab) - 1)]
            ranks = zipf_ranks(n, V, w.zipf_s, g)
            shared = not w.namespaced and w.n_features > 1
            ids = rank_to_id(ranks, w.salt(0 if shared else f))
        vals.append(w.feature_key(f, ids))
        lens.append(L)
    values = np.concatenate(vals) if vals else np.zeros(0, dtype=np.int64)
    lens = np.concatenate(lens) if lens else np.zeros(0, dtype=np.int64)
    offsets = np.zeros(lens.size + 1, dtype=np.int64)
    np.cumsum(lens, out=offsets[1:])
    return Batch(values=values.astype(np.int64), offsets=offsets, n_features=len(feats), batch=B)


def make_grad(w: Workload, b: Batch, step: int = 0, nan_in_masked: bool = False) -> np.ndarray:
    """Upstream gradient N(0,1): fp32 ``[G, D]`` for pooled modes; for the padded
    sequence mode ``[G, L, D]`` as fp32 values already rounded to bf16 when the
    gradient dtype is bf16 (returned as float32 holding bf16-representable values)."""
    g = rng(w.index, 100 + int(w.mini), step)
    if padded(w.mode):
        L = w.pad_len
        x = g.standard_normal((b.bags, L, w.dim), dtype=np.float32)
        if w.grad_dtype == BF16:
            x = bf16_representable(x)
        if nan_in_masked:
            lens = np.diff(b.offsets)
            t = np.arange(L)[None, :]
            masked = t >= lens[:, None]
            x[masked] = np.nan
        return x
    return g.standard_normal((b.bags, w.dim), dtype=np.float32)


def bf16_representable(x: np.ndarray) -> np.ndarray:
    """Truncate fp32 values to bf16-representable ones (drops the low 16 bits).

    Input data only: this picks gradient values that a bf16 tensor can hold
    exactly, so both paths read identical numbers."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) & np.uint32(0xFFFF0000)
    return u.view(np.float32)


# ---------------------------------------------------------------------------
# pre-population key lists (enumeration order: feature-major, rank order)
# ---------------------------------------------------------------------------


def prepop_member(w: Workload, f: int, ids: np.ndarray) -> np.ndarray:
    """Deterministic ~90% subset used by the "frac90" pre-population."""
    return (_fmix(ids, 0x9090 + 7919 * f) % np.uint64(10)) != 0


def prepop_keys(w: Workload, chunk: int = 1 << 22) -> Iterator[np.ndarray]:
    """Keys present in the table before the first step, in enumeration order."""
    if w.prepop == "none":
        return
    if w.prepop == "pool":
        sizes = pool_sizes(w, 0)
        for f in range(w.n_features):
            for r0 in range(1, int(sizes[f]) + 1, chunk):
                r = np.arange(r0, min(int(sizes[f]) + 1, r0 + chunk), dtype=np.int64)
                yield w.feature_key(f, rank_to_id(r, w.salt(f)))
        return
    feats = range(w.n_features) if w.namespaced else [0]
    for f in feats:
        V = w.vocab[min(f, len(w.vocab) - 1)]
        for r0 in range(1, V + 1, chunk):
            r = np.arange(r0, min(V + 1, r0 + chunk), dtype=np.int64)
            ids = rank_to_id(r, w.salt(f))
            if w.prepop == "frac90":
                ids = ids[prepop_member(w, f, ids)]
            yield w.feature_key(f, ids)


def prepop_count(w: Workload) -> int:
    return int(sum(k.size for k in prepop_keys(w)))


def describe(w: Workload) -> dict:
    return {"workload": w.name, "batch": w.batch, "features": w.n_features, "dim": w.dim,
            "row_dtype": "bf16" if w.row_dtype == BF16 else "f32",
            "optimizer": ["adagrad", "adam", "adamw", "adam-eps-hat", "adagrad-rowwise", "adam-rowwise"][w.opt],
            "pooling": ["sum", "mean", "none", "tile-tail"][w.mode], "pad_len": w.pad_len, "zipf_s": w.zipf_s,
            "vocab_total": int(sum(w.vocab)) if w.vocab else int(w.pool0), "mini": w.mini}


# ---------------------------------------------------------------------------
# ids partition input
# ---------------------------------------------------------------------------

# The paper benchmarks its fused ids partition on one million ids.  The
# stand-in: the 26 single-hot features of workload 1 (Zipf 1.05 over
# log-uniform vocabularies, feature id in the high bits) at 38462 bags, i.e.
# 1,000,012 ids of one merged same-dim request, split over the 8 GPUs of one
# node.
IDS_PARTITION_BATCH = 38462
IDS_PARTITION_SHARDS = 8
IDS_PARTITION_SEED = 0x0DDBA11CAFEF00D5


def ids_partition_values(step: int = 0, batch: int = IDS_PARTITION_BATCH) -> np.ndarray:
    """The ids of one ids-partition call (int64, feature-major)."""
    return make_batch(workload(1), step, batch=batch).values


# ---------------------------------------------------------------------------
# feature-transform columns (bucketize, mod)
# ---------------------------------------------------------------------------

# The paper benchmarks its fused bucketize and mod on 100 columns of 10,000
# values each.  Stand-ins: log-normal float features (prices) with 63
# boundaries per column at the column distribution's quantiles (rounded to
# cents, so some values hit a boundary exactly); int64 ids (Zipf ranks through
# the 40-bit bijection, some negative) with a modulus per column drawn
# log-uniformly in [1e2, 1e7].
FEATURE_COLUMNS = 100
FEATURE_VALUES = 10_000
FEATURE_BOUNDS = 63


def _col_offsets(sizes: np.ndarray) -> np.ndarray:
    off = np.zeros(len(sizes) + 1, dtype=np.int64)
    np.cumsum(sizes, out=off[1:])
    return off


def bucketize_columns(ncols: int = FEATURE_COLUMNS, nvals=FEATURE_VALUES, nbounds=FEATURE_BOUNDS, step: int = 0):
    """(values fp32 [n], col_offsets int64 [ncols+1], boundaries fp32, bnd_offsets int64 [ncols+1]).
    ``nvals`` / ``nbounds`` may be ints or per-column arrays."""
    g = rng(40, step)
    sizes = np.broadcast_to(np.asarray(nvals, dtype=np.int64), (ncols,)).copy()
    nb = np.broadcast_to(np.asarray(nbounds, dtype=np.int64), (ncols,)).copy()
    vals, bnds = [], []
    for c in range(ncols):
        mu, sigma = g.uniform(0.0, 6.0), g.uniform(0.3, 1.5)
        x = np.round(g.lognormal(mu, sigma, size=int(sizes[c])), 2).astype(np.float32)
        q = np.quantile(g.lognormal(mu, sigma, size=4096), np.linspace(0, 1, int(nb[c]) + 2)[1:-1]) if nb[c] else []
        vals.append(x)
        bnds.append(np.sort(np.round(np.asarray(q, dtype=np.float64), 2)).astype(np.float32))
    return (np.concatenate(vals) if vals else np.zeros(0, np.float32), _col_offsets(sizes),
            np.concatenate(bnds) if bnds else np.zeros(0, np.float32), _col_offsets(nb))


def mod_columns(ncols: int = FEATURE_COLUMNS, nvals=FEATURE_VALUES, step: int = 0):
    """(values int64 [n], col_offsets int64 [ncols+1], moduli int64 [ncols])."""
    g = rng(41, step)
    sizes = np.broadcast_to(np.asarray(nvals, dtype=np.int64), (ncols,)).copy()
    vals = []
    for c in range(ncols):
        ids = rank_to_id(zipf_ranks(int(sizes[c]), 10**6, 1.1, g), 7919 * c + 11)
        sign = np.where(g.random(int(sizes[c])) < 0.1, -1, 1)
        vals.append(ids * sign)
    moduli = np.round(10.0 ** g.uniform(2.0, 7.0, size=ncols)).astype(np.int64)
    return (np.concatenate(vals).astype(np.int64) if vals else np.zeros(0, np.int64), _col_offsets(sizes), moduli)
