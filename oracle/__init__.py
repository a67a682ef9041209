"""CPU oracle for the sparse embedding step — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It wraps ``oracle/oracle.cpp`` (a plain
sequential C++17 restatement of the method, fp64 sums) with ctypes and numpy;
it never imports the product package and the product never imports it.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# RS_ORACLE_LIB names another build of oracle.cpp (the sanitizer tier's)
LIB_PATH = os.environ.get("RS_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")

OK, EINVAL, ENOMEM, EFULL, EKEY = 0, 1, 2, 3, 4
SUM, MEAN, NONE, TAIL = 0, 1, 2, 3
F32, BF16 = 0, 1
ADAGRAD, ADAM, ADAMW, ADAM_TF, ADAGRAD_RW, ADAM_RW = 0, 1, 2, 3, 4, 5

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(LIB_PATH)
        p = C.c_void_p
        i64, i32, u64 = C.c_int64, C.c_int, C.c_uint64
        L.or_mix64.restype = u64
        L.or_mix64.argtypes = [u64]
        L.or_bf16_rne.restype = C.c_uint16
        L.or_bf16_rne.argtypes = [C.c_float]
        L.or_bf16_to_f32.restype = C.c_float
        L.or_bf16_to_f32.argtypes = [C.c_uint16]
        L.or_init_row.restype = None
        L.or_init_row.argtypes = [u64, i64, i32, C.c_float, C.c_float, p]
        L.or_create.restype = p
        L.or_create.argtypes = [i32, i32, i32, C.c_float, C.c_float, u64, i64]
        L.or_destroy.argtypes = [p]
        L.or_size.restype = i64
        L.or_size.argtypes = [p]
        L.or_step_count.restype = i64
        L.or_step_count.argtypes = [p]
        L.or_set_step_count.argtypes = [p, i64]
        L.or_dedup.restype = i64
        L.or_dedup.argtypes = [p, i64, p, p]
        L.or_ids_partition.restype = i64
        L.or_ids_partition.argtypes = [p, i64, i32, u64, p, p, p, p]
        L.or_bucketize.restype = i32
        L.or_bucketize.argtypes = [p, p, i32, p, p, p]
        L.or_mod.restype = i32
        L.or_mod.argtypes = [p, p, i32, p, p]
        L.or_evict.restype = i64
        L.or_evict.argtypes = [p, C.c_uint32]
        L.or_compact.restype = i64
        L.or_compact.argtypes = [p]
        L.or_rows_allocated.restype = i64
        L.or_rows_allocated.argtypes = [p]
        L.or_clock.restype = C.c_uint32
        L.or_clock.argtypes = [p]
        L.or_find_or_insert.restype = i32
        L.or_find_or_insert.argtypes = [p, p, i64, p, p]
        L.or_read_rows.restype = i64
        L.or_read_rows.argtypes = [p, p, i64, p, p]
        L.or_write_rows.restype = None
        L.or_write_rows.argtypes = [p, p, i64, p, p]
        L.or_export.restype = i64
        L.or_export.argtypes = [p, p, p, i64]
        L.or_forward.restype = i32
        L.or_forward.argtypes = [p, p, p, i64, i64, i32, i64, p, p, p, p, p, p, p]
        L.or_backward.restype = i32
        L.or_backward.argtypes = [p, i64, p, i64, i32, i32, i64, p, p]
        L.or_optimizer.restype = i32
        L.or_optimizer.argtypes = [p, p, i64, p, C.c_double, C.c_double, C.c_double, C.c_double, C.c_double]
        L.or_step.restype = i32
        L.or_step.argtypes = [p, p, p, i64, i64, i32, i64, p, C.c_double, C.c_double, C.c_double,
                              C.c_double, C.c_double, p, p, p, p]
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def mix64(x: int) -> int:
    return int(lib().or_mix64(x & 0xFFFFFFFFFFFFFFFF))


def bf16_rne(x: float) -> int:
    return int(lib().or_bf16_rne(float(x)))


def bf16_to_f32(h: int) -> float:
    return float(lib().or_bf16_to_f32(h))


def init_row(seed: int, key: int, dim: int, lo: float, hi: float) -> np.ndarray:
    out = np.empty(dim, dtype=np.float32)
    lib().or_init_row(seed & 0xFFFFFFFFFFFFFFFF, int(key), dim, lo, hi, _p(out))
    return out


def dedup(values: np.ndarray):
    """(status, unique int64[U], inverse int32[N]) in first-occurrence order."""
    v = _c(values, np.int64)
    n = v.size
    u = np.empty(max(n, 1), dtype=np.int64)
    inv = np.empty(max(n, 1), dtype=np.int32)
    U = lib().or_dedup(_p(v), n, _p(u), _p(inv))
    if U < 0:
        return -U, None, None
    return OK, u[:U].copy(), inv[:n].copy()


def ids_partition(values: np.ndarray, nshards: int, owner_seed: int = 0):
    """Dedup + split by owner shard: (keys int64[U], shard_offsets int64[G+1],
    inverse int32[N], n_rejected).  Shard s holds keys[offsets[s]:offsets[s+1]],
    in first-occurrence order; owner(k) = mix64(k ^ owner_seed) mod G."""
    v = _c(values, np.int64)
    n = v.size
    keys = np.empty(max(n, 1), dtype=np.int64)
    offs = np.empty(max(nshards, 0) + 1, dtype=np.int64)
    inv = np.empty(max(n, 1), dtype=np.int32)
    rej = np.zeros(1, dtype=np.int64)
    U = lib().or_ids_partition(_p(v), n, int(nshards), owner_seed & 0xFFFFFFFFFFFFFFFF, _p(keys), _p(offs),
                               _p(inv), _p(rej))
    if U < 0:
        raise ValueError("ids_partition: invalid arguments")
    return keys[:U].copy(), offs.copy(), inv[:n].copy(), int(rej[0])


def bucketize(values, col_offsets, boundaries, bnd_offsets) -> np.ndarray:
    """Bucket of every value of every column (int64), TF Bucketize semantics."""
    v = _c(values, np.float32)
    co = _c(col_offsets, np.int64)
    b = _c(boundaries, np.float32)
    bo = _c(bnd_offsets, np.int64)
    out = np.empty(max(v.size, 1), dtype=np.int64)
    if lib().or_bucketize(_p(v), _p(co), co.size - 1, _p(b if b.size else np.zeros(1, np.float32)), _p(bo),
                          _p(out)) != 0:
        raise ValueError("bucketize: invalid arguments")
    return out[:v.size].copy()


def mod(values, col_offsets, moduli) -> np.ndarray:
    """Floor modulus of every id by its column's modulus (int64)."""
    v = _c(values, np.int64)
    co = _c(col_offsets, np.int64)
    m = _c(moduli, np.int64)
    out = np.empty(max(v.size, 1), dtype=np.int64)
    if lib().or_mod(_p(v), _p(co), co.size - 1, _p(m if m.size else np.zeros(1, np.int64)), _p(out)) != 0:
        raise ValueError("mod: invalid arguments")
    return out[:v.size].copy()


def backward(offsets, inverse, U, dim, mode, pad_len, grad):
    off = _c(offsets, np.int64)
    inv = _c(inverse, np.int32)
    g = _c(grad, np.float32)
    gu = np.empty((max(U, 1), dim), dtype=np.float64)
    lib().or_backward(_p(off), off.size - 1, _p(inv), U, dim, mode, pad_len, _p(g), _p(gu))
    return gu[:U]


class Table:
    """The oracle's two-tier store: an unordered_map IDMap and dense row vectors."""

    def __init__(self, dim, row_dtype=F32, opt=ADAGRAD, lo=-0.01, hi=0.01, seed=0, max_live=-1):
        self.dim, self.row_dtype, self.opt = dim, row_dtype, opt
        self.h = lib().or_create(dim, row_dtype, opt, lo, hi, seed & 0xFFFFFFFFFFFFFFFF, max_live)
        if not self.h:
            raise ValueError("bad oracle table descriptor")

    def __del__(self):
        h = getattr(self, "h", None)
        if h and _lib is not None:
            _lib.or_destroy(h)
            self.h = None

    @property
    def nstate(self):
        """Per-element state vectors (row-wise optimizers: their vectors; the
        row scalar is extra)."""
        return {ADAGRAD: 1, ADAGRAD_RW: 0, ADAM_RW: 1}.get(self.opt, 2)

    @property
    def state_shape(self):
        """Shape of one row's state: (nstate, dim), or (state elements,) for
        the row-wise optimizers ([acc] or [m (dim) | v])."""
        if self.opt in (ADAGRAD_RW, ADAM_RW):
            return (self.nstate * self.dim + 1,)
        return (self.nstate, self.dim)

    def size(self) -> int:
        return int(lib().or_size(self.h))

    def evict(self, max_age: int) -> int:
        """Remove the keys not looked up in the last max_age calls (age > max_age)."""
        return int(lib().or_evict(self.h, max_age & 0xFFFFFFFF))

    def compact(self) -> int:
        """Move the live rows above the live count into the free rows below it
        (k-th above into k-th free below, both ascending); returns the rows moved."""
        return int(lib().or_compact(self.h))

    def rows_allocated(self) -> int:
        return int(lib().or_rows_allocated(self.h))

    @property
    def clock(self) -> int:
        return int(lib().or_clock(self.h))

    @property
    def t(self) -> int:
        return int(lib().or_step_count(self.h))

    @t.setter
    def t(self, v: int):
        lib().or_set_step_count(self.h, int(v))

    def find_or_insert(self, keys):
        k = _c(keys, np.int64)
        rows = np.empty(max(k.size, 1), dtype=np.int64)
        nn = np.zeros(1, dtype=np.int64)
        st = lib().or_find_or_insert(self.h, _p(k), k.size, _p(rows), _p(nn))
        return st, rows[:k.size].copy(), int(nn[0])

    def read_rows(self, keys):
        k = _c(keys, np.int64)
        w = np.full((k.size, self.dim), np.nan, dtype=np.float32)
        s = np.full((k.size, *self.state_shape), np.nan, dtype=np.float32)
        found = lib().or_read_rows(self.h, _p(k), k.size, _p(w), _p(s))
        return int(found), w, s

    def write_rows(self, keys, w, state=None):
        k = _c(keys, np.int64)
        w = _c(w, np.float32)
        s = None if state is None else _c(state, np.float32)
        lib().or_write_rows(self.h, _p(k), k.size, _p(w), _p(s))

    def export(self):
        n = int(lib().or_export(self.h, None, None, 0))
        keys = np.empty(max(n, 1), dtype=np.int64)
        rows = np.empty(max(n, 1), dtype=np.int64)
        lib().or_export(self.h, _p(keys), _p(rows), n)
        return keys[:n], rows[:n]

    def forward(self, values, offsets, mode, pad_len=0):
        v = _c(values, np.int64)
        off = _c(offsets, np.int64)
        n, bags = v.size, off.size - 1
        if mode in (NONE, TAIL):
            out = np.zeros((bags, pad_len, self.dim), dtype=np.float64)
            mask = np.zeros((bags, pad_len), dtype=np.uint8)
        else:
            out = np.zeros((bags, self.dim), dtype=np.float64)
            mask = None
        uniq = np.empty(max(n, 1), dtype=np.int64)
        inv = np.empty(max(n, 1), dtype=np.int32)
        rows = np.empty(max(n, 1), dtype=np.int64)
        U = np.zeros(1, dtype=np.int64)
        nn = np.zeros(1, dtype=np.int64)
        st = lib().or_forward(self.h, _p(v), _p(off), n, bags, mode, pad_len, _p(out), _p(mask),
                              _p(uniq), _p(inv), _p(rows), _p(U), _p(nn))
        u = int(U[0])
        return dict(status=st, out=out, mask=mask, unique=uniq[:u].copy(), inverse=inv[:n].copy(),
                    rows=rows[:u].copy(), U=u, n_new=int(nn[0]))

    def optimizer(self, rows, grad, lr, eps=1e-8, beta1=0.9, beta2=0.999, weight_decay=0.0):
        r = _c(rows, np.int64)
        g = _c(grad, np.float32)
        return lib().or_optimizer(self.h, _p(r), r.size, _p(g), lr, eps, beta1, beta2, weight_decay)

    def step(self, values, offsets, mode, grad, lr, eps=1e-8, beta1=0.9, beta2=0.999, pad_len=0,
             weight_decay=0.0):
        v = _c(values, np.int64)
        off = _c(offsets, np.int64)
        g = _c(grad, np.float32)
        n, bags = v.size, off.size - 1
        if mode in (NONE, TAIL):
            out = np.zeros((bags, pad_len, self.dim), dtype=np.float64)
            mask = np.zeros((bags, pad_len), dtype=np.uint8)
        else:
            out = np.zeros((bags, self.dim), dtype=np.float64)
            mask = None
        U = np.zeros(1, dtype=np.int64)
        nn = np.zeros(1, dtype=np.int64)
        st = lib().or_step(self.h, _p(v), _p(off), n, bags, mode, pad_len, _p(g), lr, eps, beta1, beta2, weight_decay,
                           _p(out), _p(mask), _p(U), _p(nn))
        return dict(status=st, out=out, mask=mask, U=int(U[0]), n_new=int(nn[0]))
