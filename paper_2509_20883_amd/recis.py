"""Python binding of librecis_mi355x.so (ctypes; argument marshalling only).

Every step of the embedding path runs in the library's HIP kernels; PyTorch is
used here only for device memory and the current HIP stream.  There is no
fallback: if the library is not built, or no GPU is present, calls raise.

Names follow the C ABI (include/recis_mi355x.h): ht_create, ht_find_or_insert,
lookup_pool_fwd, lookup_pool_bwd, sparse_opt_step, lookup_pool_bwd_opt,
ids_partition, fused_bucketize, fused_mod.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Tuple

import torch

PKG = os.path.dirname(os.path.abspath(__file__))
# RS_LIB names another build of the library (e.g. a variant being measured)
LIB_PATH = os.environ.get("RS_LIB") or os.path.join(PKG, "librecis_mi355x.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "recis_mi355x.h")

OK, EINVAL, ENOMEM, EFULL, EKEY, EHIP = 0, 1, 2, 3, 4, 5
STATUS_NAMES = {0: "RS_OK", 1: "RS_EINVAL", 2: "RS_ENOMEM", 3: "RS_EFULL", 4: "RS_EKEY", 5: "RS_EHIP"}
SUM, MEAN, NONE, TAIL = 0, 1, 2, 3
F32, BF16 = 0, 1
ADAGRAD, ADAM, ADAMW, ADAM_TF, ADAGRAD_RW, ADAM_RW = 0, 1, 2, 3, 4, 5
# kernel ids of rs_set_kernel_events ("occ" and "init_rows" bracket the same
# launch; "bwd_long" brackets the hot-key unit sums and their finish)
KERNELS = {"tile_dedup": 0, "partition": 1, "compact_insert": 2, "init_rows": 3, "pool": 4,
           "bwd_short": 5, "bwd_long": 6, "opt": 7, "occ": 8, "occ_list": 9}


class RecisError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class TableDesc(C.Structure):
    _fields_ = [("dim", C.c_int32), ("row_dtype", C.c_int32), ("optimizer", C.c_int32),
                ("init_lo", C.c_float), ("init_hi", C.c_float), ("seed", C.c_uint64),
                ("capacity_slots", C.c_int64), ("max_load", C.c_float), ("block_rows", C.c_int64),
                ("auto_grow", C.c_int32), ("evictable", C.c_int32)]


ALLOC_FN = C.CFUNCTYPE(C.c_void_p, C.c_size_t, C.c_void_p)
FREE_FN = C.CFUNCTYPE(None, C.c_void_p, C.c_void_p)


class Allocator(C.Structure):
    _fields_ = [("alloc", ALLOC_FN), ("free", FREE_FN), ("ctx", C.c_void_p)]


class TorchAllocator:
    """rs_allocator backed by PyTorch's caching allocator (current stream).

    fail_after: return NULL from the (fail_after + 1)-th allocation on (tests
    of the RS_ENOMEM path)."""

    def __init__(self, device=None, fail_after: Optional[int] = None):
        self.device = torch.cuda.current_device() if device is None else device
        self.fail_after = fail_after
        self.calls = 0
        self.live = {}
        self._a = ALLOC_FN(self._alloc)
        self._f = FREE_FN(self._free)
        self.struct = Allocator(self._a, self._f, None)

    def _alloc(self, nbytes, ctx):
        self.calls += 1
        if self.fail_after is not None and self.calls > self.fail_after:
            return None
        try:
            p = torch.cuda.caching_allocator_alloc(int(nbytes), self.device)
        except Exception:  # an exception must not cross the C callback
            return None
        self.live[p] = int(nbytes)
        return p

    def _free(self, ptr, ctx):
        if ptr in self.live:
            del self.live[ptr]
            torch.cuda.caching_allocator_delete(ptr)


class OptParams(C.Structure):
    _fields_ = [("lr", C.c_double), ("eps", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double),
                ("weight_decay", C.c_double)]


class RsCtx(C.Structure):
    _fields_ = [("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t),
                ("unique", C.c_void_p), ("inverse", C.c_void_p), ("rows", C.c_void_p),
                ("scalars", C.c_void_p), ("offsets", C.c_void_p), ("table", C.c_void_p),
                ("n", C.c_int64), ("bags", C.c_int64), ("pad_len", C.c_int64),
                ("mode", C.c_int32), ("dim", C.c_int32), ("priv", C.c_int64 * 16)]


_lib = None


def lib() -> C.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RecisError(EHIP, f"{LIB_PATH} is not built; run paper_2509_20883_amd/build.py")
    L = C.CDLL(LIB_PATH)
    p, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
    sig = {
        "rs_version": (C.c_int, []),
        "rs_last_error": (C.c_char_p, []),
        "ht_create": (C.c_int, [C.POINTER(TableDesc), C.POINTER(Allocator), p, C.POINTER(p)]),
        "ht_destroy": (C.c_int, [p]),
        "ht_find_or_insert": (C.c_int, [p, p, i64, p, p, p]),
        "ht_find": (C.c_int, [p, p, i64, p, p]),
        "ht_size": (C.c_int, [p, C.POINTER(i64), p]),
        "rs_table_check": (C.c_int, [p, p]),
        "ht_capacity": (C.c_int, [p, C.POINTER(i64)]),
        "ht_export": (C.c_int, [p, p, p, i64, p, p]),
        "ht_read_rows": (C.c_int, [p, p, i64, p, p, p]),
        "ht_reserve": (C.c_int, [p, i64, p]),
        "lookup_workspace_bytes": (C.c_size_t, [i64, i64, i64, p]),
        "lookup_pool_fwd": (C.c_int, [p, p, p, i64, i64, i32, i64, p, p, C.POINTER(RsCtx), i32, p]),
        "lookup_prepare": (C.c_int, [p, p, p, i64, i64, i32, i64, C.POINTER(RsCtx), i32, p]),
        "lookup_pool_prepared": (C.c_int, [p, C.POINTER(RsCtx), p, p, p]),
        "lookup_pool_bwd": (C.c_int, [p, C.POINTER(RsCtx), p, p, p]),
        "sparse_opt_step": (C.c_int, [p, C.POINTER(RsCtx), p, C.POINTER(OptParams), p]),
        "lookup_pool_bwd_opt": (C.c_int, [p, C.POINTER(RsCtx), p, C.POINTER(OptParams), p]),
        "rs_set_kernel_events": (C.c_int, [p, i32, p, p]),
        "ht_evict": (C.c_int, [p, C.c_uint32, C.POINTER(i64), p]),
        "ht_compact": (C.c_int, [p, C.POINTER(i64), C.POINTER(i64), p]),
        "ids_partition_workspace_bytes": (C.c_size_t, [i64, i32]),
        "ids_partition": (C.c_int, [p, i64, i32, C.c_uint64, p, p, p, p, p, C.c_size_t, p]),
        "fused_bucketize": (C.c_int, [p, i64, p, i32, p, p, p, i32, p]),
        "fused_mod": (C.c_int, [p, i64, p, i32, p, p, i32, p]),
        "rs_bandwidth_probe": (C.c_int, [i32, p, i64, p, i64, p, i64, i32, p]),
        "ids_partition_static": (C.c_int, [p, i64, i32, C.c_uint64, p, p, p, p, p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def _check(st: int):
    if st != OK:
        raise RecisError(st, lib().rs_last_error().decode())


def _stream() -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype: torch.dtype) -> torch.Tensor:
    if not t.is_cuda:
        raise RecisError(EINVAL, "tensors must be on the GPU")
    if t.dtype != dtype:
        raise RecisError(EINVAL, f"expected {dtype}, got {t.dtype}")
    return t.contiguous()


class Ctx:
    """Forward context: the caller-owned workspace plus the rs_ctx struct."""

    def __init__(self):
        self.ws: Optional[torch.Tensor] = None
        self.c = RsCtx()
        self.keep = ()

    def ensure(self, nbytes: int, device):
        if self.ws is None or self.ws.numel() < nbytes:
            self.ws = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        self.c.workspace = self.ws.data_ptr()
        self.c.workspace_bytes = self.ws.numel()

    def _view(self, ptr: int, count: int, dtype: torch.dtype) -> torch.Tensor:
        off = ptr - self.ws.data_ptr()
        es = torch.empty(0, dtype=dtype).element_size()
        return self.ws[off:off + count * es].view(dtype)

    def scalars(self) -> torch.Tensor:
        """Device int64[4]: U, inserted, occurrences kept, live rows before."""
        return self._view(self.c.scalars, 4, torch.int64)

    def unique(self, U: int) -> torch.Tensor:
        return self._view(self.c.unique, U, torch.int64)

    def inverse(self) -> torch.Tensor:
        return self._view(self.c.inverse, self.c.n, torch.int32)

    def rows(self, U: int) -> torch.Tensor:
        return self._view(self.c.rows, U, torch.int64)


def ids_partition_workspace_bytes(n: int, nshards: int) -> int:
    return int(lib().ids_partition_workspace_bytes(n, nshards))


class IdsPartition:
    """Ids partition (dedup + split by owner shard) with a reusable workspace.

    ``__call__(values, nshards, owner_seed)`` enqueues the call on the current
    stream and returns device tensors (keys int64 [n], shard_offsets int64
    [nshards+1], inverse int32 [n], info int64 [2] = {U, error bits}); the
    first U keys are valid, shard s holds keys[offsets[s]:offsets[s+1]].
    """

    def __init__(self):
        self.ws: Optional[torch.Tensor] = None

    def __call__(self, values: torch.Tensor, nshards: int, owner_seed: int = 0, keys=None, shard_offsets=None,
                 inverse=None, info=None):
        v = _dev(values, torch.int64)
        n = v.numel()
        need = ids_partition_workspace_bytes(n, nshards)
        if need == 0:
            raise RecisError(EINVAL, "n must be in [0, 2^28] and nshards in [1, 1024]")
        if self.ws is None or self.ws.numel() < need:
            self.ws = torch.empty(need, dtype=torch.uint8, device=v.device)
        if keys is None:
            keys = torch.empty(max(n, 1), dtype=torch.int64, device=v.device)
        if shard_offsets is None:
            shard_offsets = torch.empty(nshards + 1, dtype=torch.int64, device=v.device)
        if inverse is None:
            inverse = torch.empty(max(n, 1), dtype=torch.int32, device=v.device)
        if info is None:
            info = torch.empty(2, dtype=torch.int64, device=v.device)
        _check(lib().ids_partition(_ptr(v), n, nshards, owner_seed & 0xFFFFFFFFFFFFFFFF, _ptr(keys),
                                   _ptr(shard_offsets), _ptr(inverse), _ptr(info), _ptr(self.ws), self.ws.numel(),
                                   _stream()))
        return keys[:max(n, 0)], shard_offsets, inverse[:n], info


IDS_STATIC_MAX_IDS = 1 << 20


def ids_partition_static(values: torch.Tensor, nshards: int, owner_seed: int, keys: torch.Tensor,
                         shard_offsets: torch.Tensor, inverse: torch.Tensor, info: torch.Tensor) -> None:
    """ids_partition with the library's own fixed workspace: allocates nothing.

    Every tensor is the caller's (contiguous, on the GPU): keys int64 [>= n],
    shard_offsets int64 [nshards + 1], inverse int32 [>= n], info int64 [2];
    n = values.numel() <= IDS_STATIC_MAX_IDS.  Calls on one GPU share the
    workspace: overlapping calls race.
    """
    for t, dt in ((values, torch.int64), (keys, torch.int64), (shard_offsets, torch.int64), (inverse, torch.int32),
                  (info, torch.int64)):
        if not t.is_cuda or t.dtype != dt or not t.is_contiguous():
            raise RecisError(EINVAL, f"expected a contiguous GPU {dt} tensor")
    n = values.numel()
    if keys.numel() < n or inverse.numel() < n or shard_offsets.numel() < nshards + 1 or info.numel() < 2:
        raise RecisError(EINVAL, "output tensors too small")
    _check(lib().ids_partition_static(_ptr(values), n, nshards, owner_seed & 0xFFFFFFFFFFFFFFFF, _ptr(keys),
                                      _ptr(shard_offsets), _ptr(inverse), _ptr(info), _stream()))


def ids_partition(values: torch.Tensor, nshards: int, owner_seed: int = 0):
    """One-off ids partition (allocates its workspace); see IdsPartition."""
    return IdsPartition()(values, nshards, owner_seed)


def fused_bucketize(values: torch.Tensor, col_offsets: torch.Tensor, boundaries: torch.Tensor,
                    bnd_offsets: torch.Tensor, out: Optional[torch.Tensor] = None,
                    validate: bool = False) -> torch.Tensor:
    """Bucket (int64) of every fp32 value of every column; one launch."""
    v = _dev(values, torch.float32)
    co = _dev(col_offsets, torch.int64)
    b = _dev(boundaries, torch.float32)
    bo = _dev(bnd_offsets, torch.int64)
    if out is None:
        out = torch.empty(v.numel(), dtype=torch.int64, device=v.device)
    _check(lib().fused_bucketize(_ptr(v), v.numel(), _ptr(co), co.numel() - 1, _ptr(b), _ptr(bo), _ptr(out),
                                 int(validate), _stream()))
    return out


def fused_mod(values: torch.Tensor, col_offsets: torch.Tensor, moduli: torch.Tensor,
              out: Optional[torch.Tensor] = None, validate: bool = False) -> torch.Tensor:
    """Floor modulus (int64) of every id by its column's modulus; one launch."""
    v = _dev(values, torch.int64)
    co = _dev(col_offsets, torch.int64)
    m = _dev(moduli, torch.int64)
    if out is None:
        out = torch.empty(v.numel(), dtype=torch.int64, device=v.device)
    _check(lib().fused_mod(_ptr(v), v.numel(), _ptr(co), co.numel() - 1, _ptr(m), _ptr(out), int(validate),
                           _stream()))
    return out


PROBES = {"read": 0, "write": 1, "copy": 2, "gather": 3, "rmw": 4}


def bandwidth_probe(kind: str, a: torch.Tensor, b: Optional[torch.Tensor] = None, idx: Optional[torch.Tensor] = None,
                    n: Optional[int] = None, row_bytes: int = 0):
    """Enqueue one bandwidth probe (measurement reference) on the current stream.

    read / write / copy: n bytes (default: all of a); gather / rmw: the rows
    of row_bytes of a named by idx (int64), gathered into b or updated in place.
    """
    if not a.is_cuda or (b is not None and not b.is_cuda) or (idx is not None and not idx.is_cuda):
        raise RecisError(EINVAL, "probe buffers must be on the GPU")
    ab = a.numel() * a.element_size()
    bb = 0 if b is None else b.numel() * b.element_size()
    if idx is not None:
        idx = _dev(idx, torch.int64)
    if n is None:
        n = idx.numel() if kind in ("gather", "rmw") else ab
    _check(lib().rs_bandwidth_probe(PROBES[kind], _ptr(a), ab, _ptr(b), bb, _ptr(idx), n, row_bytes, _stream()))


class Table:
    """A dynamic embedding table (IDMap + Blocks) on the current GPU."""

    def __init__(self, dim: int, row_dtype: int = F32, optimizer: int = ADAGRAD, init_lo: float = -0.01,
                 init_hi: float = 0.01, seed: int = 0, capacity_slots: int = 1 << 17, max_load: float = 0.75,
                 block_rows: int = 1 << 16, auto_grow: bool = True, evictable: bool = False,
                 allocator: Optional[TorchAllocator] = None):
        d = TableDesc(dim, row_dtype, optimizer, init_lo, init_hi, seed & 0xFFFFFFFFFFFFFFFF, capacity_slots,
                      max_load, block_rows, int(bool(auto_grow)), int(bool(evictable)))
        h = C.c_void_p()
        self.allocator = allocator  # kept alive for the table's lifetime (its callbacks free the memory)
        _check(lib().ht_create(C.byref(d), C.byref(allocator.struct) if allocator else None, _stream(), C.byref(h)))
        self.h = h
        self.dim, self.row_dtype, self.optimizer = dim, row_dtype, optimizer
        # per-element state vectors; the row-wise optimizers add one scalar per row
        self.nstate = {ADAGRAD: 1, ADAGRAD_RW: 0, ADAM_RW: 1}.get(optimizer, 2)
        self.state_shape = ((self.nstate * dim + 1,) if optimizer in (ADAGRAD_RW, ADAM_RW)
                            else (self.nstate, dim))
        self.device = torch.device("cuda", torch.cuda.current_device())

    def close(self):
        if getattr(self, "h", None) and self.h.value:
            st = lib().ht_destroy(self.h)
            self.h = C.c_void_p()
            _check(st)

    def __del__(self):
        try:
            if getattr(self, "h", None) and self.h.value and _lib is not None:
                _lib.ht_destroy(self.h)
                self.h = C.c_void_p()
        except Exception:
            pass

    # ---------------------------------------------------------------- IDMap
    def find_or_insert(self, keys: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
        k = _dev(keys, torch.int64)
        rows = torch.empty_like(k)
        nins = torch.zeros(1, dtype=torch.int64, device=k.device)
        _check(lib().ht_find_or_insert(self.h, _ptr(k), k.numel(), _ptr(rows), _ptr(nins), _stream()))
        return rows, nins

    def find(self, keys: torch.Tensor) -> torch.Tensor:
        k = _dev(keys, torch.int64)
        rows = torch.empty_like(k)
        _check(lib().ht_find(self.h, _ptr(k), k.numel(), _ptr(rows), _stream()))
        return rows

    def size(self) -> int:
        v = C.c_int64()
        _check(lib().ht_size(self.h, C.byref(v), _stream()))
        return v.value

    def evict(self, max_age: int) -> int:
        """Drop the keys not looked up in the last max_age lookup calls; returns the count."""
        v = C.c_int64()
        _check(lib().ht_evict(self.h, max_age & 0xFFFFFFFF, C.byref(v), _stream()))
        return v.value

    def compact(self) -> Tuple[int, int]:
        """Move the live rows above the live count into the free rows below it;
        returns (rows moved, bytes of Blocks memory released).  Synchronizes."""
        m, b = C.c_int64(), C.c_int64()
        _check(lib().ht_compact(self.h, C.byref(m), C.byref(b), _stream()))
        return m.value, b.value

    def check(self):
        _check(lib().rs_table_check(self.h, _stream()))

    def capacity(self) -> int:
        v = C.c_int64()
        _check(lib().ht_capacity(self.h, C.byref(v)))
        return v.value

    def reserve(self, live_upper_bound: int):
        _check(lib().ht_reserve(self.h, live_upper_bound, _stream()))

    def export(self) -> Tuple[torch.Tensor, torch.Tensor]:
        live = self.size()
        keys = torch.empty(max(live, 1), dtype=torch.int64, device=self.device)
        rows = torch.empty(max(live, 1), dtype=torch.int64, device=self.device)
        nd = torch.zeros(1, dtype=torch.int64, device=self.device)
        _check(lib().ht_export(self.h, _ptr(keys), _ptr(rows), live, _ptr(nd), _stream()))
        return keys[:live], rows[:live]

    def read_rows(self, rows: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
        r = _dev(rows, torch.int64)
        w = torch.empty(r.numel(), self.dim, dtype=torch.float32, device=r.device)
        s = torch.empty(r.numel(), *self.state_shape, dtype=torch.float32, device=r.device)
        _check(lib().ht_read_rows(self.h, _ptr(r), r.numel(), _ptr(w), _ptr(s), _stream()))
        return w, s

    # ---------------------------------------------------------------- step
    def workspace_bytes(self, n: int, bags: int, pad_len: int = 0) -> int:
        return int(lib().lookup_workspace_bytes(n, bags, pad_len, self.h))

    def forward(self, values: torch.Tensor, offsets: torch.Tensor, mode: int, pad_len: int = 0,
                ctx: Optional[Ctx] = None, out: Optional[torch.Tensor] = None,
                mask: Optional[torch.Tensor] = None, validate: bool = False):
        v = _dev(values, torch.int64)
        o = _dev(offsets, torch.int64)
        n, bags = v.numel(), o.numel() - 1
        ctx = ctx or Ctx()
        ctx.ensure(self.workspace_bytes(n, bags, pad_len), v.device)
        if mode in (NONE, TAIL):
            odt = torch.bfloat16 if self.row_dtype == BF16 else torch.float32
            if out is None:
                out = torch.empty(bags, pad_len, self.dim, dtype=odt, device=v.device)
            if mask is None:
                mask = torch.empty(bags, pad_len, dtype=torch.uint8, device=v.device)
        elif out is None:
            out = torch.empty(bags, self.dim, dtype=torch.float32, device=v.device)
        ctx.keep = (v, o)
        _check(lib().lookup_pool_fwd(self.h, _ptr(v), _ptr(o), n, bags, mode, pad_len, _ptr(out), _ptr(mask),
                                     C.byref(ctx.c), int(validate), _stream()))
        return out, mask, ctx

    def prepare(self, values: torch.Tensor, offsets: torch.Tensor, mode: int, pad_len: int = 0,
                ctx: Optional[Ctx] = None, validate: bool = False, stream=None) -> Ctx:
        """First half of the forward (dedup, find-or-insert, bookkeeping) on `stream`."""
        v = _dev(values, torch.int64)
        o = _dev(offsets, torch.int64)
        n, bags = v.numel(), o.numel() - 1
        ctx = ctx or Ctx()
        ctx.ensure(self.workspace_bytes(n, bags, pad_len), v.device)
        ctx.keep = (v, o)
        st = C.c_void_p(stream.cuda_stream) if stream is not None else _stream()
        _check(lib().lookup_prepare(self.h, _ptr(v), _ptr(o), n, bags, mode, pad_len, C.byref(ctx.c),
                                    int(validate), st))
        return ctx

    def pool(self, ctx: Ctx, out: Optional[torch.Tensor] = None, mask: Optional[torch.Tensor] = None):
        """Second half of the forward: gather + pool of a prepared ctx."""
        c = ctx.c
        dev = ctx.ws.device
        if c.mode in (NONE, TAIL):
            odt = torch.bfloat16 if self.row_dtype == BF16 else torch.float32
            if out is None:
                out = torch.empty(c.bags, c.pad_len, self.dim, dtype=odt, device=dev)
            if mask is None:
                mask = torch.empty(c.bags, c.pad_len, dtype=torch.uint8, device=dev)
        elif out is None:
            out = torch.empty(c.bags, self.dim, dtype=torch.float32, device=dev)
        _check(lib().lookup_pool_prepared(self.h, C.byref(ctx.c), _ptr(out), _ptr(mask), _stream()))
        return out, mask

    def _grad(self, ctx: Ctx, grad_out: torch.Tensor) -> torch.Tensor:
        c = ctx.c
        if c.mode in (NONE, TAIL):
            want, dt = c.bags * c.pad_len * self.dim, (torch.bfloat16 if self.row_dtype == BF16 else torch.float32)
        else:
            want, dt = c.bags * self.dim, torch.float32
        if grad_out.numel() != want or grad_out.dtype != dt or not grad_out.is_cuda:
            raise RecisError(EINVAL, f"grad_out must be a GPU {dt} tensor with {want} elements")
        return grad_out.contiguous()

    def backward(self, ctx: Ctx, grad_out: torch.Tensor, grad_unique: Optional[torch.Tensor] = None):
        g = self._grad(ctx, grad_out)
        if grad_unique is None:
            grad_unique = torch.empty(max(ctx.c.n, 1), self.dim, dtype=torch.float32, device=g.device)
        _check(lib().lookup_pool_bwd(self.h, C.byref(ctx.c), _ptr(g), _ptr(grad_unique), _stream()))
        return grad_unique

    def optimizer_step(self, ctx: Ctx, grad_unique: torch.Tensor, lr: float, eps: float = 1e-8,
                       beta1: float = 0.9, beta2: float = 0.999, weight_decay: float = 0.0):
        p = OptParams(lr, eps, beta1, beta2, weight_decay)
        _check(lib().sparse_opt_step(self.h, C.byref(ctx.c), _ptr(grad_unique), C.byref(p), _stream()))

    def backward_optimizer(self, ctx: Ctx, grad_out: torch.Tensor, lr: float, eps: float = 1e-8,
                           beta1: float = 0.9, beta2: float = 0.999, weight_decay: float = 0.0):
        g = self._grad(ctx, grad_out)
        p = OptParams(lr, eps, beta1, beta2, weight_decay)
        _check(lib().lookup_pool_bwd_opt(self.h, C.byref(ctx.c), _ptr(g), C.byref(p), _stream()))

    def set_kernel_events(self, kernel: str, start, stop):
        """Record torch.cuda.Event `start` / `stop` around every launch of `kernel`."""
        if start is not None and (not start.cuda_event or not stop.cuda_event):
            # torch creates the underlying hipEvent_t on its first record()
            start.record()
            stop.record()
        s = None if start is None else C.c_void_p(start.cuda_event)
        e = None if stop is None else C.c_void_p(stop.cuda_event)
        _check(lib().rs_set_kernel_events(self.h, KERNELS[kernel], s, e))
