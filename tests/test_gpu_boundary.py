"""The boundary's error and ownership paths, on the GPU (through the C ABI).

  * validate = 1 rejects malformed CSR offsets with RS_EINVAL (host check,
    before any kernel is enqueued);
  * offsets that do not cover every id (validate = 0) give in-bounds work:
    the covered bags pool correctly and the backward gives the uncovered ids
    no gradient row;
  * an allocator that returns NULL gives RS_ENOMEM, at creation and when the
    table has to grow, and the table stays consistent afterwards;
  * a table whose IDMap, Blocks and workspace all come from PyTorch's caching
    allocator matches the oracle step by step while it grows;
  * the optimizer's bf16 store rounds ties to even.
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


def test_validate_rejects_malformed_offsets():
    _log("validate: malformed offsets")
    w = W.workload(0)
    b = W.make_batch(w, 0)
    gt = P.gpu_table(w)
    v = P.to_dev(b.values)
    good = b.offsets.copy()
    bad = {"first offset not 0": np.concatenate([[1], good[1:]]),
           "last offset not n": np.concatenate([good[:-1], [good[-1] - 1]]),
           "decreasing": good.copy()}
    bad["decreasing"][5], bad["decreasing"][6] = good[6], good[5] - 1
    for name, off in bad.items():
        with pytest.raises(R.RecisError) as e:
            gt.forward(v, P.to_dev(off.astype(np.int64)), w.mode, validate=True)
        assert e.value.status == R.EINVAL, name
    # the same call with well-formed offsets goes through, and nothing was latched
    gt.forward(v, P.to_dev(good), w.mode, validate=True)
    gt.check()
    gt.close()


@pytest.mark.parametrize("k", [0, 2])
def test_offsets_not_covering_every_id_stay_in_bounds(k):
    """validate = 0 and offsets that leave ids outside every bag: the kernels
    stay in bounds (positions clamped to [0, n), occurrence-list entries
    outside the gradient rows skipped); covered bags pool exactly as
    defined, and the backward sums over the covered ids only (the uncovered
    ones contribute nothing).  The workspace starts as random bytes."""
    w = W.workload(k, mini=(k != 0))
    _log("uncovered ids without validation", w.name)
    b = W.make_batch(w, 0)
    off = b.offsets.copy()
    off[0] = off[1]      # the first bag's ids are in no bag
    off[-1] = off[-2]    # nor the last bag's
    assert off[0] > 0 and off[-1] < b.n and np.all(np.diff(off) >= 0)
    gt = P.gpu_table(w)
    ctx = R.Ctx()
    ctx.ensure(gt.workspace_bytes(b.n, b.bags), torch.device("cuda"))
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    ctx.ws.copy_(torch.randint(0, 256, ctx.ws.shape, dtype=torch.uint8, device="cuda", generator=g))
    out, _, ctx = gt.forward(P.to_dev(b.values), P.to_dev(off), w.mode, ctx=ctx)
    grad = W.make_grad(w, b, 0)
    gu = gt.backward(ctx, P.to_dev(grad))
    gt.optimizer_step(ctx, gu, w.lr, w.eps)
    torch.cuda.synchronize()
    gt.check()
    U = int(ctx.scalars()[0].item())
    st, u_ref, inv_ref = O.dedup(b.values)
    assert st == O.OK and U == u_ref.size
    assert np.array_equal(ctx.inverse().cpu().numpy(), inv_ref)
    # the backward over the bags as given: ids outside them contribute nothing
    gu_ref = O.backward(off, inv_ref, U, w.dim, w.mode, 0, grad)
    gu_abs = O.backward(off, inv_ref, U, w.dim, w.mode, 0, np.abs(grad))
    P.assert_sum_close(gu.cpu().numpy()[:U], gu_ref, gu_abs, what="gradient of the covered ids")
    # covered bags: the sum of the initial rows of their ids
    ot = P.oracle_table(w)
    ot.find_or_insert(u_ref)
    _, rows0, _ = ot.read_rows(u_ref)
    o = out.cpu().numpy()
    lens = np.diff(off)
    bag = np.repeat(np.arange(b.bags), lens)
    pos = np.arange(off[0], off[-1])
    ref = np.zeros((b.bags, w.dim))
    np.add.at(ref, bag, rows0[inv_ref[pos]].astype(np.float64))
    scale = np.zeros((b.bags, w.dim))
    np.add.at(scale, bag, np.abs(rows0[inv_ref[pos]].astype(np.float64)))
    if w.mode == R.MEAN:
        ref /= np.maximum(lens, 1)[:, None]
        scale /= np.maximum(lens, 1)[:, None]
    P.assert_sum_close(o, ref, scale, what="covered bags")
    gt.close()


def test_allocator_returning_null_gives_enomem():
    _log("allocator returning NULL")
    w = W.workload(0)
    with pytest.raises(R.RecisError) as e:
        P.gpu_table(w, allocator=R.TorchAllocator(fail_after=0))
    assert e.value.status == R.ENOMEM
    # creation takes three allocations (IDMap, scalars, Blocks chunk table);
    # the first forward then needs Blocks rows and gets NULL
    alloc = R.TorchAllocator(fail_after=3)
    gt = P.gpu_table(w, allocator=alloc)
    b = W.make_batch(w, 0)
    with pytest.raises(R.RecisError) as e:
        gt.forward(P.to_dev(b.values), P.to_dev(b.offsets), w.mode)
    assert e.value.status == R.ENOMEM
    # the table stays consistent: nothing was inserted, and with memory again
    # the same batch goes through and matches the oracle
    assert gt.size() == 0
    alloc.fail_after = None
    ot = P.oracle_table(w)
    P.run_step_parity(w, gt, ot, b, W.make_grad(w, b, 0), 0)
    gt.check()
    gt.close()
    assert not alloc.live, "every allocation was returned"


@pytest.mark.parametrize("k", [0, 2])
def test_torch_allocator_backs_a_growing_table(k):
    """IDMap, Blocks and workspace from PyTorch's caching allocator: small
    Blocks chunks (many of them) and a small IDMap that rehashes."""
    w = W.workload(k, mini=(k != 0))
    _log("torch allocator", w.name)
    alloc = R.TorchAllocator()
    before = torch.cuda.memory_allocated()
    gt = P.gpu_table(w, allocator=alloc, block_rows=1024, capacity_slots=1 << 12)
    ot = P.oracle_table(w)
    for step in range(3):
        b = W.make_batch(w, step)
        U, nn = P.run_step_parity(w, gt, ot, b, W.make_grad(w, b, step), step)
        _log(f"  step {step}: U={U} new={nn} capacity={gt.capacity()}")
    assert gt.capacity() > (1 << 12)                   # the IDMap grew
    assert torch.cuda.memory_allocated() > before      # the table lives in torch's pool
    assert len(alloc.live) > gt.size() // 1024         # one allocation per chunk of 1024 rows
    gt.check()
    gt.close()
    assert not alloc.live


def test_bf16_optimizer_store_rounds_ties_to_even():
    """Rows initialised to exactly 1.0 (lo = hi = 1), Adagrad with eps = 0 and
    upstream gradients of +-1 on single-id bags: the update is exactly
    lr * sign(g), so w - lr*sign(g) lands on a bf16 tie or an exact value:
      lr = 2^-9, g = +1: 1 - 2^-9, a tie between 0x3F7F (odd) and 0x3F80 -> 0x3F80
      lr = 2^-8, g = -1: 1 + 2^-8, a tie between 0x3F80 and 0x3F81 (odd)  -> 0x3F80
      lr = 2^-8, g = +1: 1 - 2^-8 = 0x3F7F exactly
    (truncation would give 0x3F7F in the first case, rounding half up 0x3F81
    in the second)."""
    _log("bf16 ties")
    keys = np.arange(1, 65, dtype=np.int64) * 1000003
    offs = np.arange(keys.size + 1, dtype=np.int64)
    for lr, sign, want in ((2.0 ** -9, 1.0, 0x3F80), (2.0 ** -8, -1.0, 0x3F80), (2.0 ** -8, 1.0, 0x3F7F)):
        gt = R.Table(16, R.BF16, R.ADAGRAD, 1.0, 1.0, 7, 1 << 10, 0.75, 1024)
        ot = O.Table(16, row_dtype=O.BF16, opt=O.ADAGRAD, lo=1.0, hi=1.0, seed=7)
        grad = np.full((keys.size, 16), sign, dtype=np.float32)
        _, _, ctx = gt.forward(P.to_dev(keys), P.to_dev(offs), R.SUM)
        gt.backward_optimizer(ctx, P.to_dev(grad), lr, 0.0)
        wg, sg = gt.read_rows(ctx.rows(keys.size))
        wg = wg.cpu().numpy()
        bits = (wg.view(np.uint32) >> 16).astype(np.uint32)
        assert np.all((wg.view(np.uint32) & 0xFFFF) == 0)  # bf16 values widened exactly
        assert np.all(bits == want), (lr, sign, np.unique(bits))
        assert np.all(sg.cpu().numpy() == 1.0)             # acc = g^2
        r = ot.step(keys, offs, O.SUM, grad, lr, 0.0)
        assert r["status"] == O.OK
        _, wr, _ = ot.read_rows(keys)
        assert np.array_equal(wg, wr)                      # the oracle rounds the same way
        gt.close()
