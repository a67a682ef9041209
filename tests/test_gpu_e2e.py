"""End-to-end parity over three consecutive steps, with no re-synchronisation.

The GPU table and the oracle table each run fwd -> fused bwd + optimizer for
three steps from the same seeded inputs, each side on its own rows (the
stage-wise tests instead restart the oracle from the GPU's rows every step).
After every step:
  * unique keys, inverse, inserted count: bit-exact;
  * pooled output: within 1e-5 * sum |x| per element, plus the rows' carried
    difference (the sum over the bag of the bound on each row's difference);
  * rows and optimizer state of every key of the step: within the fp32
    optimizer bound of the step (tests/parity.py::opt_bounds), the gradient
    allowed 1e-5 of its summed magnitudes, and the bounds of the key's
    earlier steps carried into it to first order.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2509_20883_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


class Carried:
    """Per-key bounds on |GPU - oracle| for the row and its state."""

    def __init__(self, dim, state_shape):
        self.keys = np.zeros(0, dtype=np.int64)
        self.bw = np.zeros((0, dim))
        self.bs = np.zeros((0,) + tuple(state_shape))

    def get(self, keys):
        bw = np.zeros((keys.size,) + self.bw.shape[1:])
        bs = np.zeros((keys.size,) + self.bs.shape[1:])
        if self.keys.size:
            i = np.searchsorted(self.keys, keys)
            i = np.minimum(i, self.keys.size - 1)
            hit = self.keys[i] == keys
            bw[hit] = self.bw[i[hit]]
            bs[hit] = self.bs[i[hit]]
        return bw, bs

    def put(self, keys, bw, bs):
        allk = np.union1d(self.keys, keys)
        nbw = np.zeros((allk.size,) + self.bw.shape[1:])
        nbs = np.zeros((allk.size,) + self.bs.shape[1:])
        if self.keys.size:
            j = np.searchsorted(allk, self.keys)
            nbw[j], nbs[j] = self.bw, self.bs
        j = np.searchsorted(allk, keys)
        nbw[j], nbs[j] = bw, bs
        self.keys, self.bw, self.bs = allk, nbw, nbs


@pytest.mark.parametrize("k", [0, 1, 2])
def test_three_steps_end_to_end(k):
    w = W.workload(k, mini=(k != 0))
    _log("end to end, 3 steps:", w.name, "mini" if w.mini else "full")
    gt, ot = P.gpu_table(w), P.oracle_table(w)
    P.prepopulate(w, gt, ot)
    carried = Carried(w.dim, ot.state_shape)
    for step in range(3):
        b = W.make_batch(w, step)
        grad = W.make_grad(w, b, step)
        st, uniq, inv = O.dedup(b.values)
        assert st == O.OK
        # the oracle inserts the step's new keys first (first-occurrence
        # order, as its step would), so their starting rows can be read
        st, _, n_new = ot.find_or_insert(uniq)
        assert st == O.OK
        _, w0, s0 = ot.read_rows(uniq)
        dw0, ds0 = carried.get(uniq)
        # GPU step
        out, _, ctx = gt.forward(P.to_dev(b.values), P.to_dev(b.offsets), w.mode)
        gt.backward_optimizer(ctx, P.to_dev(grad), w.lr, w.eps, w.beta1, w.beta2, w.weight_decay)
        sc = ctx.scalars().cpu().numpy()
        U = int(sc[0])
        assert U == uniq.size and int(sc[1]) == n_new, (U, uniq.size, int(sc[1]), n_new)
        assert np.array_equal(ctx.unique(U).cpu().numpy(), uniq)
        assert np.array_equal(ctx.inverse().cpu().numpy(), inv)
        w1, s1 = [x.cpu().numpy() for x in gt.read_rows(ctx.rows(U))]
        # oracle step on its own rows
        r = ot.step(b.values, b.offsets, w.mode, grad, w.lr, w.eps, w.beta1, w.beta2,
                    weight_decay=w.weight_decay)
        assert r["status"] == O.OK and r["U"] == U
        _, w1_ref, s1_ref = ot.read_rows(uniq)
        # pooled output: summation tolerance + the carried row differences
        tol = P.abs_pooled(w0, inv, b.offsets, w.mode) * 1e-5 + P.abs_pooled(dw0, inv, b.offsets, w.mode)
        P.assert_sum_close(out.cpu().numpy(), r["out"], tol, rel=1.0, what=f"step {step} pooled")
        # rows and state
        gu = O.backward(b.offsets, inv, U, w.dim, w.mode, 0, grad)
        gabs = O.backward(b.offsets, inv, U, w.dim, w.mode, 0, np.abs(grad))
        dg = 1e-5 * gabs + np.abs(gu) * 2.0 ** -23
        bw, bs = P.opt_bounds(w.opt, w.row_dtype, w0, s0, gu, dg, w.lr, w.eps, w.beta1, w.beta2, ot.t, w1_ref,
                              w.weight_decay, dw0=dw0, ds0=ds0)
        P.assert_opt_close(w1, s1, w1_ref, s1_ref, (bw, bs), what=f"step {step} rows")
        carried.put(uniq, bw, bs)
        _log(f"  step {step}: N={b.n} U={U} new={n_new} max |dw| {np.abs(w1 - w1_ref).max():.3g}")
    gt.check()
    assert gt.size() == ot.size()
    gt.close()
