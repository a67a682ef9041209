"""Helpers shared by the GPU parity tests: build matching GPU / oracle tables,
run one step on both from the same seeded inputs, and compare them at the
stated tolerances.

Tolerances (fp32 arithmetic against the oracle's fp64):
  pooled / per-unique gradient sums: |err| <= 1e-5 * sum |terms| per element
  optimizer (stage-wise, same gradient on both sides): first-order fp32
    error bound, 1e-6 of the magnitude of the terms of every operation
    (opt_bounds); bf16 rows additionally 1e-2 * |w_ref| + 1e-6 or one bf16 ulp
  integers (unique, inverse, rows, present set) and copied rows: bit-exact
"""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2509_20883_amd import recis as R
from paper_2509_20883_amd import workloads as W


def gpu_table(w: W.Workload, **kw) -> R.Table:
    args = dict(dim=w.dim, row_dtype=w.row_dtype, optimizer=w.opt, init_lo=w.init_lo, init_hi=w.init_hi,
                seed=w.table_seed, capacity_slots=w.capacity_slots, max_load=w.max_load,
                block_rows=w.block_rows, auto_grow=True)
    args.update(kw)
    return R.Table(**args)


def oracle_table(w: W.Workload, max_live: int = -1) -> O.Table:
    return O.Table(w.dim, row_dtype=w.row_dtype, opt=w.opt, lo=w.init_lo, hi=w.init_hi, seed=w.table_seed,
                   max_live=max_live)


def prepopulate(w: W.Workload, gt: R.Table, ot: O.Table = None):
    for keys in W.prepop_keys(w):
        gt.find_or_insert(torch.from_numpy(keys).cuda())
        if ot is not None:
            ot.find_or_insert(keys)


def to_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def assert_sum_close(got, ref, abs_terms, rel=1e-5, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    bound = rel * np.asarray(abs_terms, dtype=np.float64) + 1e-30
    err = np.abs(got - ref)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance, e.g. at {idx.tolist()}: "
                             f"got {got[tuple(idx[0])]}, ref {ref[tuple(idx[0])]}, bound {bound[tuple(idx[0])]}")


def abs_pooled(ot_rows_w: np.ndarray, inverse: np.ndarray, offsets: np.ndarray, mode: int) -> np.ndarray:
    """sum_{i in bag} |x_i| per element (the pooled-output tolerance scale)."""
    lens = np.diff(offsets)
    bag_of = np.repeat(np.arange(len(lens)), lens)
    acc = np.zeros((len(lens), ot_rows_w.shape[1]))
    valid = inverse >= 0
    np.add.at(acc, bag_of[valid], np.abs(ot_rows_w[inverse[valid]].astype(np.float64)))
    if mode == O.MEAN:
        acc[lens > 0] /= lens[lens > 0, None]
    return acc


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    a = np.abs(x.astype(np.float32))
    e = np.floor(np.log2(np.maximum(a, 1e-38)))
    return 2.0 ** (e - 7)


def opt_bounds(opt, row_dtype, w0, s0, g, dg, lr, eps, b1, b2, t, w_ref, wd=0.0, dw0=0.0, ds0=0.0):
    """Error bounds of an fp32 optimizer step against the fp64 oracle.

    Each fp32 operation is allowed 1e-6 of the magnitude of its terms (about
    16 units of fp32 rounding), so cancellation in m = b1*m + (1-b1)*g or in
    w - update is bounded by the terms, not the result; `dg` is an extra
    uncertainty of the gradient itself (0 when both sides use the same one),
    propagated to first order.  dw0 / ds0 (shapes of w0 / s0) bound how far
    the GPU's starting row and state already are from the oracle's (earlier
    steps without re-synchronisation; Adagrad and the Adam family): they are
    carried through the step to first order.  Returns (bound_w, bound_state)."""
    f = np.float64
    w0, g, dg, w_ref = (np.asarray(x, f) for x in (w0, g, dg, w_ref))
    s0 = np.asarray(s0, f)
    ds0 = np.broadcast_to(np.asarray(ds0, f), s0.shape)
    dw0 = np.broadcast_to(np.asarray(dw0, f), w0.shape)
    ag = np.abs(g)
    if opt in (O.ADAGRAD_RW, O.ADAM_RW):
        # the row mean of g^2: an fp32 tree sum over the row (a few roundings
        # per level) plus the gradient's own uncertainty
        D = g.shape[1]
        ms = (g * g).mean(axis=1)
        d_ms = 4e-6 * ms + (2 * ag * dg + dg * dg).mean(axis=1) + 1e-37
        if opt == O.ADAGRAD_RW:
            acc1 = s0[:, 0] + ms
            b_acc = 1e-6 * acc1 + d_ms
            sq = np.sqrt(acc1)
            dsq = np.minimum(b_acc / np.maximum(2 * sq, 1e-30), np.sqrt(b_acc))
            den = (sq + eps)[:, None]
            upd = lr * ag / den
            d_upd = lr * (dg / den + ag * dsq[:, None] / den ** 2) + 1e-6 * upd
            b_state = b_acc[:, None]
        else:
            bc1, bc2 = 1.0 - b1 ** t, 1.0 - b2 ** t
            m1 = b1 * s0[:, :D] + (1 - b1) * g
            v1 = b2 * s0[:, D] + (1 - b2) * ms
            b_m = 1e-6 * (b1 * np.abs(s0[:, :D]) + (1 - b1) * ag) + (1 - b1) * dg + 1e-37
            b_v = 1e-6 * (b2 * s0[:, D] + (1 - b2) * ms) + (1 - b2) * d_ms
            sq = np.sqrt(v1 / bc2)
            dsq = np.minimum((b_v / bc2) / np.maximum(2 * sq, 1e-30), np.sqrt(b_v / bc2))
            den = (sq + eps)[:, None]
            mh = np.abs(m1) / bc1
            upd = lr * mh / den
            d_upd = lr * ((b_m / bc1) / den + mh * dsq[:, None] / den ** 2) + 1e-6 * upd
            b_state = np.concatenate([b_m, b_v[:, None]], axis=1)
    elif opt == O.ADAGRAD:
        acc1 = s0[:, 0] + g * g
        b_acc = 1e-6 * acc1 + 2 * ag * dg + dg * dg + ds0[:, 0] + 1e-37
        sq = np.sqrt(acc1)
        dsq = np.minimum(b_acc / np.maximum(2 * sq, 1e-30), np.sqrt(b_acc))
        upd = lr * ag / (sq + eps)
        d_upd = lr * (dg / (sq + eps) + ag * dsq / (sq + eps) ** 2) + 1e-6 * upd
        b_state = b_acc[:, None, :]
    else:
        bc1, bc2 = 1.0 - b1 ** t, 1.0 - b2 ** t
        m1 = b1 * s0[:, 0] + (1 - b1) * g
        v1 = b2 * s0[:, 1] + (1 - b2) * g * g
        b_m = 1e-6 * (b1 * np.abs(s0[:, 0]) + (1 - b1) * ag) + (1 - b1) * dg + b1 * ds0[:, 0] + 1e-37
        b_v = (1e-6 * (b2 * s0[:, 1] + (1 - b2) * g * g) + (1 - b2) * (2 * ag * dg + dg * dg) + b2 * ds0[:, 1]
               + 1e-37)
        if opt == O.ADAM_TF:
            # w -= lr_t m / (sqrt(v) + eps), lr_t = lr sqrt(bc2) / bc1
            lrt = lr * np.sqrt(bc2) / bc1
            sq = np.sqrt(v1)
            dsq = np.minimum(b_v / np.maximum(2 * sq, 1e-30), np.sqrt(b_v))
            upd = lrt * np.abs(m1) / (sq + eps)
            d_upd = lrt * (b_m / (sq + eps) + np.abs(m1) * dsq / (sq + eps) ** 2) + 1e-6 * upd
        else:
            mh, vh = np.abs(m1) / bc1, v1 / bc2
            sq = np.sqrt(vh)
            dsq = np.minimum((b_v / bc2) / np.maximum(2 * sq, 1e-30), np.sqrt(b_v / bc2))
            upd = lr * mh / (sq + eps)
            d_upd = lr * ((b_m / bc1) / (sq + eps) + mh * dsq / (sq + eps) ** 2) + 1e-6 * upd
            if opt == O.ADAMW:  # w -= (lr wd) w first: one more rounded product
                d_upd = d_upd + 1e-6 * lr * wd * np.abs(w0)
        b_state = np.stack([b_m, b_v], axis=1)
    if row_dtype == O.BF16:
        b_w = np.maximum(1e-2 * np.abs(w_ref) + 1e-6, 1.01 * bf16_ulp(w_ref)) + d_upd + dw0
    else:
        b_w = 1e-6 * np.maximum(np.maximum(np.abs(w0), np.abs(w_ref)), lr) + d_upd + dw0
    return b_w, b_state


def assert_opt_close(w_gpu, s_gpu, w_ref, s_ref, bounds, what=""):
    b_w, b_s = bounds
    err = np.abs(np.asarray(w_gpu, np.float64) - np.asarray(w_ref, np.float64))
    if (err > b_w).any():
        i = np.argwhere(err > b_w)[0]
        raise AssertionError(f"{what}: {(err > b_w).sum()} row elements out of tolerance, e.g. {i.tolist()}: "
                             f"gpu {w_gpu[tuple(i)]} ref {w_ref[tuple(i)]} bound {b_w[tuple(i)]}")
    se = np.abs(np.asarray(s_gpu, np.float64) - np.asarray(s_ref, np.float64))
    if (se > b_s).any():
        i = np.argwhere(se > b_s)[0]
        raise AssertionError(f"{what}: {(se > b_s).sum()} state elements out of tolerance, e.g. {i.tolist()}: "
                             f"gpu {s_gpu[tuple(i)]} ref {s_ref[tuple(i)]} bound {b_s[tuple(i)]}")


def run_step_parity(w: W.Workload, gt: R.Table, ot: O.Table, batch: W.Batch, grad: np.ndarray, step: int,
                    check_rows_exact: bool = True):
    """One step on both sides; compares every stage.  Returns (U, n_new)."""
    v, off = batch.values, batch.offsets
    pad = w.pad_len if w.mode in (O.NONE, O.TAIL) else 0
    out, mask, ctx = gt.forward(to_dev(v), to_dev(off), w.mode, pad_len=pad)
    torch.cuda.synchronize()
    ref = ot.forward(v, off, w.mode, pad_len=pad)
    assert ref["status"] == O.OK
    sc = ctx.scalars().cpu().numpy()
    U = int(sc[0])
    assert U == ref["U"], f"U {U} vs {ref['U']}"
    assert int(sc[1]) == ref["n_new"], f"inserted {sc[1]} vs {ref['n_new']}"
    assert np.array_equal(ctx.unique(U).cpu().numpy(), ref["unique"]), "unique differs"
    assert np.array_equal(ctx.inverse().cpu().numpy(), ref["inverse"]), "inverse differs"
    g_rows = ctx.rows(U).cpu().numpy()
    if check_rows_exact:
        assert np.array_equal(g_rows, ref["rows"]), "row ids differ"
    # pre-optimizer rows of every unique key (GPU), and the oracle's view of them
    w0, s0 = gt.read_rows(ctx.rows(U))
    w0, s0 = w0.cpu().numpy(), s0.cpu().numpy()
    _, w0_ref, s0_ref = ot.read_rows(ref["unique"])
    # rows found or inserted this step hold the same bits on both sides
    assert np.array_equal(w0, w0_ref) and np.array_equal(s0, s0_ref), "rows before the optimizer differ"
    # forward output
    if w.mode in (O.NONE, O.TAIL):
        o = out.float().cpu().numpy()
        assert np.array_equal(o, ref["out"].astype(np.float32)), "padded gather differs"
        assert np.array_equal(mask.cpu().numpy(), ref["mask"]), "mask differs"
    else:
        scale = abs_pooled(w0_ref, ref["inverse"], off, w.mode)
        assert_sum_close(out.cpu().numpy(), ref["out"], scale, what=f"step {step} pooled")
    # backward (per-unique sums), stage-wise
    gdev = to_dev(grad)
    if w.mode in (O.NONE, O.TAIL) and w.row_dtype == O.BF16:
        gdev = gdev.to(torch.bfloat16)
    gu = gt.backward(ctx, gdev)
    gu_gpu = gu[:U].cpu().numpy()
    gfin = np.where(np.isfinite(grad), grad, 0).astype(np.float32)
    gu_ref = O.backward(off, ref["inverse"], U, w.dim, w.mode, pad, grad)
    gu_abs = O.backward(off, ref["inverse"], U, w.dim, w.mode, pad, np.abs(gfin))
    assert_sum_close(gu_gpu, gu_ref, gu_abs, what=f"step {step} grad_unique")
    # optimizer, stage-wise: oracle starts from the GPU's pre-state and grads
    gt.optimizer_step(ctx, gu, w.lr, w.eps, w.beta1, w.beta2, w.weight_decay)
    w1, s1 = gt.read_rows(ctx.rows(U))
    w1, s1 = w1.cpu().numpy(), s1.cpu().numpy()
    ot.write_rows(ref["unique"], w0, s0)
    ot.optimizer(ref["rows"], gu_gpu, w.lr, w.eps, w.beta1, w.beta2, weight_decay=w.weight_decay)
    _, w1_ref, s1_ref = ot.read_rows(ref["unique"])
    bounds = opt_bounds(w.opt, w.row_dtype, w0, s0, gu_gpu, 0.0, w.lr, w.eps, w.beta1, w.beta2, ot.t, w1_ref,
                        w.weight_decay)
    assert_opt_close(w1, s1, w1_ref, s1_ref, bounds, what=f"step {step} optimizer")
    # the next step starts both sides from the GPU's updated rows (stage-wise
    # parity: fp32 vs fp64 optimizer rounding is not carried into later steps)
    ot.write_rows(ref["unique"], w1, s1)
    return U, int(sc[1])
