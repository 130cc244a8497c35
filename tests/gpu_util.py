"""Helpers of the GPU parity tests: run the HIP path through the C ABI and
judge its outputs with the oracle's lockstep verifier."""
from __future__ import annotations

import sys

import numpy as np


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_fit(W, bits, P, G, tol, grid=None, with_err=True, dense=False):
    """mpq_fit_layer (histogram search up to d = 32768) or, with dense=True,
    mpq_fit_layer_dense, through the C ABI."""
    import torch
    from paper_2002_09049_amd import mpq
    Wd = to_dev(W)
    codes, scales, counts, err = mpq.fit_layer(Wd, bits, P, G, tol, grid=grid, with_err=with_err,
                                               dense=dense)
    torch.cuda.synchronize()
    return (codes.cpu().numpy(), scales.cpu().numpy(), counts.cpu().numpy(),
            None if err is None else err.cpu().numpy())


def assert_parity(orc, W, bits, P, G, tol, out, grid=None, channels=None):
    """Lockstep check (rules V1-V4) of every listed channel; returns the
    verifier's report.  tol is rounded to fp32 as the C ABI takes it."""
    codes, scales, counts, err = out
    tol32 = float(np.float32(tol))
    v = orc.verify(W, bits, P, G, tol32, codes, scales, counts, err, grid=grid, channels=channels)
    bad = np.nonzero(v["status"])[0]
    assert bad.size == 0, (f"{bad.size} channels fail: channels {v['channels'][bad][:8]} "
                           f"status {v['status'][bad][:8]}")
    return v


def free_running_diff(orc, W, bits, P, G, tol, out, grid=None, channels=None):
    """Compare with the oracle's own free-running fit.  Returns the number of
    channels whose (codes, scales, counts) differ."""
    codes, scales, counts, _ = out
    tol32 = float(np.float32(tol))
    Ws = W if channels is None else W[channels]
    oc, os_, on, _ = orc.fit(Ws, bits, P, G, tol32, grid=grid)
    if channels is not None:
        codes, scales, counts = codes[channels], scales[channels], counts[channels]
    diff = (on != counts) | (os_ != scales).any(axis=1) | (oc != codes).any(axis=(1, 2))
    return int(diff.sum())
