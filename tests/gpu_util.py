"""Helpers of the GPU parity tests: run a generated case through the C ABI
(via the ctypes binding) and through the oracle, on the same inputs."""
import os
import sys
import time
from contextlib import contextmanager

import numpy as np
import torch

from paper_2006_10226_amd import qnn as Q
from oracle import oracle as O
import workloads as W


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@contextmanager
def env(**kw):
    old = {k: os.environ.get(k) for k in kw}
    os.environ.update({k: str(v) for k, v in kw.items()})
    try:
        yield
    finally:
        for k, v in old.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def xdtype(a: np.ndarray) -> str:
    return {np.dtype(np.uint8): "u8", np.dtype(np.int8): "i8"}[a.dtype]


def make_plan(c: W.ConvCase, N=None, y_ldc=None, y_coff=0):
    """Plan for a ConvCase (conv, depthwise or dense)."""
    w = dev(c.w)
    bias = None if c.bias is None else dev(c.bias)
    if c.dense:
        M, K = c.x.shape
        return Q.dense_plan(M, K, xdtype(c.x), c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.s_y, c.zp_y, c.yt,
                            c.act, c.rounding, y_ldc), (w, bias)
    shape = c.x.shape if N is None else (N,) + c.x.shape[1:]
    if c.depthwise:
        p = Q.depthwise_conv2d_plan(shape, xdtype(c.x), c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride, c.pads,
                                    1, c.s_y, c.zp_y, c.yt, c.act, c.rounding, y_ldc, y_coff)
    else:
        p = Q.conv2d_plan(shape, xdtype(c.x), c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride, c.pads, 1,
                          c.s_y, c.zp_y, c.yt, c.act, c.rounding, y_ldc, y_coff)
    return p, (w, bias)


def run_gpu(c: W.ConvCase, one_shot=False):
    """Output of the HIP path for a case, as numpy."""
    x = dev(c.x)
    if one_shot:
        w = dev(c.w)
        bias = None if c.bias is None else dev(c.bias)
        if c.dense:
            y = Q.dense(x, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.s_y, c.zp_y, c.yt, c.act, c.rounding)
        elif c.depthwise:
            y = Q.depthwise_conv2d(x, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride, c.pads, 1, c.s_y, c.zp_y,
                                   c.yt, c.act, c.rounding)
        else:
            y = Q.conv2d(x, c.s_x, c.zp_x, w, c.s_w, c.zp_w, bias, c.stride, c.pads, 1, c.s_y, c.zp_y, c.yt,
                         c.act, c.rounding)
    else:
        p, keep = make_plan(c)
        y = p.run(x)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    return y.cpu().numpy()


def run_oracle(c: W.ConvCase):
    """Full oracle output of a case."""
    if c.dense:
        return O.dense(c.x, c.s_x, c.zp_x, c.w, c.s_w, c.zp_w, c.bias, c.s_y, c.zp_y, c.yt, c.act, c.rounding)
    return O.conv2d(c.x, c.s_x, c.zp_x, c.w, c.s_w, c.zp_w, c.bias, c.s_y, c.zp_y, c.yt, c.act, c.rounding,
                    c.stride, c.pads, (1, 1), c.depthwise)


def oracle_points(c: W.ConvCase, idx):
    """Oracle outputs at flat output indices (conv / depthwise)."""
    acc = O.conv2d_acc_points(c.x, c.zp_x, c.w, idx, c.zp_w, c.bias, c.stride, c.pads, (1, 1), c.depthwise)
    if c.yt == "i32":
        return acc
    return O.requantize_points(acc, idx, c.K, c.s_x, c.s_w, c.s_y, c.zp_y, c.yt, c.act, c.rounding)


def assert_equal(got, ref, what):
    got = np.asarray(got)
    ref = np.asarray(ref)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    bad = np.flatnonzero(got.reshape(-1).astype(np.int64) != ref.reshape(-1).astype(np.int64))
    if bad.size:
        i = bad[0]
        raise AssertionError(f"{what}: {bad.size} of {got.size} outputs differ; first at flat {i}: "
                             f"gpu {got.reshape(-1)[i]} oracle {ref.reshape(-1)[i]}")
