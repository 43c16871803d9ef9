"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every symbol of include/qnn.h, the fixed-point multiplier the
library derives agrees with the oracle's independent derivation, and every
validation error path returns its status without touching the device."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def Q():
    from paper_2006_10226_amd import qnn
    qnn.lib()
    return qnn


def _header_functions():
    text = open(os.path.join(ROOT, "include", "qnn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qnn_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(Q):
    declared = _header_functions()
    assert len(declared) >= 17
    assert sorted(Q.EXPORTS) == declared
    L = Q.lib()
    for name in declared:
        assert hasattr(L, name), name
    assert L.qnn_abi_version() == 1
    for code, name in enumerate(Q.STATUS):
        assert L.qnn_status_string(code).decode() == name


def test_multiplier_agrees_with_oracle(Q, oracle):
    """The library and the oracle derive (mult, shift) independently from
    the same rule; they must agree on random scale triples."""
    rng = np.random.default_rng(0)
    n = 100000
    s_x = (10.0 ** rng.uniform(-4, 0, n)).astype(np.float32)
    s_w = (10.0 ** rng.uniform(-5, -1, n)).astype(np.float32)
    s_y = (10.0 ** rng.uniform(-4, 1, n)).astype(np.float32)
    for i in range(n):
        M = (float(s_x[i]) * float(s_w[i])) / float(s_y[i])
        assert Q.quantize_multiplier(M) == oracle.quantize_multiplier(M)
    for M in (0.0, 1.0, 0.5, 2.0**-80, 1e-300, 2.0**29, float(np.nextafter(1.0, 0.0))):
        assert Q.quantize_multiplier(M) == oracle.quantize_multiplier(M)
    for M in (2.0**30, float("inf"), float("nan"), -1.0):
        with pytest.raises(Q.QnnError) as e:
            Q.quantize_multiplier(M)
        assert e.value.status_name == "QNN_ERR_QPARAM"


FAKE = ctypes.c_void_p(0x10000)   # never dereferenced: validation fails first


def _conv(Q, **kw):
    """Call qnn_conv2d with defaults overridden by kw; returns (status, msg)."""
    a = dict(x=FAKE, xt=Q.UINT8, N=1, H=8, W=8, C=16, xs=0.02, xz=128,
             w=FAKE, K=32, R=3, S=3, ws=[0.01], wz=[0], bias=None,
             cp=(1, 1, 1, 1, 1, 1, 1, 1), y=FAKE, yt=Q.UINT8, ys=0.05, yz=0,
             act=(-(2**31), 2**31 - 1), rnd=Q.HALF_UP, y_ldc=32, y_coff=0, xn=1, yn=1)
    a.update(kw)
    xq = Q._Q(a["xs"], a["xz"], a["xn"])
    wq = Q._Q(a["ws"], a["wz"], len(np.atleast_1d(a["ws"])))
    yq = Q._Q(a["ys"], a["yz"], a["yn"])
    st = Q.lib().qnn_conv2d(None, a["x"], a["xt"], a["N"], a["H"], a["W"], a["C"], xq.q, a["w"], a["K"],
                            a["R"], a["S"], wq.q, a["bias"], Q.ConvParams(*a["cp"]), a["y"], a["yt"], yq.q,
                            Q.Clamp(*a["act"]), a["rnd"], a["y_ldc"], a["y_coff"])
    return Q.STATUS[st], Q.lib().qnn_last_error().decode()


@pytest.mark.parametrize("kw,expect", [
    (dict(x=None), "QNN_ERR_NULL"),
    (dict(y=None), "QNN_ERR_NULL"),
    (dict(w=None), "QNN_ERR_NULL"),
    (dict(xt=2), "QNN_ERR_DTYPE"),
    (dict(yt=7), "QNN_ERR_DTYPE"),
    (dict(rnd=5), "QNN_ERR_QPARAM"),
    (dict(H=0), "QNN_ERR_SHAPE"),
    (dict(C=0), "QNN_ERR_SHAPE"),
    (dict(N=-1), "QNN_ERR_SHAPE"),
    (dict(cp=(0, 1, 1, 1, 1, 1, 1, 1)), "QNN_ERR_SHAPE"),
    (dict(cp=(1, 1, -1, 1, 1, 1, 1, 1)), "QNN_ERR_SHAPE"),
    (dict(cp=(1, 1, 1, 1, 1, 1, 0, 1)), "QNN_ERR_SHAPE"),
    (dict(R=11, cp=(1, 1, 0, 0, 0, 0, 1, 1)), "QNN_ERR_SHAPE"),
    (dict(y_ldc=31), "QNN_ERR_SHAPE"),
    (dict(y_ldc=40, y_coff=9), "QNN_ERR_SHAPE"),
    (dict(y_coff=-1), "QNN_ERR_SHAPE"),
    (dict(xs=0.0), "QNN_ERR_QPARAM"),
    (dict(xs=float("nan")), "QNN_ERR_QPARAM"),
    (dict(xs=-0.5), "QNN_ERR_QPARAM"),
    (dict(xz=256), "QNN_ERR_QPARAM"),
    (dict(xt=1, xz=128), "QNN_ERR_QPARAM"),
    (dict(wz=[128]), "QNN_ERR_QPARAM"),
    (dict(ws=[0.01] * 5, wz=[0] * 5), "QNN_ERR_QPARAM"),
    (dict(ws=[float("inf")]), "QNN_ERR_QPARAM"),
    (dict(ys=0.0), "QNN_ERR_QPARAM"),
    (dict(yz=-1), "QNN_ERR_QPARAM"),
    (dict(yt=1, yz=200), "QNN_ERR_QPARAM"),
    (dict(act=(300, 400)), "QNN_ERR_QPARAM"),
    (dict(act=(10, 5)), "QNN_ERR_QPARAM"),
    (dict(ys=1e-13), "QNN_ERR_QPARAM"),          # multiplier >= 2^30
    (dict(C=4096, R=3, S=3, xz=0, wz=[127]), "QNN_ERR_OVERFLOW"),   # 36864 * 255 * 255 >= 2^31
    (dict(N=2**20, H=64, W=64), "QNN_ERR_UNSUPPORTED"),
    # 9 channels padded to 12 for the gather: N*H*W*9 < 2^31 <= N*H*W*12
    (dict(H=14000, W=14000, C=9, K=4, y_ldc=4), "QNN_ERR_UNSUPPORTED"),
])
def test_conv_validation_errors(Q, kw, expect):
    st, msg = _conv(Q, **kw)
    assert st == expect, msg
    assert msg


def test_overflow_bound_is_tight(Q):
    """J * 255 * 255 < 2^31 passes validation for J = 33025 - 1 taps when
    x and w zero points are at the dtype edge; one more tap fails."""
    # C * R * S = J; with zp_x = 0 (uint8) max|x-zp| = 255, zp_w = 127 gives max|w-zp| = 255
    st, msg = _conv(Q, C=33026, R=1, S=1, K=4, cp=(1, 1, 0, 0, 0, 0, 1, 1), xz=0, wz=[127], y_ldc=4,
                    H=1, W=1)
    assert st == "QNN_ERR_OVERFLOW", msg
    st, msg = _conv(Q, C=33025, R=1, S=1, K=4, cp=(1, 1, 0, 0, 0, 0, 1, 1), xz=0, wz=[127], y_ldc=4,
                    H=1, W=1, N=0)
    assert st == "QNN_OK", msg    # N = 0: valid no-op, nothing launched


def test_requantize_and_add_validation(Q):
    L = Q.lib()
    q1 = Q._Q(0.1, 0, 1)
    qz = Q._Q(0.1, 3, 1)
    qc = Q._Q([0.1, 0.2, 0.3], [0, 0, 0], 3)
    none = Q.Clamp(-(2**31), 2**31 - 1)
    cases = [
        (dict(xt=Q.INT32, xq=qz), "QNN_ERR_QPARAM"),    # int32 input needs zp 0
        (dict(count=10, channels=3, xq=qc), "QNN_ERR_SHAPE"),
        (dict(count=12, channels=4, xq=qc), "QNN_ERR_QPARAM"),
        (dict(yt=5), "QNN_ERR_DTYPE"),
        (dict(x=None), "QNN_ERR_NULL"),
        (dict(act=Q.Clamp(200, 100)), "QNN_ERR_QPARAM"),
    ]
    for kw, expect in cases:
        a = dict(x=FAKE, xt=Q.UINT8, count=12, channels=3, xq=q1, y=FAKE, yt=Q.UINT8, yq=q1, act=none,
                 rnd=Q.HALF_UP)
        a.update(kw)
        st = L.qnn_requantize(None, a["x"], a["xt"], a["count"], a["channels"], a["xq"].q, a["y"], a["yt"],
                              a["yq"].q, a["act"], a["rnd"])
        assert Q.STATUS[st] == expect, (kw, L.qnn_last_error())
    # add: per-tensor only, 8-bit only
    st = L.qnn_add(None, FAKE, Q.UINT8, qc.q, FAKE, Q.UINT8, q1.q, 12, FAKE, Q.UINT8, q1.q, none, 0)
    assert Q.STATUS[st] == "QNN_ERR_QPARAM"
    st = L.qnn_add(None, FAKE, Q.INT32, q1.q, FAKE, Q.UINT8, q1.q, 12, FAKE, Q.UINT8, q1.q, none, 0)
    assert Q.STATUS[st] == "QNN_ERR_DTYPE"
    st = L.qnn_add(None, None, Q.UINT8, q1.q, FAKE, Q.UINT8, q1.q, 12, FAKE, Q.UINT8, q1.q, none, 0)
    assert Q.STATUS[st] == "QNN_ERR_NULL"
    st = L.qnn_add(None, None, Q.UINT8, q1.q, None, Q.UINT8, q1.q, 0, None, Q.UINT8, q1.q, none, 0)
    assert Q.STATUS[st] == "QNN_OK"     # count 0: no-op


def test_plan_null_handling(Q):
    L = Q.lib()
    assert Q.STATUS[L.qnn_plan_run(None, None, FAKE, FAKE, None)] == "QNN_ERR_NULL"
    assert L.qnn_plan_workspace_size(None) == 0
    assert L.qnn_plan_describe(None) == b""
    L.qnn_plan_destroy(None)
    st = L.qnn_conv2d_plan_create(None, None, Q.UINT8, 1, 8, 8, 16, Q._Q(0.1, 0, 1).q, FAKE, 8, 3, 3,
                                  Q._Q(0.1, 0, 1).q, None, Q.ConvParams(1, 1, 1, 1, 1, 1, 1, 1), Q.UINT8,
                                  Q._Q(0.1, 0, 1).q, Q.Clamp(0, 255), 0, 8, 0)
    assert Q.STATUS[st] == "QNN_ERR_NULL"


def test_dense_and_depthwise_validation(Q):
    L = Q.lib()
    q1 = Q._Q(0.1, 0, 1)
    none = Q.Clamp(-(2**31), 2**31 - 1)
    st = L.qnn_dense(None, FAKE, Q.UINT8, 16, 64, q1.q, FAKE, 32, q1.q, None, FAKE, Q.INT8, q1.q, none, 0, 16)
    assert Q.STATUS[st] == "QNN_ERR_SHAPE"      # y_ldc < Nd
    st = L.qnn_dense(None, FAKE, Q.UINT8, -1, 64, q1.q, FAKE, 32, q1.q, None, FAKE, Q.INT8, q1.q, none, 0, 32)
    assert Q.STATUS[st] == "QNN_ERR_SHAPE"
    st = L.qnn_depthwise_conv2d(None, FAKE, Q.UINT8, 1, 8, 8, 16, q1.q, FAKE, 3, 3, Q._Q([0.1] * 8, [0] * 8, 8).q,
                                None, Q.ConvParams(1, 1, 1, 1, 1, 1, 1, 1), FAKE, Q.UINT8, q1.q, none, 0, 16, 0)
    assert Q.STATUS[st] == "QNN_ERR_QPARAM"     # 8 weight scales for 16 channels


def test_tuning_file_paths(Q, tmp_path):
    """The kernel-choice file: a missing file starts empty, a readable one
    is parsed, an unreadable path is an error, None switches it off."""
    missing = tmp_path / "none.txt"
    Q.set_tuning_file(str(missing))
    assert not missing.exists()          # nothing is written before a plan is timed
    f = tmp_path / "tune.txt"
    f.write_text("conv:x0:n1:h8 2 4\nconv:x1:n1:h8 3 1\ngarbage\n")
    Q.set_tuning_file(str(f))
    with pytest.raises(Q.QnnError) as e:
        Q.set_tuning_file(str(f / "below_a_file"))
    assert e.value.status_name == "QNN_ERR_UNSUPPORTED"
    Q.set_tuning_file(None)
