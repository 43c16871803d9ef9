"""qnn_plan_run_timed: the same bytes as qnn_plan_run, and the two events
that the main kernel records at its own start and end give a positive
duration no longer than events bracketing the whole call."""
import pytest
import torch

import workloads as W
from gpu_util import Q, assert_equal, dev, log, make_plan

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["s14b1_3x3", "stem7x7s2"])
def test_timed_run_matches_and_times_the_kernel(name):
    layer = [l for l in W.resnet50() if l.name == name][0]
    c = W.conv_case(layer, 2, seed=9)
    p, keep = make_plan(c)
    x = dev(c.x)
    ref = p.run(x)
    out = torch.empty_like(ref)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    o1, o2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    o1.record()
    p.run_timed(x, out, None, a, b)
    o2.record()
    torch.cuda.synchronize()
    k, outer = a.elapsed_time(b), o1.elapsed_time(o2)
    log(f"{name}: kernel {k * 1e3:.2f} us, bracketed call {outer * 1e3:.2f} us ({p.describe()})")
    assert 0.0 < k <= outer * 1.05 + 1e-3
    assert_equal(out.cpu().numpy(), ref.cpu().numpy(), name)
    p.close()


def test_timed_run_rejects_requantize_plans():
    p = Q.requantize_plan((64,), "u8", 0.1, 3, 0.2, 5)
    x = torch.zeros(64, dtype=torch.uint8, device="cuda")
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with pytest.raises(Q.QnnError):
        p.run_timed(x, torch.empty_like(x), None, a, b)
    p.close()
