"""Full-tensor GPU parity of the benchmark configurations: every output
byte of all 53 ResNet-50 conv layers at batch 32 (the inputs bench.py
times, seeds 3000 + layer), with the kernels the committed choice file
names (the same ones bench.py and its profiles run), against the full
oracle (conv accumulator of Eq. (2) plus bias, requantize of Eq. (5));
and every output byte of the MobileNet-V2 b64 and Inception-v3 b64
workloads, set up by bench.py's own layer list."""
import os
import shutil

import pytest
import torch

import workloads as W
from gpu_util import O, Q, assert_equal, dev, log, make_plan, run_oracle

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHOICES = os.path.join(ROOT, "workloads", "choices", "resnet50_b32.txt")


@pytest.fixture()
def committed_choices(tmp_path):
    if not os.path.exists(CHOICES):
        pytest.skip("no committed kernel choices")
    path = tmp_path / "choices.txt"
    shutil.copyfile(CHOICES, path)   # shapes timed anew are appended to the copy
    Q.set_tuning_file(str(path))
    yield path
    Q.set_tuning_file(None)


def test_resnet50_batch32_every_byte(committed_choices):
    timed = 0
    for i, layer in enumerate(W.resnet50()):
        c = W.conv_case(layer, 32, seed=3000 + i)
        p, keep = make_plan(c)
        d = p.describe()
        y = p.run(dev(c.x))
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        p.close()
        log(f"resnet50 b32 {layer.name}: {d}")
        assert_equal(y, run_oracle(c), f"{layer.name} ({d})")
        del c, y
    # every layer found its kernel in the committed file (none was timed)
    appended = len(open(committed_choices).read().splitlines()) - len(open(CHOICES).read().splitlines())
    assert appended == timed, f"{appended} layer shapes were missing from {CHOICES}"


@pytest.fixture()
def mobilenet_choices(tmp_path):
    src = os.path.join(ROOT, "workloads", "choices", "mobilenet_v2_b64.txt")
    if not os.path.exists(src):
        pytest.skip("no committed kernel choices")
    path = tmp_path / "choices.txt"
    shutil.copyfile(src, path)
    Q.set_tuning_file(str(path))
    yield path
    Q.set_tuning_file(None)


def _every_byte(workload):
    import bench
    layers, _ = bench._layers(workload)
    for kind, layer, c in layers:
        if kind == "add":
            y = Q.add(dev(c.a), c.s_a, c.zp_a, dev(c.b), c.s_b, c.zp_b, c.s_o, c.zp_o, c.yt, c.act,
                      c.rounding).cpu().numpy()
            ref = O.add(c.a, c.s_a, c.zp_a, c.b, c.s_b, c.zp_b, c.s_o, c.zp_o, c.yt, c.act, c.rounding)
            assert_equal(y, ref, c.name)
            continue
        p, keep = make_plan(c)
        d = p.describe()
        y = p.run(dev(c.x))
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        p.close()
        log(f"{workload} {layer.name}: {d}")
        assert_equal(y, run_oracle(c), f"{layer.name} ({d})")
        del c, y


def test_mobilenet_v2_batch64_every_byte(mobilenet_choices):
    _every_byte("mobilenet_v2_b64")


def test_inception_v3_batch64_every_byte():
    _every_byte("inception_v3_b64")
