"""Replays of a captured HIP graph against eager runs.  bench.py times
steps replayed from one graph; these tests capture the same steps (its
plans, tensors, split reductions with their arrival counters, fused
residual adds, one-shot adds and pools) and check, byte for byte, that
every replay writes what the eager run wrote, with eager work, output
scribbles and synchronizations between the replays."""
import os
import shutil

import pytest
import torch

from gpu_util import log

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _capture(items):
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for it in items:
                it.run()
    torch.cuda.synchronize()
    return g


def _check_replays(items, outs, what, reps=3):
    """outs: name -> tensor written by the step.  The eager run is the
    reference; each replay follows a scribble over every output and an
    eager run of the first step."""
    for it in items:
        it.run()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in outs.items()}
    g = _capture(items)
    for rep in range(reps):
        for v in outs.values():
            v.fill_(90)
        items[0].run()   # the program's own eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k, v in outs.items():
            assert torch.equal(v, ref[k]), f"{what}: replay {rep}, tensor {k}"
    log(f"{what}: {len(items)} steps, {len(outs)} tensors, {reps} replays equal to the eager run")


@pytest.mark.parametrize("workload", ["resnet50_b1_chain", "mobilenet_v2_b1_chain", "inception_v3_mixed5_b1_chain"])
def test_chain_replays(workload):
    import bench
    t = {}
    items, _ = bench.setup_chain(workload, fuse=True, tensors=t)
    outs = {k: v for k, v in t.items() if k != "x0"}
    _check_replays(items, outs, workload)


@pytest.mark.parametrize("workload", ["resnet50_b1", "dense_bert"])
def test_layer_set_replays(workload):
    """Independent layers as bench.py times them (split reductions among
    the batch-1 choices), each with its own workspace."""
    import bench
    items, _ = bench.setup(workload)
    outs = {f"{i}:{it.name}": it.out for i, it in enumerate(items)}
    splits = sum(1 for it in items if "ksplit" in getattr(it, "desc", ""))
    log(f"{workload}: {splits} plans in the split form")
    _check_replays(items, outs, workload)


@pytest.mark.parametrize("workload", ["resnet50_b32", "mobilenet_v2_b64"])
def test_benchmark_replays(workload, tmp_path):
    """The benchmark stacks with their committed kernel choices, set up as
    bench.py sets them up."""
    import bench
    from paper_2006_10226_amd import qnn as Q
    path = tmp_path / "choices.txt"
    shutil.copy(os.path.join(ROOT, bench.CHOICE_FILES[workload]), path)
    Q.set_tuning_file(str(path))
    try:
        items, _ = bench.setup(workload)
        outs = {f"{i}:{it.name}": it.out for i, it in enumerate(items)}
        _check_replays(items, outs, workload, reps=2)
    finally:
        Q.set_tuning_file(None)
