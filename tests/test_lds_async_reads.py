"""The kernels that read LDS with inline assembly retire every such read
before its registers are touched, on every control-flow path (checked on
the gfx950 assembly the compiler produces; no GPU needed)."""
import os
import re
import shutil
import subprocess

import pytest

import lds_hazards as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2006_10226_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _kernel(text):
    return H.kernels("_Zkernel:\n" + text + "\n.Lfunc_end0:\n")["_Zkernel"]


def test_checker_flags_use_before_wait():
    k = _kernel("""
    ds_read_b128 v[2:5], v10
    v_add_u32_e32 v3, 1, v3
    s_endpgm""")
    assert len(H.hazards(k)) == 1


def test_checker_accepts_wait_before_use():
    k = _kernel("""
    ds_read_b128 v[2:5], v10
    ds_read_b128 v[6:9], v10
    s_waitcnt lgkmcnt(1)
    v_add_u32_e32 v3, 1, v3
    s_waitcnt lgkmcnt(0)
    v_add_u32_e32 v7, 1, v7
    s_endpgm""")
    assert H.hazards(k) == {}


def test_checker_follows_a_branch_around_the_wait():
    # the taken branch skips the wait: the use after the label is a hazard
    k = _kernel("""
    ds_read_b128 v[2:5], v10
    s_cbranch_scc1 .LBB0_2
    s_waitcnt lgkmcnt(0)
.LBB0_2:
    v_mov_b32_e32 v4, 0
    s_endpgm""")
    assert len(H.hazards(k)) == 1


def test_checker_scalar_loads_void_partial_waits():
    # a scalar load may return first, so lgkmcnt(1) does not retire the read
    k = _kernel("""
    ds_read_b128 v[2:5], v10
    s_load_dword s4, s[0:1], 0x0
    s_waitcnt lgkmcnt(1)
    v_mov_b32_e32 v2, 0
    s_endpgm""")
    assert len(H.hazards(k)) == 1


def test_checker_loop_carried_read():
    # a read issued at the bottom of a loop is still pending at the top
    k = _kernel("""
.LBB0_1:
    v_mov_b32_e32 v3, 0
    ds_read_b128 v[2:5], v10
    s_cbranch_scc1 .LBB0_1
    s_waitcnt lgkmcnt(0)
    s_endpgm""")
    assert len(H.hazards(k)) == 1


_SOURCES = ["conv_dma.hip", "conv_dma_fused.hip", "conv_tap.hip", "conv_wave.hip", "conv_halo.hip", "conv_window.hip"]
_ASM = {}


def _asm(src, tmp_path_factory):
    """gfx950 assembly of one source; the first call compiles every source
    these tests read, side by side."""
    if not _ASM:
        d = tmp_path_factory.mktemp("asm")
        procs = {}
        for name in _SOURCES:
            cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "--cuda-device-only", "-S", "-O3", "-std=c++17",
                   "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                   "-mllvm", "-disable-promote-alloca-to-lds", os.path.join(CSRC, name),
                   "-o", str(d / (name + ".s"))]
            procs[name] = subprocess.Popen(cmd, stdout=subprocess.DEVNULL, stderr=subprocess.PIPE, text=True)
        for name, p in procs.items():
            err = p.communicate()[1]
            assert p.returncode == 0, err[-2000:]
            _ASM[name] = (d / (name + ".s")).read_text()
    return _ASM[src]


needs_hipcc = pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not available")


@needs_hipcc
@pytest.mark.parametrize("src", ["conv_dma.hip", "conv_dma_fused.hip", "conv_wave.hip"])
def test_kernels_retire_async_lds_reads(src, tmp_path_factory):
    ks = H.kernels(_asm(src, tmp_path_factory))
    assert len(ks) > 0
    bad = {name: H.hazards(lines) for name, lines in ks.items()}
    bad = {k: v for k, v in bad.items() if v}
    assert not bad, {k[:80]: sorted(v.items())[:3] for k, v in bad.items()}


@needs_hipcc
@pytest.mark.parametrize("src", _SOURCES)
def test_counted_wait_kernels_use_no_scratch(src, tmp_path_factory):
    # These kernels wait for their staged loads with explicit counts of
    # outstanding vector-memory operations; a register spill would add
    # scratch loads and stores to that count and release a wait early.
    text = _asm(src, tmp_path_factory)
    sizes = re.findall(r"^\s*\.amdhsa_kernel\s+(\S+)|\.amdhsa_private_segment_fixed_size\s+(\d+)", text, re.M)
    kernels, name = {}, None
    for k, size in sizes:
        if k:
            name = k
        elif name is not None:
            kernels[name] = int(size)
            name = None
    assert kernels
    spilled = {k[:100]: v for k, v in kernels.items() if v}
    assert not spilled, spilled
