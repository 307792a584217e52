"""Rules for the gfx950 code that hipcc generates for the HIP library (CPU only: the device
code is cross-compiled to assembly here, nothing runs).

* M0 is written only by the direct-to-LDS load helpers, each time right before the load
  that uses it.  Their inline assembly clobbers M0, which the compiler reserves and cannot
  save around an asm statement, so no other instruction may rely on it.
* No packed fp32 vector instructions (the build turns them off).
* No writes through the scalar data cache: scalar stores, scalar atomics, its write-back
  or discard.
"""
from __future__ import annotations

import concurrent.futures
import os
import re
import subprocess
import tempfile

import pytest

from paper_2503_08467_amd import build as B

SOURCES = sorted(f for f in B.sources() if f.endswith(".hip"))


def _device_asm(src: str, outdir: str) -> list:
    out = os.path.join(outdir, os.path.basename(src) + ".s")
    flags = [f for f in B.HIPCC_FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [B.hipcc(), *flags, "--cuda-device-only", "-S", "-I", os.path.join(B.ROOT, "include"), "-o", out, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    insts = []
    for line in open(out):
        t = line.split(";", 1)[0].strip()
        if not t or t.startswith(".") or t.endswith(":"):
            continue
        insts.append(t)
    return insts


@pytest.fixture(scope="module")
def asm():
    try:
        B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    with tempfile.TemporaryDirectory() as d:
        with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
            return dict(zip(SOURCES, ex.map(lambda s: _device_asm(s, d), SOURCES)))


def test_m0_only_feeds_direct_lds_loads(asm):
    m0 = re.compile(r"\bm0\b")
    # the pipelined GEMM and the route kernel do load through M0 (the check is not vacuous)
    for name in ("ffn.hip", "route.hip"):
        insts = next(v for k, v in asm.items() if k.endswith(name))
        assert sum(t.startswith("global_load_lds_") for t in insts) > 0, name
    for src, insts in asm.items():
        for i, t in enumerate(insts):
            if not m0.search(t):
                continue
            assert re.fullmatch(r"s_mov_b32 m0, s\d+", t), f"{os.path.basename(src)}: {t}"
            assert i + 1 < len(insts) and insts[i + 1].startswith("global_load_lds_"), \
                f"{os.path.basename(src)}: M0 set but not used by the next instruction: {insts[i + 1:i + 2]}"


def test_no_packed_fp32(asm):
    bad = re.compile(r"^v_pk_(fma|mul|add)_f32\b")
    for src, insts in asm.items():
        hits = [t for t in insts if bad.match(t)]
        assert not hits, f"{os.path.basename(src)}: {hits[:3]}"


def test_no_scalar_cache_writes(asm):
    bad = re.compile(r"^(s_store|s_buffer_store|s_scratch_store|s_atomic|s_buffer_atomic|s_dcache_wb|"
                     r"s_dcache_discard)")
    for src, insts in asm.items():
        hits = [t for t in insts if bad.match(t)]
        assert not hits, f"{os.path.basename(src)}: {hits[:3]}"
