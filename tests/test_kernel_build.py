"""Build invariants of the gfx950 code object, checked on the CPU from the compiler's own
assembly of this repository's kernels.

The GEMM main loops wait for their global->LDS and global->register loads with hand-counted
`s_waitcnt vmcnt(N)`. Scratch (register-spill) loads and stores also count in vmcnt, so a spill
inside a main loop would let those waits pass early and the MFMAs read stale LDS. Every GEMM
kernel's main loop must therefore be free of scratch instructions, and must contain the MFMA and
load mix the kernel is designed around.
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2603_16428_amd import build as B

GEMMS = [f"_ZN3lce11gemm_kernelI{t}Li{e}EEEvNS_8GemmArgsE" for t in ("DF16b", "f") for e in range(4)]


@pytest.fixture(scope="module")
def asm():
    with tempfile.TemporaryDirectory() as d:
        cmd = [B.HIPCC] + [f for f in B.FLAGS if f != "-shared"] + ["-c", "--save-temps"] + B.SOURCES + \
              ["-o", os.path.join(d, "lce.o")]
        r = subprocess.run(cmd, cwd=d, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        files = [f for f in os.listdir(d) if f.endswith(".s") and "gfx950" in f]
        assert files, os.listdir(d)
        return open(os.path.join(d, files[0])).read()


def _main_loop(asm_text, name):
    start = asm_text.index(name + ":")
    end = asm_text.index(".Lfunc_end", start)
    body = asm_text[start:end].splitlines()
    lo = next(i for i, l in enumerate(body) if "Loop Header" in l)
    hi = next(i for i, l in enumerate(body) if i > lo and "s_cbranch" in l)
    return [l.strip() for l in body[lo:hi + 1] if l.strip() and not l.strip().startswith(";")]


@pytest.mark.parametrize("name", GEMMS)
def test_gemm_main_loop_has_no_scratch_traffic(asm, name):
    loop = _main_loop(asm, name)
    scratch = [l for l in loop if l.startswith("scratch_") or re.match(r"buffer_(load|store)\S*\s.*\boff\b", l)]
    assert not scratch, scratch[:4]
    mfma = [l for l in loop if l.startswith("v_mfma")]
    dma = [l for l in loop if l.startswith("buffer_load") and l.endswith("lds")]
    vload = [l for l in loop if l.startswith("buffer_load") and not l.endswith("lds")]
    writes = [l for l in loop if l.startswith("ds_write")]
    # Two K-tiles per loop trip: 2 x 64 MFMA steps (x4 for fp32's 32x32x2), 2 x 8 loads of each kind.
    assert len(mfma) == (128 if "DF16b" in name else 512), len(mfma)
    assert len(dma) == 16 and len(vload) == 16 and len(writes) == 16
