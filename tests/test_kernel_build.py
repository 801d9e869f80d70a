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

# Element types: bf16 (DF16b), fp16 (DF16_), fp32 (f).
TYPES = ("DF16b", "DF16_", "f")
# gemm_kernel (both operands through LDS): the dH GEMM (epilogue 2, A K-contiguous, B MN-contiguous).
LDS_GEMMS = [f"_ZN3lce11gemm_kernelI{t}Li2ELb0ELb1ELb0EEEvNS_8GemmArgsE" for t in TYPES]
# gemm_xb_kernel (B from a blocked copy, straight to registers): (epilogue, A MN-contiguous, per-chunk
# K check) of the logits GEMMs (forward / backward, with and without the K check) and dW.
XB_VARIANTS = [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1), (3, 1, 0)]
XB_GEMMS = [f"_ZN3lce14gemm_xb_kernelI{t}Li{e}ELb{a}ELb{c}EEEvNS_8GemmArgsE" for t in TYPES for e, a, c in XB_VARIANTS]
GEMMS = LDS_GEMMS + XB_GEMMS


@pytest.fixture(scope="module")
def asm():
    with tempfile.TemporaryDirectory() as d:
        cmd = [B.HIPCC] + [f for f in B.FLAGS if f != "-shared"] + ["-c", "--save-temps"] + B.KERNEL_SOURCES + \
              ["-o", os.path.join(d, "lce.o")]
        r = subprocess.run(cmd, cwd=d, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        files = [f for f in os.listdir(d) if f.endswith(".s") and "gfx950" in f]
        assert files, os.listdir(d)
        return open(os.path.join(d, files[0])).read()


def _main_loop(asm_text, name, with_prologue=False):
    # The K-loop: the innermost loop (gemm_xb_kernel runs it inside a loop over tiles).
    start = asm_text.index(name + ":")
    end = asm_text.index(".Lfunc_end", start)
    body = asm_text[start:end].splitlines()
    depth = max(int(m.group(1)) for l in body for m in [re.search(r"Loop Header: Depth=(\d+)", l)] if m)
    lo = next(i for i, l in enumerate(body) if f"Loop Header: Depth={depth}" in l)
    # The loop's back edge: the branch to the header's label (the body may hold other branches).
    label = next(body[i].split(":")[0].strip() for i in range(lo, -1, -1) if re.match(r"^\.LBB\w+:", body[i]))
    hi = next(i for i, l in enumerate(body) if i > lo and re.match(r"\s*s_(c)?branch\S*\s+" + re.escape(label) + r"\s*$", l))
    if with_prologue:
        lo = 0
    return [l.strip() for l in body[lo:hi + 1] if l.strip() and not l.strip().startswith(";")]


@pytest.mark.parametrize("name", GEMMS)
def test_gemm_pipeline_fill_has_no_scratch_traffic(asm, name):
    # The prologue's waits are hand-counted too: no spill traffic from the kernel's start to the
    # end of the main loop.
    code = _main_loop(asm, name, with_prologue=True)
    scratch = [l for l in code if l.startswith("scratch_") or re.match(r"buffer_(load|store)\S*\s.*\boff\b", l)]
    assert not scratch, scratch[:4]


@pytest.mark.parametrize("name", GEMMS)
def test_gemm_main_loop_has_no_scratch_traffic(asm, name):
    loop = _main_loop(asm, name)
    scratch = [l for l in loop if l.startswith("scratch_") or re.match(r"buffer_(load|store)\S*\s.*\boff\b", l)]
    assert not scratch, scratch[:4]
    mfma = [l for l in loop if l.startswith("v_mfma")]
    dma = [l for l in loop if l.startswith("buffer_load") and l.endswith("lds")]
    vload = [l for l in loop if l.startswith("buffer_load") and not l.endswith("lds")]
    writes = [l for l in loop if l.startswith("ds_write")]
    tr = [l for l in loop if l.startswith("ds_read_b64_tr_b16")]
    # Two K-tiles per loop trip: 2 x 64 MFMA steps (x4 for fp32's 32x32x2). gemm_kernel: 2 x 8 loads
    # of each kind, B written to LDS. gemm_xb_kernel: A by LDS-DMA (2 x 8), B fragments straight to
    # registers (2 x 16), nothing written to LDS.
    assert len(mfma) == (128 if "DF16" in name else 512), len(mfma)
    xb = name in XB_GEMMS
    if xb:
        assert len(dma) == 16 and len(vload) == 32 and len(writes) == 0, (len(dma), len(vload), len(writes))
    else:
        assert len(dma) == 16 and len(vload) == 16 and len(writes) == 16
    # MN-contiguous 16-bit operands read from LDS: 2 transposing reads per fragment x 4 fragments per
    # K-pair x 4 K-pairs per K-tile x 2 K-tiles.
    flags = [int(f[0]) for f in name.split("ELb")[1:]]
    n_mn = flags[0] if xb else flags[0] + flags[1]
    assert len(tr) == (2 * 4 * 4 * 2 * n_mn if "DF16" in name else 0), len(tr)


# ---- LDS layout model: the index formulas of the GEMM loaders and fragment reads -------------
# These restate, in Python, the per-lane formulas of gemm_kernel (Operand::init / offset /
# fragment) and check that every fragment read finds the element the loader put there.

def _swz_k(r):
    return (r ^ (r >> 3)) & 7


def _swz_mn(k):
    return (4 if k & 1 else 0) ^ (10 if k & 2 else 0) ^ (16 if k & 8 else 0)


def test_k_contiguous_layout_model():
    ld = 1000  # any pitch (elements); bf16
    stored = {}  # LDS byte -> (row, k) element index of its first bf16
    for w in range(4):
        for j in range(8):
            for lane in range(64):
                row_off = (64 * w + (lane >> 3)) * ld * 2
                slot_x = ((lane & 7) ^ (lane >> 3)) << 4
                off = row_off + j * 8 * ld * 2 + (slot_x ^ (j << 4))
                row, kbyte = divmod(off, ld * 2)
                lds = (8 * w + j) * 1024 + lane * 16
                stored[lds] = (row, kbyte // 2)
    for wsub in (0, 128):
        for i in range(4):
            for lane in range(64):
                sw = _swz_k(i * 32 + (lane & 31))
                for p in range(4):
                    c = 2 * p + (lane >> 5)
                    lds = (wsub + 32 * i + (lane & 31)) * 128 + ((c ^ sw) << 4)
                    assert stored[lds] == (wsub + 32 * i + (lane & 31), 8 * c)


def test_mn_contiguous_bf16_layout_model():
    ld = 4096
    stored = {}  # LDS byte -> (k-row, column) of its first bf16
    for w in range(4):
        for j in range(8):
            for lane in range(64):
                row_off = (16 * w + (lane >> 5)) * ld * 2
                slot_x = ((lane & 31) ^ (4 * (lane >> 5))) << 4
                xj = ((10 if j & 1 else 0) ^ (16 if (j >> 2) & 1 else 0)) << 4
                off = row_off + j * 2 * ld * 2 + (slot_x ^ xj)
                kr, cbyte = divmod(off, ld * 2)
                lds = (8 * w + j) * 1024 + lane * 16
                assert kr == 2 * (8 * w + j) + (lane >> 5)
                for e in range(8):
                    stored[lds + 2 * e] = (kr, cbyte // 2 + e)
    conflicts = 0
    for wsub in (0, 128):
        g_ = [lane >> 4 for lane in range(64)]
        for i in range(4):
            for p in range(4):
                for s in range(2):
                    got, addrs = {}, []
                    for lane in range(64):
                        g, ip = lane >> 4, lane & 15
                        r0 = 8 * (g >> 1) + (ip >> 2)
                        col = wsub + 16 * (g & 1) + 4 * (ip & 3)
                        frag0 = r0 * 512 + (((col >> 3) ^ _swz_mn(r0)) << 4) + 8 * ((col >> 2) & 1)
                        a = (frag0 ^ (i << 6)) + (16 * p + 4 * s) * 512
                        addrs.append(a)
                        got[lane] = [stored[a + 2 * e] for e in range(4)]   # 4 consecutive columns
                    for lane in range(64):   # the transposed delivery of ds_read_b64_tr_b16
                        g, jj = lane >> 4, lane & 15
                        recv = [got[16 * g + 4 * e + jj // 4][jj % 4] for e in range(4)]
                        k0 = 16 * p + 8 * (lane >> 5) + 4 * s
                        assert recv == [(k0 + e, wsub + 32 * i + (lane & 31)) for e in range(4)]
                    for nb, grp in ((32, 16), (64, 32)):
                        for g0 in range(0, 64, grp):
                            banks = [((a // 4) + b) % nb for a in addrs[g0:g0 + grp] for b in (0, 1)]
                            conflicts += len(banks) - len(set(banks))
    assert conflicts == 0


# ---- Blocked operand B of gemm_xb_kernel: the two blocking kernels and the GEMM's loads ---------
# Restated from block_k_kernel, block_mn_kernel and gemm_xb_kernel's load_b: both blocking kernels
# must put element (n, k) at the same byte, and the GEMM's B load for K-pair q of column block jb
# must hand lane l the column and the K bytes that the A fragment of the same lane covers (K-pair
# q = 4 t + p of K-tile t, lane half h: bytes [32 q + 16 h, +16) of the row).

def _blocked_from_k(N, K, esz, KP, NB):
    out = {}  # byte -> (n, k) of the element there, or None for padding
    for frag in range(NB * KP):
        jb, q = divmod(frag, KP)
        for l in range(64):
            n, k = 32 * jb + (l & 31), (32 * q + 16 * (l >> 5)) // esz
            for e in range(16 // esz):
                out[frag * 1024 + l * 16 + e * esz] = (n, k + e) if (n < N and k < K) else None
    return out


def _blocked_from_mn(N, K, esz, KP, NB):
    vec, rows, pieces = 16 // esz, 128 // esz, 32 // (16 // esz)
    out = {}
    for jb in range(NB):
        for grp in range((KP + 3) // 4):
            tile = {}
            for t in range(256):   # staging: thread t loads row t / pieces, piece t % pieces
                r, pc = divmod(t, pieces)
                k, n = grp * rows + r, 32 * jb + pc * vec
                for e in range(vec):
                    tile[(r, pc * vec + e)] = (n + e, k) if (k < K and n < N) else None
            for t in range(256):   # gather: thread t writes lane t % 64 of fragment 4 grp + t / 64
                q = grp * 4 + (t >> 6)
                if q >= KP:
                    continue
                l = t & 63
                kr = (t >> 6) * (32 // esz) + (l >> 5) * vec
                for e in range(vec):
                    out[(jb * KP + q) * 1024 + l * 16 + e * esz] = tile[(kr + e, l & 31)]
    return out


def _check_definition(layout, N, K, esz, KP, NB):
    # Every element of B appears once, at the byte the layout defines; everything else is padding.
    placed = [v for v in layout.values() if v is not None]
    assert sorted(placed) == sorted((n, k) for n in range(N) for k in range(K))
    for byte, v in layout.items():
        if v is not None:
            frag, rem = divmod(byte, 1024)
            l, off = divmod(rem, 16)
            jb, q = divmod(frag, KP)
            assert v == (32 * jb + (l & 31), (32 * q + 16 * (l >> 5) + off) // esz)


@pytest.mark.parametrize("N,K,esz", [(70, 200, 2), (33, 40, 4)])
def test_blocked_from_k_ragged_columns(N, K, esz):
    # block_k_kernel (logits GEMM: columns = tokens, any count; K = H, whole 16-byte pieces).
    KP = -(-(K * esz) // 128) * 128 // 32
    NB = -(-N // 32)
    _check_definition(_blocked_from_k(N, K, esz, KP, NB), N, K, esz, KP, NB)


@pytest.mark.parametrize("N,K,esz", [(72, 37, 2), (36, 13, 4)])
def test_blocked_from_mn_ragged_k(N, K, esz):
    # block_mn_kernel (dW GEMM: columns = H, whole 16-byte pieces; K = tokens, any count).
    KP = -(-(K * esz) // 128) * 128 // 32
    NB = -(-N // 32)
    _check_definition(_blocked_from_mn(N, K, esz, KP, NB), N, K, esz, KP, NB)


# N and K as both kernels require (whole 16-byte pieces on both axes), so that both apply.
@pytest.mark.parametrize("N,K,esz", [(72, 200, 2), (64, 256, 2), (36, 40, 4), (96, 72, 4), (8, 8, 2)])
def test_blocked_operand_layout_model(N, K, esz):
    KP = -(-(K * esz) // 128) * 128 // 32
    NB = -(-N // 32)
    a = _blocked_from_k(N, K, esz, KP, NB)
    b = _blocked_from_mn(N, K, esz, KP, NB)
    assert a == b
    _check_definition(a, N, K, esz, KP, NB)
    # The GEMM's B loads (wave column blocks jb0 .. jb0 + 3, split starting at K-pair q0 = 0).
    for jb in range(NB):
        for q in range(KP):
            soff = (jb * KP + q) * 1024
            for l in range(64):
                got = [a[soff + l * 16 + e * esz] for e in range(16 // esz)]
                t, p = divmod(q, 4)
                h = l >> 5
                kbytes = 128 * t + 32 * p + 16 * h          # the A fragment's K bytes for this lane
                want = [(32 * jb + (l & 31), kbytes // esz + e) for e in range(16 // esz)]
                assert [g for g in got if g is not None] == [w for w in want if w[0] < N and w[1] < K]
