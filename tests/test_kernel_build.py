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
# gemm_xb_kernel (B blocked, straight to registers): (epilogue, A layout 0 K-contiguous / 1 MN-
# contiguous / 2 blocked, per-chunk K check) of the logits GEMMs (forward / backward, with and
# without the K check), dH and dW.
XB_VARIANTS = [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1), (2, 1, 0), (3, 2, 0)]
GEMMS = [f"_ZN3lce14gemm_xb_kernelI{t}Li{e}ELi{a}ELb{c}EEEvNS_8GemmArgsE" for t in TYPES for e, a, c in XB_VARIANTS]


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
    # Two K-tiles per loop trip: 2 x 64 MFMA steps (x4 for fp32's 32x32x2); A by LDS-DMA (2 x 8), B
    # fragments straight to registers (2 x 16), nothing written to LDS.
    assert len(mfma) == (128 if "DF16" in name else 512), len(mfma)
    assert len(dma) == 16 and len(vload) == 32 and len(writes) == 0, (len(dma), len(vload), len(writes))
    # A in the MN-contiguous LDS layout (MN-contiguous or blocked), 16-bit: 2 transposing reads per
    # fragment x 4 fragments per K-pair x 4 K-pairs per K-tile x 2 K-tiles.
    layout = int(name.split("ELi")[1][0])
    assert len(tr) == (2 * 4 * 4 * 2 if "DF16" in name and layout > 0 else 0), len(tr)


# ---- LDS layout model: the index formulas of the GEMM loaders and fragment reads -------------
# These restate, in Python, the per-lane formulas of operand A's loader (Operand::init / offset /
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
# Restated from block_k_block, block_mn_block and gemm_xb_kernel's load_b: both blocking kernels
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
    # block_k_block (logits GEMM: columns = tokens, any count; K = H, whole 16-byte pieces).
    KP = -(-(K * esz) // 128) * 128 // 32
    NB = -(-N // 32)
    _check_definition(_blocked_from_k(N, K, esz, KP, NB), N, K, esz, KP, NB)


@pytest.mark.parametrize("N,K,esz", [(72, 37, 2), (36, 13, 4)])
def test_blocked_from_mn_ragged_k(N, K, esz):
    # block_mn_block (dW GEMM: columns = H, whole 16-byte pieces; K = tokens, any count).
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


# ---- Blocked operand A (dZ of the dW GEMM) and the writers of e / dZ ----------------------------
# Restated from Operand::init / rsrc (A_BLK), the LSE epilogue's blocked store and dlogits_block.

def _blocked_decode(off, KP, esz):
    # Byte offset into the blocked buffer -> (column = token, first K element = vocabulary id).
    jb, rem = divmod(off, KP * 1024)
    q, r = divmod(rem, 1024)
    lf, b = divmod(r, 16)
    assert b == 0
    return 32 * jb + (lf & 31), (32 * q + 16 * (lf >> 5)) // esz


@pytest.mark.parametrize("KP", [32, 16032])
def test_blocked_a_fp32_loader_fetches_the_mn_loaders_pieces(KP):
    # fp32 blocked A: relative to the K-tile's first token and the tile's first id, load j of wave
    # w, lane l must fetch the piece (K-row, ids) that the MN-contiguous loader puts in the same
    # LDS slot, inside the descriptor's range (the tile's ids in the K-tile's one token block).
    esz = 4
    for w in range(4):
        for j in range(8):
            for lane in range(64):
                off = 8 * w * 16 + j * 16 + (lane << 9)
                assert _blocked_decode(off, KP, esz) == (8 * w + j, 4 * lane)
                assert off + 16 <= 256 * esz * 32


@pytest.mark.parametrize("KP", [16, 8016])
def test_blocked_a_16bit_loads_whole_fragments(KP):
    # 16-bit blocked A: each load reads one whole fragment (1 KB, contiguous), slot 8w + j holds
    # fragment (w/2, 8 (w%2) + j), and with one token block left in the K-tile the descriptor's
    # range (the tile's ids in that block) takes exactly the first block's loads.
    esz, tile_bytes = 2, 256 * 2 * 32
    for w in range(4):
        for j in range(8):
            offs = []
            for lane in range(64):
                slot_x = (lane ^ (4 * (lane >> 5))) << 4
                offs.append((w >> 1) * KP * 1024 + (w & 1) * 8192 + j * 1024 + (slot_x ^ (128 if j & 1 else 0)))
            base = (w >> 1) * KP * 1024 + (8 * (w & 1) + j) * 1024
            assert sorted(offs) == list(range(base, base + 1024, 16))
            assert all((o + 16 <= tile_bytes) == (w < 2) for o in offs)


@pytest.mark.parametrize("esz", [2, 4])
def test_lse_epilogue_stores_e_blocked(esz):
    # The LSE_BWD epilogue: for block (i, j) of the wave at (mw, nw), lane l's token is column
    # nw + 32 j + l%32 and its piece of each fragment of that token block is at l * 16.
    KP = 64 if esz == 2 else 128
    for mw, nw in ((0, 0), (128, 128), (768, 224)):
        for j in range(4):
            for i in range(4):
                for lane in range(64):
                    h = lane >> 5
                    tok = nw + 32 * j + (lane & 31)
                    e_blk = ((nw + 32 * j) >> 5) * KP * 1024 + lane * 16
                    if esz == 2:
                        # after regroup32: ids 8h .. and 16 + 8h .. of the 32-id segment
                        lo = e_blk + ((mw + 32 * i) >> 4) * 1024
                        assert _blocked_decode(lo, KP, esz) == (tok, mw + 32 * i + 8 * h)
                        assert _blocked_decode(lo + 1024, KP, esz) == (tok, mw + 32 * i + 16 + 8 * h)
                    else:
                        for q in range(4):
                            off = e_blk + ((mw + 32 * i + 8 * q) >> 3) * 1024
                            assert _blocked_decode(off, KP, esz) == (tok, mw + 32 * i + 8 * q + 4 * h)


@pytest.mark.parametrize("esz", [2, 4])
def test_dlogits_pieces(esz):
    # dlogits_job: block (b, jb), wave w, lane l, piece k -- its token and ids, and the claim
    # that the four pieces of a lane lie in one 128-id slice; the grid writes every piece once.
    KP, NB = 32 if esz == 2 else 64, 3
    seen = set()
    for jb in range(NB):
        for b in range(KP // 16):
            for w in range(4):
                for lane in range(64):
                    q0 = 16 * b + 4 * w
                    v0 = (q0 * 32 + 16 * (lane >> 5)) // esz
                    slices = set()
                    for k in range(4):
                        off = (jb * KP + q0) * 1024 + lane * 16 + k * 1024
                        v = v0 + k * (32 // esz)
                        assert _blocked_decode(off, KP, esz) == (32 * jb + (lane & 31), v)
                        slices |= {(v + e) // 128 for e in range(16 // esz)}
                        seen.add(off)
                    assert len(slices) == 1 and slices == {v0 // 128}
    assert seen == set(range(0, NB * KP * 1024, 16))


def test_blocked_a_16bit_lds_layout_model():
    # 16-bit blocked A: whole-fragment loads with a piece permutation, and the transposing fragment
    # reads (as in test_mn_contiguous_bf16_layout_model): every lane must receive the four tokens
    # of its id that the MFMA expects, with no LDS bank conflicts.
    KP, esz = 64, 2
    stored = {}   # LDS byte -> (token, id) of its first bf16, relative to the K-tile and the tile
    for w in range(4):
        for j in range(8):
            row_off = (w >> 1) * KP * 1024 + (w & 1) * 8192
            for lane in range(64):
                slot_x = (lane ^ (4 * (lane >> 5))) << 4
                off = row_off + j * 1024 + (slot_x ^ (128 if j & 1 else 0))
                tok, idx = _blocked_decode(off, KP, esz)
                lds = (8 * w + j) * 1024 + lane * 16
                for e in range(8):
                    stored[lds + 2 * e] = (tok, idx + e)
    assert len(stored) == 32 * 1024 // 2
    conflicts = 0
    for wsub in (0, 128):
        for i in range(4):
            for p in range(4):
                for s in range(2):
                    got, addrs = {}, []
                    for lane in range(64):
                        g, ip = lane >> 4, lane & 15
                        h = (ip & 3) >> 1
                        frag0 = (wsub // 16 + (g & 1)) * 1024 + 16 * ((ip >> 2) + 4 * h + 8 * ((g >> 1) ^ (g & 1)) + 32 * h) + 8 * (ip & 1)
                        a = ((frag0) ^ (64 * s)) + 16384 * (p >> 1) + 256 * (p & 1) + 2048 * i
                        addrs.append(a)
                        got[lane] = [stored[a + 2 * e] for e in range(4)]   # 4 consecutive ids of a token
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


# ---- aux_kernel: several bandwidth-bound jobs in one launch -----------------------------------
# Restated from aux_kernel's dispatch: block b runs the first job whose range holds it, at its index
# within that range; block_mn's range is its old (NB, ceil(KP / 4)) grid with the column block
# fastest; prepare's last block (index ceil(N / 4)) is the counting block.

def _aux_dispatch(counts, b):
    for job, n in counts:
        if b < n:
            return job, b
        b -= n
    return None, None


@pytest.mark.parametrize("N,NB,KPm,with_dl,with_loss", [(8192, 128, 256, True, False), (37, 3, 4, False, True),
                                                        (1, 1, 1, True, True), (2048, 64, 64, False, False)])
def test_aux_job_partition(N, NB, KPm, with_dl, with_loss):
    prep = (N + 3) // 4 + 1
    bk = (NB * KPm * 64 + 255) // 256
    bmn = NB * ((KPm + 3) // 4)
    dl = 7 if with_dl else 0
    loss = 1 if with_loss else 0
    counts = [("prep", prep), ("bk", bk), ("bmn", bmn), ("dl", dl), ("loss", loss)]
    seen = {job: [] for job, _ in counts}
    total = sum(n for _, n in counts)
    for b in range(total):
        job, i = _aux_dispatch(counts, b)
        seen[job].append(i)
    assert _aux_dispatch(counts, total) == (None, None)
    for job, n in counts:
        assert seen[job] == list(range(n)), job
    grid = sorted((i % NB, i // NB) for i in seen["bmn"])
    assert grid == sorted((jb, g) for jb in range(NB) for g in range((KPm + 3) // 4))
    # prepare: token blocks of four tokens, then the counting block
    assert [i for i in seen["prep"] if i * 4 >= N] == [prep - 1]
