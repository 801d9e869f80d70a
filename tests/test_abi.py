"""The C ABI on the CPU: the library loads, exports every function include/lce.h declares, and
rejects invalid arguments before it touches the GPU. No case here passes validation, so nothing
is ever launched (the pointers below are never dereferenced)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lce.h")

OK, INVALID, UNSUPPORTED, WS_SMALL, HIP = 0, 1, 2, 3, 4
BF16, FP32, FP16 = 1, 0, 2
NONE, MEAN, SUM = 0, 1, 2
FAKE = ctypes.c_void_p(0x1000)  # non-null, never dereferenced: every call below fails validation


@pytest.fixture(scope="module")
def lib():
    from paper_2603_16428_amd import lce
    return lce.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lce_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert names == sorted(["lce_workspace_size", "lce_plan_info", "lce_auto_chunk_tokens", "lce_forward",
                            "lce_forward_no_alloc",
                            "lce_forward_backward", "lce_rmsnorm_workspace_size", "lce_rmsnorm_forward",
                            "lce_rmsnorm_forward_backward", "lce_host_adam_step", "lce_head_train_step",
                            "lce_timing_enable",
                            "lce_timing_read", "lce_status_string"])
    for n in names:
        assert hasattr(lib, n), n


def test_binding_names_match_header():
    from paper_2603_16428_amd import lce
    assert sorted(lce.EXPORTED) == _declared_functions()


def test_status_strings(lib):
    for code, name in [(0, b"LCE_OK"), (1, b"LCE_ERR_INVALID_ARGUMENT"), (2, b"LCE_ERR_UNSUPPORTED"),
                       (3, b"LCE_ERR_WORKSPACE_TOO_SMALL"), (4, b"LCE_ERR_HIP"), (99, b"LCE_ERR_UNKNOWN")]:
        assert lib.lce_status_string(code) == name


def test_workspace_size(lib):
    ws = lib.lce_workspace_size
    assert ws(0, 8, 8, BF16, 1, 0) == 0
    assert ws(8, 0, 8, BF16, 1, 0) == 0
    assert ws(8, 8, 0, BF16, 1, 0) == 0
    assert ws(8, 8, 8, 7, 1, 0) == 0
    assert ws(8, 12, 8, BF16, 1, 0) == 0          # H not a multiple of 8 for bf16
    assert ws(8, 12, 8, FP16, 1, 0) == 0          # nor for fp16
    assert ws(8, 12, 8, FP32, 1, 0) > 0           # fine for fp32
    assert ws(8, 16, 8, FP16, 1, 0) == ws(8, 16, 8, BF16, 1, 0) > 0  # same 2-byte layout
    assert ws(300, 64, 100, BF16, 1, 100) == 0    # chunk must be a multiple of 64 when < N
    # a chunk's blocked copy of X_c (128 bytes per token at H = 64 in bf16) must stay below 2^31 bytes
    assert ws(2 ** 24 - 64, 64, 256, BF16, 1, 2 ** 24 - 64) > 0
    assert ws(2 ** 24, 64, 256, BF16, 1, 2 ** 24) == 0
    fwd = ws(8192, 4096, 128256, BF16, 0, 0)
    bwd = ws(8192, 4096, 128256, BF16, 1, 0)
    assert 0 < fwd < bwd
    # The workspace is O(n_c*V + V*H + N*H): at a fixed chunk size, doubling N adds only N*H-sized
    # buffers, never another N*V of logits.
    a = ws(8192, 4096, 128256, BF16, 1, 4096)
    b = ws(16384, 4096, 128256, BF16, 1, 4096)
    assert 0 < b - a <= 8192 * 4096 * 2 + 8192 * 64
    assert lib.lce_auto_chunk_tokens(8192, 4096, 128256, BF16) == 4096
    # Qwen: min(H, N/2) = 3584 would give five chunks, above bf16's carry limit of four; four chunks
    # of 4096 cost 156 MB more e buffer instead of a 2.18 GB fp32 accumulator. fp16's limit is 9.
    assert lib.lce_auto_chunk_tokens(16384, 3584, 152064, BF16) == 4096
    assert lib.lce_auto_chunk_tokens(16384, 3584, 152064, FP16) == 3584
    assert lib.lce_auto_chunk_tokens(4096, 12288, 32768, BF16) == 2048
    assert lib.lce_auto_chunk_tokens(37, 72, 1000, BF16) == 37  # one chunk
    # Forward only: one chunk up to 16384 tokens (per-slice partials, no logits-shaped buffer).
    one = ws(8192, 4096, 128256, BF16, 0, 8192)
    assert fwd == one
    assert ws(8192, 4096, 128256, BF16, 0, 4096) < one < bwd / 4
    assert ws(40000, 4096, 128256, BF16, 0, 0) == ws(40000, 4096, 128256, BF16, 0, 16384)


def _fwd(lib, **kw):
    a = dict(hidden=FAKE, weight=FAKE, labels=FAKE, N=16, H=64, V=100, dtype=BF16, ignore=-100,
             red=MEAN, loss=FAKE, lse=None, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return lib.lce_forward(a["hidden"], a["weight"], a["labels"], a["N"], a["H"], a["V"], a["dtype"],
                           a["ignore"], a["red"], a["loss"], a["lse"], a["ws"], a["wsb"], a["stream"])


def _fb(lib, **kw):
    a = dict(hidden=FAKE, weight=FAKE, labels=FAKE, N=16, H=64, V=100, dtype=BF16, ignore=-100,
             red=MEAN, loss=FAKE, dh=FAKE, dw=FAKE, chunk=0, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return lib.lce_forward_backward(a["hidden"], a["weight"], a["labels"], a["N"], a["H"], a["V"],
                                    a["dtype"], a["ignore"], a["red"], a["loss"], a["dh"], a["dw"],
                                    a["chunk"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(hidden=None), INVALID), (dict(weight=None), INVALID), (dict(labels=None), INVALID),
    (dict(loss=None), INVALID), (dict(N=0), INVALID), (dict(H=-1), INVALID), (dict(V=0), INVALID),
    (dict(dtype=5), INVALID), (dict(dtype=3), INVALID), (dict(red=3), INVALID), (dict(H=60), UNSUPPORTED),
    (dict(dtype=FP16, H=60), UNSUPPORTED),
    (dict(ws=None), WS_SMALL), (dict(wsb=16), WS_SMALL),
])
def test_forward_validation(lib, kw, status):
    assert _fwd(lib, **kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dh=None), INVALID), (dict(dw=None), INVALID), (dict(red=NONE), INVALID),
    (dict(red=7), INVALID), (dict(chunk=-1), INVALID), (dict(N=300, chunk=100), INVALID),
    (dict(H=20), UNSUPPORTED), (dict(wsb=0), WS_SMALL), (dict(ws=None), WS_SMALL),
])
def test_forward_backward_validation(lib, kw, status):
    assert _fb(lib, **kw) == status


# ---- the RMSNorm variant -------------------------------------------------------------------------

def test_rmsnorm_workspace_size(lib):
    ws = lib.lce_rmsnorm_workspace_size
    assert ws(0, 8, 8, BF16, 1, 0) == 0
    assert ws(8, 12, 8, BF16, 1, 0) == 0           # same shape rules as the plain step
    assert ws(65535 * 64, 8, 8, BF16, 1, 64) > 0   # rows of 64 per backward block: grid y <= 65535
    assert ws(65535 * 64 + 1, 8, 8, BF16, 1, 64) == 0
    assert ws(65535 * 64 + 1, 8, 8, BF16, 0, 64) > 0
    base = lib.lce_workspace_size(8192, 4096, 128256, BF16, 1, 0)
    extra = ws(8192, 4096, 128256, BF16, 1, 0) - base
    # x [N,H] bf16, dX [N,H] fp32, one chunk's fp32 dH partials (4096 x 4096 here), r and s [N],
    # ceil(N/64) x H fp32 partials (+ alignment): O(N H), no N x V.
    top = 8192 * 4096 * (2 + 4) + 4096 * 4096 * 4 + 2 * 8192 * 4 + 128 * 4096 * 4 + 8 * 256
    assert 8192 * 4096 * 6 <= extra <= top
    fwd = ws(8192, 4096, 128256, BF16, 0, 0) - lib.lce_workspace_size(8192, 4096, 128256, BF16, 0, 0)
    assert 8192 * 4096 * 2 <= fwd < extra


def _rfwd(lib, **kw):
    a = dict(hidden=FAKE, gamma=FAKE, weight=FAKE, labels=FAKE, N=16, H=64, V=100, dtype=BF16, eps=1e-5,
             ignore=-100, red=MEAN, loss=FAKE, lse=None, normed=None, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return lib.lce_rmsnorm_forward(a["hidden"], a["gamma"], a["weight"], a["labels"], a["N"], a["H"], a["V"],
                                   a["dtype"], a["eps"], a["ignore"], a["red"], a["loss"], a["lse"], a["normed"],
                                   a["ws"], a["wsb"], a["stream"])


def _rfb(lib, **kw):
    a = dict(hidden=FAKE, gamma=FAKE, weight=FAKE, labels=FAKE, N=16, H=64, V=100, dtype=BF16, eps=1e-5,
             ignore=-100, red=MEAN, loss=FAKE, dh=FAKE, dg=FAKE, dw=FAKE, chunk=0, ws=FAKE, wsb=1 << 30,
             stream=None)
    a.update(kw)
    return lib.lce_rmsnorm_forward_backward(a["hidden"], a["gamma"], a["weight"], a["labels"], a["N"], a["H"],
                                            a["V"], a["dtype"], a["eps"], a["ignore"], a["red"], a["loss"],
                                            a["dh"], a["dg"], a["dw"], a["chunk"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(gamma=None), INVALID), (dict(hidden=None), INVALID), (dict(eps=-1.0), INVALID),
    (dict(eps=float("nan")), INVALID), (dict(eps=float("inf")), INVALID), (dict(red=3), INVALID),
    (dict(H=60), UNSUPPORTED), (dict(wsb=16), WS_SMALL),
])
def test_rmsnorm_forward_validation(lib, kw, status):
    assert _rfwd(lib, **kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(dg=None), INVALID), (dict(dh=None), INVALID), (dict(dw=None), INVALID), (dict(red=NONE), INVALID),
    (dict(eps=-0.5), INVALID), (dict(H=20), UNSUPPORTED), (dict(wsb=0), WS_SMALL),
])
def test_rmsnorm_forward_backward_validation(lib, kw, status):
    assert _rfb(lib, **kw) == status


# ---- the output-layer training step ---------------------------------------------------------------

def _head(lib, **kw):
    from paper_2603_16428_amd import lce as L
    cfg = kw.pop("cfg", L.AdamConfig(1e-3, 0.9, 0.999, 1e-8, 0.0))
    a = dict(hidden=FAKE, labels=FAKE, N=16, H=64, V=100, dtype=BF16, ignore=-100, red=MEAN, chunk=0, w=FAKE,
             dh=FAKE, dw=FAKE, loss=FAKE, master=FAKE, m=FAKE, v=FAKE, gh=FAKE, ph=FAKE, step=1, blocks=4,
             threads=0, overlap=1, ws=FAKE, wsb=1 << 30, stream=None)
    a.update(kw)
    return lib.lce_head_train_step(a["hidden"], a["labels"], a["N"], a["H"], a["V"], a["dtype"], a["ignore"],
                                   a["red"], a["chunk"], a["w"], a["dh"], a["dw"], a["loss"], a["master"], a["m"],
                                   a["v"], a["gh"], a["ph"], ctypes.byref(cfg), a["step"], a["blocks"], a["threads"],
                                   a["overlap"], a["ws"], a["wsb"], a["stream"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(master=None), INVALID), (dict(gh=None), INVALID), (dict(ph=None), INVALID), (dict(step=0), INVALID),
    (dict(blocks=0), INVALID), (dict(blocks=257), INVALID), (dict(threads=-1), INVALID), (dict(red=NONE), INVALID),
    (dict(dtype=FP32), UNSUPPORTED), (dict(dtype=9), INVALID), (dict(H=60), UNSUPPORTED), (dict(wsb=8), WS_SMALL),
])
def test_head_train_step_validation(lib, kw, status):
    assert _head(lib, **kw) == status


def test_head_train_step_rejects_bad_optimizer_settings(lib):
    from paper_2603_16428_amd import lce as L
    for cfg in (L.AdamConfig(-1e-3, 0.9, 0.999, 1e-8, 0.0), L.AdamConfig(1e-3, 1.0, 0.999, 1e-8, 0.0),
                L.AdamConfig(1e-3, 0.9, 0.999, 0.0, 0.0), L.AdamConfig(1e-3, 0.9, 0.999, 1e-8, -0.5)):
        assert _head(lib, cfg=cfg) == INVALID


def test_gpu_parity_cases_cover_every_path():
    """The whole-oracle GPU parity cases (tests/test_gpu_parity.py) reach every way the backward can
    run, by the library's own plan: for each dtype, a dH contraction that stores its rows directly
    (one chunk, and several with dW added to across chunks) and one split over the vocabulary;
    for the 16-bit types, dW carried across chunks in fp32; and a chunk count at each carry limit."""
    import test_gpu_parity as gp
    from paper_2603_16428_amd import lce
    import torch
    dt = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32}
    cases = [(N, H, V, d, c) for N, H, V, d, c in gp.RAGGED + gp.NAN_WS]
    cases += [(N, H, V, d, c) for N, H, V, d, c, _ in gp.UNSPLIT]
    cases += [(16384, 4096, 4096, "bf16", c) for c in (4096, 1024, 0)]   # test_many_chunks_llama_width
    cases += [(4096, 1024, 4096, "fp16", c) for c in (512, 256)]         # test_many_chunks_fp16
    seen = set()
    for N, H, V, d, c in cases:
        p = lce.plan_info(N, H, V, dt[d], True, c)
        seen.add((d, "unsplit" if p["dh_splits"] == 1 else "split", "1 chunk" if p["chunks"] == 1 else "chunks",
                  "fp32 carry" if p["dw_fp32_carry"] else "own carry"))
    for d in ("bf16", "fp16", "fp32"):
        assert (d, "unsplit", "1 chunk", "own carry") in seen, d
        assert (d, "unsplit", "chunks", "own carry") in seen, d
        assert (d, "split", "chunks", "own carry") in seen, d
    for d in ("bf16", "fp16"):
        assert any(k[0] == d and k[3] == "fp32 carry" for k in seen), d
    # The full-size workloads run unsplit (Llama, Qwen) and split (Mistral-Large).
    assert lce.plan_info(8192, 4096, 128256, torch.bfloat16)["dh_splits"] == 1
    assert lce.plan_info(16384, 3584, 152064, torch.bfloat16)["dh_splits"] == 1
    assert lce.plan_info(4096, 12288, 32768, torch.bfloat16)["dh_splits"] > 1


def test_plan_info(lib):
    from paper_2603_16428_amd import lce
    info = lce.PlanInfo()
    assert lib.lce_plan_info(8, 8, 8, BF16, 1, 0, None) == INVALID
    assert lib.lce_plan_info(0, 8, 8, BF16, 1, 0, ctypes.byref(info)) == INVALID
    assert lib.lce_plan_info(8, 12, 8, BF16, 1, 0, ctypes.byref(info)) == UNSUPPORTED
    for args in [(8192, 4096, 128256, BF16, 1, 0), (8192, 4096, 128256, BF16, 0, 0), (300, 136, 4099, FP32, 1, 64),
                 (16384, 4096, 4096, BF16, 1, 1024), (65536, 4096, 128256, FP16, 1, 0)]:
        assert lib.lce_plan_info(*args, ctypes.byref(info)) == OK
        assert info.workspace_bytes == lib.lce_workspace_size(*args)
        assert info.chunks == -(-args[0] // info.chunk_tokens)
        if args[4]:
            assert info.chunk_tokens == (args[5] or lib.lce_auto_chunk_tokens(*args[:4]))
            assert 0 < info.fallback_flags_offset and info.fallback_flags_offset + 4 * info.chunks <= info.workspace_bytes
        else:
            assert info.dh_splits == 0 and info.fallback_flags_offset == 0
    # The fp32 carry costs V x H fp32 of workspace.
    assert lib.lce_plan_info(16384, 4096, 4096, BF16, 1, 1024, ctypes.byref(info)) == OK and info.dw_fp32_carry == 1
    with_acc = info.workspace_bytes
    assert lib.lce_plan_info(16384, 4096, 4096, BF16, 1, 4096, ctypes.byref(info)) == OK and info.dw_fp32_carry == 0
    assert lib.lce_workspace_size(16384, 4096, 4096, FP32, 1, 1024) > 0
    assert with_acc - lib.lce_workspace_size(16384, 4096, 4096, BF16, 1, 4096) >= 4096 * 4096 * 4 - 3 * 1024 * 4096 * 2


def test_no_alloc_forward_rejects_before_launching(lib):
    # Invalid arguments as for lce_forward; sizes whose workspace cannot fit the static scratch even
    # at 64 tokens per chunk: LCE_ERR_WORKSPACE_TOO_SMALL, decided on the host before any HIP call.
    f = lib.lce_forward_no_alloc
    assert f(None, FAKE, FAKE, 8, 8, 8, BF16, -100, MEAN, FAKE, None, None) == INVALID
    assert f(FAKE, FAKE, FAKE, 8, 8, 8, BF16, -100, 7, FAKE, None, None) == INVALID
    assert f(FAKE, FAKE, FAKE, 8, 12, 8, BF16, -100, MEAN, FAKE, None, None) == UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, 8 << 20, 4096, 128256, BF16, -100, MEAN, FAKE, None, None) == WS_SMALL
    assert f(FAKE, FAKE, FAKE, 4096, 1 << 20, 256, BF16, -100, MEAN, FAKE, None, None) == WS_SMALL
