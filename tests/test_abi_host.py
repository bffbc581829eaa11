"""Host-only checks of the C ABI: the library loads, exports every declared symbol
and rejects invalid arguments before any HIP call (no kernel is launched here)."""
import ctypes
import os
import re

import pytest

from paper_2607_08779_amd import ssq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssq.h")

EINVAL, EALIGN, ESCRATCH = -1, -2, -4
COUNTERS = 65536                    # fixed arrival-counter region at the front of a workspace
P16 = ctypes.c_void_p(1 << 20)      # aligned dummy pointers: never dereferenced, because
P2 = ctypes.c_void_p((1 << 20) + 2)  # every call below fails validation first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssq_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == ["ssq_export_gguf", "ssq_gguf_block_bytes",
                                    "ssq_matmul", "ssq_matmul_f32", "ssq_matmul_min",
                                    "ssq_matmul_min_f32", "ssq_matmul_min_ws",
                                    "ssq_matmul_noalloc", "ssq_matmul_q8", "ssq_matmul_q8_min",
                                    "ssq_matmul_workspace_size", "ssq_matmul_ws",
                                    "ssq_quantize", "ssq_quantize_act_q8",
                                    "ssq_quantize_diag", "ssq_quantize_diag_f32",
                                    "ssq_quantize_f32", "ssq_quantize_min", "ssq_quantize_min_f32",
                                    "ssq_sign_diagnostics", "ssq_sign_diagnostics_f32",
                                    "ssq_strerror"]


def test_library_exports_every_declared_symbol():
    lib = ssq.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_strerror_never_null():
    for st in (0, -1, -2, -3, -4, 7, -99):
        assert isinstance(ssq.ssq_strerror(st), str) and ssq.ssq_strerror(st)


@pytest.mark.parametrize("args", [
    dict(q=5), dict(q=1), dict(group=16), dict(group=48), dict(mode=3), dict(mode=-1),
    dict(cols=48), dict(rows=-1), dict(cols=-32), dict(mode=2),          # ASYM without zp
    dict(zp=P16),                                                         # zp with a sym mode
    dict(W=None), dict(codes=None), dict(scales=None),
])
def test_quantize_rejects_invalid_arguments(args):
    a = dict(W=P16, rows=4, cols=64, group=32, q=4, mode=0, codes=P16, scales=P16, zp=None)
    a.update(args)
    for fn in (ssq.lib().ssq_quantize, ssq.lib().ssq_quantize_f32):
        assert fn(a["W"], a["rows"], a["cols"], a["group"], a["q"], a["mode"], a["codes"],
                  a["scales"], a["zp"]) == EINVAL


@pytest.mark.parametrize("which", ["W", "codes", "scales"])
def test_quantize_rejects_misaligned_pointers(which):
    a = dict(W=P16, codes=P16, scales=P16)
    a[which] = ctypes.c_void_p((1 << 20) + (1 if which == "scales" else 8))
    st = ssq.lib().ssq_quantize(a["W"], 4, 64, 32, 4, 0, a["codes"], a["scales"], None)
    assert st == EALIGN


def test_quantize_empty_is_a_noop():
    for rows, cols in ((0, 64), (4, 0), (0, 0)):
        assert ssq.lib().ssq_quantize(None, rows, cols, 32, 4, 0, None, None, None) == 0


@pytest.mark.parametrize("args", [
    dict(K=0), dict(K=48), dict(K=-32), dict(K=(1 << 22) + 32), dict(M=-1), dict(N=-1), dict(q=8),
    dict(group=96),
    dict(x=None), dict(codes=None), dict(scales=None), dict(y=None),
])
def test_matmul_rejects_invalid_arguments(args):
    a = dict(x=P16, M=2, codes=P16, scales=P16, zp=None, N=8, K=64, group=32, q=4, y=P16)
    a.update(args)
    for fn in (ssq.lib().ssq_matmul, ssq.lib().ssq_matmul_f32):
        assert fn(a["x"], a["M"], a["codes"], a["scales"], a["zp"], a["N"], a["K"], a["group"],
                  a["q"], a["y"], None) == EINVAL


@pytest.mark.parametrize("which", ["x", "codes", "y", "scales"])
def test_matmul_rejects_misaligned_pointers(which):
    a = dict(x=P16, codes=P16, y=P16, scales=P16)
    a[which] = P2 if which != "scales" else ctypes.c_void_p((1 << 20) + 1)
    st = ssq.lib().ssq_matmul(a["x"], 2, a["codes"], a["scales"], None, 8, 64, 32, 4, a["y"], None)
    assert st == EALIGN


def test_matmul_empty_is_a_noop():
    for M, N in ((0, 8), (2, 0)):
        assert ssq.lib().ssq_matmul(None, M, None, None, None, N, 64, 32, 4, None, None) == 0


def test_workspace_size_rules():
    lib = ssq.lib()
    # M=512 x N=4096 has 64 output tiles of 256x128, too few for 256 CUs: split 4 ways
    n = lib.ssq_matmul_workspace_size(512, 4096, 14336, 32, 4)
    assert n == COUNTERS + 64 * 4 * 256 * 128 * 4      # fixed counter region + partials
    assert lib.ssq_matmul_workspace_size(2048, 4096, 14336, 32, 4) == 0   # one full round of 256 tiles
    assert lib.ssq_matmul_workspace_size(2048, 12288, 4096, 32, 4) == 0   # three full rounds
    # 896 tiles: three rounds, then the last 128 tiles cut in two K slices
    assert lib.ssq_matmul_workspace_size(2048, 14336, 4096, 32, 4) == COUNTERS + 128 * 2 * 256 * 128 * 4
    # 1088 tiles: four rounds, then 64 tiles cut four ways
    assert lib.ssq_matmul_workspace_size(2048, 17408, 5120, 32, 4) == COUNTERS + 64 * 4 * 256 * 128 * 4
    assert lib.ssq_matmul_workspace_size(512, 28672, 8192, 32, 4) == 0    # last round 3/4 full: kept
    assert lib.ssq_matmul_workspace_size(1, 4096, 14336, 32, 4) == 0      # GEMV never splits
    # batched decode: 32 row blocks of 128 rows, 16 slices of K, one 16-token block
    assert lib.ssq_matmul_workspace_size(16, 4096, 14336, 32, 4) == COUNTERS + 32 * 16 * 8 * 256 * 4
    assert lib.ssq_matmul_workspace_size(32, 4096, 14336, 32, 4) == COUNTERS + 32 * 16 * 8 * 512 * 4
    assert lib.ssq_matmul_workspace_size(512, 4096, 48, 32, 4) == 0       # invalid K
    assert lib.ssq_matmul_workspace_size(512, 4096, 256, 32, 4) == 0      # too few steps


def test_noalloc_rejects_problems_beyond_its_scratch():
    """ssq_matmul_noalloc refuses, before any HIP call, a split that needs more than its
    64 MiB static scratch: 131072 x 8192 at M = 16 needs 1024 row blocks x 8 slices of
    partials (exactly 64 MiB) plus the counter region."""
    lib = ssq.lib()
    need = lib.ssq_matmul_workspace_size(16, 131072, 8192, 32, 4)
    assert need == COUNTERS + (64 << 20)
    st = lib.ssq_matmul_noalloc(P16, 16, P16, P16, None, 131072, 8192, 32, 4, P16, None)
    assert st == ESCRATCH and "64 MiB" in ssq.ssq_strerror(st)
    # invalid arguments are still reported as such
    assert lib.ssq_matmul_noalloc(P16, 16, P16, P16, None, 8, 48, 32, 4, P16, None) == EINVAL
    assert lib.ssq_matmul_noalloc(P2, 16, P16, P16, None, 8, 64, 32, 4, P16, None) == EALIGN
    assert lib.ssq_matmul_noalloc(None, 0, None, None, None, 8, 64, 32, 4, None, None) == 0


def test_matmul_ws_rejects_misaligned_workspace():
    st = ssq.lib().ssq_matmul_ws(P16, 2, P16, P16, None, 8, 64, 32, 4, P16,
                                 ctypes.c_void_p((1 << 20) + 16), 1 << 20, None)
    assert st == EALIGN


def test_binding_fails_loudly_without_library(monkeypatch):
    monkeypatch.setattr(ssq, "LIB_PATH", "/nonexistent/libssq.so")
    monkeypatch.setattr(ssq, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        ssq.lib()


# ---------------------------------------------------------------------------
# The binary16-minimum entry points (App. B.1 Q*_1 layout).
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("args", [
    dict(q=5), dict(group=16), dict(cols=48), dict(rows=-1),
    dict(W=None), dict(codes=None), dict(scales=None), dict(mins=None),
])
def test_quantize_min_rejects_invalid_arguments(args):
    a = dict(W=P16, rows=4, cols=64, group=32, q=4, codes=P16, scales=P16, mins=P16)
    a.update(args)
    for fn in (ssq.lib().ssq_quantize_min, ssq.lib().ssq_quantize_min_f32):
        assert fn(a["W"], a["rows"], a["cols"], a["group"], a["q"], a["codes"], a["scales"],
                  a["mins"]) == EINVAL


def test_min_entry_points_reject_misaligned_minimums():
    odd = ctypes.c_void_p((1 << 20) + 1)
    assert ssq.lib().ssq_quantize_min(P16, 4, 64, 32, 4, P16, P16, odd) == EALIGN
    assert ssq.lib().ssq_matmul_min(P16, 2, P16, P16, odd, 8, 64, 32, 4, P16, None) == EALIGN
    assert ssq.lib().ssq_matmul_min_f32(P16, 2, P16, P16, odd, 8, 64, 32, 4, P16, None) == EALIGN
    assert ssq.lib().ssq_matmul_min_ws(P16, 2, P16, P16, odd, 8, 64, 32, 4, P16, None, 0, None) == EALIGN


@pytest.mark.parametrize("args", [dict(K=48), dict(M=-1), dict(q=8), dict(x=None), dict(mins=None)])
def test_matmul_min_rejects_invalid_arguments(args):
    a = dict(x=P16, M=2, codes=P16, scales=P16, mins=P16, N=8, K=64, group=32, q=4, y=P16)
    a.update(args)
    for fn in (ssq.lib().ssq_matmul_min, ssq.lib().ssq_matmul_min_f32):
        assert fn(a["x"], a["M"], a["codes"], a["scales"], a["mins"], a["N"], a["K"], a["group"],
                  a["q"], a["y"], None) == EINVAL
    assert ssq.lib().ssq_matmul_min_ws(a["x"], a["M"], a["codes"], a["scales"], a["mins"], a["N"],
                                       a["K"], a["group"], a["q"], a["y"], None, 0, None) == EINVAL


def test_min_entry_points_empty_is_a_noop():
    assert ssq.lib().ssq_quantize_min(None, 0, 64, 32, 4, None, None, None) == 0
    assert ssq.lib().ssq_matmul_min(None, 0, None, None, None, 8, 64, 32, 4, None, None) == 0
    assert ssq.lib().ssq_matmul_min_ws(None, 2, None, None, None, 0, 64, 32, 4, None, None, 0, None) == 0


@pytest.mark.parametrize("args", [
    dict(q=5), dict(group=16), dict(cols=48), dict(rows=-1),
    dict(W=None), dict(margin=None), dict(gain=None),
])
def test_sign_diagnostics_rejects_invalid_arguments(args):
    a = dict(W=P16, rows=4, cols=64, group=32, q=4, margin=P16, gain=P16, tally=P16)
    a.update(args)
    for fn in (ssq.lib().ssq_sign_diagnostics, ssq.lib().ssq_sign_diagnostics_f32):
        assert fn(a["W"], a["rows"], a["cols"], a["group"], a["q"], a["margin"], a["gain"],
                  a["tally"]) == EINVAL


def test_sign_diagnostics_alignment_and_empty():
    lib = ssq.lib()
    assert lib.ssq_sign_diagnostics(P16, 4, 64, 32, 4, P2, ctypes.c_void_p((1 << 20) + 2), None) == EALIGN
    assert lib.ssq_sign_diagnostics(P16, 4, 64, 32, 4, P16, P16, ctypes.c_void_p((1 << 20) + 4)) == EALIGN
    assert lib.ssq_sign_diagnostics(None, 0, 64, 32, 4, None, None, None) == 0


def test_binding_refuses_host_tensors():
    """A CPU tensor never reaches a kernel: the binding raises before any launch."""
    import torch
    W = torch.zeros((4, 64), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensors"):
        ssq.ssq_quantize(W, 32, 4, ssq.SIGNED_SYM)
    with pytest.raises(ValueError, match="GPU tensors"):
        ssq.ssq_sign_diagnostics(W, 32, 4)


@pytest.mark.parametrize("args,status", [
    (dict(K=48), EINVAL), (dict(M=-1), EINVAL), (dict(x=None), EINVAL), (dict(q=None), EINVAL),
    (dict(d=None), EINVAL), (dict(x=P2), EALIGN), (dict(q=P2), EALIGN),
    (dict(d=ctypes.c_void_p((1 << 20) + 1)), EALIGN),
])
def test_quantize_act_q8_rejects_invalid_arguments(args, status):
    a = dict(x=P16, M=2, K=64, q=P16, d=P16)
    a.update(args)
    assert ssq.lib().ssq_quantize_act_q8(a["x"], a["M"], a["K"], a["q"], a["d"], None) == status


def test_quantize_act_q8_empty_is_a_no_op():
    assert ssq.lib().ssq_quantize_act_q8(None, 0, 64, None, None, None) == 0


@pytest.mark.parametrize("args,status", [
    (dict(q=5), EINVAL), (dict(group=16), EINVAL), (dict(K=48), EINVAL), (dict(K=1 << 23), EINVAL),
    (dict(qx=None), EINVAL), (dict(dx=None), EINVAL), (dict(codes=None), EINVAL), (dict(y=None), EINVAL),
    (dict(qx=P2), EALIGN), (dict(codes=P2), EALIGN), (dict(dx=ctypes.c_void_p((1 << 20) + 1)), EALIGN),
])
def test_matmul_q8_rejects_invalid_arguments(args, status):
    a = dict(qx=P16, dx=P16, M=1, codes=P16, scales=P16, zp=None, N=4, K=64, group=32, q=4, y=P16)
    a.update(args)
    lib = ssq.lib()
    assert lib.ssq_matmul_q8(a["qx"], a["dx"], a["M"], a["codes"], a["scales"], a["zp"], a["N"], a["K"],
                             a["group"], a["q"], a["y"], None) == status
    assert lib.ssq_matmul_q8_min(a["qx"], a["dx"], a["M"], a["codes"], a["scales"], P16, a["N"], a["K"],
                                 a["group"], a["q"], a["y"], None) == status


def test_matmul_q8_min_requires_minimums():
    assert ssq.lib().ssq_matmul_q8_min(P16, P16, 1, P16, P16, None, 4, 64, 32, 4, P16, None) == EINVAL


@pytest.mark.parametrize("args,status", [
    (dict(q=5), EINVAL), (dict(group=16), EINVAL), (dict(cols=48), EINVAL), (dict(W=None), EINVAL),
    (dict(codes=None), EINVAL), (dict(margin=None), EINVAL), (dict(gain=None), EINVAL),
    (dict(W=P2), EALIGN), (dict(margin=ctypes.c_void_p((1 << 20) + 1)), EALIGN), (dict(gain=P2), EALIGN),
])
def test_quantize_diag_rejects_invalid_arguments(args, status):
    a = dict(W=P16, rows=4, cols=64, group=32, q=4, codes=P16, scales=P16, margin=P16, gain=P16)
    a.update(args)
    for fn in (ssq.lib().ssq_quantize_diag, ssq.lib().ssq_quantize_diag_f32):
        assert fn(a["W"], a["rows"], a["cols"], a["group"], a["q"], a["codes"], a["scales"], a["margin"],
                  a["gain"]) == status


@pytest.mark.parametrize("args,status", [
    (dict(q=3), EINVAL), (dict(q=5), EINVAL), (dict(group=16), EINVAL), (dict(cols=48), EINVAL),
    (dict(rows=-1), EINVAL), (dict(codes=None), EINVAL), (dict(scales=None), EINVAL), (dict(out=None), EINVAL),
    (dict(codes=P2), EALIGN), (dict(scales=ctypes.c_void_p((1 << 20) + 1)), EALIGN),
    (dict(out=ctypes.c_void_p((1 << 20) + 1)), EALIGN), (dict(mins=ctypes.c_void_p((1 << 20) + 1)), EALIGN),
])
def test_export_gguf_rejects_invalid_arguments(args, status):
    a = dict(codes=P16, scales=P16, mins=None, rows=4, cols=64, group=32, q=4, out=P16)
    a.update(args)
    assert ssq.lib().ssq_export_gguf(a["codes"], a["scales"], a["mins"], a["rows"], a["cols"], a["group"],
                                     a["q"], a["out"], None) == status


def test_export_gguf_block_sizes_and_empty():
    """Block sizes of App. B.1's formats table; an empty matrix is a no-op."""
    lib = ssq.lib()
    assert [lib.ssq_gguf_block_bytes(q, m) for q in (4, 2) for m in (0, 1)] == [18, 20, 10, 12]
    assert lib.ssq_gguf_block_bytes(3, 0) == 0
    assert lib.ssq_export_gguf(None, None, None, 0, 64, 32, 4, None, None) == 0
