"""C-ABI checks that need no GPU: the library loads, exports every function declared in
include/hsa.h, and rejects bad arguments before any launch with the documented codes."""
import ctypes
import os
import re

import pytest

import paper_2504_16795_amd as hsa
from paper_2504_16795_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUPPORTED, WS_SMALL = 0, 1, 2, 3


def declared_functions():
    src = open(os.path.join(ROOT, "include", "hsa.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hsa_\w+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    return hsa.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(binding.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def P(**kw):
    base = dict(B=2, L=256, H=16, G=2, d=128, S=64, k=8, dtype=hsa.HSA_DTYPE_BF16)
    base.update(kw)
    return hsa.make_params(**base)


FAKE = ctypes.c_void_p(0x10000)          # aligned, never dereferenced (rejected earlier)


def fwd(lib, p, Q=FAKE, ws=None, nb=0):
    return lib.hsa_forward(ctypes.byref(p), Q, FAKE, FAKE, FAKE, FAKE, FAKE, ws, nb, None)


@pytest.mark.parametrize("kw,code", [
    (dict(H=15), INVALID), (dict(G=0), INVALID), (dict(k=0), INVALID), (dict(S=0), INVALID),
    (dict(d=96), UNSUPPORTED), (dict(S=48), UNSUPPORTED), (dict(k=33), UNSUPPORTED),
    (dict(H=34, G=2), UNSUPPORTED), (dict(dtype=7), INVALID), (dict(B=-1), INVALID),
    (dict(dtype=hsa.HSA_DTYPE_F32, S=128, d=128), UNSUPPORTED),
])
def test_forward_rejects_bad_shapes(lib, kw, code):
    assert fwd(lib, P(**kw)) == code
    assert lib.hsa_attn_last_error().decode() != ""


def test_flags_reserved(lib):
    p = P()
    for bit in (4, 8, 1 << 31):
        p.flags = bit
        assert fwd(lib, p) == UNSUPPORTED
    p.flags = binding.HSA_FLAG_STICK_BREAKING | binding.HSA_FLAG_SOFTMAX_OFF_BY_ONE | 8
    assert fwd(lib, p) == UNSUPPORTED


@pytest.mark.parametrize("kw,flags", [
    (dict(stick_breaking=True), binding.HSA_FLAG_STICK_BREAKING),
    (dict(off_by_one=True), binding.HSA_FLAG_SOFTMAX_OFF_BY_ONE),
    (dict(stick_breaking=True, off_by_one=True),
     binding.HSA_FLAG_STICK_BREAKING | binding.HSA_FLAG_SOFTMAX_OFF_BY_ONE)])
def test_variant_flags_accepted(lib, kw, flags):
    """The stick-breaking and off-by-one flags pass validation: the call then fails on the
    NULL Q."""
    p = P(**kw)
    assert p.flags == flags
    assert fwd(lib, p, Q=None) == INVALID
    assert "Q" in lib.hsa_attn_last_error().decode()


def test_null_and_misaligned_pointers(lib):
    assert fwd(lib, P(), Q=None) == INVALID
    assert "Q" in lib.hsa_attn_last_error().decode()
    assert fwd(lib, P(), Q=ctypes.c_void_p(0x10004)) == INVALID
    assert "aligned" in lib.hsa_attn_last_error().decode()


def test_workspace_checks(lib):
    p = P()
    need = lib.hsa_attn_workspace_size(ctypes.byref(p), hsa.HSA_OP_BACKWARD)
    assert need > 0
    st = lib.hsa_backward(ctypes.byref(p), *([FAKE] * 10), FAKE, need - 1, None)
    assert st == WS_SMALL
    assert lib.hsa_attn_workspace_size(ctypes.byref(P(H=15)), hsa.HSA_OP_BACKWARD) == 0
    assert lib.hsa_attn_workspace_size(ctypes.byref(p), hsa.HSA_OP_DECODE) > 0
    assert lib.hsa_attn_workspace_size(ctypes.byref(p), hsa.HSA_OP_SELECT) == 0


def test_landmark_range_checks(lib):
    p = P()
    assert lib.hsa_landmarks(ctypes.byref(p), FAKE, FAKE, 0, 2, 1, None) == INVALID
    assert lib.hsa_landmarks(ctypes.byref(p), FAKE, FAKE, 0, 0, 5, None) == INVALID
    assert lib.hsa_landmarks(ctypes.byref(p), FAKE, FAKE, 3, 0, 4, None) == INVALID
    # empty range and empty batch are no-ops that launch nothing
    assert lib.hsa_landmarks(ctypes.byref(p), FAKE, FAKE, 0, 2, 2, None) == OK
    assert lib.hsa_landmarks(ctypes.byref(P(B=0)), None, None, 0, 0, 4, None) == OK


def test_decode_checks(lib):
    p = P(G=32, H=32)
    assert lib.hsa_decode(ctypes.byref(p), *([FAKE] * 4), 1, None, FAKE, FAKE, FAKE, FAKE,
                          1 << 20, None) == UNSUPPORTED
    p = P()
    assert lib.hsa_decode(ctypes.byref(p), *([FAKE] * 4), 5, None, FAKE, FAKE, FAKE, FAKE,
                          1 << 20, None) == INVALID


def test_status_strings(lib):
    for s in range(5):
        assert lib.hsa_attn_status_string(s)
    assert lib.hsa_attn_status_string(99) == b"unknown status"


def test_wide_selection_rows_only_for_selection_calls(lib):
    """Rows of 256 / 512 / 1024 columns are a selection over inputs of its own: accepted by
    the selection calls (one row per group, bf16), refused by the attention calls."""
    wide = P(H=2, G=2, d=1024)
    assert fwd(lib, wide) == UNSUPPORTED
    assert lib.hsa_attn_workspace_size(ctypes.byref(wide), hsa.HSA_OP_SELECT_BACKWARD) > 0
    assert lib.hsa_attn_workspace_size(ctypes.byref(wide), hsa.HSA_OP_BACKWARD) == 0
    # a NULL Q passes the shape checks first: INVALID, not UNSUPPORTED
    assert lib.hsa_select_topk(ctypes.byref(wide), None, FAKE, FAKE, FAKE, None, 0,
                               None) == INVALID
    for bad in (P(H=16, G=2, d=1024), P(H=2, G=2, d=1024, dtype=hsa.HSA_DTYPE_F32),
                P(H=2, G=2, d=384)):
        assert lib.hsa_select_topk(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, None, 0,
                                   None) == UNSUPPORTED


def test_backward_attn_and_select_backward_check_arguments(lib):
    p = P()
    n = lib.hsa_attn_workspace_size(ctypes.byref(p), hsa.HSA_OP_BACKWARD)
    ws = ctypes.c_void_p(0x20000)
    args = [FAKE] * 9
    # dw is required
    assert lib.hsa_backward_attn(ctypes.byref(p), *args, None, 0, ws, n, None) == INVALID
    assert "dw" in lib.hsa_attn_last_error().decode()
    assert lib.hsa_backward_attn(ctypes.byref(p), *args, FAKE, 0, ws, 16, None) == WS_SMALL
    sp = P(H=2, G=2, d=1024)
    m = lib.hsa_attn_workspace_size(ctypes.byref(sp), hsa.HSA_OP_SELECT_BACKWARD)
    assert lib.hsa_select_backward(ctypes.byref(sp), FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                                   ws, m, None) == INVALID
    assert "dw" in lib.hsa_attn_last_error().decode()
    assert lib.hsa_select_backward(ctypes.byref(sp), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                   ws, m - 1, None) == WS_SMALL


def test_kernel_path_hook(lib):
    """hsa_attn_set_path: per-op kernel-family override, validated, read back, restored."""
    from paper_2504_16795_amd import binding as B
    assert lib.hsa_attn_get_path(B.HSA_OP_FORWARD) == B.HSA_PATH_AUTO
    assert lib.hsa_attn_set_path(B.HSA_OP_FORWARD, B.HSA_PATH_CHUNK_MAJOR) == 0
    assert lib.hsa_attn_get_path(B.HSA_OP_FORWARD) == B.HSA_PATH_CHUNK_MAJOR
    assert lib.hsa_attn_get_path(B.HSA_OP_BACKWARD) == B.HSA_PATH_AUTO
    # a family the op has no kernel of, an op without families, an unknown path
    assert lib.hsa_attn_set_path(B.HSA_OP_BACKWARD, B.HSA_PATH_CHUNK_MAJOR) == 1
    assert lib.hsa_attn_set_path(B.HSA_OP_FORWARD, B.HSA_PATH_TWO_PASS) == 1
    assert lib.hsa_attn_set_path(B.HSA_OP_FORWARD, B.HSA_PATH_FUSED) == 1
    assert lib.hsa_attn_set_path(B.HSA_OP_BACKWARD, B.HSA_PATH_FUSED) == 0
    assert lib.hsa_attn_get_path(B.HSA_OP_BACKWARD) == B.HSA_PATH_FUSED
    assert lib.hsa_attn_set_path(B.HSA_OP_LANDMARKS, B.HSA_PATH_GENERIC) == 1
    assert lib.hsa_attn_set_path(B.HSA_OP_SELECT, 99) == 1
    assert lib.hsa_attn_set_path(-1, B.HSA_PATH_TWO_PASS) == 1
    assert lib.hsa_attn_get_path(B.HSA_OP_LANDMARKS) == -1
    assert lib.hsa_attn_set_path(-1, B.HSA_PATH_GENERIC) == 0
    for op in (B.HSA_OP_SELECT, B.HSA_OP_FORWARD, B.HSA_OP_BACKWARD, B.HSA_OP_DECODE):
        assert lib.hsa_attn_get_path(op) == B.HSA_PATH_GENERIC
    assert lib.hsa_attn_set_path(-1, B.HSA_PATH_AUTO) == 0
    for op in (B.HSA_OP_SELECT, B.HSA_OP_FORWARD, B.HSA_OP_BACKWARD, B.HSA_OP_DECODE):
        assert lib.hsa_attn_get_path(op) == B.HSA_PATH_AUTO


def test_decode_noalloc_checks(lib):
    """hsa_decode_noalloc refuses shapes whose scratch exceeds its per-GPU array, before any
    launch, and accepts an empty batch."""
    from paper_2504_16795_amd import binding as B
    p = B.make_params(4096, 1 << 20, 16, 2, 128, 64, 8, 1)
    need = lib.hsa_attn_workspace_size(ctypes.byref(p), B.HSA_OP_DECODE)
    assert need > (8 << 20)
    fake = ctypes.c_void_p(1 << 20)
    r = lib.hsa_decode_noalloc(ctypes.byref(p), fake, fake, fake, fake, 0, None, fake, fake,
                               fake, None)
    assert r == UNSUPPORTED
    assert "scratch" in lib.hsa_attn_last_error().decode()
    p0 = B.make_params(0, 1 << 20, 16, 2, 128, 64, 8, 1)
    assert lib.hsa_decode_noalloc(ctypes.byref(p0), None, None, None, None, 0, None, None,
                                  None, None, None) == OK
    # the 1M-token decode workload fits
    p1 = B.make_params(8, 1 << 20, 16, 2, 128, 64, 8, 1)
    assert lib.hsa_attn_workspace_size(ctypes.byref(p1), B.HSA_OP_DECODE) <= (8 << 20)


def test_no_cpu_fallback():
    """The product path has no CPU route: a missing library raises, and CPU tensors are
    refused before any call into the library."""
    import torch
    with pytest.raises(RuntimeError, match="not built"):
        binding.load(os.path.join(ROOT, "no_such_library.so"))
    K = torch.zeros((1, 128, 2, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensor"):
        hsa.hsa_landmarks(K, 64)
