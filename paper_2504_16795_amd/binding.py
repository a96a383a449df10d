"""Thin ctypes binding of libhsa_mi355x.so (C ABI in include/hsa.h).

Argument marshalling only: shape/dtype checks, output and workspace allocation through
torch, the current HIP stream, and status-to-exception translation.  Every step of the
operator runs in the library's HIP kernels; there is no fallback of any kind, and a
missing library raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhsa_mi355x.so")

HSA_DTYPE_F32, HSA_DTYPE_BF16 = 0, 1
(HSA_OP_LANDMARKS, HSA_OP_SELECT, HSA_OP_FORWARD, HSA_OP_BACKWARD, HSA_OP_DECODE,
 HSA_OP_SELECT_BACKWARD, HSA_OP_DECODE_HOST) = range(7)
(HSA_PATH_AUTO, HSA_PATH_GENERIC, HSA_PATH_TWO_PASS, HSA_PATH_CHUNK_MAJOR,
 HSA_PATH_TILE_MAJOR, HSA_PATH_FUSED) = range(6)
HSA_FLAG_STICK_BREAKING = 2
HSA_FLAG_SOFTMAX_OFF_BY_ONE = 1
STATUS = {0: "OK", 1: "INVALID_ARGUMENT", 2: "UNSUPPORTED", 3: "WORKSPACE_TOO_SMALL", 4: "HIP"}

_lib = None


class HsaParams(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seqlen", ctypes.c_int32),
                ("n_qheads", ctypes.c_int32), ("n_kvheads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("chunk", ctypes.c_int32),
                ("topk", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("sm_scale", ctypes.c_float), ("sel_scale", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


class HsaError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__("%s failed: %s (%s)" % (where, STATUS.get(status, status), detail))
        self.status = status


EXPORTED = ("hsa_landmarks", "hsa_select_topk", "hsa_forward", "hsa_backward", "hsa_decode",
            "hsa_backward_attn", "hsa_select_backward", "hsa_decode_host",
            "hsa_attn_workspace_size", "hsa_attn_status_string", "hsa_attn_last_error",
            "hsa_attn_timing_enable", "hsa_attn_timing_select", "hsa_attn_timing_collect",
            "hsa_attn_set_path", "hsa_attn_get_path", "hsa_decode_noalloc")


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError("HSA HIP library not built: %s (run __graft_entry__.build())" % p)
    lib = ctypes.CDLL(p)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    PP = ctypes.POINTER(HsaParams)
    lib.hsa_landmarks.argtypes = [PP, P, P, I32, I32, I32, P]
    lib.hsa_select_topk.argtypes = [PP, P, P, P, P, P, SZ, P]
    lib.hsa_forward.argtypes = [PP, P, P, P, P, P, P, P, SZ, P]
    lib.hsa_backward.argtypes = [PP, P, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.hsa_decode.argtypes = [PP, P, P, P, P, I32, P, P, P, P, P, SZ, P]
    lib.hsa_backward_attn.argtypes = [PP, P, P, P, P, P, P, P, P, P, P, I32, P, SZ, P]
    lib.hsa_select_backward.argtypes = [PP, P, P, P, P, P, P, P, P, SZ, P]
    lib.hsa_decode_host.argtypes = [PP, P, P, P, P, I32, P, P, P, P, P, SZ, P]
    lib.hsa_decode_noalloc.argtypes = [PP, P, P, P, P, I32, P, P, P, P, P]
    for f in ("hsa_landmarks", "hsa_select_topk", "hsa_forward", "hsa_backward", "hsa_decode",
              "hsa_backward_attn", "hsa_select_backward", "hsa_decode_host",
              "hsa_decode_noalloc"):
        getattr(lib, f).restype = I32
    lib.hsa_attn_workspace_size.argtypes = [PP, ctypes.c_int]
    lib.hsa_attn_workspace_size.restype = SZ
    lib.hsa_attn_status_string.argtypes = [I32]
    lib.hsa_attn_status_string.restype = ctypes.c_char_p
    lib.hsa_attn_last_error.argtypes = []
    lib.hsa_attn_last_error.restype = ctypes.c_char_p
    lib.hsa_attn_timing_enable.argtypes = [ctypes.c_int]
    lib.hsa_attn_timing_enable.restype = I32
    lib.hsa_attn_timing_select.argtypes = [ctypes.c_char_p]
    lib.hsa_attn_timing_select.restype = I32
    lib.hsa_attn_timing_collect.argtypes = [ctypes.c_char_p, SZ]
    lib.hsa_attn_timing_collect.restype = ctypes.c_int
    lib.hsa_attn_set_path.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.hsa_attn_set_path.restype = I32
    lib.hsa_attn_get_path.argtypes = [ctypes.c_int]
    lib.hsa_attn_get_path.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def set_path(op: int, path: int) -> None:
    """Serve `op` with the kernel family `path` (hsa_attn_set_path; HSA_PATH_AUTO restores
    the default); process-wide."""
    _check(load().hsa_attn_set_path(int(op), int(path)), "hsa_attn_set_path")


def get_path(op: int) -> int:
    return int(load().hsa_attn_get_path(int(op)))


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return HSA_DTYPE_F32
    if t == torch.bfloat16:
        return HSA_DTYPE_BF16
    raise TypeError("unsupported dtype %s (float32 or bfloat16)" % t)


def make_params(B, L, H, G, d, S, k, dtype, sm_scale=0.0, sel_scale=0.0,
                stick_breaking=False, off_by_one=False) -> HsaParams:
    code = dtype if isinstance(dtype, int) else _dtype_code(dtype)
    flags = (HSA_FLAG_STICK_BREAKING if stick_breaking else 0) | \
        (HSA_FLAG_SOFTMAX_OFF_BY_ONE if off_by_one else 0)
    return HsaParams(int(B), int(L), int(H), int(G), int(d), int(S), int(k), code,
                     float(sm_scale), float(sel_scale), flags)


def workspace_size(p: HsaParams, op: int) -> int:
    return int(load().hsa_attn_workspace_size(ctypes.byref(p), op))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(dev: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _check(status: int, where: str):
    if status != 0:
        detail = load().hsa_attn_last_error().decode()
        raise HsaError(status, where, detail)


def _need(t: torch.Tensor, name: str, shape=None, dtype=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be a GPU tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if dtype is not None and t.dtype != dtype:
        raise ValueError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))


def _workspace(p: HsaParams, op: int, dev, ws: Optional[torch.Tensor]):
    n = workspace_size(p, op)
    if ws is None:
        ws = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)
    return ws, ws.numel() * ws.element_size()


def hsa_landmarks(K: torch.Tensor, S: int, kbar_dtype: torch.dtype = torch.float32,
                  chunk_begin: int = 0, chunk_end: Optional[int] = None,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Kbar [B, floor(L/S), G, d] = mean of each chunk's keys (chunks [begin, end))."""
    B, L, G, d = K.shape
    C = L // S
    _need(K, "K")
    p = make_params(B, L, G, G, d, S, 1, K.dtype)
    if out is None:
        out = torch.empty((B, C, G, d), dtype=kbar_dtype, device=K.device)
    _need(out, "Kbar", (B, C, G, d), kbar_dtype, K.device)
    end = C if chunk_end is None else chunk_end
    _check(load().hsa_landmarks(ctypes.byref(p), _ptr(K), _ptr(out), _dtype_code(kbar_dtype),
                                int(chunk_begin), int(end), _stream(K.device)), "hsa_landmarks")
    return out


def hsa_select_topk(Q: torch.Tensor, Kbar: torch.Tensor, G: int, S: int, k: int,
                    sel_scale: float = 0.0, idx: Optional[torch.Tensor] = None,
                    w: Optional[torch.Tensor] = None,
                    stick_breaking: bool = False) -> Tuple[torch.Tensor, torch.Tensor]:
    """idx int32 [B, L, G, k] (descending chunk order, -1 pad), w float32 [B, L, G, k]:
    softmax weights over the selected scores, or stick-breaking ones in slot order."""
    B, L, H, d = Q.shape
    _need(Q, "Q")
    _need(Kbar, "Kbar", (B, L // S, G, d), torch.float32, Q.device)
    p = make_params(B, L, H, G, d, S, k, Q.dtype, 0.0, sel_scale, stick_breaking)
    if idx is None:
        idx = torch.empty((B, L, G, k), dtype=torch.int32, device=Q.device)
    if w is None:
        w = torch.empty((B, L, G, k), dtype=torch.float32, device=Q.device)
    _need(idx, "idx", (B, L, G, k), torch.int32, Q.device)
    _need(w, "w", (B, L, G, k), torch.float32, Q.device)
    _check(load().hsa_select_topk(ctypes.byref(p), _ptr(Q), _ptr(Kbar), _ptr(idx), _ptr(w), None,
                                  0, _stream(Q.device)), "hsa_select_topk")
    return idx, w


def hsa_forward(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, idx: torch.Tensor,
                w: torch.Tensor, S: int, sm_scale: float = 0.0,
                out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None,
                off_by_one: bool = False) -> torch.Tensor:
    """O [B, L, H, d] = sum_i w_i softmax(beta q K_c^T) V_c over the selected chunks (the
    softmax off by one with off_by_one)."""
    B, L, H, d = Q.shape
    G, k = K.shape[2], idx.shape[-1]
    _need(Q, "Q")
    _need(K, "K", (B, L, G, d), Q.dtype, Q.device)
    _need(V, "V", (B, L, G, d), Q.dtype, Q.device)
    _need(idx, "idx", (B, L, G, k), torch.int32, Q.device)
    _need(w, "w", (B, L, G, k), torch.float32, Q.device)
    p = make_params(B, L, H, G, d, S, k, Q.dtype, sm_scale, off_by_one=off_by_one)
    if out is None:
        out = torch.empty_like(Q)
    _need(out, "O", Q.shape, Q.dtype, Q.device)
    ws, nb = _workspace(p, HSA_OP_FORWARD, Q.device, workspace)
    _check(load().hsa_forward(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(idx), _ptr(w),
                              _ptr(out), _ptr(ws), nb, _stream(Q.device)), "hsa_forward")
    return out


def hsa_backward(Q, K, V, Kbar, idx, w, dO, S: int, sm_scale: float = 0.0,
                 sel_scale: float = 0.0, out=None, workspace: Optional[torch.Tensor] = None,
                 stick_breaking: bool = False, off_by_one: bool = False):
    """(dQ, dK, dV) of sum(dO * O) with the selection held fixed; stick_breaking states
    how w was formed from the scores (the score term of the gradient depends on it),
    off_by_one which softmax the forward took inside a chunk."""
    B, L, H, d = Q.shape
    G, k = K.shape[2], idx.shape[-1]
    for t, n, shp in ((Q, "Q", None), (K, "K", (B, L, G, d)), (V, "V", (B, L, G, d)),
                      (dO, "dO", (B, L, H, d))):
        _need(t, n, shp, Q.dtype, Q.device)
    _need(Kbar, "Kbar", (B, L // S, G, d), torch.float32, Q.device)
    _need(idx, "idx", (B, L, G, k), torch.int32, Q.device)
    _need(w, "w", (B, L, G, k), torch.float32, Q.device)
    p = make_params(B, L, H, G, d, S, k, Q.dtype, sm_scale, sel_scale, stick_breaking,
                    off_by_one)
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    dQ, dK, dV = out
    ws, nb = _workspace(p, HSA_OP_BACKWARD, Q.device, workspace)
    _check(load().hsa_backward(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(Kbar), _ptr(idx),
                               _ptr(w), _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws), nb,
                               _stream(Q.device)), "hsa_backward")
    return dQ, dK, dV


def hsa_backward_attn(Q, K, V, idx, w, dO, S: int, sm_scale: float = 0.0, out=None,
                      dw: Optional[torch.Tensor] = None, accumulate_dw: bool = False,
                      workspace: Optional[torch.Tensor] = None, off_by_one: bool = False):
    """(dQ, dK, dV, dw) of sum(dO * O) for one layer whose selection comes from inputs of
    its own: no score term reaches Q or K; dw [B, L, G, k] float32 = d loss / d w, written,
    or added to the given dw with accumulate_dw."""
    B, L, H, d = Q.shape
    G, k = K.shape[2], idx.shape[-1]
    for t, n, shp in ((Q, "Q", None), (K, "K", (B, L, G, d)), (V, "V", (B, L, G, d)),
                      (dO, "dO", (B, L, H, d))):
        _need(t, n, shp, Q.dtype, Q.device)
    _need(idx, "idx", (B, L, G, k), torch.int32, Q.device)
    _need(w, "w", (B, L, G, k), torch.float32, Q.device)
    if dw is None:
        if accumulate_dw:
            raise ValueError("accumulate_dw needs the dw to add to")
        dw = torch.empty((B, L, G, k), dtype=torch.float32, device=Q.device)
    _need(dw, "dw", (B, L, G, k), torch.float32, Q.device)
    p = make_params(B, L, H, G, d, S, k, Q.dtype, sm_scale, off_by_one=off_by_one)
    if out is None:
        out = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    dQ, dK, dV = out
    ws, nb = _workspace(p, HSA_OP_BACKWARD, Q.device, workspace)
    _check(load().hsa_backward_attn(ctypes.byref(p), _ptr(Q), _ptr(K), _ptr(V), _ptr(idx),
                                    _ptr(w), _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(dw),
                                    1 if accumulate_dw else 0, _ptr(ws), nb,
                                    _stream(Q.device)), "hsa_backward_attn")
    return dQ, dK, dV, dw


def hsa_select_backward(Qs, Ks, idx, w, dw, G: int, S: int, sel_scale: float = 0.0,
                        stick_breaking: bool = False, out=None,
                        workspace: Optional[torch.Tensor] = None):
    """(dQs, dKs) through the selection scores s = alpha q~ . Ks_c for d loss / d w = dw:
    Qs [B, L, G h, d_sel] (h = 1 for selection inputs of their own), Ks [B, C, G, d_sel]
    float32; dQs like Qs, dKs [B, C, G, d_sel] float32."""
    B, L, H, d = Qs.shape
    k = idx.shape[-1]
    C = L // S
    _need(Qs, "Qs")
    _need(Ks, "Ks", (B, C, G, d), torch.float32, Qs.device)
    for t, n in ((idx, "idx"), (w, "w"), (dw, "dw")):
        _need(t, n, (B, L, G, k), torch.int32 if n == "idx" else torch.float32, Qs.device)
    p = make_params(B, L, H, G, d, S, k, Qs.dtype, 0.0, sel_scale, stick_breaking)
    if out is None:
        out = (torch.empty_like(Qs), torch.empty((B, C, G, d), dtype=torch.float32,
                                                 device=Qs.device))
    dQs, dKs = out
    ws, nb = _workspace(p, HSA_OP_SELECT_BACKWARD, Qs.device, workspace)
    _check(load().hsa_select_backward(ctypes.byref(p), _ptr(Qs), _ptr(Ks), _ptr(idx), _ptr(w),
                                      _ptr(dw), _ptr(dQs), _ptr(dKs), _ptr(ws), nb,
                                      _stream(Qs.device)), "hsa_select_backward")
    return dQs, dKs


def hsa_decode(q, Kcache, Vcache, Kbar_cache, S: int, k: int,
               cache_len: Optional[torch.Tensor] = None, sm_scale: float = 0.0,
               sel_scale: float = 0.0, out=None, workspace: Optional[torch.Tensor] = None,
               stick_breaking: bool = False, off_by_one: bool = False):
    """One query token per sequence at position cache_len[b]: (o [B,H,d], idx, w [B,G,k])."""
    B, H, d = q.shape
    Ncap, G = Kcache.shape[1], Kcache.shape[2]
    _need(q, "q")
    _need(Kcache, "Kcache", (B, Ncap, G, d), q.dtype, q.device)
    _need(Vcache, "Vcache", (B, Ncap, G, d), q.dtype, q.device)
    _need(Kbar_cache, "Kbar_cache", (B, Ncap // S, G, d), None, q.device)
    if cache_len is not None:
        _need(cache_len, "cache_len", (B,), torch.int32, q.device)
    p = make_params(B, Ncap, H, G, d, S, k, q.dtype, sm_scale, sel_scale, stick_breaking,
                    off_by_one)
    if out is None:
        out = (torch.empty_like(q), torch.empty((B, G, k), dtype=torch.int32, device=q.device),
               torch.empty((B, G, k), dtype=torch.float32, device=q.device))
    o, idx, w = out
    ws, nb = _workspace(p, HSA_OP_DECODE, q.device, workspace)
    _check(load().hsa_decode(ctypes.byref(p), _ptr(q), _ptr(Kcache), _ptr(Vcache),
                             _ptr(Kbar_cache), _dtype_code(Kbar_cache.dtype), _ptr(cache_len),
                             _ptr(o), _ptr(idx), _ptr(w), _ptr(ws), nb, _stream(q.device)),
           "hsa_decode")
    return o, idx, w


def hsa_decode_noalloc(q, Kcache, Vcache, Kbar_cache, S: int, k: int,
                       cache_len: Optional[torch.Tensor] = None, sm_scale: float = 0.0,
                       sel_scale: float = 0.0, out=None, stick_breaking: bool = False,
                       off_by_one: bool = False):
    """hsa_decode without a workspace: the library's per-GPU scratch array serves instead
    (calls overlapping on one GPU race).  Pass `out` to allocate nothing at all."""
    B, H, d = q.shape
    Ncap, G = Kcache.shape[1], Kcache.shape[2]
    _need(q, "q")
    _need(Kcache, "Kcache", (B, Ncap, G, d), q.dtype, q.device)
    _need(Vcache, "Vcache", (B, Ncap, G, d), q.dtype, q.device)
    _need(Kbar_cache, "Kbar_cache", (B, Ncap // S, G, d), None, q.device)
    if cache_len is not None:
        _need(cache_len, "cache_len", (B,), torch.int32, q.device)
    p = make_params(B, Ncap, H, G, d, S, k, q.dtype, sm_scale, sel_scale, stick_breaking,
                    off_by_one)
    if out is None:
        out = (torch.empty_like(q), torch.empty((B, G, k), dtype=torch.int32, device=q.device),
               torch.empty((B, G, k), dtype=torch.float32, device=q.device))
    o, idx, w = out
    _check(load().hsa_decode_noalloc(ctypes.byref(p), _ptr(q), _ptr(Kcache), _ptr(Vcache),
                                     _ptr(Kbar_cache), _dtype_code(Kbar_cache.dtype),
                                     _ptr(cache_len), _ptr(o), _ptr(idx), _ptr(w),
                                     _stream(q.device)),
           "hsa_decode_noalloc")
    return o, idx, w


def hsa_decode_host(q, Kcache_host, Vcache_host, Kbar_cache, S: int, k: int,
                    cache_len: Optional[torch.Tensor] = None, sm_scale: float = 0.0,
                    sel_scale: float = 0.0, out=None, workspace: Optional[torch.Tensor] = None,
                    stick_breaking: bool = False, off_by_one: bool = False):
    """hsa_decode with the key / value cache [B, N_cap, G, d] in pinned host memory (CPU
    tensors from pin_memory); q, the landmark cache and the outputs live on the GPU."""
    B, H, d = q.shape
    Ncap, G = Kcache_host.shape[1], Kcache_host.shape[2]
    _need(q, "q")
    for t, n in ((Kcache_host, "Kcache_host"), (Vcache_host, "Vcache_host")):
        if not isinstance(t, torch.Tensor) or t.is_cuda or not t.is_pinned():
            raise ValueError("%s must be a pinned CPU tensor" % n)
        if not t.is_contiguous() or tuple(t.shape) != (B, Ncap, G, d) or t.dtype != q.dtype:
            raise ValueError("%s must be a contiguous %s tensor of shape %s"
                             % (n, q.dtype, (B, Ncap, G, d)))
    _need(Kbar_cache, "Kbar_cache", (B, Ncap // S, G, d), None, q.device)
    if cache_len is not None:
        _need(cache_len, "cache_len", (B,), torch.int32, q.device)
    p = make_params(B, Ncap, H, G, d, S, k, q.dtype, sm_scale, sel_scale, stick_breaking,
                    off_by_one)
    if out is None:
        out = (torch.empty_like(q), torch.empty((B, G, k), dtype=torch.int32, device=q.device),
               torch.empty((B, G, k), dtype=torch.float32, device=q.device))
    o, idx, w = out
    ws, nb = _workspace(p, HSA_OP_DECODE_HOST, q.device, workspace)
    _check(load().hsa_decode_host(ctypes.byref(p), _ptr(q), ctypes.c_void_p(Kcache_host.data_ptr()),
                                  ctypes.c_void_p(Vcache_host.data_ptr()), _ptr(Kbar_cache),
                                  _dtype_code(Kbar_cache.dtype), _ptr(cache_len), _ptr(o),
                                  _ptr(idx), _ptr(w), _ptr(ws), nb, _stream(q.device)),
           "hsa_decode_host")
    return o, idx, w


def timing_enable(on: bool = True) -> None:
    """Bracket every kernel launch of the library with HIP events on its stream."""
    load().hsa_attn_timing_enable(1 if on else 0)


def timing_select(name: Optional[str] = None) -> None:
    """Time only the kernels called `name` (None: every kernel)."""
    load().hsa_attn_timing_select(name.encode() if name else None)


def timing_collect() -> dict:
    """{kernel name: (launches, total ms)} for the launches recorded since the last call."""
    lib = load()
    n = lib.hsa_attn_timing_collect(None, 0)
    buf = ctypes.create_string_buffer(n + 4096)
    while lib.hsa_attn_timing_collect(buf, len(buf)) > len(buf):
        buf = ctypes.create_string_buffer(2 * len(buf))
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out
