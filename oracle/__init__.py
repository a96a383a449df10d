"""Python front-end of the HSA oracle (plain fp64 C, see hsa_oracle.h).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the GPU product path never does, and this
package imports nothing from it.

Full tensors use the operator layouts
    Q, dO, O, dQ : [B, L, H, d]     K, V, dK, dV : [B, L, G, d]
    Kbar         : [B, C, G, d]     idx, w       : [B, L, G, k]
and are split into independent (batch, group) slices for the C routines.  Inputs may be
float32 / bfloat16-valued float32 / float64; they are converted exactly to float64.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "hsa_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


class _Dims(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int64), ("h", ctypes.c_int32), ("d", ctypes.c_int32),
                ("S", ctypes.c_int32), ("k", ctypes.c_int32), ("alpha", ctypes.c_double),
                ("beta", ctypes.c_double), ("stick", ctypes.c_int32),
                ("off_by_one", ctypes.c_int32), ("sep", ctypes.c_int32)]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, no fast-math, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-fPIC", "-shared", "-Wall", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        srcs = (_SRC, os.path.join(_HERE, "hsa_oracle.h"))
        if not os.path.exists(_LIB_PATH) or \
                os.path.getmtime(_LIB_PATH) < max(os.path.getmtime(f) for f in srcs):
            build(force=True)          # absent, or older than its sources
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I64 = ctypes.c_int64
        DP = ctypes.POINTER(_Dims)
        lib.hsa_oracle_landmarks.argtypes = [DP, P, P]
        lib.hsa_oracle_select.argtypes = [DP, P, P, I64, P, P, P, P, P]
        lib.hsa_oracle_forward.argtypes = [DP, P, P, P, P, P, I64, P, P]
        lib.hsa_oracle_backward_q.argtypes = [DP, P, P, P, P, P, P, P, I64, P, P, P, P]
        lib.hsa_oracle_select_backward.argtypes = [DP, P, P, P, P, P, P, P, P]
        lib.hsa_oracle_backward_kv.argtypes = [DP, P, P, P, P, P, P, P, I64, P, P, P]
        lib.hsa_oracle_decode.argtypes = [DP, P, P, P, P, I64, P, P, P, P]
        lib.hsa_oracle_scores.argtypes = [DP, P, P, I64, I64, P, P]
        lib.hsa_oracle_slot_weights.argtypes = [DP, P, P, I64, I64, P, P, P]
        for f in ("landmarks", "select", "forward", "backward_q", "backward_kv", "decode",
                  "select_backward", "scores", "slot_weights"):
            getattr(lib, "hsa_oracle_" + f).restype = None
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):                       # torch tensor
        x = x.detach().float().cpu().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def default_scales(h: int, d: int):
    """alpha = 1/sqrt(h*d) (group dimension d_g = h*d_h), beta = 1/sqrt(d)."""
    return 1.0 / math.sqrt(h * d), 1.0 / math.sqrt(d)


def dims(L, h, d, S, k, alpha=None, beta=None, stick=False, off_by_one=False,
         sep=False) -> _Dims:
    """Slice dimensions; stick selects stick-breaking chunk weights (Sec. 3.1.1) instead of
    the softmax over the selected scores; off_by_one the softmax off by one for the
    attention inside a chunk (the paper's kernels, Sec. 3.1.2) instead of the softmax; sep
    a selection over inputs of its own (Sec. 3.1), whose score term the attention backward
    leaves out."""
    a0, b0 = default_scales(h, d)
    return _Dims(int(L), int(h), int(d), int(S), int(k),
                 float(a0 if alpha is None else alpha), float(b0 if beta is None else beta),
                 1 if stick else 0, 1 if off_by_one else 0, 1 if sep else 0)


# ----------------------------------------------------------------------------------
# per-(b, g) slice API
# ----------------------------------------------------------------------------------

def landmarks_slice(dm: _Dims, K: np.ndarray) -> np.ndarray:
    K = _f64(K)
    C = dm.L // dm.S
    out = np.zeros((C, dm.d))
    if C:
        _load().hsa_oracle_landmarks(ctypes.byref(dm), _p(K), _p(out))
    return out


def _rows(rows, L):
    if rows is None:
        return None, L
    r = np.ascontiguousarray(rows, dtype=np.int64)
    assert r.ndim == 1 and (r.size == 0 or (r.min() >= 0 and r.max() < L))
    return r, r.size


def select_slice(dm: _Dims, Q, Kbar, rows=None):
    Q, Kbar = _f64(Q), _f64(Kbar)
    r, n = _rows(rows, dm.L)
    idx = np.empty((n, dm.k), np.int32)
    w = np.empty((n, dm.k))
    gap = np.empty((n,))
    ss = np.empty((n, dm.k))
    if n:
        _load().hsa_oracle_select(ctypes.byref(dm), _p(Q), _p(Kbar), n, _p(r), _p(idx),
                                  _p(w), _p(gap), _p(ss))
    return idx, w, gap, ss


def scores_at(dm: _Dims, q, Kbar, pos):
    """Group scores [n, C] of n queries q [n, h, d] at sequence positions pos [n] against
    every landmark row of Kbar [C, d]; NaN where c >= floor(pos / S) (not a candidate)."""
    q, Kbar = _f64(q), _f64(Kbar)
    pos = np.ascontiguousarray(pos, dtype=np.int64)
    n, C = pos.size, Kbar.shape[0]
    assert q.shape == (n, dm.h, dm.d) and Kbar.shape[1] == dm.d
    s = np.empty((n, C))
    if n and C:
        _load().hsa_oracle_scores(ctypes.byref(dm), _p(q), _p(Kbar), C, n, _p(pos), _p(s))
    return s


def slot_weights_at(dm: _Dims, q, Kbar, pos, idx):
    """The weight rule (softmax, or stick-breaking with dm.stick) applied to the GIVEN slots
    idx [n, k] of n queries q [n, h, d] at positions pos [n]: [n, k], 0 in empty slots."""
    q, Kbar = _f64(q), _f64(Kbar)
    pos = np.ascontiguousarray(pos, dtype=np.int64)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    n, C = pos.size, Kbar.shape[0]
    assert q.shape == (n, dm.h, dm.d) and idx.shape == (n, dm.k)
    w = np.zeros((n, dm.k))
    if n and C:
        _load().hsa_oracle_slot_weights(ctypes.byref(dm), _p(q), _p(Kbar), C, n, _p(pos),
                                        _p(idx), _p(w))
    return w


def forward_slice(dm: _Dims, Q, K, V, idx, w, rows=None):
    Q, K, V, w = _f64(Q), _f64(K), _f64(V), _f64(w)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    r, n = _rows(rows, dm.L)
    O = np.empty((n, dm.h, dm.d))
    if n:
        _load().hsa_oracle_forward(ctypes.byref(dm), _p(Q), _p(K), _p(V), _p(idx), _p(w),
                                   n, _p(r), _p(O))
    return O


def backward_q_slice(dm: _Dims, Q, K, V, Kbar, idx, w, dO, rows=None, with_dw=False):
    Q, K, V, Kbar, w, dO = map(_f64, (Q, K, V, Kbar, w, dO))
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    r, n = _rows(rows, dm.L)
    dQ = np.empty((n, dm.h, dm.d))
    ds = np.empty((n, dm.k))
    dw = np.empty((n, dm.k))
    if n:
        _load().hsa_oracle_backward_q(ctypes.byref(dm), _p(Q), _p(K), _p(V), _p(Kbar),
                                      _p(idx), _p(w), _p(dO), n, _p(r), _p(dQ), _p(ds),
                                      _p(dw))
    return (dQ, ds, dw) if with_dw else (dQ, ds)


def select_backward_slice(dm: _Dims, Q, Kbar, idx, w, dw):
    """(dQ [L, h, d], dKbar [C, d], ds [L, k]) of one slice through the selection scores."""
    Q, Kbar, w, dw = map(_f64, (Q, Kbar, w, dw))
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    C = dm.L // dm.S
    dQ = np.empty((dm.L, dm.h, dm.d))
    dKbar = np.zeros((C, dm.d))
    ds = np.empty((dm.L, dm.k))
    if dm.L:
        _load().hsa_oracle_select_backward(ctypes.byref(dm), _p(Q),
                                           _p(Kbar if C else np.zeros((1, dm.d))), _p(idx),
                                           _p(w), _p(dw), _p(dQ),
                                           _p(dKbar if C else np.zeros((1, dm.d))), _p(ds))
    return dQ, dKbar, ds


def backward_kv_slice(dm: _Dims, Q, K, V, idx, w, dO, ds, chunks=None):
    Q, K, V, w, dO, ds = map(_f64, (Q, K, V, w, dO, ds))
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    C = dm.L // dm.S
    c, n = _rows(chunks, C)
    dK = np.empty((n, dm.S, dm.d))
    dV = np.empty((n, dm.S, dm.d))
    if n:
        _load().hsa_oracle_backward_kv(ctypes.byref(dm), _p(Q), _p(K), _p(V), _p(idx),
                                       _p(w), _p(dO), _p(ds), n, _p(c), _p(dK), _p(dV))
    return dK, dV


# ----------------------------------------------------------------------------------
# full-tensor API
# ----------------------------------------------------------------------------------

def _shape(Q, K):
    B, L, H, d = Q.shape
    G = K.shape[2]
    assert H % G == 0 and K.shape[:2] == (B, L) and K.shape[3] == d
    return B, L, H, G, d, H // G


def landmarks(K, S: int) -> np.ndarray:
    """Kbar [B, C, G, d] (fp64) of every complete chunk."""
    K = _f64(K)
    B, L, G, d = K.shape
    C = L // S
    out = np.zeros((B, C, G, d))
    for b in range(B):
        for g in range(G):
            out[b, :, g] = landmarks_slice(dims(L, 1, d, S, 1), K[b, :, g])
    return out


def select(Q, Kbar, G: int, S: int, k: int, alpha=None, stick=False):
    """idx [B,L,G,k] int32, w [B,L,G,k], gap [B,L,G], selected scores [B,L,G,k]."""
    Q, Kbar = _f64(Q), _f64(Kbar)
    B, L, H, d = Q.shape
    h = H // G
    idx = np.empty((B, L, G, k), np.int32)
    w = np.empty((B, L, G, k))
    gap = np.empty((B, L, G))
    ss = np.empty((B, L, G, k))
    for b in range(B):
        for g in range(G):
            dm = dims(L, h, d, S, k, alpha, None, stick)
            i, ww, gp, s = select_slice(dm, Q[b, :, g * h:(g + 1) * h], Kbar[b, :, g])
            idx[b, :, g], w[b, :, g], gap[b, :, g], ss[b, :, g] = i, ww, gp, s
    return idx, w, gap, ss


def forward(Q, K, V, idx, w, S: int, beta=None, off_by_one=False):
    Q, K, V, w = map(_f64, (Q, K, V, w))
    B, L, H, G, d, h = _shape(Q, K)
    k = idx.shape[-1]
    O = np.empty((B, L, H, d))
    for b in range(B):
        for g in range(G):
            dm = dims(L, h, d, S, k, None, beta, off_by_one=off_by_one)
            O[b, :, g * h:(g + 1) * h] = forward_slice(
                dm, Q[b, :, g * h:(g + 1) * h], K[b, :, g], V[b, :, g],
                np.ascontiguousarray(idx[b, :, g]), w[b, :, g])
    return O


def backward(Q, K, V, idx, w, dO, S: int, alpha=None, beta=None, stick=False,
             off_by_one=False, separate=False):
    """dQ, dK, dV (fp64) of sum(dO * O) with the selection held fixed (weights a function of
    the selected scores: softmax, or stick-breaking with stick).  separate: the scores come
    from selection inputs of their own, so no score term reaches Q or K; returns
    (dQ, dK, dV, dw) with dw [B, L, G, k] = d loss / d w."""
    Q, K, V, w, dO = map(_f64, (Q, K, V, w, dO))
    B, L, H, G, d, h = _shape(Q, K)
    k = idx.shape[-1]
    C = L // S
    dQ = np.empty((B, L, H, d))
    dK = np.zeros((B, L, G, d))
    dV = np.zeros((B, L, G, d))
    dW = np.zeros((B, L, G, k))
    for b in range(B):
        for g in range(G):
            dm = dims(L, h, d, S, k, alpha, beta, stick, off_by_one, separate)
            Qs = np.ascontiguousarray(Q[b, :, g * h:(g + 1) * h])
            dOs = np.ascontiguousarray(dO[b, :, g * h:(g + 1) * h])
            Ks, Vs = np.ascontiguousarray(K[b, :, g]), np.ascontiguousarray(V[b, :, g])
            ids, ws = np.ascontiguousarray(idx[b, :, g]), np.ascontiguousarray(w[b, :, g])
            Kb = landmarks_slice(dm, Ks)
            dq, ds, dw = backward_q_slice(dm, Qs, Ks, Vs, Kb, ids, ws, dOs, with_dw=True)
            dQ[b, :, g * h:(g + 1) * h] = dq
            dW[b, :, g] = dw
            if C:
                dk, dv = backward_kv_slice(dm, Qs, Ks, Vs, ids, ws, dOs, ds)
                dK[b, :C * S, g] = dk.reshape(C * S, d)
                dV[b, :C * S, g] = dv.reshape(C * S, d)
    return (dQ, dK, dV, dW) if separate else (dQ, dK, dV)


def select_backward(Q, Kbar, idx, w, dw, G: int, S: int, alpha=None, stick=False):
    """Gradient through the selection scores s = alpha (sum_j q_j) . Kbar_c for d loss / d w
    = dw [B, L, G, k]: (dQ [B, L, H, d], dKbar [B, C, G, d], ds [B, L, G, k]).  For a
    selection over inputs of its own, Q is [B, L, G, d_sel] (h = 1) and Kbar the chunk
    representations [B, C, G, d_sel]."""
    Q, Kbar, w, dw = map(_f64, (Q, Kbar, w, dw))
    B, L, H, d = Q.shape
    h = H // G
    k = idx.shape[-1]
    C = L // S
    dQ = np.empty((B, L, H, d))
    dKbar = np.zeros((B, C, G, d))
    ds = np.empty((B, L, G, k))
    for b in range(B):
        for g in range(G):
            dm = dims(L, h, d, S, k, alpha, None, stick)
            dq, dkb, dsl = select_backward_slice(
                dm, np.ascontiguousarray(Q[b, :, g * h:(g + 1) * h]),
                np.ascontiguousarray(Kbar[b, :, g]), np.ascontiguousarray(idx[b, :, g]),
                np.ascontiguousarray(w[b, :, g]), np.ascontiguousarray(dw[b, :, g]))
            dQ[b, :, g * h:(g + 1) * h] = dq
            dKbar[b, :, g] = dkb
            ds[b, :, g] = dsl
    return dQ, dKbar, ds


def decode(q, Kc, Vc, Kbar_cache, cache_len: Sequence[int], S: int, k: int,
           alpha=None, beta=None, stick=False, off_by_one=False):
    """Single-token decode: q [B,H,d]; Kc, Vc [B,N,G,d]; Kbar_cache [B,Cc,G,d] (given).

    Returns o [B,H,d], idx [B,G,k], w [B,G,k], gap [B,G]."""
    q = _f64(q)
    B, H, d = q.shape
    G = Kc.shape[2]
    h = H // G
    o = np.empty((B, H, d))
    idx = np.empty((B, G, k), np.int32)
    w = np.empty((B, G, k))
    gap = np.empty((B, G))
    lib = _load()
    for b in range(B):
        n = int(cache_len[b])
        nch = n // S
        for g in range(G):
            dm = dims(n, h, d, S, k, alpha, beta, stick, off_by_one)
            qs = np.ascontiguousarray(q[b, g * h:(g + 1) * h])
            # only the candidate chunks are read
            Ks = _f64(Kc[b, :nch * S, g]) if nch else np.zeros((1, d))
            Vs = _f64(Vc[b, :nch * S, g]) if nch else np.zeros((1, d))
            Kb = _f64(Kbar_cache[b, :nch, g]) if nch else np.zeros((1, d))
            ii = np.empty(k, np.int32)
            ww = np.empty(k)
            oo = np.empty((h, d))
            gp = np.empty(1)
            lib.hsa_oracle_decode(ctypes.byref(dm), _p(qs), _p(Ks), _p(Vs), _p(Kb), n,
                                  _p(ii), _p(ww), _p(oo), _p(gp))
            o[b, g * h:(g + 1) * h], idx[b, g], w[b, g], gap[b, g] = oo, ii, ww, gp[0]
    return o, idx, w, gap
