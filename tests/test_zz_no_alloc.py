"""hsa_decode_noalloc (the decode entry point that allocates nothing: its scratch is the
library's per-GPU device array) against hsa_decode with a workspace, through the C ABI, on
two calls in a row, the second with a smaller input; both also against the oracle."""
import ctypes

import numpy as np
import pytest
import torch

import hsa_synth
from parity import check_decode, decode_case

pytestmark = pytest.mark.gpu

Shape = hsa_synth.HsaShape


def _call_noalloc(lib, hsa, inp, Kbar, S, k, lens, stick=False):
    q, Kc, Vc = inp["q"], inp["Kc"], inp["Vc"]
    B, H, d = q.shape
    N, G = Kc.shape[1], Kc.shape[2]
    p = hsa.make_params(B, N, H, G, d, S, k, q.dtype, stick_breaking=stick)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o = torch.full_like(q, float("nan"))
    idx = torch.full((B, G, k), 777, dtype=torch.int32, device="cuda")
    w = torch.full((B, G, k), float("nan"), dtype=torch.float32, device="cuda")
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    kdt = 1 if Kbar.dtype == torch.bfloat16 else 0
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    r = lib.hsa_decode_noalloc(ctypes.byref(p), P(q), P(Kc), P(Vc), P(Kbar), kdt, P(cache_len),
                               P(o), P(idx), P(w), st)
    assert r == 0, lib.hsa_attn_last_error().decode()
    return o, idx, w, cache_len


@pytest.mark.parametrize("dtype,kbar_dtype,stick", [("bf16", torch.bfloat16, False),
                                                    ("f32", torch.float32, True)])
def test_decode_noalloc_matches_decode(hsa_gpu, dtype, kbar_dtype, stick):
    lib = hsa_gpu.load()
    d = 128 if dtype == "bf16" else 64
    S, k = 64, 8
    # first call: 4 sequences of 8256 cached tokens; second: 2 sequences of 4160 and k = 5
    for B, N, kk, lens, seed in ((4, 8192 + 64, k, [8192 + 64, 8192, 5000, 64], 91),
                                 (2, 4096 + 64, 5, [4096 + 30, 700], 92)):
        shape = Shape(B, N, 16, 2, d, S, kk, dtype)
        print("\n[gpu] decode_noalloc %s B=%d N=%d k=%d" % (dtype, B, N, kk), flush=True)
        inp, Kbar = decode_case(shape, seed, lens, kbar_dtype)
        o, idx, w, cache_len = _call_noalloc(lib, hsa_gpu, inp, Kbar, S, kk, lens, stick)
        od, idxd, wd = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, S, kk,
                                          cache_len=cache_len, stick_breaking=stick)
        torch.cuda.synchronize()
        assert torch.equal(idx, idxd) and torch.equal(w, wd) and torch.equal(o, od)
        check_decode(shape, inp, Kbar, lens, o, idx, w, stick=stick)
