"""GPU parity of the decode step with the key / value cache in host memory (Sec. 3.2 and the
offloading of Sec. 4.4: only the landmark cache stays on the GPU; the selected chunks are
fetched from pinned host memory every step).

The host path runs the same scan, merge and attend kernels as the device-resident decode,
with a gather from the host cache in between, so its outputs must equal hsa_decode's bit
for bit on the same cache contents; both are also checked against the oracle.
"""
import ctypes

import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import check_decode, decode_case

pytestmark = pytest.mark.gpu

Shape = hsa_synth.HsaShape


def banner(name, what):
    print("\n[gpu] %s: %s" % (name, what), flush=True)


CASES = [
    # (dtype, d, k, kbar dtype, stick, off by one): bf16 h = 8, d = 128, S = 64 takes the
    # MFMA attend kernel, f32 the finish + combine kernels
    ("bf16", 128, 8, torch.float32, False, False),
    ("bf16", 128, 20, torch.bfloat16, True, True),
    ("f32", 64, 8, torch.float32, False, False),
    ("f32", 64, 5, torch.bfloat16, True, True),
]


@pytest.mark.parametrize("dtype,d,k,kbar_dtype,stick,off1", CASES)
def test_decode_host_matches_device_decode_and_oracle(hsa_gpu, dtype, d, k, kbar_dtype, stick,
                                                      off1):
    shape = Shape(3, 4096 + 64, 16, 2, d, 64, k, dtype)
    banner("decode_host_%s_k%d_stick%d_off%d" % (dtype, k, stick, off1), "hsa_decode_host")
    lens = [4096, 4096 + 40, 64 * 5 + 3]
    inp, Kbar = decode_case(shape, 71, lens, kbar_dtype)
    Kc, Vc, q = inp["Kc"], inp["Vc"], inp["q"]
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    Kh, Vh = Kc.cpu().pin_memory(), Vc.cpu().pin_memory()
    o, idx, w = hsa_gpu.hsa_decode_host(q, Kh, Vh, Kbar, 64, k, cache_len=cache_len,
                                        stick_breaking=stick, off_by_one=off1)
    od, idxd, wd = hsa_gpu.hsa_decode(q, Kc, Vc, Kbar, 64, k, cache_len=cache_len,
                                      stick_breaking=stick, off_by_one=off1)
    torch.cuda.synchronize()
    assert torch.equal(idx, idxd)
    assert torch.equal(w, wd)
    assert torch.equal(o, od)
    check_decode(shape, inp, Kbar, lens, o, idx, w, stick=stick, off_by_one=off1)


def test_decode_host_refuses_memory_that_is_not_pinned_host_memory(hsa_gpu):
    """Pageable host memory and device memory are refused before any launch."""
    banner("decode_host_checks", "argument checks")
    B, N, H, G, d, S, k = 2, 512, 16, 2, 128, 64, 4
    lib = hsa_gpu.load()
    p = hsa_gpu.make_params(B, N, H, G, d, S, k, torch.bfloat16)
    q = torch.zeros((B, H, d), dtype=torch.bfloat16, device="cuda")
    Kbar = torch.zeros((B, N // S, G, d), dtype=torch.float32, device="cuda")
    o = torch.empty_like(q)
    idx = torch.empty((B, G, k), dtype=torch.int32, device="cuda")
    w = torch.empty((B, G, k), dtype=torch.float32, device="cuda")
    nws = hsa_gpu.workspace_size(p, hsa_gpu.HSA_OP_DECODE_HOST)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    pageable = torch.zeros((B, N, G, d), dtype=torch.bfloat16)
    device = torch.zeros((B, N, G, d), dtype=torch.bfloat16, device="cuda")
    pinned = torch.zeros((B, N, G, d), dtype=torch.bfloat16).pin_memory()
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    for bad in (pageable, device):
        r = lib.hsa_decode_host(ctypes.byref(p), P(q), P(bad), P(pinned), P(Kbar), 0, None,
                                P(o), P(idx), P(w), P(ws), nws, None)
        assert r == 1, r
        assert "pinned" in lib.hsa_attn_last_error().decode()
    # pinned caches are accepted (all-zero contents: a valid call)
    r = lib.hsa_decode_host(ctypes.byref(p), P(q), P(pinned), P(pinned), P(Kbar), 0, None,
                            P(o), P(idx), P(w), P(ws), nws, None)
    assert r == 0
    torch.cuda.synchronize()
    with pytest.raises(ValueError):
        hsa_gpu.hsa_decode_host(q, pageable, pinned, Kbar, S, k)
