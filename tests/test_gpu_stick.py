"""GPU parity of the stick-breaking chunk weights (Sec. 3.1.1): selection, decode and every
backward path against the oracle run with stick-breaking weights.

The forward takes the weights as given, so only the calls that form the weights (selection,
decode) or differentiate through them (the score term of the backward) change with the flag.
"""
import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import (W_ATOL, assert_close, assert_indices, check_decode, decode_case,
                    make_case, oracle_reference, to_dev)

pytestmark = pytest.mark.gpu

Shape = hsa_synth.HsaShape

CASES = {
    # name: (shape, seed, kind); the first three take the chunk-major fused backward,
    # wide_S128 the two-pass one, the f32 cases the generic one
    "L4K_like_bf16": (Shape(2, 1024, 16, 2, 128, 64, 8, "bf16"), 52, "iid"),
    "ragged_mfma_bf16": (Shape(1, 1000, 16, 2, 128, 64, 8, "bf16"), 53, "iid"),
    "k24_bf16": (Shape(1, 2048, 16, 2, 128, 32, 24, "bf16"), 54, "iid"),
    "k32_bf16": (Shape(1, 2304, 16, 2, 128, 64, 32, "bf16"), 55, "long"),
    "wide_S128_bf16": (Shape(1, 1024, 32, 4, 128, 128, 4, "bf16"), 5, "lowrank"),
    "ragged_f32": (Shape(2, 1000, 8, 2, 64, 32, 5, "f32"), 57, "iid"),
    "k20_d64_f32": (Shape(1, 1500, 4, 2, 64, 32, 20, "f32"), 58, "iid"),
}

_cache = {}


def case(name):
    if name not in _cache:
        shape, seed, kind = CASES[name]
        inp, _ = make_case(shape, seed, kind=kind, mu_std=0.0 if kind == "lowrank" else 0.5)
        ref = oracle_reference(inp, shape, stick=True)
        dev = {n: to_dev(v, shape) for n, v in inp.items()}
        _cache[name] = (shape, inp, ref, dev)
    return _cache[name]


def banner(name, what):
    print("\n[gpu] %s: %s" % (name, what), flush=True)


def _dev32(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


@pytest.mark.parametrize("name", list(CASES))
def test_select_stick(hsa_gpu, name):
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_select_topk, stick-breaking weights")
    Kbar = _dev32(ref["Kbar"].astype(np.float32))
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k,
                                     stick_breaking=True)
    torch.cuda.synchronize()
    sure, loose = assert_indices(idx, ref["idx"], ref["gap"], shape.S)
    assert loose == 0
    got = w.cpu().numpy()
    assert np.max(np.abs(got - ref["w"])) <= W_ATOL
    assert np.all(got.sum(-1) <= 1 + 1e-6)         # the leftover mass goes to no chunk


@pytest.mark.parametrize("two_pass", [False, True])
@pytest.mark.parametrize("name", list(CASES))
def test_backward_stick(hsa_gpu, name, two_pass, kernel_path):
    shape, inp, ref, dev = case(name)
    fused_shape = shape.dtype == "bf16" and shape.d == 128 and shape.S == 64 \
        and shape.H // shape.G == 8
    if two_pass and not fused_shape:
        pytest.skip("the two-pass switch only changes the path of the fused shapes")
    banner(name, "hsa_backward, stick-breaking (%s)" % ("two-pass" if two_pass else "default"))
    if two_pass:
        kernel_path(hsa_gpu.HSA_OP_BACKWARD, hsa_gpu.HSA_PATH_TWO_PASS)
    got = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], _dev32(ref["Kbar"].astype(np.float32)),
                               _dev32(ref["idx"]), _dev32(ref["w"].astype(np.float32)), dev["dO"],
                               shape.S, stick_breaking=True)
    torch.cuda.synchronize()
    for n, g_ in zip(("dQ", "dK", "dV"), got):
        assert_close(n, shape, g_, ref[n])


@pytest.mark.parametrize("name", ["L4K_like_bf16", "ragged_mfma_bf16", "wide_S128_bf16",
                                  "ragged_f32"])
def test_backward_stick_empty_slots(hsa_gpu, name):
    """Empty slots mixed into a stick-breaking selection: they hold no share of the stick,
    so the later slots' b are recovered from the valid slots only, on both sides."""
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_backward, stick-breaking with empty slots")
    rng = np.random.default_rng(59)
    ncand = (np.arange(shape.L) // shape.S)[None, :, None, None]
    u = rng.random(ref["idx"].shape)
    idx = np.where(u < 0.1, -1, ref["idx"])
    idx = np.where((u >= 0.1) & (u < 0.2), ncand + rng.integers(0, 3, idx.shape), idx)
    idx = idx.astype(np.int32)
    idx_o = np.where((idx < 0) | (idx >= ncand), -1, idx).astype(np.int32)
    w = ref["w"].astype(np.float32)
    want = oracle.backward(inp["Q"], inp["K"], inp["V"], idx_o, w, inp["dO"], shape.S,
                           stick=True)
    got = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], _dev32(ref["Kbar"].astype(np.float32)),
                               _dev32(idx), _dev32(w), dev["dO"], shape.S, stick_breaking=True)
    torch.cuda.synchronize()
    for n, g_, r in zip(("dQ", "dK", "dV"), got, want):
        assert_close(n, shape, g_, r)


@pytest.mark.parametrize("name", ["L4K_like_bf16", "ragged_f32"])
def test_pipeline_stick(hsa_gpu, name):
    """landmarks -> select -> forward -> backward on the GPU, all with the flag."""
    shape, inp, ref, dev = case(name)
    banner(name, "pipeline, stick-breaking")
    Kbar = hsa_gpu.hsa_landmarks(dev["K"], shape.S)
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k,
                                     stick_breaking=True)
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    dQ, dK, dV = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"],
                                      shape.S, stick_breaking=True)
    torch.cuda.synchronize()
    assert_indices(idx, ref["idx"], ref["gap"], shape.S)
    assert_close("O", shape, O, ref["O"], o_abs=ref["O_abs"])
    for n, t in (("dQ", dQ), ("dK", dK), ("dV", dV)):
        assert_close(n, shape, t, ref[n])


@pytest.mark.parametrize("k", [8, 20])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_stick(hsa_gpu, dtype, k):
    shape = Shape(3, 4096 + 64, 16, 2, 128 if dtype == "bf16" else 64, 64, k, dtype)
    banner("decode_stick_%s_k%d" % (dtype, k), "hsa_decode, stick-breaking")
    lens = [4096, 4096 + 40, 64 * 5 + 3]
    inp, Kbar = decode_case(shape, 61, lens)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, 64, k,
                                   cache_len=cache_len, stick_breaking=True)
    torch.cuda.synchronize()
    check_decode(shape, inp, Kbar, lens, o, idx, w, stick=True)
