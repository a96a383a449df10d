"""GPU parity of a selection over inputs of its own shared by several layers (Sec. 3.1: the
selection query and chunk representations come from projections of their own, of the
group dimension d_g = h d_h; Sec. 4.4: one selection serves every HSA layer):
hsa_select_topk on the selection inputs (rows up to 1024 long), hsa_backward_attn per
layer (no score term, dw out or accumulated), hsa_select_backward of the summed dw.
"""
import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import (MIN_GAP, W_ATOL, assert_close, assert_indices, make_case,
                    oracle_reference, to_dev)

pytestmark = pytest.mark.gpu

Shape = hsa_synth.HsaShape


def banner(name, what):
    print("\n[gpu] %s: %s" % (name, what), flush=True)


def _dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x)).cuda()
    return t.to(dtype) if dtype is not None else t


def selection_inputs(B, L, G, S, k, dsel, seed, bf16=True, stick=False):
    """Selection queries Qs [B, L, G, dsel] (bf16-exact when bf16) and chunk representations
    Ks [B, C, G, dsel] float32, N(0, 1) each, so the scores alpha Qs . Ks (alpha =
    1/sqrt(dsel)) are about N(0, 1); query rows are redrawn until every token's top-k gap
    is >= MIN_GAP."""
    g = hsa_synth.philox(seed, 91)
    Qs = g.standard_normal((B, L, G, dsel)).astype(np.float32)
    Ks = g.standard_normal((B, L // S, G, dsel)).astype(np.float32)
    if bf16:
        Qs = hsa_synth.round_bf16(Qs)
    for attempt in range(32):
        _, _, gap, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
        bad = gap < MIN_GAP
        if not bad.any():
            return Qs, Ks
        new = hsa_synth.philox(seed, 92, attempt).standard_normal(Qs.shape).astype(np.float32)
        if bf16:
            new = hsa_synth.round_bf16(new)
        Qs[bad] = new[bad]
    raise RuntimeError("gap enforcement failed")


@pytest.mark.parametrize("stick", [False, True])
@pytest.mark.parametrize("dsel,k", [(256, 8), (512, 16), (1024, 8), (1024, 32), (128, 8)])
def test_select_on_selection_inputs(hsa_gpu, dsel, k, stick):
    B, L, G, S = 2, 1024, 2, 32
    banner("sel_%d_k%d_stick%d" % (dsel, k, stick), "hsa_select_topk on selection inputs")
    Qs, Ks = selection_inputs(B, L, G, S, k, dsel, 300 + dsel + k, stick=stick)
    idx_ref, w_ref, gap, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
    idx, w = hsa_gpu.hsa_select_topk(_dev(Qs, torch.bfloat16), _dev(Ks), G, S, k,
                                     stick_breaking=stick)
    torch.cuda.synchronize()
    sure, loose = assert_indices(idx, idx_ref, gap, S)
    assert loose == 0
    assert np.max(np.abs(w.cpu().numpy() - w_ref)) <= W_ATOL


ATTN_CASES = {
    # name: (shape, seed, options): the fused chunk-major path, the two-pass path (forced, and
    # at S = 128) and the generic kernels
    "fused_bf16": (Shape(2, 1024, 16, 2, 128, 64, 8, "bf16"), 401, {}),
    "two_pass_bf16": (Shape(1, 1000, 16, 2, 128, 64, 8, "bf16"), 402, {"two_pass": True}),
    "S128_bf16": (Shape(1, 1024, 32, 4, 128, 128, 4, "bf16"), 403, {}),
    "generic_f32": (Shape(2, 1000, 8, 2, 64, 32, 5, "f32"), 404, {}),
}


@pytest.mark.parametrize("off1", [False, True])
@pytest.mark.parametrize("name", list(ATTN_CASES))
def test_backward_attn(hsa_gpu, name, off1, kernel_path):
    shape, seed, env = ATTN_CASES[name]
    banner(name, "hsa_backward_attn (off by one %d)" % off1)
    if env.get("two_pass"):
        kernel_path(hsa_gpu.HSA_OP_BACKWARD, hsa_gpu.HSA_PATH_TWO_PASS)
    inp, _ = make_case(shape, seed, logit_shift=-4.5 if off1 else 0.0)
    ref = oracle_reference(inp, shape, backward=False)
    dQ_r, dK_r, dV_r, dw_r = oracle.backward(inp["Q"], inp["K"], inp["V"], ref["idx"],
                                             ref["w"], inp["dO"], shape.S, off_by_one=off1,
                                             separate=True)
    dev = {n: to_dev(v, shape) for n, v in inp.items()}
    idx, w = _dev(ref["idx"]), _dev(ref["w"].astype(np.float32))
    dQ, dK, dV, dw = hsa_gpu.hsa_backward_attn(dev["Q"], dev["K"], dev["V"], idx, w, dev["dO"],
                                               shape.S, off_by_one=off1)
    torch.cuda.synchronize()
    for n, g_, r in (("dQ", dQ, dQ_r), ("dK", dK, dK_r), ("dV", dV, dV_r)):
        assert_close(n, shape, g_, r)
    # dw: a sum over heads of fp32 dot products of bf16 rows; the gradient bound
    assert_close("dw", shape, dw, dw_r)
    # accumulation: a second call adds its dw to the first
    _, _, _, dw2 = hsa_gpu.hsa_backward_attn(dev["Q"], dev["K"], dev["V"], idx, w, dev["dO"],
                                             shape.S, off_by_one=off1, dw=dw.clone(),
                                             accumulate_dw=True)
    torch.cuda.synchronize()
    assert torch.allclose(dw2, 2 * dw, rtol=1e-6, atol=0)


@pytest.mark.parametrize("stick", [False, True])
@pytest.mark.parametrize("dsel,dtype", [(1024, "bf16"), (128, "bf16"), (64, "f32")])
def test_select_backward(hsa_gpu, dsel, dtype, stick):
    B, L, G, S, k = 2, 1024, 2, 32, 8
    banner("selbwd_%d_%s_stick%d" % (dsel, dtype, stick), "hsa_select_backward")
    Qs, Ks = selection_inputs(B, L, G, S, k, dsel, 500 + dsel, bf16=dtype == "bf16",
                              stick=stick)
    idx, w, _, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
    dw = hsa_synth.philox(501, 1).standard_normal(w.shape).astype(np.float32)
    dQs_r, dKs_r, _ = oracle.select_backward(Qs, Ks, idx, w, dw, G, S, stick=stick)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dQs, dKs = hsa_gpu.hsa_select_backward(_dev(Qs, tdt), _dev(Ks), _dev(idx),
                                           _dev(w.astype(np.float32)), _dev(dw), G, S,
                                           stick_breaking=stick)
    torch.cuda.synchronize()
    shape = Shape(B, L, G, G, dsel, S, k, dtype)
    assert_close("dQs", shape, dQs, dQs_r)
    assert_close("dKs", shape, dKs, dKs_r)
    # chunks nobody could select (the last one) get zeros
    assert torch.all(dKs[:, -1] == 0)


@pytest.mark.parametrize("stick,off1", [(False, False), (True, True)])
def test_three_layers_share_one_selection(hsa_gpu, stick, off1):
    """Sec. 4.4's setting: one selection over inputs of their own (d_sel = h d_h = 1024)
    serves three attention layers; forward per layer, backward per layer with dw
    accumulated, then the selection backward, all on the GPU, against the oracle."""
    shape = Shape(1, 2048, 16, 2, 128, 64, 8, "bf16")
    B, L, H, G, d, S, k = shape.B, shape.L, shape.H, shape.G, shape.d, shape.S, shape.k
    dsel = (H // G) * d
    banner("shared_x3_stick%d_off%d" % (stick, off1), "select once, 3 layers fwd + bwd")
    Qs, Ks = selection_inputs(B, L, G, S, k, dsel, 601, stick=stick)
    layers = [make_case(shape, 610 + l, gap=False, logit_shift=-1.5 if off1 else 0.0)[0]
              for l in range(3)]
    idx_r, w_r, gap, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
    idx, w = hsa_gpu.hsa_select_topk(_dev(Qs, torch.bfloat16), _dev(Ks), G, S, k,
                                     stick_breaking=stick)
    torch.cuda.synchronize()
    assert_indices(idx, idx_r, gap, S)
    assert np.max(np.abs(w.cpu().numpy() - w_r)) <= W_ATOL
    dw = torch.zeros((B, L, G, k), dtype=torch.float32, device="cuda")
    dw_r = np.zeros(w_r.shape)
    for l, inp in enumerate(layers):
        dev = {n: to_dev(v, shape) for n, v in inp.items()}
        O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, S, off_by_one=off1)
        got = hsa_gpu.hsa_backward_attn(dev["Q"], dev["K"], dev["V"], idx, w, dev["dO"], S,
                                        off_by_one=off1, dw=dw, accumulate_dw=l > 0)
        torch.cuda.synchronize()
        O_r = oracle.forward(inp["Q"], inp["K"], inp["V"], idx_r, w_r, S, off_by_one=off1)
        O_abs = oracle.forward(inp["Q"], inp["K"], np.abs(inp["V"]), idx_r, np.abs(w_r), S,
                               off_by_one=off1)
        assert_close("O[%d]" % l, shape, O, O_r, o_abs=O_abs)
        want = oracle.backward(inp["Q"], inp["K"], inp["V"], idx_r, w_r, inp["dO"], S,
                               stick=stick, off_by_one=off1, separate=True)
        for n, g_, r in zip(("dQ", "dK", "dV"), got[:3], want[:3]):
            assert_close("%s[%d]" % (n, l), shape, g_, r)
        dw_r += want[3]
    sel_shape = Shape(B, L, G, G, dsel, S, k, "bf16")
    assert_close("dw", sel_shape, dw, dw_r)
    dQs, dKs = hsa_gpu.hsa_select_backward(_dev(Qs, torch.bfloat16), _dev(Ks), idx, w, dw, G, S,
                                           stick_breaking=stick)
    torch.cuda.synchronize()
    dQs_r, dKs_r, _ = oracle.select_backward(Qs, Ks, idx_r, w_r, dw_r, G, S, stick=stick)
    assert_close("dQs", sel_shape, dQs, dQs_r)
    assert_close("dKs", sel_shape, dKs, dKs_r)
