"""Full-size parity: the benchmark workloads at their real shapes, run through the same entry
points and workspace sizing as bench.py, checked against the fp64 oracle on sampled outputs
(the oracle computes them one by one: sampled tokens for selection, O and dQ; sampled chunks
for dK and dV, with ds of every token that selected them).

The inputs are the bench's plain draws (no gap enforcement), so selected indices are
compared bit-exactly where the oracle's top-k gap is >= 1e-3; elsewhere the selection must
be a valid one (every chosen chunk's fp64 score within 1e-4 of the oracle's n-th best, the
weights those of the weight rule on the chosen chunks).  O, dQ, dK, dV are compared given
the selection the GPU made (its idx and w are the oracle's inputs), which the selection
checks have validated.
"""
import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import assert_close, check_decode, check_selection, to_dev

pytestmark = pytest.mark.gpu

N_ROWS = 192        # sampled tokens per (b, g) slice
N_CHUNKS = 4        # sampled chunks per slice


def banner(name, what):
    print("\n[gpu] %s: %s" % (name, what), flush=True)


def pipeline(hsa, sh, dev):
    """landmarks -> select -> forward -> backward, as one bench step."""
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    Q, K, V, dO = dev["Q"], dev["K"], dev["V"], dev["dO"]
    Kbar = torch.empty((B, L // S, G, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((B, L, G, k), dtype=torch.int32, device="cuda")
    w = torch.empty((B, L, G, k), dtype=torch.float32, device="cuda")
    O = torch.empty_like(Q)
    grads = (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    p = hsa.make_params(B, L, H, G, d, S, k, Q.dtype)
    ws_f = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_FORWARD)), dtype=torch.uint8,
                       device="cuda")
    ws_b = torch.empty(max(1, hsa.workspace_size(p, hsa.HSA_OP_BACKWARD)), dtype=torch.uint8,
                       device="cuda")
    hsa.hsa_landmarks(K, S, out=Kbar)
    hsa.hsa_select_topk(Q, Kbar, G, S, k, idx=idx, w=w)
    hsa.hsa_forward(Q, K, V, idx, w, S, out=O, workspace=ws_f)
    hsa.hsa_backward(Q, K, V, Kbar, idx, w, dO, S, out=grads, workspace=ws_b)
    torch.cuda.synchronize()
    return Kbar, idx, w, O, grads


def check_slice(name, sh, inp, gpu, b, g, rng, all_rows_ds=False):
    """Sampled parity of one (b, g) slice."""
    Kbar, idx, w, O, (dQ, dK, dV) = gpu
    L, G, h, d, S, k = sh.L, sh.G, sh.H // sh.G, sh.d, sh.S, sh.k
    C = L // S
    dm = oracle.dims(L, h, d, S, k)
    hs = slice(g * h, (g + 1) * h)
    Qs = np.ascontiguousarray(inp["Q"][b, :, hs], dtype=np.float64)
    dOs = np.ascontiguousarray(inp["dO"][b, :, hs], dtype=np.float64)
    Ks = np.ascontiguousarray(inp["K"][b, :, g], dtype=np.float64)
    Vs = np.ascontiguousarray(inp["V"][b, :, g], dtype=np.float64)
    gKbar = Kbar[b, :, g].cpu().numpy().astype(np.float64)
    gi = np.ascontiguousarray(idx[b, :, g].cpu().numpy())
    gw = w[b, :, g].cpu().numpy().astype(np.float64)

    # landmarks (all chunks of the slice)
    kb_ref = oracle.landmarks_slice(dm, Ks)
    assert np.max(np.abs(gKbar - kb_ref)) <= 1e-6 * np.max(np.abs(kb_ref)) + 1e-7

    # selection on sampled tokens (first and last tokens included)
    rows = np.unique(np.concatenate([[0, S, L - 1], rng.choice(L, N_ROWS, replace=False)]))
    ridx, rw, gap, _ = oracle.select_slice(dm, Qs, kb_ref, rows)
    exact, valid = check_selection(dm, Qs[rows], kb_ref, rows, gi[rows], gw[rows], ridx, rw, gap)
    print("[parity] %s b=%d g=%d: %d sampled tokens index-exact, %d below the gap checked "
          "for validity" % (name, b, g, exact, valid), flush=True)

    # forward on the sampled tokens, given the GPU's selection
    o_ref = oracle.forward_slice(dm, Qs, Ks, Vs, gi, gw, rows)
    o_abs = oracle.forward_slice(dm, Qs, Ks, np.abs(Vs), gi, np.abs(gw), rows)
    trows = torch.from_numpy(rows).cuda()
    assert_close("O", sh, O[b, trows][:, hs], o_ref, o_abs=o_abs)

    # dQ on the sampled tokens
    dq_ref, _ = oracle.backward_q_slice(dm, Qs, Ks, Vs, gKbar, gi, gw, dOs, rows)
    assert_close("dQ", sh, dQ[b, trows][:, hs], dq_ref)

    # dK, dV of sampled chunks: ds of every token that selected one of them
    chunks = np.unique(np.concatenate([[0, C - 1], rng.choice(C, N_CHUNKS, replace=False)]))
    if all_rows_ds:
        sel_rows = np.arange(L)
    else:
        sel_rows = np.nonzero(np.isin(gi, chunks).any(axis=1))[0]
    ds = np.zeros((L, k))
    if sel_rows.size:
        _, ds_rows = oracle.backward_q_slice(dm, Qs, Ks, Vs, gKbar, gi, gw, dOs, sel_rows)
        ds[sel_rows] = ds_rows
    dk_ref, dv_ref = oracle.backward_kv_slice(dm, Qs, Ks, Vs, gi, gw, dOs, ds, chunks)
    key_rows = (chunks[:, None] * S + np.arange(S)[None, :]).reshape(-1)
    tkeys = torch.from_numpy(key_rows).cuda()
    assert_close("dK", sh, dK[b, tkeys, g], dk_ref.reshape(-1, d))
    assert_close("dV", sh, dV[b, tkeys, g], dv_ref.reshape(-1, d))


def run_training(hsa_gpu, name, slices):
    wl = hsa_synth.WORKLOADS[name]
    sh = wl["shape"]
    banner(name, "full-size pipeline (%s)" % (sh,))
    inp = hsa_synth.make_training_inputs(name)
    dev = {n: to_dev(v, sh) for n, v in inp.items()}
    gpu = pipeline(hsa_gpu, sh, dev)
    del dev
    rng = np.random.default_rng(7)
    for b, g in slices:
        banner(name, "oracle samples of slice b=%d g=%d" % (b, g))
        check_slice(name, sh, inp, gpu, b, g, rng)


def test_fullsize_L4K(hsa_gpu):
    run_training(hsa_gpu, "L4K_bf16", [(0, 0), (7, 1)])


def test_fullsize_L64K(hsa_gpu):
    run_training(hsa_gpu, "L64K_bf16", [(0, 1)])


def test_fullsize_wide_L16K(hsa_gpu):
    run_training(hsa_gpu, "wide_L16K_bf16", [(3, 2)])


def test_fullsize_decode_1M(hsa_gpu):
    """The bench's decode step (8 sequences at 2^20 cached tokens, bf16 landmark cache) for
    two sampled sequences: the oracle decodes against the same landmark cache; groups below
    the gap are checked for a valid selection."""
    wl = hsa_synth.WORKLOADS["decode_1M_bf16"]
    sh = wl["shape"]
    banner("decode_1M_bf16", "full-size decode")
    inp = hsa_synth.make_decode_inputs(sh, wl["seed"], device="cuda")
    q, Kc, Vc = inp["q"], inp["Kc"], inp["Vc"]
    kbar = hsa_gpu.hsa_landmarks(Kc, sh.S, kbar_dtype=torch.bfloat16)
    o, idx, w = hsa_gpu.hsa_decode(q, Kc, Vc, kbar, sh.S, sh.k)
    torch.cuda.synchronize()
    for b in (0, 5):
        banner("decode_1M_bf16", "oracle decode of sequence %d" % b)
        sub = {"q": q[b:b + 1].cpu(), "Kc": Kc[b:b + 1].cpu(), "Vc": Vc[b:b + 1].cpu()}
        check_decode(sh, sub, kbar[b:b + 1], [sh.L], o[b:b + 1], idx[b:b + 1], w[b:b + 1],
                     require_exact=False)
        gi = idx[b:b + 1].cpu().numpy()
        for g in range(sh.G):
            assert int(inp["planted"][b, g]) in gi[0, g].tolist()


def test_fullsize_decode_1M_host_cache(hsa_gpu):
    """The bench's decode step with the key / value cache in pinned host memory: bitwise the
    outputs of the HBM-resident decode, and one sequence against the oracle."""
    wl = hsa_synth.WORKLOADS["decode_1M_bf16"]
    sh = wl["shape"]
    banner("decode_1M_bf16", "full-size decode, cache in host memory")
    inp = hsa_synth.make_decode_inputs(sh, wl["seed"], device="cuda")
    q, Kc, Vc = inp["q"], inp["Kc"], inp["Vc"]
    kbar = hsa_gpu.hsa_landmarks(Kc, sh.S, kbar_dtype=torch.bfloat16)
    o, idx, w = hsa_gpu.hsa_decode(q, Kc, Vc, kbar, sh.S, sh.k)
    Kh = torch.empty(Kc.shape, dtype=Kc.dtype, pin_memory=True)
    Vh = torch.empty(Vc.shape, dtype=Vc.dtype, pin_memory=True)
    Kh.copy_(Kc)
    Vh.copy_(Vc)
    oh, idxh, wh = hsa_gpu.hsa_decode_host(q, Kh, Vh, kbar, sh.S, sh.k)
    torch.cuda.synchronize()
    assert torch.equal(idxh, idx) and torch.equal(wh, w) and torch.equal(oh, o)
    b = 2
    banner("decode_1M_bf16", "oracle decode of sequence %d" % b)
    sub = {"q": q[b:b + 1].cpu(), "Kc": Kh[b:b + 1], "Vc": Vh[b:b + 1]}
    check_decode(sh, sub, kbar[b:b + 1], [sh.L], oh[b:b + 1], idxh[b:b + 1], wh[b:b + 1],
                 require_exact=False)


def test_fullsize_shared_x3_L4K(hsa_gpu):
    """The bench's step of three layers sharing one selection over inputs of its own
    (B8 L4096 H16/G2 d128 S64 k8, d_sel = 1024): selection, per-layer forward and
    attention-only backward (dw accumulated), selection backward; sampled tokens and chunks
    of two slices against the oracle, given the GPU's selection (checked on its own)."""
    name = "shared_x3_L4K_bf16"
    sh = hsa_synth.WORKLOADS[name]["shape"]
    B, L, H, G, d, S, k = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S, sh.k
    h, C = H // G, L // S
    dsel = h * d
    banner(name, "full-size shared-selection step")
    layers, Qs, Ks = hsa_synth.make_shared_selection_inputs(name)
    idx, w = hsa_gpu.hsa_select_topk(Qs, Ks, G, S, k)
    dw = torch.empty((B, L, G, k), dtype=torch.float32, device="cuda")
    outs = []
    for i, lay in enumerate(layers):
        O = hsa_gpu.hsa_forward(lay["Q"], lay["K"], lay["V"], idx, w, S)
        grads = hsa_gpu.hsa_backward_attn(lay["Q"], lay["K"], lay["V"], idx, w, lay["dO"], S,
                                          dw=dw, accumulate_dw=i > 0)
        outs.append((O,) + tuple(grads[:3]))
    dQs, dKs = hsa_gpu.hsa_select_backward(Qs, Ks, idx, w, dw, G, S)
    torch.cuda.synchronize()
    rng = np.random.default_rng(17)
    f64 = lambda t: np.ascontiguousarray(t.float().cpu().numpy(), dtype=np.float64)
    for b, g in ((0, 0), (7, 1)):
        banner(name, "oracle samples of slice b=%d g=%d" % (b, g))
        hs = slice(g * h, (g + 1) * h)
        gi = np.ascontiguousarray(idx[b, :, g].cpu().numpy())
        gw = f64(w[b, :, g])
        rows = np.unique(np.concatenate([[0, S, L - 1], rng.choice(L, N_ROWS, replace=False)]))
        trows = torch.from_numpy(rows).cuda()
        # selection on the sampled tokens
        dms = oracle.dims(L, 1, dsel, S, k)
        Qss, Kss = f64(Qs[b, :, g]).reshape(L, 1, dsel), f64(Ks[b, :, g])
        ridx, rw, gap, _ = oracle.select_slice(dms, Qss, Kss, rows)
        check_selection(dms, Qss[rows], Kss, rows, gi[rows], gw[rows], ridx, rw, gap)
        # each layer: O and dQ of the sampled tokens, dK and dV of sampled chunks
        dm = oracle.dims(L, h, d, S, k, sep=True)
        chunks = np.unique(np.concatenate([[0, C - 1], rng.choice(C, N_CHUNKS, replace=False)]))
        key_rows = torch.from_numpy((chunks[:, None] * S + np.arange(S)[None, :]).reshape(-1)).cuda()
        dw_ref = np.zeros((rows.size, k))
        for lay, (O, dQ, dK, dV) in zip(layers, outs):
            Ql, dOl = f64(lay["Q"][b, :, hs]), f64(lay["dO"][b, :, hs])
            Kl, Vl = f64(lay["K"][b, :, g]), f64(lay["V"][b, :, g])
            o_ref = oracle.forward_slice(dm, Ql, Kl, Vl, gi, gw, rows)
            o_abs = oracle.forward_slice(dm, Ql, Kl, np.abs(Vl), gi, np.abs(gw), rows)
            assert_close("O", sh, O[b, trows][:, hs], o_ref, o_abs=o_abs)
            dq_ref, _, dwl = oracle.backward_q_slice(dm, Ql, Kl, Vl, np.zeros((C, d)), gi, gw,
                                                     dOl, rows, with_dw=True)
            assert_close("dQ", sh, dQ[b, trows][:, hs], dq_ref)
            dw_ref += dwl
            dk_ref, dv_ref = oracle.backward_kv_slice(dm, Ql, Kl, Vl, gi, gw, dOl,
                                                      np.zeros((L, k)), chunks)
            assert_close("dK", sh, dK[b, key_rows, g], dk_ref.reshape(-1, d))
            assert_close("dV", sh, dV[b, key_rows, g], dv_ref.reshape(-1, d))
        assert_close("dw", sh, dw[b, trows, g], dw_ref)
        # the selection backward of the slice, given the GPU's summed dw
        dqs_ref, dks_ref, _ = oracle.select_backward_slice(dms, Qss, Kss, gi, gw, f64(dw[b, :, g]))
        assert_close("dQs", sh, dQs[b, trows, g], dqs_ref[rows, 0])
        assert_close("dKs", sh, dKs[b, :, g], dks_ref)
