"""Full-size parity: the benchmark workloads at their real shapes, run through the same entry
points and workspace sizing as bench.py, checked against the fp64 oracle on sampled outputs
(the oracle computes them one by one: sampled tokens for selection, O and dQ; sampled chunks
for dK and dV, with ds of every token that selected them).

The inputs are the bench's plain draws (no gap enforcement), so selected indices are
compared bit-exactly where the oracle's top-k gap is >= 1e-3 and checked for validity
elsewhere.  O, dQ, dK, dV are compared given the selection the GPU made (its idx and w are
the oracle's inputs): the selection itself is checked separately.
"""
import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import W_ATOL, assert_close, assert_indices, to_dev

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
    assert_indices(torch.from_numpy(gi[rows][None, :, None]), ridx[None, :, None],
                   gap[None, :, None], S, tokens=rows)
    sure = gap >= 1e-3
    assert np.max(np.abs(gw[rows][sure] - rw[sure]), initial=0.0) <= W_ATOL

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
    two sampled sequences: the oracle decodes against the same landmark cache."""
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
        ro, ridx, rw, rgap = oracle.decode(q[b:b + 1].cpu(), Kc[b:b + 1].cpu(),
                                           Vc[b:b + 1].cpu(), kbar[b:b + 1].float().cpu(),
                                           [sh.L], sh.S, sh.k)
        ro_abs = oracle.decode(q[b:b + 1].cpu(), Kc[b:b + 1].cpu(), Vc[b:b + 1].abs().cpu(),
                               kbar[b:b + 1].float().cpu(), [sh.L], sh.S, sh.k)[0]
        gi = idx[b:b + 1].cpu().numpy()
        sure = rgap >= 1e-3
        assert np.array_equal(gi[sure], ridx[sure])
        assert np.max(np.abs(w[b:b + 1].cpu().numpy() - rw)[sure], initial=0.0) <= W_ATOL
        assert_close("o", sh, o[b:b + 1], ro, o_abs=ro_abs)
        for g in range(sh.G):
            assert int(inp["planted"][b, g]) in gi[0, g].tolist()
