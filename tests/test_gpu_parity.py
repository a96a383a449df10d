"""GPU parity: every entry point of the HIP library against the fp64 oracle.

Sizes are small enough for the oracle to finish in seconds, yet span several query tiles,
several landmark blocks and ragged tails.  Every case prints its name before the GPU work.
"""
import numpy as np
import pytest
import torch

import hsa_synth
import oracle
from parity import (W_ATOL, assert_close, assert_indices, attention_abs, check_decode,
                    decode_case, make_case, oracle_reference, to_dev, torch_dtype)

pytestmark = pytest.mark.gpu

Shape = hsa_synth.HsaShape

CASES = {
    # name: (shape, seed, kind[, per-chunk key offset scale mu_std; default 0.5, 0 for
    # "lowrank"])
    "tiny_f32": (Shape(1, 1024, 4, 1, 64, 64, 4, "f32"), 1, "iid"),
    "L4K_like_bf16": (Shape(2, 1024, 16, 2, 128, 64, 8, "bf16"), 2, "iid"),
    "long_like_bf16": (Shape(1, 2048, 16, 2, 128, 64, 8, "bf16"), 3, "long"),
    "wide_like_bf16": (Shape(1, 1024, 32, 4, 128, 128, 4, "bf16"), 5, "lowrank"),
    "ragged_f32": (Shape(2, 1000, 8, 2, 64, 32, 5, "f32"), 11, "iid"),
    "ragged_bf16": (Shape(1, 777, 6, 2, 64, 16, 7, "bf16"), 12, "iid"),
    "h1_S128_bf16": (Shape(1, 1100, 3, 3, 128, 128, 3, "bf16"), 13, "iid"),
    "k_exceeds_chunks_f32": (Shape(1, 300, 4, 2, 64, 64, 8, "f32"), 14, "iid"),
    "no_candidates_bf16": (Shape(2, 50, 8, 1, 128, 64, 4, "bf16"), 15, "iid"),
    "ragged_mfma_bf16": (Shape(1, 1000, 16, 2, 128, 64, 8, "bf16"), 16, "iid"),
    "wide_k16_bf16": (Shape(1, 2304, 32, 4, 128, 128, 16, "bf16"), 17, "lowrank"),
    "k24_bf16": (Shape(1, 2048, 16, 2, 128, 32, 24, "bf16"), 18, "iid"),
    # the largest k (32 slots: the widest selection lists, slot tables and dQ completion)
    "k32_bf16": (Shape(1, 2560, 16, 2, 128, 64, 32, "bf16"), 25, "iid"),
    "k20_d64_f32": (Shape(1, 1500, 4, 2, 64, 32, 20, "f32"), 19, "iid"),
    # float32 with d = 128 (the largest float32 chunk: S d = 8192), generic kernels
    "f32_d128": (Shape(1, 1024, 8, 2, 128, 64, 4, "f32"), 22, "iid"),
    # keys dominated by their chunk's offset (about 23 times the per-key spread): dQ is a
    # strongly cancelling sum over each chunk's keys
    "key_offset_bf16": (Shape(1, 1024, 16, 2, 128, 64, 8, "bf16"), 21, "iid", 2.0),
    # more than 1024 chunks: the selection bitmap is built over two chunk ranges (generic
    # key pass, and the chunk-major forward and fused backward)
    "C1062_S16_f32": (Shape(1, 17000, 2, 1, 64, 16, 4, "f32"), 23, "iid"),
    "C1040_bf16": (Shape(1, 66560, 8, 1, 128, 64, 2, "bf16"), 24, "iid"),
    # the most query heads per KV head (16; generic kernels, the selection's head sum in
    # several load rounds), ragged length
    "h16_bf16": (Shape(1, 1100, 16, 1, 128, 64, 8, "bf16"), 26, "iid"),
    # one slot: every weight is 1 and the score gradient vanishes (ds = w (dw - w dw) = 0)
    "k1_bf16": (Shape(1, 1024, 16, 2, 128, 64, 1, "bf16"), 27, "iid"),
}

_cache = {}


def case(name):
    if name not in _cache:
        shape, seed, kind, *rest = CASES[name]
        mu_std = rest[0] if rest else (0.0 if kind == "lowrank" else 0.5)
        inp, stats = make_case(shape, seed, kind=kind, mu_std=mu_std)
        ref = oracle_reference(inp, shape)
        dev = {n: to_dev(v, shape) for n, v in inp.items()}
        _cache[name] = (shape, inp, ref, dev)
    return _cache[name]


def banner(name, what):
    print("\n[gpu] %s: %s" % (name, what), flush=True)


@pytest.mark.parametrize("name", list(CASES))
def test_landmarks(hsa_gpu, name):
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_landmarks")
    Kbar = hsa_gpu.hsa_landmarks(dev["K"], shape.S)
    torch.cuda.synchronize()
    got = Kbar.cpu().numpy().astype(np.float64)
    want = ref["Kbar"]
    assert got.shape == want.shape
    if want.size:
        err = np.max(np.abs(got - want))
        assert err <= 1e-6 * np.max(np.abs(want)) + 1e-7, err


def test_landmarks_exact_and_bf16_cache(hsa_gpu):
    banner("exact", "hsa_landmarks on exactly representable keys; bf16 output")
    g = hsa_synth.philox(7, 1)
    K = (g.integers(-64, 64, size=(2, 512, 2, 128)) / 16.0).astype(np.float32)
    Kd = torch.from_numpy(K).cuda().to(torch.bfloat16)
    want = oracle.landmarks(K, 64)
    got = hsa_gpu.hsa_landmarks(Kd, 64).cpu().numpy()
    assert np.array_equal(got.astype(np.float64), want)
    got16 = hsa_gpu.hsa_landmarks(Kd, 64, kbar_dtype=torch.bfloat16)
    want16 = hsa_synth.round_bf16(want.astype(np.float32))
    assert np.array_equal(got16.float().cpu().numpy(), want16)
    # partial range leaves the other chunks untouched
    out = torch.full((2, 8, 2, 128), 7.0, device="cuda")
    hsa_gpu.hsa_landmarks(Kd, 64, chunk_begin=2, chunk_end=5, out=out)
    o = out.cpu().numpy()
    assert np.all(o[:, :2] == 7.0) and np.all(o[:, 5:] == 7.0)
    assert np.array_equal(o[:, 2:5].astype(np.float64), want[:, 2:5])


@pytest.mark.parametrize("name", list(CASES))
def test_select(hsa_gpu, name):
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_select_topk")
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k)
    torch.cuda.synchronize()
    sure, loose = assert_indices(idx, ref["idx"], ref["gap"], shape.S)
    assert loose == 0
    err = np.max(np.abs(w.cpu().numpy() - ref["w"])) if w.numel() else 0.0
    assert err <= W_ATOL, err


@pytest.mark.parametrize("name", list(CASES))
def test_forward(hsa_gpu, name):
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_forward (oracle selection)")
    idx = torch.from_numpy(ref["idx"]).cuda()
    w = torch.from_numpy(ref["w"].astype(np.float32)).cuda()
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    torch.cuda.synchronize()
    assert_close("O", shape, O, ref["O"], o_abs=ref["O_abs"])


@pytest.mark.parametrize("name", list(CASES))
def test_backward(hsa_gpu, name):
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_backward (oracle selection)")
    idx = torch.from_numpy(ref["idx"]).cuda()
    w = torch.from_numpy(ref["w"].astype(np.float32)).cuda()
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    dQ, dK, dV = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"],
                                      shape.S)
    torch.cuda.synchronize()
    assert_close("dQ", shape, dQ, ref["dQ"])
    assert_close("dK", shape, dK, ref["dK"])
    assert_close("dV", shape, dV, ref["dV"])


@pytest.mark.parametrize("name", ["tiny_f32", "L4K_like_bf16", "ragged_bf16", "wide_like_bf16"])
def test_end_to_end_pipeline(hsa_gpu, name):
    """landmarks -> select -> forward -> backward, all on the GPU."""
    shape, inp, ref, dev = case(name)
    banner(name, "pipeline")
    Kbar = hsa_gpu.hsa_landmarks(dev["K"], shape.S)
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k)
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    dQ, dK, dV = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"],
                                      shape.S)
    torch.cuda.synchronize()
    assert_indices(idx, ref["idx"], ref["gap"], shape.S)
    assert_close("O", shape, O, ref["O"], o_abs=ref["O_abs"])
    for n, t in (("dQ", dQ), ("dK", dK), ("dV", dV)):
        assert_close(n, shape, t, ref[n])


@pytest.mark.parametrize("name", ["L4K_like_bf16", "wide_like_bf16", "tiny_f32", "C1062_S16_f32"])
def test_backward_is_bitwise_deterministic(hsa_gpu, name):
    """Two calls give the same bits: the fused pass (L4K_like), the two-pass backward with
    its key pass split over workgroups (wide_like, S = 128) and the generic kernels with
    their per-split partials (tiny, and more than 1024 chunks)."""
    shape, inp, ref, dev = case(name)
    banner(name, "backward determinism")
    Kbar = hsa_gpu.hsa_landmarks(dev["K"], shape.S)
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k)
    r1 = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"], shape.S)
    r2 = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"], shape.S)
    torch.cuda.synchronize()
    for a, b in zip(r1, r2):
        assert torch.equal(a, b)


@pytest.mark.parametrize("name", ["L4K_like_bf16", "C1040_bf16", "tiny_f32"])
def test_forward_is_bitwise_deterministic(hsa_gpu, name):
    """Two calls give the same bits: the tile-major forward (L4K_like), the chunk-major one
    with its per-(token, slot) partials summed in slot order (more than 256 chunks) and the
    generic kernel."""
    shape, inp, ref, dev = case(name)
    banner(name, "forward determinism")
    idx = torch.from_numpy(ref["idx"]).cuda()
    w = torch.from_numpy(ref["w"].astype(np.float32)).cuda()
    o1 = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    o2 = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_outputs_fully_overwritten(hsa_gpu):
    shape, inp, ref, dev = case("ragged_bf16")
    banner("ragged_bf16", "overwrite semantics")
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    idx = torch.full((shape.B, shape.L, shape.G, shape.k), 12345, dtype=torch.int32,
                     device="cuda")
    w = torch.full_like(idx, 0, dtype=torch.float32).fill_(float("nan"))
    hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k, idx=idx, w=w)
    O = torch.full_like(dev["Q"], float("nan"))
    hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S, out=O)
    outs = tuple(torch.full_like(x, float("nan")) for x in (dev["Q"], dev["K"], dev["V"]))
    hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"], shape.S,
                         out=outs)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), ref["idx"])
    for t in (w, O) + outs:
        assert torch.isfinite(t.float()).all()


@pytest.mark.parametrize("kbar_dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode(hsa_gpu, dtype, kbar_dtype):
    shape = Shape(3, 4096 + 64, 16, 2, 128 if dtype == "bf16" else 64, 64, 8, dtype)
    banner("decode_%s_kbar_%s" % (dtype, kbar_dtype), "hsa_decode")
    lens = [4096, 4096 + 40, 1000]            # full chunks, a partial tail, a short cache
    inp, Kbar = decode_case(shape, 21, lens, kbar_dtype)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, 64, 8,
                                   cache_len=cache_len)
    torch.cuda.synchronize()
    check_decode(shape, inp, Kbar, lens, o, idx, w)
    for b in range(3):
        for g in range(2):
            p = inp["planted"][b, g].item()
            if p < lens[b] // 64:          # the planted chunk is a candidate: it must win
                assert p in idx[b, g].tolist()


@pytest.mark.parametrize("k", [3, 20])
def test_decode_many_slots(hsa_gpu, k):
    """k above the 8 waves of the attention stage (a wave attends several chunks in turn)
    and caches with fewer complete chunks than k."""
    shape = Shape(2, 4096, 16, 2, 128, 64, k, "bf16")
    banner("decode_k%d" % k, "hsa_decode")
    lens = [64 * 5 + 7, 4096]
    inp, Kbar = decode_case(shape, 23, lens)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, 64, k,
                                   cache_len=cache_len)
    torch.cuda.synchronize()
    check_decode(shape, inp, Kbar, lens, o, idx, w)
    assert np.all(idx.cpu().numpy()[0, :, 5:] == -1)     # 5 complete chunks in sequence 0


@pytest.mark.parametrize("stick,off1", [(False, False), (True, True)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_short_caches(hsa_gpu, dtype, stick, off1):
    """Caches of 0, S - 1, S, S + 1 and 2 S + 5 tokens: no candidate (o = 0, idx = -1,
    w = 0), exactly one (w = 1 for the softmax, sigmoid(s) for stick-breaking), two."""
    S = 64
    shape = Shape(5, 4096, 16, 2, 128 if dtype == "bf16" else 64, S, 8, dtype)
    banner("decode_short_%s_stick%d_off%d" % (dtype, stick, off1), "hsa_decode, short caches")
    lens = [0, S - 1, S, S + 1, 2 * S + 5]
    inp, Kbar = decode_case(shape, 25, lens)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, S, 8,
                                   cache_len=cache_len, stick_breaking=stick, off_by_one=off1)
    torch.cuda.synchronize()
    check_decode(shape, inp, Kbar, lens, o, idx, w, stick=stick, off_by_one=off1)
    gi, gw, go = idx.cpu().numpy(), w.cpu().numpy(), o.float().cpu().numpy()
    assert np.all(gi[:2] == -1) and np.all(gw[:2] == 0) and np.all(go[:2] == 0)
    assert np.all(gi[2:4, :, 0] == 0) and np.all(gi[2:4, :, 1:] == -1)
    assert np.all(gi[4, :, :2] == [1, 0]) and np.all(gi[4, :, 2:] == -1)
    if not stick:
        assert np.all(gw[2:4, :, 0] == 1.0) and np.all(gw[2:4, :, 1:] == 0)


def test_decode_matches_forward_row(hsa_gpu):
    """Decode at position t equals row t of the forward (same K, V, landmarks)."""
    shape, inp, ref, dev = case("L4K_like_bf16")
    banner("L4K_like_bf16", "decode vs forward row")
    t = 777
    Kbar = hsa_gpu.hsa_landmarks(dev["K"], shape.S)
    idx, w = hsa_gpu.hsa_select_topk(dev["Q"], Kbar, shape.G, shape.S, shape.k)
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    q = dev["Q"][:, t].contiguous()
    cl = torch.full((shape.B,), t, dtype=torch.int32, device="cuda")
    o, di, dw = hsa_gpu.hsa_decode(q, dev["K"], dev["V"], Kbar, shape.S, shape.k, cache_len=cl)
    torch.cuda.synchronize()
    assert torch.equal(di, idx[:, t])
    assert torch.allclose(dw, w[:, t], rtol=0, atol=1e-6)
    # both sides are rounded to bf16 (a GPU-to-GPU comparison): the element bound with one
    # full ulp
    assert_close("o", shape, o, O[:, t].double().cpu().numpy(), ulps=2.0, contract=False)


def test_empty_batch_is_noop(hsa_gpu):
    banner("empty", "B = 0")
    Q = torch.empty((0, 128, 8, 64), device="cuda", dtype=torch.bfloat16)
    K = torch.empty((0, 128, 2, 64), device="cuda", dtype=torch.bfloat16)
    Kbar = hsa_gpu.hsa_landmarks(K, 64)
    idx, w = hsa_gpu.hsa_select_topk(Q, Kbar, 2, 64, 4)
    O = hsa_gpu.hsa_forward(Q, K, K, idx, w, 64)
    assert O.shape == Q.shape


def _scrambled_selection(ref, shape, seed, repeats):
    """The oracle's selection with empty slots mixed in: -1, the token's own chunk or a
    later one, and an index far past the end; with `repeats`, some slots also repeat the
    token's slot-0 chunk.  Returns (idx, w) as given to the library and the idx the
    oracle sees, where every entry outside [0, floor(t / S)) is -1 (an empty slot)."""
    rng = np.random.default_rng(seed)
    idx = ref["idx"].copy()
    w = rng.uniform(0.05, 1.0, idx.shape).astype(np.float32)
    ncand = (np.arange(shape.L) // shape.S)[None, :, None, None]
    u = rng.random(idx.shape)
    idx = np.where(u < 0.08, -1, idx)
    idx = np.where((u >= 0.08) & (u < 0.16), ncand + rng.integers(0, 3, idx.shape), idx)
    idx = np.where((u >= 0.16) & (u < 0.18), 1 << 30, idx)
    if repeats:
        rep = (rng.random(idx.shape) < 0.15) & (np.arange(shape.k) > 0)
        idx = np.where(rep, idx[..., :1], idx)
    idx = idx.astype(np.int32)
    idx_oracle = np.where((idx < 0) | (idx >= ncand), -1, idx).astype(np.int32)
    return idx, w, idx_oracle


@pytest.mark.parametrize("name", ["ragged_mfma_bf16", "wide_like_bf16", "ragged_f32"])
def test_forward_empty_and_repeated_slots(hsa_gpu, name):
    """Empty slots add nothing; a chunk given in several slots adds each slot's weight."""
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_forward, empty and repeated slots")
    idx, w, idx_o = _scrambled_selection(ref, shape, 31, repeats=True)
    want = oracle.forward(inp["Q"], inp["K"], inp["V"], idx_o, w, shape.S)
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], torch.from_numpy(idx).cuda(),
                            torch.from_numpy(w).cuda(), shape.S)
    torch.cuda.synchronize()
    assert_close("O", shape, O, want, o_abs=attention_abs(inp, idx_o, w, shape.S),
                 contract=False)


@pytest.mark.parametrize("name", ["ragged_mfma_bf16", "wide_like_bf16", "ragged_f32"])
def test_backward_empty_slots(hsa_gpu, name):
    """Empty slots (outside the token's candidates) carry no weight and no gradient."""
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_backward, empty slots")
    idx, w, idx_o = _scrambled_selection(ref, shape, 32, repeats=False)
    # the valid entries left are a subset of the oracle's selection, so they stay distinct
    want = oracle.backward(inp["Q"], inp["K"], inp["V"], idx_o, w, inp["dO"], shape.S)
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    got = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, torch.from_numpy(idx).cuda(),
                               torch.from_numpy(w).cuda(), dev["dO"], shape.S)
    torch.cuda.synchronize()
    for n, g_, r in zip(("dQ", "dK", "dV"), got, want):
        assert_close(n, shape, g_, r, contract=False)


@pytest.mark.parametrize("name", ["L4K_like_bf16", "long_like_bf16", "ragged_mfma_bf16",
                                  "key_offset_bf16", "no_candidates_bf16"])
def test_forward_chunk_major(hsa_gpu, name, kernel_path):
    """The chunk-major forward (the default for bf16, h = 8, d = 128, S = 64 sequences of at
    least 256 chunks), forced on the parity shapes with HSA_PATH_CHUNK_MAJOR."""
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_forward, chunk-major path")
    kernel_path(hsa_gpu.HSA_OP_FORWARD, hsa_gpu.HSA_PATH_CHUNK_MAJOR)
    idx = torch.from_numpy(ref["idx"]).cuda()
    w = torch.from_numpy(ref["w"].astype(np.float32)).cuda()
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], idx, w, shape.S)
    torch.cuda.synchronize()
    assert_close("O", shape, O, ref["O"], o_abs=ref["O_abs"])


def test_forward_chunk_major_repeated_slots(hsa_gpu, kernel_path):
    """Empty and repeated slots on the chunk-major forward: a chunk given in several slots
    adds each slot's weight (one partial carries their sum)."""
    name = "ragged_mfma_bf16"
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_forward, chunk-major path, empty and repeated slots")
    kernel_path(hsa_gpu.HSA_OP_FORWARD, hsa_gpu.HSA_PATH_CHUNK_MAJOR)
    idx, w, idx_o = _scrambled_selection(ref, shape, 31, repeats=True)
    want = oracle.forward(inp["Q"], inp["K"], inp["V"], idx_o, w, shape.S)
    O = hsa_gpu.hsa_forward(dev["Q"], dev["K"], dev["V"], torch.from_numpy(idx).cuda(),
                            torch.from_numpy(w).cuda(), shape.S)
    torch.cuda.synchronize()
    assert_close("O", shape, O, want, o_abs=attention_abs(inp, idx_o, w, shape.S),
                 contract=False)


@pytest.mark.parametrize("name", ["ragged_mfma_bf16", "L4K_like_bf16", "key_offset_bf16"])
def test_backward_repeated_slots(hsa_gpu, name, kernel_path):
    """Slots that repeat a chunk: the fused chunk-major backward (bf16, h = 8, d = 128,
    S = 64) gives the gradient of the forward, which adds each slot's weighted attention, so
    it matches the oracle's slot-by-slot sums."""
    kernel_path(hsa_gpu.HSA_OP_BACKWARD, hsa_gpu.HSA_PATH_FUSED)
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_backward, empty and repeated slots")
    idx, w, idx_o = _scrambled_selection(ref, shape, 33, repeats=True)
    srt = np.sort(idx_o, axis=-1)
    assert ((srt[..., 1:] == srt[..., :-1]) & (srt[..., 1:] >= 0)).any()   # repeats present
    want = oracle.backward(inp["Q"], inp["K"], inp["V"], idx_o, w, inp["dO"], shape.S)
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    got = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, torch.from_numpy(idx).cuda(),
                               torch.from_numpy(w).cuda(), dev["dO"], shape.S)
    torch.cuda.synchronize()
    for n, g_, r in zip(("dQ", "dK", "dV"), got, want):
        assert_close(n, shape, g_, r, contract=False)


@pytest.mark.parametrize("name", ["L4K_like_bf16", "ragged_mfma_bf16", "key_offset_bf16",
                                  "no_candidates_bf16"])
def test_backward_two_pass(hsa_gpu, name, kernel_path):
    """The two-pass MFMA backward (query pass, then key pass), which serves S = 128 and
    is selectable for S = 64 with HSA_PATH_TWO_PASS."""
    shape, inp, ref, dev = case(name)
    banner(name, "hsa_backward, two-pass path")
    kernel_path(hsa_gpu.HSA_OP_BACKWARD, hsa_gpu.HSA_PATH_TWO_PASS)
    idx = torch.from_numpy(ref["idx"]).cuda()
    w = torch.from_numpy(ref["w"].astype(np.float32)).cuda()
    Kbar = torch.from_numpy(ref["Kbar"].astype(np.float32)).cuda()
    dQ, dK, dV = hsa_gpu.hsa_backward(dev["Q"], dev["K"], dev["V"], Kbar, idx, w, dev["dO"],
                                      shape.S)
    torch.cuda.synchronize()
    assert_close("dQ", shape, dQ, ref["dQ"])
    assert_close("dK", shape, dK, ref["dK"])
    assert_close("dV", shape, dV, ref["dV"])


@pytest.mark.parametrize("shape", [Shape(1, 20480, 16, 2, 128, 64, 8, "bf16"),
                                   Shape(1, 8192, 4, 1, 64, 16, 20, "f32")],
                         ids=["C320_bf16", "C512_d64_k20_f32"])
def test_select_many_candidates(hsa_gpu, shape):
    """Sequences with more than 256 complete chunks: the selection splits each tile's
    candidates over its waves and merges their lists."""
    banner("select_%dx%d" % (shape.L, shape.S), "hsa_select_topk, many candidates")
    inp, _ = make_case(shape, 41, kind="iid")
    Kbar_ref = oracle.landmarks(inp["K"], shape.S)
    idx_ref, w_ref, gap, _ = oracle.select(inp["Q"], Kbar_ref, shape.G, shape.S, shape.k)
    Q = to_dev(inp["Q"], shape)
    Kbar = torch.from_numpy(Kbar_ref.astype(np.float32)).cuda()
    idx, w = hsa_gpu.hsa_select_topk(Q, Kbar, shape.G, shape.S, shape.k)
    torch.cuda.synchronize()
    sure, loose = assert_indices(idx, idx_ref, gap, shape.S)
    assert loose == 0
    assert np.max(np.abs(w.cpu().numpy() - w_ref)) <= W_ATOL


@pytest.mark.parametrize("L", [4160, 4161], ids=["64_candidates", "65_candidates"])
def test_select_block_boundary(hsa_gpu, L):
    """The last tokens see exactly 64 candidate chunks (one full block: the selection's
    single-stage form) or 65 (a second block of one chunk: the double-buffered form)."""
    shape = Shape(1, L, 16, 2, 128, 64, 8, "bf16")
    banner("select_L%d" % L, "hsa_select_topk, candidate block boundary")
    inp, _ = make_case(shape, 43, kind="iid")
    Kbar_ref = oracle.landmarks(inp["K"], shape.S)
    idx_ref, w_ref, gap, _ = oracle.select(inp["Q"], Kbar_ref, shape.G, shape.S, shape.k)
    Q = to_dev(inp["Q"], shape)
    Kbar = torch.from_numpy(Kbar_ref.astype(np.float32)).cuda()
    idx, w = hsa_gpu.hsa_select_topk(Q, Kbar, shape.G, shape.S, shape.k)
    torch.cuda.synchronize()
    sure, loose = assert_indices(idx, idx_ref, gap, shape.S)
    assert loose == 0
    assert np.max(np.abs(w.cpu().numpy() - w_ref)) <= W_ATOL
    # no index beyond the last candidate: 63 (L = 4160) or 64 (L = 4161)
    assert int(idx.max()) <= (L - 1) // 64 - 1


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_decode_more_than_64_slices(hsa_gpu, dtype):
    """A cache of more than 64 scan slices (S = 16, 16385 chunks): the merge of the slice
    candidates takes the workgroup tournament instead of the one-wave list merge.  The
    queries are gap-enforced, so all four (b, g) groups are compared index by index."""
    d = 64 if dtype == "f32" else 128
    S, k = 16, 8
    N = (64 * 256 + 1) * S
    shape = Shape(2, N, 16, 2, d, S, k, dtype)
    banner("decode_%d_slices_%s" % (65, dtype), "hsa_decode, tournament merge")
    lens = [N, N - 5 * S - 3]
    inp, Kbar = decode_case(shape, 29, lens)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, S, k,
                                   cache_len=cache_len)
    torch.cuda.synchronize()
    assert check_decode(shape, inp, Kbar, lens, o, idx, w) == 4


def test_decode_f32_d128(hsa_gpu):
    """Decode in float32 with d = 128 (the finish + combine kernels at S d = 8192)."""
    shape = Shape(2, 4096 + 64, 8, 2, 128, 64, 6, "f32")
    banner("decode_f32_d128", "hsa_decode")
    lens = [4096 + 64, 64 * 7 + 9]
    inp, Kbar = decode_case(shape, 31, lens)
    cache_len = torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, idx, w = hsa_gpu.hsa_decode(inp["q"], inp["Kc"], inp["Vc"], Kbar, 64, 6,
                                   cache_len=cache_len)
    torch.cuda.synchronize()
    check_decode(shape, inp, Kbar, lens, o, idx, w)
