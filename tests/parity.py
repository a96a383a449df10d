"""Shared helpers of the GPU parity tests: seeded inputs, the oracle reference and the
tolerances (written here, used by every GPU test).

Tolerances (fixed in advance, independent of the measured error):
  - fp32 mode: max-abs error <= 1e-4 for outputs and gradients;
  - bf16 mode, the operator's bound (2e-2 of the reference's RMS), applied to the error of
    the computation: |got - ref| <= 2e-2 * RMS(ref) + hulp(got) element-wise, where
    hulp(got) is half an ulp of bfloat16 at the stored value, i.e. the most the rounding of
    an exact result to the bf16 output can add.  No bf16-output implementation can do
    better: the oracle's own fp64 result rounded to bf16 misses max |err| <= 2e-2 RMS by up
    to 3.6x on these tensors (max |ref| / RMS(ref) is 6 to 30, and half an ulp is up to
    2^-8 |ref|).  Asserted wherever the chunk weights come from a selection (softmax or
    stick-breaking), for O, dQ, dK, dV, decode o, dw and the selection backward's dQs, dKs;
    tests that inject unnormalised weights of their own skip it (contract=False);
  - bf16 mode, in addition, element-wise bounds that follow the rounding steps:
      attention outputs O: |got - ref| <= 2^-8 (O_abs + |ref|), with
      O_abs = sum_i |w_i| sum_s P_s |V_s| (the same operator applied to |V| and |w|): a
      bf16 rounding of the weighted probabilities w P / sum (relative error <= 2^-9) and
      one of the output (<= 2^-9 |O|), every other step fp32 on exact bf16 products, and a
      factor-2 margin (the kernels carry w P as a bf16 pair hi + lo, so their error stays
      well inside it);
      gradients: |got - ref| <= 2e-2 * RMS(ref) + 2^-8 * |ref|;
  - selected chunk indices: bit-exact for every token whose oracle top-k score gap is
    >= 1e-3; below that gap, a valid selection: the right count, distinct, descending,
    candidates only, every chosen chunk's fp64 score >= the oracle's n-th best score - 1e-4
    (fp32 score error is ~1e-6 at most), and weights equal to the weight rule applied to
    the oracle's scores of the chosen chunks within 1e-5;
  - chunk weights: max-abs <= 1e-5 (fp32 softmax of fp32 scores whose error is ~1e-7);
  - landmarks: max-abs <= 1e-6 * max|Kbar| + 1e-7 (fp32 mean of S values).
Every bf16 comparison records max(|err| - hulp(got)) / (2e-2 RMS(ref)) (the contract ratio,
asserted <= 1), the raw max |err| / (2e-2 RMS(ref)) and the same raw ratio of the oracle's
result rounded to bf16 (the floor); the session prints them.
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch

import hsa_synth
import oracle
from oracle.gapfix import enforce_gap

MIN_GAP = 1e-3
F32_ATOL = 1e-4
BF16_RMS_FRAC = 2e-2
W_ATOL = 1e-5
SCORE_SLACK = 1e-4

# (test id, tensor name, contract ratio, max |err| / element bound, asserted, raw ratio,
#  rounding floor)
RATIOS = []


def half_ulp_bf16(x: np.ndarray) -> np.ndarray:
    """Half an ulp of bfloat16 (8 significant bits) at each value: 2^(e - 8) for |x| in
    [2^e, 2^(e + 1)), 0 at 0."""
    a = np.abs(x)
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(e - 8.0), 0.0)


def torch_dtype(shape):
    return torch.bfloat16 if shape.dtype == "bf16" else torch.float32


def to_dev(x: np.ndarray, shape) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(torch_dtype(shape))


def logit_shift_coord(shape, shift):
    """The value a (bf16-exact) whose square over sqrt(d) is about |shift|: coordinate 0 of
    every key set to sign(shift) a and of every query to a adds sign(shift) a^2 / sqrt(d)
    to every intra-chunk logit beta q.k (beta = 1/sqrt(d))."""
    a = math.sqrt(abs(shift) * math.sqrt(shape.d))
    return float(hsa_synth.round_bf16(np.array([a], np.float32))[0])


def make_case(shape, seed, kind="iid", mu_std=0.5, gap=True, logit_shift=0.0):
    """Seeded inputs of one case, gap-enforced.  logit_shift moves every intra-chunk logit
    by about that constant (see logit_shift_coord): the softmax does not see it, the
    softmax off by one does.  Every key then has the same coordinate 0, so a token's
    selection scores all move by one constant and its selection and gap do not change; the
    keys are set before the gap enforcement (which may redraw queries) and the queries
    after it."""
    inp = hsa_synth.make_training_inputs(shape, seed, kind=kind, mu_std=mu_std)
    if logit_shift:
        a = logit_shift_coord(shape, logit_shift)
        inp["K"][..., 0] = math.copysign(a, logit_shift)
    stats = enforce_gap(inp, shape, seed, MIN_GAP) if gap else None
    if logit_shift:
        inp["Q"][..., 0] = a
    return inp, stats


def oracle_reference(inp, shape, backward=True, stick=False, off_by_one=False):
    """The oracle's landmarks, selection, forward and (optionally) backward of one case,
    with softmax or (stick) stick-breaking chunk weights, and the softmax or (off_by_one)
    the softmax off by one inside a chunk."""
    S, k, G = shape.S, shape.k, shape.G
    ref = {"Kbar": oracle.landmarks(inp["K"], S)}
    idx, w, gap, _ = oracle.select(inp["Q"], ref["Kbar"], G, S, k, stick=stick)
    ref.update(idx=idx, w=w, gap=gap)
    ref["O"] = oracle.forward(inp["Q"], inp["K"], inp["V"], idx, w, S, off_by_one=off_by_one)
    ref["O_abs"] = attention_abs(inp, idx, w, S, off_by_one)
    if backward:
        ref["dQ"], ref["dK"], ref["dV"] = oracle.backward(inp["Q"], inp["K"], inp["V"], idx, w,
                                                           inp["dO"], S, stick=stick,
                                                           off_by_one=off_by_one)
    return ref


def attention_abs(inp, idx, w, S, off_by_one=False):
    """O_abs of the attention bound: the oracle forward on |V| and |w|."""
    return oracle.forward(inp["Q"], inp["K"], np.abs(inp["V"]), idx, np.abs(w), S,
                          off_by_one=off_by_one)


BF16_HALF_ULP = 2.0 ** -8


def tol(shape, ref: np.ndarray, ulps: float = 1.0, o_abs=None):
    """Element-wise tolerance array (see the module docstring); o_abs selects the bound of
    attention outputs."""
    if shape.dtype == "f32":
        return np.full(ref.shape, F32_ATOL)
    if o_abs is not None:
        return ulps * BF16_HALF_ULP * (o_abs + np.abs(ref))
    rms = float(np.sqrt(np.mean(np.square(ref)))) if ref.size else 0.0
    return BF16_RMS_FRAC * rms + ulps * BF16_HALF_ULP * np.abs(ref)


def assert_close(name, shape, got: torch.Tensor, ref: np.ndarray, ulps: float = 1.0,
                 o_abs=None, contract: bool = True):
    """fp32: max-abs <= 1e-4.  bf16: the element-wise bound and, with contract (weights
    from a selection), max |err| <= 2e-2 RMS(ref) over the tensor."""
    g = got.detach().float().cpu().numpy().astype(np.float64)
    assert g.shape == ref.shape, (name, g.shape, ref.shape)
    assert np.all(np.isfinite(g)), name + " has non-finite values"
    if not ref.size:
        return 0.0
    err = np.abs(g - ref)
    t = tol(shape, ref, ulps, o_abs)
    worst = int(np.argmax(err - t))
    elem_ratio = float(np.max(err / np.maximum(t, 1e-300)))
    rms_ratio = None
    if shape.dtype != "f32":
        unit = BF16_RMS_FRAC * float(np.sqrt(np.mean(np.square(ref))))
        beyond = float(np.max(err - half_ulp_bf16(g)))
        floor_err = float(np.max(np.abs(hsa_synth.round_bf16(ref.astype(np.float32)) - ref)))
        if unit > 0:
            rms_ratio, raw, floor = beyond / unit, float(err.max()) / unit, floor_err / unit
        else:
            rms_ratio = raw = floor = 0.0 if err.max() == 0 else math.inf
        RATIOS.append((os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0], name,
                       rms_ratio, elem_ratio, bool(contract), raw, floor))
        print("[parity] %s: max|err| = %.3e; beyond the output's half-ulp %.3f of 2e-2 RMS(ref)"
              "%s (raw %.3f, rounded oracle %.3f); %.3f of the element bound"
              % (name, err.max(), rms_ratio, "" if contract else " (not asserted)", raw, floor,
                 elem_ratio), flush=True)
    assert np.all(err <= t), "%s: error %.3e > tolerance %.3e at flat index %d (max-abs %.3e)" % (
        name, err.flat[worst], t.flat[worst], worst, err.max())
    if contract and rms_ratio is not None:
        assert rms_ratio <= 1.0, ("%s: error beyond the output's half-ulp is %.3f x 2e-2 RMS(ref)"
                                  % (name, rms_ratio))
    return float(err.max())


def assert_indices(idx_gpu: torch.Tensor, ref_idx: np.ndarray, gap: np.ndarray, S: int,
                   tokens=None):
    """Bit-exact where the oracle gap is >= MIN_GAP; elsewhere only validity is checked
    (distinct, descending, in range, the right count).  tokens[i] is the sequence position
    of row i along axis 1 (default: row i is token i)."""
    got = idx_gpu.cpu().numpy()
    sure = gap >= MIN_GAP                                    # [B, L, G]
    bad = np.nonzero((got != ref_idx).any(-1) & sure)
    assert bad[0].size == 0, "index mismatch at %s" % (list(zip(*bad))[:5],)
    k = got.shape[-1]
    for b, t, g in zip(*np.nonzero(~sure)):
        row = got[b, t, g]
        valid = row[row >= 0]
        pos = int(tokens[t]) if tokens is not None else int(t)
        assert len(valid) == min(k, pos // S)
        assert np.all(row[len(valid):] == -1)
        assert np.all(np.diff(valid) < 0) and np.all(valid < pos // S)
    return int(sure.sum()), int((~sure).sum())


def check_selection(dm, q, Kbar, pos, got_idx, got_w, ref_idx, ref_w, gap):
    """Selection of n queries q [n, h, d] at positions pos [n] against landmarks Kbar [C, d]
    (one (b, g) slice; dm from oracle.dims with the weight rule): bit-exact indices and
    weights within 1e-5 where the oracle gap is >= 1e-3; elsewhere a valid selection: the
    right count, distinct, descending, candidates only, each chosen chunk's fp64 score at
    least the oracle's n-th best - SCORE_SLACK, and weights equal to the weight rule on the
    oracle's scores of the chosen chunks within 1e-5.  Returns (#exact rows, #valid rows)."""
    got_idx = np.asarray(got_idx)
    got_w = np.asarray(got_w, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.int64)
    sure = gap >= MIN_GAP
    bad = np.nonzero((got_idx != ref_idx).any(-1) & sure)[0]
    assert bad.size == 0, "index mismatch at rows %s" % (pos[bad][:5],)
    if sure.any():
        assert np.max(np.abs(got_w[sure] - ref_w[sure])) <= W_ATOL
    loose = np.nonzero(~sure)[0]
    if loose.size == 0:
        return int(sure.sum()), 0
    k = got_idx.shape[-1]
    C = Kbar.shape[0]
    s = oracle.scores_at(dm, q[loose], Kbar, pos[loose])
    for r, row in enumerate(loose):
        gi = got_idx[row]
        nc = min(int(pos[row]) // dm.S, C)
        n = min(k, nc)
        valid = gi[gi >= 0]
        assert len(valid) == n and np.all(gi[n:] == -1), (pos[row], gi)
        assert np.all(np.diff(valid) < 0) and np.all(valid < nc), (pos[row], gi)
        nth = np.sort(s[r, :nc])[::-1][n - 1]
        assert np.all(s[r, valid] >= nth - SCORE_SLACK), (
            "row %d: chosen scores %s below the %d-th best %.6e" % (pos[row], s[r, valid], n, nth))
    w_rule = oracle.slot_weights_at(dm, q[loose], Kbar, pos[loose], got_idx[loose])
    assert np.max(np.abs(got_w[loose] - w_rule)) <= W_ATOL, np.max(np.abs(got_w[loose] - w_rule))
    return int(sure.sum()), int(loose.size)


def decode_case(shape, seed, lens, kbar_dtype=torch.float32, gap=True, key_coord0=None):
    """Decode inputs (hsa_synth.make_decode_inputs on the GPU) with the landmark cache of
    the given dtype; with gap, the query of every (b, g) whose top-k gap at lens[b] is below
    1e-3 is redrawn, so every group's selection is index-exact.  key_coord0: coordinate 0
    of every cached key is set to this value first (a common logit shift)."""
    from oracle.gapfix import enforce_decode_gap
    inp = hsa_synth.make_decode_inputs(shape, seed, device="cuda")
    if key_coord0 is not None:
        inp["Kc"][..., 0] = key_coord0
    kb = oracle.landmarks(inp["Kc"], shape.S).astype(np.float32)
    Kbar = torch.from_numpy(kb).cuda().to(kbar_dtype)
    if gap:
        inp["redrawn"] = enforce_decode_gap(inp, Kbar, lens, shape.S, shape.k)
    return inp, Kbar


def check_decode(shape, inp, Kbar, lens, o, idx, w, stick=False, off_by_one=False,
                 require_exact=True):
    """The GPU decode (o, idx, w) against the oracle's decode of the same cache: every
    (b, g) with a top-k gap >= 1e-3 index-exact with weights within 1e-5 and its heads'
    outputs within the bounds; any other group a valid selection (check_selection), its
    outputs not compared.  require_exact: every group must be exact (gap-enforced input).
    Returns the number of exact groups."""
    q, Kc, Vc = inp["q"], inp["Kc"], inp["Vc"]
    S, k = shape.S, shape.k
    B, H, d = q.shape
    G = Kc.shape[2]
    h = H // G
    ro, ridx, rw, rgap = oracle.decode(q, Kc, Vc, Kbar.float(), lens, S, k, stick=stick,
                                       off_by_one=off_by_one)
    ro_abs = oracle.decode(q, Kc, Vc.abs(), Kbar.float(), lens, S, k, stick=stick,
                           off_by_one=off_by_one)[0]
    gi, gw = idx.cpu().numpy(), w.cpu().numpy()
    qn = q.double().cpu().numpy()
    for b in range(B):
        for g in range(G):
            dm = oracle.dims(int(lens[b]), h, d, S, k, stick=stick)
            check_selection(dm, qn[b, g * h:(g + 1) * h][None], Kbar[b, :, g].float(),
                            [lens[b]], gi[b, g][None], gw[b, g][None], ridx[b, g][None],
                            rw[b, g][None], rgap[b, g][None])
    sure = rgap >= MIN_GAP
    if require_exact:
        assert sure.all(), "groups below the gap: %s" % (list(zip(*np.nonzero(~sure))),)
    hm = np.repeat(sure, h, axis=1)
    if hm.any():
        assert_close("o", shape, o[torch.from_numpy(hm).cuda()], ro[hm], o_abs=ro_abs[hm])
    return int(sure.sum())
