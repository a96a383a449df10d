"""Shared helpers of the GPU parity tests: seeded inputs, the oracle reference and the
tolerances (written here, used by every GPU test).

Tolerances (fixed in advance, independent of the measured error):
  - fp32 mode: max-abs error <= 1e-4 for outputs and gradients;
  - bf16 mode, attention outputs O: |got - ref| <= 2^-8 (O_abs + |ref|) element-wise, with
    O_abs = sum_i |w_i| sum_s P_s |V_s| (the same operator applied to |V| and |w|).  The
    bf16 kernels round the weighted probabilities w P / sum to bf16 (relative error <=
    2^-9) and the output once (<= 2^-9 |O|); every other step is fp32 on exact bf16
    products.  The bound is that error sum with a factor-2 margin;
  - bf16 mode, gradients: |got - ref| <= 2e-2 * RMS(ref) + 2^-8 * |ref| element-wise: the
    operator's bound relative to the gradient RMS plus half an ulp of the bf16 output
    format at the reference value (the final rounding to bf16, which no implementation
    avoids);
  - selected chunk indices: bit-exact for every token whose oracle top-k score gap is
    >= 1e-3 (gap-enforced inputs make that every token);
  - chunk weights: max-abs <= 1e-5 (fp32 softmax of fp32 scores whose error is ~1e-7);
  - landmarks: max-abs <= 1e-6 * max|Kbar| + 1e-7 (fp32 mean of S values).
"""
from __future__ import annotations

import math

import numpy as np
import torch

import hsa_synth
import oracle
from oracle.gapfix import enforce_gap

MIN_GAP = 1e-3
F32_ATOL = 1e-4
BF16_RMS_FRAC = 2e-2
W_ATOL = 1e-5


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
                 o_abs=None):
    g = got.detach().float().cpu().numpy().astype(np.float64)
    assert g.shape == ref.shape, (name, g.shape, ref.shape)
    assert np.all(np.isfinite(g)), name + " has non-finite values"
    if not ref.size:
        return 0.0
    err = np.abs(g - ref)
    t = tol(shape, ref, ulps, o_abs)
    worst = int(np.argmax(err - t))
    assert np.all(err <= t), "%s: error %.3e > tolerance %.3e at flat index %d (max-abs %.3e)" % (
        name, err.flat[worst], t.flat[worst], worst, err.max())
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
