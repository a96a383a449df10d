"""Score-gap enforcement for parity inputs (test infrastructure).

Index parity is only well defined when the k-th and (k+1)-th group scores of a token are
separated by more than the rounding error of either side.  For every (b, t, g) whose fp64
gap (computed by the oracle from the dtype-rounded tensors) is below `min_gap`, the h query
heads of that group at that token are redrawn from a sub-seeded stream of the input
generator, up to `max_attempts` times.  A token's queries only affect its own selection,
so the fix is local.
"""
from __future__ import annotations

import math

import numpy as np

import hsa_synth
from . import dims, landmarks_slice, scores_at, select_slice


def enforce_gap(inp: dict, shape: "hsa_synth.HsaShape", seed: int, min_gap: float = 1e-3,
                max_attempts: int = 64, alpha=None) -> dict:
    """Redraw query rows in place until every token's top-k gap is >= min_gap.

    Returns statistics {'redrawn': count of (b,t,g) rows redrawn, 'rows': total rows}."""
    Q, K = inp["Q"], inp["K"]
    B, L, H, d = Q.shape
    G, S, k, h = shape.G, shape.S, shape.k, shape.H // shape.G
    qstd = float(np.std(Q[:, :min(L, 256)])) or 1.0 / math.sqrt(d)
    redrawn = 0
    for b in range(B):
        for g in range(G):
            dm = dims(L, h, d, S, k, alpha)
            Kb = landmarks_slice(dm, np.ascontiguousarray(K[b, :, g]))
            _, _, gap, _ = select_slice(dm, Q[b, :, g * h:(g + 1) * h], Kb)
            bad = np.nonzero(gap < min_gap)[0]
            attempt = 0
            while bad.size:
                if attempt >= max_attempts:
                    raise RuntimeError("gap enforcement failed for %d rows" % bad.size)
                for t in bad:
                    hsa_synth.redraw_query_rows(Q, seed, b, int(t), g, h, attempt, qstd,
                                                shape.dtype)
                if attempt == 0:
                    redrawn += bad.size
                _, _, gap2, _ = select_slice(dm, Q[b, :, g * h:(g + 1) * h], Kb, rows=bad)
                bad = bad[gap2 < min_gap]
                attempt += 1
    return {"redrawn": int(redrawn), "rows": int(B * L * G)}


def decode_gap(q, Kbar, lens, S: int, k: int, alpha=None):
    """Top-k score gap [B, G] of the decode queries q [B, H, d] (torch or numpy) at positions
    lens[b] against the landmark cache Kbar [B, C, G, d]: s_(k) - s_(k+1), +inf with at most
    k candidates."""
    q = np.asarray(q.detach().double().cpu()) if hasattr(q, "detach") else np.asarray(q, np.float64)
    B, H, d = q.shape
    G = Kbar.shape[2]
    h = H // G
    gap = np.full((B, G), np.inf)
    for b in range(B):
        nc = int(lens[b]) // S
        if nc <= k:
            continue
        kb = Kbar[b, :nc, :].float() if hasattr(Kbar, "float") else Kbar[b, :nc]
        for g in range(G):
            dm = dims(int(lens[b]), h, d, S, k, alpha)
            s = scores_at(dm, q[b, g * h:(g + 1) * h][None], kb[:, g], [int(lens[b])])[0]
            srt = np.sort(s)[::-1]
            gap[b, g] = srt[k - 1] - srt[k]
    return gap


def enforce_decode_gap(inp: dict, Kbar, lens, S: int, k: int, min_gap: float = 1e-3,
                       max_attempts: int = 64, alpha=None) -> int:
    """Redraw the decode query of every (b, g) whose top-k gap is < min_gap (in place, with
    hsa_synth.redraw_decode_query, which keeps the planted chunk aligned with the group);
    returns the number of groups redrawn."""
    q, u, seed = inp["q"], inp["u"], inp["seed"]
    gap = decode_gap(q, Kbar, lens, S, k, alpha)
    bad = list(zip(*np.nonzero(gap < min_gap)))
    for b, g in bad:
        for attempt in range(max_attempts + 1):
            if attempt == max_attempts:
                raise RuntimeError("decode gap enforcement failed for (%d, %d)" % (b, g))
            hsa_synth.redraw_decode_query(q, u, seed, int(b), int(g), attempt)
            one = decode_gap(q[b:b + 1], Kbar[b:b + 1], [lens[b]], S, k, alpha)
            if one[0, g] >= min_gap:
                break
    return len(bad)
