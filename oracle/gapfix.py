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
from . import dims, landmarks_slice, select_slice


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
