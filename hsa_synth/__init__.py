"""Seeded synthetic inputs for the HSA operator (shared by the GPU path and the oracle).

This module only draws random tensors with the shapes and value distributions of the
workloads; it contains none of the operator's arithmetic (no pooling, scoring, top-k,
softmax or attention).  Every tensor comes from its own counter-based Philox stream keyed
by (seed, tensor id, block), so a tensor does not depend on the order in which other
tensors were drawn, and a block of rows can be regenerated on its own.

Layouts follow the operator's problem statement: queries carry H = G*h heads and keys /
values one head per group (grouped-query attention, Sec. 3.1 "Notations"):

    Q, dO : [B, L, H, d]      K, V : [B, L, G, d]

bf16 workloads are returned as float32 arrays whose values are exactly representable in
bfloat16 (round-to-nearest-even of the float32 draw), so both sides see identical bits.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

__all__ = [
    "HsaShape", "WORKLOADS", "philox", "round_bf16", "make_training_inputs",
    "make_decode_inputs", "redraw_query_rows", "redraw_decode_query",
]

# tensor ids of the Philox key; one stream per tensor
_TID = {"Q": 1, "K": 2, "V": 3, "dO": 4, "mu": 5, "plant_pos": 6, "plant_dir": 7,
        "plant_keys": 8, "lowrank_U": 9, "lowrank_c": 10, "lowrank_a": 11,
        "lowrank_xi": 12, "redraw": 13, "kc": 14, "vc": 15, "q1": 16}


@dataclasses.dataclass(frozen=True)
class HsaShape:
    """Problem size: batch, sequence length, query heads, KV heads, head dim, chunk, top-k."""
    B: int
    L: int
    H: int
    G: int
    d: int
    S: int
    k: int
    dtype: str = "bf16"          # "f32" or "bf16": element type of Q, K, V, O and gradients

    @property
    def h(self) -> int:
        return self.H // self.G

    @property
    def C(self) -> int:          # number of complete chunks
        return self.L // self.S


# The five workloads (shapes of the paper's 370M model family, Sec. 4.1 and App. B:
# chunk 64, top-8, GQA).  K keeps a per-chunk mean offset so that landmark scores
# are separated: with i.i.d. keys the top-k score gaps fall far below 1e-3, while a
# constant shift of a chunk's keys leaves the intra-chunk softmax unchanged and moves only
# the selection and the weights.
WORKLOADS: Dict[str, dict] = {
    "tiny_f32": dict(shape=HsaShape(1, 1024, 4, 1, 64, 64, 4, "f32"), seed=1,
                     kind="iid", mu_std=0.5),
    "L4K_bf16": dict(shape=HsaShape(8, 4096, 16, 2, 128, 64, 8, "bf16"), seed=2,
                     kind="iid", mu_std=0.5),
    "L64K_bf16": dict(shape=HsaShape(1, 65536, 16, 2, 128, 64, 8, "bf16"), seed=3,
                      kind="long", mu_std=0.5),
    "decode_1M_bf16": dict(shape=HsaShape(8, 1 << 20, 16, 2, 128, 64, 8, "bf16"), seed=4,
                           kind="decode", mu_std=0.5),
    "wide_L16K_bf16": dict(shape=HsaShape(4, 16384, 32, 4, 128, 128, 16, "bf16"), seed=5,
                           kind="lowrank", mu_std=0.0),
    # three attention layers sharing one selection over inputs of their own (d_sel = h d)
    "shared_x3_L4K_bf16": dict(shape=HsaShape(8, 4096, 16, 2, 128, 64, 8, "bf16"), seed=2504,
                               kind="shared", mu_std=0.0, layers=3),
}


def philox(seed: int, tid: int, *sub: int) -> np.random.Generator:
    """Counter-based Philox-4x64 stream keyed by (seed, tensor id, sub-block ids)."""
    k0 = ((int(seed) & 0xFFFFFFFF) << 32) | (int(tid) & 0xFFFFFFFF)
    k1 = 0
    for s in sub:
        k1 = (k1 * 1000003 + (int(s) & 0xFFFFFFFFFFFF) + 1) & 0xFFFFFFFFFFFFFFFF
    return np.random.Generator(np.random.Philox(key=np.array([k0, k1], dtype=np.uint64)))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)


def _normal(seed: int, tid: int, shape, std: float, block_rows: Optional[int] = None) -> np.ndarray:
    """N(0, std^2) float32 tensor; drawn per leading-index block so slices are regenerable."""
    out = np.empty(shape, dtype=np.float32)
    lead = shape[0]
    for b in range(lead):
        g = philox(seed, tid, b)
        out[b] = g.standard_normal(shape[1:], dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def _cast(x: np.ndarray, dtype: str) -> np.ndarray:
    return round_bf16(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_training_inputs(name_or_shape, seed: Optional[int] = None, kind: str = "iid",
                         mu_std: float = 0.5, with_grad: bool = True) -> Dict[str, np.ndarray]:
    """Q, K, V (and dO) for a forward+backward workload.

    kind "iid":     Q, V ~ N(0,1)/sqrt(d); K ~ N(0,1)/sqrt(d) + mu[b,c,g,:],
                    mu ~ N(0, mu_std^2) per element, constant over the S keys of chunk c.
    kind "long":    as "iid" but K ~ N(0,1) + mu (unit-scale keys).
    kind "lowrank": rank-16 shared structure; per group an orthonormal U_g (d x 16),
                    K[t] = (U_g c[b,g,chunk(t)] + 0.1 eps)/sqrt(d),
                    Q[t, g*h+j] = (U_g (a[b,g] + 0.5 xi[t,j]) + 0.1 eps')/sqrt(d).
    dO ~ N(0, 1).
    """
    if isinstance(name_or_shape, str):
        wl = WORKLOADS[name_or_shape]
        shape, seed, kind, mu_std = wl["shape"], wl["seed"], wl["kind"], wl["mu_std"]
    else:
        shape = name_or_shape
        assert seed is not None
    B, L, H, G, d, S = shape.B, shape.L, shape.H, shape.G, shape.d, shape.S
    sc = 1.0 / math.sqrt(d)
    C_all = -(-L // S)
    out: Dict[str, np.ndarray] = {}
    if kind in ("iid", "long"):
        q = _normal(seed, _TID["Q"], (B, L, H, d), sc)
        kstd = 1.0 if kind == "long" else sc
        k = _normal(seed, _TID["K"], (B, L, G, d), kstd)
        if mu_std > 0:
            mu = _normal(seed, _TID["mu"], (B, C_all, G, d), mu_std)
            k = k.reshape(B, L, G, d)
            k += np.repeat(mu, S, axis=1)[:, :L]
        v = _normal(seed, _TID["V"], (B, L, G, d), sc)
    elif kind == "lowrank":
        r = 16
        h = H // G
        U = np.empty((G, d, r), dtype=np.float32)
        for g in range(G):
            a = philox(seed, _TID["lowrank_U"], g).standard_normal((d, r))
            U[g] = np.linalg.qr(a)[0].astype(np.float32)
        cch = _normal(seed, _TID["lowrank_c"], (B, C_all, G, r), 1.0)
        abar = _normal(seed, _TID["lowrank_a"], (B, G, r), 1.0)
        xi = _normal(seed, _TID["lowrank_xi"], (B, L, H, r), 0.5)
        k = np.einsum("gdr,bcgr->bcgd", U, cch).astype(np.float32)
        k = np.repeat(k, S, axis=1)[:, :L]
        k += _normal(seed, _TID["K"], (B, L, G, d), 0.1)
        k *= np.float32(sc)
        xi = xi.reshape(B, L, G, h, r) + abar[:, None, :, None, :]
        q = np.einsum("gdr,blgjr->blgjd", U, xi).astype(np.float32).reshape(B, L, H, d)
        q += _normal(seed, _TID["Q"], (B, L, H, d), 0.1)
        q *= np.float32(sc)
        v = _normal(seed, _TID["V"], (B, L, G, d), sc)
    else:
        raise ValueError(kind)
    out["Q"] = _cast(q, shape.dtype)
    out["K"] = _cast(k, shape.dtype)
    out["V"] = _cast(v, shape.dtype)
    if with_grad:
        out["dO"] = _cast(_normal(seed, _TID["dO"], (B, L, H, d), 1.0), shape.dtype)
    return out


def redraw_query_rows(Q: np.ndarray, seed: int, b: int, t: int, g: int, h: int,
                      attempt: int, std: float, dtype: str) -> None:
    """Replace the h query heads of group g at (b, t) by a fresh draw (sub-seeded)."""
    d = Q.shape[-1]
    x = philox(seed, _TID["redraw"], b, t, g, attempt).standard_normal((h, d), dtype=np.float32)
    Q[b, t, g * h:(g + 1) * h] = _cast(x * np.float32(std), dtype)


def make_decode_inputs(shape: HsaShape, seed: int, n_cache: Optional[int] = None,
                       mu_std: float = 0.5, plant: bool = True, device: str = "cpu"):
    """One query token per sequence against a KV cache of n_cache tokens (torch tensors).

    The cache is large (8 x 2^20 tokens), so it is drawn with torch's seeded Philox
    generator on `device`; the same (seed, device) always gives the same tensors.

    q[b, g*h+j] = 0.5 u[b,g] + N(0,1)/sqrt(d) with u[b,g] a random unit direction.
    Cache K ~ N(0,1)/sqrt(d) + mu[b,c,g,:] (mu ~ N(0, mu_std^2)), V ~ N(0,1)/sqrt(d).
    A planted chunk p[b,g] (uniform over the complete chunks) gets keys
    r (0.9 u + sqrt(0.19) v_s) with v_s random unit vectors orthogonal to u and
    r = mu_std*sqrt(d) (the typical norm of a chunk's mean key), so its keys have
    cosine 0.9 with the shared query direction: a passkey-like chunk that must be selected.
    Returns q [B,H,d], Kc, Vc [B,N,G,d] in the workload dtype, planted [B,G] (int64) and
    the query directions u [B,G,d] (float64).
    """
    import torch
    B, H, G, d, S = shape.B, shape.H, shape.G, shape.d, shape.S
    h = H // G
    N = shape.L if n_cache is None else n_cache
    sc = 1.0 / math.sqrt(d)
    tdt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32

    def gen(tid, *sub):
        g = torch.Generator(device=device)
        k1 = 0
        for s in sub:
            k1 = (k1 * 1000003 + int(s) + 1) & 0xFFFFFFFF
        g.manual_seed(((int(seed) & 0xFFFF) << 40) | ((tid & 0xFF) << 32) | k1)
        return g

    u = torch.randn((B, G, d), generator=gen(_TID["plant_dir"]), device=device,
                    dtype=torch.float64)
    u /= u.norm(dim=-1, keepdim=True)
    q = torch.randn((B, G, h, d), generator=gen(_TID["q1"]), device=device) * sc
    q += 0.5 * u[:, :, None, :].float()
    q = q.reshape(B, H, d).to(tdt)
    C_all = -(-N // S)
    kc = torch.empty((B, N, G, d), device=device, dtype=tdt)
    vc = torch.empty((B, N, G, d), device=device, dtype=tdt)
    for b in range(B):
        x = torch.randn((N, G, d), generator=gen(_TID["kc"], b), device=device) * sc
        if mu_std > 0:
            mu = torch.randn((C_all, G, d), generator=gen(_TID["mu"], b), device=device)
            x.view(-1, G, d)[: (N // S) * S].view(N // S, S, G, d).add_(
                (mu[: N // S] * mu_std)[:, None])
            if N % S:
                x[(N // S) * S:] += mu[N // S] * mu_std
        kc[b] = x.to(tdt)
        del x
        vc[b] = (torch.randn((N, G, d), generator=gen(_TID["vc"], b), device=device)
                 * sc).to(tdt)
    planted = torch.full((B, G), -1, dtype=torch.int64)
    C = N // S
    if plant and C > 0:
        r = mu_std * math.sqrt(d) if mu_std > 0 else 1.0
        for b in range(B):
            for g in range(G):
                p = int(torch.randint(0, C, (1,), generator=gen(_TID["plant_pos"], b, g),
                                      device=device).item())
                planted[b, g] = p
                x = torch.randn((S, d), generator=gen(_TID["plant_keys"], b, g),
                                device=device, dtype=torch.float64)
                ub = u[b, g]
                x -= (x @ ub)[:, None] * ub[None, :]
                x /= x.norm(dim=-1, keepdim=True)
                keys = r * (0.9 * ub[None, :] + math.sqrt(0.19) * x)
                kc[b, p * S:(p + 1) * S, g] = keys.to(tdt)
    return {"q": q, "Kc": kc, "Vc": vc, "planted": planted, "u": u, "seed": seed}


def redraw_decode_query(q, u, seed: int, b: int, g: int, attempt: int) -> None:
    """Replace the h query heads of group g of sequence b (q [B, H, d], a torch tensor) by
    0.5 u[b, g] + a fresh N(0, 1/d) draw (sub-seeded by (b, g, attempt)): the same
    distribution as make_decode_inputs, so the planted chunk stays aligned with the group."""
    import torch
    B, H, d = q.shape
    G = u.shape[1]
    h = H // G
    x = philox(seed, _TID["redraw"], b, g, attempt, 1).standard_normal((h, d))
    row = 0.5 * u[b, g].double().cpu()[None, :] + torch.from_numpy(x) / math.sqrt(d)
    q[b, g * h:(g + 1) * h] = row.to(q.dtype).to(q.device)


def make_shared_selection_inputs(name: str = "shared_x3_L4K_bf16", device: str = "cuda"):
    """Inputs of several attention layers sharing one selection over inputs of its own
    (torch tensors, drawn with torch's seeded Philox generator on `device`).

    Per layer: Q, K, V ~ N(0, 1/d), dO ~ N(0, 1) (workload dtype).  Selection queries
    Qs [B, L, G, h d] ~ N(0, 1) (workload dtype) and chunk representations Ks [B, C, G, h d]
    ~ N(0, 1) float32, so the scores Qs . Ks / sqrt(h d) are about N(0, 1).
    Returns (layers: list of dicts, Qs, Ks)."""
    import torch
    wl = WORKLOADS[name]
    sh = wl["shape"]
    B, L, H, G, d, S = sh.B, sh.L, sh.H, sh.G, sh.d, sh.S
    dsel = (H // G) * d
    tdt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(wl["seed"])

    def rnd(*shape, std=1.0, dt=tdt):
        return (torch.randn(shape, generator=gen, device=device) * std).to(dt)

    sc = d ** -0.5
    layers = [dict(Q=rnd(B, L, H, d, std=sc), K=rnd(B, L, G, d, std=sc),
                   V=rnd(B, L, G, d, std=sc), dO=rnd(B, L, H, d)) for _ in range(wl["layers"])]
    Qs = rnd(B, L, G, dsel)
    Ks = rnd(B, L // S, G, dsel, dt=torch.float32)
    return layers, Qs, Ks
