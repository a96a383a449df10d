"""Pins of the fp64 oracle against facts fixed outside the oracle's own code.

Each test checks the oracle against brute force, a closed form, an invariant, or a
library routine that the operator reduces to in a special case (CPU only):
  - landmarks: exact mean of exactly representable keys; the mean-of-logits identity
    q . Kbar_c = mean_s q . k_s (App. A, mean-pooled relevance);
  - selection: brute force over all chunk subsets; ties to the lower chunk index;
    invariance of the selected set to positive query scaling;
  - weights: sum to 1, equal 1 for k = 1, padded slots;
  - forward: S=1, h=1, k>=L reduces to causal attention without the diagonal (torch
    SDPA); S=1 with small k to top-k token attention (torch.topk); k=1 to attention over
    the single best chunk (torch SDPA); all-past selection to a dense two-level softmax;
    per-chunk key shifts leave the output unchanged when the weights are held fixed;
  - backward: central finite differences of sum(dO*O) (selection fixed, weights moving
    with the scores) and torch float64 autograd of a gather+softmax formulation;
  - decode: equals the forward's row at the same position.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import hsa_synth
import oracle

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def rnd(seed, *shape, std=1.0):
    return hsa_synth.philox(seed, 99, *shape).standard_normal(shape) * std


def small_problem(seed, L=24, h=2, d=4, S=3, k=3, mu=1.0, G=1, B=1):
    Q = rnd(seed, B, L, G * h, d)
    K = rnd(seed + 1, B, L, G, d)
    C_all = -(-L // S)
    K += np.repeat(rnd(seed + 2, B, C_all, G, d, std=mu), S, axis=1)[:, :L]
    V = rnd(seed + 3, B, L, G, d)
    dO = rnd(seed + 4, B, L, G * h, d)
    return Q, K, V, dO


# ------------------------------------------------------------------ landmarks ----

def test_landmarks_exact_mean_of_representable_keys():
    g = hsa_synth.philox(11, 1)
    K = g.integers(-64, 64, size=(2, 256, 3, 8)).astype(np.float64) / 16.0
    Kb = oracle.landmarks(K, 64)
    ref = K.reshape(2, 4, 64, 3, 8).mean(axis=2)
    assert np.array_equal(Kb, ref)


def test_landmarks_ragged_tail_ignored():
    K = rnd(3, 1, 70, 1, 5)
    Kb = oracle.landmarks(K, 16)
    assert Kb.shape == (1, 4, 1, 5)
    np.testing.assert_allclose(Kb[0, 3, 0], K[0, 48:64, 0].mean(0), rtol=0, atol=1e-14)


def test_mean_of_logits_identity():
    """App. A: q . Kbar_c equals the mean over the chunk of the token logits q . k_s."""
    K = rnd(5, 1, 128, 1, 16)
    q = rnd(6, 16)
    Kb = oracle.landmarks(K, 32)[0, :, 0]
    logits = K[0, :, 0] @ q
    np.testing.assert_allclose(Kb @ q, logits.reshape(4, 32).mean(1), rtol=1e-13, atol=1e-13)


# ------------------------------------------------------------------ selection ----

def brute_force_select(scores, ncand, k):
    """All subsets of size min(k, ncand): maximal score sum, ties -> lexicographically
    smallest ascending index tuple; returned in descending chunk order."""
    n = min(k, ncand)
    if n == 0:
        return []
    best, best_sum = None, -np.inf
    for sub in itertools.combinations(range(ncand), n):
        ssum = float(sum(scores[c] for c in sub))
        if ssum > best_sum + 1e-12:
            best, best_sum = sub, ssum
    return sorted(best, reverse=True)


@pytest.mark.parametrize("seed,k", [(21, 1), (22, 3), (23, 5)])
def test_select_brute_force(seed, k):
    L, h, d, S = 40, 3, 5, 4
    Q, K, _, _ = small_problem(seed, L=L, h=h, d=d, S=S, k=k)
    Kb = oracle.landmarks(K, S)
    idx, w, gap, ss = oracle.select(Q, Kb, 1, S, k)
    alpha = 1.0 / math.sqrt(h * d)
    for t in range(L):
        ncand = t // S
        scores = alpha * (Q[0, t].sum(0) @ Kb[0, :, 0].T)
        want = brute_force_select(scores, ncand, k)
        got = [int(c) for c in idx[0, t, 0] if c >= 0]
        assert got == want, (t, got, want)
        assert all(c == -1 for c in idx[0, t, 0, len(want):])
        if want:
            ref_w = torch.softmax(torch.tensor(scores[want]), 0).numpy()
            np.testing.assert_allclose(w[0, t, 0, :len(want)], ref_w, rtol=1e-12, atol=1e-14)
        assert np.all(w[0, t, 0, len(want):] == 0)


def test_select_ties_go_to_lower_index():
    # d = 1, h = 1, q = 1: scores are alpha * Kbar, with exact ties at the top-2 boundary
    S = 1
    vals = np.array([3., 5., 5., 2., 5., 1.])
    K = vals.reshape(1, 6, 1, 1)
    L = 7
    Kfull = np.zeros((1, L, 1, 1))
    Kfull[0, :6] = K[0]
    Q = np.ones((1, L, 1, 1))
    idx, w, gap, _ = oracle.select(Q, oracle.landmarks(Kfull, S), 1, S, 2)
    # token 6 sees chunks 0..5; the top-2 among {1, 2, 4} (all 5.0) are 1 and 2
    assert list(idx[0, 6, 0]) == [2, 1]
    assert gap[0, 6, 0] == 0.0
    np.testing.assert_allclose(w[0, 6, 0], [0.5, 0.5])


def test_select_positive_query_scaling_keeps_indices():
    Q, K, _, _ = small_problem(31, L=48, h=2, d=6, S=4, k=3)
    Kb = oracle.landmarks(K, 4)
    i1, w1, _, _ = oracle.select(Q, Kb, 1, 4, 3)
    i2, w2, _, _ = oracle.select(Q * 3.7, Kb, 1, 4, 3)
    assert np.array_equal(i1, i2)
    assert not np.allclose(w1[0, 40:], w2[0, 40:])


def test_select_k_at_least_all_candidates_is_noop():
    Q, K, _, _ = small_problem(33, L=32, h=2, d=4, S=4, k=8)
    Kb = oracle.landmarks(K, 4)
    idx, w, gap, _ = oracle.select(Q, Kb, 1, 4, 8)
    for t in range(32):
        n = t // 4
        assert list(idx[0, t, 0, :n]) == list(range(n - 1, -1, -1))
        assert np.isinf(gap[0, t, 0])


def test_weights_sum_to_one_and_k1():
    Q, K, _, _ = small_problem(35, L=64, h=2, d=4, S=4, k=4)
    Kb = oracle.landmarks(K, 4)
    _, w, _, _ = oracle.select(Q, Kb, 1, 4, 4)
    s = w[0, 4:, 0].sum(-1)
    np.testing.assert_allclose(s, 1.0, rtol=0, atol=1e-14)
    assert np.all(w[0, :4] == 0)
    _, w1, _, _ = oracle.select(Q, Kb, 1, 4, 1)
    assert np.all(w1[0, 4:, 0, 0] == 1.0)


def test_stick_breaking_weights_telescope_and_k1():
    """Stick-breaking weights (Sec. 3.1.1): slot i takes the share sigmoid(s_i) of what the
    earlier slots left, so the weights sum to 1 - prod(1 - sigmoid(s)) (telescoping), stay
    below 1, and k = 1 gives sigmoid of the best score; the indices do not depend on the
    weight rule."""
    Q, K, _, _ = small_problem(37, L=64, h=2, d=4, S=4, k=4, mu=1.5)
    Kb = oracle.landmarks(K, 4)
    idx_s, w, _, ss = oracle.select(Q, Kb, 1, 4, 4, stick=True)
    idx_m, _, _, _ = oracle.select(Q, Kb, 1, 4, 4)
    assert np.array_equal(idx_s, idx_m)
    sig = 1.0 / (1.0 + np.exp(-ss[0, 4:, 0]))
    valid = idx_s[0, 4:, 0] >= 0
    left = np.prod(np.where(valid, 1.0 - sig, 1.0), axis=-1)
    np.testing.assert_allclose(w[0, 4:, 0].sum(-1), 1.0 - left, rtol=1e-14, atol=1e-15)
    assert np.all(w[0, 4:, 0].sum(-1) < 1.0) and np.all(w >= 0)
    assert np.all(w[0, :4] == 0)
    _, w1, _, s1 = oracle.select(Q, Kb, 1, 4, 1, stick=True)
    np.testing.assert_allclose(w1[0, 4:, 0, 0], 1.0 / (1.0 + np.exp(-s1[0, 4:, 0, 0])),
                               rtol=1e-15, atol=0)


def test_stick_breaking_most_recent_chunk_breaks_first():
    """The stick is broken in descending chunk order (Sec. 3.1.1 sorts the selected chunks
    before the weights): the most recent selected chunk takes sigmoid of its own score,
    whatever the others score, and the oldest takes what all the more recent ones left.
    Scores are recomputed here with numpy from the plain definition."""
    Q, K, _, _ = small_problem(41, L=96, h=2, d=4, S=4, k=5, mu=1.5)
    Kb = oracle.landmarks(K, 4)
    idx, w, _, _ = oracle.select(Q, Kb, 1, 4, 5, stick=True)
    alpha = 1.0 / np.sqrt(2 * 4)
    sig = lambda x: 1.0 / (1.0 + np.exp(-x))
    checked = 0
    for t in range(96):
        sel = [int(c) for c in idx[0, t, 0] if c >= 0]
        if len(sel) < 2:
            continue
        s = {c: alpha * Q[0, t].sum(0) @ Kb[0, c, 0] for c in sel}
        newest, oldest = max(sel), min(sel)
        wt = dict(zip(sel, w[0, t, 0][:len(sel)]))
        assert abs(wt[newest] - sig(s[newest])) < 1e-14
        rest = np.prod([1.0 - sig(s[c]) for c in sel if c != oldest])
        assert abs(wt[oldest] - sig(s[oldest]) * rest) < 1e-14
        checked += 1
    assert checked > 50


@pytest.mark.parametrize("seed,k", [(51, 1), (52, 3), (53, 6)])
def test_gap_is_the_order_statistic_of_a_brute_force_sort(seed, k):
    """gap = s_(n) - s_(n+1) of the descending score order (n = min(k, #candidates)), +inf
    when every candidate is selected; checked against numpy's sort of the scores of the
    concatenated group query against the landmark tiled over the heads (Sec. 3.1: the
    group query has dimension h d), a formulation the oracle does not use."""
    L, h, d, S = 60, 3, 5, 4
    Q, K, _, _ = small_problem(seed, L=L, h=h, d=d, S=S, k=k)
    Kb = oracle.landmarks(K, S)
    _, _, gap, _ = oracle.select(Q, Kb, 1, S, k)
    alpha = 1.0 / math.sqrt(h * d)
    tiled = np.tile(Kb[0, :, 0], (1, h))                      # [C, h d]
    checked = 0
    for t in range(L):
        ncand = t // S
        n = min(k, ncand)
        if ncand <= n:
            assert np.isinf(gap[0, t, 0]), t
            continue
        s = np.sort(alpha * (tiled[:ncand] @ Q[0, t].reshape(-1)))[::-1]
        assert abs(gap[0, t, 0] - (s[n - 1] - s[n])) <= 1e-13, (t, gap[0, t, 0], s[n - 1] - s[n])
        checked += 1
    assert checked > 20


def test_gap_at_exact_ties_and_one_below():
    """Exact ties give gap 0; moving the (n+1)-th score down by exactly 1/2 gives 1/2 (the
    n-th and (n+1)-th order statistics, not the (n-1)-th or the (n+2)-th)."""
    S, L = 1, 8
    q = np.ones((1, L, 1, 1))
    for vals, k, want in (([4., 9., 7., 7., 1., 3., 2.], 2, 0.0),     # 9 7 | 7
                          ([4., 9., 7., 6.5, 1., 3., 2.], 2, 0.5),    # 9 7 | 6.5
                          ([4., 9., 7., 6.5, 1., 3., 2.], 3, 2.5),    # 9 7 6.5 | 4
                          ([4., 9., 7., 6.5, 1., 3., 2.], 1, 2.0)):   # 9 | 7
        K = np.zeros((1, L, 1, 1))
        K[0, :7, 0, 0] = vals
        _, _, gap, _ = oracle.select(q, oracle.landmarks(K, S), 1, S, k)
        assert gap[0, 7, 0] == want, (vals, k)


def test_scores_at_match_the_tiled_group_query():
    """scores_at: alpha (sum_j q_j) . Kbar_c for the candidates, NaN beyond, checked against
    the concatenated group query against the tiled landmark."""
    L, h, d, S = 50, 2, 6, 5
    Q, K, _, _ = small_problem(55, L=L, h=h, d=d, S=S, k=2)
    Kb = oracle.landmarks(K, S)[0, :, 0]
    dm = oracle.dims(L, h, d, S, 2)
    pos = np.array([0, 4, 5, 23, 49])
    s = oracle.scores_at(dm, Q[0, pos], Kb, pos)
    tiled = np.tile(Kb, (1, h))
    for r, t in enumerate(pos):
        nc = t // S
        want = (tiled[:nc] @ Q[0, t].reshape(-1)) / math.sqrt(h * d)
        np.testing.assert_allclose(s[r, :nc], want, rtol=1e-13, atol=1e-15)
        assert np.all(np.isnan(s[r, nc:]))


@pytest.mark.parametrize("stick", [False, True])
def test_slot_weights_at(stick):
    """The weight rule on given slots: on the oracle's own selection it is the oracle's w;
    on another selection it is torch.softmax of the scores of its valid slots (or the
    stick-breaking product in the given slot order), with empty slots at 0."""
    L, h, d, S, k = 80, 2, 4, 4, 4
    Q, K, _, _ = small_problem(57, L=L, h=h, d=d, S=S, k=k, mu=1.5)
    Kb = oracle.landmarks(K, S)[0, :, 0]
    dm = oracle.dims(L, h, d, S, k, stick=stick)
    rows = np.arange(L)
    idx, w, _, _ = oracle.select_slice(dm, Q[0], Kb)
    np.testing.assert_allclose(oracle.slot_weights_at(dm, Q[0], Kb, rows, idx), w,
                               rtol=0, atol=1e-15)
    # another selection: arbitrary candidate chunks in arbitrary slot order, some empty
    rng = np.random.default_rng(3)
    other = np.full((L, k), -1, np.int32)
    for t in range(L):
        nc = t // S
        if nc:
            m = rng.integers(1, min(k, nc) + 1)
            other[t, :m] = rng.choice(nc, m, replace=False)
    other[5::7, 0] = 10 ** 6                       # past the candidates: empty
    got = oracle.slot_weights_at(dm, Q[0], Kb, rows, other)
    alpha = 1.0 / math.sqrt(h * d)
    for t in range(L):
        valid = [(i, int(c)) for i, c in enumerate(other[t]) if 0 <= c < t // S]
        want = np.zeros(k)
        if valid:
            sc = torch.tensor([alpha * Q[0, t].sum(0) @ Kb[c] for _, c in valid])
            if stick:
                b = torch.sigmoid(sc)
                left = torch.cumprod(torch.cat([torch.ones(1, dtype=b.dtype), 1 - b[:-1]]), 0)
                ww = (b * left).numpy()
            else:
                ww = torch.softmax(sc, 0).numpy()
            for (i, _), x in zip(valid, ww):
                want[i] = x
        np.testing.assert_allclose(got[t], want, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------- forward ----

def sdpa(q, k, v, scale, mask=None):
    return torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q), torch.tensor(k), torch.tensor(v), attn_mask=mask, scale=scale).numpy()


def test_S1_full_k_is_causal_attention_without_diagonal():
    L, d = 33, 8
    Q = rnd(41, 1, L, 1, d)
    K = rnd(42, 1, L, 1, d)
    V = rnd(43, 1, L, 1, d)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, 1), 1, 1, L)
    O = oracle.forward(Q, K, V, idx, w, 1)
    mask = torch.tril(torch.ones(L, L, dtype=torch.bool), diagonal=-1)
    ref = sdpa(Q[0, 1:, 0], K[0, :, 0], V[0, :, 0], 1.0 / math.sqrt(d), mask[1:])
    np.testing.assert_allclose(O[0, 1:, 0], ref, rtol=1e-11, atol=1e-12)
    assert np.all(O[0, 0] == 0)


def test_S1_small_k_is_topk_token_attention():
    L, d, k = 40, 6, 5
    Q = rnd(45, 1, L, 1, d)
    K = rnd(46, 1, L, 1, d)
    V = rnd(47, 1, L, 1, d)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, 1), 1, 1, k)
    O = oracle.forward(Q, K, V, idx, w, 1)
    q, kk, v = (torch.tensor(x[0, :, 0]) for x in (Q, K, V))
    logits = (q @ kk.T) / math.sqrt(d)
    for t in range(1, L):
        n = min(k, t)
        top = torch.topk(logits[t, :t], n)
        ref = torch.softmax(top.values, 0) @ v[top.indices]
        np.testing.assert_allclose(O[0, t, 0], ref.numpy(), rtol=1e-11, atol=1e-12)


def test_k1_is_attention_over_the_best_chunk():
    L, h, d, S = 64, 3, 8, 8
    Q, K, V, _ = small_problem(51, L=L, h=h, d=d, S=S, k=1)
    Kb = oracle.landmarks(K, S)
    idx, w, _, _ = oracle.select(Q, Kb, 1, S, 1)
    O = oracle.forward(Q, K, V, idx, w, S)
    for t in range(S, L):
        scores = Q[0, t].sum(0) @ Kb[0, :t // S, 0].T
        c = int(np.argmax(scores))
        assert idx[0, t, 0, 0] == c
        ref = sdpa(Q[0, t], K[0, c * S:(c + 1) * S, 0], V[0, c * S:(c + 1) * S, 0],
                   1.0 / math.sqrt(d))
        np.testing.assert_allclose(O[0, t], ref, rtol=1e-11, atol=1e-12)


def test_all_past_selection_is_dense_two_level_softmax():
    L, h, d, S = 48, 2, 5, 6
    C = L // S
    Q, K, V, _ = small_problem(55, L=L, h=h, d=d, S=S, k=C)
    Kb = oracle.landmarks(K, S)
    idx, w, _, _ = oracle.select(Q, Kb, 1, S, C)
    O = oracle.forward(Q, K, V, idx, w, S)
    Kt = torch.tensor(K[0, :, 0]).reshape(C, S, d)
    Vt = torch.tensor(V[0, :, 0]).reshape(C, S, d)
    alpha = 1.0 / math.sqrt(h * d)
    for t in range(L):
        n = t // S
        if n == 0:
            assert np.all(O[0, t] == 0)
            continue
        q = torch.tensor(Q[0, t])
        wts = torch.softmax(alpha * (Kt[:n].mean(1) @ q.sum(0)), 0)
        per_chunk = torch.nn.functional.scaled_dot_product_attention(
            q[None].expand(n, h, d), Kt[:n], Vt[:n], scale=1.0 / math.sqrt(d))
        ref = (wts[:, None, None] * per_chunk).sum(0)
        np.testing.assert_allclose(O[0, t], ref.numpy(), rtol=1e-11, atol=1e-12)


def test_S1_off_by_one_is_sigmoid_gated_token_attention():
    """S = 1, h = 1, k >= L with the softmax off by one: each chunk is one key, whose
    attention is exp(z) / (1 + exp(z)) = sigmoid(z), so O_t = sum_{c<t} softmax_c(alpha
    q.k_c) sigmoid(beta q.k_c) v_c."""
    L, d = 30, 8
    Q = rnd(141, 1, L, 1, d)
    K = rnd(142, 1, L, 1, d)
    V = rnd(143, 1, L, 1, d)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, 1), 1, 1, L)
    O = oracle.forward(Q, K, V, idx, w, 1, off_by_one=True)
    q, kk, v = (torch.tensor(x[0, :, 0]) for x in (Q, K, V))
    logits = (q @ kk.T) / math.sqrt(d)
    assert np.all(O[0, 0] == 0)
    for t in range(1, L):
        ref = (torch.softmax(logits[t, :t], 0) * torch.sigmoid(logits[t, :t])) @ v[:t]
        np.testing.assert_allclose(O[0, t, 0], ref.numpy(), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("key_scale", [1.0, 40.0])
def test_k1_off_by_one_is_attention_with_a_null_key(key_scale):
    """k = 1 with the softmax off by one equals plain attention over the chosen chunk's keys
    plus one all-zero key (logit exactly 0) whose value is zero; key_scale = 40 puts the
    logits far beyond exp's range on both sides."""
    L, h, d, S = 64, 3, 8, 8
    Q, K, V, _ = small_problem(151, L=L, h=h, d=d, S=S, k=1)
    K = K * key_scale
    Kb = oracle.landmarks(K, S)
    idx, w, _, _ = oracle.select(Q, Kb, 1, S, 1)
    O = oracle.forward(Q, K, V, idx, w, S, off_by_one=True)
    zero = np.zeros((1, d))
    for t in range(S, L):
        c = int(idx[0, t, 0, 0])
        ref = sdpa(Q[0, t], np.concatenate([zero, K[0, c * S:(c + 1) * S, 0]]),
                   np.concatenate([zero, V[0, c * S:(c + 1) * S, 0]]), 1.0 / math.sqrt(d))
        np.testing.assert_allclose(O[0, t], ref, rtol=1e-11, atol=1e-13)
    # the normaliser is at least 1: a chunk can take less than its weight, never more
    O_abs = oracle.forward(Q, K, np.abs(V), idx, w, S, off_by_one=True)
    O_std = oracle.forward(Q, K, np.abs(V), idx, w, S)
    assert np.all(O_abs <= O_std * (1 + 1e-12))


def test_per_chunk_key_shift_leaves_output_unchanged():
    L, h, d, S = 64, 2, 6, 8
    Q, K, V, _ = small_problem(57, L=L, h=h, d=d, S=S, k=3)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, S), 1, S, 3)
    O1 = oracle.forward(Q, K, V, idx, w, S)
    K2 = K.copy()
    K2[0, 2 * S:3 * S, 0] += rnd(58, d)
    O2 = oracle.forward(Q, K2, V, idx, w, S)
    np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)


# ------------------------------------------------------------------ backward ----

def _loss(Q, K, V, dO, S, k, idx_ref, stick=False, off1=False):
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, S), K.shape[2], S, k, stick=stick)
    assert np.array_equal(idx, idx_ref), "selection moved under the perturbation"
    return float((oracle.forward(Q, K, V, idx, w, S, off_by_one=off1) * dO).sum())


@pytest.mark.parametrize("G,stick,off1", [(1, False, False), (2, False, False),
                                          (1, True, False), (2, True, False),
                                          (2, False, True), (1, True, True)])
def test_backward_finite_differences(G, stick, off1):
    L, h, d, S, k = 12, 2, 3, 2, 2
    Q, K, V, dO = small_problem(61 + G, L=L, h=h, d=d, S=S, k=k, mu=2.0, G=G)
    idx, w, gap, _ = oracle.select(Q, oracle.landmarks(K, S), G, S, k, stick=stick)
    assert gap[np.isfinite(gap)].min() > 1e-4
    dQ, dK, dV = oracle.backward(Q, K, V, idx, w, dO, S, stick=stick, off_by_one=off1)
    eps = 1e-6
    for name, X, grad in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        num = np.zeros_like(X)
        it = np.nditer(X, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            Xp, Xm = X.copy(), X.copy()
            Xp[i] += eps
            Xm[i] -= eps
            args = {"Q": Q, "K": K, "V": V}
            args[name] = Xp
            fp = _loss(args["Q"], args["K"], args["V"], dO, S, k, idx, stick, off1)
            args[name] = Xm
            fm = _loss(args["Q"], args["K"], args["V"], dO, S, k, idx, stick, off1)
            num[i] = (fp - fm) / (2 * eps)
        np.testing.assert_allclose(grad, num, rtol=1e-5, atol=1e-7, err_msg=name)


def torch_hsa_forward(Q, K, V, idx, S, alpha, beta, stick=False, off1=False):
    """Gather + softmax formulation (fixed idx; weights from the scores) in autograd;
    stick: weights by stick-breaking over the slots (sigmoid, then a cumulative product of
    the complements); off1: the chunk's softmax taken over its logits and one extra 0,
    whose column is then dropped."""
    B, L, H, d = Q.shape
    G = K.shape[2]
    h = H // G
    k = idx.shape[-1]
    C = L // S
    O = torch.zeros_like(Q)
    Kc = K[:, :C * S].reshape(B, C, S, G, d)
    Vc = V[:, :C * S].reshape(B, C, S, G, d)
    Kbar = Kc.mean(2)                                            # [B, C, G, d]
    for b in range(B):
        for g in range(G):
            for t in range(L):
                sel = [int(c) for c in idx[b, t, g] if c >= 0]
                if not sel:
                    continue
                q = Q[b, t, g * h:(g + 1) * h]                   # [h, d]
                s = alpha * (Kbar[b, sel, g] @ q.sum(0))         # [n]
                if stick:
                    bb = torch.sigmoid(s)
                    left = torch.cumprod(torch.cat([torch.ones_like(bb[:1]), 1 - bb[:-1]]), 0)
                    wts = bb * left
                else:
                    wts = torch.softmax(s, 0)
                kk = Kc[b, sel, :, g]                             # [n, S, d]
                vv = Vc[b, sel, :, g]
                z = beta * torch.einsum("jd,nsd->njs", q, kk)
                if off1:
                    p = torch.softmax(torch.cat([torch.zeros_like(z[..., :1]), z], -1), -1)[..., 1:]
                else:
                    p = torch.softmax(z, -1)
                o = torch.einsum("njs,nsd->njd", p, vv)
                O[b, t, g * h:(g + 1) * h] = (wts[:, None, None] * o).sum(0)
    return O


@pytest.mark.parametrize("stick,off1", [(False, False), (True, False), (False, True),
                                        (True, True)])
def test_backward_matches_torch_autograd(stick, off1):
    L, h, d, S, k, G = 40, 2, 4, 4, 3, 2
    Q, K, V, dO = small_problem(71, L=L, h=h, d=d, S=S, k=k, G=G)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, S), G, S, k, stick=stick)
    dQ, dK, dV = oracle.backward(Q, K, V, idx, w, dO, S, stick=stick, off_by_one=off1)
    Qt, Kt, Vt = (torch.tensor(x, requires_grad=True) for x in (Q, K, V))
    O = torch_hsa_forward(Qt, Kt, Vt, idx, S, 1 / math.sqrt(h * d), 1 / math.sqrt(d), stick,
                          off1)
    np.testing.assert_allclose(O.detach().numpy(),
                               oracle.forward(Q, K, V, idx, w, S, off_by_one=off1),
                               rtol=1e-12, atol=1e-13)
    (O * torch.tensor(dO)).sum().backward()
    np.testing.assert_allclose(dQ, Qt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dK, Kt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dV, Vt.grad.numpy(), rtol=1e-10, atol=1e-12)


def test_backward_row_and_chunk_subsets_match_full():
    L, h, d, S, k = 48, 2, 4, 4, 3
    Q, K, V, dO = small_problem(73, L=L, h=h, d=d, S=S, k=k)
    idx, w, _, _ = oracle.select(Q, oracle.landmarks(K, S), 1, S, k)
    dQ, dK, dV = oracle.backward(Q, K, V, idx, w, dO, S)
    dm = oracle.dims(L, h, d, S, k)
    Qs, dOs = Q[0, :, :h], dO[0, :, :h]
    Kb = oracle.landmarks_slice(dm, K[0, :, 0])
    rows = np.array([47, 5, 30])
    dq, ds_rows = oracle.backward_q_slice(dm, Qs, K[0, :, 0], V[0, :, 0], Kb, idx[0, :, 0],
                                          w[0, :, 0], dOs, rows=rows)
    np.testing.assert_allclose(dq, dQ[0, rows], rtol=0, atol=1e-15)
    _, ds = oracle.backward_q_slice(dm, Qs, K[0, :, 0], V[0, :, 0], Kb, idx[0, :, 0],
                                    w[0, :, 0], dOs)
    ch = np.array([7, 0, 3])
    dk, dv = oracle.backward_kv_slice(dm, Qs, K[0, :, 0], V[0, :, 0], idx[0, :, 0],
                                      w[0, :, 0], dOs, ds, chunks=ch)
    for i, c in enumerate(ch):
        np.testing.assert_allclose(dk[i], dK[0, c * S:(c + 1) * S, 0], rtol=0, atol=1e-15)
        np.testing.assert_allclose(dv[i], dV[0, c * S:(c + 1) * S, 0], rtol=0, atol=1e-15)


# -------------------------------------------------------------------- decode ----

@pytest.mark.parametrize("off1", [False, True])
@pytest.mark.parametrize("t", [64, 67, 100, 31])
def test_decode_equals_forward_row(t, off1):
    L, h, d, S, k, G = 128, 2, 8, 8, 3, 2
    Q, K, V, _ = small_problem(81, L=L, h=h, d=d, S=S, k=k, G=G)
    Kb = oracle.landmarks(K, S)
    idx, w, _, _ = oracle.select(Q, Kb, G, S, k)
    O = oracle.forward(Q, K, V, idx, w, S, off_by_one=off1)
    o, di, dw, _ = oracle.decode(Q[:, t], K, V, Kb, [t], S, k, off_by_one=off1)
    assert np.array_equal(di[0], idx[0, t])
    np.testing.assert_allclose(dw[0], w[0, t], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(o[0], O[0, t], rtol=1e-12, atol=1e-14)


def test_decode_planted_chunk_is_selected():
    shape = hsa_synth.HsaShape(2, 8192, 16, 2, 128, 64, 8, "bf16")
    inp = hsa_synth.make_decode_inputs(shape, 4)
    Kb = oracle.landmarks(inp["Kc"], 64)
    o, idx, w, gap = oracle.decode(inp["q"], inp["Kc"], inp["Vc"], Kb, [8192, 8192], 64, 8)
    for b in range(2):
        for g in range(2):
            assert inp["planted"][b, g].item() in set(idx[b, g].tolist())


# ------------------------------------------------- selection over its own inputs ----

def _shared_selection_loss(Qs, Ks, layers, S, k, stick, off1, idx_ref):
    """Sec. 3.1 / Sec. 4.4: one selection from the selection inputs (Qs [B, L, G, d_sel],
    Ks [B, C, G, d_sel]) serves every layer; loss = sum over layers of sum(O_l * dO_l)."""
    G = Ks.shape[2]
    idx, w, _, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
    assert np.array_equal(idx, idx_ref), "selection moved under the perturbation"
    return sum(float((oracle.forward(Q, K, V, idx, w, S, off_by_one=off1) * dO).sum())
               for Q, K, V, dO in layers)


@pytest.mark.parametrize("stick,off1", [(False, False), (True, True)])
def test_shared_selection_finite_differences(stick, off1):
    """Two layers sharing a selection over separate inputs: each layer's backward without
    the score term, plus the selection backward of the summed dw, is the gradient of the
    summed loss w.r.t. every input (central differences, step 1e-6)."""
    L, h, d, S, k, G, dsel = 12, 2, 3, 2, 2, 2, 4
    C = L // S
    Qs = rnd(201, 1, L, G, dsel)
    Ks = rnd(202, 1, C, G, dsel, std=1.5)
    layers = [small_problem(210 + 10 * l, L=L, h=h, d=d, S=S, k=k, mu=1.0, G=G)
              for l in range(2)]
    idx, w, gap, _ = oracle.select(Qs, Ks, G, S, k, stick=stick)
    assert gap[np.isfinite(gap)].min() > 1e-4
    grads, dw = [], np.zeros_like(w)
    for Q, K, V, dO in layers:
        dQ, dK, dV, dwl = oracle.backward(Q, K, V, idx, w, dO, S, stick=stick,
                                          off_by_one=off1, separate=True)
        grads.append((dQ, dK, dV))
        dw += dwl
    dQs, dKs, _ = oracle.select_backward(Qs, Ks, idx, w, dw, G, S, stick=stick)
    eps = 1e-6

    def fd(X, put):
        num = np.zeros_like(X)
        it = np.nditer(X, flags=["multi_index"])
        for _ in it:
            i = it.multi_index
            Xp, Xm = X.copy(), X.copy()
            Xp[i] += eps
            Xm[i] -= eps
            num[i] = (put(Xp) - put(Xm)) / (2 * eps)
        return num

    loss = lambda Qs_, Ks_, ls_: _shared_selection_loss(Qs_, Ks_, ls_, S, k, stick, off1, idx)
    np.testing.assert_allclose(dQs, fd(Qs, lambda X: loss(X, Ks, layers)), rtol=1e-5,
                               atol=1e-7, err_msg="Qs")
    np.testing.assert_allclose(dKs, fd(Ks, lambda X: loss(Qs, X, layers)), rtol=1e-5,
                               atol=1e-7, err_msg="Ks")
    for l, (Q, K, V, dO) in enumerate(layers):
        for pos, name in ((0, "Q"), (1, "K"), (2, "V")):
            def put(X, pos=pos, l=l):
                ls_ = [list(t) for t in layers]
                ls_[l][pos] = X
                return loss(Qs, Ks, [tuple(t) for t in ls_])
            np.testing.assert_allclose(grads[l][pos], fd(layers[l][pos], put), rtol=1e-5,
                                       atol=1e-7, err_msg="layer %d %s" % (l, name))


@pytest.mark.parametrize("stick", [False, True])
def test_fused_score_term_is_the_selection_backward_of_the_head_sum(stick):
    """The fused form scores with q~ = sum_j q_j and Kbar = mean of the chunk's keys: its
    gradient is the attention-only gradient plus the selection backward of those inputs,
    with dKbar reaching every key of the chunk as dKbar / S."""
    L, h, d, S, k, G = 48, 2, 4, 4, 3, 2
    Q, K, V, dO = small_problem(231, L=L, h=h, d=d, S=S, k=k, G=G)
    Kb = oracle.landmarks(K, S)
    idx, w, _, _ = oracle.select(Q, Kb, G, S, k, stick=stick)
    dQ, dK, dV = oracle.backward(Q, K, V, idx, w, dO, S, stick=stick)
    dQa, dKa, dVa, dw = oracle.backward(Q, K, V, idx, w, dO, S, stick=stick, separate=True)
    dQs, dKb, _ = oracle.select_backward(Q, Kb, idx, w, dw, G, S, stick=stick)
    np.testing.assert_allclose(dV, dVa, rtol=0, atol=0)
    np.testing.assert_allclose(dQ, dQa + dQs, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(dK, dKa + np.repeat(dKb / S, S, axis=1), rtol=1e-12,
                               atol=1e-14)
