"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own formula: they use hand-derived
closed forms (tests/golden), expectations proved in the paper (Lemma 1 and
Lemma 6, checked by Monte Carlo within a standard-error bound), brute force on
tiny inputs, a library attention routine for the special case where Radar
selects every segment, and invariants of exact attention.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch

from oracle import radar_oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# Eq. 4 / Eq. 5 worked by hand
# --------------------------------------------------------------------------
def _expr(s):
    return float(eval(s, {"__builtins__": {}}, {"sqrt": math.sqrt,
                                                "exp": math.exp}))


def _load_cases(path):
    cases, cur = [], None
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, _, rest = line.partition(" ")
        if key == "case":
            cur = {"name": rest, "x": []}
            cases.append(cur)
        elif key == "d":
            cur["d"] = int(rest)
        elif key == "omega":
            cur["omega"] = [[_expr(v) for v in row.split()]
                            for row in rest.split(";")]
        elif key == "x":
            cur["x"].append([_expr(v) for v in rest.split()])
        elif key in ("phi", "mean"):
            cur.setdefault(key, []).append([_expr(v) for v in rest.split()])
    return cases


CASES = _load_cases(os.path.join(GOLDEN, "phi_closed_forms.txt"))


@pytest.mark.parametrize("case", CASES, ids=[c["name"] for c in CASES])
def test_phi_and_segment_mean_closed_forms(case):
    omega = np.array(case["omega"])
    x = np.array(case["x"])
    assert x.shape[1] == case["d"] == omega.shape[1]
    if "phi" in case:
        got = orc.random_features(x, omega)
        np.testing.assert_allclose(got, np.array(case["phi"]), rtol=1e-14,
                                   atol=0)
    if "mean" in case:
        got = orc.segment_summaries(x, omega, c=len(x))
        np.testing.assert_allclose(got, np.array(case["mean"]), rtol=1e-14,
                                   atol=0)


# --------------------------------------------------------------------------
# Lemma 1 and Lemma 6 (Monte Carlo over Omega, 5 standard errors)
# --------------------------------------------------------------------------
def _unit_scaled(rng, d, norm):
    """A vector whose scaled copy x' = x / d^(1/4) has the given norm."""
    v = rng.standard_normal(d)
    return v / np.linalg.norm(v) * norm * d ** 0.25


@pytest.mark.parametrize("d,nu,nv,seed", [(8, 0.8, 0.6, 0), (16, 1.0, 0.5, 1),
                                          (4, 0.3, 0.9, 2)])
def test_lemma1_expectation(d, nu, nv, seed):
    # E_Omega[phi(u) . phi(v)] = exp(u.v / sqrt(d))          (Lemma 1)
    rng = np.random.default_rng(seed)
    u, v = _unit_scaled(rng, d, nu), _unit_scaled(rng, d, nv)
    n, M = 64, 3000
    est = np.array([orc.random_features(u, om) @ orc.random_features(v, om)
                    for om in rng.standard_normal((M, n, d))])
    target = math.exp(u @ v / math.sqrt(d))
    up, vp = u / d ** 0.25, v / d ** 0.25
    # per-feature variance from Lemma 6 (property 4) on the scaled vectors
    var_f = math.exp(2 * up @ vp) * (math.exp((up + vp) @ (up + vp)) - 1)
    se = math.sqrt(var_f / (n * M))
    assert abs(est.mean() - target) <= 5 * se, (est.mean(), target, se)


def _features_f(x, omega):
    """f_{x'}(omega_i) = sqrt(n) * phi(x)_i (Definition 5 vs Eq. 4)."""
    return orc.random_features(x, omega) * math.sqrt(omega.shape[0])


def test_lemma6_mean_and_variance():
    rng = np.random.default_rng(7)
    d, N = 4, 1_000_000
    om = rng.standard_normal((N, d))
    u = _unit_scaled(rng, d, 0.7)
    v = _unit_scaled(rng, d, 0.4)
    up, vp = u / d ** 0.25, v / d ** 0.25
    fu, fv = _features_f(u, om), _features_f(v, om)
    # property 1: non-negative
    assert (fu >= 0).all() and (fv >= 0).all()
    # property 2: E[f_u] = 1, Var[f_u] = e^{|u|^2} - 1 (property 4 with v=0)
    se = math.sqrt((math.exp(up @ up) - 1) / N)
    assert abs(fu.mean() - 1) <= 5 * se
    # property 3: E[f_u f_v] = e^{u.v}
    p = fu * fv
    var_p = math.exp(2 * up @ vp) * (math.exp((up + vp) @ (up + vp)) - 1)
    assert abs(p.mean() - math.exp(up @ vp)) <= 5 * math.sqrt(var_p / N)
    # property 4: Var[f_u f_v] = e^{2u.v}(e^{|u+v|^2} - 1); SE of the sample
    # variance from the sample's own fourth central moment
    c = p - p.mean()
    se_var = math.sqrt(max(np.mean(c ** 4) - np.mean(c ** 2) ** 2, 0) / N)
    assert abs(c.var() - var_p) <= 5 * se_var, (c.var(), var_p, se_var)


def test_lemma6_covariance():
    rng = np.random.default_rng(11)
    d, N = 4, 1_000_000
    om = rng.standard_normal((N, d))
    u, v, z = (_unit_scaled(rng, d, r) for r in (0.5, 0.6, 0.4))
    up, vp, zp = (x / d ** 0.25 for x in (u, v, z))
    a = _features_f(u, om) * _features_f(z, om)
    b = _features_f(v, om) * _features_f(z, om)
    # property 5: Cov(f_u f_z, f_v f_z) = e^{(u+v).z}(e^{(u+z).(v+z)} - 1)
    target = math.exp((up + vp) @ zp) * (math.exp((up + zp) @ (vp + zp)) - 1)
    prod = (a - a.mean()) * (b - b.mean())
    se = prod.std() / math.sqrt(N)
    assert abs(prod.mean() - target) <= 5 * se, (prod.mean(), target, se)


def test_segment_score_expectation():
    # E_Omega[phi(q) . phi_bar(seg s)] = (1/c) sum_{j in s} exp(q.k_j/sqrt(d))
    # (Lemma 1 + linearity of Eq. 5 / Eq. 6); pins segment boundaries and 1/c.
    rng = np.random.default_rng(3)
    d, c, n_seg, n, M = 8, 3, 4, 64, 3000
    K = rng.standard_normal((c * n_seg + 2, d)) * 0.35
    q = rng.standard_normal(d) * 0.35
    acc = np.zeros(n_seg)
    sq = np.zeros(n_seg)
    for om in rng.standard_normal((M, n, d)):
        sc = orc.segment_scores(orc.random_features(q, om),
                                orc.segment_summaries(K, om, c))
        acc += sc
        sq += sc * sc
    mean = acc / M
    se = np.sqrt((sq / M - mean ** 2) / M)
    target = np.array([np.mean(np.exp(K[s * c:(s + 1) * c] @ q / math.sqrt(d)))
                       for s in range(n_seg)])
    assert (np.abs(mean - target) <= 5 * se).all(), (mean, target, se)
    # only full segments are summarised (the 2-token tail is not)
    assert orc.segment_summaries(K, om, c).shape == (n_seg, n)


def test_planted_constant_segments():
    # A segment whose c keys are all u_s has embedding phi(u_s), so a segment
    # boundary off by one would mix neighbours.
    rng = np.random.default_rng(5)
    d, c, n_seg, n = 6, 5, 7, 32
    U = rng.standard_normal((n_seg, d))
    K = np.repeat(U, c, axis=0)
    om = rng.standard_normal((n, d))
    got = orc.segment_summaries(K, om, c)
    for s in range(n_seg):
        np.testing.assert_allclose(got[s], orc.random_features(U[s], om),
                                   rtol=1e-13)
    # c = 1: the embedding of a one-token segment is that token's feature
    np.testing.assert_allclose(orc.segment_summaries(K, om, 1),
                               orc.random_features(K, om), rtol=1e-13)


# --------------------------------------------------------------------------
# top-k: brute force over subsets, tie order
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n_cand,k,seed", [(1, 1, 0), (5, 2, 1), (9, 4, 2),
                                           (12, 5, 3), (7, 7, 4), (6, 9, 5)])
def test_top_segments_brute_force(n_cand, k, seed):
    rng = np.random.default_rng(seed)
    sc = rng.standard_normal(n_cand)
    sel = orc.top_segments(sc, k)
    k_eff = min(k, n_cand)
    assert len(sel) == k_eff and len(set(sel.tolist())) == k_eff
    best = max(itertools.combinations(range(n_cand), k_eff),
               key=lambda s: sum(sc[list(s)]))
    assert set(sel.tolist()) == set(best)
    assert all(sc[sel[i]] >= sc[sel[i + 1]] for i in range(k_eff - 1))


def test_top_segments_ties_lower_index_first():
    sc = np.array([1.0, 3.0, 2.0, 3.0, 2.0, 3.0, 0.5])
    assert orc.top_segments(sc, 2).tolist() == [1, 3]
    assert orc.top_segments(sc, 4).tolist() == [1, 3, 5, 2]
    assert orc.top_segments(sc, 5).tolist() == [1, 3, 5, 2, 4]


# --------------------------------------------------------------------------
# window / buffer bookkeeping
# --------------------------------------------------------------------------
@pytest.mark.parametrize("c", [1, 3, 8])
@pytest.mark.parametrize("w", [0, 1, 5, 8, 20])
def test_window_partition(c, w):
    for t in range(1, 70):
        ws, n_cand = orc.window_split(t, c, w)
        assert ws % c == 0 and n_cand * c == ws and 0 <= ws <= t
        # W holds at least min(t, w) and at most w + c - 1 tokens
        assert min(t, w) <= t - ws <= w + c - 1
        # candidates + W partition [0, t): with every candidate selected the
        # attended tokens are exactly 0..t-1, each once
        toks = orc.attended_tokens(range(n_cand), c, ws, t)
        assert toks.tolist() == list(range(t))


@pytest.mark.parametrize("c", [1, 2, 5])
def test_window_zero_is_algorithm1_buffer(c):
    # With w = 0 the window is the unregistered buffer of Algorithm 1 at a
    # fixed segment length: simulate the buffer as a state machine (append
    # each new token; once it holds c tokens they become a segment).
    buffer, segments = [], 0
    for t in range(1, 60):
        buffer.append(t - 1)
        if len(buffer) == c:
            segments += 1
            buffer = []
        ws, n_cand = orc.window_split(t, c, 0)
        assert n_cand == segments
        assert list(range(ws, t)) == buffer


# --------------------------------------------------------------------------
# attention: library routine and invariants
# --------------------------------------------------------------------------
def _sdpa(q, K, V, mask=None):
    """torch's scaled_dot_product_attention in fp64 on the CPU."""
    qt = torch.as_tensor(q, dtype=torch.float64)[None, None, None, :]
    Kt = torch.as_tensor(K, dtype=torch.float64)[None, None]
    Vt = torch.as_tensor(V, dtype=torch.float64)[None, None]
    m = None if mask is None else torch.as_tensor(mask)[None, None, None, :]
    return torch.nn.functional.scaled_dot_product_attention(
        qt, Kt, Vt, attn_mask=m)[0, 0, 0].numpy()


@pytest.mark.parametrize("B,Hq,Hkv,d,t,c,w,n", [
    (1, 2, 2, 16, 50, 8, 8, 32),     # MHA, partial tail
    (2, 4, 2, 8, 37, 4, 6, 16),      # GQA
    (1, 3, 1, 8, 5, 4, 16, 16),      # t < w: window only
    (1, 2, 2, 8, 64, 8, 0, 16),      # w = 0, segment-aligned t
    (1, 1, 1, 4, 1, 1, 0, 8),        # a single token
])
def test_all_segments_selected_is_full_attention(B, Hq, Hkv, d, t, c, w, n):
    # k >= number of candidates: S = [0, t) and the output is exact causal
    # softmax attention (Eq. 1-2).
    rng = np.random.default_rng(t + d)
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, t + 3, d))
    V = rng.standard_normal((B, Hkv, t + 3, d))
    om = rng.standard_normal((n, d))
    summ = np.stack([np.stack([orc.segment_summaries(K[b, g, :t], om, c)
                               for g in range(Hkv)]) for b in range(B)])
    _, n_cand = orc.window_split(t, c, w)
    res = orc.decode(q, K, V, om, summ, t, max(n_cand, 1), c, w)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            ref = _sdpa(q[b, h], K[b, h // G, :t], V[b, h // G, :t])
            np.testing.assert_allclose(res["out"][b, h], ref, rtol=1e-12,
                                       atol=1e-13)


def test_attend_matches_masked_library_attention():
    rng = np.random.default_rng(9)
    d, T = 16, 40
    q, K, V = (rng.standard_normal(s) for s in (d, (T, d), (T, d)))
    toks = np.array(sorted(rng.choice(T, 13, replace=False)))
    mask = np.zeros(T, dtype=bool)
    mask[toks] = True
    np.testing.assert_allclose(orc.attend(q, K, V, toks), _sdpa(q, K, V, mask),
                               rtol=1e-12, atol=1e-13)


def test_attention_invariants():
    rng = np.random.default_rng(13)
    d, T = 8, 30
    q = rng.standard_normal(d)
    V = rng.standard_normal((T, d))
    toks = np.arange(3, 21)
    # identical keys: uniform weights, the output is the mean of V over S
    K = np.tile(rng.standard_normal(d), (T, 1))
    np.testing.assert_allclose(orc.attend(q, K, V, toks), V[toks].mean(0),
                               rtol=1e-13)
    K = rng.standard_normal((T, d)) * 3
    # constant V: the output is that value
    Vc = np.tile(rng.standard_normal(d), (T, 1))
    np.testing.assert_allclose(orc.attend(q, K, Vc, toks), Vc[0], rtol=1e-13)
    # a single token: the output is its value
    np.testing.assert_allclose(orc.attend(q, K, V, np.array([7])), V[7],
                               rtol=1e-15)
    # permutation invariance over S
    perm = rng.permutation(toks)
    np.testing.assert_allclose(orc.attend(q, K, V, perm),
                               orc.attend(q, K, V, toks), rtol=1e-13)
    # large logits: subtracting the max keeps exp finite
    np.testing.assert_allclose(orc.attend(q * 400, K, Vc, toks), Vc[0],
                               rtol=1e-13)


def test_gqa_heads_attend_group_union_plus_window():
    rng = np.random.default_rng(21)
    B, Hq, Hkv, d, c, w, n, k = 1, 4, 2, 8, 4, 5, 32, 2
    t = 43
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, t, d))
    V = rng.standard_normal((B, Hkv, t, d))
    om = rng.standard_normal((n, d))
    summ = np.stack([np.stack([orc.segment_summaries(K[0, g], om, c)
                               for g in range(Hkv)])])
    res = orc.decode(q, K, V, om, summ, t, k, c, w)
    ws, n_cand = orc.window_split(t, c, w)
    G = Hq // Hkv
    for g in range(Hkv):
        heads = range(g * G, (g + 1) * G)
        sel = set(res["selected"][0, list(heads)].ravel().tolist())
        assert res["union"][(0, g)] == sorted(sel)
        mask = np.zeros(t, dtype=bool)
        mask[ws:t] = True
        for s in sel:
            mask[s * c:(s + 1) * c] = True
        # attended tokens = |U| c + |W|   (Appendix A, final attention step)
        assert mask.sum() == len(sel) * c + (t - ws)
        for h in heads:
            np.testing.assert_allclose(res["out"][0, h],
                                       _sdpa(q[0, h], K[0, g], V[0, g], mask),
                                       rtol=1e-12, atol=1e-13)
    # each head's selection is its own top-k over the candidates
    for h in range(Hq):
        sc = res["scores"][(0, h)]
        assert len(sc) == n_cand
        top = res["selected"][0, h]
        assert (sc[top] >= np.sort(sc)[-k] - 1e-15).all()


def test_selection_finds_planted_segment():
    # A query equal to a key that is far larger than the rest picks that key's
    # segment first: the approximate segment score follows the true segment
    # attention when the gap is large (Theorem 2).
    rng = np.random.default_rng(17)
    d, c, n, T = 16, 8, 256, 96
    K = rng.standard_normal((T, d)) * 0.3
    K[45] = rng.standard_normal(d) * 1.5
    om = rng.standard_normal((n, d))
    summ = orc.segment_summaries(K, om, c)
    sc = orc.segment_scores(orc.random_features(K[45], om), summ)
    assert orc.top_segments(sc, 1)[0] == 45 // c


# --------------------------------------------------------------------------
# Algorithm 1's restructuring schedule
# --------------------------------------------------------------------------
def test_sqrt_schedule_matches_algorithm1_state_machine():
    # Run Algorithm 1's bookkeeping literally (1-based tokens): t <- t + 1;
    # if sqrt(t) is an integer, c <- sqrt(t) and the buffer W is emptied,
    # otherwise token t joins W. The schedule must reproduce c, the
    # candidate segments (c segments of c tokens) and W at every t.
    c, W = 0, []
    for t in range(1, 3000):
        r = math.isqrt(t)
        if r * r == t:
            c, W = r, []
        else:
            W.append(t)
        cs, w = orc.sqrt_schedule(t)
        ws, n_cand = orc.window_split(t, cs, w)
        assert cs == c and n_cand == c and ws == c * c
        # W holds the 1-based tokens c^2 + 1 .. t, i.e. 0-based [c^2, t)
        assert list(range(ws, t)) == [j - 1 for j in W]
        # the buffer never exceeds 2 sqrt(t) - 1 tokens (Section 2.2)
        assert len(W) <= 2 * math.sqrt(t) - 1


def test_sqrt_schedule_decode_is_algorithm1_query():
    # At a restructure step the query attends only the selected segments;
    # with every segment selected that is full attention over [0, t).
    rng = np.random.default_rng(31)
    d, n, t = 8, 32, 49
    c, w = orc.sqrt_schedule(t)
    assert (c, w) == (7, 0)
    q = rng.standard_normal((1, 1, d))
    K = rng.standard_normal((1, 1, t, d))
    V = rng.standard_normal((1, 1, t, d))
    om = rng.standard_normal((n, d))
    summ = orc.segment_summaries(K[0, 0], om, c)[None, None]
    res = orc.decode(q, K, V, om, summ, t, c, c, w)
    np.testing.assert_allclose(res["out"][0, 0], _sdpa(q[0, 0], K[0, 0], V[0, 0]),
                               rtol=1e-12, atol=1e-13)
    # with k = 2 the attended set is exactly two segments (W is empty)
    res = orc.decode(q, K, V, om, summ, t, 2, c, w)
    toks = orc.attended_tokens(res["selected"][0, 0], c, c * c, t)
    assert len(toks) == 2 * c


# --------------------------------------------------------------------------
# exact segment search (segment attention mass beta)
# --------------------------------------------------------------------------
def test_exact_mass_one_token_segments_is_token_topk():
    # c = 1: beta_s = exp(q . k_s / sqrt(d)), so the exact search is the
    # token top-k of the problem statement (Eq. 3) by the logit itself.
    rng = np.random.default_rng(41)
    d, T, k = 16, 40, 7
    q = rng.standard_normal(d)
    K = rng.standard_normal((T, d)) * 2
    lnb = orc.exact_segment_mass(q, K, 1, T)
    np.testing.assert_allclose(lnb, K @ q / 4.0, rtol=1e-13, atol=1e-13)
    assert orc.top_segments(lnb, k).tolist() == np.argsort(-(K @ q))[:k].tolist()


def test_exact_mass_constant_segment_and_full_normaliser():
    rng = np.random.default_rng(43)
    d, c, ns = 9, 6, 5
    q = rng.standard_normal(d) * 3
    U = rng.standard_normal((ns, d)) * 3
    K = np.repeat(U, c, axis=0)
    # identical keys: beta_s = c exp(q . u_s / sqrt(d))
    np.testing.assert_allclose(orc.exact_segment_mass(q, K, c, ns),
                               np.log(c) + U @ q / 3.0, rtol=1e-13)
    # the segments' masses add up to the softmax normaliser of the tokens
    K = rng.standard_normal((c * ns, d)) * 3
    lnz = torch.logsumexp(torch.as_tensor(K @ q / 3.0), 0).item()
    lnb = orc.exact_segment_mass(q, K, c, ns)
    assert abs(np.log(np.exp(lnb - lnb.max()).sum()) + lnb.max() - lnz) < 1e-12


def test_radar_score_estimates_exact_mass():
    # E_Omega[phi(q) . phi_bar(s)] = beta_s / c (Lemma 1 with Eq. 5-6): the
    # random-feature score is an unbiased estimate of the exact mass.
    rng = np.random.default_rng(47)
    d, c, ns, n, M = 8, 4, 5, 64, 3000
    K = rng.standard_normal((c * ns, d)) * 0.35
    q = rng.standard_normal(d) * 0.35
    beta = np.exp(orc.exact_segment_mass(q, K, c, ns))
    est = np.zeros(ns)
    sq = np.zeros(ns)
    for om in rng.standard_normal((M, n, d)):
        a = orc.segment_scores(orc.random_features(q, om),
                               orc.segment_summaries(K, om, c))
        est += a
        sq += a * a
    mean = est / M
    se = np.sqrt((sq / M - mean ** 2) / M)
    assert (np.abs(mean - beta / c) <= 5 * se).all(), (mean, beta / c, se)


def test_decode_exact_all_selected_is_full_attention():
    rng = np.random.default_rng(53)
    B, Hq, Hkv, d, t, c, w = 1, 4, 2, 8, 45, 4, 6
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, t, d))
    V = rng.standard_normal((B, Hkv, t, d))
    _, n_cand = orc.window_split(t, c, w)
    res = orc.decode_exact(q, K, V, t, n_cand, c, w)
    for h in range(Hq):
        np.testing.assert_allclose(res["out"][0, h],
                                   _sdpa(q[0, h], K[0, h // 2], V[0, h // 2]),
                                   rtol=1e-12, atol=1e-13)


# --------------------------------------------------------------------------
# serving options: attention sinks, per-head GQA attention, ragged batches
# --------------------------------------------------------------------------
def _summ(K, om, c, n_sink, B, Hkv, t):
    return np.stack([np.stack([orc.segment_summaries(K[b, g, :t], om, c,
                                                     offset=n_sink)
                               for g in range(Hkv)]) for b in range(B)])


@pytest.mark.parametrize("t,c,w,n_sink", [
    (50, 8, 8, 4), (50, 8, 0, 1), (3, 4, 2, 5), (5, 4, 2, 5), (64, 8, 0, 8),
    (100, 7, 3, 20), (21, 4, 30, 2)])
def test_sink_layout_partitions_the_context(t, c, w, n_sink):
    """Sinks, candidate segments and the window are disjoint and cover
    [0, t); the candidates are whole c-blocks after the sinks; the window
    holds at least min(w, t - sinks) and fewer than w + c tokens."""
    ws, n_cand = orc.window_split(t, c, w, n_sink)
    toks = orc.attended_tokens(range(n_cand), c, ws, t, n_sink)
    assert sorted(toks.tolist()) == list(range(t))
    sink = min(n_sink, t)
    assert ws == sink + n_cand * c
    rest = t - sink
    if rest <= w:
        assert t - ws == rest
    else:
        assert w <= t - ws <= w + c - 1
    if t <= n_sink:
        assert (ws, n_cand) == (t, 0)


@pytest.mark.parametrize("t,c,w,n_sink,Hq,Hkv", [
    (50, 8, 8, 4, 2, 2), (37, 4, 6, 3, 4, 2), (5, 4, 2, 9, 2, 1),
    (64, 8, 0, 8, 2, 2), (9, 4, 0, 1, 1, 1)])
def test_sinks_all_selected_is_full_attention(t, c, w, n_sink, Hq, Hkv):
    rng = np.random.default_rng(t + n_sink)
    B, d, n = 2, 8, 16
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, t + 2, d))
    V = rng.standard_normal((B, Hkv, t + 2, d))
    om = rng.standard_normal((n, d))
    summ = _summ(K, om, c, n_sink, B, Hkv, t)
    _, n_cand = orc.window_split(t, c, w, n_sink)
    G = Hq // Hkv
    for per_head in (False, True):
        res = orc.decode(q, K, V, om, summ, t, max(n_cand, 1), c, w,
                         n_sink=n_sink, per_head=per_head)
        ex = orc.decode_exact(q, K, V, t, max(n_cand, 1), c, w,
                              n_sink=n_sink, per_head=per_head)
        for b in range(B):
            for h in range(Hq):
                ref = _sdpa(q[b, h], K[b, h // G, :t], V[b, h // G, :t])
                np.testing.assert_allclose(res["out"][b, h], ref, rtol=1e-12,
                                           atol=1e-13)
                np.testing.assert_allclose(ex["out"][b, h], ref, rtol=1e-12,
                                           atol=1e-13)


def test_sink_is_attended_even_when_unselected():
    """One sink key aligned with the query carries almost all the softmax
    weight: the output tends to that token's value although no segment
    holds it (exp(-25) bounds the rest)."""
    rng = np.random.default_rng(5)
    d, t, c, w, n = 8, 60, 4, 4, 32
    q = rng.standard_normal((1, 1, d))
    q /= np.linalg.norm(q)
    K = rng.standard_normal((1, 1, t, d)) * 0.3
    K[0, 0, 0] = 75.0 * q[0, 0]                 # logit 75 / sqrt(8) ~ 26.5
    V = rng.standard_normal((1, 1, t, d))
    om = rng.standard_normal((n, d))
    summ = _summ(K, om, c, 1, 1, 1, t)
    res = orc.decode(q, K, V, om, summ, t, 1, c, w, n_sink=1)
    assert 0 not in res["selected"][0, 0]       # segment ids count after sinks
    np.testing.assert_allclose(res["out"][0, 0], V[0, 0, 0], atol=1e-8)
    # without the sink option token 0 sits in segment 0 and may be dropped
    summ0 = _summ(K, om, c, 0, 1, 1, t)
    res0 = orc.decode(q, K, V, om, summ0, t, 1, c, w)
    toks0 = orc.attended_tokens(res0["selected"][0, 0], c, res0["ws"], t)
    assert (0 in toks0) == np.allclose(res0["out"][0, 0], V[0, 0, 0],
                                       atol=1e-8)


def test_sink_summaries_are_the_shifted_segments():
    rng = np.random.default_rng(8)
    K = rng.standard_normal((70, 8))
    om = rng.standard_normal((16, 8))
    # the offset path equals the hand-pinned offset-0 path on shifted keys
    got = orc.segment_summaries(K, om, 6, offset=5)
    assert got.shape == ((70 - 5) // 6, 16)
    np.testing.assert_array_equal(got, orc.segment_summaries(K[5:], om, 6))
    np.testing.assert_array_equal(
        orc.segment_summaries(K, om, 6, n_seg=7, first=3, offset=5), got[3:7])


def test_per_head_gqa_is_mha_on_repeated_kv():
    """Per-head GQA attention equals MHA (one kv head per query head) on the
    group's K / V and summaries repeated per head: there each head's union
    is its own selection."""
    rng = np.random.default_rng(17)
    B, Hq, Hkv, d, c, w, n, k, t, s0 = 2, 8, 2, 8, 4, 5, 32, 2, 61, 3
    G = Hq // Hkv
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, t, d))
    V = rng.standard_normal((B, Hkv, t, d))
    om = rng.standard_normal((n, d))
    summ = _summ(K, om, c, s0, B, Hkv, t)
    gqa = orc.decode(q, K, V, om, summ, t, k, c, w, n_sink=s0, per_head=True)
    Kr, Vr, Sr = (np.repeat(x, G, axis=1) for x in (K, V, summ))
    mha = orc.decode(q, Kr, Vr, om, Sr, t, k, c, w, n_sink=s0)
    np.testing.assert_array_equal(gqa["selected"], mha["selected"])
    np.testing.assert_allclose(gqa["out"], mha["out"], rtol=1e-13, atol=1e-14)
    # the union mode differs from it once the group's selections differ
    uni = orc.decode(q, K, V, om, summ, t, k, c, w, n_sink=s0)
    np.testing.assert_array_equal(uni["selected"], gqa["selected"])
    differ = [(b, g) for b in range(B) for g in range(Hkv)
              if len(uni["union"][(b, g)]) > k]
    assert differ
    b, g = differ[0]
    assert not np.allclose(uni["out"][b, g * G:(g + 1) * G],
                           gqa["out"][b, g * G:(g + 1) * G])


def test_ragged_batch_is_per_sequence_decode():
    rng = np.random.default_rng(23)
    B, Hq, Hkv, d, c, w, n, k, s0 = 4, 4, 2, 8, 5, 6, 32, 3, 2
    lens = [9, 64, 1, 40]
    T = max(lens)
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, T, d))
    V = rng.standard_normal((B, Hkv, T, d))
    om = rng.standard_normal((n, d))
    summ = _summ(K, om, c, s0, B, Hkv, T)
    for per_head in (False, True):
        rag = orc.decode(q, K, V, om, summ, lens, k, c, w, n_sink=s0,
                         per_head=per_head)
        rex = orc.decode_exact(q, K, V, lens, k, c, w, n_sink=s0,
                               per_head=per_head)
        for b, tb in enumerate(lens):
            one = orc.decode(q[b:b + 1], K[b:b + 1, :, :tb], V[b:b + 1, :, :tb],
                             om, summ[b:b + 1], tb, k, c, w, n_sink=s0,
                             per_head=per_head)
            np.testing.assert_array_equal(rag["selected"][b], one["selected"][0])
            np.testing.assert_allclose(rag["out"][b], one["out"][0], rtol=1e-14)
            ex1 = orc.decode_exact(q[b:b + 1], K[b:b + 1, :, :tb],
                                   V[b:b + 1, :, :tb], tb, k, c, w, n_sink=s0,
                                   per_head=per_head)
            np.testing.assert_allclose(rex["out"][b], ex1["out"][0], rtol=1e-14)
            assert rag["n_cand_b"][b] == orc.window_split(tb, c, w, s0)[1]
