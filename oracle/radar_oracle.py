"""Plain fp64 CPU oracle for Radar's decode-time path.

TEST INFRASTRUCTURE ONLY. Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this module. The HIP library never
calls it, shares no code with it, and the product path has no CPU fallback.

Everything is float64 numpy. Inputs (fp32 or bf16 tensors) are widened exactly
by the caller (`np.float64(x)` of an fp32 / bf16 value is exact). Each function
cites the part of the paper it writes out: "Radar: Fast Long-Context Decoding
for Any Transformer" (ICLR 2025), Section 2 (Eq. 1-6), Algorithm 1 in
Appendix A, Lemma 1 / Lemma 6 for the random-feature map.

Readings taken where the paper is silent or inconsistent (full list with
reasons in the design notes):
  * omega_i is the i-th ROW of Omega [n][d] (the text says column).
  * x' = x / d^(1/4) scales queries and keys alike.
  * only full segments of c tokens are summarised; the unsummarised tail and
    the recent window form the buffer W, which is always attended.
  * W = [ws, t) with ws = c * floor(max(0, t - w) / c); candidate segments
    are the ws / c segments wholly before ws.
  * top-k order: score descending, then segment index ascending; k_eff =
    min(k, number of candidates).
  * grouped-query attention: each query head selects its own top-k; every
    head of a group attends the union of its group's selections plus W.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "random_features", "segment_summaries", "window_split", "segment_scores",
    "top_segments", "attended_tokens", "attend", "decode_head", "decode",
    "full_attention", "sqrt_schedule", "exact_segment_mass", "decode_exact",
]


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def random_features(x, omega):
    """Positive random-feature map phi_Omega (Section 2.2, Eq. 4).

    phi(x)_i = n^(-1/2) * exp(omega_i . x' - |x'|^2 / 2),  x' = x / d^(1/4),
    with omega_i the i-th row of Omega.

    x: [..., d]; omega: [n, d]. Returns [..., n].
    """
    x = _f64(x)
    omega = _f64(omega)
    d = x.shape[-1]
    n = omega.shape[0]
    assert omega.shape[1] == d
    xp = x / d ** 0.25
    proj = xp @ omega.T                                  # omega_i . x'
    half_sq = 0.5 * np.sum(xp * xp, axis=-1, keepdims=True)
    return np.exp(proj - half_sq) / np.sqrt(n)


def segment_summaries(keys, omega, c, n_seg=None, first=0):
    """Segment embeddings (Section 2.2, Eq. 5): the mean of phi over the c keys
    of each segment. Segment s (0-based) holds tokens [s*c, s*c + c).

    keys: [T, d] of one head; returns [n_seg - first, n] for segments
    first .. n_seg-1 (n_seg defaults to floor(T / c), the full segments).
    """
    keys = _f64(keys)
    if n_seg is None:
        n_seg = keys.shape[0] // c
    n = np.asarray(omega).shape[0]
    out = np.empty((n_seg - first, n))
    for s in range(first, n_seg):
        out[s - first] = random_features(keys[s * c:(s + 1) * c], omega).mean(0)
    return out


def window_split(t, c, w):
    """Partition of the context [0, t) used at a decode step (Algorithm 1's
    buffer W, generalised to a recent window of at least w tokens).

    Returns (ws, n_cand): W = [ws, t) is always attended; segments
    0 .. n_cand-1 (tokens [0, ws)) are the scoring candidates.
    """
    ws = c * (max(0, t - w) // c)
    return ws, ws // c


def segment_scores(phi_q, summaries):
    """Approximate segment attention a_s = phi(q) . phi_bar(segment s)
    (Section 2.2, Eq. 6) for every row of `summaries` [S, n]."""
    return _f64(summaries) @ _f64(phi_q)


def top_segments(scores, k):
    """Indices of the k segments with the highest scores (Algorithm 1,
    selection step), ordered by score descending, ties by lower index.
    Returns min(k, len(scores)) indices."""
    scores = _f64(scores)
    order = sorted(range(len(scores)), key=lambda s: (-scores[s], s))
    return np.asarray(order[:min(k, len(scores))], dtype=np.int64)


def attended_tokens(segments, c, ws, t):
    """Token positions attended: the union of the selected segments' tokens
    and the window W = [ws, t) (Algorithm 1, S <- S u W)."""
    segs = sorted(set(int(s) for s in segments))
    toks = [np.arange(s * c, s * c + c) for s in segs]
    toks.append(np.arange(ws, t))
    return np.concatenate(toks).astype(np.int64)


def attend(q, K, V, tokens):
    """Exact softmax attention of one query over the token set S
    (Section 2.1, Eq. 1-2, restricted to S as in Algorithm 1's output step):
    o = sum_{j in S} exp(q.k_j / sqrt(d)) v_j / sum_{j in S} exp(q.k_j / sqrt(d)).
    The max logit is subtracted before exponentiating (exact in real arithmetic).
    """
    q = _f64(q)
    Ks = _f64(K[tokens])
    Vs = _f64(V[tokens])
    d = q.shape[-1]
    logits = Ks @ q / np.sqrt(d)
    e = np.exp(logits - logits.max())
    return (e @ Vs) / e.sum()


def full_attention(q, K, V, t):
    """Causal attention of the query at position t-1 over all t tokens
    (Eq. 1-2)."""
    return attend(q, K, V, np.arange(t))


def decode_head(phi_q, summaries, n_cand, k):
    """Scores and top-k of one query head over the candidate segments."""
    sc = segment_scores(phi_q, summaries[:n_cand])
    sel = top_segments(sc, k)
    return sc, sel


def decode(q, K, V, omega, summaries, t, k, c, w):
    """One decode step for every (batch, query head) (Algorithm 1, querying
    procedure): phi(q) -> segment scores over the candidates -> top-k ->
    union over the query heads sharing a kv head -> exact attention over the
    union's tokens plus the window.

    q: [B, Hq, d]; K, V: [B, Hkv, >=t, d]; summaries: [B, Hkv, >=n_cand, n]
    (the oracle's own, from `segment_summaries`); t: current length (the
    query's own token is position t-1).

    Returns dict with
      out      [B, Hq, d]
      selected [B, Hq, k] int64, -1 padded, ordered as `top_segments`
      sel_scores [B, Hq, k] (nan padded)
      scores   list per (b, h): all candidate scores
      union    list per (b, g): sorted union of the group's selections
      ws, n_cand
    """
    q = _f64(q)
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    ws, n_cand = window_split(t, c, w)
    k_eff = min(k, n_cand)
    out = np.zeros((B, Hq, d))
    selected = -np.ones((B, Hq, k), dtype=np.int64)
    sel_scores = np.full((B, Hq, k), np.nan)
    scores = {}
    union = {}
    for b in range(B):
        for g in range(Hkv):
            heads = range(g * G, (g + 1) * G)
            picks = []
            for h in heads:
                phi_q = random_features(q[b, h], omega)
                sc, sel = decode_head(phi_q, summaries[b, g], n_cand, k)
                scores[(b, h)] = sc
                selected[b, h, :k_eff] = sel
                sel_scores[b, h, :k_eff] = sc[sel]
                picks.extend(sel.tolist())
            union[(b, g)] = sorted(set(picks))
            toks = attended_tokens(union[(b, g)], c, ws, t)
            for h in heads:
                out[b, h] = attend(q[b, h], K[b, g], V[b, g], toks)
    return dict(out=out, selected=selected, sel_scores=sel_scores,
                scores=scores, union=union, ws=ws, n_cand=n_cand, k_eff=k_eff)


def sqrt_schedule(t):
    """Algorithm 1's dynamic restructuring (Section 2.2, Appendix A): the
    segment length is reset to sqrt(t) whenever t is a perfect square, the c
    segments of c tokens then cover [0, c^2), and every later token waits in
    the buffer W until the next perfect square. At context length t >= 1
    this gives c = floor(sqrt(t)) and W = [c^2, t).

    Returns (c, w) such that window_split(t, c, w) reproduces that state:
    w = t - c^2, so ws = c * floor(c^2 / c) = c^2 and the candidates are
    the c restructured segments."""
    assert t >= 1
    c = int(np.floor(np.sqrt(t)))
    while c * c > t:
        c -= 1
    while (c + 1) * (c + 1) <= t:
        c += 1
    return c, t - c * c


def exact_segment_mass(q, keys, c, n_cand):
    """Exact segment attention mass (the quantity Theorem 2's proof calls
    beta): beta_s = sum over the c keys of segment s of exp(q . k / sqrt(d)),
    the unnormalised attention weight the segment carries. Selecting the k
    largest is the exact segment search of the ablation study (Section 3.3).
    Returns ln(beta_s) for s < n_cand (the log keeps large logits finite;
    each segment subtracts its own max logit before exponentiating)."""
    q = _f64(q)
    keys = _f64(keys)
    d = q.shape[-1]
    out = np.empty(n_cand)
    for s in range(n_cand):
        lg = keys[s * c:(s + 1) * c] @ q / np.sqrt(d)
        m = lg.max()
        out[s] = m + np.log(np.exp(lg - m).sum())
    return out


def decode_exact(q, K, V, t, k, c, w):
    """decode() with the exact segment search in place of the random-feature
    scores: every query head selects the k segments with the largest
    beta_s; the union over the heads sharing a kv head plus the window is
    attended exactly. Returns the same dict as decode() with `scores` and
    `sel_scores` holding ln(beta)."""
    q = _f64(q)
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    ws, n_cand = window_split(t, c, w)
    k_eff = min(k, n_cand)
    out = np.zeros((B, Hq, d))
    selected = -np.ones((B, Hq, k), dtype=np.int64)
    sel_scores = np.full((B, Hq, k), np.nan)
    scores, union = {}, {}
    for b in range(B):
        for g in range(Hkv):
            heads = range(g * G, (g + 1) * G)
            picks = []
            for h in heads:
                sc = exact_segment_mass(q[b, h], K[b, g], c, n_cand)
                sel = top_segments(sc, k)
                scores[(b, h)] = sc
                selected[b, h, :k_eff] = sel
                sel_scores[b, h, :k_eff] = sc[sel]
                picks.extend(sel.tolist())
            union[(b, g)] = sorted(set(picks))
            toks = attended_tokens(union[(b, g)], c, ws, t)
            for h in heads:
                out[b, h] = attend(q[b, h], K[b, g], V[b, g], toks)
    return dict(out=out, selected=selected, sel_scores=sel_scores,
                scores=scores, union=union, ws=ws, n_cand=n_cand, k_eff=k_eff)
