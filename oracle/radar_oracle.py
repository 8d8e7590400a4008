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


def segment_summaries(keys, omega, c, n_seg=None, first=0, offset=0):
    """Segment embeddings (Section 2.2, Eq. 5): the mean of phi over the c keys
    of each segment. Segment s (0-based) holds tokens [offset + s*c,
    offset + s*c + c); offset is the number of sink tokens that precede the
    segments (0 without sinks).

    keys: [T, d] of one head; returns [n_seg - first, n] for segments
    first .. n_seg-1 (n_seg defaults to floor((T - offset) / c), the full
    segments).
    """
    keys = _f64(keys)
    if n_seg is None:
        n_seg = max(0, keys.shape[0] - offset) // c
    n = np.asarray(omega).shape[0]
    out = np.empty((n_seg - first, n))
    for s in range(first, n_seg):
        lo = offset + s * c
        out[s - first] = random_features(keys[lo:lo + c], omega).mean(0)
    return out


def window_split(t, c, w, n_sink=0):
    """Partition of the context [0, t) used at a decode step (Algorithm 1's
    buffer W, generalised to a recent window of at least w tokens).

    Returns (ws, n_cand): W = [ws, t) is always attended; segments
    0 .. n_cand-1 are the scoring candidates. Without sinks they cover
    [0, ws). With n_sink attention-sink tokens, tokens [0, min(n_sink, t))
    are always attended and belong to no segment; segment s covers
    [n_sink + s*c, n_sink + s*c + c), and the split applies to the tokens
    after the sinks: ws = n_sink + c * floor(max(0, t - n_sink - w) / c)
    (ws = t when t <= n_sink).
    """
    sink = min(n_sink, t)
    rest = t - sink
    ws_rel = c * (max(0, rest - w) // c)
    return sink + ws_rel, ws_rel // c


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


def attended_tokens(segments, c, ws, t, n_sink=0):
    """Token positions attended: the sink tokens [0, min(n_sink, ws)), the
    union of the selected segments' tokens and the window W = [ws, t)
    (Algorithm 1, S <- S u W)."""
    segs = sorted(set(int(s) for s in segments))
    toks = [np.arange(0, min(n_sink, ws))]
    toks += [np.arange(n_sink + s * c, n_sink + s * c + c) for s in segs]
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


def _decode(q, K, V, t, k, c, w, n_sink, per_head, head_scores):
    """Shared body of decode() and decode_exact(): head_scores(b, g, h,
    n_cand) gives one query head's candidate scores."""
    q = _f64(q)
    B, Hq, d = q.shape
    Hkv = K.shape[1]
    G = Hq // Hkv
    lens = [int(t)] * B if np.ndim(t) == 0 else [int(x) for x in t]
    assert len(lens) == B
    out = np.zeros((B, Hq, d))
    selected = -np.ones((B, Hq, k), dtype=np.int64)
    sel_scores = np.full((B, Hq, k), np.nan)
    scores, union = {}, {}
    ws_b, nc_b, ke_b = [], [], []
    for b in range(B):
        tb = lens[b]
        ws, n_cand = window_split(tb, c, w, n_sink)
        k_eff = min(k, n_cand)
        ws_b.append(ws); nc_b.append(n_cand); ke_b.append(k_eff)
        for g in range(Hkv):
            heads = range(g * G, (g + 1) * G)
            own = {}
            for h in heads:
                sc = head_scores(b, g, h, n_cand)
                sel = top_segments(sc, k)
                scores[(b, h)] = sc
                selected[b, h, :k_eff] = sel
                sel_scores[b, h, :k_eff] = sc[sel]
                own[h] = sel.tolist()
            union[(b, g)] = sorted(set(s for h in heads for s in own[h]))
            for h in heads:
                segs = own[h] if per_head else union[(b, g)]
                toks = attended_tokens(segs, c, ws, tb, n_sink)
                out[b, h] = attend(q[b, h], K[b, g], V[b, g], toks)
    res = dict(out=out, selected=selected, sel_scores=sel_scores,
               scores=scores, union=union, ws_b=ws_b, n_cand_b=nc_b,
               k_eff_b=ke_b)
    if np.ndim(t) == 0:
        res.update(ws=ws_b[0], n_cand=nc_b[0], k_eff=ke_b[0])
    return res


def decode(q, K, V, omega, summaries, t, k, c, w, n_sink=0, per_head=False):
    """One decode step for every (batch, query head) (Algorithm 1, querying
    procedure): phi(q) -> segment scores over the candidates -> top-k ->
    union over the query heads sharing a kv head -> exact attention over the
    union's tokens plus the window.

    q: [B, Hq, d]; K, V: [B, Hkv, >=t, d]; summaries: [B, Hkv, >=n_cand, n]
    (the oracle's own, from `segment_summaries` with offset=n_sink); t:
    current length (the query's own token is position t-1), one int for the
    whole batch or one per sequence (a ragged batch: each sequence b is
    decoded at its own length t[b]).

    Options outside the paper's single-head description:
      n_sink    tokens [0, n_sink) are attention sinks (always attended,
                never in a segment); see window_split.
      per_head  grouped-query attention where every query head attends its
                own selection plus W instead of its group's union.

    Returns dict with
      out      [B, Hq, d]
      selected [B, Hq, k] int64, -1 padded, ordered as `top_segments`
      sel_scores [B, Hq, k] (nan padded)
      scores   list per (b, h): all candidate scores
      union    list per (b, g): sorted union of the group's selections
      ws_b, n_cand_b, k_eff_b  per sequence; ws, n_cand, k_eff when t is
                one int
    """
    q64 = _f64(q)

    def head_scores(b, g, h, n_cand):
        phi_q = random_features(q64[b, h], omega)
        return decode_head(phi_q, summaries[b, g], n_cand, k)[0]
    return _decode(q64, K, V, t, k, c, w, n_sink, per_head, head_scores)


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


def exact_segment_mass(q, keys, c, n_cand, offset=0):
    """Exact segment attention mass (the quantity Theorem 2's proof calls
    beta): beta_s = sum over the c keys of segment s of exp(q . k / sqrt(d)),
    the unnormalised attention weight the segment carries. Selecting the k
    largest is the exact segment search of the ablation study (Section 3.3).
    Returns ln(beta_s) for s < n_cand (the log keeps large logits finite;
    each segment subtracts its own max logit before exponentiating).
    Segment s covers keys [offset + s*c, offset + s*c + c)."""
    q = _f64(q)
    keys = _f64(keys)
    d = q.shape[-1]
    out = np.empty(n_cand)
    for s in range(n_cand):
        lo = offset + s * c
        lg = keys[lo:lo + c] @ q / np.sqrt(d)
        m = lg.max()
        out[s] = m + np.log(np.exp(lg - m).sum())
    return out


def decode_exact(q, K, V, t, k, c, w, n_sink=0, per_head=False):
    """decode() with the exact segment search in place of the random-feature
    scores: every query head selects the k segments with the largest
    beta_s; the union over the heads sharing a kv head (or, per_head, the
    head's own selection) plus the sinks and the window is attended exactly.
    Returns the same dict as decode() with `scores` and `sel_scores`
    holding ln(beta)."""
    q64 = _f64(q)

    def head_scores(b, g, h, n_cand):
        return exact_segment_mass(q64[b, h], K[b, g], c, n_cand, offset=n_sink)
    return _decode(q64, K, V, t, k, c, w, n_sink, per_head, head_scores)
