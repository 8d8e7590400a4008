"""Statistical checks of the method itself on the fp64 oracle (opt-in:
`pytest -m slow`). They pin the random-feature scores to the paper's
probability bounds, which no exact formula can:

  * Lemma 9 (Appendix B, the scaled form of Lemma 8): two segments u and v
    with beta_u <= beta_v are mis-ordered by their Radar scores with
    probability at most 2 exp(-(sqrt(n) (a'_v - a'_u) / (sqrt(2)
    exp(zeta^2 / sqrt(d))))^2), a'_x = beta_x / (beta_u + beta_v).
  * Theorem 2 (Section 2.3, proof in Appendix C) in the form its proof
    derives: with c segments, a_i = beta_i / sum_j beta_j and gap
    eps = a_1 - max_{i > 1} a_i, the top segment is missed with probability
    at most 2 (c - 1) exp(-n eps^2 / (8 a_1^2 exp(2 zeta^2 / sqrt(d)))).
  * Convergence (Section 3.3's n study; Theorem 2): on planted inputs with
    gaps between the segment masses, Radar's top-k converges to the exact
    segment search's top-k as n grows from 2^8 to 2^16.

The bounds are one-sided (the observed rates are far below them). Each
check draws Omega many times and compares the observed rate with the bound
plus three binomial standard errors."""
import numpy as np
import pytest

from oracle import radar_oracle as orc

pytestmark = pytest.mark.slow


def _radar_scores(z, segs, omega, c):
    """Eq. 6 scores of the segments `segs` [S*c, d] for query z."""
    summ = orc.segment_summaries(segs, omega, c)
    return orc.segment_scores(orc.random_features(z, omega), summ)


def _beta(z, keys, c):
    return np.exp(orc.exact_segment_mass(z, keys, c, len(keys) // c))


def _segment(rng, d, c, proj, e):
    """c keys of norm <= 1 whose projection on the unit vector e is about
    `proj`: proj * e plus a small orthogonal part."""
    x = rng.standard_normal((c, d)) * 0.15
    x -= np.outer(x @ e, e)
    x += np.outer(proj + rng.standard_normal(c) * 0.02, e)
    nrm = np.linalg.norm(x, axis=1, keepdims=True)
    return x / np.maximum(nrm, 1.0)


@pytest.mark.parametrize("proj_u,proj_v", [(0.2, 0.6), (0.1, 0.7), (-0.2, 0.5)])
def test_lemma9_pairwise_misorder_rate(proj_u, proj_v):
    rng = np.random.default_rng(int(100 * (proj_u + 2) + 10 * proj_v))
    d, c, M = 4, 8, 3000
    e = np.zeros(d); e[0] = 1.0
    z = e.copy()                                    # |z| = 1
    u = _segment(rng, d, c, proj_u, e)
    v = _segment(rng, d, c, proj_v, e)
    bu, bv = _beta(z, u, c)[0], _beta(z, v, c)[0]
    assert bu < bv
    zeta = max(np.linalg.norm(np.vstack([u, v, z[None]]), axis=1))
    assert zeta <= 1.0 + 1e-12
    gap = (bv - bu) / (bu + bv)                     # a'_v - a'_u
    rates = {}
    for n in (256, 1024, 2048):
        bound = 2 * np.exp(-(np.sqrt(n) * gap / (np.sqrt(2) * np.exp(zeta ** 2 / np.sqrt(d)))) ** 2)
        bad = 0
        for _ in range(M):
            om = rng.standard_normal((n, d))
            s = _radar_scores(z, np.vstack([u, v]), om, c)
            bad += s[0] >= s[1]
        rate = bad / M
        rates[n] = rate
        if bound < 1:
            slack = 3 * np.sqrt(bound * (1 - bound) / M) + 1 / M
            assert rate <= bound + slack, (n, rate, bound)
    # more features, fewer mis-orders
    assert rates[2048] <= rates[256]


def test_theorem2_top_segment_found():
    rng = np.random.default_rng(7)
    d, c, M = 4, 4, 2000
    e = np.zeros(d); e[0] = 1.0
    z = e.copy()
    projs = [0.9, 0.35, 0.3, 0.2]                   # segment 0 leads
    keys = np.vstack([_segment(rng, d, c, p, e) for p in projs])
    beta = _beta(z, keys, c)
    a = beta / beta.sum()
    assert np.argmax(a) == 0
    eps = a[0] - a[1:].max()
    zeta = max(np.linalg.norm(np.vstack([keys, z[None]]), axis=1))
    checked = 0
    for n in (512, 1024, 2048):
        delta = 2 * (c - 1) * np.exp(-n * eps ** 2 / (8 * a[0] ** 2 * np.exp(2 * zeta ** 2 / np.sqrt(d))))
        miss = 0
        for _ in range(M):
            om = rng.standard_normal((n, d))
            miss += int(np.argmax(_radar_scores(z, keys, om, c)) != 0)
        rate = miss / M
        if delta < 1:
            checked += 1
            slack = 3 * np.sqrt(delta * (1 - delta) / M) + 1 / M
            assert rate <= delta + slack, (n, rate, delta)
    assert checked >= 2


def test_topk_converges_to_exact_segment_search():
    rng = np.random.default_rng(1)
    d, c, S, k, draws = 16, 16, 32, 4, 16
    e = np.zeros(d); e[0] = 1.0
    q = 2.0 * e
    keys = rng.standard_normal((S * c, d)) * 0.35
    keys[:, 0] = rng.uniform(-1.0, 0.4, S * c)
    planted = rng.choice(S, 8, replace=False)
    for j, s in enumerate(planted):                 # graded masses, ~3% apart
        keys[s * c:(s + 1) * c, 0] = 1.5 - 0.1 * j + rng.standard_normal(c) * 0.05
    lnb = orc.exact_segment_mass(q, keys, c, S)
    exact = orc.top_segments(lnb, k).tolist()
    recall, same = {}, {}
    for p in (8, 10, 12, 14, 16):
        n = 1 << p
        r, eq = [], 0
        for _ in range(draws):
            om = rng.standard_normal((n, d))
            sel = orc.top_segments(_radar_scores(q, keys, om, c), k).tolist()
            r.append(len(set(sel) & set(exact)) / k)
            eq += sel == exact
        recall[p], same[p] = float(np.mean(r)), eq
    # the small-n selections miss some of the exact top-k ...
    assert recall[8] < 1.0
    # ... and the recall does not fall as n grows, reaching the exact
    # selection, in order, for every draw at n = 2^16
    ps = sorted(recall)
    for a, b in zip(ps, ps[1:]):
        assert recall[b] >= recall[a] - 1.0 / (k * draws), recall
    assert recall[16] == 1.0 and same[16] == draws, (recall, same)
