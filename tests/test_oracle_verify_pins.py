"""Pins for the oracle's verification (Appendix A.1, Eq. 5; Algorithm 1).

None of these tests restates the oracle's arithmetic.  They check it against
what the paper and the mathematics fix:
  * the paper's exactness claim (the emitted tokens follow the target), by
    exhaustive enumeration over tiny vocabularies with the oracle treated as a
    black box whose decision thresholds are located by bisection over the
    float32 uniforms;
  * special cases that reduce to library routines (inverse-transform sampling
    via numpy's searchsorted, argmax chains);
  * the expected accepted length of Eq. 1, itself pinned to the figures the
    paper prints (tests/golden/eq1_expected_length.txt).
"""
import itertools
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eq1_expected_length.txt")
U_STEPS = 1 << 24  # the uniforms are k * 2^-24


def eq1_expected_length(alpha, k):
    """Eq. 1 of the paper."""
    return (1.0 - alpha ** (k + 1)) / (1.0 - alpha)


def test_eq1_matches_printed_factors():
    rows = [l.split() for l in open(GOLDEN) if l.strip() and not l.startswith("#")]
    n = 0
    for r in rows:
        if len(r) == 5:
            _, _, a1, a2, printed = r
            f = eq1_expected_length(float(a2), 5) / eq1_expected_length(float(a1), 5)
            assert abs(f - float(printed)) <= 0.01 + 1e-9, r
            n += 1
        else:
            _, a, k, printed = r
            assert round(eq1_expected_length(float(a), int(k)), 1) == float(printed), r
            n += 1
    assert n == 10


# --------------------------------------------------------------------------
# Black-box helpers
# --------------------------------------------------------------------------

def _run(target, draft, y, ua, ur, T):
    out = ref.verify(target, draft, y, ua, ur, T)
    return int(out["accepted_len"][0]), out["out_tokens"][0]


def _first_false(pred, lo=0, hi=U_STEPS):
    """Smallest k in [lo, hi) with pred(k) False, given pred monotone
    True...True False...False; returns hi if pred is True throughout."""
    if not pred(lo):
        return lo
    a, b = lo, hi
    while b - a > 1:
        m = (a + b) // 2
        if pred(m):
            a = m
        else:
            b = m
    return b


def _step_masses(f, lo=0, hi=U_STEPS):
    """For a monotone step function f on integers [lo, hi), the mass (count /
    U_STEPS) of each value."""
    out = {}
    while lo < hi:
        v = f(lo)
        end = _first_false(lambda k: f(k) == v, lo, hi)
        out[v] = out.get(v, 0.0) + (end - lo) / U_STEPS
        lo = end
    return out


def _random_table(g, V, zero_frac):
    p = g.gamma(0.7, size=V)
    if V > 1:
        zero = g.random(V) < zero_frac
        if zero.all():
            zero[g.integers(V)] = False
        p[zero] = 0.0
    return p / p.sum()


def _emission_distribution(ptab, qtab, V, k, T):
    """Distribution of the emitted token sequence of one verification step,
    integrated exactly (on the 2^-24 grid) over both kinds of uniform."""
    emitted = {}
    with np.errstate(divide="ignore"):
        for y in itertools.product(range(V), repeat=k):
            py = 1.0
            for i in range(k):
                py *= qtab[tuple(y[:i])][y[i]]
            if py == 0.0:
                continue
            # logits whose temperature softmax is the table row
            target = np.stack([T * np.log(ptab[tuple(y[:i])]) for i in range(k + 1)])[None]
            draft = np.stack([T * np.log(qtab[tuple(y[:i])]) for i in range(k)])[None]
            yy = np.array([y], np.int32)

            # acceptance threshold of each position, earlier positions forced
            # to accept with u = 0
            thresholds = []
            for i in range(k):
                def accepted(kk, i=i):
                    ua = np.zeros((1, k), np.float32)
                    ua[0, i] = kk / U_STEPS
                    a, _ = _run(target, draft, yy, ua, np.zeros(1, np.float32), T)
                    return a > i
                thresholds.append(_first_false(accepted))
            reach = 1.0
            for a in range(k + 1):
                if a < k:
                    p_a = reach * (1.0 - thresholds[a] / U_STEPS)
                else:
                    p_a = reach
                if p_a > 0.0:
                    ua = np.zeros((1, k), np.float32)
                    if a < k:
                        ua[0, a] = thresholds[a] / U_STEPS  # first rejecting u
                    def extra(kk, ua=ua, a=a):
                        acc, toks = _run(target, draft, yy, ua,
                                         np.array([kk / U_STEPS], np.float32), T)
                        assert acc == a
                        return int(toks[a])
                    for c, mass in _step_masses(extra).items():
                        seq = tuple(y[:a]) + (c,)
                        emitted[seq] = emitted.get(seq, 0.0) + py * p_a * mass
                if a < k:
                    reach *= thresholds[a] / U_STEPS
    return emitted


@pytest.mark.parametrize("V,k,T,seed", [(2, 1, 1.0, 0), (3, 2, 1.0, 1), (3, 3, 0.6, 2),
                                        (4, 2, 1.3, 3), (8, 1, 1.0, 4), (5, 2, 1.0, 5)])
def test_enumeration_emits_target_distribution(V, k, T, seed):
    """Exactness (Section 3 and Appendix A.1): the emitted tokens follow the
    target.  For every j <= k+1 and prefix z:
      P(step emits >= j tokens and they start with z)
        = prod_{i<j} min(p_i, q_i)(z_i) * p_j(z_j),
    and hence, given the step emitted >= j tokens starting with z_<j, the j-th
    one is distributed as p_j( . | z_<j)."""
    g = np.random.default_rng(seed)
    ptab = {z: _random_table(g, V, 0.25) for j in range(k + 1)
            for z in itertools.product(range(V), repeat=j)}
    qtab = {z: _random_table(g, V, 0.25) for j in range(k)
            for z in itertools.product(range(V), repeat=j)}
    emitted = _emission_distribution(ptab, qtab, V, k, T)
    assert abs(sum(emitted.values()) - 1.0) < 1e-6
    tol = 2e-6 * (k + 2)
    for j in range(1, k + 2):
        for z in itertools.product(range(V), repeat=j):
            got = sum(m for s, m in emitted.items() if len(s) >= j and s[:j] == z)
            want = 1.0
            for i in range(j - 1):
                want *= min(ptab[z[:i]][z[i]], qtab[z[:i]][z[i]])
            want *= ptab[z[:j - 1]][z[j - 1]]
            assert abs(got - want) < tol, (j, z, got, want)
    # the first emitted token alone follows p_1
    for c in range(V):
        got = sum(m for s, m in emitted.items() if s[0] == c)
        assert abs(got - ptab[()][c]) < tol


def test_identical_rows_accept_everything():
    """p == q gives p(y)/q(y) == 1 > u for every u in [0,1): all k accepted."""
    g = np.random.default_rng(7)
    B, K, V = 6, 5, 50
    t = g.normal(0, 2, (B, K + 1, V)).astype(np.float32)
    d = t[:, :K].copy()
    y = g.integers(0, V, (B, K)).astype(np.int32)
    ua = np.full((B, K), 1.0 - 2.0 ** -24, np.float32)
    ur = g.random(B).astype(np.float32)
    out = ref.verify(t, d, y, ua, ur, 0.9)
    assert (out["accepted_len"] == K).all()
    assert (out["out_tokens"][:, :K] == y).all()
    assert (out["reject_mask"] == 0).all()


def test_bonus_token_is_inverse_transform_sample():
    """With every proposal accepted, the extra token is a draw from p at the
    bonus row (Eq. 5, case a = k): compare with numpy's searchsorted over the
    cumulative sum of scipy's softmax."""
    g = np.random.default_rng(8)
    B, K, V, T = 64, 3, 37, 0.8
    t = g.normal(0, 2, (B, K + 1, V))
    d = t[:, :K].copy()
    y = g.integers(0, V, (B, K)).astype(np.int32)
    ua = np.zeros((B, K), np.float32)
    ur = (g.integers(0, U_STEPS, B) / U_STEPS).astype(np.float32)
    out = ref.verify(t, d, y, ua, ur, T)
    for b in range(B):
        p = scipy.special.softmax(t[b, K] / float(np.float32(T)))
        cdf = np.cumsum(p)
        want = int(np.searchsorted(cdf, float(ur[b]) * cdf[-1], side="right"))
        assert out["accepted_len"][b] == K
        assert out["out_tokens"][b, K] == want
        assert abs(out["margin_cdf"][b] - min(cdf[want] - ur[b] * cdf[-1],
                                              ur[b] * cdf[-1] - (cdf[want - 1] if want else 0))) < 1e-12


def test_zero_target_probability_rejects():
    """A proposal the target gives probability 0 is never accepted; the
    correction token is never a zero-mass token of max(0, p - q)."""
    g = np.random.default_rng(9)
    B, K, V = 32, 2, 20
    t = g.normal(0, 1, (B, K + 1, V))
    d = g.normal(0, 1, (B, K, V))
    y = g.integers(0, V, (B, K)).astype(np.int32)
    for b in range(B):
        t[b, 0, y[b, 0]] = -np.inf
    ua = np.zeros((B, K), np.float32)
    ur = g.random(B).astype(np.float32)
    out = ref.verify(t, d, y, ua, ur, 1.0)
    assert (out["accepted_len"] == 0).all()
    assert (out["reject_mask"][:, 0] == 1).all()
    for b in range(B):
        p = scipy.special.softmax(t[b, 0])
        q = scipy.special.softmax(d[b, 0])
        assert p[out["out_tokens"][b, 0]] > q[out["out_tokens"][b, 0]]


def test_acceptance_threshold_is_probability_ratio():
    """u just below p(y)/q(y) accepts and u just above rejects; the recorded
    margin is |u - p/q|.  V = 2 rows with hand-computable probabilities."""
    # p = (0.2, 0.8), q = (0.4, 0.6): proposal 0 has ratio exactly 0.5
    t = np.log(np.array([[[0.2, 0.8], [0.5, 0.5]]]))
    d = np.log(np.array([[[0.4, 0.6]]]))
    y = np.array([[0]], np.int32)
    for u, acc in [(0.4999999, 1), (0.5000001, 0)]:
        out = ref.verify(t, d, y, np.array([[u]], np.float32), np.array([0.3], np.float32), 1.0)
        assert out["accepted_len"][0] == acc
        assert abs(out["margin_accept"][0, 0] - abs(np.float32(u) - 0.5)) < 1e-12
    # rejected: max(0, p - q) = (0, 0.2), so the correction is token 1 whatever u_res is
    out = ref.verify(t, d, y, np.array([[0.9]], np.float32), np.array([0.0], np.float32), 1.0)
    assert out["out_tokens"][0].tolist() == [1, -1]
    assert abs(out["margin_cdf"][0] - 0.0) < 1e-12  # u_res = 0 sits on the lower edge


def test_residual_margin_is_absolute_mass():
    """After a rejection the residual max(0, p - q) has total Z < 1, and the
    recorded CDF margin is the distance from u*Z to the nearer edge of the
    drawn token's interval in probability mass, not divided by Z.  Hand
    case: p = (0.5, 0.1, 0.4), q = (0.3, 0.5, 0.2), proposal 1 (ratio 0.2)
    rejected; r = (0.2, 0, 0.2), Z = 0.4."""
    t = np.log(np.array([[[0.5, 0.1, 0.4], [1 / 3, 1 / 3, 1 / 3]]]))
    d = np.log(np.array([[[0.3, 0.5, 0.2]]]))
    y = np.array([[1]], np.int32)
    for u, tok, lo, hi in [(0.3, 0, 0.0, 0.2), (0.55, 2, 0.2, 0.4), (0.125, 0, 0.0, 0.2)]:
        uf = float(np.float32(u))
        out = ref.verify(t, d, y, np.array([[0.9]], np.float32), np.array([uf], np.float32), 1.0)
        assert out["accepted_len"][0] == 0 and out["reject_mask"][0, 0] == 1
        assert out["out_tokens"][0].tolist() == [tok, -1]
        c = uf * 0.4
        assert abs(out["margin_cdf"][0] - min(hi - c, c - lo)) < 1e-12, (u, out["margin_cdf"][0])


def test_greedy_is_argmax_chain():
    """T = 0: accept while the proposal equals the target argmax (numpy's
    argmax, which also breaks ties towards the lowest index)."""
    g = np.random.default_rng(10)
    B, K, V = 40, 4, 9
    t = g.integers(-3, 3, (B, K + 1, V)).astype(np.float32)  # many ties
    am = np.argmax(t, axis=-1)
    y = am[:, :K].copy().astype(np.int32)
    flip = g.random((B, K)) < 0.3
    y[flip] = g.integers(0, V, flip.sum())
    out = ref.verify(t, None, y, None, None, 0.0)
    for b in range(B):
        a = next((i for i in range(K) if y[b, i] != am[b, i]), K)
        assert out["accepted_len"][b] == a
        assert out["out_tokens"][b, :a].tolist() == y[b, :a].tolist()
        assert out["out_tokens"][b, a] == am[b, a]
        assert (out["out_tokens"][b, a + 1:] == -1).all()
        assert out["reject_mask"][b].sum() == (1 if a < K else 0)


def test_expected_accepted_length_follows_eq1():
    """Eq. 1 with i.i.d. acceptance: every position scores the same (p, q)
    pair, so each proposal is accepted with alpha = sum_y min(p, q) and
    E[a + 1] = (1 - alpha^(k+1)) / (1 - alpha).  Monte Carlo over 20000
    sequences drawn by the oracle."""
    g = np.random.default_rng(11)
    B, K, V = 20000, 5, 12
    tp = g.normal(0, 1.0, V)
    tq = tp + g.normal(0, 0.8, V)
    p, q = scipy.special.softmax(tp), scipy.special.softmax(tq)
    alpha = np.minimum(p, q).sum()
    t = np.broadcast_to(tp, (B, K + 1, V)).copy()
    d = np.broadcast_to(tq, (B, K, V)).copy()
    y = np.array([g.choice(V, size=K, p=q) for _ in range(B)], np.int32)
    ua = g.random((B, K)).astype(np.float32)
    ur = g.random(B).astype(np.float32)
    out = ref.verify(t, d, y, ua, ur, 1.0)
    a = out["accepted_len"]
    emitted = (a + 1).mean()
    want = eq1_expected_length(alpha, K)
    sd = (a + 1).std() / math.sqrt(B)
    assert abs(emitted - want) < 5 * sd, (emitted, want, sd)
    # P(a >= j) = alpha^j: the step exits at the first rejection
    for j in range(1, K + 1):
        frac = (a >= j).mean()
        assert abs(frac - alpha ** j) < 5 * math.sqrt(alpha ** j * (1 - alpha ** j) / B) + 1e-9


def test_invalid_rows_are_flagged():
    g = np.random.default_rng(12)
    B, K, V = 4, 3, 10
    t = g.normal(0, 1, (B, K + 1, V)).astype(np.float32)
    d = g.normal(0, 1, (B, K, V)).astype(np.float32)
    y = g.integers(0, V, (B, K)).astype(np.int32)
    y[1, 2] = V            # out-of-range token
    dl = np.array([3, 3, 0, 2], np.int32)   # k_b = 0 is invalid
    t[3, 0, :] = -np.inf   # no finite logit in a row that is read
    ua = np.zeros((B, K), np.float32)
    ur = np.zeros(B, np.float32)
    out = ref.verify(t, d, y, ua, ur, 1.0, draft_len=dl)
    assert out["accepted_len"].tolist()[1:] == [-1, -1, -1]
    assert out["accepted_len"][0] >= 0
    assert (out["out_tokens"][1:] == -1).all()


def test_ragged_lengths_use_bonus_row_kb():
    """k_b < K: target row k_b is the bonus row; later rows are padding and
    are never read (NaN there changes nothing)."""
    g = np.random.default_rng(13)
    B, K, V = 5, 4, 16
    t = g.normal(0, 1, (B, K + 1, V))
    d = t[:, :K].copy()
    dl = np.array([1, 2, 3, 4, 2], np.int32)
    for b in range(B):
        t[b, dl[b] + 1:] = np.nan
        d[b, dl[b]:] = np.nan
    y = g.integers(0, V, (B, K)).astype(np.int32)
    ur = g.random(B).astype(np.float32)
    out = ref.verify(t, d, y, np.zeros((B, K), np.float32), ur, 1.0, draft_len=dl)
    assert out["accepted_len"].tolist() == dl.tolist()
    for b in range(B):
        p = scipy.special.softmax(t[b, dl[b]])
        cdf = np.cumsum(p)
        want = int(np.searchsorted(cdf, float(ur[b]) * cdf[-1], side="right"))
        assert out["out_tokens"][b, dl[b]] == want
