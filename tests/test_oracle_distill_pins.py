"""Pins for the oracle's distillation divergences and gradients (Section 4.1,
Eq. 2-4).

The values are checked against scipy's library routines (relative entropy,
Jensen-Shannon distance), closed forms (Bernoulli KL, the JSD of disjoint
supports), invariants (D(p, p) = 0, shift invariance, gradients summing to
zero) and central finite differences of the oracle's own loss, which tie its
closed-form gradients to its divergence values.
"""
import math

import numpy as np
import pytest
import scipy.spatial.distance
import scipy.special
import scipy.stats

from oracle import ref

KINDS = ("fkl", "rkl", "jsd")


def _rows(seed, B, K, V, scale=2.0, noise=1.0):
    g = np.random.default_rng(seed)
    t = g.normal(0, scale, (B, K, V))
    s = t + g.normal(0, noise, (B, K, V))
    return t, s


@pytest.mark.parametrize("kind", KINDS)
def test_divergence_of_identical_rows_is_zero(kind):
    t, _ = _rows(0, 3, 2, 64)
    out = ref.distill(t, t.copy(), kind, beta=0.3, tau=0.9)
    assert np.all(np.abs(out["row_loss"]) <= 1e-15)
    assert np.all(np.abs(out["grad"]) <= 1e-15)


@pytest.mark.parametrize("tau", [1.0, 0.7, 2.5])
def test_forward_and_reverse_kl_match_scipy(tau):
    t, s = _rows(1, 2, 3, 100)
    f = ref.distill(t, s, "fkl", tau=tau)
    r = ref.distill(t, s, "rkl", tau=tau)
    for b in range(2):
        for i in range(3):
            p = scipy.special.softmax(t[b, i] / tau)
            q = scipy.special.softmax(s[b, i] / tau)
            assert math.isclose(f["row_loss"][b, i], scipy.stats.entropy(p, q), rel_tol=1e-11)
            assert math.isclose(r["row_loss"][b, i], scipy.stats.entropy(q, p), rel_tol=1e-11)


def test_jsd_half_matches_scipy_jensenshannon():
    """At beta = 1/2, JSD is the square of scipy's Jensen-Shannon distance
    (natural log)."""
    t, s = _rows(2, 2, 2, 80)
    out = ref.distill(t, s, "jsd", beta=0.5, tau=1.0)
    for b in range(2):
        for i in range(2):
            p = scipy.special.softmax(t[b, i])
            q = scipy.special.softmax(s[b, i])
            js = scipy.spatial.distance.jensenshannon(p, q) ** 2
            assert math.isclose(out["row_loss"][b, i], js, rel_tol=1e-9)


@pytest.mark.parametrize("beta", [0.1, 0.5, 0.9])
def test_jsd_general_beta_matches_scipy_entropy(beta):
    """Eq. 3 with m = beta p + (1-beta) q, via scipy's relative entropy."""
    t, s = _rows(3, 1, 3, 50)
    out = ref.distill(t, s, "jsd", beta=beta, tau=1.2)
    for i in range(3):
        p = scipy.special.softmax(t[0, i] / 1.2)
        q = scipy.special.softmax(s[0, i] / 1.2)
        m = beta * p + (1 - beta) * q
        want = beta * scipy.stats.entropy(p, m) + (1 - beta) * scipy.stats.entropy(q, m)
        assert math.isclose(out["row_loss"][0, i], want, rel_tol=1e-10)


@pytest.mark.parametrize("beta", [0.5, 0.2, 0.85])
def test_jsd_bounds_and_disjoint_supports(beta):
    """0 <= JSD_beta <= H(beta) = -beta ln beta - (1-beta) ln(1-beta), with
    equality exactly when p and q have disjoint supports (ln 2 at beta = 1/2)."""
    hb = -beta * math.log(beta) - (1 - beta) * math.log(1 - beta)
    t, s = _rows(4, 4, 4, 30, scale=4.0, noise=4.0)
    out = ref.distill(t, s, "jsd", beta=beta)
    assert np.all(out["row_loss"] >= 0) and np.all(out["row_loss"] <= hb)
    V = 10
    td = np.full((1, 1, V), -np.inf)
    sd = np.full((1, 1, V), -np.inf)
    td[0, 0, :4] = np.arange(4)
    sd[0, 0, 4:] = np.arange(6) * 0.5
    out = ref.distill(td, sd, "jsd", beta=beta)
    assert math.isclose(out["row_loss"][0, 0], hb, rel_tol=1e-13)


@pytest.mark.parametrize("beta", [0.0, 1.0])
def test_jsd_is_identically_zero_at_the_endpoints(beta):
    """Eq. 3 at beta = 1 is KL(p || p) (+ 0 x KL(q || p)), at beta = 0 it is
    0 x KL(p || q) + KL(q || q): zero, with a zero gradient, whatever p and
    q are -- also for disjoint supports, where the weight-0 KL is infinite
    and must be left out rather than multiplied by 0."""
    t, s = _rows(11, 2, 3, 40, scale=3.0, noise=2.0)
    out = ref.distill(t, s, "jsd", beta=beta, tau=0.8)
    assert np.all(np.isfinite(out["row_loss"])) and np.all(np.abs(out["row_loss"]) <= 1e-14)
    assert np.all(np.isfinite(out["grad"])) and np.all(np.abs(out["grad"]) <= 1e-14)
    V = 6
    td = np.full((1, 2, V), -np.inf)
    sd = np.full((1, 2, V), -np.inf)
    td[0, :, :3] = [0.0, 1.0, 2.0]
    sd[0, :, 2:] = [0.5, -1.0, 0.0, 3.0]      # overlapping support (token 2)
    sd[0, 1, 2] = -np.inf                     # row 1: disjoint supports
    out = ref.distill(td, sd, "jsd", beta=beta)
    assert np.all(np.isfinite(out["row_loss"])) and np.all(np.abs(out["row_loss"]) <= 1e-14)
    assert np.all(np.isfinite(out["grad"])) and np.all(np.abs(out["grad"]) <= 1e-14)
    assert out["loss_sum"] == 0.0 or abs(out["loss_sum"]) <= 1e-14
    # just inside the endpoints the divergence is small and positive, bounded
    # by H(beta') (disjoint supports reach the bound)
    bp = 1e-6 if beta == 0.0 else 1 - 1e-6
    hb = -bp * math.log(bp) - (1 - bp) * math.log(1 - bp)
    near = ref.distill(td, sd, "jsd", beta=bp)["row_loss"][0]
    assert 0 < near[0] < hb and math.isclose(near[1], hb, rel_tol=1e-9)


@pytest.mark.parametrize("tau", [1.0, 0.5])
def test_bernoulli_closed_forms(tau):
    """V = 2: the softmax is a logistic sigmoid and KL is the textbook
    Bernoulli divergence."""
    t = np.array([[[0.3, 1.7]]])
    s = np.array([[[-0.4, 0.2]]])
    a = 1 / (1 + math.exp(-(t[0, 0, 1] - t[0, 0, 0]) / tau))   # p(token 1)
    c = 1 / (1 + math.exp(-(s[0, 0, 1] - s[0, 0, 0]) / tau))   # q(token 1)
    kl = lambda x, y: x * math.log(x / y) + (1 - x) * math.log((1 - x) / (1 - y))
    f = ref.distill(t, s, "fkl", tau=tau)["row_loss"][0, 0]
    r = ref.distill(t, s, "rkl", tau=tau)["row_loss"][0, 0]
    assert math.isclose(f, kl(a, c), rel_tol=1e-12)
    assert math.isclose(r, kl(c, a), rel_tol=1e-12)


def test_forward_kl_gradient_is_softmax_difference():
    """At tau = 1 the forward-KL gradient is softmax(draft) - softmax(target)."""
    t, s = _rows(5, 2, 2, 40)
    g = ref.distill(t, s, "fkl", tau=1.0)["grad"]
    want = scipy.special.softmax(s, axis=-1) - scipy.special.softmax(t, axis=-1)
    assert np.max(np.abs(g - want)) < 1e-15


@pytest.mark.parametrize("kind,beta,tau", [("fkl", 0.5, 1.0), ("fkl", 0.5, 0.6),
                                           ("rkl", 0.5, 1.0), ("rkl", 0.5, 1.7),
                                           ("jsd", 0.5, 1.0), ("jsd", 0.2, 0.8),
                                           ("jsd", 0.9, 1.3)])
def test_gradients_match_central_finite_differences(kind, beta, tau):
    """d(sum_n mask_n D_n)/d s by central differences of the oracle's own loss,
    V <= 16, fp64 inputs."""
    B, K, V = 2, 2, 13
    t, s = _rows(6, B, K, V, scale=1.5, noise=1.0)
    mask = np.array([[1, 0], [1, 1]], np.uint8)
    g = ref.distill(t, s, kind, beta=beta, tau=tau, mask=mask)["grad"]
    h = 1e-6
    fd = np.zeros_like(s)
    for idx in np.ndindex(s.shape):
        sp = s.copy(); sp[idx] += h
        sm = s.copy(); sm[idx] -= h
        lp = ref.distill(t, sp, kind, beta=beta, tau=tau, mask=mask, grad=False)["loss_sum"]
        lm = ref.distill(t, sm, kind, beta=beta, tau=tau, mask=mask, grad=False)["loss_sum"]
        fd[idx] = (lp - lm) / (2 * h)
    assert np.max(np.abs(g - fd)) < 5e-9, np.max(np.abs(g - fd))
    assert np.all(g[0, 1] == 0.0)          # masked row has zero gradient


@pytest.mark.parametrize("kind", KINDS)
def test_gradient_sums_to_zero_and_shift_invariance(kind):
    """Adding a constant to a row leaves softmax unchanged, so the loss is
    invariant and the gradient sums to zero along the vocabulary."""
    t, s = _rows(7, 2, 3, 64)
    a = ref.distill(t, s, kind, beta=0.4, tau=0.9)
    b = ref.distill(t + 3.0, s - 5.0, kind, beta=0.4, tau=0.9)
    assert np.max(np.abs(a["grad"].sum(-1))) < 1e-15
    assert np.allclose(a["row_loss"], b["row_loss"], rtol=1e-10, atol=1e-13)
    assert np.allclose(a["grad"], b["grad"], rtol=1e-9, atol=1e-15)


def test_masked_mean_and_sum_hand_example():
    """Three rows: disjoint supports (JSD_1/2 = ln 2), the same masked out, and
    identical rows (JSD = 0): sum = ln 2, count = 2, mean = ln 2 / 2."""
    V = 6
    t = np.full((1, 3, V), -np.inf)
    s = np.full((1, 3, V), -np.inf)
    t[0, 0, :3] = 0.0; s[0, 0, 3:] = 0.0
    t[0, 1, :3] = 0.0; s[0, 1, 3:] = 0.0
    t[0, 2] = np.arange(V); s[0, 2] = np.arange(V)
    out = ref.distill(t, s, "jsd", beta=0.5, mask=np.array([[1, 0, 1]], np.uint8))
    assert math.isclose(out["loss_sum"], math.log(2), rel_tol=1e-14)
    assert math.isclose(out["loss_mean"], math.log(2) / 2, rel_tol=1e-14)
    assert out["row_loss"][0, 1] == 0.0
    empty = ref.distill(t, s, "jsd", mask=np.zeros((1, 3), np.uint8))
    assert empty["loss_mean"] == 0.0 and empty["loss_sum"] == 0.0
    assert np.all(empty["grad"] == 0.0)


def test_teacher_batch_stride_reads_first_k_target_rows():
    """Distilling against a [B, K+1, V] target with batch stride (K+1)V uses
    its first K rows."""
    g = np.random.default_rng(8)
    B, K, V = 3, 2, 20
    target = g.normal(0, 1, (B, K + 1, V))
    s = g.normal(0, 1, (B, K, V))
    a = ref.distill(target, s, "rkl", teacher_batch_stride=(K + 1) * V,
                    student_batch_stride=K * V, B=B, K=K)
    b = ref.distill(target[:, :K].copy(), s, "rkl")
    assert np.array_equal(a["row_loss"], b["row_loss"])
    assert np.array_equal(a["grad"], b["grad"])


def test_round_bf16_is_single_rne_rounding():
    """fp64 -> bf16 agrees with torch's float32 -> bfloat16 conversion (RNE)
    wherever the value is exact in float32, and avoids the double rounding of
    going through float32 on a hand-made case."""
    import torch
    g = np.random.default_rng(9)
    x = g.normal(0, 3, 4000).astype(np.float32).astype(np.float64)
    x = np.concatenate([x, [0.0, -0.0, 1e-40, 3e38, -3.3e38, 1.0, 1.00390625]])
    want = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ref.round_bf16(x), want)
    # 1 + 2^-8 is a bf16 tie (rounds to even: 1.0); 1 + 2^-8 + 2^-30 is not a
    # tie in fp64 and must round up, although float32 would turn it into the tie
    y = np.array([1 + 2.0 ** -8, 1 + 2.0 ** -8 + 2.0 ** -30])
    r = ref.round_bf16(y)
    assert r[0] == 0x3F80 and r[1] == 0x3F81
    flags = ref.bf16_midpoint_flags(y)
    assert flags.tolist() == [True, True]
    assert ref.bf16_midpoint_flags(np.array([1.25]))[0] == False
