"""Pins for the oracle's token sampling: the draft's proposals y ~ q
(Algorithm 1) and mixed sampling y ~ beta p + (1 - beta) q (Section 4.1).

None of these tests restates the oracle's arithmetic.  They check it against
what the mathematics fixes:
  * one row alone reduces to textbook inverse-transform sampling, done here
    with scipy's softmax and numpy's cumsum + searchsorted;
  * V = 2 has a closed form through the logistic function;
  * disjoint supports make the mixture weight directly visible;
  * stratified uniforms u_k = (k + 1/2)/M land in each token's interval
    M * pi_j times, up to one at each end, which fixes the whole mixture;
  * shifting a row by a constant or scaling logits and temperature together
    changes nothing;
  * greedy sampling is numpy's argmax (first maximum).
"""
import numpy as np
import pytest
import scipy.special

from oracle import ref


def rng(seed):
    return np.random.default_rng(seed)


def softmax(x, T):
    return scipy.special.softmax(np.asarray(x, np.float64) / T, axis=-1)


def textbook(pi, u):
    """Inverse-transform sampling: the first j with cumsum(pi)[j] > u * sum(pi)."""
    c = np.cumsum(pi)
    return int(np.searchsorted(c, np.float64(u) * c[-1], side="right"))


@pytest.mark.parametrize("beta", [1.0, 0.0])
@pytest.mark.parametrize("T", [1.0, 0.6, 2.5])
def test_one_row_is_inverse_transform_sampling(beta, T):
    g = rng(int(10 * T) + int(beta))
    N, V = 24, 200
    x = g.normal(0.0, 2.0, (N, V))
    u = g.random(N).astype(np.float32)
    r = ref.sample(x if beta == 1.0 else None, x if beta == 0.0 else None, T, beta, u)
    for n in range(N):
        pi = softmax(x[n], T)
        if r["margin"][n] > 1e-9:  # away from a rounding tie between the two summations
            assert r["tokens"][n] == textbook(pi, u[n]), n
    assert np.all(r["margin"] >= 0.0)


@pytest.mark.parametrize("beta", [0.25, 0.5, 0.9])
def test_mixture_midpoints_reach_every_token(beta):
    """u at the middle of each token's interval draws that token; tokens whose
    logits are -inf in both rows are never drawn."""
    g = rng(int(beta * 100))
    V, T = 8, 0.8
    p = g.normal(0.0, 1.5, V)
    q = g.normal(0.0, 1.5, V)
    p[[2, 5]] = -np.inf
    q[[2, 6]] = -np.inf
    pi = beta * softmax(p, T) + (1.0 - beta) * softmax(q, T)
    c = np.concatenate([[0.0], np.cumsum(pi)])
    for j in range(V):
        if pi[j] == 0.0:
            continue
        u = np.float32((c[j] + c[j + 1]) / 2.0)
        r = ref.sample(p[None], q[None], T, beta, np.array([u]))
        assert r["tokens"][0] == j
    us = (np.arange(4096, dtype=np.float64) + 0.5) / 4096
    r = ref.sample(np.tile(p, (4096, 1)), np.tile(q, (4096, 1)), T, beta, us.astype(np.float32))
    assert 2 not in set(r["tokens"].tolist())


def test_two_token_closed_form():
    """V = 2: token 0 iff u < pi_0 = beta s((p0-p1)/T) + (1-beta) s((q0-q1)/T)."""
    g = rng(7)
    N = 400
    p = g.normal(0.0, 2.0, (N, 2))
    q = g.normal(0.0, 2.0, (N, 2))
    T, beta = 0.7, 0.35
    u = g.random(N).astype(np.float32)
    r = ref.sample(p, q, T, beta, u)
    pi0 = beta * scipy.special.expit((p[:, 0] - p[:, 1]) / T) + \
        (1 - beta) * scipy.special.expit((q[:, 0] - q[:, 1]) / T)
    far = np.abs(u.astype(np.float64) - pi0) > 1e-12
    assert np.array_equal(r["tokens"][far], np.where(u[far] < pi0[far], 0, 1))


@pytest.mark.parametrize("beta", [0.2, 0.5, 0.8])
def test_beta_weights_the_first_row(beta):
    """p puts all mass on token 0, q on token 1: token 0 exactly when u < beta."""
    p = np.array([[0.0, -np.inf, -np.inf]])
    q = np.array([[-np.inf, 0.0, -np.inf]])
    for u in (0.0, beta * 0.5, beta - 1e-6, beta + 1e-6, 0.999):
        r = ref.sample(p, q, 1.0, beta, np.array([u], np.float32))
        assert r["tokens"][0] == (0 if np.float32(u) < beta else 1)


@pytest.mark.parametrize("beta,T", [(0.5, 1.0), (0.3, 0.7), (1.0, 1.3), (0.0, 0.9)])
def test_stratified_counts_match_the_mixture(beta, T):
    g = rng(int(beta * 10 + T * 100))
    V, M = 16, 8192
    p = g.normal(0.0, 1.0, V)
    q = g.normal(0.0, 1.0, V)
    pi = beta * softmax(p, T) + (1.0 - beta) * softmax(q, T)
    u = ((np.arange(M) + 0.5) / M).astype(np.float32)
    r = ref.sample(np.tile(p, (M, 1)) if beta > 0 else None, np.tile(q, (M, 1)) if beta < 1 else None,
                   T, beta, u)
    counts = np.bincount(r["tokens"], minlength=V)
    assert np.all(np.abs(counts - M * pi) <= 1.0 + 1e-9), (counts, M * pi)


def test_shift_and_temperature_invariance():
    g = rng(11)
    N, V = 64, 50
    p = g.normal(0.0, 1.0, (N, V))
    q = g.normal(0.0, 1.0, (N, V))
    u = g.random(N).astype(np.float32)
    a = ref.sample(p, q, 0.5, 0.4, u)
    b = ref.sample(p + g.normal(0, 5, (N, 1)), q - 3.0, 0.5, 0.4, u)
    c = ref.sample(2.0 * p, 2.0 * q, 1.0, 0.4, u)  # exact scaling of logits and temperature
    ok = a["margin"] > 1e-9
    assert np.array_equal(a["tokens"][ok], b["tokens"][ok])
    assert np.array_equal(a["tokens"], c["tokens"])


def test_greedy_is_first_argmax():
    g = rng(3)
    x = np.round(g.normal(0.0, 1.0, (40, 30)), 1)  # many ties
    r = ref.sample(None, x, 0.0, 0.0)
    assert np.array_equal(r["tokens"], np.argmax(x, axis=1))
    assert np.all(np.isnan(r["margin"]))
    r = ref.sample(x, None, 0.0, 1.0)
    assert np.array_equal(r["tokens"], np.argmax(x, axis=1))


def test_invalid_rows_and_arguments():
    x = np.zeros((3, 5))
    x[1] = -np.inf
    u = np.full(3, 0.5, np.float32)
    r = ref.sample(None, x, 1.0, 0.0, u)
    assert r["tokens"].tolist()[1] == -1 and r["tokens"][0] >= 0 and r["tokens"][2] >= 0
    # The row with weight 0 is never read: -inf there is harmless.
    r = ref.sample(np.zeros((3, 5)), x, 1.0, 1.0, u)
    assert (r["tokens"] >= 0).all()
    for bad in [dict(T=-1.0, beta=0.5), dict(T=1.0, beta=1.5), dict(T=0.0, beta=0.5)]:
        with pytest.raises(ValueError):
            ref.sample(x, x, bad["T"], bad["beta"], u)
    with pytest.raises(ValueError):
        ref.sample(None, x, 1.0, 0.5, u)  # p needed when beta > 0


def test_bf16_rows_and_row_strides():
    """bf16 inputs are converted exactly; a strided view of a [B, K, V] tensor
    samples the same rows as a contiguous copy."""
    g = rng(5)
    B, K, V = 6, 3, 40
    t = g.normal(0.0, 2.0, (B, K, V)).astype(np.float32)
    bits = (t.view(np.uint32) >> 16).astype(np.uint16)  # truncation gives exact bf16 values
    exact = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    u = g.random(B).astype(np.float32)
    view = bits[:, 1, :]  # row stride K*V elements
    a = ref.sample(None, view, 0.9, 0.0, u)
    b = ref.sample(None, np.ascontiguousarray(exact[:, 1, :]), 0.9, 0.0, u)
    assert np.array_equal(a["tokens"], b["tokens"])
