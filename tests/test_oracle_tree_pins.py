"""Pins for the oracle's multi-candidate (tree) verification.

The rule (candidates drawn independently from the draft distribution at
their parent, tested in order, each rejection replacing the distribution
the next one is tested against by the normalised residual of Eq. 5) is
pinned by:
  - exactness, by exhaustive enumeration at V <= 4 over every candidate
    assignment with both kinds of uniform integrated exactly on the 2^-24
    grid: given the accepted prefix w, the next emitted token follows the
    target's p(. | w) (the property that makes the paper's verification
    lossless, Section 3 and Appendix A.1);
  - a chain (one child per node) reducing to the pinned single-candidate
    verification, sampling and greedy;
  - a hand-computed two-candidate rejection and residual draw;
  - greedy on a tree, identical rows, invalid trees.
"""
import itertools

import numpy as np
import pytest

from oracle import ref

U_STEPS = 1 << 24


def _first_false(pred, lo=0, hi=U_STEPS):
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
    out = {}
    while lo < hi:
        v = f(lo)
        end = _first_false(lambda k: f(k) == v, lo, hi)
        out[v] = out.get(v, 0.0) + (end - lo) / U_STEPS
        lo = end
    return out


def _table(g, V):
    p = g.gamma(0.7, size=V)
    zero = g.random(V) < 0.25
    if zero.all():
        zero[g.integers(V)] = False
    p[zero] = 0.0
    return p / p.sum()


def _emissions(parent, ptab, qtab, V, T):
    """Distribution of (accepted candidate tokens, extra token) over every
    assignment of candidate tokens (node n ~ q at its parent, independently)
    and both kinds of uniform, integrated exactly."""
    N = len(parent)
    kids = {v: [n for n in range(1, N) if parent[n] == v] for v in range(N)}
    out = {}
    with np.errstate(divide="ignore"):
        for toks in itertools.product(range(V), repeat=N - 1):
            tok = (0,) + toks
            path = {0: ()}
            for n in range(1, N):
                path[n] = path[parent[n]] + (tok[n],)
            w = 1.0
            for n in range(1, N):
                w *= qtab[path[parent[n]]][tok[n]]
            if w == 0.0:
                continue
            target = np.stack([T * np.log(ptab[path[n]]) for n in range(N)])[None]
            draft = np.stack([T * np.log(qtab[path[n]]) for n in range(N)])[None]
            par = np.array([[-1] + list(parent[1:])], np.int32)
            nt = np.array([tok], np.int32)

            def run(ua, ur):
                o = ref.verify_tree(target, draft, par, nt, ua[None], np.array([ur], np.float32), T)
                return o["accepted_len"][0], o["out_tokens"][0], o["path_nodes"][0]

            def walk(v, ua, weight, depth):
                # children of v tested in order; ua holds the choices made so far
                ua = ua.copy()
                for c in kids[v]:
                    def accepted(kk, c=c):
                        u2 = ua.copy()
                        u2[c] = kk / U_STEPS
                        a, _, pn = run(u2, 0.0)
                        return a > depth and pn[depth] == c
                    th = _first_false(accepted)
                    if th > 0:
                        u2 = ua.copy()
                        u2[c] = 0.0
                        walk(c, u2, weight * th / U_STEPS, depth + 1)
                    if th == U_STEPS:
                        return
                    ua[c] = th / U_STEPS  # the first rejecting uniform
                    weight *= 1.0 - th / U_STEPS

                def extra(kk):
                    a, ot, _ = run(ua, kk / U_STEPS)
                    assert a == depth
                    return tuple(int(t) for t in ot[:depth + 1])
                for seq, m in _step_masses(extra).items():
                    out[seq] = out.get(seq, 0.0) + w * weight * m

            walk(0, np.zeros(N, np.float32), 1.0, 0)
    return out


TREES = {
    "two candidates": [-1, 0, 0],
    "three candidates": [-1, 0, 0, 0],
    "two levels": [-1, 0, 0, 1, 2],
    "uneven": [-1, 0, 0, 1, 1, 3],
}


@pytest.mark.parametrize("name,V,T,seed", [("two candidates", 4, 1.0, 0), ("three candidates", 3, 1.0, 1),
                                           ("two levels", 3, 0.7, 2), ("uneven", 2, 1.3, 3),
                                           ("two candidates", 3, 1.0, 4)])
def test_tree_enumeration_emits_target_distribution(name, V, T, seed):
    parent = TREES[name]
    depth = 0
    for n in range(1, len(parent)):
        d, v = 1, parent[n]
        while v != 0:
            d, v = d + 1, parent[v]
        depth = max(depth, d)
    g = np.random.default_rng(seed)
    ptab = {z: _table(g, V) for j in range(depth + 1) for z in itertools.product(range(V), repeat=j)}
    qtab = {z: _table(g, V) for j in range(depth + 1) for z in itertools.product(range(V), repeat=j)}
    em = _emissions(parent, ptab, qtab, V, T)
    assert abs(sum(em.values()) - 1.0) < 1e-6
    tol = 4e-6 * (depth + 2)
    # For every accepted prefix w (j - 1 accepted candidates) the next token
    # follows p(. | w): P(emits >= j tokens starting w z) = A(w) p_w(z), where
    # A(w) = P(the first j - 1 emitted tokens are accepted candidates w).
    for j in range(1, depth + 2):
        for w in itertools.product(range(V), repeat=j - 1):
            A = sum(m for s, m in em.items() if len(s) >= j and s[:j - 1] == w)
            for z in range(V):
                got = sum(m for s, m in em.items() if len(s) >= j and s[:j] == w + (z,))
                assert abs(got - A * ptab[w][z]) < tol, (j, w, z, got, A * ptab[w][z])
    for z in range(V):  # the first token alone follows p at the root
        assert abs(sum(m for s, m in em.items() if s[0] == z) - ptab[()][z]) < tol


def _chain(target, draft, y):
    """The single-candidate step as a chain tree: node n (1..K) proposes
    y[n-1] under its parent n-1; node K is the leaf whose row is the bonus
    row."""
    B, K1, V = target.shape
    K = K1 - 1
    par = np.tile(np.arange(-1, K, dtype=np.int32), (B, 1))
    nt = np.concatenate([np.zeros((B, 1), np.int32), y.astype(np.int32)], axis=1)
    dr = None if draft is None else np.concatenate([draft, draft[:, :1]], axis=1)
    return par, nt, dr


@pytest.mark.parametrize("T", [1.0, 0.6, 0.0])
def test_chain_tree_is_single_candidate_verification(T):
    g = np.random.default_rng(7)
    B, K, V = 64, 4, 50
    t = g.normal(0, 2, (B, K + 1, V))
    d = t[:, :K] + g.normal(0, 1, (B, K, V))
    y = g.integers(0, V, (B, K)).astype(np.int32)
    if T == 0.0:
        y[::2] = np.argmax(t[::2, :K], -1)
    ua = g.random((B, K)).astype(np.float32)
    ur = g.random(B).astype(np.float32)
    want = ref.verify(t, None if T == 0 else d, y, ua, ur, T)
    par, nt, dr = _chain(t, d, y)
    ua_t = np.concatenate([np.zeros((B, 1), np.float32), ua], axis=1)
    got = ref.verify_tree(t, None if T == 0 else dr, par, nt, ua_t, ur, T)
    assert np.array_equal(got["accepted_len"], want["accepted_len"])
    assert np.array_equal(got["out_tokens"], want["out_tokens"])
    acc = want["accepted_len"]
    for b in range(B):
        assert got["path_nodes"][b, :acc[b]].tolist() == list(range(1, acc[b] + 1))
    if T > 0:
        assert np.allclose(got["margin_cdf"], want["margin_cdf"], rtol=0, atol=1e-15)


def test_two_rejected_candidates_draw_from_the_second_residual():
    """p = (0.5, 0.3, 0.2), q = (0.2, 0.2, 0.6), two candidates of token 2.
    First test: 0.2/0.6 = 1/3, rejected at u = 0.5; the residual is
    norm(max(0, p - q)) = (0.75, 0.25, 0).  Second test: 0/0.6 = 0, always
    rejected; residual max(0, (0.75, 0.25, 0) - q) = (0.55, 0.05, 0), total
    0.6, normalised (11/12, 1/12, 0).  u_res = 0.95 lies in token 1's
    interval; the CDF margin is in the units of the unnormalised residual
    (as Eq. 5's single residual): u*Z = 0.57, edges 0.55 and 0.6."""
    t = np.log(np.array([[[0.5, 0.3, 0.2], [1.0, 1.0, 1.0], [1.0, 1.0, 1.0]]]))
    d = np.log(np.array([[[0.2, 0.2, 0.6], [1.0, 1.0, 1.0], [1.0, 1.0, 1.0]]]))
    par = np.array([[-1, 0, 0]], np.int32)
    nt = np.array([[0, 2, 2]], np.int32)
    for ur, tok in [(0.95, 1), (0.5, 0)]:
        o = ref.verify_tree(t, d, par, nt, np.array([[0.0, 0.5, 0.0]], np.float32), np.array([ur], np.float32), 1.0)
        assert o["accepted_len"][0] == 0 and o["out_tokens"][0].tolist() == [tok, -1, -1]
        assert abs(o["margin_accept"][0, 1] - abs(0.5 - 1 / 3)) < 1e-12
        assert abs(o["margin_accept"][0, 2] - 0.0) < 1e-12  # u = 0, ratio = 0
        c = float(np.float32(ur)) * 0.6
        want = min(0.6 - c, c - 0.55) if tok == 1 else min(0.55 - c, c)
        assert abs(o["margin_cdf"][0] - want) < 1e-12
    # the first candidate accepted (u below 1/3): the walk moves to node 1, a
    # leaf, whose uniform row gives the bonus token
    o = ref.verify_tree(t, d, par, nt, np.array([[0.0, 0.3, 0.0]], np.float32), np.array([0.7], np.float32), 1.0)
    assert o["accepted_len"][0] == 1 and o["path_nodes"][0].tolist() == [1, -1, -1]
    assert o["out_tokens"][0].tolist() == [2, 2, -1]


def test_identical_rows_accept_the_first_candidate():
    g = np.random.default_rng(9)
    B, V = 16, 30
    par = np.array([-1, 0, 0, 0, 1, 1, 4], np.int32)
    N = len(par)
    t = g.normal(0, 2, (B, N, V))
    nt = g.integers(0, V, (B, N)).astype(np.int32)
    o = ref.verify_tree(t, t.copy(), np.tile(par, (B, 1)), nt, g.random((B, N)).astype(np.float32),
                        g.random(B).astype(np.float32), 0.9)
    # ratio = 1 > u for the first child at every level: path 1, 4, 6
    assert (o["accepted_len"] == 3).all()
    assert (o["path_nodes"][:, :3] == [1, 4, 6]).all()
    assert (o["out_tokens"][:, :3] == nt[:, [1, 4, 6]]).all()


def test_greedy_tree_follows_the_argmax():
    """T = 0: at each node the first child whose token is the target argmax
    is accepted; the argmax is emitted where no child matches."""
    g = np.random.default_rng(10)
    B, V = 32, 20
    par = np.array([-1, 0, 0, 0, 2, 2, 3], np.int32)
    N = len(par)
    t = g.normal(0, 1, (B, N, V))
    am = np.argmax(t, -1)
    nt = g.integers(0, V, (B, N)).astype(np.int32)
    nt[: B // 2, 2] = am[: B // 2, 0]
    nt[: B // 2, 3] = am[: B // 2, 0]      # a later duplicate is not taken
    nt[: B // 4, 5] = am[: B // 4, 2]
    o = ref.verify_tree(t, None, np.tile(par, (B, 1)), nt, None, None, 0.0)
    for b in range(B):
        v, path = 0, []
        while True:
            kids = [n for n in range(N) if n > 0 and par[n] == v and nt[b, n] == am[b, v]]
            if not kids:
                break
            v = kids[0]
            path.append(v)
        assert o["accepted_len"][b] == len(path)
        assert o["path_nodes"][b, :len(path)].tolist() == path
        assert o["out_tokens"][b, len(path)] == am[b, v]


def test_invalid_trees_and_rows():
    g = np.random.default_rng(11)
    B, V = 5, 12
    par = np.tile(np.array([-1, 0, 0, 1], np.int32), (B, 1))
    N = 4
    t = g.normal(0, 1, (B, N, V))
    d = g.normal(0, 1, (B, N, V))
    nt = g.integers(0, V, (B, N)).astype(np.int32)
    par[0, 3] = 3            # not an earlier node
    nt[1, 2] = V             # token outside the vocabulary
    t[2, 0] = -np.inf        # the root row has no finite logit
    par[3, 1] = -2           # negative parent
    o = ref.verify_tree(t, d, par, nt, np.full((B, N), 0.999, np.float32), g.random(B).astype(np.float32), 1.0)
    assert o["accepted_len"][:4].tolist() == [-1, -1, -1, -1]
    assert (o["out_tokens"][:4] == -1).all() and (o["path_nodes"][:4] == -1).all()
    assert o["accepted_len"][4] >= 0
