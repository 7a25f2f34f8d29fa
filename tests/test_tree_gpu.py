"""Parity of multi-candidate (tree) verification (osd_verify_tree) with the
fp64 oracle (ref.verify_tree).

The bar is osd_verify's: accepted lengths, emitted tokens and accepted nodes
bit-exact, except for sequences where a decision the oracle evaluated (every
candidate test along its walk, and the final draw's CDF margin in absolute
mass) lies within 1e-6 of its boundary, or whose residual ran out of mass;
those are counted and printed.
"""
import numpy as np
import pytest

from oracle import ref
from paper_2310_07177_amd import synth
from tests._helpers import MARGIN, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def osd():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2310_07177_amd as m
    m.lib()
    return m


def run_tree(osd, x):
    import torch
    T = x["T"]
    out = osd.osd_verify_tree(to_device(x["target"]), None if T == 0 else to_device(x["draft"]),
                              to_device(x["parent"]), to_device(x["tokens"]),
                              None if T == 0 else to_device(x["u_accept"]),
                              None if T == 0 else to_device(x["u_resample"]), T)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in out]


def tree_at_risk(r):
    with np.errstate(invalid="ignore"):
        acc = (np.nan_to_num(r["margin_accept"], nan=np.inf) < MARGIN).any(axis=1)
    return acc | (np.nan_to_num(r["margin_cdf"], nan=np.inf) < MARGIN) | (r["z_fallback"] != 0)


def check_tree(osd, x, label, max_excluded_frac=0.1):
    acc, toks, nodes = run_tree(osd, x)
    T = x["T"]
    r = ref.verify_tree(x["target"], None if T == 0 else x["draft"], x["parent"], x["tokens"],
                        None if T == 0 else x["u_accept"], None if T == 0 else x["u_resample"], T)
    risky = tree_at_risk(r)
    bad = [b for b in np.nonzero(~risky)[0]
           if acc[b] != r["accepted_len"][b] or not np.array_equal(toks[b], r["out_tokens"][b])
           or not np.array_equal(nodes[b], r["path_nodes"][b])]
    assert not bad, (f"{label}: {len(bad)} sequences differ, first b={bad[0]}: gpu a={acc[bad[0]]} "
                     f"toks={toks[bad[0]].tolist()} nodes={nodes[bad[0]].tolist()} | oracle "
                     f"a={r['accepted_len'][bad[0]]} toks={r['out_tokens'][bad[0]].tolist()} "
                     f"nodes={r['path_nodes'][bad[0]].tolist()}")
    print(f"[{label}] compared {int((~risky).sum())} sequences, excluded {int(risky.sum())} (margin < 1e-6); "
          f"mean accepted {acc[acc >= 0].mean() if (acc >= 0).any() else 0:.3f}", flush=True)
    assert risky.sum() <= max(1, max_excluded_frac * len(acc))
    return r, acc


def test_tree_medusa_shape_full_batch(osd):
    """B=16 sequences, a 64-node tree (branching 4, 3, 2, 1), V = 32000 bf16."""
    for seed in range(2):
        check_tree(osd, synth.config_medusa_tree(seed), f"medusa tree seed={seed}")


@pytest.mark.parametrize("V,dtype", [(5, "bf16"), (1001, "bf16"), (4096, "bf16"), (8000, "bf16"), (16384, "bf16"),
                                     (24000, "bf16"), (32768, "bf16"), (4100, "f32"), (16384, "f32")])
def test_tree_random_shapes_and_vocabularies(osd, V, dtype):
    """Random trees (node n's parent uniform over 0..n-1) of up to 40 nodes,
    every tile of both layouts (unaligned rows take one workgroup per node;
    V = 8000 and 24000 bf16 end in a partial round of the streaming
    layout's 1024x1 and 1024x3 tiles)."""
    g = synth.rng(V)
    for k, N in enumerate((2, 9, 40)):
        par = np.stack([synth.random_tree_parents(g, N) for _ in range(6)])
        x = synth.tree_inputs(6, par, V, dtype, T=0.8, seed=V + k, target_std=2.0, draft_noise=0.7)
        check_tree(osd, x, f"random tree N={N} V={V} {dtype}")


@pytest.mark.parametrize("T", [0.6, 1.5])
def test_tree_temperatures_and_wide_nodes(osd, T):
    """A root with 20 candidates (many recursive rejections) and a second
    level of 6."""
    par = synth.tree_parents((20, 1, 6), max_nodes=64)
    x = synth.tree_inputs(12, par, 8192, "bf16", T=T, seed=int(T * 10), target_std=2.5, draft_noise=2.0)
    check_tree(osd, x, f"wide tree T={T}")


def test_tree_greedy(osd):
    x = synth.tree_inputs(16, synth.tree_parents((4, 3, 2, 1)), 32000, "bf16", T=0.0, seed=3, target_std=2.0,
                          draft_noise=0.3)
    r, acc = check_tree(osd, x, "greedy tree", max_excluded_frac=0.0)
    assert (acc > 0).any()


def test_tree_chain_equals_osd_verify(osd):
    """One child per node: the tree is the single-candidate step, and the
    outputs equal osd_verify's on the same rows."""
    import torch
    x = synth.verify_inputs(32, 6, 8192, "bf16", T=0.9, seed=9, draft_noise=0.6)
    B, K = 32, 6
    par = np.tile(np.arange(-1, K, dtype=np.int32), (B, 1))
    tree = dict(target=x["target"], draft=np.concatenate([x["draft"], x["draft"][:, :1]], axis=1), parent=par,
                tokens=np.concatenate([np.zeros((B, 1), np.int32), x["tokens"].astype(np.int32)], axis=1),
                u_accept=np.concatenate([np.zeros((B, 1), np.float32), x["u_accept"]], axis=1),
                u_resample=x["u_resample"], T=x["T"])
    _, acc = check_tree(osd, tree, "chain tree")
    ta, tt, tn = run_tree(osd, tree)
    va, vt, vm = osd.osd_verify(to_device(x["target"]), to_device(x["draft"]),
                                to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]),
                                to_device(x["u_resample"]), x["T"])
    torch.cuda.synchronize()
    assert np.array_equal(ta, va.cpu().numpy())
    assert np.array_equal(tt[:, :K + 1], vt.cpu().numpy())


def test_tree_identical_rows_and_invalid_trees(osd):
    import torch
    g = synth.rng(5)
    B, V = 10, 3000
    par = np.tile(synth.tree_parents((3, 2)), (B, 1))
    N = par.shape[1]
    x = synth.tree_inputs(B, par, V, "bf16", T=1.0, seed=17)
    x["draft"] = x["target"].copy()      # identical rows: the first child is always accepted
    x["parent"] = x["parent"].copy()
    x["parent"][0, 5] = 7                 # not an earlier node
    x["tokens"][1, 2] = V                 # token outside the vocabulary
    x["parent"][2, 1] = -1                # a second root
    x["target"][3, 0, :] = 0xFF80         # the root row has no finite logit
    acc, toks, nodes = run_tree(osd, x)
    assert acc[:4].tolist() == [-1] * 4 and (toks[:4] == -1).all() and (nodes[:4] == -1).all()
    first = [n for n in range(1, N) if par[0, n] == 0][0]
    second = [n for n in range(1, N) if par[0, n] == first][0]
    assert (acc[4:] == 2).all() and (nodes[4:, :2] == [first, second]).all()
    check_tree(osd, {k: (v[4:] if isinstance(v, np.ndarray) and v.shape[:1] == (B,) else v) for k, v in x.items()},
               "identical rows")


def test_tree_all_candidates_rejected(osd):
    """Every candidate at the root has target probability 0: all are
    rejected, and the token comes from the last residual, whose mass lies
    only where p > 0 (never on a candidate)."""
    B, V = 16, 2048
    par = synth.tree_parents((5, 1))
    x = synth.tree_inputs(B, par, V, "bf16", T=1.0, seed=23, draft_noise=1.5)
    roots = [n for n in range(1, len(par)) if par[n] == 0]
    for b in range(B):
        for c in roots:
            x["target"][b, 0, x["tokens"][b, c]] = 0xFF80
    r, acc = check_tree(osd, x, "all rejected at the root")
    assert (acc == 0).all()
    toks = run_tree(osd, x)[1]
    for b in range(B):
        assert toks[b, 0] not in [x["tokens"][b, c] for c in roots]


def test_tree_workspace_reuse_and_determinism(osd):
    import torch
    from paper_2310_07177_amd import binding
    for seed, (B, N) in enumerate([(8, 64), (3, 5), (8, 64), (40, 17)]):
        g = synth.rng(100 + seed)
        par = np.stack([synth.random_tree_parents(g, N) for _ in range(B)])
        x = synth.tree_inputs(B, par, 4000, "bf16", T=1.0, seed=30 + seed, draft_noise=0.8)
        a = run_tree(osd, x)
        b = run_tree(osd, x)
        for u, v in zip(a, b):
            assert np.array_equal(u, v)
        check_tree(osd, x, f"reuse B={B} N={N}")
    torch.cuda.synchronize()
    for key, ws in binding._workspaces.items():
        if key[2] == "verify_tree":
            assert int(ws.count_nonzero()) == 0
