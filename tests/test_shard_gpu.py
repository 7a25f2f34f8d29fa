"""Parity of the vocabulary-sharded verification (osd_shard_verify_stats,
osd_shard_verify_mass, osd_shard_verify_draw) with the fp64 oracle.

G ranks are played on one GPU: rank g's slice is a contiguous copy of columns
[v_g, v_{g+1}) of the workload's logits; the all-gathers of the phase
records are a torch.stack in rank order and the closing all-reduce MAX of
out_tokens is an amax over the ranks (torch stands in for the collectives,
which carry no arithmetic of the method).  The merged result must equal the
oracle's verification of the whole rows under the same rule as osd_verify:
bit-exact outside the 1e-6 margin band.  The per-rank records are checked as
well: each slice's normaliser against scipy's logsumexp of that slice, and
every rank must emit the same accepted lengths and reject masks, with the
extra token on exactly one rank.
"""
import numpy as np
import pytest

from oracle import ref
from paper_2310_07177_amd import synth
from tests._helpers import compare_verify, to_device

pytestmark = pytest.mark.gpu

ROW_STATS = np.dtype([("s_target", "<f8"), ("s_draft", "<f8"), ("k_target", "<f4"), ("k_draft", "<f4"),
                      ("t_y", "<f4"), ("d_y", "<f4"), ("argmax", "<i4"), ("flags", "<i4")])
assert ROW_STATS.itemsize == 40


@pytest.fixture(scope="module")
def osd():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2310_07177_amd as m
    m.lib()
    return m


def even_bounds(V, G):
    q, r = divmod(V, G)
    sizes = [q + (1 if g < r else 0) for g in range(G)]
    return np.concatenate([[0], np.cumsum(sizes)]).astype(int).tolist()


def run_sharded(osd, x, bounds, want_records=False):
    """The three phases on every rank, with the exchanges in between."""
    import torch
    T = x["T"]
    G = len(bounds) - 1
    V = x["target"].shape[-1]
    target = to_device(x["target"])
    draft = None if T == 0 else to_device(x["draft"])
    tokens = to_device(x["tokens"].astype(np.int32))
    dl = to_device(x.get("draft_len"))
    u_acc = None if T == 0 else to_device(x["u_accept"])
    u_res = None if T == 0 else to_device(x["u_resample"])
    tg = [target[:, :, bounds[g]:bounds[g + 1]].contiguous() for g in range(G)]
    dg = [None if draft is None else draft[:, :, bounds[g]:bounds[g + 1]].contiguous() for g in range(G)]
    stats = [osd.osd_shard_verify_stats(tg[g], dg[g], tokens, T, bounds[g], V, draft_len=dl) for g in range(G)]
    stats_all = torch.stack(stats)                      # all-gather, rank order
    mass = [osd.osd_shard_verify_mass(tg[g], dg[g], tokens, u_acc, T, stats_all, draft_len=dl)
            for g in range(G)]
    mass_all = torch.stack(mass)                        # all-gather, rank order
    outs = [osd.osd_shard_verify_draw(tg[g], dg[g], tokens, u_res, T, bounds[g], g, mass_all, draft_len=dl)
            for g in range(G)]
    torch.cuda.synchronize()
    accs = [o[0].cpu().numpy() for o in outs]
    toks = [o[1].cpu().numpy() for o in outs]
    rms = [o[2].cpu().numpy() for o in outs]
    for g in range(1, G):                               # every rank agrees
        assert np.array_equal(accs[g], accs[0]) and np.array_equal(rms[g], rms[0]), g
    merged = np.max(np.stack(toks), axis=0)             # all-reduce MAX
    acc = accs[0]
    if T > 0:
        # the extra token comes from exactly one rank
        for b in np.nonzero(acc >= 0)[0]:
            holders = [g for g in range(G) if toks[g][b, acc[b]] >= 0]
            assert len(holders) == 1, (b, holders)
    res = (acc, merged, rms[0])
    if want_records:
        return res, stats_all.cpu().numpy()
    return res


def oracle_verify(x):
    T = x["T"]
    return ref.verify(x["target"], None if T == 0 else x["draft"], x["tokens"],
                      None if T == 0 else x["u_accept"], None if T == 0 else x["u_resample"], T,
                      draft_len=x.get("draft_len"))


def check(osd, x, bounds, label, max_excluded_frac=0.1):
    acc, toks, rmask = run_sharded(osd, x, bounds)
    r = oracle_verify(x)
    n, ex = compare_verify(r, acc, toks, rmask, label)
    print(f"[{label}] G={len(bounds) - 1} compared {n} sequences, excluded {ex} (margin < 1e-6)", flush=True)
    assert ex <= max(1, max_excluded_frac * len(acc))
    return r, acc


@pytest.mark.parametrize("G", [1, 3, 7])
def test_shard_tiny_fp32(osd, G):
    """fp32 rows of 1000 split unevenly (element-wise loads)."""
    for seed in range(3):
        check(osd, synth.config_tiny(seed), even_bounds(1000, G), f"tiny seed {seed}")


@pytest.mark.parametrize("sigma", [0.25, 1.0, 2.0])
def test_shard_llama_vocab(osd, sigma):
    for seed in range(2):
        check(osd, synth.config_llama_vocab(sigma, seed), even_bounds(32000, 8), f"llama sigma={sigma} seed={seed}")


def test_shard_t5_vocab_full_batch(osd):
    x = synth.config_t5_vocab(0)
    check(osd, x, even_bounds(32128, 4), "t5 B=64 K=8 G=4")


def test_shard_t5_vocab_greedy(osd):
    x = synth.config_t5_vocab(1, greedy=True)
    check(osd, x, even_bounds(32128, 4), "t5 greedy G=4", max_excluded_frac=0.0)


def test_shard_greedy_ties_across_slices(osd):
    """Massive ties: the lowest global id wins, also when equal maxima sit in
    different slices."""
    g = np.random.default_rng(5)
    B, K, V = 16, 4, 3000
    t = g.integers(-2, 3, (B, K + 1, V)).astype(np.float32)
    x = dict(target=synth.to_bf16(t), draft=None, tokens=np.argmax(t[:, :K], -1).astype(np.int32),
             u_accept=None, u_resample=None, T=0.0)
    x["tokens"][::3, 1] = 0
    check(osd, x, [0, 5, 1000, 1001, 2999, 3000], "greedy ties", max_excluded_frac=0.0)


def test_shard_large_vocab_ragged(osd):
    """V = 128256 over 8 ranks (16032 each, the tensor-parallel shape) with
    ragged proposal lengths."""
    x = synth.config_large_vocab(seed=0, B=24)
    # With 128256 tokens the drawn token's mass is often of order 1e-6, so
    # the oracle's 1e-6 CDF margin excludes a larger share of sequences (the
    # expected share is the sum over tokens of min(p_j, 2e-6), ~0.1-0.2 here).
    check(osd, x, even_bounds(128256, 8), "V=128256 ragged G=8", max_excluded_frac=0.3)


def test_shard_uneven_slices(osd):
    """Slices of 1, 7, 8, 9 and the rest: rows shorter than one chunk, one
    chunk, and a ragged tail; bf16 (element-wise loads where a row is not a
    16-byte multiple)."""
    x = synth.verify_inputs(10, 5, 4000, "bf16", T=0.9, seed=12, target_std=2.0, draft_noise=0.8)
    check(osd, x, [0, 1, 8, 16, 25, 4000], "uneven slices")


def test_shard_ragged_lengths_and_invalid_rows(osd):
    x = synth.verify_inputs(12, 6, 5000, "bf16", T=1.0, seed=3, ragged=True, draft_noise=0.3)
    x["draft_len"][0] = 0        # invalid k_b
    x["draft_len"][1] = 7        # invalid k_b > K
    x["tokens"][2, 0] = 5000     # out-of-range proposal
    x["tokens"][3, x["draft_len"][3] - 1] = -3
    x["target"][4, 0, :] = 0xFF80  # a row without finite logits that the test reaches
    x["draft_len"][5] = 3          # the same after a certain rejection (never reached)
    x["target"][5, 0, :] = 0xFF80
    x["target"][5, 0, 17] = synth.to_bf16(np.float32([0.0]))[0]
    x["draft"][5, 0, :] = synth.to_bf16(np.float32([0.0]))[0]
    x["tokens"][5, 0] = 3
    x["target"][5, 1, :] = 0xFF80
    r, acc = check(osd, x, even_bounds(5000, 4), "ragged + invalid G=4")
    assert acc[:5].tolist() == [-1] * 5
    assert acc[5] == 0 and r["out_tokens"][5, 0] == 17


def test_shard_identical_rows_accept_all(osd):
    x = synth.verify_inputs(16, 8, 32128, "bf16", T=0.7, seed=4)
    x["draft"] = x["target"][:, :8].copy()
    x["u_accept"][:] = np.float32(1 - 2 ** -24)
    acc, toks, rmask = run_sharded(osd, x, even_bounds(32128, 8))
    assert (acc == 8).all() and (rmask == 0).all()


def test_shard_neg_inf_entries(osd):
    x = synth.verify_inputs(8, 4, 3000, "f32", T=1.0, seed=9, draft_noise=1.5)
    g = np.random.default_rng(1)
    x["target"][g.random(x["target"].shape) < 0.3] = -np.inf
    x["draft"][g.random(x["draft"].shape) < 0.3] = -np.inf
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(5), x["draft"], 1.0)
    check(osd, x, even_bounds(3000, 5), "-inf entries G=5")


def test_shard_whole_slice_neg_inf(osd):
    """A slice that holds no finite logit of a row (all its mass elsewhere)."""
    x = synth.verify_inputs(8, 3, 2048, "bf16", T=1.0, seed=21, draft_noise=0.5)
    x["target"][:, :, 1024:] = 0xFF80
    x["draft"][:, :, 1024:] = 0xFF80
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(6), x["draft"], 1.0)
    check(osd, x, [0, 1024, 2048], "empty second slice")


def test_shard_records_match_slice_logsumexp(osd):
    """Each rank's record of each row: (k + log2 s) ln 2 is the log-sum-exp of
    the slice at temperature T (scipy, fp64), and the proposal's logits are
    picked up exactly by the rank that holds them."""
    from scipy.special import logsumexp
    x = synth.config_llama_vocab(1.0, seed=4)
    bounds = even_bounds(32000, 8)
    (acc, _, _), rec = run_sharded(osd, x, bounds, want_records=True)
    rec = rec.reshape(-1).view(ROW_STATS).reshape(rec.shape[:3])
    T, K = x["T"], x["K"]
    t = synth.as_f32(x["target"]).astype(np.float64)
    d = synth.as_f32(x["draft"]).astype(np.float64)
    for g in range(8):
        v0, v1 = bounds[g], bounds[g + 1]
        for b in range(x["B"]):
            for i in range(K + 1):
                r = rec[g, b, i]
                lse = logsumexp(t[b, i, v0:v1] / T)
                got = (float(r["k_target"]) + np.log2(r["s_target"])) * np.log(2.0)
                assert abs(got - lse) <= 1e-6 * max(1.0, abs(lse)), (g, b, i, got, lse)
                if i < K:
                    lsd = logsumexp(d[b, i, v0:v1] / T)
                    got = (float(r["k_draft"]) + np.log2(r["s_draft"])) * np.log(2.0)
                    assert abs(got - lsd) <= 1e-6 * max(1.0, abs(lsd)), (g, b, i, got, lsd)
                    y = int(x["tokens"][b, i])
                    holds = v0 <= y < v1
                    assert bool(r["flags"] & 1) == holds
                    if holds:
                        assert r["t_y"] == np.float32(t[b, i, y]) and r["d_y"] == np.float32(d[b, i, y])


def test_shard_deterministic_and_reusable(osd):
    x = synth.config_t5_vocab(3, B=16)
    a = run_sharded(osd, x, even_bounds(32128, 8))
    b = run_sharded(osd, x, even_bounds(32128, 8))
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


def test_shard_gap_in_slices_invalidates_the_sequence(osd):
    """Slices that do not cover the vocabulary (a caller's mistake the host
    cannot see): a sequence is invalid (-1) when the test reaches a proposal
    that no rank holds; sequences whose tested proposals all lie inside the
    slices are still verified exactly like the whole rows (the oracle), as
    long as the residual draw does not need the missing columns.  Nothing
    faults."""
    import torch
    B, K, V = 16, 3, 3000
    x = synth.verify_inputs(B, K, V, "f32", T=1.0, seed=51, target_std=2.0, draft_noise=1.0)
    # the gap [1000, 1100) holds no probability in either row, so the draws
    # of the whole rows and of the covered slices coincide
    x["target"][:, :, 1000:1100] = -np.inf
    x["draft"][:, :, 1000:1100] = -np.inf
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(9), x["draft"], 1.0)
    x["tokens"][:4, 0] = 1050  # proposals inside the gap (p = q = 0 there)
    slices = [(0, 1000), (1100, 3000)]
    t, d = to_device(x["target"]), to_device(x["draft"])
    y = to_device(x["tokens"].astype(np.int32))
    ua, ur = to_device(x["u_accept"]), to_device(x["u_resample"])
    tg = [t[:, :, a:e].contiguous() for a, e in slices]
    dg = [d[:, :, a:e].contiguous() for a, e in slices]
    G = len(slices)
    st = torch.stack([osd.osd_shard_verify_stats(tg[g], dg[g], y, 1.0, slices[g][0], V) for g in range(G)])
    ms = torch.stack([osd.osd_shard_verify_mass(tg[g], dg[g], y, ua, 1.0, st) for g in range(G)])
    outs = [osd.osd_shard_verify_draw(tg[g], dg[g], y, ur, 1.0, slices[g][0], g, ms) for g in range(G)]
    toks = torch.stack([o[1] for o in outs]).amax(0).cpu().numpy()
    acc = outs[0][0].cpu().numpy()
    torch.cuda.synchronize()
    assert acc[:4].tolist() == [-1] * 4 and (toks[:4] == -1).all()
    r = oracle_verify(x)
    ok = np.arange(B) >= 4
    n, ex = compare_verify({k: (v[ok] if isinstance(v, np.ndarray) else v) for k, v in r.items()},
                           acc[ok], toks[ok], outs[0][2].cpu().numpy()[ok], "gap in slices")
    print(f"[gap in slices] compared {n}, excluded {ex}", flush=True)
