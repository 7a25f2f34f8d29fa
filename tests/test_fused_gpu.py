"""Parity of the fused entry point (osd_verify_distill) with the fp64 oracle.

One call verifies a step and distils it: the oracle side is ref.verify on the
step and ref.distill on target rows 0..K-1 and the draft rows at
tau = temperature, with the same mask.  The bar is that of the separate
entry points (tests/test_parity_gpu.py): exact discrete outputs outside the
1e-6 margin band, fp32 losses within 1e-5 relative, bf16 gradients within
2e-3 absolute of the oracle's fp64 value rounded to bf16 (midpoints
excluded), fp32 gradients within 2e-6.
"""
import numpy as np
import pytest

from oracle import ref
from paper_2310_07177_amd import synth
from tests._helpers import (compare_grad_bf16, compare_grad_f32, compare_losses,
                            compare_verify, to_device)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def osd():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    import paper_2310_07177_amd as m
    m.lib()
    return m


def run_fused(osd, x, kind, beta, mask):
    import torch
    out = osd.osd_verify_distill(to_device(x["target"]), to_device(x["draft"]),
                                 to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]),
                                 to_device(x["u_resample"]), x["T"], kind, beta,
                                 distill_mask=to_device(mask), draft_len=to_device(x.get("draft_len")))
    torch.cuda.synchronize()
    acc, toks, rmask, loss, rows, g = out
    if g.dtype == torch.bfloat16:
        g = g.cpu().view(torch.int16).numpy().view(np.uint16)
    else:
        g = g.cpu().numpy()
    return (acc.cpu().numpy(), toks.cpu().numpy(), rmask.cpu().numpy(), loss.cpu().numpy(),
            rows.cpu().numpy(), g)


def check_fused(osd, x, kind, beta, mask, label, max_excluded_frac=0.1, loss_atol=1e-7):
    acc, toks, rmask, loss, rows, g = run_fused(osd, x, kind, beta, mask)
    B, K, V = x["target"].shape[0], x["target"].shape[1] - 1, x["target"].shape[2]
    rv = ref.verify(x["target"], x["draft"], x["tokens"], x["u_accept"], x["u_resample"], x["T"],
                    draft_len=x.get("draft_len"))
    n, ex = compare_verify(rv, acc, toks, rmask, label)
    assert ex <= max(1, max_excluded_frac * B)
    rd = ref.distill(x["target"], x["draft"], kind, beta=beta, tau=x["T"], mask=mask, B=B, K=K,
                     teacher_batch_stride=(K + 1) * V, student_batch_stride=K * V)
    compare_losses(rows, rd["row_loss"], atol=loss_atol, label=f"{label} row loss")
    compare_losses(loss, [rd["loss_mean"], rd["loss_sum"]], atol=np.array([loss_atol, loss_atol * rows.size]),
                   label=f"{label} loss")
    if g.dtype == np.uint16:
        gx = compare_grad_bf16(g, rd["grad"], label)
    else:
        compare_grad_f32(g, rd["grad"], label)
        gx = 0
    print(f"[{label}] compared {n} sequences, excluded {ex}; loss {loss.tolist()}; "
          f"{gx} midpoint gradient elements excluded", flush=True)
    return rv, acc, loss


@pytest.mark.parametrize("kind", ["jsd", "rkl", "fkl"])
def test_fused_t5_vocab_full_batch(osd, kind):
    """B=64 k=8 V=32128 bf16, T = tau = 0.7, every row distilled."""
    x = synth.config_t5_vocab(0)
    check_fused(osd, x, kind, 0.5, np.ones((x["B"], x["K"]), np.uint8), f"fused t5 {kind}")


@pytest.mark.parametrize("sigma", [1.0, 2.0])
def test_fused_llama_vocab(osd, sigma):
    """B=8 k=5 V=32000 bf16 at acceptance rates from about 0.9 to 0.4, forward
    KL (the divergence this workload specifies) with a random mask."""
    x = synth.config_llama_vocab(sigma, 0)
    mask = (np.random.default_rng(int(sigma * 8)).random((x["B"], x["K"])) < 0.5).astype(np.uint8)
    check_fused(osd, x, "fkl", 0.5, mask, f"fused llama sigma={sigma}")


def test_fused_llama_vocab_small_divergence(osd):
    """Nearly identical rows (sigma = 0.25, D ~ 0.02 nats, a token with
    p ~ 0.92 far above its thread's first chunk): the log-ratios must come
    from the same rounded exponents as the normalisers, or the row loss is
    off by ~4e-5 relative."""
    x = synth.config_llama_vocab(0.25, 0)
    mask = (np.random.default_rng(2).random((x["B"], x["K"])) < 0.5).astype(np.uint8)
    check_fused(osd, x, "fkl", 0.5, mask, "fused llama sigma=0.25")


@pytest.mark.parametrize("beta", [0.3, 0.7])
def test_fused_llama_vocab_jsd(osd, beta):
    """JSD on the sigma = 1 Llama-vocab step (divergence ~0.1 nats per row)."""
    x = synth.config_llama_vocab(1.0, 1)
    mask = (np.random.default_rng(7).random((x["B"], x["K"])) < 0.5).astype(np.uint8)
    check_fused(osd, x, "jsd", beta, mask, f"fused llama jsd beta={beta}")


def test_fused_tiny_fp32(osd):
    x = synth.config_tiny(0)
    check_fused(osd, x, "fkl", 0.5, x["mask"], "fused tiny fp32")


@pytest.mark.parametrize("V,dtype", [(1000, "bf16"), (8192, "bf16"), (8200, "bf16"), (20000, "bf16"), (4100, "f32"),
                                     (1001, "bf16"), (40000, "bf16")])
def test_fused_vocab_sizes(osd, V, dtype):
    """Streaming tiles of several sizes (256x1, 1024x1, 1024x2, 1024x3, the
    partial ones ending in a part-filled round), an unaligned row length and
    a vocabulary above the streaming tiles (the last two take the two-call
    path inside the entry point)."""
    x = synth.verify_inputs(6, 4, V, dtype, T=0.9, seed=V % 97, target_std=2.5, draft_noise=0.8)
    mask = (np.random.default_rng(V).random((6, 4)) < 0.7).astype(np.uint8)
    check_fused(osd, x, "rkl", 0.5, mask, f"fused V={V} {dtype}")


def test_fused_ragged_and_invalid(osd):
    """Ragged proposal lengths, invalid lengths and tokens, rows without a
    finite logit (read or skipped), and distilled padding rows."""
    x = synth.verify_inputs(12, 6, 5000, "bf16", T=1.0, seed=3, ragged=True, draft_noise=1.0)
    V = x["target"].shape[2]
    x["draft_len"][0] = 0        # invalid k_b
    x["draft_len"][1] = 7        # invalid k_b > K
    x["tokens"][2, 0] = V        # out-of-range proposal
    x["tokens"][3, x["draft_len"][3] - 1] = -3
    x["target"][4, 0, :] = 0xFF80  # no finite logit at position 0 (read: invalid)
    x["draft_len"][5] = 3
    x["target"][5, 0, :] = 0xFF80
    x["target"][5, 0, 17] = synth.to_bf16(np.float32([0.0]))[0]
    x["draft"][5, 0, :] = synth.to_bf16(np.float32([0.0]))[0]
    x["tokens"][5, 0] = 3        # p(y) = 0: always rejected
    mask = np.ones((12, 6), np.uint8)
    mask[4, 0] = 0               # keep the all -inf teacher row out of the distillation
    mask[5, 1] = 0
    x["target"][5, 1, :] = 0xFF80
    rv, acc, _ = check_fused(osd, x, "jsd", 0.5, mask, "fused ragged + invalid")
    assert acc[:5].tolist() == [-1] * 5
    assert acc[5] == 0 and rv["out_tokens"][5, 0] == 17


def test_fused_identical_rows(osd):
    """Draft = target: every proposal accepted, divergence and gradient 0."""
    x = synth.verify_inputs(16, 8, 32128, "bf16", T=0.7, seed=4)
    x["draft"] = x["target"][:, :8].copy()
    x["u_accept"][:] = np.float32(0.5)
    acc, toks, rmask, loss, rows, g = run_fused(osd, x, "jsd", 0.5, None)
    assert (acc == 8).all() and (rmask == 0).all()
    assert np.all(np.abs(rows) <= 1e-6) and abs(loss[1]) <= 1e-6 * rows.size
    assert np.all(np.abs(synth.bf16_to_f32(g)) <= 1e-6)


def test_fused_matches_separate_calls_and_is_deterministic(osd):
    """Same step through osd_verify + osd_distill_loss_grad and through the
    fused entry point: identical discrete outputs outside the margin band,
    identical row losses and gradients; two fused calls are bitwise equal."""
    import torch
    x = synth.config_t5_vocab(5)
    B, K, V = x["B"], x["K"], x["V"]
    mask = np.ones((B, K), np.uint8)
    a = run_fused(osd, x, "jsd", 0.5, mask)
    b = run_fused(osd, x, "jsd", 0.5, mask)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    acc, toks, rmask = osd.osd_verify(to_device(x["target"]), to_device(x["draft"]),
                                      to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]),
                                      to_device(x["u_resample"]), x["T"])
    loss, rows, g = osd.osd_distill_loss_grad(to_device(x["target"]), to_device(x["draft"]), "jsd", 0.5,
                                              x["T"], mask=to_device(mask), B=B, K=K,
                                              teacher_batch_stride=(K + 1) * V, student_batch_stride=K * V)
    torch.cuda.synchronize()
    rv = ref.verify(x["target"], x["draft"], x["tokens"], x["u_accept"], x["u_resample"], x["T"])
    from tests._helpers import at_risk
    ok = ~at_risk(rv)
    assert np.array_equal(a[0][ok], acc.cpu().numpy()[ok])
    assert np.array_equal(a[1][ok], toks.cpu().numpy()[ok])
    assert np.array_equal(a[4], rows.cpu().numpy())
    assert np.array_equal(a[5], g.cpu().view(torch.int16).numpy().view(np.uint16))


def test_fused_high_acceptance_bonus_rows(osd):
    """B=64 k=8 V=32128: draft = target except one boosted proposal logit in
    16 sequences (a rejection at a chosen position, in either round of the
    workgroups' items); the other 48 accept all 8 proposals and draw the
    bonus token from the target row k_b, which the workgroups must read."""
    x = synth.verify_inputs(64, 8, 32128, "bf16", T=0.7, seed=11)
    x["draft"] = x["target"][:, :8].copy()
    x["u_accept"][:] = np.float32(0.5)
    rng = np.random.default_rng(5)
    rej = {int(b): int(rng.integers(0, 8)) for b in rng.choice(64, 16, replace=False)}
    for b, j in rej.items():
        y = x["tokens"][b, j]
        x["draft"][b, j, y] = synth.to_bf16(synth.bf16_to_f32(x["draft"][b, j, y:y + 1]) + np.float32(4.0))[0]
    # Rows with D = 0 exactly: each of the V fp32 terms p (log p - log m)
    # carries a rounding error of a few units of 2^-24 times |log2 p|, so the
    # computed row loss is zero only to about 2^-24 * (entropy in bits) * a
    # few, i.e. below 1e-6 at V = 32128 (the identical-rows test's bound).
    _, acc, _ = check_fused(osd, x, "jsd", 0.5, np.ones((64, 8), np.uint8), "fused high acceptance",
                            loss_atol=1e-6)
    want = np.array([rej.get(b, 8) for b in range(64)])
    assert np.array_equal(acc, want)


@pytest.mark.parametrize("side", ["draft", "target"])
def test_fused_jsd_one_sided_neg_inf(osd, side):
    """-inf logits in the draft rows only (q = 0 where p > 0) or in the target
    rows only, with JSD distillation of every row: verification and the
    divergence agree with the oracle."""
    x = synth.verify_inputs(6, 4, 6000, "bf16", T=1.0, seed=31, target_std=2.0, draft_noise=1.0)
    g = np.random.default_rng(37)
    holes = g.random(x[side].shape) < 0.25
    x[side][holes] = 0xFF80
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(8), x["draft"], 1.0)
    mask = np.ones((6, 4), np.uint8)
    check_fused(osd, x, "jsd", 0.5, mask, f"fused one-sided -inf ({side})")


@pytest.mark.parametrize("beta", [0.0, 1.0])
def test_fused_jsd_endpoints_are_zero(osd, beta):
    """JSD at beta in {0, 1} is identically 0 (the term of weight 0 is left
    out): zero losses and gradient rows, while verification is unaffected."""
    x = synth.verify_inputs(8, 4, 8192, "bf16", T=0.9, seed=43, target_std=2.5, draft_noise=1.5)
    holes = np.random.default_rng(3).random(x["draft"].shape) < 0.2
    x["draft"][holes] = 0xFF80
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(9), x["draft"], 0.9)
    mask = np.ones((8, 4), np.uint8)
    _, _, loss = check_fused(osd, x, "jsd", beta, mask, f"fused jsd beta={beta}")
    acc, toks, rmask, loss, rows, g = run_fused(osd, x, "jsd", beta, mask)
    assert loss.tolist() == [0.0, 0.0] and not rows.any()
    assert np.all(synth.bf16_to_f32(g) == 0.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind,side", [("fkl", "target"), ("rkl", "draft")])
def test_fused_kl_one_sided_neg_inf(osd, kind, side, dtype):
    """-inf logits on the side that keeps the divergence finite (FKL: target
    holes, p = 0 < q; RKL: draft holes, q = 0 < p): the gradient at a hole is
    q/tau (FKL) or 0 (RKL), and the draws use each side's own probability."""
    V = 8192 if dtype == "bf16" else 4100
    x = synth.verify_inputs(6, 4, V, dtype, T=1.0, seed=47, target_std=2.0, draft_noise=1.0)
    holes = np.random.default_rng(53).random(x[side].shape) < 0.25
    x[side][holes] = 0xFF80 if dtype == "bf16" else -np.inf
    x["tokens"] = synth.gumbel_max_tokens(synth.rng(10), x["draft"], 1.0)
    check_fused(osd, x, kind, 0.5, np.ones((6, 4), np.uint8), f"fused {kind} one-sided -inf ({side}) {dtype}")


def test_fused_nan_logits_give_invalid_rows(osd):
    """A NaN logit in a target or draft row that the test reaches invalidates
    the sequence, as in osd_verify."""
    x = synth.verify_inputs(8, 4, 8192, "bf16", T=1.0, seed=59, draft_noise=0.5)
    x["target"][0, 0, 100] = np.uint16(0x7FC0)
    x["draft"][1, 0, 7] = np.uint16(0x7FC0)
    mask = np.ones((8, 4), np.uint8)
    mask[:2] = 0                          # a NaN row has no finite divergence
    acc, toks, rmask, loss, rows, g = run_fused(osd, x, "fkl", 0.5, mask)
    assert acc[0] == -1 and acc[1] == -1 and (toks[:2] == -1).all() and not rmask[:2].any()
    rv = ref.verify(x["target"], x["draft"], x["tokens"], x["u_accept"], x["u_resample"], x["T"])
    keep = np.arange(8) >= 2
    rr = {k: (v[keep] if isinstance(v, np.ndarray) and v.shape[:1] == (8,) else v) for k, v in rv.items()}
    compare_verify(rr, acc[keep], toks[keep], rmask[keep], "fused nan rows")
    assert np.isfinite(loss).all()


# --------------------------------------------------------------------------
# Error-index mode: distil the row at each sequence's first rejection
# --------------------------------------------------------------------------

def run_rejected(osd, x, kind, beta):
    import torch
    out = osd.osd_verify_distill_rejected(to_device(x["target"]), to_device(x["draft"]),
                                          to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]),
                                          to_device(x["u_resample"]), x["T"], kind, beta,
                                          draft_len=to_device(x.get("draft_len")))
    torch.cuda.synchronize()
    acc, toks, rmask, loss, rows, g = out
    if g.dtype == torch.bfloat16:
        g = g.cpu().view(torch.int16).numpy().view(np.uint16)
    else:
        g = g.cpu().numpy()
    return (acc.cpu().numpy(), toks.cpu().numpy(), rmask.cpu().numpy(), loss.cpu().numpy(),
            rows.cpu().numpy(), g)


def check_rejected(osd, x, kind, beta, label, max_excluded_frac=0.1):
    """Against ref.verify, then ref.distill with the verification's reject
    mask (the kernel's own mask, which equals the oracle's on every sequence
    compared exactly; a sequence inside the margin band may legitimately
    reject elsewhere, and its distilled row follows its own outcome)."""
    acc, toks, rmask, loss, rows, g = run_rejected(osd, x, kind, beta)
    B, K, V = x["target"].shape[0], x["target"].shape[1] - 1, x["target"].shape[2]
    rv = ref.verify(x["target"], x["draft"], x["tokens"], x["u_accept"], x["u_resample"], x["T"],
                    draft_len=x.get("draft_len"))
    n, ex = compare_verify(rv, acc, toks, rmask, label)
    assert ex <= max(1, max_excluded_frac * B)
    rd = ref.distill(x["target"], x["draft"], kind, beta=beta, tau=x["T"], mask=rmask, B=B, K=K,
                     teacher_batch_stride=(K + 1) * V, student_batch_stride=K * V)
    compare_losses(rows, rd["row_loss"], label=f"{label} row loss")
    compare_losses(loss, [rd["loss_mean"], rd["loss_sum"]], label=f"{label} loss")
    if g.dtype == np.uint16:
        gx = compare_grad_bf16(g, rd["grad"], label)
        gf = synth.bf16_to_f32(g)
    else:
        compare_grad_f32(g, rd["grad"], label)
        gx, gf = 0, g
    off = rmask == 0
    assert not rows[off].any() and not gf[off].any(), "rows outside the first rejections must be zero"
    print(f"[{label}] compared {n} sequences, excluded {ex}; {int(rmask.sum())} rows distilled; "
          f"loss {loss.tolist()}; {gx} midpoint gradient elements excluded", flush=True)
    return acc, rmask, loss


@pytest.mark.parametrize("sigma", [0.25, 1.0, 2.0])
def test_rejected_llama_vocab(osd, sigma):
    """B=8 k=5 V=32000 bf16, forward KL on the rejected positions (the
    workload's own reading of which rows are distilled), three acceptance
    rates."""
    for seed in range(3):
        check_rejected(osd, synth.config_llama_vocab(sigma, seed), "fkl", 0.5, f"rejected llama sigma={sigma} seed={seed}")


@pytest.mark.parametrize("kind", ["jsd", "rkl", "fkl"])
def test_rejected_t5_vocab_full_batch(osd, kind):
    check_rejected(osd, synth.config_t5_vocab(0), kind, 0.5, f"rejected t5 {kind}")


def test_rejected_ragged_and_invalid(osd):
    """Ragged lengths; invalid lengths and tokens (a bad token anywhere in a
    sequence leaves its rejected row undistilled); a row without finite
    logits; p(y) = 0 at position 0."""
    x = synth.verify_inputs(12, 6, 5008, "bf16", T=1.0, seed=5, ragged=True, draft_noise=1.0)
    V = x["target"].shape[2]
    x["draft_len"][0] = 0
    x["draft_len"][1] = 7
    x["tokens"][2, x["draft_len"][2] - 1] = V    # out of range at the last position
    x["target"][4, 0, :] = 0xFF80
    x["draft_len"][5] = 3
    x["target"][5, 0, :] = 0xFF80
    x["target"][5, 0, 17] = synth.to_bf16(np.float32([0.0]))[0]
    x["draft"][5, 0, :] = synth.to_bf16(np.float32([0.0]))[0]
    x["tokens"][5, 0] = 3
    acc, rmask, _ = check_rejected(osd, x, "jsd", 0.5, "rejected ragged + invalid")
    assert acc[:3].tolist() == [-1] * 3 and acc[4] == -1 and acc[5] == 0
    assert not rmask[:5].any() and rmask[5, 0] == 1


@pytest.mark.parametrize("V,dtype", [(4100, "f32"), (1001, "bf16"), (40000, "bf16")])
def test_rejected_vocab_sizes(osd, V, dtype):
    """fp32 rows, an unaligned row length and a vocabulary above the
    streaming tiles (the last two take osd_verify + osd_distill_loss_grad
    inside the entry point)."""
    x = synth.verify_inputs(6, 4, V, dtype, T=0.9, seed=V % 89, target_std=2.5, draft_noise=0.8)
    check_rejected(osd, x, "rkl", 0.5, f"rejected V={V} {dtype}")


def test_rejected_matches_separate_calls(osd):
    """The same step as osd_verify, then osd_distill_loss_grad on its
    reject_mask: identical outputs (the two verifications' draws agree
    outside the margin band; row losses and gradients bit for bit), and two
    fused calls are bitwise equal."""
    import torch
    x = synth.config_t5_vocab(3)
    B, K, V = x["B"], x["K"], x["V"]
    a = run_rejected(osd, x, "jsd", 0.5)
    b = run_rejected(osd, x, "jsd", 0.5)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)
    acc, toks, rmask = osd.osd_verify(to_device(x["target"]), to_device(x["draft"]),
                                      to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]),
                                      to_device(x["u_resample"]), x["T"])
    loss, rows, g = osd.osd_distill_loss_grad(to_device(x["target"]), to_device(x["draft"]), "jsd", 0.5, x["T"],
                                              mask=rmask, B=B, K=K, teacher_batch_stride=(K + 1) * V,
                                              student_batch_stride=K * V)
    torch.cuda.synchronize()
    rv = ref.verify(x["target"], x["draft"], x["tokens"], x["u_accept"], x["u_resample"], x["T"])
    from tests._helpers import at_risk
    ok = ~at_risk(rv)
    assert np.array_equal(a[2][ok], rmask.cpu().numpy()[ok])
    assert np.array_equal(a[4][ok], rows.cpu().numpy()[ok])
    assert np.array_equal(a[5][ok], g.cpu().view(torch.int16).numpy().view(np.uint16)[ok])
    compare_losses(a[3], loss.cpu().numpy(), rtol=1e-6, label="fused vs separate loss")


def test_rejected_without_reject_mask_output(osd):
    """reject_mask is optional: the streaming path and the two-call path
    (which then keeps the mask in the workspace) give the same results."""
    import ctypes
    import torch
    from paper_2310_07177_amd import binding
    L = binding.lib()
    for V in (8192, 40000):
        x = synth.verify_inputs(8, 4, V, "bf16", T=1.0, seed=V % 7, draft_noise=1.0)
        want = run_rejected(osd, x, "fkl", 0.5)
        B, K = 8, 4
        dev = torch.device("cuda")
        acc = torch.empty(B, dtype=torch.int32, device=dev)
        toks = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
        loss = torch.empty(2, dtype=torch.float32, device=dev)
        rows = torch.empty(B, K, dtype=torch.float32, device=dev)
        g = torch.empty(B, K, V, dtype=torch.bfloat16, device=dev)
        ws = torch.zeros(L.osd_verify_distill_workspace_bytes(B, K), dtype=torch.uint8, device=dev)
        t, d = to_device(x["target"]), to_device(x["draft"])
        y, ua, ur = to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]), to_device(x["u_resample"])
        P = lambda z: ctypes.c_void_p(z.data_ptr())
        st = L.osd_verify_distill_rejected(P(t), P(d), binding.OSD_BF16, B, K, V, P(y), None, P(ua), P(ur),
                                           ctypes.c_float(1.0), P(acc), P(toks), None, binding.OSD_FKL,
                                           ctypes.c_float(0.5), P(loss), P(rows), P(g), P(ws), ws.numel(),
                                           ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0
        torch.cuda.synchronize()
        assert np.array_equal(acc.cpu().numpy(), want[0]) and np.array_equal(toks.cpu().numpy(), want[1])
        assert np.array_equal(loss.cpu().numpy(), want[3]) and np.array_equal(rows.cpu().numpy(), want[4])
        assert np.array_equal(g.cpu().view(torch.int16).numpy().view(np.uint16), want[5])
        assert int(ws.count_nonzero()) == 0, "the workspace is left zero"


SPECULATIVE = r'''
import sys
sys.path.insert(0, ".")
import numpy as np
from paper_2310_07177_amd import synth
from tests import test_fused_gpu as t
import paper_2310_07177_amd as osd
osd.lib()
import ctypes
_hip = ctypes.CDLL("libamdhip64.so")
_hip.hipGetErrorString.restype = ctypes.c_char_p
_orig = osd.binding.OsdError.__init__
def _init(self, fn, status):
    e = _hip.hipGetLastError()
    print("HIP last error", e, _hip.hipGetErrorString(e), flush=True)
    _orig(self, fn, status)
osd.binding.OsdError.__init__ = _init
# every rejecting workgroup at a position > 0 that has not seen an earlier
# rejection itself draws and distils without looking at the decisions
t.check_rejected(osd, synth.config_t5_vocab(0), "jsd", 0.5, "speculative rejected t5 jsd")
t.check_rejected(osd, synth.config_llama_vocab(2.0, 1), "fkl", 0.5, "speculative rejected llama sigma=2")
x = synth.verify_inputs(40, 8, 8192, "f32", T=0.8, seed=71, ragged=True, draft_noise=1.5)
t.check_rejected(osd, x, "rkl", 0.5, "speculative rejected ragged f32")
t.check_fused(osd, synth.config_t5_vocab(1), "jsd", 0.5, np.ones((64, 8), np.uint8), "speculative masked t5 jsd")
print("SPECULATIVE_OK", flush=True)
'''


def test_rejected_speculative_rows_are_cleared(osd):
    """With the fused kernel's bound on looks at earlier decisions set to 0
    (OSD_FUSED_POLLS, read once per process, so in a child process), every
    rejection at a position > 0 is drawn and distilled speculatively; the
    last workgroup must clear the rows that turn out not to be first.  The
    results must still equal the oracle's."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, OSD_FUSED_POLLS="0")
    r = subprocess.run([sys.executable, "-u", "-c", SPECULATIVE], cwd=root, env=env, capture_output=True, text=True,
                       timeout=150)
    print(r.stdout[-3000:], r.stderr[-3000:], flush=True)
    assert r.returncode == 0 and "SPECULATIVE_OK" in r.stdout


@pytest.mark.parametrize("V", [4096, 32128])
def test_fused_extreme_finite_logits(osd, V):
    """The fused step on bf16 rows with logits at the edges of the f16 range
    and beyond, and rows of denormals (both branches of the thread maxima),
    against the oracle."""
    from tests.test_parity_gpu import extreme_rows
    B, K = 4, 3
    x = synth.verify_inputs(B, K, V, "bf16", T=0.9, seed=43)
    t, s = extreme_rows(B, K, V, 47)
    x["target"], x["draft"] = synth.to_bf16(t), synth.to_bf16(s)
    # One-hot and tied rows put many decisions exactly on their boundaries
    # (such sequences are excluded from the token comparison by the margin
    # rule); losses and gradients are compared on every row.
    check_fused(osd, x, "jsd", 0.5, np.ones((B, K), np.uint8), f"extreme fused V={V}", max_excluded_frac=1.0)
