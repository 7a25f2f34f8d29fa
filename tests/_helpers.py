"""Shared test helpers: moving synthetic inputs to the GPU and comparing the
HIP path with the oracle under the parity rules (exact discrete outputs except
where an evaluated decision has a margin below 1e-6; fp32 losses within 1e-5
relative; bf16 gradients within 2e-3 absolute except at bf16 rounding
midpoints)."""
import numpy as np

MARGIN = 1e-6
LOSS_RTOL = 1e-5
BF16_GRAD_ATOL = 2e-3
F32_GRAD_ATOL = 2e-6


def to_device(a, device="cuda"):
    import torch
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:  # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def at_risk(ref):
    """Sequences whose oracle decisions sit within MARGIN of a boundary (or
    used the Z == 0 fallback): excluded from the exact comparison."""
    ma = ref["margin_accept"]
    with np.errstate(invalid="ignore"):
        close_acc = np.nan_to_num(ma, nan=np.inf) < MARGIN
    close_cdf = np.nan_to_num(ref["margin_cdf"], nan=np.inf) < MARGIN
    return close_acc.any(axis=1) | close_cdf | (ref["z_fallback"] != 0)


def compare_verify(ref, acc, toks, rmask, label=""):
    """Exact comparison outside the margin band; returns (#compared, #excluded)."""
    risky = at_risk(ref)
    ok = ~risky
    bad = []
    for b in np.nonzero(ok)[0]:
        if (acc[b] != ref["accepted_len"][b] or not np.array_equal(toks[b], ref["out_tokens"][b])
                or not np.array_equal(rmask[b], ref["reject_mask"][b])):
            bad.append(b)
    assert not bad, (f"{label}: {len(bad)} sequences differ, first b={bad[0]}: "
                     f"gpu a={acc[bad[0]]} toks={toks[bad[0]].tolist()} | "
                     f"oracle a={ref['accepted_len'][bad[0]]} toks={ref['out_tokens'][bad[0]].tolist()}")
    return int(ok.sum()), int(risky.sum())


def compare_losses(gpu, ref, rtol=LOSS_RTOL, atol=1e-7, label=""):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(gpu - ref)
    lim = rtol * np.abs(ref) + atol
    worst = int(np.argmax(err - lim)) if err.size else 0
    assert np.all(err <= lim), (f"{label}: loss mismatch at {worst}: gpu={gpu.flat[worst]!r} "
                                f"oracle={ref.flat[worst]!r}")


def compare_grad_bf16(gpu_bits, ref_f64, label=""):
    """|gpu - RNE_bf16(oracle)| <= 2e-3, excluding elements whose exact value
    lies within 2^-20 |g| of a bf16 rounding midpoint.  Returns #excluded."""
    from oracle import ref as oref
    want = oref.round_bf16(ref_f64)
    g = oref.bf16_to_f64(gpu_bits)
    w = oref.bf16_to_f64(want)
    mid = oref.bf16_midpoint_flags(ref_f64)
    err = np.abs(g - w)
    bad = (err > BF16_GRAD_ATOL) & ~mid
    assert not bad.any(), (f"{label}: {int(bad.sum())} gradient elements off by > 2e-3, "
                           f"max {float(err[~mid].max())}")
    # Where |g| >= 1e-2 the fp32 arithmetic is accurate to well under 2^-14
    # relative (no cancellation to speak of), so away from that band around a
    # rounding midpoint the kernel's round-to-nearest-even must land on the
    # very same bf16 value: this catches a wrong rounding mode.
    wide = oref.bf16_midpoint_flags(ref_f64, rel=2.0 ** -14)
    flips = (g != w) & ~wide & np.isfinite(ref_f64) & (np.abs(ref_f64) >= 1e-2)
    assert not flips.any(), (f"{label}: {int(flips.sum())} gradient elements not the RNE bf16 "
                             f"of the exact value (first at {np.argwhere(flips)[0].tolist()})")
    return int(mid.sum())


def compare_grad_f32(gpu, ref_f64, label=""):
    err = np.abs(np.asarray(gpu, np.float64) - ref_f64)
    lim = F32_GRAD_ATOL + 1e-5 * np.abs(ref_f64)
    assert np.all(err <= lim), f"{label}: fp32 gradient max error {float(err.max())}"
