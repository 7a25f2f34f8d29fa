"""Canary guard bands around every output buffer.

Each output is a window inside a larger allocation filled with a canary byte;
after the call, the bytes before and after every window must be untouched.
The shapes are the ones most likely to write past an end: ragged proposal
lengths, row lengths that are not a multiple of a chunk (V = 1, 7, 1001),
outputs that are not 16-byte aligned, long streamed rows, and trees (both
layouts of the tree kernel: V = 4096 bf16 takes the streaming one).  The
calls go through the C ABI directly, with raw pointers into the windows.
"""
import ctypes

import numpy as np
import pytest

from paper_2310_07177_amd import binding, synth
from tests._helpers import to_device

pytestmark = pytest.mark.gpu

CANARY = 0x5A
GUARD = 4096


@pytest.fixture(scope="module")
def L():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    return binding.lib()


class Guarded:
    """A window of `nbytes` at byte offset GUARD + shift inside a canary-filled
    allocation."""

    def __init__(self, nbytes, shift=0):
        import torch
        self.n, self.off = int(nbytes), GUARD + shift
        self.buf = torch.full((self.n + 2 * GUARD + 64,), CANARY, dtype=torch.uint8, device="cuda")

    @property
    def ptr(self):
        return ctypes.c_void_p(self.buf.data_ptr() + self.off)

    def check(self, label):
        b = self.buf.cpu().numpy()
        before, after = b[:self.off], b[self.off + self.n:]
        assert (before == CANARY).all(), f"{label}: {int((before != CANARY).sum())} bytes written before the buffer"
        assert (after == CANARY).all(), f"{label}: {int((after != CANARY).sum())} bytes written after the buffer"


def stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def zeros_ws(n):
    import torch
    return torch.zeros(max(int(n), 256), dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("V,dtype,shift", [(1, "bf16", 0), (7, "bf16", 4), (1001, "bf16", 0), (1001, "f32", 8),
                                           (8192, "bf16", 0), (70001, "bf16", 4)])
def test_verify_and_distill_outputs_stay_in_bounds(L, V, dtype, shift):
    import torch
    x = synth.verify_inputs(5, 6, V, dtype, T=1.0, seed=V % 17, draft_noise=0.8, ragged=True)
    x["draft_len"][0] = 0  # an invalid row too
    B, K = 5, 6
    dt = binding.OSD_BF16 if dtype == "bf16" else binding.OSD_F32
    eb = 2 if dtype == "bf16" else 4
    t, d = to_device(x["target"]), to_device(x["draft"])
    y, ua, ur = to_device(x["tokens"].astype(np.int32)), to_device(x["u_accept"]), to_device(x["u_resample"])
    dl = to_device(x["draft_len"])
    acc, toks, rm = Guarded(4 * B, shift), Guarded(4 * B * (K + 1), shift), Guarded(B * K, shift + 1)
    ws = zeros_ws(L.osd_verify_workspace_bytes(B, K))
    assert L.osd_verify(ptr(t), ptr(d), dt, B, K, V, ptr(y), ptr(dl), ptr(ua), ptr(ur), ctypes.c_float(1.0),
                        acc.ptr, toks.ptr, rm.ptr, ptr(ws), ws.numel(), stream()) == 0
    torch.cuda.synchronize()
    for g, n in ((acc, "accepted_len"), (toks, "out_tokens"), (rm, "reject_mask")):
        g.check(f"verify V={V} {dtype} {n}")
    # distillation of every row, then the fused entry points
    mask = to_device(np.ones((B, K), np.uint8))
    for kind in (binding.OSD_FKL, binding.OSD_JSD):
        loss, rows, grad = Guarded(8, shift), Guarded(4 * B * K, shift), Guarded(B * K * V * eb, shift)
        wsd = zeros_ws(L.osd_distill_workspace_bytes(B, K))
        assert L.osd_distill_loss_grad(ptr(t), (K + 1) * V, ptr(d), K * V, dt, B, K, V, ptr(mask), kind,
                                       ctypes.c_float(0.5), ctypes.c_float(0.9), loss.ptr, rows.ptr, grad.ptr,
                                       ptr(wsd), wsd.numel(), stream()) == 0
        torch.cuda.synchronize()
        for g, n in ((loss, "loss"), (rows, "row_loss"), (grad, "grad")):
            g.check(f"distill kind={kind} V={V} {dtype} {n}")
    outs = [Guarded(4 * B, shift), Guarded(4 * B * (K + 1), shift), Guarded(B * K, shift + 1), Guarded(8, shift),
            Guarded(4 * B * K, shift), Guarded(B * K * V * eb, shift)]
    wsf = zeros_ws(L.osd_verify_distill_workspace_bytes(B, K))
    assert L.osd_verify_distill(ptr(t), ptr(d), dt, B, K, V, ptr(y), ptr(dl), ptr(ua), ptr(ur), ctypes.c_float(1.0),
                                outs[0].ptr, outs[1].ptr, outs[2].ptr, ptr(mask), binding.OSD_RKL,
                                ctypes.c_float(0.5), outs[3].ptr, outs[4].ptr, outs[5].ptr, ptr(wsf), wsf.numel(),
                                stream()) == 0
    torch.cuda.synchronize()
    for j, g in enumerate(outs):
        g.check(f"verify_distill V={V} {dtype} output {j}")
    outs = [Guarded(4 * B, shift), Guarded(4 * B * (K + 1), shift), Guarded(B * K, shift + 1), Guarded(8, shift),
            Guarded(4 * B * K, shift), Guarded(B * K * V * eb, shift)]
    assert L.osd_verify_distill_rejected(ptr(t), ptr(d), dt, B, K, V, ptr(y), ptr(dl), ptr(ua), ptr(ur),
                                         ctypes.c_float(1.0), outs[0].ptr, outs[1].ptr, outs[2].ptr, binding.OSD_FKL,
                                         ctypes.c_float(0.5), outs[3].ptr, outs[4].ptr, outs[5].ptr, ptr(wsf),
                                         wsf.numel(), stream()) == 0
    torch.cuda.synchronize()
    for j, g in enumerate(outs):
        g.check(f"verify_distill_rejected V={V} {dtype} output {j}")


@pytest.mark.parametrize("V,dtype", [(7, "bf16"), (1001, "f32"), (4096, "bf16"), (70001, "bf16")])
def test_sample_and_tree_outputs_stay_in_bounds(L, V, dtype):
    import torch
    dt = binding.OSD_BF16 if dtype == "bf16" else binding.OSD_F32
    x = synth.sample_inputs(9, V, dtype, seed=V % 11)
    p, q, u = to_device(x["p"]), to_device(x["q"]), to_device(x["u"])
    for beta, T in ((0.5, 1.0), (0.0, 0.8), (1.0, 0.0)):
        out = Guarded(4 * 9, 4)
        ws = zeros_ws(L.osd_sample_workspace_bytes(9))
        assert L.osd_sample(ptr(p), V, ptr(q), V, dt, 9, V, ctypes.c_float(T), ctypes.c_float(beta), ptr(u),
                            out.ptr, ptr(ws), ws.numel(), stream()) == 0
        torch.cuda.synchronize()
        out.check(f"sample V={V} beta={beta} T={T}")
    if V > 32768:
        return  # beyond the tree kernel's rows
    g = synth.rng(V)
    par = np.stack([synth.random_tree_parents(g, 11) for _ in range(3)])
    tx = synth.tree_inputs(3, par, V, dtype, T=0.9, seed=V % 7)
    B, N = 3, 11
    args = [to_device(tx[k]) for k in ("target", "draft", "parent", "tokens", "u_accept", "u_resample")]
    for T in (0.9, 0.0):
        outs = [Guarded(4 * B, 4), Guarded(4 * B * N, 4), Guarded(4 * B * N, 8)]
        ws = zeros_ws(L.osd_verify_tree_workspace_bytes(B, N))
        assert L.osd_verify_tree(ptr(args[0]), ptr(args[1]), dt, B, N, V, ptr(args[2]), ptr(args[3]), ptr(args[4]),
                                 ptr(args[5]), ctypes.c_float(T), outs[0].ptr, outs[1].ptr, outs[2].ptr, ptr(ws),
                                 ws.numel(), stream()) == 0
        torch.cuda.synchronize()
        for j, o in enumerate(outs):
            o.check(f"tree V={V} T={T} output {j}")
