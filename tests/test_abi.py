"""The C ABI library loads, exports every function include/osd.h declares,
and rejects host-checkable mistakes before touching the GPU (no kernel is
launched by any call in this file)."""
import ctypes
import os
import re

import pytest

import paper_2310_07177_amd as osd
from paper_2310_07177_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "osd.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(osd_[a-z_]+)\s*\(", src)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = osd.lib()
    for name in declared_functions():
        assert hasattr(L, name), name
        assert getattr(L, name) is not None


def test_status_strings_and_limits():
    L = osd.lib()
    for s in (0, -1, -2, -3, -4, -5):
        assert L.osd_status_string(s).startswith(b"OSD_")
    assert L.osd_max_vocab(binding.OSD_BF16) >= 128256
    assert L.osd_max_vocab(binding.OSD_F32) >= 32768
    assert L.osd_max_vocab(7) == 0


def test_workspace_sizes():
    L = osd.lib()
    assert L.osd_verify_workspace_bytes(64, 8) >= 4 * (64 * 9 + 64)
    assert L.osd_verify_workspace_bytes(0, 8) == 0
    assert L.osd_verify_workspace_bytes(4, 17) == 0
    assert L.osd_distill_workspace_bytes(16384, 1) >= 8 * 16384
    assert L.osd_distill_workspace_bytes(-1, 1) == 0


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation
FAKE_MISALIGNED = ctypes.c_void_p(0x1004)


def verify(**kw):
    a = dict(target=FAKE, draft=FAKE, dtype=1, B=2, K=3, V=64, tokens=FAKE, dlen=None,
             ua=FAKE, ur=FAKE, T=1.0, acc=FAKE, toks=FAKE, rmask=None, ws=FAKE, wsb=1 << 20,
             stream=None)
    a.update(kw)
    return osd.lib().osd_verify(a["target"], a["draft"], a["dtype"], a["B"], a["K"], a["V"],
                                a["tokens"], a["dlen"], a["ua"], a["ur"], a["T"], a["acc"],
                                a["toks"], a["rmask"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(target=None), -1), (dict(tokens=None), -1), (dict(acc=None), -1), (dict(toks=None), -1),
    (dict(draft=None), -1), (dict(ua=None), -1), (dict(ur=None), -1),
    (dict(B=0), -1), (dict(K=0), -1), (dict(V=0), -1), (dict(K=17), -1), (dict(dtype=5), -1),
    (dict(V=1 << 20), -2), (dict(dtype=0, V=70000), -2),
    (dict(T=-1.0), -1), (dict(T=float("nan")), -1), (dict(T=float("inf")), -1),
    (dict(ws=None), -4), (dict(wsb=16), -4), (dict(ws=ctypes.c_void_p(0x1001)), -4),
])
def test_verify_rejects_bad_arguments(kw, status):
    assert verify(**kw) == status


def distill(**kw):
    a = dict(t=FAKE, ts=3 * 64, s=FAKE, ss=2 * 64, dtype=1, B=2, K=2, V=64, mask=None, kind=0,
             beta=0.5, tau=1.0, loss=FAKE, rows=None, grad=None, ws=FAKE, wsb=1 << 20, stream=None)
    a.update(kw)
    return osd.lib().osd_distill_loss_grad(a["t"], a["ts"], a["s"], a["ss"], a["dtype"], a["B"],
                                           a["K"], a["V"], a["mask"], a["kind"], a["beta"],
                                           a["tau"], a["loss"], a["rows"], a["grad"], a["ws"],
                                           a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(t=None), -1), (dict(s=None), -1), (dict(loss=None), -1),
    (dict(B=0), -1), (dict(K=-1), -1), (dict(V=0), -1), (dict(dtype=3), -1), (dict(kind=3), -1),
    (dict(tau=0.0), -1), (dict(tau=-2.0), -1), (dict(tau=float("nan")), -1),
    (dict(beta=-0.1), -1), (dict(beta=1.5), -1), (dict(beta=float("nan")), -1),
    (dict(ts=10), -1), (dict(ss=10), -1),
    (dict(V=1 << 20), -2),
    (dict(ws=None), -4), (dict(wsb=8), -4),
])
def test_distill_rejects_bad_arguments(kw, status):
    assert distill(**kw) == status


def test_binding_fails_loudly_without_gpu_tensors():
    import torch
    t = torch.zeros(1, 2, 8)
    with pytest.raises(ValueError):
        osd.osd_verify(t, t[:, :1].contiguous(), torch.zeros(1, 1, dtype=torch.int32),
                       torch.zeros(1, 1), torch.zeros(1), 1.0)


def fused(**kw):
    a = dict(target=FAKE, draft=FAKE, dtype=1, B=2, K=3, V=64, tokens=FAKE, dlen=None, ua=FAKE, ur=FAKE,
             T=0.8, acc=FAKE, toks=FAKE, rmask=None, mask=None, kind=2, beta=0.5, loss=FAKE, rows=None,
             grad=None, ws=FAKE, wsb=1 << 20, stream=None)
    a.update(kw)
    return osd.lib().osd_verify_distill(a["target"], a["draft"], a["dtype"], a["B"], a["K"], a["V"],
                                        a["tokens"], a["dlen"], a["ua"], a["ur"], a["T"], a["acc"],
                                        a["toks"], a["rmask"], a["mask"], a["kind"], a["beta"], a["loss"],
                                        a["rows"], a["grad"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(target=None), -1), (dict(draft=None), -1), (dict(tokens=None), -1), (dict(ua=None), -1),
    (dict(ur=None), -1), (dict(acc=None), -1), (dict(toks=None), -1), (dict(loss=None), -1),
    (dict(B=0), -1), (dict(K=0), -1), (dict(K=17), -1), (dict(V=0), -1), (dict(dtype=2), -1),
    (dict(V=1 << 20), -2),
    (dict(T=0.0), -1), (dict(T=-1.0), -1), (dict(T=float("nan")), -1), (dict(T=float("inf")), -1),
    (dict(kind=3), -1), (dict(beta=1.01), -1), (dict(beta=float("nan")), -1),
    (dict(ws=None), -4), (dict(wsb=64), -4), (dict(ws=ctypes.c_void_p(0x1008)), -4),
])
def test_fused_rejects_bad_arguments(kw, status):
    assert fused(**kw) == status


def test_fused_workspace_covers_both_entry_points():
    L = osd.lib()
    for B, K in [(1, 1), (64, 8), (256, 16)]:
        assert L.osd_verify_distill_workspace_bytes(B, K) >= (L.osd_verify_workspace_bytes(B, K)
                                                             + L.osd_distill_workspace_bytes(B, K))
    assert L.osd_verify_distill_workspace_bytes(4, 17) == 0
    assert L.osd_verify_distill_workspace_bytes(0, 4) == 0


def sample(**kw):
    a = dict(p=FAKE, ps=64, q=FAKE, qs=64, dtype=1, N=4, V=64, T=0.8, beta=0.5, u=FAKE, out=FAKE,
             ws=None, wsb=0, stream=None)
    a.update(kw)
    return osd.lib().osd_sample(a["p"], a["ps"], a["q"], a["qs"], a["dtype"], a["N"], a["V"], a["T"],
                                a["beta"], a["u"], a["out"], a["ws"], a["wsb"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(N=0), -1), (dict(V=0), -1), (dict(dtype=2), -1), (dict(V=1 << 20, ps=1 << 20, qs=1 << 20), -2),
    (dict(T=-1.0), -1), (dict(T=float("nan")), -1), (dict(T=float("inf")), -1),
    (dict(beta=-0.1), -1), (dict(beta=1.5), -1), (dict(beta=float("nan")), -1),
    (dict(T=0.0), -1),                       # argmax of a mixture
    (dict(p=None), -1), (dict(q=None), -1), (dict(u=None), -1), (dict(out=None), -1),
    (dict(ps=63), -1), (dict(qs=10), -1),
    (dict(beta=1.0, p=None), -1), (dict(beta=0.0, q=None), -1),
    (dict(ws=FAKE, wsb=4 * 272 - 1), -4), (dict(ws=FAKE_MISALIGNED, wsb=4 * 272), -4),
])
def test_sample_rejects_bad_arguments(kw, status):
    assert sample(**kw) == status


def test_sample_workspace_size():
    L = osd.lib()
    assert L.osd_sample_workspace_bytes(4) == 4 * 272
    assert L.osd_sample_workspace_bytes(0) == 0


def test_binding_sample_fails_loudly_without_gpu_tensors():
    import torch
    with pytest.raises(ValueError):
        osd.osd_sample(torch.zeros(2, 8), None, 1.0, 1.0, torch.zeros(2))


# Vocabulary-sharded verification (three phases, one call per rank each).


def shard_stats(**kw):
    a = dict(t=FAKE, d=FAKE, dtype=1, B=4, K=3, Vs=64, v0=64, V=256, y=FAKE, kl=None, T=0.8, out=FAKE,
             stream=None)
    a.update(kw)
    return osd.lib().osd_shard_verify_stats(a["t"], a["d"], a["dtype"], a["B"], a["K"], a["Vs"], a["v0"], a["V"],
                                            a["y"], a["kl"], a["T"], a["out"], a["stream"])


def shard_mass(**kw):
    a = dict(t=FAKE, d=FAKE, dtype=1, B=4, K=3, Vs=64, G=4, y=FAKE, kl=None, u=FAKE, T=0.8, stats=FAKE,
             out=FAKE, stream=None)
    a.update(kw)
    return osd.lib().osd_shard_verify_mass(a["t"], a["d"], a["dtype"], a["B"], a["K"], a["Vs"], a["G"], a["y"],
                                           a["kl"], a["u"], a["T"], a["stats"], a["out"], a["stream"])


def shard_draw(**kw):
    a = dict(t=FAKE, d=FAKE, dtype=1, B=4, K=3, Vs=64, v0=64, G=4, g=1, y=FAKE, kl=None, u=FAKE, T=0.8,
             mass=FAKE, acc=FAKE, toks=FAKE, rmask=None, stream=None)
    a.update(kw)
    return osd.lib().osd_shard_verify_draw(a["t"], a["d"], a["dtype"], a["B"], a["K"], a["Vs"], a["v0"], a["G"],
                                           a["g"], a["y"], a["kl"], a["u"], a["T"], a["mass"], a["acc"],
                                           a["toks"], a["rmask"], a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), -1), (dict(K=0), -1), (dict(K=17), -1), (dict(Vs=0), -1), (dict(dtype=5), -1),
    (dict(Vs=(1 << 17) + 8, V=1 << 19, v0=0), -2), (dict(V=(1 << 19) + 64), -2),
    (dict(v0=-1), -1), (dict(v0=200), -1), (dict(V=0), -1),
    (dict(T=-1.0), -1), (dict(T=float("nan")), -1), (dict(T=float("inf")), -1),
    (dict(t=None), -1), (dict(d=None), -1), (dict(y=None), -1), (dict(out=None), -1),
    (dict(out=FAKE_MISALIGNED), -1),  # records must be 8-byte aligned
])
def test_shard_stats_rejects_bad_arguments(kw, status):
    assert shard_stats(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), -1), (dict(K=17), -1), (dict(Vs=(1 << 17) + 8), -2),
    (dict(G=0), -1), (dict(G=65), -1), (dict(T=-0.5), -1),
    (dict(t=None), -1), (dict(d=None), -1), (dict(u=None), -1), (dict(stats=None), -1), (dict(out=None), -1),
    (dict(stats=FAKE_MISALIGNED), -1), (dict(out=FAKE_MISALIGNED), -1),
])
def test_shard_mass_rejects_bad_arguments(kw, status):
    assert shard_mass(**kw) == status


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), -1), (dict(K=17), -1), (dict(Vs=(1 << 17) + 8), -2),
    (dict(G=0), -1), (dict(G=65), -1), (dict(g=-1), -1), (dict(g=4), -1), (dict(v0=-3), -1),
    (dict(v0=(1 << 19) - 32), -1), (dict(T=float("nan")), -1),
    (dict(t=None), -1), (dict(d=None), -1), (dict(u=None), -1), (dict(mass=None), -1), (dict(acc=None), -1),
    (dict(toks=None), -1), (dict(mass=FAKE_MISALIGNED), -1),
])
def test_shard_draw_rejects_bad_arguments(kw, status):
    assert shard_draw(**kw) == status


def test_binding_shard_fails_loudly_without_gpu_tensors():
    import torch
    with pytest.raises(ValueError):
        osd.osd_shard_verify_stats(torch.zeros(2, 3, 8), torch.zeros(2, 2, 8), torch.zeros(2, 2, dtype=torch.int32),
                                   1.0, 0, 8)


def test_shard_record_layout_matches_header(tmp_path):
    """The record sizes and field offsets the binding and the tests assume are
    the ones a C compiler gives the structs declared in include/osd.h."""
    import subprocess
    src = tmp_path / "layout.c"
    src.write_text(
        '#include <stddef.h>\n#include <stdio.h>\n#include "osd.h"\n'
        "int main(void) {\n"
        '  printf("%zu %zu %zu %zu %zu %zu %zu %zu\\n", sizeof(osd_shard_row_stats), sizeof(osd_shard_mass),\n'
        "         offsetof(osd_shard_row_stats, k_target), offsetof(osd_shard_row_stats, argmax),\n"
        "         offsetof(osd_shard_row_stats, flags), offsetof(osd_shard_mass, s_target),\n"
        "         offsetof(osd_shard_mass, accepted), offsetof(osd_shard_mass, token));\n"
        "  return 0;\n}\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split()]
    assert got == [binding.SHARD_ROW_STATS_BYTES, binding.SHARD_MASS_BYTES, 16, 32, 36, 16, 40, 44]


def test_verify_noalloc_rejects_before_touching_the_gpu():
    """The allocation-free verification checks its arguments, then its size
    against the library's scratch, before any HIP call."""
    L = osd.lib()
    args = lambda B, K, **kw: (kw.get("t", FAKE), FAKE, 1, B, K, 64, FAKE, None, FAKE, FAKE,
                               kw.get("T", 1.0), FAKE, FAKE, None, None)
    assert L.osd_verify_noalloc(*args(2, 3, t=None)) == -1
    assert L.osd_verify_noalloc(*args(2, 17)) == -1
    assert L.osd_verify_noalloc(*args(2, 3, T=float("nan"))) == -1
    big = 4096  # 4096 x 9 rows need more than OSD_VERIFY_NOALLOC_SCRATCH_BYTES
    assert L.osd_verify_workspace_bytes(big, 8) > binding.OSD_VERIFY_NOALLOC_SCRATCH_BYTES
    assert L.osd_verify_noalloc(*args(big, 8)) == binding.OSD_ERR_SCRATCH
    assert L.osd_verify_workspace_bytes(1024, 8) <= binding.OSD_VERIFY_NOALLOC_SCRATCH_BYTES


def test_verify_tree_rejects_bad_arguments():
    """Host checks of osd_verify_tree (nothing is launched)."""
    L = osd.lib()
    def call(**kw):
        a = dict(t=FAKE, d=FAKE, dtype=1, B=2, N=5, V=64, par=FAKE, tok=FAKE, ua=FAKE, ur=FAKE, T=1.0,
                 acc=FAKE, toks=FAKE, nodes=None, ws=FAKE, wsb=1 << 20)
        a.update(kw)
        return L.osd_verify_tree(a["t"], a["d"], a["dtype"], a["B"], a["N"], a["V"], a["par"], a["tok"], a["ua"],
                                 a["ur"], a["T"], a["acc"], a["toks"], a["nodes"], a["ws"], a["wsb"], None)
    assert call(t=None) == -1 and call(par=None) == -1 and call(tok=None) == -1 and call(acc=None) == -1
    assert call(d=None) == -1 and call(ua=None) == -1 and call(ur=None) == -1
    assert call(N=0) == -1 and call(N=65) == -1 and call(B=0) == -1 and call(V=0) == -1 and call(dtype=3) == -1
    assert call(V=32769) == -2 and call(dtype=0, V=16385) == -2
    assert call(T=-1.0) == -1 and call(T=float("nan")) == -1
    assert call(ws=None) == -4 and call(wsb=8) == -4
    assert L.osd_verify_tree_workspace_bytes(4, 64) >= 4 * (4 + 4 * 64)
    assert L.osd_verify_tree_workspace_bytes(4, 65) == 0 and L.osd_verify_tree_workspace_bytes(0, 4) == 0


def test_sharded_slices_beyond_the_register_tile_are_unsupported():
    """A rank's slice is held in registers: up to 65536 bf16 / 32768 fp32."""
    L = osd.lib()
    args = lambda Vs, dt: (FAKE, FAKE, dt, 2, 3, Vs, 0, 2 * Vs, FAKE, None, ctypes.c_float(1.0), FAKE, None)
    assert L.osd_shard_verify_stats(*args(65537, 1)) == -2
    assert L.osd_shard_verify_stats(*args(32769, 0)) == -2
