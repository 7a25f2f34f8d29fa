"""The library's calls captured in a HIP graph and replayed.

The library allocates nothing and clears its own workspace with its kernels
(no memset nodes), so a captured step can be replayed.  Each replay is
checked bit for bit against the eager result of the same call, with other
eager calls on other inputs (sharing the workspaces) and synchronisations
between the replays.
"""
import ctypes

import numpy as np
import pytest

from paper_2310_07177_amd import binding, synth

pytestmark = pytest.mark.gpu


def _dev(a, dev):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


def test_graph_replays_match_eager():
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    L = binding.lib()
    B, K, V = 16, 5, 8192
    sets = []
    for seed in (3, 4):
        x = synth.verify_inputs(B, K, V, "bf16", T=0.8, seed=seed, target_std=2.5, draft_noise=1.0)
        s = {k: _dev(x[k], dev) for k in ("target", "draft", "u_accept", "u_resample")}
        s["tokens"] = _dev(x["tokens"].astype(np.int32), dev)
        s["mask"] = torch.ones(B, K, dtype=torch.uint8, device=dev)
        s["acc"] = torch.empty(B, dtype=torch.int32, device=dev)
        s["toks"] = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
        s["rmask"] = torch.empty(B, K, dtype=torch.uint8, device=dev)
        s["loss"] = torch.empty(2, dtype=torch.float32, device=dev)
        s["rows"] = torch.empty(B, K, dtype=torch.float32, device=dev)
        s["grad"] = torch.empty(B, K, V, dtype=torch.bfloat16, device=dev)
        sets.append(s)
    stream = torch.cuda.Stream(dev)
    stream.wait_stream(torch.cuda.current_stream(dev))
    hs = ctypes.c_void_p(stream.cuda_stream)
    vws = torch.zeros(L.osd_verify_workspace_bytes(B, K), dtype=torch.uint8, device=dev)
    dws = torch.zeros(L.osd_distill_workspace_bytes(B, K), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    P = lambda t: ctypes.c_void_p(t.data_ptr())

    def step(s, T):
        st = L.osd_verify(P(s["target"]), P(s["draft"]), binding.OSD_BF16, B, K, V, P(s["tokens"]), None,
                          P(s["u_accept"]) if T > 0 else None, P(s["u_resample"]) if T > 0 else None,
                          ctypes.c_float(T), P(s["acc"]), P(s["toks"]), P(s["rmask"]), P(vws), vws.numel(), hs)
        assert st == 0
        st = L.osd_distill_loss_grad(P(s["target"]), (K + 1) * V, P(s["draft"]), K * V, binding.OSD_BF16,
                                     B, K, V, P(s["mask"]), binding.OSD_JSD, ctypes.c_float(0.5),
                                     ctypes.c_float(0.8), P(s["loss"]), P(s["rows"]), P(s["grad"]),
                                     P(dws), dws.numel(), hs)
        assert st == 0

    def outputs(s):
        return [s[k].clone() for k in ("acc", "toks", "rmask", "loss", "rows", "grad")]

    for T in (0.8, 0.0):
        a, b = sets
        with torch.cuda.stream(stream):
            step(a, T)
        torch.cuda.synchronize()
        eager = outputs(a)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            step(a, T)
        for rep in range(3):
            for k in ("acc", "toks", "rmask", "loss", "rows", "grad"):
                a[k].zero_()
            torch.cuda.synchronize()
            with torch.cuda.stream(stream):
                g.replay()
            torch.cuda.synchronize()
            for e, o in zip(eager, outputs(a)):
                assert torch.equal(e, o), f"T={T} replay {rep}"
            with torch.cuda.stream(stream):  # eager work on other inputs between replays
                step(b, T)
            torch.cuda.synchronize()
        assert int(vws.count_nonzero()) == 0 and int(dws.count_nonzero()) == 0


def test_graph_replays_match_eager_fused():
    """The same for the fused entry point (osd_verify_distill)."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    L = binding.lib()
    B, K, V = 16, 5, 8192
    sets = []
    for seed in (5, 6):
        x = synth.verify_inputs(B, K, V, "bf16", T=0.8, seed=seed, target_std=2.5, draft_noise=1.0)
        s = {k: _dev(x[k], dev) for k in ("target", "draft", "u_accept", "u_resample")}
        s["tokens"] = _dev(x["tokens"].astype(np.int32), dev)
        s["mask"] = _dev((np.random.default_rng(seed).random((B, K)) < 0.7).astype(np.uint8), dev)
        s["acc"] = torch.empty(B, dtype=torch.int32, device=dev)
        s["toks"] = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
        s["rmask"] = torch.empty(B, K, dtype=torch.uint8, device=dev)
        s["loss"] = torch.empty(2, dtype=torch.float32, device=dev)
        s["rows"] = torch.empty(B, K, dtype=torch.float32, device=dev)
        s["grad"] = torch.empty(B, K, V, dtype=torch.bfloat16, device=dev)
        sets.append(s)
    stream = torch.cuda.Stream(dev)
    stream.wait_stream(torch.cuda.current_stream(dev))
    hs = ctypes.c_void_p(stream.cuda_stream)
    ws = torch.zeros(L.osd_verify_distill_workspace_bytes(B, K), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    P = lambda t: ctypes.c_void_p(t.data_ptr())

    def step(s):
        st = L.osd_verify_distill(P(s["target"]), P(s["draft"]), binding.OSD_BF16, B, K, V, P(s["tokens"]), None,
                                  P(s["u_accept"]), P(s["u_resample"]), ctypes.c_float(0.8), P(s["acc"]),
                                  P(s["toks"]), P(s["rmask"]), P(s["mask"]), binding.OSD_JSD, ctypes.c_float(0.5),
                                  P(s["loss"]), P(s["rows"]), P(s["grad"]), P(ws), ws.numel(), hs)
        assert st == 0

    def outputs(s):
        return [s[k].clone() for k in ("acc", "toks", "rmask", "loss", "rows", "grad")]

    a, b = sets
    with torch.cuda.stream(stream):
        step(a)
    torch.cuda.synchronize()
    eager = outputs(a)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        step(a)
    for rep in range(3):
        for k in ("acc", "toks", "rmask", "loss", "rows", "grad"):
            a[k].zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        for e, o in zip(eager, outputs(a)):
            assert torch.equal(e, o), f"replay {rep}"
        with torch.cuda.stream(stream):
            step(b)
        torch.cuda.synchronize()
    assert int(ws.count_nonzero()) == 0


def test_concurrent_calls_on_two_streams():
    """Fused calls on two streams at once, each with its own workspace (the
    way bench.py keeps two steps in flight): every output equals that of the
    same call made alone, and both workspaces end zeroed."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    L = binding.lib()
    B, K, V = 64, 8, 32128
    sets = []
    for seed in (7, 8, 9, 10):
        x = synth.verify_inputs(B, K, V, "bf16", T=0.7, seed=seed, target_std=2.5, draft_scale=0.7,
                                draft_noise=1.5)
        s = {k: _dev(x[k], dev) for k in ("target", "draft", "u_accept", "u_resample")}
        s["tokens"] = _dev(x["tokens"].astype(np.int32), dev)
        s["acc"] = torch.empty(B, dtype=torch.int32, device=dev)
        s["toks"] = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
        s["rmask"] = torch.empty(B, K, dtype=torch.uint8, device=dev)
        s["loss"] = torch.empty(2, dtype=torch.float32, device=dev)
        s["rows"] = torch.empty(B, K, dtype=torch.float32, device=dev)
        s["grad"] = torch.empty(B, K, V, dtype=torch.bfloat16, device=dev)
        sets.append(s)
    streams = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]
    wss = [torch.zeros(L.osd_verify_distill_workspace_bytes(B, K), dtype=torch.uint8, device=dev)
           for _ in streams]
    torch.cuda.synchronize()
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    keys = ("acc", "toks", "rmask", "loss", "rows", "grad")

    def call(s, j):
        st = L.osd_verify_distill(P(s["target"]), P(s["draft"]), binding.OSD_BF16, B, K, V, P(s["tokens"]),
                                  None, P(s["u_accept"]), P(s["u_resample"]), ctypes.c_float(0.7), P(s["acc"]),
                                  P(s["toks"]), P(s["rmask"]), None, binding.OSD_JSD, ctypes.c_float(0.5),
                                  P(s["loss"]), P(s["rows"]), P(s["grad"]), P(wss[j]), wss[j].numel(),
                                  ctypes.c_void_p(streams[j].cuda_stream))
        assert st == 0

    alone = []
    for s in sets:
        call(s, 0)
        torch.cuda.synchronize()
        alone.append([s[k].clone() for k in keys])
    for rep in range(3):
        for s in sets:
            for k in keys:
                s[k].zero_()
        torch.cuda.synchronize()
        for i, s in enumerate(sets):  # sets 0, 2 on stream 0; 1, 3 on stream 1
            call(s, i % 2)
        torch.cuda.synchronize()
        for i, s in enumerate(sets):
            for k, want in zip(keys, alone[i]):
                assert torch.equal(s[k], want), f"rep {rep} set {i} {k}"
    assert all(int(w.count_nonzero()) == 0 for w in wss)


def test_graph_replays_match_eager_sharded():
    """The three phases of the vocabulary-sharded verification for 4 ranks
    (12 calls, the exchanges being the shared record arrays) captured once
    and replayed; each replay equals the eager result."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    dev = torch.device("cuda:0")
    L = binding.lib()
    B, K, V, G = 16, 5, 8192, 4
    Vs = V // G
    x = synth.verify_inputs(B, K, V, "bf16", T=0.8, seed=7, target_std=2.5, draft_noise=1.0, ragged=True)
    t, d = _dev(x["target"], dev), _dev(x["draft"], dev)
    tg = [t[:, :, g * Vs:(g + 1) * Vs].contiguous() for g in range(G)]
    dg = [d[:, :, g * Vs:(g + 1) * Vs].contiguous() for g in range(G)]
    y, kl = _dev(x["tokens"].astype(np.int32), dev), _dev(x["draft_len"], dev)
    ua, ur = _dev(x["u_accept"], dev), _dev(x["u_resample"], dev)
    stats = torch.zeros(G, B, K + 1, binding.SHARD_ROW_STATS_BYTES, dtype=torch.uint8, device=dev)
    mass = torch.zeros(G, B, binding.SHARD_MASS_BYTES, dtype=torch.uint8, device=dev)
    acc = torch.empty(G, B, dtype=torch.int32, device=dev)
    toks = torch.empty(G, B, K + 1, dtype=torch.int32, device=dev)
    rm = torch.empty(G, B, K, dtype=torch.uint8, device=dev)
    stream = torch.cuda.Stream(dev)
    stream.wait_stream(torch.cuda.current_stream(dev))
    hs = ctypes.c_void_p(stream.cuda_stream)
    torch.cuda.synchronize()
    P = lambda a: ctypes.c_void_p(a.data_ptr())
    cT = ctypes.c_float(x["T"])

    def step():
        for g in range(G):
            assert L.osd_shard_verify_stats(P(tg[g]), P(dg[g]), binding.OSD_BF16, B, K, Vs, g * Vs, V, P(y), P(kl),
                                            cT, P(stats[g]), hs) == 0
        for g in range(G):
            assert L.osd_shard_verify_mass(P(tg[g]), P(dg[g]), binding.OSD_BF16, B, K, Vs, G, P(y), P(kl), P(ua),
                                           cT, P(stats), P(mass[g]), hs) == 0
        for g in range(G):
            assert L.osd_shard_verify_draw(P(tg[g]), P(dg[g]), binding.OSD_BF16, B, K, Vs, g * Vs, G, g, P(y), P(kl),
                                           P(ur), cT, P(mass), P(acc[g]), P(toks[g]), P(rm[g]), hs) == 0

    with torch.cuda.stream(stream):
        step()
    torch.cuda.synchronize()
    eager = [a.clone() for a in (stats, mass, acc, toks, rm)]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        step()
    for rep in range(3):
        for a in (stats, mass, acc, toks, rm):
            a.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            g.replay()
        torch.cuda.synchronize()
        for e, o in zip(eager, (stats, mass, acc, toks, rm)):
            assert torch.equal(e, o), f"replay {rep}"
