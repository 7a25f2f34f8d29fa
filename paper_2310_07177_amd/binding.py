"""Thin Python binding of libosd (include/osd.h).

The functions carry the C ABI's names and only marshal arguments: torch
supplies device memory and the current stream, every computation happens in
the HIP kernels behind the C ABI.  There is no fallback: if the library or a
GPU is missing, the call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libosd.so")

OSD_OK, OSD_ERR_INVALID_ARG, OSD_ERR_UNSUPPORTED, OSD_ERR_DEVICE, OSD_ERR_WORKSPACE, OSD_ERR_SCRATCH = 0, -1, -2, -3, -4, -5
OSD_VERIFY_NOALLOC_SCRATCH_BYTES = 4 << 20
OSD_F32, OSD_BF16 = 0, 1
OSD_FKL, OSD_RKL, OSD_JSD = 0, 1, 2
OSD_MAX_K = 16
OSD_MAX_SHARDS = 64
OSD_MAX_TREE_NODES = 64
# Byte sizes of the sharded verification's records (osd_shard_row_stats,
# osd_shard_mass in include/osd.h); the binding keeps them as uint8 tensors.
SHARD_ROW_STATS_BYTES = 40
SHARD_MASS_BYTES = 48
KINDS = {"fkl": OSD_FKL, "rkl": OSD_RKL, "jsd": OSD_JSD}

EXPORTS = ("osd_max_vocab", "osd_status_string", "osd_verify_workspace_bytes", "osd_verify", "osd_verify_noalloc",
           "osd_distill_workspace_bytes", "osd_distill_loss_grad", "osd_verify_distill_workspace_bytes",
           "osd_verify_distill", "osd_verify_distill_rejected", "osd_verify_tree_workspace_bytes", "osd_verify_tree",
           "osd_sample_workspace_bytes", "osd_sample", "osd_shard_verify_stats", "osd_shard_verify_mass",
           "osd_shard_verify_draw")

_lib = None
_lock = threading.Lock()


class OsdError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed: {lib().osd_status_string(status).decode()}")


def lib():
    """Load libosd.so (built in-tree by paper_2310_07177_amd.build)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                                   "`python -m paper_2310_07177_amd.build`")
            L = ctypes.CDLL(LIB_PATH)
            vp, i32, i64, f32, sz = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                     ctypes.c_float, ctypes.c_size_t)
            L.osd_max_vocab.restype = i32
            L.osd_max_vocab.argtypes = [i32]
            L.osd_status_string.restype = ctypes.c_char_p
            L.osd_status_string.argtypes = [i32]
            L.osd_verify_workspace_bytes.restype = sz
            L.osd_verify_workspace_bytes.argtypes = [i32, i32]
            L.osd_verify.restype = i32
            L.osd_verify.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32,
                                     vp, vp, vp, vp, sz, vp]
            L.osd_verify_noalloc.restype = i32
            L.osd_verify_noalloc.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp, vp, vp]
            L.osd_distill_workspace_bytes.restype = sz
            L.osd_distill_workspace_bytes.argtypes = [i32, i32]
            L.osd_distill_loss_grad.restype = i32
            L.osd_distill_loss_grad.argtypes = [vp, i64, vp, i64, i32, i32, i32, i32, vp, i32,
                                                f32, f32, vp, vp, vp, vp, sz, vp]
            L.osd_verify_distill_workspace_bytes.restype = sz
            L.osd_verify_distill_workspace_bytes.argtypes = [i32, i32]
            L.osd_verify_distill.restype = i32
            L.osd_verify_distill.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp, vp,
                                             vp, i32, f32, vp, vp, vp, vp, sz, vp]
            L.osd_verify_distill_rejected.restype = i32
            L.osd_verify_distill_rejected.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp,
                                                      vp, i32, f32, vp, vp, vp, vp, sz, vp]
            L.osd_verify_tree_workspace_bytes.restype = sz
            L.osd_verify_tree_workspace_bytes.argtypes = [i32, i32]
            L.osd_verify_tree.restype = i32
            L.osd_verify_tree.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp, vp, vp, sz, vp]
            L.osd_sample.restype = i32
            L.osd_sample_workspace_bytes.restype = sz
            L.osd_sample_workspace_bytes.argtypes = [i32]
            L.osd_sample.argtypes = [vp, i64, vp, i64, i32, i32, i32, f32, f32, vp, vp, vp, sz, vp]
            L.osd_shard_verify_stats.restype = i32
            L.osd_shard_verify_stats.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, vp, vp, f32, vp, vp]
            L.osd_shard_verify_mass.restype = i32
            L.osd_shard_verify_mass.argtypes = [vp, vp, i32, i32, i32, i32, i32, vp, vp, vp, f32, vp, vp, vp]
            L.osd_shard_verify_draw.restype = i32
            L.osd_shard_verify_draw.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, i32, vp, vp, vp, f32,
                                                vp, vp, vp, vp, vp]
            _lib = L
    return _lib


def _torch():
    import torch
    return torch


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t):
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return OSD_BF16
    if t.dtype == torch.float32:
        return OSD_F32
    raise TypeError(f"logits must be bfloat16 or float32, got {t.dtype}")


def _check_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("every tensor argument must live on the GPU")


def _stream_handle(device):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


# Zero-initialised workspaces, one per (device, stream, kind, size): the kernels
# leave them zeroed, so they are reused across calls on the same stream.
_workspaces = {}


def workspace(kind, nbytes, device):
    torch = _torch()
    stream = torch.cuda.current_stream(device).cuda_stream
    key = (str(device), stream, kind)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        ws = torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device)
        _workspaces[key] = ws
    return ws


def osd_max_vocab(dtype_code: int) -> int:
    return lib().osd_max_vocab(dtype_code)


def osd_verify(target_logits, draft_logits, draft_tokens, u_accept, u_resample, temperature,
               draft_len=None, out=None):
    """Speculative-sampling verification through the C ABI.

    target_logits [B, K+1, V], draft_logits [B, K, V] (bf16 or fp32, on the
    GPU; draft may be None for temperature 0), draft_tokens [B, K] int32,
    u_accept [B, K] / u_resample [B] float32 (None for temperature 0),
    draft_len [B] int32 or None.  Returns (accepted_len [B], out_tokens
    [B, K+1], reject_mask [B, K]) as new (or the given `out`) GPU tensors."""
    torch = _torch()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_cuda(target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len)
    dev = target_logits.device
    for t in (target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if draft_tokens.dtype != torch.int32 or (draft_len is not None and draft_len.dtype != torch.int32):
        raise TypeError("draft_tokens and draft_len must be int32")
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, K + 1, dtype=torch.int32, device=dev),
               torch.empty(B, K, dtype=torch.uint8, device=dev))
    acc, toks, rmask = out
    L = lib()
    nbytes = L.osd_verify_workspace_bytes(B, K)
    ws = workspace("verify", nbytes, dev)
    st = L.osd_verify(_ptr(target_logits), _ptr(draft_logits), _dtype_code(target_logits), B, K, V,
                      _ptr(draft_tokens), _ptr(draft_len), _ptr(u_accept), _ptr(u_resample),
                      float(temperature), _ptr(acc), _ptr(toks), _ptr(rmask), _ptr(ws),
                      ws.numel(), _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_verify", st)
    return acc, toks, rmask


def osd_verify_noalloc(target_logits, draft_logits, draft_tokens, u_accept, u_resample, temperature,
                       draft_len=None, out=None):
    """osd_verify through the allocation-free entry point: no workspace, the
    library's per-GPU scratch array instead (calls that overlap on one GPU
    race).  Arguments and results as osd_verify; the outputs must be given
    (`out`) by a caller that cannot allocate."""
    torch = _torch()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_cuda(target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len)
    dev = target_logits.device
    for t in (target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if draft_tokens.dtype != torch.int32 or (draft_len is not None and draft_len.dtype != torch.int32):
        raise TypeError("draft_tokens and draft_len must be int32")
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, K + 1, dtype=torch.int32, device=dev),
               torch.empty(B, K, dtype=torch.uint8, device=dev))
    acc, toks, rmask = out
    st = lib().osd_verify_noalloc(_ptr(target_logits), _ptr(draft_logits), _dtype_code(target_logits), B, K, V,
                                  _ptr(draft_tokens), _ptr(draft_len), _ptr(u_accept), _ptr(u_resample),
                                  float(temperature), _ptr(acc), _ptr(toks), _ptr(rmask), _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_verify_noalloc", st)
    return acc, toks, rmask


def osd_distill_loss_grad(teacher_logits, student_logits, kind, beta=0.5, tau=1.0, mask=None,
                          B=None, K=None, teacher_batch_stride=None, student_batch_stride=None,
                          grad=True, row_loss=True, out=None):
    """Masked distillation divergence and gradient through the C ABI.

    By default teacher and student are [B, K, V]; pass B, K and explicit
    batch strides (elements) to distil the first K rows of a [B, K+1, V]
    target.  Returns (loss [2] fp32 = {mean, sum}, row_loss [B, K] fp32 or
    None, grad [B, K, V] or None)."""
    torch = _torch()
    _check_cuda(teacher_logits, student_logits, mask)
    dev = student_logits.device
    V = student_logits.shape[-1]
    if B is None:
        B, K = student_logits.shape[0], student_logits.shape[1]
    if teacher_batch_stride is None:
        teacher_batch_stride = teacher_logits.stride(0)
    if student_batch_stride is None:
        student_batch_stride = student_logits.stride(0)
    if teacher_logits.dtype != student_logits.dtype:
        raise TypeError("teacher and student logits must share a dtype")
    if mask is not None and (mask.dtype != torch.uint8 or not mask.is_contiguous()):
        raise TypeError("mask must be a contiguous uint8 tensor")
    kind_code = KINDS[kind] if isinstance(kind, str) else int(kind)
    if out is None:
        out = (torch.empty(2, dtype=torch.float32, device=dev),
               torch.empty(B, K, dtype=torch.float32, device=dev) if row_loss else None,
               torch.empty(B, K, V, dtype=student_logits.dtype, device=dev) if grad else None)
    loss, rows, g = out
    L = lib()
    nbytes = L.osd_distill_workspace_bytes(B, K)
    ws = workspace("distill", nbytes, dev)
    st = L.osd_distill_loss_grad(_ptr(teacher_logits), int(teacher_batch_stride),
                                 _ptr(student_logits), int(student_batch_stride),
                                 _dtype_code(student_logits), B, K, V, _ptr(mask), kind_code,
                                 float(beta), float(tau), _ptr(loss), _ptr(rows), _ptr(g),
                                 _ptr(ws), ws.numel(), _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_distill_loss_grad", st)
    return loss, rows, g


def osd_verify_distill(target_logits, draft_logits, draft_tokens, u_accept, u_resample, temperature,
                       kind, beta=0.5, distill_mask=None, draft_len=None, grad=True, row_loss=True):
    """Verification and distillation of one step in one pass through the C
    ABI: the results of osd_verify(...) and of osd_distill_loss_grad on the
    first K target rows and the draft rows at tau = temperature.

    Returns (accepted_len [B], out_tokens [B, K+1], reject_mask [B, K],
    loss [2], row_loss [B, K] or None, grad [B, K, V] or None)."""
    torch = _torch()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_cuda(target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len, distill_mask)
    dev = target_logits.device
    for t in (target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len, distill_mask):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if draft_tokens.dtype != torch.int32 or (draft_len is not None and draft_len.dtype != torch.int32):
        raise TypeError("draft_tokens and draft_len must be int32")
    if target_logits.dtype != draft_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    if distill_mask is not None and distill_mask.dtype != torch.uint8:
        raise TypeError("distill_mask must be uint8")
    kind_code = KINDS[kind] if isinstance(kind, str) else int(kind)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    toks = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
    rmask = torch.empty(B, K, dtype=torch.uint8, device=dev)
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    rows = torch.empty(B, K, dtype=torch.float32, device=dev) if row_loss else None
    g = torch.empty(B, K, V, dtype=draft_logits.dtype, device=dev) if grad else None
    L = lib()
    ws = workspace("verify_distill", L.osd_verify_distill_workspace_bytes(B, K), dev)
    st = L.osd_verify_distill(_ptr(target_logits), _ptr(draft_logits), _dtype_code(target_logits), B, K, V,
                              _ptr(draft_tokens), _ptr(draft_len), _ptr(u_accept), _ptr(u_resample),
                              float(temperature), _ptr(acc), _ptr(toks), _ptr(rmask), _ptr(distill_mask),
                              kind_code, float(beta), _ptr(loss), _ptr(rows), _ptr(g), _ptr(ws), ws.numel(),
                              _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_verify_distill", st)
    return acc, toks, rmask, loss, rows, g


def osd_verify_distill_rejected(target_logits, draft_logits, draft_tokens, u_accept, u_resample, temperature,
                                kind, beta=0.5, draft_len=None, grad=True, row_loss=True):
    """Verification and distillation of the row at each sequence's first
    rejection (the error index), in one pass through the C ABI: the results
    of osd_verify(...) and of osd_distill_loss_grad with mask = reject_mask
    at tau = temperature.  Returns what osd_verify_distill returns."""
    torch = _torch()
    B, K1, V = target_logits.shape
    K = K1 - 1
    _check_cuda(target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len)
    dev = target_logits.device
    for t in (target_logits, draft_logits, draft_tokens, u_accept, u_resample, draft_len):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if draft_tokens.dtype != torch.int32 or (draft_len is not None and draft_len.dtype != torch.int32):
        raise TypeError("draft_tokens and draft_len must be int32")
    if target_logits.dtype != draft_logits.dtype:
        raise TypeError("target and draft logits must share a dtype")
    kind_code = KINDS[kind] if isinstance(kind, str) else int(kind)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    toks = torch.empty(B, K + 1, dtype=torch.int32, device=dev)
    rmask = torch.empty(B, K, dtype=torch.uint8, device=dev)
    loss = torch.empty(2, dtype=torch.float32, device=dev)
    rows = torch.empty(B, K, dtype=torch.float32, device=dev) if row_loss else None
    g = torch.empty(B, K, V, dtype=draft_logits.dtype, device=dev) if grad else None
    L = lib()
    ws = workspace("verify_distill", L.osd_verify_distill_workspace_bytes(B, K), dev)
    st = L.osd_verify_distill_rejected(_ptr(target_logits), _ptr(draft_logits), _dtype_code(target_logits), B, K,
                                       V, _ptr(draft_tokens), _ptr(draft_len), _ptr(u_accept), _ptr(u_resample),
                                       float(temperature), _ptr(acc), _ptr(toks), _ptr(rmask), kind_code,
                                       float(beta), _ptr(loss), _ptr(rows), _ptr(g), _ptr(ws), ws.numel(),
                                       _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_verify_distill_rejected", st)
    return acc, toks, rmask, loss, rows, g


def osd_verify_tree(target_logits, draft_logits, parent, node_tokens, u_accept, u_resample, temperature):
    """Multi-candidate (tree) verification through the C ABI.  target_logits,
    draft_logits [B, N, V] (draft may be None at temperature 0), parent and
    node_tokens [B, N] int32, u_accept [B, N] and u_resample [B] float32 (None
    at temperature 0).  Returns (accepted_len [B], out_tokens [B, N],
    path_nodes [B, N])."""
    torch = _torch()
    B, N, V = target_logits.shape
    _check_cuda(target_logits, draft_logits, parent, node_tokens, u_accept, u_resample)
    dev = target_logits.device
    for t in (target_logits, draft_logits, parent, node_tokens, u_accept, u_resample):
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if parent.dtype != torch.int32 or node_tokens.dtype != torch.int32:
        raise TypeError("parent and node_tokens must be int32")
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    toks = torch.empty(B, N, dtype=torch.int32, device=dev)
    nodes = torch.empty(B, N, dtype=torch.int32, device=dev)
    L = lib()
    ws = workspace("verify_tree", L.osd_verify_tree_workspace_bytes(B, N), dev)
    st = L.osd_verify_tree(_ptr(target_logits), _ptr(draft_logits), _dtype_code(target_logits), B, N, V,
                           _ptr(parent), _ptr(node_tokens), _ptr(u_accept), _ptr(u_resample), float(temperature),
                           _ptr(acc), _ptr(toks), _ptr(nodes), _ptr(ws), ws.numel(), _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_verify_tree", st)
    return acc, toks, nodes


def osd_sample(p_logits, q_logits, temperature, beta, u=None, out=None):
    """Token sampling through the C ABI: pi = beta softmax(p/T) +
    (1 - beta) softmax(q/T) per row, inverse CDF with u (argmax at T == 0).

    p_logits, q_logits: [N, V] bf16 or fp32 GPU tensors whose rows are
    contiguous (a row stride other than V is passed through, e.g. a slice
    [:, i, :] of a [B, K+1, V] tensor); either may be None when its weight is
    0.  u: [N] float32 (None at T == 0).  Returns out_tokens [N] int32."""
    torch = _torch()
    ref = p_logits if p_logits is not None else q_logits
    if ref is None:
        raise ValueError("p_logits or q_logits is needed")
    _check_cuda(p_logits, q_logits, u)
    for t in (p_logits, q_logits):
        if t is not None and (t.dim() != 2 or t.stride(1) != 1 or t.dtype != ref.dtype or t.shape != ref.shape):
            raise ValueError("logit rows must be [N, V] views of one dtype with contiguous rows")
    if u is not None and (u.dtype != torch.float32 or not u.is_contiguous()):
        raise TypeError("u must be a contiguous float32 tensor")
    N, V = ref.shape
    if out is None:
        out = torch.empty(N, dtype=torch.int32, device=ref.device)
    stride = lambda t: 0 if t is None else (t.stride(0) if N > 1 else V)
    L = lib()
    ws = workspace("sample", L.osd_sample_workspace_bytes(N), ref.device)
    st = L.osd_sample(_ptr(p_logits), stride(p_logits), _ptr(q_logits), stride(q_logits),
                      _dtype_code(ref), N, V, float(temperature), float(beta), _ptr(u), _ptr(out),
                      _ptr(ws), ws.numel(), _stream_handle(ref.device))
    if st != OSD_OK:
        raise OsdError("osd_sample", st)
    return out


def _shard_args(target_shard, draft_shard, draft_tokens, draft_len, temperature, *more):
    torch = _torch()
    _check_cuda(target_shard, draft_shard, draft_tokens, draft_len, *more)
    for t in (target_shard, draft_shard, draft_tokens, draft_len) + more:
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor arguments must be contiguous")
    if draft_tokens.dtype != torch.int32 or (draft_len is not None and draft_len.dtype != torch.int32):
        raise TypeError("draft_tokens and draft_len must be int32")
    if temperature != 0 and draft_shard is not None and draft_shard.dtype != target_shard.dtype:
        raise TypeError("target and draft logits must share a dtype")
    B, K1, Vs = target_shard.shape
    return B, K1 - 1, Vs


def osd_shard_verify_stats(target_shard, draft_shard, draft_tokens, temperature, v_begin, V, draft_len=None,
                           out=None):
    """Phase 1 of vocabulary-sharded verification on this rank's slice
    (target_shard [B, K+1, V_g], draft_shard [B, K, V_g], columns
    v_begin .. v_begin+V_g-1 of a V-token vocabulary).  Returns the
    osd_shard_row_stats records as a uint8 tensor [B, K+1, 40]."""
    torch = _torch()
    B, K, Vs = _shard_args(target_shard, draft_shard, draft_tokens, draft_len, temperature)
    if out is None:
        out = torch.empty(B, K + 1, SHARD_ROW_STATS_BYTES, dtype=torch.uint8, device=target_shard.device)
    st = lib().osd_shard_verify_stats(_ptr(target_shard), _ptr(draft_shard), _dtype_code(target_shard), B, K, Vs,
                                      int(v_begin), int(V), _ptr(draft_tokens), _ptr(draft_len),
                                      float(temperature), _ptr(out), _stream_handle(target_shard.device))
    if st != OSD_OK:
        raise OsdError("osd_shard_verify_stats", st)
    return out


def osd_shard_verify_mass(target_shard, draft_shard, draft_tokens, u_accept, temperature, stats_all,
                          draft_len=None, out=None):
    """Phase 2: stats_all [G, B, K+1, 40] holds the records of every rank in
    rank order (the all-gather of phase 1).  Returns this rank's
    osd_shard_mass records as a uint8 tensor [B, 48]."""
    torch = _torch()
    B, K, Vs = _shard_args(target_shard, draft_shard, draft_tokens, draft_len, temperature, u_accept, stats_all)
    G = stats_all.shape[0]
    if tuple(stats_all.shape) != (G, B, K + 1, SHARD_ROW_STATS_BYTES) or stats_all.dtype != torch.uint8:
        raise ValueError("stats_all must be a uint8 tensor [G, B, K+1, 40]")
    if out is None:
        out = torch.empty(B, SHARD_MASS_BYTES, dtype=torch.uint8, device=target_shard.device)
    st = lib().osd_shard_verify_mass(_ptr(target_shard), _ptr(draft_shard), _dtype_code(target_shard), B, K, Vs,
                                     G, _ptr(draft_tokens), _ptr(draft_len), _ptr(u_accept), float(temperature),
                                     _ptr(stats_all), _ptr(out), _stream_handle(target_shard.device))
    if st != OSD_OK:
        raise OsdError("osd_shard_verify_mass", st)
    return out


def osd_shard_verify_draw(target_shard, draft_shard, draft_tokens, u_resample, temperature, v_begin, shard,
                          mass_all, draft_len=None, out=None):
    """Phase 3: mass_all [G, B, 48] holds every rank's phase-2 records in rank
    order.  Returns (accepted_len [B], out_tokens [B, K+1], reject_mask
    [B, K]); out_tokens carries the extra token only on the rank that drew
    it (-1 on the others), so an all-reduce MAX over the ranks completes it."""
    torch = _torch()
    B, K, Vs = _shard_args(target_shard, draft_shard, draft_tokens, draft_len, temperature, u_resample, mass_all)
    G = mass_all.shape[0]
    if tuple(mass_all.shape) != (G, B, SHARD_MASS_BYTES) or mass_all.dtype != torch.uint8:
        raise ValueError("mass_all must be a uint8 tensor [G, B, 48]")
    dev = target_shard.device
    if out is None:
        out = (torch.empty(B, dtype=torch.int32, device=dev),
               torch.empty(B, K + 1, dtype=torch.int32, device=dev),
               torch.empty(B, K, dtype=torch.uint8, device=dev))
    acc, toks, rmask = out
    st = lib().osd_shard_verify_draw(_ptr(target_shard), _ptr(draft_shard), _dtype_code(target_shard), B, K, Vs,
                                     int(v_begin), G, int(shard), _ptr(draft_tokens), _ptr(draft_len),
                                     _ptr(u_resample), float(temperature), _ptr(mass_all), _ptr(acc), _ptr(toks),
                                     _ptr(rmask), _stream_handle(dev))
    if st != OSD_OK:
        raise OsdError("osd_shard_verify_draw", st)
    return acc, toks, rmask
