"""ctypes front end of the fp64 CPU oracle (test infrastructure only).

Every function takes and returns numpy arrays on the host.  Logit arrays are
float32, float64, or uint16 holding bf16 bit patterns; the dtype is inferred
from the array.  The arithmetic lives in ``osd_ref.cpp``; this module only
marshals arguments.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F32, BF16, F64 = 0, 1, 2
FKL, RKL, JSD = 0, 1, 2
KINDS = {"fkl": FKL, "rkl": RKL, "jsd": JSD}

_lib = None


def lib():
    global _lib
    if _lib is None:
        path = os.environ.get("OSD_REF_LIB")  # a rebuilt copy, for mutation tests
        if path is None:
            path = _build.LIB
            if not os.path.exists(path):
                _build.build()
        L = ctypes.CDLL(path)
        vp, i32, i64, f32, f64 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                  ctypes.c_float, ctypes.c_double)
        L.osd_ref_verify.restype = i32
        L.osd_ref_verify.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp,
                                     f32, vp, vp, vp, vp, vp, vp]
        L.osd_ref_distill_loss_grad.restype = i32
        L.osd_ref_distill_loss_grad.argtypes = [vp, i64, vp, i64, i32, i32, i32,
                                                i32, vp, i32, f64, f64, vp, vp, vp]
        L.osd_ref_verify_tree.restype = i32
        L.osd_ref_verify_tree.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp, vp, vp, vp, vp, vp]
        L.osd_ref_sample.restype = i32
        L.osd_ref_sample.argtypes = [vp, i64, vp, i64, i32, i32, i32, f32, f64, vp, vp, vp]
        L.osd_ref_round_bf16.restype = None
        L.osd_ref_round_bf16.argtypes = [vp, vp, i64]
        L.osd_ref_bf16_midpoint_flags.restype = None
        L.osd_ref_bf16_midpoint_flags.argtypes = [vp, vp, i64, f64]
        _lib = L
    return _lib


def _dtype_code(a):
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float64:
        return F64
    raise TypeError(f"unsupported logit dtype {a.dtype}")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype=None):
    if a is None:
        return None
    return np.ascontiguousarray(a if dtype is None else a.astype(dtype, copy=False))


def verify(target, draft, draft_tokens, u_accept, u_resample, temperature,
           draft_len=None):
    """Oracle verification.  target [B,K+1,V], draft [B,K,V] (may be None when
    temperature == 0).  Returns a dict of numpy arrays: accepted_len [B],
    out_tokens [B,K+1], reject_mask [B,K], margin_accept [B,K] (NaN where no
    test was evaluated), margin_cdf [B], z_fallback [B]."""
    target = _c(target)
    B, K1, V = target.shape
    K = K1 - 1
    draft = _c(draft)
    if draft is not None:
        assert draft.shape == (B, K, V) and draft.dtype == target.dtype
    toks = _c(draft_tokens, np.int32)
    assert toks.shape == (B, K)
    dl = _c(draft_len, np.int32)
    ua = _c(u_accept, np.float32)
    ur = _c(u_resample, np.float32)
    acc = np.empty(B, np.int32)
    out = np.empty((B, K + 1), np.int32)
    rmask = np.empty((B, K), np.uint8)
    ma = np.empty((B, K), np.float64)
    mc = np.empty(B, np.float64)
    zf = np.empty(B, np.int32)
    rc = lib().osd_ref_verify(_ptr(target), _ptr(draft), _dtype_code(target), B, K, V,
                              _ptr(toks), _ptr(dl), _ptr(ua), _ptr(ur),
                              float(temperature), _ptr(acc), _ptr(out), _ptr(rmask),
                              _ptr(ma), _ptr(mc), _ptr(zf))
    if rc != 0:
        raise ValueError(f"osd_ref_verify rejected its arguments (rc={rc})")
    return dict(accepted_len=acc, out_tokens=out, reject_mask=rmask,
                margin_accept=ma, margin_cdf=mc, z_fallback=zf)


def distill(teacher, student, kind, beta=0.5, tau=1.0, mask=None, grad=True,
            teacher_batch_stride=None, student_batch_stride=None, B=None, K=None):
    """Oracle divergence + gradient.  By default teacher and student are
    [B,K,V] contiguous; pass explicit batch strides (elements) with B and K to
    distil the first K rows of a [B,K+1,V] target.  Returns dict with
    loss (mean, sum), row_loss [B,K] and grad [B,K,V] (fp64) if requested."""
    teacher = _c(teacher)
    student = _c(student)
    V = teacher.shape[-1]
    if B is None:
        B, K = student.shape[0], student.shape[1]
    if teacher_batch_stride is None:
        teacher_batch_stride = teacher.shape[1] * V
    if student_batch_stride is None:
        student_batch_stride = student.shape[1] * V
    assert teacher.dtype == student.dtype
    m = _c(mask, np.uint8)
    loss = np.empty(2, np.float64)
    rows = np.empty((B, K), np.float64)
    g = np.empty((B, K, V), np.float64) if grad else None
    kind_code = KINDS[kind] if isinstance(kind, str) else int(kind)
    rc = lib().osd_ref_distill_loss_grad(_ptr(teacher), int(teacher_batch_stride),
                                         _ptr(student), int(student_batch_stride),
                                         _dtype_code(teacher), B, K, V, _ptr(m),
                                         kind_code, float(beta), float(tau),
                                         _ptr(loss), _ptr(rows), _ptr(g))
    if rc != 0:
        raise ValueError(f"osd_ref_distill_loss_grad rejected its arguments (rc={rc})")
    return dict(loss_mean=loss[0], loss_sum=loss[1], row_loss=rows, grad=g)


def verify_tree(target, draft, parent, node_tokens, u_accept, u_resample, temperature):
    """Oracle multi-candidate (tree) verification.  target, draft [B, N, V]
    (draft may be None when temperature == 0), parent and node_tokens [B, N]
    int32, u_accept [B, N], u_resample [B].  Returns a dict: accepted_len [B],
    out_tokens [B, N], path_nodes [B, N], margin_accept [B, N], margin_cdf [B],
    z_fallback [B]."""
    target = _c(target)
    B, N, V = target.shape
    draft = _c(draft)
    if draft is not None:
        assert draft.shape == (B, N, V) and draft.dtype == target.dtype
    par = _c(parent, np.int32)
    tok = _c(node_tokens, np.int32)
    assert par.shape == (B, N) and tok.shape == (B, N)
    ua = _c(u_accept, np.float32)
    ur = _c(u_resample, np.float32)
    acc = np.empty(B, np.int32)
    out = np.empty((B, N), np.int32)
    pn = np.empty((B, N), np.int32)
    ma = np.empty((B, N), np.float64)
    mc = np.empty(B, np.float64)
    zf = np.empty(B, np.int32)
    rc = lib().osd_ref_verify_tree(_ptr(target), _ptr(draft), _dtype_code(target), B, N, V, _ptr(par), _ptr(tok),
                                   _ptr(ua), _ptr(ur), float(temperature), _ptr(acc), _ptr(out), _ptr(pn),
                                   _ptr(ma), _ptr(mc), _ptr(zf))
    if rc != 0:
        raise ValueError(f"osd_ref_verify_tree rejected its arguments (rc={rc})")
    return dict(accepted_len=acc, out_tokens=out, path_nodes=pn, margin_accept=ma, margin_cdf=mc, z_fallback=zf)


def sample(p, q, temperature, beta, u=None):
    """Oracle token sampling.  p and q are [N, V] (either may be None when its
    weight is 0: p needs beta > 0, q needs beta < 1); rows may be views with a
    row stride (the leading axis stride is passed through).  Returns a dict:
    tokens [N] int32 (-1 for an invalid row) and margin [N] (NaN for greedy
    and invalid rows)."""
    def rows(a):
        if a is None:
            return None, 0
        a = np.asarray(a)
        assert a.ndim == 2 and a.strides[1] == a.itemsize, "rows must be contiguous along V"
        return a, (a.strides[0] // a.itemsize if a.shape[0] > 1 else a.shape[1])
    p, ps = rows(p)
    q, qs = rows(q)
    ref = p if p is not None else q
    N, V = ref.shape
    uu = _c(u, np.float32)
    out = np.empty(N, np.int32)
    mg = np.empty(N, np.float64)
    pp = None if p is None else ctypes.c_void_p(p.ctypes.data)
    qp = None if q is None else ctypes.c_void_p(q.ctypes.data)
    rc = lib().osd_ref_sample(pp, int(ps), qp, int(qs), _dtype_code(ref), N, V, float(temperature),
                              float(beta), _ptr(uu), _ptr(out), _ptr(mg))
    if rc != 0:
        raise ValueError(f"osd_ref_sample rejected its arguments (rc={rc})")
    return dict(tokens=out, margin=mg)


def round_bf16(x):
    """fp64 -> bf16 bit patterns (uint16), round to nearest even, one rounding."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.uint16)
    lib().osd_ref_round_bf16(_ptr(x), _ptr(out), x.size)
    return out


def bf16_midpoint_flags(x, rel=2.0 ** -20):
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, np.uint8)
    lib().osd_ref_bf16_midpoint_flags(_ptr(x), _ptr(out), x.size, float(rel))
    return out.astype(bool)


def bf16_to_f64(bits):
    """Exact widening of bf16 bit patterns (a format conversion, no arithmetic
    of the method)."""
    b = np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)
