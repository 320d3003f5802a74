"""ctypes binding of libprq.so (include/prq.h) -- argument marshalling only.

Every step of the hot path runs in the library: ``prq_prepare`` in its native
host code, ``prq_quant_act`` / ``prq_gemm`` / ``prq_grouped_gemm`` in its HIP
kernels.  torch supplies device memory (``data_ptr()``) and the stream
(``torch.cuda.current_stream().cuda_stream``); torch is imported before the
library is loaded so both use one HIP runtime instance.  There is no fallback:
a missing library raises ``ImportError`` at import time.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime the library binds to)

from . import build as _build

PRQ_OK, PRQ_EINVAL, PRQ_EALIGN, PRQ_EDEVICE, PRQ_EUNSUPPORTED, PRQ_EWORKSPACE = 0, -1, -2, -3, -4, -5
SCALE_MODES = {"smooth": 0, "act_only": 1, "none": 2}
GEMM_AUTO, GEMM_TILE, GEMM_STREAM, GEMM_STREAM_K = 0, 1, 2, 3
HEADER = os.path.join(_build.INCLUDE, "prq.h")

if not os.path.exists(_build.LIB):
    raise ImportError(f"{_build.LIB} is not built; run `python -m paper_2609_22106_amd.build`")
_lib = ctypes.CDLL(_build.LIB)

_p = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_sz = ctypes.c_size_t


def _decl(name, restype, argtypes):
    fn = getattr(_lib, name)
    fn.restype = restype
    fn.argtypes = argtypes
    return fn


_strerror = _decl("prq_strerror", ctypes.c_char_p, [ctypes.c_int])
_abi_version = _decl("prq_abi_version", ctypes.c_int, [])
_prepare = _decl("prq_prepare", ctypes.c_int,
                 [_p, _i32, _i32, _p, _i32, ctypes.c_double, _i32, _i32, _p, _p, _p, _p, _p, _p, _p])
_prepare_ex = _decl("prq_prepare_ex", ctypes.c_int,
                    [_p, _i32, _i32, _p, _i32, ctypes.c_double, _i32, _i32, _i32, _p, _p, _p, _p, _p,
                     _p, _p])
PREPARE_E8M0_SEARCH = 1
_expand = _decl("prq_expand_producer", ctypes.c_int, [_p, _p, _i32, _i32, _p, _p, _i32, _p, _p])
_evaluate = _decl("prq_evaluate_nrmse", ctypes.c_int,
                  [_p, _i32, _i32, _p, _i32, _p, _i32, ctypes.c_double, _i32, _i32, _i32, _p, _p])
_search = _decl("prq_search_alpha", ctypes.c_int,
                [_p, _i32, _i32, _p, _i32, _p, _i32, _i32, _i32, _i32, _p, _p, _p])
_quant_act = _decl("prq_quant_act", ctypes.c_int,
                   [_p, _i64, _i32, _i32, _i32, _p, _p, _p, _i32, _p, _p, _p])
_packed_bytes = _decl("prq_packed_weight_bytes", ctypes.c_int,
                      [_i32, _i32, _i32, ctypes.POINTER(_sz), ctypes.POINTER(_sz)])
_pack = _decl("prq_pack_weight", ctypes.c_int, [_p, _p, _i32, _i32, _i32, _p, _p, _p])
_gemm_ws = _decl("prq_gemm_workspace_bytes", _sz, [_i32, _i32, _i32])
_gemm_ws_ex = _decl("prq_gemm_workspace_bytes_ex", _sz, [_i32, _i32, _i32, _i32, _i32])
_gemm = _decl("prq_gemm", ctypes.c_int, [_p, _p, _i32, _p, _p, _i32, _i32, _p, _p, _sz, _p])
_gemm_ex = _decl("prq_gemm_ex", ctypes.c_int,
                 [_p, _p, _i32, _p, _p, _i32, _i32, _p, _p, _sz, _i32, _i32, _p])
_gemm_noalloc = _decl("prq_gemm_noalloc", ctypes.c_int, [_p, _p, _i32, _p, _p, _i32, _i32, _p, _p])
_gemm_noalloc_max = _decl("prq_gemm_noalloc_max_workspace_bytes", _sz, [])
_packed_act_bytes = _decl("prq_packed_act_bytes", ctypes.c_int,
                          [_i32, _i32, ctypes.POINTER(_sz), ctypes.POINTER(_sz)])
_quant_act_packed = _decl("prq_quant_act_packed", ctypes.c_int,
                          [_p, _i64, _i32, _i32, _i32, _p, _p, _p, _i32, _p, _p, _p])
_swiglu_quant = _decl("prq_swiglu_quant", ctypes.c_int, [_p, _p, _i64, _i32, _i32, _p, _p, _p])
_swiglu_quant_packed = _decl("prq_swiglu_quant_packed", ctypes.c_int,
                             [_p, _p, _i64, _i32, _i32, _p, _p, _p])
_gemm_packed_ws = _decl("prq_gemm_packed_workspace_bytes", _sz, [_i32, _i32, _i32])
_gemm_packed = _decl("prq_gemm_packed", ctypes.c_int,
                     [_p, _p, _i32, _p, _p, _i32, _i32, _p, _p, _sz, _p])
_ggemm_packed = _decl("prq_grouped_gemm_packed", ctypes.c_int,
                      [_p, _p, _p, _i32, _i32, _p, _p, _i32, _i32, _p, _p])
_ggemm_ws = _decl("prq_grouped_gemm_workspace_bytes", _sz, [_i32, _i32, _i32, _i32])
_ggemm = _decl("prq_grouped_gemm", ctypes.c_int,
               [_p, _p, _p, _i32, _i32, _p, _p, _i32, _i32, _p, _p, _sz, _p])
_ggemm_ex = _decl("prq_grouped_gemm_ex", ctypes.c_int,
                  [_p, _p, _p, _i32, _i32, _p, _p, _i32, _i32, _p, _p, _sz, _i32, _p])


class PRQError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {prq_strerror(status)} (status {status})")


def _check(status, where):
    if status != PRQ_OK:
        raise PRQError(status, where)


def prq_strerror(status):
    return _strerror(int(status)).decode()


def prq_abi_version():
    return int(_abi_version())


def exported_symbols():
    """Names of the functions include/prq.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(prq_\w+)\s*\(", text)))


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# --------------------------------------------------------------- prepare ---
def prq_prepare(W_bf16, Xcal_bf16, alpha, k_tail, scale_mode="smooth", with_col_err=False,
                scale_search=False):
    """Offline calibration/export (host).  W_bf16 [N, K] and Xcal_bf16 [T, K]
    are uint16 numpy arrays of bf16 bit patterns.  Returns numpy arrays.
    scale_search: the weight-side E8M0 block-scale search (prq_prepare_ex)."""
    W = np.ascontiguousarray(W_bf16, dtype=np.uint16)
    X = np.ascontiguousarray(Xcal_bf16, dtype=np.uint16)
    N, K = W.shape
    T = X.shape[0]
    if X.shape[1] != K:
        raise ValueError("calibration activations must have K columns")
    K_aug = K + int(k_tail)
    out = {
        "scale": np.empty(K, np.float32), "inv_scale": np.empty(K, np.float32),
        "perm": np.empty(K, np.int32), "inv_scale_pos": np.empty(K, np.float32),
        "Wq": np.empty((N, max(K_aug, 0) // 2), np.uint8),
        "Wsc": np.empty((N, max(K_aug, 0) // 32), np.uint8),
    }
    col_err = np.empty(K, np.float64) if with_col_err else None
    st = _prepare_ex(_ptr(W), N, K, _ptr(X), T, float(alpha), int(k_tail), SCALE_MODES[scale_mode],
                     PREPARE_E8M0_SEARCH if scale_search else 0,
                     _ptr(out["scale"]), _ptr(out["inv_scale"]), _ptr(out["perm"]),
                     _ptr(out["inv_scale_pos"]), _ptr(out["Wq"]), _ptr(out["Wsc"]), _ptr(col_err))
    _check(st, "prq_prepare")
    if with_col_err:
        out["col_err"] = col_err
    return out


def prq_expand_producer(W_up_bf16, W_gate_bf16, inv_scale, perm, k_tail):
    """Offline copy (host): (W_up_aug, W_gate_aug or None), each [C + k, H]
    bf16 bit patterns (uint16)."""
    up = _bf16_host(W_up_bf16, "W_up")
    gate = None if W_gate_bf16 is None else _bf16_host(W_gate_bf16, "W_gate")
    C, H = up.shape
    if gate is not None and gate.shape != up.shape:
        raise ValueError("W_gate must have W_up's shape")
    inv = np.ascontiguousarray(inv_scale, dtype=np.float32)
    p = np.ascontiguousarray(perm, dtype=np.int32)
    if inv.shape != (C,) or p.shape != (C,):
        raise ValueError("inv_scale and perm must have C entries")
    up_aug = np.empty((C + int(k_tail), H), np.uint16)
    gate_aug = None if gate is None else np.empty((C + int(k_tail), H), np.uint16)
    _check(_expand(_ptr(up), _ptr(gate), C, H, _ptr(inv), _ptr(p), int(k_tail), _ptr(up_aug),
                   _ptr(gate_aug)), "prq_expand_producer")
    return up_aug, gate_aug


# ------------------------------------------------------------ evaluation ---
def _bf16_host(a, name):
    a = np.ascontiguousarray(a)
    if a.dtype not in (np.uint16, np.int16) or a.ndim != 2:
        raise ValueError(f"{name} must be a 2-D array of bf16 bit patterns (uint16)")
    return a


def prq_evaluate_nrmse(W_bf16, Xcal_bf16, X_bf16, alpha, k_tail, scale_mode="smooth",
                       scale_search=False, stream=None):
    """y-NRMSE of one configuration on the rows X (offline; host arrays)."""
    W, Xc, X = _bf16_host(W_bf16, "W"), _bf16_host(Xcal_bf16, "Xcal"), _bf16_host(X_bf16, "X")
    N, K = W.shape
    if Xc.shape[1] != K or X.shape[1] != K:
        raise ValueError("activations must have K columns")
    out = ctypes.c_double()
    st = _evaluate(_ptr(W), N, K, _ptr(Xc), Xc.shape[0], _ptr(X), X.shape[0], float(alpha),
                   int(k_tail), SCALE_MODES[scale_mode], PREPARE_E8M0_SEARCH if scale_search else 0,
                   ctypes.byref(out), _stream(stream))
    _check(st, "prq_evaluate_nrmse")
    return float(out.value)


def prq_search_alpha(W_bf16, Xcal_bf16, alphas, k_tail, scale_mode="smooth", scale_search=False,
                     stream=None):
    """Algorithm 1's alpha search (offline): (best alpha, y-NRMSE per alpha)."""
    W, Xc = _bf16_host(W_bf16, "W"), _bf16_host(Xcal_bf16, "Xcal")
    N, K = W.shape
    if Xc.shape[1] != K:
        raise ValueError("calibration activations must have K columns")
    a = np.ascontiguousarray(alphas, dtype=np.float64)
    err = np.empty(a.size, np.float64)
    best = ctypes.c_int32()
    st = _search(_ptr(W), N, K, _ptr(Xc), Xc.shape[0], _ptr(a), a.size, int(k_tail),
                 SCALE_MODES[scale_mode], PREPARE_E8M0_SEARCH if scale_search else 0, _ptr(err),
                 ctypes.byref(best), _stream(stream))
    _check(st, "prq_search_alpha")
    return float(a[best.value]), err


# ------------------------------------------------------------- device ops ---
# The library receives bare pointers and cannot see buffer extents, so the
# binding checks every tensor against the sizes it passes (shape, dtype,
# contiguity) and that it lives on a GPU, before anything is launched.
def _need(t, name, dtype, shape=None, min_numel=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype not in (dtype if isinstance(dtype, tuple) else (dtype,)):
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name} has {t.numel()} elements, needs at least {min_numel}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _on_gpu(**tensors):
    for name, t in tensors.items():
        if t is not None and not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")


_BF16_LIKE = (torch.int16, torch.uint16, torch.bfloat16)


def prq_quant_act(X, K, k_tail, inv_scale_pos=None, perm=None, group_offsets=None, G=1,
                  Aq=None, Asc=None, stream=None):
    """Quantize bf16 activations X [M, ld] (device) -> (Aq [M, K_aug/2], Asc [M, K_aug/32]).
    inv_scale_pos[p] = 1/s_{perm[p]} (prq_prepare's ``inv_scale_pos``)."""
    if not isinstance(X, torch.Tensor) or X.dim() != 2 or X.dtype not in _BF16_LIKE:
        raise ValueError("X must be a 2-D tensor of bf16 values (or their int16 bit patterns)")
    M = X.shape[0]
    K_aug = K + k_tail
    if X.shape[1] < K or (M > 1 and X.stride(0) < K) or X.stride(1) != 1:
        raise ValueError(f"X rows must hold K={K} contiguous values (shape {tuple(X.shape)}, "
                         f"strides {X.stride()})")
    if Aq is None:
        Aq = torch.empty((M, K_aug // 2), dtype=torch.uint8, device=X.device)
    if Asc is None:
        Asc = torch.empty((M, K_aug // 32), dtype=torch.uint8, device=X.device)
    _need(Aq, "Aq", torch.uint8, (M, K_aug // 2))
    _need(Asc, "Asc", torch.uint8, (M, K_aug // 32))
    if inv_scale_pos is not None:
        _need(inv_scale_pos, "inv_scale_pos", torch.float32, min_numel=G * K)
    if perm is not None:
        _need(perm, "perm", torch.int32, min_numel=G * K)
    if G > 1:
        if group_offsets is None:
            raise ValueError("G > 1 needs group_offsets")
        _need(group_offsets, "group_offsets", torch.int32, min_numel=G + 1)
    _on_gpu(X=X, Aq=Aq, Asc=Asc, inv_scale_pos=inv_scale_pos, perm=perm,
            group_offsets=group_offsets if G > 1 else None)
    ld = X.stride(0) if M > 1 else K
    st = _quant_act(_ptr(X), ld, M, K, k_tail, _ptr(inv_scale_pos), _ptr(perm), _ptr(group_offsets), G,
                    _ptr(Aq), _ptr(Asc), _stream(stream))
    _check(st, "prq_quant_act")
    return Aq, Asc


class PackedWeight:
    """Device buffers of a weight in the GEMM's packed layout (include/prq.h)."""

    def __init__(self, Wp, Wps, E, N, K_aug):
        self.Wp, self.Wps, self.E, self.N, self.K_aug = Wp, Wps, E, N, K_aug

    def check_sizes(self):
        cb, sb = prq_packed_weight_bytes(self.E, self.N, self.K_aug)
        _need(self.Wp, "W.Wp", torch.uint8, min_numel=cb)
        _need(self.Wps, "W.Wps", torch.uint8, min_numel=sb)


def _check_gemm_operands(Aq, Asc, W, Y, M):
    _need(Aq, "Aq", torch.uint8, (M, W.K_aug // 2))
    _need(Asc, "Asc", torch.uint8, (M, W.K_aug // 32))
    _need(Y, "Y", torch.float32, (M, W.N))
    W.check_sizes()
    _on_gpu(Aq=Aq, Asc=Asc, Y=Y, Wp=W.Wp, Wps=W.Wps)


def prq_packed_weight_bytes(E, N, K_aug):
    cb, sb = _sz(0), _sz(0)
    _check(_packed_bytes(E, N, K_aug, ctypes.byref(cb), ctypes.byref(sb)), "prq_packed_weight_bytes")
    return int(cb.value), int(sb.value)


def prq_pack_weight(Wq, Wsc, stream=None):
    """Canonical device Wq [N, K_aug/2] / Wsc [N, K_aug/32] (or [E, N, ...]) ->
    PackedWeight in the layout the GEMM kernels read."""
    if not isinstance(Wq, torch.Tensor) or Wq.dim() not in (2, 3):
        raise ValueError("Wq must be a [N, K_aug/2] or [E, N, K_aug/2] tensor")
    E = Wq.shape[0] if Wq.dim() == 3 else 1
    N = Wq.shape[-2]
    K_aug = Wq.shape[-1] * 2
    _need(Wq, "Wq", torch.uint8)
    _need(Wsc, "Wsc", torch.uint8, tuple(Wq.shape[:-1]) + (K_aug // 32,))
    _on_gpu(Wq=Wq, Wsc=Wsc)
    cb, sb = prq_packed_weight_bytes(E, N, K_aug)
    Wp = torch.empty(cb, dtype=torch.uint8, device=Wq.device)
    Wps = torch.empty(sb, dtype=torch.uint8, device=Wq.device)
    _check(_pack(_ptr(Wq), _ptr(Wsc), E, N, K_aug, _ptr(Wp), _ptr(Wps), _stream(stream)),
           "prq_pack_weight")
    return PackedWeight(Wp, Wps, E, N, K_aug)


def prq_gemm_workspace_bytes(M, N, K_aug, variant=GEMM_AUTO, splits=0):
    return int(_gemm_ws_ex(M, N, K_aug, variant, splits))


def prq_gemm(Aq, Asc, W, Y=None, workspace=None, variant=GEMM_AUTO, splits=0, stream=None):
    """Y [M, N] float32 = deq(A_aug) deq(W_aug)^T over K_aug (device); W is a
    PackedWeight (E = 1)."""
    M = Aq.shape[0]
    N, K_aug = W.N, W.K_aug
    if W.E != 1:
        raise ValueError("prq_gemm takes a single weight (E = 1); use prq_grouped_gemm")
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=W.Wp.device)
    _check_gemm_operands(Aq, Asc, W, Y, M)
    need = prq_gemm_workspace_bytes(M, N, K_aug, variant, splits)
    if workspace is None and need:
        workspace = torch.zeros(need, dtype=torch.uint8, device=W.Wp.device)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
        _on_gpu(workspace=workspace)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = _gemm_ex(_ptr(Aq), _ptr(Asc), M, _ptr(W.Wp), _ptr(W.Wps), N, K_aug, _ptr(Y),
                  _ptr(workspace), ws_bytes, variant, splits, _stream(stream))
    _check(st, "prq_gemm")
    return Y


def prq_gemm_noalloc_max_workspace_bytes():
    return int(_gemm_noalloc_max())


def prq_gemm_noalloc(Aq, Asc, W, Y, stream=None):
    """prq_gemm (AUTO) with the library's own device scratch as its workspace:
    nothing is allocated, Y [M, N] float32 must be given."""
    M = Aq.shape[0]
    if W.E != 1:
        raise ValueError("prq_gemm_noalloc takes a single weight (E = 1)")
    _check_gemm_operands(Aq, Asc, W, Y, M)
    st = _gemm_noalloc(_ptr(Aq), _ptr(Asc), M, _ptr(W.Wp), _ptr(W.Wps), W.N, W.K_aug, _ptr(Y),
                       _stream(stream))
    _check(st, "prq_gemm_noalloc")
    return Y


class PackedAct:
    """Device buffers of an activation in the packed layout (include/prq.h)."""

    def __init__(self, Ap, Aps, M, K_aug):
        self.Ap, self.Aps, self.M, self.K_aug = Ap, Aps, M, K_aug

    def check_sizes(self):
        cb, sb = prq_packed_act_bytes(self.M, self.K_aug)
        _need(self.Ap, "A.Ap", torch.uint8, min_numel=cb)
        _need(self.Aps, "A.Aps", torch.uint8, min_numel=sb)


def prq_packed_act_bytes(M, K_aug):
    cb, sb = _sz(0), _sz(0)
    _check(_packed_act_bytes(M, K_aug, ctypes.byref(cb), ctypes.byref(sb)), "prq_packed_act_bytes")
    return int(cb.value), int(sb.value)


def prq_quant_act_packed(X, K, k_tail, inv_scale_pos=None, perm=None, out=None, stream=None,
                         group_offsets=None, G=1):
    """prq_quant_act into the packed activation layout -> PackedAct.
    out: a PackedAct of the same M and K_aug to write into (else allocated).
    G > 1: rows sorted by group, group_offsets [G + 1] device int32, and
    inv_scale_pos / perm hold G rows of K (one per expert)."""
    if not isinstance(X, torch.Tensor) or X.dim() != 2 or X.dtype not in _BF16_LIKE:
        raise ValueError("X must be a 2-D tensor of bf16 values (or their int16 bit patterns)")
    M = X.shape[0]
    K_aug = K + k_tail
    if X.shape[1] < K or (M > 1 and X.stride(0) < K) or X.stride(1) != 1:
        raise ValueError(f"X rows must hold K={K} contiguous values (shape {tuple(X.shape)}, "
                         f"strides {X.stride()})")
    if out is None:
        cb, sb = prq_packed_act_bytes(M, K_aug)
        out = PackedAct(torch.empty(cb, dtype=torch.uint8, device=X.device),
                        torch.empty(sb, dtype=torch.uint8, device=X.device), M, K_aug)
    if out.M != M or out.K_aug != K_aug:
        raise ValueError(f"out holds {out.M} rows of K_aug {out.K_aug}, expected {M} x {K_aug}")
    out.check_sizes()
    if inv_scale_pos is not None:
        _need(inv_scale_pos, "inv_scale_pos", torch.float32, min_numel=G * K)
    if perm is not None:
        _need(perm, "perm", torch.int32, min_numel=G * K)
    if G > 1:
        if group_offsets is None:
            raise ValueError("G > 1 needs group_offsets")
        _need(group_offsets, "group_offsets", torch.int32, min_numel=G + 1)
    _on_gpu(X=X, Ap=out.Ap, Aps=out.Aps, inv_scale_pos=inv_scale_pos, perm=perm,
            group_offsets=group_offsets if G > 1 else None)
    ld = X.stride(0) if M > 1 else K
    st = _quant_act_packed(_ptr(X), ld, M, K, k_tail, _ptr(inv_scale_pos), _ptr(perm),
                           _ptr(group_offsets) if G > 1 else None, G, _ptr(out.Ap), _ptr(out.Aps),
                           _stream(stream))
    _check(st, "prq_quant_act_packed")
    return out


def prq_swiglu_quant(gate, up, K_aug, packed=False, out=None, stream=None):
    """Q(SiLU(gate) * up) of the expanded producers' bf16 outputs [M, >= K_aug]
    (offline copy, producer side): row-major (Aq, Asc) or, with packed=True, a
    PackedAct.  out: (Aq, Asc) or a PackedAct to write into (else allocated)."""
    for name, t in (("gate", gate), ("up", up)):
        if not isinstance(t, torch.Tensor) or t.dim() != 2 or t.dtype not in _BF16_LIKE:
            raise ValueError(f"{name} must be a 2-D tensor of bf16 values (or their int16 bit patterns)")
        if t.shape[1] < K_aug or t.stride(1) != 1:
            raise ValueError(f"{name} rows must hold K_aug={K_aug} contiguous values "
                             f"(shape {tuple(t.shape)}, strides {t.stride()})")
    if gate.shape != up.shape or gate.stride() != up.stride():
        raise ValueError(f"gate {tuple(gate.shape)} / {gate.stride()} and up {tuple(up.shape)} / "
                         f"{up.stride()} must have the same shape and strides")
    M = gate.shape[0]
    ld = gate.stride(0) if M > 1 else K_aug
    if packed:
        if out is None:
            cb, sb = prq_packed_act_bytes(M, K_aug)
            out = PackedAct(torch.empty(cb, dtype=torch.uint8, device=gate.device),
                            torch.empty(sb, dtype=torch.uint8, device=gate.device), M, K_aug)
        if out.M != M or out.K_aug != K_aug:
            raise ValueError(f"out holds {out.M} rows of K_aug {out.K_aug}, expected {M} x {K_aug}")
        out.check_sizes()
        A, As = out.Ap, out.Aps
    else:
        if out is None:
            out = (torch.empty((M, K_aug // 2), dtype=torch.uint8, device=gate.device),
                   torch.empty((M, K_aug // 32), dtype=torch.uint8, device=gate.device))
        A, As = out
        _need(A, "Aq", torch.uint8, (M, K_aug // 2))
        _need(As, "Asc", torch.uint8, (M, K_aug // 32))
    _on_gpu(gate=gate, up=up, A=A, As=As)
    fn = _swiglu_quant_packed if packed else _swiglu_quant
    st = fn(_ptr(gate), _ptr(up), ld, M, K_aug, _ptr(A), _ptr(As), _stream(stream))
    _check(st, "prq_swiglu_quant_packed" if packed else "prq_swiglu_quant")
    return out


def prq_gemm_packed_workspace_bytes(M, N, K_aug):
    return int(_gemm_packed_ws(M, N, K_aug))


def prq_gemm_packed(A, W, Y=None, workspace=None, stream=None):
    """Y [M, N] float32 = Eq. 3 over K_aug for a PackedAct A and a PackedWeight W (E = 1).
    workspace: uint8 device tensor of prq_gemm_packed_workspace_bytes (split along
    K when the planner wants it; without it the call runs unsplit)."""
    if W.E != 1:
        raise ValueError("prq_gemm_packed takes a single weight (E = 1)")
    if A.K_aug != W.K_aug:
        raise ValueError(f"K_aug differs: activation {A.K_aug}, weight {W.K_aug}")
    M, N = A.M, W.N
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=W.Wp.device)
    _need(Y, "Y", torch.float32, (M, N))
    A.check_sizes()
    W.check_sizes()
    _on_gpu(Ap=A.Ap, Aps=A.Aps, Y=Y, Wp=W.Wp, Wps=W.Wps)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
        _on_gpu(workspace=workspace)
    ws_bytes = workspace.numel() if workspace is not None else 0
    st = _gemm_packed(_ptr(A.Ap), _ptr(A.Aps), M, _ptr(W.Wp), _ptr(W.Wps), N, W.K_aug, _ptr(Y),
                      _ptr(workspace), ws_bytes, _stream(stream))
    _check(st, "prq_gemm_packed")
    return Y


def prq_grouped_gemm_packed(A, group_offsets, W, Y=None, stream=None):
    """prq_grouped_gemm on a PackedAct A (rows sorted by expert, from
    prq_quant_act_packed with the same group_offsets); Y [M_total, N] float32."""
    if A.K_aug != W.K_aug:
        raise ValueError(f"K_aug differs: activation {A.K_aug}, weight {W.K_aug}")
    M, E, N = A.M, W.E, W.N
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=W.Wp.device)
    _need(Y, "Y", torch.float32, (M, N))
    _need(group_offsets, "group_offsets", torch.int32, (E + 1,))
    A.check_sizes()
    W.check_sizes()
    _on_gpu(Ap=A.Ap, Aps=A.Aps, Y=Y, Wp=W.Wp, Wps=W.Wps, group_offsets=group_offsets)
    st = _ggemm_packed(_ptr(A.Ap), _ptr(A.Aps), _ptr(group_offsets), E, M, _ptr(W.Wp), _ptr(W.Wps),
                       N, W.K_aug, _ptr(Y), _stream(stream))
    _check(st, "prq_grouped_gemm_packed")
    return Y


def prq_grouped_gemm_workspace_bytes(M_total, E, N, K_aug):
    return int(_ggemm_ws(M_total, E, N, K_aug))


def prq_grouped_gemm(Aq, Asc, group_offsets, W, Y=None, workspace=None, variant=GEMM_AUTO,
                     stream=None):
    """Rows sorted by expert; W a PackedWeight of E experts; Y [M_total, N] float32."""
    M = Aq.shape[0]
    E, N, K_aug = W.E, W.N, W.K_aug
    if Y is None:
        Y = torch.empty((M, N), dtype=torch.float32, device=W.Wp.device)
    _need(group_offsets, "group_offsets", torch.int32, (E + 1,))
    _check_gemm_operands(Aq, Asc, W, Y, M)
    _on_gpu(group_offsets=group_offsets)
    if workspace is not None:
        _need(workspace, "workspace", torch.uint8)
        _on_gpu(workspace=workspace)
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    st = _ggemm_ex(_ptr(Aq), _ptr(Asc), _ptr(group_offsets), E, M, _ptr(W.Wp), _ptr(W.Wps), N,
                   K_aug, _ptr(Y), _ptr(workspace), ws_bytes, variant, _stream(stream))
    _check(st, "prq_grouped_gemm")
    return Y
