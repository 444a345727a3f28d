"""Thin ctypes binding of libpixelfly.so (include/pixelfly.h).

Argument marshalling only: every compute step runs in the library's HIP
kernels.  Functions carry the C names; device buffers may be given as torch
tensors (their data_ptr() is passed) or as integer device addresses, streams
as torch.cuda.Stream objects, raw hipStream_t integers or None (the current
torch stream when torch is importable, else the null stream).  A non-zero
status raises PixelflyError with the library's detail message.  There is no
fallback: if libpixelfly.so is missing the import of this module fails.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpixelfly.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "pixelfly.h")

PF_OK, PF_ERR_INVALID_ARG, PF_ERR_UNSUPPORTED = 0, -1, -2
PF_ERR_WORKSPACE, PF_ERR_HIP, PF_ERR_NOMEM, PF_ERR_STATE = -3, -4, -5, -6
PF_BF16, PF_FP32 = 0, 1
PF_EPI_NONE, PF_EPI_GELU = 0, 1
PF_OP_NT, PF_OP_NN, PF_OP_TN = 0, 1, 2
# Kernel classes of the timing hook (pf_kernel_class).
KERNEL_CLASSES = ["spmm_fwd", "spmm_bwd_data", "sddmm", "lowrank_t", "lowrank_s", "reduce",
                  "gelu_bwd", "attn_fwd", "attn_bwd_dq", "attn_bwd_dkv", "dense", "butterfly"]
PF_KERNEL_COUNT = len(KERNEL_CLASSES)


class PixelflyError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"pixelfly status {status}: {msg}")
        self.status = status


# Load torch's HIP runtime first when torch is present: libpixelfly.so then
# binds to that same runtime (matched by SONAME) instead of bringing a second
# HIP/HSA runtime into the process, so torch tensors and streams are valid
# for the library.
try:
    import torch  # noqa: F401
except ImportError:
    pass

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} not built; run `python -m paper_2112_00029_amd.build` "
        "(or __graft_entry__.build())")
_lib = ctypes.CDLL(LIB_PATH)

_p = ctypes.c_void_p
_i32, _i64, _f32, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t


class pf_layout_info(ctypes.Structure):
    _fields_ = [("n_out", _i64), ("n_in", _i64), ("b", _i32), ("max_stride", _i32),
                ("eff_stride", _i32), ("s", _i32), ("nb_out", _i32), ("nb_in", _i32),
                ("nnzb", _i64), ("row_ptr", ctypes.POINTER(_i32)),
                ("col_idx", ctypes.POINTER(_i32)), ("col_ptr", ctypes.POINTER(_i32)),
                ("row_idx", ctypes.POINTER(_i32)), ("tperm", ctypes.POINTER(_i32))]


class pf_linear_plan(ctypes.Structure):
    _fields_ = [(n, _i32) for n in (
        "lowrank_t_kernel", "lowrank_t_split", "lowrank_t_tile_m", "lowrank_t_tile_n",
        "lowrank_s_kernel", "lowrank_s_split", "lowrank_s_tile_m", "lowrank_s_tile_n",
        "fwd_tile_m", "fwd_tile_n", "fwd_direct_lds", "bwd_tile_m", "bwd_tile_n",
        "bwd_direct_lds", "tn_items", "tn_split")] + [("tn_chunk", _i64),
                                                       ("workspace_bytes", ctypes.c_uint64),
                                                       ("tn_tile", _i32), ("tn_shared", _i32)]


_SIGS = {
    "pf_layout_create": (_i32, [_i64, _i64, _i32, _i32, ctypes.POINTER(_p)]),
    "pf_layout_create_from_mask": (_i32, [_i32, _i32, _i32, _p, ctypes.POINTER(_p)]),
    "pf_layout_create_attention": (_i32, [_i64, _i32, _i32, _i32, ctypes.POINTER(_p)]),
    "pf_layout_create_from_element_mask": (_i32, [_i64, _i64, _i32, _p, ctypes.POINTER(_p)]),
    "pf_layout_create_factor": (_i32, [_i64, _i32, _i32, ctypes.POINTER(_p)]),
    "pf_layout_create_butterfly": (_i32, [_i64, _i32, _i32, ctypes.POINTER(_p)]),
    "pf_butterfly_fwd": (_i32, [_p, _i64, _p, _p, _p, _p, _p]),
    "pf_butterfly_bwd_data": (_i32, [_p, _i64, _p, _p, _p, _p, _p]),
    "pf_select_mask": (_i32, [_i64, _i64, _i32, ctypes.c_double, ctypes.c_double,
                              ctypes.POINTER(_i32), ctypes.POINTER(_i32), ctypes.POINTER(_i64)]),
    "pf_layout_info_get": (_i32, [_p, ctypes.POINTER(pf_layout_info)]),
    "pf_layout_check": (_i32, [_p]),
    "pf_layout_plan_get": (_i32, [_p, ctypes.POINTER(_i32), _i32]),
    "pf_linear_plan_get": (_i32, [_p, _i32, _i64, _i32, ctypes.POINTER(pf_linear_plan)]),
    "pf_layout_upload": (_i32, [_p, _p]),
    "pf_layout_destroy": (None, [_p]),
    "pf_workspace_bytes": (_sz, [_p, _i64, _i32, _i32]),
    "pf_linear_fwd": (_i32, [_p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _p, _i32, _p, _p, _sz, _p]),
    "pf_linear_bwd_data": (_i32, [_p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _p, _i32, _p, _p, _sz,
                                  _p]),
    "pf_linear_bwd_weight": (_i32, [_p, _i32, _i64, _i32, _p, _p, _p, _p, _p, _p, _p, _p, _sz, _p]),
    "pf_linear_fwd_mixed": (_i32, [_p, _i32, _i64, _i32, _f32, _p, _p, _p, _p, _p, _p, _i32, _p, _p,
                                   _sz, _p]),
    "pf_linear_bwd_data_mixed": (_i32, [_p, _i32, _i64, _i32, _f32, _p, _p, _p, _p, _p, _p, _i32,
                                        _p, _p, _sz, _p]),
    "pf_linear_bwd_weight_mixed": (_i32, [_p, _i32, _i64, _i32, _f32, _p, _p, _p, _p, _p, _p, _p,
                                          _p, _p, _p, _sz, _p]),
    "pf_gelu_bwd": (_i32, [_i32, _i64, _p, _p, _p, _p]),
    "pf_attn_fwd": (_i32, [_p, _i32, _i32, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p]),
    "pf_attn_bwd": (_i32, [_p, _i32, _i32, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p, _p,
                           _p, _p, _sz, _p]),
    "pf_attn_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "pf_attn_bwd_noalloc": (_i32, [_p, _i32, _i32, _i32, _i32, _f32, _p, _p, _p, _p, _p, _p, _p,
                                   _p, _p, _p]),
    "pf_dense_gemm": (_i32, [_i32, _i32, _i64, _i64, _i64, _p, _p, _p, _p, _sz, _p]),
    "pf_dense_workspace_bytes": (_sz, [_i32, _i32, _i64, _i64, _i64]),
    "pf_timing_begin": (_i32, [_i32]),
    "pf_timing_end": (_i32, [ctypes.POINTER(_i32), ctypes.POINTER(ctypes.c_double)]),
    "pf_status_string": (ctypes.c_char_p, [_i32]),
    "pf_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def header_functions() -> list[str]:
    """Names of the functions include/pixelfly.h declares."""
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[a-z_ ]*?\*?\s*(pf_[a-z0-9_]+)\s*\(", text, re.M)))


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    raise TypeError(f"expected a tensor, int address or None, got {type(x)}")


def _stream(s):
    if s is None:
        try:
            import torch
            if torch.cuda.is_available() and torch.cuda.is_initialized():
                return torch.cuda.current_stream().cuda_stream
        except ImportError:
            pass
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(st: int):
    if st != PF_OK:
        raise PixelflyError(st, _lib.pf_last_error().decode())


def _dt(dtype) -> int:
    if isinstance(dtype, int):
        return dtype  # validated by the library
    name = str(dtype)
    if "bfloat16" in name or name == "bf16":
        return PF_BF16
    if "float32" in name or name == "fp32":
        return PF_FP32
    raise ValueError(f"unsupported dtype {dtype}")


class Layout:
    """Owner of a pf_layout* (destroyed with the object)."""

    def __init__(self, handle: int):
        self.handle = handle

    @property
    def _as_parameter_(self):
        return self.handle

    def __del__(self):
        h, self.handle = getattr(self, "handle", None), None
        if h and _lib is not None:
            _lib.pf_layout_destroy(h)


def pf_layout_create(n_out: int, n_in: int, b: int, max_stride: int) -> Layout:
    h = _p()
    _check(_lib.pf_layout_create(n_out, n_in, b, max_stride, ctypes.byref(h)))
    return Layout(h.value)


def pf_layout_create_from_mask(nb_out: int, nb_in: int, b: int, block_mask) -> Layout:
    """block_mask: (nb_out, nb_in) array-like, nonzero = kept block."""
    m = np.ascontiguousarray(np.asarray(block_mask).astype(bool).astype(np.uint8))
    if m.shape != (nb_out, nb_in):
        raise ValueError(f"block_mask shape {m.shape} != ({nb_out}, {nb_in})")
    h = _p()
    _check(_lib.pf_layout_create_from_mask(nb_out, nb_in, b, m.ctypes.data_as(_p), ctypes.byref(h)))
    return Layout(h.value)


def pf_layout_create_attention(seq: int, b: int, max_stride: int, global_blocks: int = 0) -> Layout:
    h = _p()
    _check(_lib.pf_layout_create_attention(seq, b, max_stride, global_blocks, ctypes.byref(h)))
    return Layout(h.value)


def pf_layout_create_from_element_mask(n_out: int, n_in: int, b: int, elem_mask) -> Layout:
    """elem_mask: (n_out, n_in) array-like, nonzero = kept element; the layout
    is its (b, b)-block cover."""
    m = np.ascontiguousarray(np.asarray(elem_mask).astype(bool).astype(np.uint8))
    if m.shape != (n_out, n_in):
        raise ValueError(f"elem_mask shape {m.shape} != ({n_out}, {n_in})")
    h = _p()
    _check(_lib.pf_layout_create_from_element_mask(n_out, n_in, b, m.ctypes.data_as(_p),
                                                   ctypes.byref(h)))
    return Layout(h.value)


def pf_layout_create_factor(n: int, b: int, k: int) -> Layout:
    h = _p()
    _check(_lib.pf_layout_create_factor(n, b, k, ctypes.byref(h)))
    return Layout(h.value)


def pf_layout_create_butterfly(n: int, b: int, max_stride: int) -> Layout:
    h = _p()
    _check(_lib.pf_layout_create_butterfly(n, b, max_stride, ctypes.byref(h)))
    return Layout(h.value)


def pf_butterfly_fwd(layout, T, X, F, Y, acts=None, stream=None) -> None:
    _check(_lib.pf_butterfly_fwd(layout.handle, T, _ptr(X), _ptr(F), _ptr(Y), _ptr(acts),
                                 _stream(stream)))


def pf_butterfly_bwd_data(layout, T, dY, F, dX, grads=None, stream=None) -> None:
    _check(_lib.pf_butterfly_bwd_data(layout.handle, T, _ptr(dY), _ptr(F), _ptr(dX),
                                      _ptr(grads), _stream(stream)))


def pf_select_mask(n_out: int, n_in: int, b: int, budget: float, lowrank_share: float = 0.25) -> dict:
    """Rank and maximum stride for a layer from a compute budget; returns
    dict(r=..., max_stride=..., params=...)."""
    r, ms, pr = _i32(), _i32(), _i64()
    _check(_lib.pf_select_mask(n_out, n_in, b, budget, lowrank_share, ctypes.byref(r),
                               ctypes.byref(ms), ctypes.byref(pr)))
    return dict(r=r.value, max_stride=ms.value, params=pr.value)


def pf_layout_info_get(layout: Layout) -> dict:
    """Layout metadata; index arrays are copied into numpy int32 arrays."""
    info = pf_layout_info()
    _check(_lib.pf_layout_info_get(layout.handle, ctypes.byref(info)))
    arr = lambda p, n: np.ctypeslib.as_array(p, shape=(n,)).copy() if n else np.zeros(0, np.int32)
    return {
        "n_out": info.n_out, "n_in": info.n_in, "b": info.b, "max_stride": info.max_stride,
        "eff_stride": info.eff_stride, "s": info.s, "nb_out": info.nb_out, "nb_in": info.nb_in,
        "nnzb": info.nnzb,
        "row_ptr": arr(info.row_ptr, info.nb_out + 1), "col_idx": arr(info.col_idx, info.nnzb),
        "col_ptr": arr(info.col_ptr, info.nb_in + 1), "row_idx": arr(info.row_idx, info.nnzb),
        "tperm": arr(info.tperm, info.nnzb),
    }


def pf_layout_check(layout: Layout) -> None:
    _check(_lib.pf_layout_check(layout.handle))


def pf_layout_plan_get(layout: Layout) -> dict:
    st = (_i32 * 10)()
    _check(_lib.pf_layout_plan_get(layout.handle, st, 10))
    keys = ["G_fwd", "fwd_tiles", "G_bwd", "bwd_tiles", "tn_items", "tn_kept",
            "G_fwd_wide", "fwd_tiles_wide", "G_bwd_wide", "bwd_tiles_wide"]
    return dict(zip(keys, list(st)))


def pf_linear_plan_get(layout: Layout, dtype, T: int, r: int) -> dict:
    """The kernels and splits a linear step of T tokens at rank r runs."""
    p = pf_linear_plan()
    _check(_lib.pf_linear_plan_get(layout.handle, _dt(dtype), T, r, ctypes.byref(p)))
    return {n: getattr(p, n) for n, _t in pf_linear_plan._fields_}


def pf_layout_upload(layout: Layout, stream=None) -> None:
    _check(_lib.pf_layout_upload(layout.handle, _stream(stream)))


def pf_layout_destroy(layout: Layout) -> None:
    h, layout.handle = layout.handle, None
    if h:
        _lib.pf_layout_destroy(h)


def pf_workspace_bytes(layout: Layout, T: int, r: int, dtype) -> int:
    return int(_lib.pf_workspace_bytes(layout.handle, T, r, _dt(dtype)))


def pf_linear_fwd(layout, dtype, T, r, X, Wblk, U, V, Y, T_lr, epi=PF_EPI_NONE,
                  Y_pre=None, workspace=None, ws_bytes=0, stream=None) -> None:
    _check(_lib.pf_linear_fwd(layout.handle, _dt(dtype), T, r, _ptr(X), _ptr(Wblk), _ptr(U),
                              _ptr(V), _ptr(Y), _ptr(T_lr), epi, _ptr(Y_pre), _ptr(workspace),
                              ws_bytes, _stream(stream)))


def pf_linear_bwd_data(layout, dtype, T, r, dY, Wblk, U, V, S, dX, epi=PF_EPI_NONE,
                       aux=None, workspace=None, ws_bytes=0, stream=None) -> None:
    _check(_lib.pf_linear_bwd_data(layout.handle, _dt(dtype), T, r, _ptr(dY), _ptr(Wblk),
                                   _ptr(U), _ptr(V), _ptr(S), _ptr(dX), epi, _ptr(aux),
                                   _ptr(workspace), ws_bytes, _stream(stream)))


def pf_linear_bwd_weight(layout, dtype, T, r, dY, X, T_lr, S, dWblk, dU, dV, workspace,
                         ws_bytes, stream=None) -> None:
    _check(_lib.pf_linear_bwd_weight(layout.handle, _dt(dtype), T, r, _ptr(dY), _ptr(X),
                                     _ptr(T_lr), _ptr(S), _ptr(dWblk), _ptr(dU), _ptr(dV),
                                     _ptr(workspace), ws_bytes, _stream(stream)))


def pf_linear_fwd_mixed(layout, dtype, T, r, gamma, X, Wblk, U, V, Y, T_lr, epi=PF_EPI_NONE,
                        Y_pre=None, workspace=None, ws_bytes=0, stream=None) -> None:
    _check(_lib.pf_linear_fwd_mixed(layout.handle, _dt(dtype), T, r, float(gamma), _ptr(X),
                                    _ptr(Wblk), _ptr(U), _ptr(V), _ptr(Y), _ptr(T_lr), epi,
                                    _ptr(Y_pre), _ptr(workspace), ws_bytes, _stream(stream)))


def pf_linear_bwd_data_mixed(layout, dtype, T, r, gamma, dY, Wblk, U, V, S, dX, epi=PF_EPI_NONE,
                             aux=None, workspace=None, ws_bytes=0, stream=None) -> None:
    _check(_lib.pf_linear_bwd_data_mixed(layout.handle, _dt(dtype), T, r, float(gamma), _ptr(dY),
                                         _ptr(Wblk), _ptr(U), _ptr(V), _ptr(S), _ptr(dX), epi,
                                         _ptr(aux), _ptr(workspace), ws_bytes, _stream(stream)))


def pf_linear_bwd_weight_mixed(layout, dtype, T, r, gamma, dY, X, Wblk, T_lr, S, dWblk, dU, dV,
                               dgamma, workspace, ws_bytes, stream=None) -> None:
    """dgamma: device buffer of one float32."""
    _check(_lib.pf_linear_bwd_weight_mixed(layout.handle, _dt(dtype), T, r, float(gamma),
                                           _ptr(dY), _ptr(X), _ptr(Wblk), _ptr(T_lr), _ptr(S),
                                           _ptr(dWblk), _ptr(dU), _ptr(dV), _ptr(dgamma),
                                           _ptr(workspace), ws_bytes, _stream(stream)))


def pf_gelu_bwd(dtype, n, dH, H_pre, dH_pre, stream=None) -> None:
    _check(_lib.pf_gelu_bwd(_dt(dtype), n, _ptr(dH), _ptr(H_pre), _ptr(dH_pre), _stream(stream)))


def pf_attn_fwd(layout, B, H, S, d, scale, Q, K, V, O, lse, stream=None) -> None:
    _check(_lib.pf_attn_fwd(layout.handle, B, H, S, d, scale, _ptr(Q), _ptr(K), _ptr(V),
                            _ptr(O), _ptr(lse), _stream(stream)))


def pf_attn_bwd(layout, B, H, S, d, scale, Q, K, V, O, lse, dO, dQ, dK, dV, workspace,
                ws_bytes, stream=None) -> None:
    _check(_lib.pf_attn_bwd(layout.handle, B, H, S, d, scale, _ptr(Q), _ptr(K), _ptr(V),
                            _ptr(O), _ptr(lse), _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV),
                            _ptr(workspace), ws_bytes, _stream(stream)))


def pf_attn_bwd_noalloc(layout, B, H, S, d, scale, Q, K, V, O, lse, dO, dQ, dK, dV,
                        stream=None) -> None:
    _check(_lib.pf_attn_bwd_noalloc(layout.handle, B, H, S, d, scale, _ptr(Q), _ptr(K), _ptr(V),
                                    _ptr(O), _ptr(lse), _ptr(dO), _ptr(dQ), _ptr(dK), _ptr(dV),
                                    _stream(stream)))


def pf_attn_workspace_bytes(B, H, S) -> int:
    return int(_lib.pf_attn_workspace_bytes(B, H, S))


def pf_dense_gemm(dtype, op, M, N, K, A, B, C, workspace=None, ws_bytes=0, stream=None) -> None:
    _check(_lib.pf_dense_gemm(_dt(dtype), op, M, N, K, _ptr(A), _ptr(B), _ptr(C),
                              _ptr(workspace), ws_bytes, _stream(stream)))


def pf_dense_workspace_bytes(dtype, op, M, N, K) -> int:
    return int(_lib.pf_dense_workspace_bytes(_dt(dtype), op, M, N, K))


def pf_timing_begin(max_launches_per_class: int) -> None:
    _check(_lib.pf_timing_begin(max_launches_per_class))


def pf_timing_end() -> dict:
    """{class name: (timed launches, mean duration in ms)}."""
    counts = (_i32 * PF_KERNEL_COUNT)()
    avg = (ctypes.c_double * PF_KERNEL_COUNT)()
    _check(_lib.pf_timing_end(counts, avg))
    return {n: (int(counts[i]), float(avg[i])) for i, n in enumerate(KERNEL_CLASSES)}


def pf_status_string(status: int) -> str:
    return _lib.pf_status_string(status).decode()


def pf_last_error() -> str:
    return _lib.pf_last_error().decode()
