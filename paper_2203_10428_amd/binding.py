"""Thin ctypes binding of libpgcn (the C ABI declared in include/pgcn.h).

Argument marshalling only: every computation runs in the library's HIP
kernels.  Device buffers are passed as raw pointers (``int``); a torch
tensor's ``data_ptr()`` or a stream's ``cuda_stream`` are the usual sources.
If the shared library is missing, importing this module raises: there is no
fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
# torch ships its own HIP runtime (SONAME libamdhip64.so.7).  Loading torch
# first makes libpgcn bind to that already-loaded runtime, so the process has
# one HIP/HSA runtime shared by torch's allocator and streams and libpgcn.
import torch  # noqa: F401

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpgcn.so")

PGCN_OK, PGCN_EINVAL, PGCN_ENOMEM, PGCN_EHIP, PGCN_EUNSUPPORTED, PGCN_EWORKSPACE = range(6)
PGCN_F32, PGCN_BF16 = 0, 1
PGCN_SETUP_HOST_ONLY, PGCN_SETUP_NO_SELF_LOOP, PGCN_SETUP_SYMMETRIC = 1, 2, 4
PGCN_PACK_FEAT, PGCN_ACCUM_GRAD = 0, 1
PGCN_MAX_WIDTH = 63740
PGCN_SOFTMAX_CE, PGCN_SIGMOID_BCE = 0, 1
PGCN_REFILL_DMA, PGCN_REFILL_FROM_HOST = 1, 2
PGCN_ORDER_AGG, PGCN_ORDER_TRANSFORM = 0, 1
PGCN_NOALLOC_SCRATCH_BYTES = 32 << 20

_vp = C.c_void_p
_i32, _i64, _u32, _f32, _sz = C.c_int32, C.c_int64, C.c_uint32, C.c_float, C.c_size_t


class pgcn_csr(C.Structure):
    _fields_ = [("n", _i64), ("rowptr", _vp), ("col", _vp)]


class pgcn_boundary_map(C.Structure):
    _fields_ = [("nparts", _i32), ("self", _i32), ("owner", _vp)]


class pgcn_info(C.Structure):
    _fields_ = [("n_inner", _i64), ("n_bd", _i64), ("nnz", _i64), ("n_send", _i64),
                ("max_row_len", _i64), ("max_row_len_t", _i64), ("nparts", _i32), ("self", _i32),
                ("host_only", _i32), ("spmm_segment", _i32), ("spmm_items", _i64),
                ("spmm_split_slots", _i64), ("spmmt_items", _i64), ("spmmt_split_slots", _i64),
                ("spmm_chunks", _i32), ("spmmt_chunks", _i32), ("symmetric", _i32), ("self_loop", _i32),
                ("spmm_chunks_narrow", _i32), ("spmmt_chunks_narrow", _i32),
                ("spmm_hub_rows", _i32), ("spmm_hub_cols", _i32), ("spmm_hub_nnz", _i64),
                ("spmmt_hub_rows", _i32), ("spmmt_hub_cols", _i32), ("spmmt_hub_nnz", _i64)]


class pgcn_arrays(C.Structure):
    _fields_ = [(n, _vp) for n in ("inner_gid", "bd_gid", "recv_ptr", "rowptr", "col", "rowptr_t",
                                    "col_t", "send_ptr", "send_idx", "inv_ptr", "inv_k", "deg")]


class pgcn_fwd_args(C.Structure):
    _fields_ = [("f_in", _i32), ("f_out", _i32), ("gemm_dtype", _i32), ("relu", _i32),
                ("ld_in", _i64), ("ld_out", _i64), ("H_in", _vp), ("H_bd", _vp), ("W", _vp),
                ("A", _vp), ("A_bf16", _vp), ("H_out", _vp), ("workspace", _vp), ("workspace_bytes", _sz),
                ("order", _i32), ("a_given", _i32), ("send_out", _vp)]


class pgcn_bwd_args(C.Structure):
    _fields_ = [("f_in", _i32), ("f_out", _i32), ("gemm_dtype", _i32), ("relu", _i32),
                ("ld_in", _i64), ("ld_out", _i64), ("J_out", _vp), ("H_out", _vp), ("A", _vp),
                ("A_bf16", _vp), ("W", _vp), ("dW", _vp), ("J_in", _vp), ("J_bd_out", _vp),
                ("workspace", _vp), ("workspace_bytes", _sz), ("order", _i32), ("H_in", _vp), ("H_bd", _vp)]


class pgcn_sage_fwd_args(C.Structure):
    _fields_ = [("f_in", _i32), ("f_out", _i32), ("gemm_dtype", _i32), ("relu", _i32),
                ("ld_in", _i64), ("ld_out", _i64), ("X_in", _vp), ("X_in_bf16", _vp), ("X_bd", _vp), ("W", _vp),
                ("A", _vp), ("A_bf16", _vp), ("H_out", _vp), ("workspace", _vp), ("workspace_bytes", _sz),
                ("order", _i32), ("send_out", _vp)]


class pgcn_sage_bwd_args(C.Structure):
    _fields_ = [("f_in", _i32), ("f_out", _i32), ("gemm_dtype", _i32), ("relu", _i32),
                ("ld_in", _i64), ("ld_out", _i64), ("J_out", _vp), ("H_out", _vp), ("A", _vp),
                ("A_bf16", _vp), ("X_in", _vp), ("X_in_bf16", _vp), ("W", _vp), ("dW", _vp), ("J_in", _vp),
                ("J_bd_out", _vp), ("workspace", _vp), ("workspace_bytes", _sz), ("order", _i32), ("X_bd", _vp)]


# every symbol include/pgcn.h declares, with its ctypes signature
SIGNATURES = {
    "pgcn_partition_setup": (_i32, [C.POINTER(pgcn_csr), C.POINTER(pgcn_boundary_map), _u32, C.POINTER(_vp)]),
    "pgcn_partition_info": (_i32, [_vp, C.POINTER(pgcn_info)]),
    "pgcn_partition_export": (_i32, [_vp, C.POINTER(pgcn_arrays)]),
    "pgcn_partition_destroy": (None, [_vp]),
    "pgcn_workspace_size": (_sz, [_vp, _i32, _i32, _i32]),
    "pgcn_layer_workspace_size": (_sz, [_vp, _i32, _i32, _i32, _i32]),
    "pgcn_layer_fwd": (_i32, [_vp, C.POINTER(pgcn_fwd_args), _vp]),
    "pgcn_layer_fwd_noalloc": (_i32, [_vp, C.POINTER(pgcn_fwd_args), _vp]),
    "pgcn_layer_bwd": (_i32, [_vp, C.POINTER(pgcn_bwd_args), _vp]),
    "pgcn_smooth_ema": (_i32, [_vp, _vp, _i64, _i32, _i64, _f32, _vp]),
    "pgcn_pack_boundary": (_i32, [_vp, _i32, _vp, _vp, _i32, _i64, _vp]),
    "pgcn_accum_smoothed": (_i32, [_vp, _vp, _vp, _f32, _vp, _i32, _i64, _vp]),
    "pgcn_loss_fwd_bwd": (_i32, [_i32, _vp, _i64, _i32, _i64, _vp, _vp, _i64, _f32, _vp, _vp, _vp, _sz, _vp]),
    "pgcn_sgd_update": (_i32, [_vp, _vp, _vp, _i64, _f32, _vp]),
    "pgcn_adam_update": (_i32, [_vp, _vp, _vp, _vp, _vp, _i64, C.c_double, C.c_double, C.c_double, C.c_double,
                                _i32, _vp]),
    "pgcn_dropout": (_i32, [_vp, _vp, _i64, _i32, _i64, _i64, C.c_double, _u32, _u32, _u32, _u32, _vp, _i64,
                            _vp]),
    "pgcn_sage_layer_fwd": (_i32, [_vp, C.POINTER(pgcn_sage_fwd_args), _vp]),
    "pgcn_sage_layer_bwd": (_i32, [_vp, C.POINTER(pgcn_sage_bwd_args), _vp]),
    "pgcn_refill_async": (_i32, [_vp, _vp, _sz, _u32, _vp]),
    "pgcn_trace_enable": (_i32, [_i32]),
    "pgcn_trace_filter": (_i32, [C.c_uint32]),
    "pgcn_trace_collect": (_i32, [_vp, _vp, _vp, _i32, C.POINTER(_i32)]),
    "pgcn_trace_disable": (_i32, []),
    "pgcn_last_error": (C.c_char_p, []),
    "pgcn_version": (_i32, []),
}


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libpgcn.so not found at {LIB_PATH}: build it with "
                          "`python -c 'import __graft_entry__ as g; g.build()'`")
    lib = C.CDLL(LIB_PATH)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


class PgcnError(RuntimeError):
    def __init__(self, code: int, where: str):
        msg = lib.pgcn_last_error().decode(errors="replace")
        super().__init__(f"{where} failed with status {code}: {msg}")
        self.code = code


def _check(code: int, where: str):
    if code != PGCN_OK:
        raise PgcnError(code, where)


def _ptr(x) -> int | None:
    """A device/host pointer from a torch tensor, a numpy array, an int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(s) -> int | None:
    if s is None or isinstance(s, int):
        return s
    return s.cuda_stream


# --------------------------------------------------------------------------
# Python-named wrappers (same names as the C entry points)
# --------------------------------------------------------------------------

class Partition:
    """Owns a pgcn_partition handle (freed by pgcn_partition_destroy)."""

    def __init__(self, handle: int):
        self.handle = handle

    def __del__(self):
        h = getattr(self, "handle", None)
        if h and lib is not None:                  # at interpreter exit the module may be torn down first
            lib.pgcn_partition_destroy(h)
            self.handle = None

    @property
    def _as_parameter_(self):
        return self.handle


def pgcn_partition_setup(n: int, rowptr: np.ndarray, col: np.ndarray, owner: np.ndarray,
                         nparts: int, self_part: int, host_only: bool = False, self_loop: bool = True,
                         symmetric: bool = False) -> Partition:
    rowptr = np.ascontiguousarray(rowptr, dtype=np.int64)
    col = np.ascontiguousarray(col, dtype=np.int32)
    owner = np.ascontiguousarray(owner, dtype=np.int32)
    csr = pgcn_csr(n, rowptr.ctypes.data, col.ctypes.data if len(col) else None)
    bmap = pgcn_boundary_map(nparts, self_part, owner.ctypes.data)
    out = _vp()
    flags = (PGCN_SETUP_HOST_ONLY if host_only else 0) | (0 if self_loop else PGCN_SETUP_NO_SELF_LOOP) | \
        (PGCN_SETUP_SYMMETRIC if symmetric else 0)
    _check(lib.pgcn_partition_setup(C.byref(csr), C.byref(bmap), flags, C.byref(out)), "pgcn_partition_setup")
    return Partition(out.value)


def pgcn_partition_info(part: Partition) -> dict:
    info = pgcn_info()
    _check(lib.pgcn_partition_info(part.handle, C.byref(info)), "pgcn_partition_info")
    return {name: getattr(info, name) for name, _ in pgcn_info._fields_}


def pgcn_partition_export(part: Partition) -> dict:
    i = pgcn_partition_info(part)
    n, b, nnz, s, P = i["n_inner"], i["n_bd"], i["nnz"], i["n_send"], i["nparts"]
    out = dict(inner_gid=np.empty(n, np.int64), bd_gid=np.empty(b, np.int64), recv_ptr=np.empty(P + 1, np.int64),
               rowptr=np.empty(n + 1, np.int64), col=np.empty(nnz, np.int32),
               rowptr_t=np.empty(n + b + 1, np.int64), col_t=np.empty(nnz, np.int32),
               send_ptr=np.empty(P + 1, np.int64), send_idx=np.empty(s, np.int32),
               inv_ptr=np.empty(n + 1, np.int64), inv_k=np.empty(s, np.int32), deg=np.empty(n + b, np.int64))
    arr = pgcn_arrays(**{k: (v.ctypes.data if v.size else None) for k, v in out.items()})
    _check(lib.pgcn_partition_export(part.handle, C.byref(arr)), "pgcn_partition_export")
    return out


def pgcn_workspace_size(part: Partition, f_in: int, f_out: int, gemm_dtype: int = PGCN_F32) -> int:
    return int(lib.pgcn_workspace_size(part.handle, f_in, f_out, gemm_dtype))


def pgcn_layer_workspace_size(part: Partition, f_in: int, f_out: int, gemm_dtype: int = PGCN_F32,
                              order: int = PGCN_ORDER_AGG) -> int:
    return int(lib.pgcn_layer_workspace_size(part.handle, f_in, f_out, gemm_dtype, order))


def pgcn_layer_fwd(part: Partition, *, f_in, f_out, gemm_dtype, relu, ld_in, ld_out, H_in, H_bd, W, A, A_bf16,
                   H_out, workspace, workspace_bytes, order=PGCN_ORDER_AGG, a_given=False, send_out=None,
                   stream=None):
    a = pgcn_fwd_args(f_in, f_out, gemm_dtype, int(relu), ld_in, ld_out, _ptr(H_in), _ptr(H_bd), _ptr(W),
                      _ptr(A), _ptr(A_bf16), _ptr(H_out), _ptr(workspace), workspace_bytes, order, int(a_given),
                      _ptr(send_out))
    _check(lib.pgcn_layer_fwd(part.handle, C.byref(a), _stream(stream)), "pgcn_layer_fwd")


def pgcn_layer_fwd_noalloc(part: Partition, *, f_in, f_out, gemm_dtype, relu, ld_in, ld_out, H_in, H_bd, W, A,
                           A_bf16, H_out, order=PGCN_ORDER_AGG, a_given=False, send_out=None, stream=None,
                           workspace=None, workspace_bytes=0):
    a = pgcn_fwd_args(f_in, f_out, gemm_dtype, int(relu), ld_in, ld_out, _ptr(H_in), _ptr(H_bd), _ptr(W),
                      _ptr(A), _ptr(A_bf16), _ptr(H_out), _ptr(workspace), workspace_bytes, order, int(a_given),
                      _ptr(send_out))
    _check(lib.pgcn_layer_fwd_noalloc(part.handle, C.byref(a), _stream(stream)), "pgcn_layer_fwd_noalloc")


def pgcn_layer_bwd(part: Partition, *, f_in, f_out, gemm_dtype, relu, ld_in, ld_out, J_out, H_out, A, A_bf16,
                   W, dW, J_in, J_bd_out, workspace, workspace_bytes, order=PGCN_ORDER_AGG, H_in=None, H_bd=None,
                   stream=None):
    a = pgcn_bwd_args(f_in, f_out, gemm_dtype, int(relu), ld_in, ld_out, _ptr(J_out), _ptr(H_out), _ptr(A),
                      _ptr(A_bf16), _ptr(W), _ptr(dW), _ptr(J_in), _ptr(J_bd_out), _ptr(workspace),
                      workspace_bytes, order, _ptr(H_in), _ptr(H_bd))
    _check(lib.pgcn_layer_bwd(part.handle, C.byref(a), _stream(stream)), "pgcn_layer_bwd")


def pgcn_smooth_ema(state, incoming, rows: int, cols: int, ld: int, gamma: float, stream=None):
    _check(lib.pgcn_smooth_ema(_ptr(state), _ptr(incoming), rows, cols, ld, gamma, _stream(stream)),
           "pgcn_smooth_ema")


def pgcn_pack_boundary(part: Partition, kind: int, src, dst, cols: int, ld: int, stream=None):
    _check(lib.pgcn_pack_boundary(part.handle, kind, _ptr(src), _ptr(dst), cols, ld, _stream(stream)),
           "pgcn_pack_boundary")


def pgcn_loss_fwd_bwd(kind: int, Z, rows: int, classes: int, ld: int, labels, targets, ld_t: int, scale: float,
                      J, loss_out, workspace, workspace_bytes: int, stream=None):
    _check(lib.pgcn_loss_fwd_bwd(kind, _ptr(Z), rows, classes, ld, _ptr(labels), _ptr(targets), ld_t, scale,
                                 _ptr(J), _ptr(loss_out), _ptr(workspace), workspace_bytes, _stream(stream)),
           "pgcn_loss_fwd_bwd")


def pgcn_sgd_update(W, G, G_peer, count: int, eta: float, stream=None):
    _check(lib.pgcn_sgd_update(_ptr(W), _ptr(G), _ptr(G_peer), count, eta, _stream(stream)), "pgcn_sgd_update")


def pgcn_adam_update(W, G, G_peer, m, v, count: int, lr: float, beta1: float, beta2: float, eps: float, t: int,
                     stream=None):
    _check(lib.pgcn_adam_update(_ptr(W), _ptr(G), _ptr(G_peer), _ptr(m), _ptr(v), count, lr, beta1, beta2, eps, t,
                                _stream(stream)), "pgcn_adam_update")


def pgcn_dropout(out, inp, rows: int, cols: int, ld: int, row0: int, p: float, seed: int, part: int, layer: int,
                 iteration: int, out_bf16=None, ld_bf16: int = 0, stream=None):
    _check(lib.pgcn_dropout(_ptr(out), _ptr(inp), rows, cols, ld, row0, p, seed, part, layer, iteration,
                            _ptr(out_bf16), ld_bf16, _stream(stream)), "pgcn_dropout")


def pgcn_sage_layer_fwd(part: Partition, *, f_in, f_out, gemm_dtype, relu, ld_in, ld_out, X_in, X_in_bf16, X_bd, W,
                        A, A_bf16, H_out, workspace, workspace_bytes, order=PGCN_ORDER_AGG, send_out=None,
                        stream=None):
    a = pgcn_sage_fwd_args(f_in, f_out, gemm_dtype, int(relu), ld_in, ld_out, _ptr(X_in), _ptr(X_in_bf16),
                           _ptr(X_bd), _ptr(W), _ptr(A), _ptr(A_bf16), _ptr(H_out), _ptr(workspace),
                           workspace_bytes, order, _ptr(send_out))
    _check(lib.pgcn_sage_layer_fwd(part.handle, C.byref(a), _stream(stream)), "pgcn_sage_layer_fwd")


def pgcn_sage_layer_bwd(part: Partition, *, f_in, f_out, gemm_dtype, relu, ld_in, ld_out, J_out, H_out, A, A_bf16,
                        X_in, X_in_bf16, W, dW, J_in, J_bd_out, workspace, workspace_bytes, order=PGCN_ORDER_AGG,
                        X_bd=None, stream=None):
    a = pgcn_sage_bwd_args(f_in, f_out, gemm_dtype, int(relu), ld_in, ld_out, _ptr(J_out), _ptr(H_out), _ptr(A),
                           _ptr(A_bf16), _ptr(X_in), _ptr(X_in_bf16), _ptr(W), _ptr(dW), _ptr(J_in),
                           _ptr(J_bd_out), _ptr(workspace), workspace_bytes, order, _ptr(X_bd))
    _check(lib.pgcn_sage_layer_bwd(part.handle, C.byref(a), _stream(stream)), "pgcn_sage_layer_bwd")


def pgcn_accum_smoothed(part: Partition, incoming, state, gamma: float, dst, cols: int, ld: int, stream=None):
    _check(lib.pgcn_accum_smoothed(part.handle, _ptr(incoming), _ptr(state), gamma, _ptr(dst), cols, ld,
                                   _stream(stream)), "pgcn_accum_smoothed")


def pgcn_refill_async(dst, src, nbytes: int, flags: int = 0, stream=None):
    _check(lib.pgcn_refill_async(_ptr(dst), _ptr(src), nbytes, flags, _stream(stream)), "pgcn_refill_async")


TRACE_KINDS = ["agg_fwd", "agg_bwd", "agg_fixup", "gemm_fwd", "gemm_dgrad", "gemm_wgrad", "wgrad_reduce", "ema",
               "pack", "accum", "loss", "sgd", "refill", "gemm_pack", "dropout", "adam", "mask_scale",
               "accum_ema"]


def pgcn_trace_enable(capacity: int):
    _check(lib.pgcn_trace_enable(capacity), "pgcn_trace_enable")


def pgcn_trace_filter(kinds=None):
    """Record only the named kinds (names of TRACE_KINDS); None records all."""
    mask = 0xFFFFFFFF if kinds is None else sum(1 << TRACE_KINDS.index(k) for k in kinds)
    _check(lib.pgcn_trace_filter(mask), "pgcn_trace_filter")


def pgcn_trace_collect(max_records: int = 1 << 16):
    """[(kind name, ms, launches)] of the records since the last collect (a record spans
    one launch, or the back-to-back chunk launches of one aggregation column range)."""
    kinds = np.zeros(max_records, np.int32)
    ms = np.zeros(max_records, np.float32)
    nl = np.zeros(max_records, np.int32)
    cnt = C.c_int32(0)
    _check(lib.pgcn_trace_collect(kinds.ctypes.data, ms.ctypes.data, nl.ctypes.data, max_records, C.byref(cnt)),
           "pgcn_trace_collect")
    n = cnt.value
    return [(TRACE_KINDS[k], float(v), int(c)) for k, v, c in zip(kinds[:n], ms[:n], nl[:n])]


def pgcn_trace_disable():
    _check(lib.pgcn_trace_disable(), "pgcn_trace_disable")


def pgcn_last_error() -> str:
    return lib.pgcn_last_error().decode(errors="replace")


def pgcn_version() -> int:
    return int(lib.pgcn_version())
