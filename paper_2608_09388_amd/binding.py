"""Python binding of libshc.so: the same entry points, torch tensors in.

Argument marshalling only -- every step of the path runs in the library's HIP
kernels.  PyTorch supplies device memory and the current HIP stream.  Before
any call the binding checks that every tensor is on the GPU, contiguous, of
the expected dtype and large enough for the sizes passed, so a kernel never
sees a buffer smaller than its launch assumes.  There is no fallback: if
libshc.so is missing or cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libshc.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "shc.h")

SHC_F32, SHC_BF16 = 0, 1
SHC_ACT_NONE, SHC_ACT_RELU = 0, 1
SHC_COMBINE_SUM, SHC_COMBINE_MEAN, SHC_COMBINE_MAX = 0, 1, 2
# largest V shc_compact_mask_table_start takes
COMPACT_TABLE_MAX_V = 19456
COMBINE = {"sum": SHC_COMBINE_SUM, "mean": SHC_COMBINE_MEAN, "max": SHC_COMBINE_MAX}
STATUS = {0: "SHC_OK", -1: "SHC_ERR_INVALID_ARG", -2: "SHC_ERR_CAPACITY",
          -3: "SHC_ERR_MISALIGNED", -4: "SHC_ERR_UNSUPPORTED", -5: "SHC_ERR_HIP"}


class ShcError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")


_lib = None

_c_i32, _c_i64, _c_ptr, _c_sz, _c_f = (ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p,
                                        ctypes.c_size_t, ctypes.c_float)

# stack executor (shc_stack_*): mirrors of the C structs, same field order
STACK_MAX_LAYERS = 16
SHC_LAYER_LINEAR, SHC_LAYER_CONV = 0, 1


class StackLayer(ctypes.Structure):
    _fields_ = [("kind", _c_i32), ("Cin", _c_i32), ("Cout", _c_i32), ("act", _c_i32),
                ("W", _c_ptr), ("bias", _c_ptr), ("plan_rows", _c_i64), ("split_rows", _c_i64),
                ("Wp", _c_ptr), ("packed_rows", _c_i64), ("packed_min_rows", _c_i64)]


class StackIndexSet(ctypes.Structure):
    _fields_ = [("coords", _c_ptr), ("inv", _c_ptr), ("row_ptr", _c_ptr), ("n_active", _c_ptr),
                ("host_count", _c_ptr), ("ws", _c_ptr), ("ws_bytes", _c_sz), ("table", _c_ptr),
                ("plan", _c_ptr * STACK_MAX_LAYERS), ("plan_bytes", _c_sz * STACK_MAX_LAYERS)]


class StackDesc(ctypes.Structure):
    _fields_ = [("B", _c_i32), ("V", _c_i32), ("K", _c_i32), ("dtype", _c_i32), ("C0", _c_i32),
                ("mask", _c_ptr), ("x", _c_ptr), ("nbr", _c_ptr),
                ("table_in_compaction", _c_i32), ("n_layers", _c_i32),
                ("layers", StackLayer * STACK_MAX_LAYERS),
                ("acts", _c_ptr * (STACK_MAX_LAYERS + 1)), ("last_alt", _c_ptr),
                ("dense_out", _c_ptr), ("incremental", _c_i32), ("prev_coords", _c_ptr),
                ("pooled", _c_ptr), ("pool_empty", _c_f), ("n_sets", _c_i32),
                ("sets", StackIndexSet * 3), ("side", _c_ptr), ("tail", _c_ptr),
                ("split_ws", _c_ptr), ("split_ws_bytes", _c_sz)]


STACK_FEED_FN = ctypes.CFUNCTYPE(ctypes.c_int, _c_ptr, _c_i64, _c_ptr)
_SIGS = {
    "shc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "shc_last_error": (ctypes.c_char_p, []),
    "shc_compact_mask_workspace": (_c_sz, [_c_i32, _c_i32]),
    "shc_compact_mask": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                        _c_ptr, _c_i64, _c_ptr, _c_sz, _c_ptr]),
    "shc_compact_mask_noalloc": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr,
                                                _c_ptr, _c_ptr, _c_i64, _c_ptr]),
    "shc_compact_mask_start": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr,
                                              _c_ptr, _c_ptr, _c_i64, _c_ptr, _c_sz, _c_ptr]),
    "shc_compact_mask_wait": (ctypes.c_int, [_c_ptr, _c_i64, _c_ptr]),
    "shc_compact_mask_table_start": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_ptr, _c_ptr,
                                                    _c_ptr, _c_ptr, _c_ptr, _c_i64, _c_ptr,
                                                    _c_i32, _c_ptr, _c_ptr, _c_sz, _c_ptr]),
    "shc_scatter_update": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_ptr, _c_i64, _c_i32,
                                          _c_i32, _c_i32, _c_i32, _c_ptr, _c_ptr]),
    "shc_clear_inactive_rows": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_i32, _c_i32, _c_ptr,
                                               _c_ptr]),
    "shc_gather_rows": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32,
                                       _c_ptr, _c_ptr]),
    "shc_gather_rows_stacked": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32,
                                               _c_i32, _c_i32, _c_ptr, _c_ptr]),
    "shc_gather_rows_masked": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32,
                                              _c_i32, _c_i32, _c_ptr, _c_ptr]),
    "shc_row_mask_from_elements": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_i32, _c_ptr,
                                                  _c_ptr]),
    "shc_combine_stacked": (ctypes.c_int, [_c_ptr, _c_i32, _c_i64, _c_i32, _c_i32, _c_i32,
                                           _c_ptr, _c_ptr]),
    "shc_sparse_linear": (ctypes.c_int, [_c_ptr, _c_i64, _c_ptr, _c_ptr, _c_i32, _c_i32, _c_i32,
                                         _c_i32, _c_ptr, _c_ptr]),
    "shc_gather_sparse_linear": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_ptr,
                                                _c_ptr, _c_i32, _c_i32, _c_i32, _c_i32, _c_ptr,
                                                _c_ptr]),
    "shc_sparse_neighbor_conv": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32,
                                                _c_ptr, _c_i32, _c_ptr, _c_ptr, _c_i32, _c_i32,
                                                _c_i32, _c_i32, _c_ptr, _c_ptr]),
    "shc_build_neighbor_table": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_ptr,
                                                _c_i32, _c_ptr, _c_ptr]),
    "shc_sparse_neighbor_conv_table": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_ptr,
                                                      _c_ptr, _c_i32, _c_i32, _c_i32, _c_i32,
                                                      _c_ptr, _c_ptr]),
    "shc_conv_split_workspace_bytes": (_c_sz, [_c_i64, _c_i32, _c_i32, _c_i32, _c_i32]),
    "shc_sparse_neighbor_conv_split": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_ptr,
                                                      _c_ptr, _c_i32, _c_i32, _c_i32, _c_i32,
                                                      _c_ptr, _c_ptr, _c_sz, _c_ptr]),
    "shc_conv_packed_weights_bytes": (_c_sz, [_c_i32, _c_i32, _c_i32, _c_i32]),
    "shc_pack_conv_weights": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_i32, _c_i32, _c_ptr,
                                             _c_sz, _c_ptr]),
    "shc_sparse_neighbor_conv_packed": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_ptr,
                                                       _c_ptr, _c_i32, _c_i32, _c_i32, _c_i32,
                                                       _c_ptr, _c_ptr]),
    "shc_conv_packed_plan_bytes": (_c_sz, [_c_i64, _c_i32, _c_i32, _c_i32, _c_i32]),
    "shc_build_conv_packed_plan": (ctypes.c_int, [_c_ptr, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32,
                                                  _c_ptr, _c_sz, _c_ptr]),
    "shc_sparse_neighbor_conv_packed_planned": (ctypes.c_int, [_c_ptr, _c_ptr, _c_sz, _c_i64,
                                                               _c_i32, _c_ptr, _c_ptr, _c_i32,
                                                               _c_i32, _c_i32, _c_i32, _c_ptr,
                                                               _c_ptr]),
    "shc_conv_plan_max_rows": (_c_i64, [_c_i32, _c_i32, _c_i32, _c_i32]),
    "shc_conv_plan_bytes": (_c_sz, [_c_i64, _c_i32, _c_i32, _c_i32, _c_i32]),
    "shc_build_conv_plan": (ctypes.c_int, [_c_ptr, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32,
                                           _c_ptr, _c_sz, _c_ptr]),
    "shc_sparse_neighbor_conv_planned": (ctypes.c_int, [_c_ptr, _c_ptr, _c_sz, _c_i64, _c_i32,
                                                        _c_ptr, _c_ptr, _c_i32, _c_i32, _c_i32,
                                                        _c_i32, _c_ptr, _c_ptr]),
    "shc_scatter": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32, _c_i32,
                                   _c_i32, _c_ptr, _c_ptr]),
    "shc_segment_group_norm": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32,
                                              _c_f, _c_i32, _c_ptr, _c_ptr]),
    "shc_mask_scores_workspace": (_c_sz, [_c_i32, _c_i64, _c_i32]),
    "shc_mask_scores": (ctypes.c_int, [_c_ptr, _c_i32, _c_i64, _c_i32, _c_i32, _c_ptr, _c_ptr,
                                       _c_ptr, _c_i32, _c_ptr, _c_ptr, _c_sz, _c_ptr]),
    "shc_segment_maxpool": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32, _c_f,
                                           _c_ptr, _c_ptr]),
    "shc_transpose_neighbors_workspace": (_c_sz, [_c_i32, _c_i32]),
    "shc_transpose_neighbors": (ctypes.c_int, [_c_ptr, _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr,
                                               _c_ptr, _c_sz, _c_ptr]),
    "shc_build_transposed_table": (ctypes.c_int, [_c_ptr, _c_ptr, _c_i64, _c_i32, _c_i32, _c_ptr,
                                                  _c_i32, _c_ptr, _c_ptr, _c_ptr]),
    "shc_sparse_linear_backward_workspace": (_c_sz, [_c_i64, _c_i32, _c_i32, _c_i32]),
    "shc_sparse_linear_backward": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i32,
                                                  _c_i32, _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr,
                                                  _c_ptr, _c_sz, _c_ptr]),
    "shc_sparse_neighbor_conv_backward_workspace": (_c_sz, [_c_i64, _c_i32, _c_i32, _c_i32,
                                                            _c_i32]),
    "shc_build_slot_pairs_workspace": (_c_sz, [_c_i64, _c_i32]),
    "shc_build_slot_pairs": (ctypes.c_int, [_c_ptr, _c_i64, _c_i32, _c_ptr, _c_ptr, _c_ptr, _c_sz,
                                            _c_ptr]),
    "shc_sparse_neighbor_conv_backward": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                                         _c_ptr, _c_ptr, _c_i32, _c_ptr, _c_ptr,
                                                         _c_ptr, _c_i64, _c_i32, _c_i32, _c_i32,
                                                         _c_i32, _c_i32, _c_ptr, _c_ptr, _c_ptr,
                                                         _c_ptr, _c_sz, _c_ptr]),
    "shc_event_create": (ctypes.c_int, [ctypes.POINTER(_c_ptr)]),
    "shc_event_record": (ctypes.c_int, [_c_ptr, _c_ptr]),
    "shc_stream_wait_event": (ctypes.c_int, [_c_ptr, _c_ptr]),
    "shc_event_synchronize": (ctypes.c_int, [_c_ptr]),
    "shc_event_destroy": (ctypes.c_int, [_c_ptr]),
    "shc_stack_create": (ctypes.c_int, [ctypes.POINTER(StackDesc), ctypes.POINTER(_c_ptr)]),
    "shc_stack_run": (ctypes.c_int, [_c_ptr, _c_i64, _c_ptr, STACK_FEED_FN, _c_ptr, _c_i32,
                                     _c_ptr, ctypes.POINTER(_c_i32), ctypes.POINTER(_c_i64),
                                     ctypes.POINTER(_c_i64)]),
    "shc_stack_destroy": (ctypes.c_int, [_c_ptr]),
}


def load(path: Optional[str] = None):
    """Load libshc.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    # SHC_LIB may name another build of the library (same ABI)
    p = path or os.environ.get("SHC_LIB") or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is not built: run `python -m paper_2608_09388_amd.build`")
    lib = ctypes.CDLL(p)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def header_symbols(header: str = HEADER):
    """Names of the functions include/shc.h declares."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(shc_[a-z_]+)\s*\(", text)))


def _check(rc: int, where: str):
    if rc != 0:
        detail = load().shc_last_error().decode(errors="replace")
        raise ShcError(rc, where, detail)


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SHC_F32
    if t.dtype == torch.bfloat16:
        return SHC_BF16
    raise TypeError(f"feature tensors must be float32 or bfloat16, got {t.dtype}")


def _dev(t: torch.Tensor, name: str, dtype=None, min_numel: int = 0):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {min_numel}")
    return t.data_ptr()


def _opt_dev(t, name, dtype=None, min_numel=0):
    return None if t is None else _dev(t, name, dtype, min_numel)


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI, minus the prefix)
# ----------------------------------------------------------------------------


def compact_mask_workspace(B: int, V: int) -> int:
    return int(load().shc_compact_mask_workspace(B, V))


def _host_count_ptr(host_count: Optional[torch.Tensor]) -> int:
    if not isinstance(host_count, torch.Tensor) or host_count.is_cuda or \
            host_count.dtype != torch.int64 or host_count.numel() < 1:
        raise ValueError("host_count must be a CPU int64 tensor of at least one element")
    return host_count.data_ptr()


def compact_mask(mask: torch.Tensor, B: int, V: int, coords: torch.Tensor, inv: torch.Tensor,
                 row_ptr: torch.Tensor, n_active: torch.Tensor, ws: torch.Tensor,
                 want_host_count: bool = True, stream=None,
                 host_count: Optional[torch.Tensor] = None) -> Optional[int]:
    """shc_compact_mask.  ``coords`` is int32 [cap][2]; returns N' if asked (syncs).

    ``host_count`` (optional) is a CPU int64 tensor that receives N'; when it
    is pinned (``pin_memory=True``) the kernel writes it directly.
    """
    lib = load()
    cap = coords.numel() // 2
    args = [_dev(mask, "mask", torch.uint8, B * V), B, V,
            _dev(coords, "coords", torch.int32) if cap > 0 else None,
            _dev(inv, "inv", torch.int32, B * V), _dev(row_ptr, "row_ptr", torch.int32, B + 1),
            _dev(n_active, "n_active", torch.int32, 1)]
    host = ctypes.c_int64(-1)
    if host_count is not None:
        hp = _host_count_ptr(host_count)
    else:
        hp = ctypes.addressof(host) if want_host_count else None
    args += [hp, cap, _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)]
    _check(lib.shc_compact_mask(*args), "shc_compact_mask")
    if host_count is not None:
        return int(host_count[0])
    return int(host.value) if want_host_count else None


def compact_mask_noalloc(mask: torch.Tensor, B: int, V: int, coords: torch.Tensor,
                         inv: torch.Tensor, row_ptr: torch.Tensor, n_active: torch.Tensor,
                         want_host_count: bool = True, stream=None,
                         host_count: Optional[torch.Tensor] = None) -> Optional[int]:
    """shc_compact_mask_noalloc: shc_compact_mask with the library's own scratch
    instead of a workspace.  Arguments and result as for compact_mask."""
    lib = load()
    cap = coords.numel() // 2
    args = [_dev(mask, "mask", torch.uint8, B * V), B, V,
            _dev(coords, "coords", torch.int32) if cap > 0 else None,
            _dev(inv, "inv", torch.int32, B * V), _dev(row_ptr, "row_ptr", torch.int32, B + 1),
            _dev(n_active, "n_active", torch.int32, 1)]
    host = ctypes.c_int64(-1)
    if host_count is not None:
        hp = _host_count_ptr(host_count)
    else:
        hp = ctypes.addressof(host) if want_host_count else None
    args += [hp, cap, _stream(stream)]
    _check(lib.shc_compact_mask_noalloc(*args), "shc_compact_mask_noalloc")
    if host_count is not None:
        return int(host_count[0])
    return int(host.value) if want_host_count else None


def gather_rows(x: torch.Tensor, coords: torch.Tensor, n_rows: int, B: int, V: int,
                S: torch.Tensor, stream=None):
    """shc_gather_rows: S[i] = x[b_i * V + v_i]."""
    C = x.shape[-1]
    dt = _dtype_code(x)
    args = [_dev(x, "x", x.dtype, B * V * C), _dev(coords, "coords", torch.int32, 2 * n_rows),
            n_rows, B, V, C, dt, _dev(S, "S", x.dtype, n_rows * C), _stream(stream)]
    _check(load().shc_gather_rows(*args), "shc_gather_rows")


def gather_rows_stacked(x: torch.Tensor, coords: torch.Tensor, n_rows: int, B: int,
                        kappa: int, V: int, S: torch.Tensor, stream=None):
    """shc_gather_rows_stacked: S[i] = x[(b'_i mod B) * V + v_i]."""
    C = x.shape[-1]
    args = [_dev(x, "x", x.dtype, B * V * C), _dev(coords, "coords", torch.int32, 2 * n_rows),
            n_rows, B, kappa, V, C, _dtype_code(x), _dev(S, "S", x.dtype, n_rows * C),
            _stream(stream)]
    _check(load().shc_gather_rows_stacked(*args), "shc_gather_rows_stacked")


def gather_rows_masked(x: torch.Tensor, me: torch.Tensor, coords: torch.Tensor, n_rows: int,
                       B: int, V: int, S: torch.Tensor, stream=None):
    """shc_gather_rows_masked: gathered rows times the per-element mask ``me`` [B*V][C]."""
    C = x.shape[-1]
    args = [_dev(x, "x", x.dtype, B * V * C), _dev(me, "me", torch.uint8, B * V * C),
            _dev(coords, "coords", torch.int32, 2 * n_rows), n_rows, B, V, C, _dtype_code(x),
            _dev(S, "S", x.dtype, n_rows * C), _stream(stream)]
    _check(load().shc_gather_rows_masked(*args), "shc_gather_rows_masked")


def row_mask_from_elements(me: torch.Tensor, B: int, V: int, m: torch.Tensor, stream=None):
    """shc_row_mask_from_elements: m[b*V + v] = any(me[b*V + v, :])."""
    C = me.numel() // (B * V)
    args = [_dev(me, "me", torch.uint8, B * V * C), B, V, C, _dev(m, "m", torch.uint8, B * V),
            _stream(stream)]
    _check(load().shc_row_mask_from_elements(*args), "shc_row_mask_from_elements")


def combine_stacked(Y: torch.Tensor, kappa: int, rows: int, out: torch.Tensor, op="mean",
                    stream=None):
    """shc_combine_stacked: out[r] = op over k of Y[k * rows + r] ('sum', 'mean', 'max')."""
    C = Y.shape[-1]
    args = [_dev(Y, "Y", Y.dtype, kappa * rows * C), kappa, rows, C, _dtype_code(Y),
            COMBINE[op] if isinstance(op, str) else int(op), _dev(out, "out", Y.dtype, rows * C),
            _stream(stream)]
    _check(load().shc_combine_stacked(*args), "shc_combine_stacked")


def sparse_linear(S: torch.Tensor, n_rows: int, W: torch.Tensor, bias: Optional[torch.Tensor],
                  out: torch.Tensor, act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_linear: out = act(S W + bias), W [Cin][Cout]."""
    Cin, Cout = W.shape
    dt = _dtype_code(S)
    args = [_dev(S, "S", S.dtype, n_rows * Cin), n_rows, _dev(W, "W", S.dtype, Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, dt, act,
            _dev(out, "out", S.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_sparse_linear(*args), "shc_sparse_linear")


def gather_sparse_linear(x: torch.Tensor, coords: torch.Tensor, n_rows: int, B: int, V: int,
                         W: torch.Tensor, bias: Optional[torch.Tensor], out: torch.Tensor,
                         act: int = SHC_ACT_RELU, stream=None):
    """shc_gather_sparse_linear: out[i] = act(x[b_i * V + v_i] W + bias)."""
    Cin, Cout = W.shape
    dt = _dtype_code(x)
    args = [_dev(x, "x", x.dtype, B * V * Cin), _dev(coords, "coords", torch.int32, 2 * n_rows),
            n_rows, B, V, _dev(W, "W", x.dtype, Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, dt, act,
            _dev(out, "out", x.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_gather_sparse_linear(*args), "shc_gather_sparse_linear")


def sparse_neighbor_conv(S: torch.Tensor, coords: torch.Tensor, inv: torch.Tensor, n_rows: int,
                         B: int, V: int, nbr: torch.Tensor, W: torch.Tensor,
                         bias: Optional[torch.Tensor], out: torch.Tensor,
                         act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv: W [K][Cin][Cout], nbr [V][K]."""
    K, Cin, Cout = W.shape
    dt = _dtype_code(S)
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(coords, "coords", torch.int32, 2 * n_rows),
            _dev(inv, "inv", torch.int32, B * V), n_rows, B, V,
            _dev(nbr, "nbr", torch.int32, V * K), K, _dev(W, "W", S.dtype, K * Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, dt, act,
            _dev(out, "out", S.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv(*args), "shc_sparse_neighbor_conv")


def build_neighbor_table(coords: torch.Tensor, inv: torch.Tensor, n_rows: int, B: int, V: int,
                         nbr: torch.Tensor, table: torch.Tensor, stream=None):
    """shc_build_neighbor_table: table[j * n_rows + i] = neighbour row of slot j, or -1."""
    K = nbr.shape[-1]
    args = [_dev(coords, "coords", torch.int32, 2 * n_rows), _dev(inv, "inv", torch.int32, B * V),
            n_rows, B, V, _dev(nbr, "nbr", torch.int32, V * K), K,
            _dev(table, "table", torch.int32, K * n_rows), _stream(stream)]
    _check(load().shc_build_neighbor_table(*args), "shc_build_neighbor_table")


def sparse_neighbor_conv_table(S: torch.Tensor, table: torch.Tensor, n_rows: int,
                               W: torch.Tensor, bias: Optional[torch.Tensor], out: torch.Tensor,
                               act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv_table: W [K][Cin][Cout], table from build_neighbor_table."""
    K, Cin, Cout = W.shape
    dt = _dtype_code(S)
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(table, "table", torch.int32, K * n_rows),
            n_rows, K, _dev(W, "W", S.dtype, K * Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, dt, act,
            _dev(out, "out", S.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_table(*args), "shc_sparse_neighbor_conv_table")


def conv_split_workspace_bytes(n_rows: int, K: int, Cin: int, Cout: int,
                               dtype: int = SHC_BF16) -> int:
    """shc_conv_split_workspace_bytes: workspace of a split conv of up to
    n_rows rows (0 when the shape takes none)."""
    return int(load().shc_conv_split_workspace_bytes(n_rows, K, Cin, Cout, dtype))


def sparse_neighbor_conv_split(S: torch.Tensor, table: torch.Tensor, n_rows: int,
                               W: torch.Tensor, bias: Optional[torch.Tensor], out: torch.Tensor,
                               workspace: torch.Tensor, act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv_split: the conv of sparse_neighbor_conv_table
    with slot 0 and the other slots apart; workspace a device byte buffer of at
    least conv_split_workspace_bytes(n_rows, ...) bytes."""
    K, Cin, Cout = W.shape
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(table, "table", torch.int32, K * n_rows),
            n_rows, K, _dev(W, "W", S.dtype, K * Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, _dtype_code(S), act,
            _dev(out, "out", S.dtype, n_rows * Cout), _dev(workspace, "workspace"),
            workspace.numel() * workspace.element_size(), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_split(*args), "shc_sparse_neighbor_conv_split")


def conv_packed_weights_bytes(K: int, Cin: int, Cout: int, dtype: int = SHC_BF16) -> int:
    """shc_conv_packed_weights_bytes: bytes of the packed weights (0: the
    shape has no packed conv)."""
    return int(load().shc_conv_packed_weights_bytes(K, Cin, Cout, dtype))


def pack_conv_weights(W: torch.Tensor, Wp: torch.Tensor, stream=None):
    """shc_pack_conv_weights: W [K][Cin][Cout] bf16 into the device buffer Wp
    (conv_packed_weights_bytes bytes)."""
    K, Cin, Cout = W.shape
    args = [_dev(W, "W", W.dtype, K * Cin * Cout), K, Cin, Cout, _dtype_code(W),
            _dev(Wp, "Wp"), Wp.numel() * Wp.element_size(), _stream(stream)]
    _check(load().shc_pack_conv_weights(*args), "shc_pack_conv_weights")


def sparse_neighbor_conv_packed(S: torch.Tensor, table: torch.Tensor, n_rows: int,
                                Wp: torch.Tensor, K: int, Cin: int, Cout: int,
                                bias: Optional[torch.Tensor], out: torch.Tensor,
                                act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv_packed: the conv of sparse_neighbor_conv_table
    with weights from pack_conv_weights."""
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(table, "table", torch.int32, K * n_rows),
            n_rows, K, _dev(Wp, "Wp"), _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout,
            _dtype_code(S), act, _dev(out, "out", S.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_packed(*args), "shc_sparse_neighbor_conv_packed")


def conv_plan_max_rows(K: int, Cin: int, Cout: int, dtype: int = SHC_BF16) -> int:
    """shc_conv_plan_max_rows: largest active-row count with a plan (0: none)."""
    return int(load().shc_conv_plan_max_rows(K, Cin, Cout, dtype))


def conv_plan_bytes(n_rows: int, K: int, Cin: int, Cout: int, dtype: int = SHC_BF16) -> int:
    """shc_conv_plan_bytes: a buffer for the plan of any set of <= n_rows rows
    (0 when none takes a plan)."""
    return int(load().shc_conv_plan_bytes(n_rows, K, Cin, Cout, dtype))


def build_conv_plan(table: torch.Tensor, n_rows: int, K: int, Cin: int, Cout: int,
                    plan: torch.Tensor, dtype: int = SHC_BF16, stream=None):
    """shc_build_conv_plan: table [K][n_rows] (int32), plan a device byte buffer."""
    args = [_dev(table, "table", torch.int32, K * n_rows), n_rows, K, Cin, Cout, dtype,
            _dev(plan, "plan"), plan.numel() * plan.element_size(), _stream(stream)]
    _check(load().shc_build_conv_plan(*args), "shc_build_conv_plan")


def sparse_neighbor_conv_planned(S: torch.Tensor, plan: torch.Tensor, n_rows: int,
                                 W: torch.Tensor, bias: Optional[torch.Tensor], out: torch.Tensor,
                                 act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv_planned: W [K][Cin][Cout], plan from build_conv_plan."""
    K, Cin, Cout = W.shape
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(plan, "plan"),
            plan.numel() * plan.element_size(), n_rows, K,
            _dev(W, "W", S.dtype, K * Cin * Cout), _opt_dev(bias, "bias", torch.float32, Cout),
            Cin, Cout, _dtype_code(S), act, _dev(out, "out", S.dtype, n_rows * Cout),
            _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_planned(*args), "shc_sparse_neighbor_conv_planned")


def scatter(S: torch.Tensor, inv: torch.Tensor, coords: torch.Tensor, n_rows: int, B: int,
            V: int, D: torch.Tensor, zero_fill: bool = True, stream=None):
    """shc_scatter: compact rows back to D [B*V][C]."""
    C = D.shape[-1]
    dt = _dtype_code(D)
    args = [_opt_dev(S, "S", D.dtype, n_rows * C) if n_rows > 0 else None,
            _dev(inv, "inv", torch.int32, B * V) if zero_fill else None,
            _dev(coords, "coords", torch.int32, 2 * n_rows) if (not zero_fill and n_rows) else None,
            n_rows, B, V, C, dt, 1 if zero_fill else 0, _dev(D, "D", D.dtype, B * V * C),
            _stream(stream)]
    _check(load().shc_scatter(*args), "shc_scatter")


def scatter_update(S: torch.Tensor, inv: torch.Tensor, coords: torch.Tensor, n_rows: int,
                   prev_coords: torch.Tensor, prev_rows: int, B: int, V: int, D: torch.Tensor,
                   stream=None):
    """shc_scatter_update: D held the zero-fill scatter of prev_coords[:prev_rows];
    afterwards it holds this set's."""
    C = D.shape[-1]
    args = [_dev(S, "S", D.dtype, n_rows * C) if n_rows else None,
            _dev(inv, "inv", torch.int32, B * V),
            _dev(coords, "coords", torch.int32, 2 * n_rows) if n_rows else None, n_rows,
            _dev(prev_coords, "prev_coords", torch.int32, 2 * prev_rows) if prev_rows else None,
            prev_rows, B, V, C, _dtype_code(D), _dev(D, "D", D.dtype, B * V * C), _stream(stream)]
    _check(load().shc_scatter_update(*args), "shc_scatter_update")


def prepare_scatter_update(S, inv, coords, prev_coords, B, V, D, stream=None) -> "Prepared":
    """shc_scatter_update with (n_rows, prev_rows) given per call."""
    C = D.shape[-1]
    args = [_dev(S, "S", D.dtype), _dev(inv, "inv", torch.int32, B * V),
            _dev(coords, "coords", torch.int32), 0, _dev(prev_coords, "prev_coords", torch.int32),
            0, B, V, C, _dtype_code(D), _dev(D, "D", D.dtype, B * V * C), _stream(stream)]
    return PreparedScatterUpdate(args, (S, inv, coords, prev_coords, D),
                                 min(S.numel() // C, coords.numel() // 2),
                                 prev_coords.numel() // 2)


def compact_mask_start(mask: torch.Tensor, B: int, V: int, coords: torch.Tensor,
                       inv: torch.Tensor, row_ptr: torch.Tensor, n_active: torch.Tensor,
                       ws: torch.Tensor, host_count: torch.Tensor, stream=None):
    """shc_compact_mask_start: launch only; ``host_count`` is a pinned CPU int64
    tensor that receives N' (read it after ``compact_mask_wait``)."""
    cap = coords.numel() // 2
    args = [_dev(mask, "mask", torch.uint8, B * V), B, V,
            _dev(coords, "coords", torch.int32) if cap > 0 else None,
            _dev(inv, "inv", torch.int32, B * V), _dev(row_ptr, "row_ptr", torch.int32, B + 1),
            _dev(n_active, "n_active", torch.int32, 1), _host_count_ptr(host_count), cap,
            _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)]
    _check(load().shc_compact_mask_start(*args), "shc_compact_mask_start")


def compact_mask_wait(host_count: torch.Tensor, cap: int, stream=None) -> int:
    """shc_compact_mask_wait: N' once it has arrived in ``host_count``."""
    _check(load().shc_compact_mask_wait(_host_count_ptr(host_count), cap, _stream(stream)),
           "shc_compact_mask_wait")
    return int(host_count[0])


def clear_inactive_rows(inv: torch.Tensor, B: int, V: int, D: torch.Tensor, stream=None):
    """shc_clear_inactive_rows: D[r] = 0 wherever inv[r] < 0, other rows untouched."""
    C = D.shape[-1]
    args = [_dev(inv, "inv", torch.int32, B * V), B, V, C, _dtype_code(D),
            _dev(D, "D", D.dtype, B * V * C), _stream(stream)]
    _check(load().shc_clear_inactive_rows(*args), "shc_clear_inactive_rows")


def segment_group_norm(S: torch.Tensor, row_ptr: torch.Tensor, n_rows: int, B: int, G: int,
                       out: torch.Tensor, eps: float = 1e-5, stream=None):
    """shc_segment_group_norm: per body and channel group, over the active rows."""
    C = S.shape[-1]
    dt = _dtype_code(S)
    args = [_dev(S, "S", S.dtype, n_rows * C) if n_rows > 0 else None,
            _dev(row_ptr, "row_ptr", torch.int32, B + 1), n_rows, B, C, G, float(eps), dt,
            _dev(out, "out", S.dtype, n_rows * C) if n_rows > 0 else None, _stream(stream)]
    _check(load().shc_segment_group_norm(*args), "shc_segment_group_norm")


def prepare_segment_group_norm(S, row_ptr, B, G, out, eps=1e-5, stream=None) -> Prepared:
    C = S.shape[-1]
    n_max = min(S.numel() // C, out.numel() // C)
    args = [_dev(S, "S", S.dtype), _dev(row_ptr, "row_ptr", torch.int32, B + 1), 0, B, C, G,
            float(eps), _dtype_code(S), _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_segment_group_norm", args, 2, n_max, (S, row_ptr, out))


def mask_scores_workspace(K: int, N: int, C: int) -> int:
    return int(load().shc_mask_scores_workspace(K, N, C))


def mask_scores(O: torch.Tensor, alpha_in: Optional[torch.Tensor], alpha_out: torch.Tensor,
                kappa: int = 0, top: Optional[torch.Tensor] = None,
                sim: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """shc_mask_scores on O [K][N][C] bf16; returns the workspace used."""
    K, N, C = O.shape
    need = mask_scores_workspace(K, N, C)
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=O.device)
    args = [_dev(O, "O", torch.bfloat16, K * N * C), K, N, C, _dtype_code(O),
            _opt_dev(alpha_in, "alpha_in", torch.float64, K),
            _dev(alpha_out, "alpha_out", torch.float64, K),
            _opt_dev(sim, "sim", torch.float64, K * K), kappa,
            _opt_dev(top, "top", torch.int32, kappa), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    _check(load().shc_mask_scores(*args), "shc_mask_scores")
    return ws


def segment_maxpool(S: torch.Tensor, row_ptr: torch.Tensor, n_rows: int, B: int,
                    P: torch.Tensor, empty_value: float = 0.0, stream=None):
    """shc_segment_maxpool: P [B][C] = per-body max of the active rows."""
    C = P.shape[-1]
    dt = _dtype_code(P)
    args = [_dev(S, "S", P.dtype, n_rows * C) if n_rows > 0 else None,
            _dev(row_ptr, "row_ptr", torch.int32, B + 1), n_rows, B, C, dt, float(empty_value),
            _dev(P, "P", P.dtype, B * C), _stream(stream)]
    _check(load().shc_segment_maxpool(*args), "shc_segment_maxpool")


class StackExecutor:
    """shc_stack_create / shc_stack_run / shc_stack_destroy.  ``desc`` is a
    filled StackDesc; ``keep`` holds the tensors it points into (alive as
    long as the executor)."""

    def __init__(self, desc: StackDesc, keep=()):
        lib = load()
        h = _c_ptr()
        self._desc, self._keep = desc, keep
        _check(lib.shc_stack_create(ctypes.byref(desc), ctypes.byref(h)), "shc_stack_create")
        self._h = h
        self._destroy = lib.shc_stack_destroy

    def run(self, steps: int, stream=None, feed=None, time_layer: int = 0, time_events=None,
            cur_set: int = 0, prev_rows: int = 0):
        """shc_stack_run; returns (n_last, cur_set, prev_rows).  ``feed(k,
        stream_handle)`` is called for every batch; an exception it raises
        ends the run and is raised here.  ``time_events``: 2 * steps HIP event
        handles (int, 0 for none) or None."""
        err = []

        def _feed(user, k, st):
            try:
                feed(int(k), st or 0)
                return 0
            except BaseException as e:  # noqa: BLE001 -- re-raised below
                err.append(e)
                return 1

        cb = STACK_FEED_FN(_feed) if feed is not None else ctypes.cast(None, STACK_FEED_FN)
        ev = None
        if time_events is not None:
            if len(time_events) != 2 * steps:
                raise ValueError(f"time_events holds {len(time_events)} handles, "
                                 f"not 2 * steps = {2 * steps}")
            ev = (_c_ptr * (2 * steps))(*[int(e) if e else None for e in time_events])
        cur = _c_i32(cur_set)
        prev = _c_i64(prev_rows)
        n = _c_i64(0)
        rc = load().shc_stack_run(self._h, steps, _stream(stream), cb, None, time_layer, ev,
                                  ctypes.byref(cur), ctypes.byref(prev), ctypes.byref(n))
        if err:
            raise err[0]
        _check(rc, "shc_stack_run")
        return int(n.value), int(cur.value), int(prev.value)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._destroy(h)
            self._h = None


class StreamEvent:
    """shc_event_*: orders work between streams of one device, and lets the
    host wait for it, without a system-scope fence at each record.  Created on
    the current device."""

    def __init__(self):
        lib = load()
        h = _c_ptr()
        _check(lib.shc_event_create(ctypes.byref(h)), "shc_event_create")
        self._h = h
        self._destroy = lib.shc_event_destroy

    def record(self, stream=None):
        _check(load().shc_event_record(self._h, _stream(stream)), "shc_event_record")

    def wait(self, stream=None):
        """Work enqueued on ``stream`` after this call waits for the last record."""
        _check(load().shc_stream_wait_event(_stream(stream), self._h), "shc_stream_wait_event")

    def synchronize(self):
        _check(load().shc_event_synchronize(self._h), "shc_event_synchronize")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self._destroy(h)
            self._h = None


# ----------------------------------------------------------------------------
# backward of the linear and conv layers
# ----------------------------------------------------------------------------

SHC_MAX_VIRTUAL_SLOTS = 64


def transpose_neighbors(nbr: torch.Tensor, stream=None):
    """shc_transpose_neighbors on nbr [V][K] int32 (device).  Returns
    (nbr_t [V][64] int32, slot_of [64] int32, Kt); waits for the stream."""
    V, K = nbr.shape
    need = int(load().shc_transpose_neighbors_workspace(V, K))
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device=nbr.device)
    nbr_t = torch.empty((V, SHC_MAX_VIRTUAL_SLOTS), dtype=torch.int32, device=nbr.device)
    slot_of = torch.empty(SHC_MAX_VIRTUAL_SLOTS, dtype=torch.int32, device=nbr.device)
    kt = ctypes.c_int32(0)
    args = [_dev(nbr, "nbr", torch.int32, V * K), V, K, _dev(nbr_t, "nbr_t"),
            _dev(slot_of, "slot_of"), ctypes.addressof(kt), _dev(ws, "ws"),
            ws.numel(), _stream(stream)]
    _check(load().shc_transpose_neighbors(*args), "shc_transpose_neighbors")
    return nbr_t, slot_of, int(kt.value)


def build_transposed_table(coords: torch.Tensor, inv: torch.Tensor, n_rows: int, B: int, V: int,
                           nbr_t: torch.Tensor, Kt: int, table_t: torch.Tensor,
                           row_slots: torch.Tensor, stream=None):
    """shc_build_transposed_table: table_t [Kt][n_rows] int32, row_slots [n_rows] int64."""
    args = [_dev(coords, "coords", torch.int32, 2 * n_rows), _dev(inv, "inv", torch.int32, B * V),
            n_rows, B, V, _dev(nbr_t, "nbr_t", torch.int32, V * Kt), Kt,
            _dev(table_t, "table_t", torch.int32, Kt * n_rows),
            _dev(row_slots, "row_slots", torch.int64, n_rows), _stream(stream)]
    _check(load().shc_build_transposed_table(*args), "shc_build_transposed_table")


def sparse_linear_backward_workspace(n_rows: int, Cin: int, Cout: int, dtype: int = SHC_BF16):
    return int(load().shc_sparse_linear_backward_workspace(n_rows, Cin, Cout, dtype))


def sparse_linear_backward(S, W, Y, dY, n_rows: int, dS=None, dW=None, db=None,
                           act: int = SHC_ACT_RELU, ws=None, stream=None):
    """shc_sparse_linear_backward; W [Cin][Cout] bf16, dW / db fp32.  Returns the workspace."""
    Cin, Cout = W.shape
    need = sparse_linear_backward_workspace(n_rows, Cin, Cout, _dtype_code(W))
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=W.device)
    dt = W.dtype
    args = [_opt_dev(S, "S", dt, n_rows * Cin), _dev(W, "W", dt, Cin * Cout),
            _opt_dev(Y, "Y", dt, n_rows * Cout), _dev(dY, "dY", dt, n_rows * Cout), n_rows, Cin,
            Cout, _dtype_code(W), act, _opt_dev(dS, "dS", dt, n_rows * Cin),
            _opt_dev(dW, "dW", torch.float32, Cin * Cout),
            _opt_dev(db, "db", torch.float32, Cout), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    _check(load().shc_sparse_linear_backward(*args), "shc_sparse_linear_backward")
    return ws


def sparse_neighbor_conv_backward_workspace(n_rows: int, K: int, Cin: int, Cout: int,
                                            dtype: int = SHC_BF16):
    return int(load().shc_sparse_neighbor_conv_backward_workspace(n_rows, K, Cin, Cout, dtype))


def build_slot_pairs(table: torch.Tensor, n_rows: int, K: int, pairs: torch.Tensor,
                     pair_ptr: torch.Tensor, ws=None, stream=None):
    """shc_build_slot_pairs: pairs [K * n_rows][2] int32, pair_ptr [K + 1] int32."""
    need = int(load().shc_build_slot_pairs_workspace(n_rows, K))
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=table.device)
    args = [_dev(table, "table", torch.int32, K * n_rows), n_rows, K,
            _dev(pairs, "pairs", torch.int32, 2 * K * n_rows),
            _dev(pair_ptr, "pair_ptr", torch.int32, K + 1), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    _check(load().shc_build_slot_pairs(*args), "shc_build_slot_pairs")
    return ws


def sparse_neighbor_conv_backward(S, table, table_t, row_slots, slot_of, Kt: int, W, Y, dY,
                                  n_rows: int, dS=None, dW=None, db=None,
                                  act: int = SHC_ACT_RELU, ws=None, stream=None, pairs=None,
                                  pair_ptr=None):
    """shc_sparse_neighbor_conv_backward; W [K][Cin][Cout] bf16, dW [K][Cin][Cout] and db fp32.
    Returns the workspace."""
    K, Cin, Cout = W.shape
    need = sparse_neighbor_conv_backward_workspace(n_rows, K, Cin, Cout, _dtype_code(W))
    if ws is None:
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=W.device)
    dt = W.dtype
    args = [_opt_dev(S, "S", dt, n_rows * Cin), _opt_dev(table, "table", torch.int32, K * n_rows),
            _opt_dev(pairs, "pairs", torch.int32, 2 * K * n_rows),
            _opt_dev(pair_ptr, "pair_ptr", torch.int32, K + 1),
            _opt_dev(table_t, "table_t", torch.int32, Kt * n_rows),
            _opt_dev(row_slots, "row_slots", torch.int64, n_rows),
            _opt_dev(slot_of, "slot_of", torch.int32, Kt), Kt, _dev(W, "W", dt, K * Cin * Cout),
            _opt_dev(Y, "Y", dt, n_rows * Cout), _dev(dY, "dY", dt, n_rows * Cout), n_rows, K,
            Cin, Cout, _dtype_code(W), act, _opt_dev(dS, "dS", dt, n_rows * Cin),
            _opt_dev(dW, "dW", torch.float32, K * Cin * Cout),
            _opt_dev(db, "db", torch.float32, Cout), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_backward(*args), "shc_sparse_neighbor_conv_backward")
    return ws


# ----------------------------------------------------------------------------
# prepared calls: every argument marshalled and checked once, against the
# capacity of the buffers; a call then only substitutes the row count
# ----------------------------------------------------------------------------


class Prepared:
    """One library call with its arguments resolved up front.

    The tensors are checked once, at their full size, so any row count up to
    ``n_max`` is valid; ``__call__(n_rows)`` enqueues the call on the stream
    captured at preparation.  The tensors are kept alive by this object.
    """

    __slots__ = ("_fn", "_args", "_n_at", "n_max", "_where", "_keep")

    def __init__(self, where: str, args, n_at: Optional[int], n_max: int, keep):
        self._fn = getattr(load(), where)
        self._args = list(args)
        self._n_at = n_at
        self.n_max = int(n_max)
        self._where = where
        self._keep = keep

    def __call__(self, n_rows: int = 0) -> int:
        if self._n_at is not None:
            if not 0 <= n_rows <= self.n_max:
                raise ValueError(f"{self._where}: n_rows = {n_rows} outside [0, {self.n_max}]")
            self._args[self._n_at] = n_rows
        rc = self._fn(*self._args)
        if rc != 0:
            _check(rc, self._where)
        return rc


class PreparedScatterUpdate:
    """shc_scatter_update marshalled once; call with (n_rows, prev_rows)."""

    def __init__(self, args, keep, n_max: int, prev_max: int):
        self._fn = load().shc_scatter_update
        self._args = list(args)
        self._keep = keep
        self.n_max, self.prev_max = int(n_max), int(prev_max)

    def __call__(self, n_rows: int, prev_rows: int) -> int:
        if not (0 <= n_rows <= self.n_max and 0 <= prev_rows <= self.prev_max):
            raise ValueError(f"shc_scatter_update: n_rows = {n_rows}, prev_rows = {prev_rows} "
                             f"outside [0, {self.n_max}] x [0, {self.prev_max}]")
        self._args[3] = n_rows
        self._args[5] = prev_rows
        rc = self._fn(*self._args)
        if rc != 0:
            _check(rc, "shc_scatter_update")
        return rc


class PreparedCompact:
    """shc_compact_mask with a pinned host count; calling it returns N'.

    ``start()`` and ``wait()`` are the two halves (shc_compact_mask_start /
    shc_compact_mask_wait): work that needs only ``inv`` can be enqueued
    between them, while the count is on its way.  Given ``nbr`` [V][K] and
    ``table``, ``start()`` is shc_compact_mask_table_start: the neighbour-row
    table of the active set ([K][N'], row stride N') is written in the same
    pass, for up to ``cap`` = coords rows (the table holds K * cap entries).
    """

    def __init__(self, mask, B, V, coords, inv, row_ptr, n_active, ws, stream=None,
                 nbr=None, table=None):
        self.host = torch.zeros(1, dtype=torch.int64, pin_memory=True)
        self._host_view = self.host.numpy()
        cap = coords.numel() // 2
        args = [_dev(mask, "mask", torch.uint8, B * V), B, V,
                _dev(coords, "coords", torch.int32) if cap > 0 else None,
                _dev(inv, "inv", torch.int32, B * V),
                _dev(row_ptr, "row_ptr", torch.int32, B + 1),
                _dev(n_active, "n_active", torch.int32, 1), self.host.data_ptr(), cap,
                _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)]
        keep = (mask, coords, inv, row_ptr, n_active, ws, self.host, nbr, table)
        self._call = Prepared("shc_compact_mask", args, None, 0, keep)
        if nbr is not None:
            K = nbr.shape[-1]
            targs = args[:9] + [_dev(nbr, "nbr", torch.int32, V * K), K,
                                _dev(table, "table", torch.int32, K * cap) if cap > 0 else None]
            targs += args[9:]
            self._start = Prepared("shc_compact_mask_table_start", targs, None, 0, keep)
        else:
            self._start = Prepared("shc_compact_mask_start", args, None, 0, keep)
        self._wait = Prepared("shc_compact_mask_wait", [self.host.data_ptr(), cap, args[-1]],
                              None, 0, keep)

    def __call__(self) -> int:
        self._call()
        return int(self._host_view[0])

    def start(self):
        self._start()

    def wait(self) -> int:
        self._wait()
        return int(self._host_view[0])


def prepare_gather_rows(x, coords, B, V, S, stream=None) -> Prepared:
    C = x.shape[-1]
    n_max = min(coords.numel() // 2, S.numel() // C)
    args = [_dev(x, "x", x.dtype, B * V * C), _dev(coords, "coords", torch.int32), 0, B, V, C,
            _dtype_code(x), _dev(S, "S", x.dtype), _stream(stream)]
    return Prepared("shc_gather_rows", args, 2, n_max, (x, coords, S))


def prepare_sparse_linear(S, W, bias, out, act=SHC_ACT_RELU, stream=None) -> Prepared:
    Cin, Cout = W.shape
    n_max = min(S.numel() // Cin, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), 0, _dev(W, "W", S.dtype, Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, _dtype_code(S), act,
            _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_linear", args, 1, n_max, (S, W, bias, out))


def prepare_build_transposed_table(coords, inv, B, V, nbr_t, Kt, table_t, row_slots,
                                   stream=None) -> Prepared:
    n_max = min(coords.numel() // 2, table_t.numel() // Kt, row_slots.numel())
    args = [_dev(coords, "coords", torch.int32), _dev(inv, "inv", torch.int32, B * V), 0, B, V,
            _dev(nbr_t, "nbr_t", torch.int32, V * Kt), Kt, _dev(table_t, "table_t", torch.int32),
            _dev(row_slots, "row_slots", torch.int64), _stream(stream)]
    return Prepared("shc_build_transposed_table", args, 2, n_max,
                    (coords, inv, nbr_t, table_t, row_slots))


def prepare_sparse_linear_backward(S, W, Y, dY, dS, dW, db, act=SHC_ACT_RELU, ws=None,
                                   stream=None) -> Prepared:
    """shc_sparse_linear_backward for any row count up to the buffers' capacity."""
    Cin, Cout = W.shape
    n_max = min(dY.numel() // Cout, S.numel() // Cin if S is not None else 1 << 62,
                dS.numel() // Cin if dS is not None else 1 << 62)
    if ws is None:
        need = sparse_linear_backward_workspace(n_max, Cin, Cout, _dtype_code(W))
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=W.device)
    dt = W.dtype
    args = [_opt_dev(S, "S", dt), _dev(W, "W", dt, Cin * Cout), _opt_dev(Y, "Y", dt),
            _dev(dY, "dY", dt), 0, Cin, Cout, _dtype_code(W), act, _opt_dev(dS, "dS", dt),
            _opt_dev(dW, "dW", torch.float32, Cin * Cout), _opt_dev(db, "db", torch.float32, Cout),
            _dev(ws, "ws"), ws.numel() * ws.element_size(), _stream(stream)]
    return Prepared("shc_sparse_linear_backward", args, 4, n_max, (S, W, Y, dY, dS, dW, db, ws))


def prepare_build_slot_pairs(table, K, pairs, pair_ptr, n_max, ws=None, stream=None) -> Prepared:
    if ws is None:
        need = int(load().shc_build_slot_pairs_workspace(n_max, K))
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=table.device)
    args = [_dev(table, "table", torch.int32), 0, K, _dev(pairs, "pairs", torch.int32),
            _dev(pair_ptr, "pair_ptr", torch.int32, K + 1), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    return Prepared("shc_build_slot_pairs", args, 1, n_max, (table, pairs, pair_ptr, ws))


def prepare_sparse_neighbor_conv_backward(S, table, table_t, row_slots, slot_of, Kt, W, Y, dY,
                                          dS, dW, db, act=SHC_ACT_RELU, ws=None,
                                          stream=None, pairs=None, pair_ptr=None) -> Prepared:
    """shc_sparse_neighbor_conv_backward for any row count up to the buffers' capacity."""
    K, Cin, Cout = W.shape
    n_max = min(dY.numel() // Cout, S.numel() // Cin if S is not None else 1 << 62,
                dS.numel() // Cin if dS is not None else 1 << 62,
                table.numel() // K if table is not None else 1 << 62,
                table_t.numel() // Kt if table_t is not None else 1 << 62)
    if ws is None:
        need = sparse_neighbor_conv_backward_workspace(n_max, K, Cin, Cout, _dtype_code(W))
        ws = torch.empty(max(need, 16), dtype=torch.uint8, device=W.device)
    dt = W.dtype
    args = [_opt_dev(S, "S", dt), _opt_dev(table, "table", torch.int32),
            _opt_dev(pairs, "pairs", torch.int32), _opt_dev(pair_ptr, "pair_ptr", torch.int32, K + 1),
            _opt_dev(table_t, "table_t", torch.int32), _opt_dev(row_slots, "row_slots", torch.int64),
            _opt_dev(slot_of, "slot_of", torch.int32), Kt, _dev(W, "W", dt, K * Cin * Cout),
            _opt_dev(Y, "Y", dt), _dev(dY, "dY", dt), 0, K, Cin, Cout, _dtype_code(W), act,
            _opt_dev(dS, "dS", dt), _opt_dev(dW, "dW", torch.float32, K * Cin * Cout),
            _opt_dev(db, "db", torch.float32, Cout), _dev(ws, "ws"),
            ws.numel() * ws.element_size(), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_backward", args, 11, n_max,
                    (S, table, pairs, pair_ptr, table_t, row_slots, slot_of, W, Y, dY, dS, dW, db,
                     ws))


def prepare_gather_sparse_linear(x, coords, B, V, W, bias, out, act=SHC_ACT_RELU,
                                 stream=None) -> Prepared:
    Cin, Cout = W.shape
    n_max = min(coords.numel() // 2, out.numel() // Cout)
    args = [_dev(x, "x", x.dtype, B * V * Cin), _dev(coords, "coords", torch.int32), 0, B, V,
            _dev(W, "W", x.dtype, Cin * Cout), _opt_dev(bias, "bias", torch.float32, Cout),
            Cin, Cout, _dtype_code(x), act, _dev(out, "out", x.dtype), _stream(stream)]
    return Prepared("shc_gather_sparse_linear", args, 2, n_max, (x, coords, W, bias, out))


def prepare_sparse_neighbor_conv(S, coords, inv, B, V, nbr, W, bias, out, act=SHC_ACT_RELU,
                                 stream=None) -> Prepared:
    K, Cin, Cout = W.shape
    n_max = min(S.numel() // Cin, coords.numel() // 2, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(coords, "coords", torch.int32),
            _dev(inv, "inv", torch.int32, B * V), 0, B, V,
            _dev(nbr, "nbr", torch.int32, V * K), K, _dev(W, "W", S.dtype, K * Cin * Cout),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, _dtype_code(S), act,
            _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv", args, 3, n_max, (S, coords, inv, nbr, W, bias, out))


def prepare_build_neighbor_table(coords, inv, B, V, nbr, table, stream=None) -> Prepared:
    K = nbr.shape[-1]
    n_max = min(coords.numel() // 2, table.numel() // K)
    args = [_dev(coords, "coords", torch.int32), _dev(inv, "inv", torch.int32, B * V), 0, B, V,
            _dev(nbr, "nbr", torch.int32, V * K), K, _dev(table, "table", torch.int32),
            _stream(stream)]
    return Prepared("shc_build_neighbor_table", args, 2, n_max, (coords, inv, nbr, table))


def prepare_sparse_neighbor_conv_table(S, table, W, bias, out, act=SHC_ACT_RELU,
                                       stream=None) -> Prepared:
    K, Cin, Cout = W.shape
    n_max = min(S.numel() // Cin, table.numel() // K, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(table, "table", torch.int32), 0, K,
            _dev(W, "W", S.dtype, K * Cin * Cout), _opt_dev(bias, "bias", torch.float32, Cout),
            Cin, Cout, _dtype_code(S), act, _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_table", args, 2, n_max, (S, table, W, bias, out))


def prepare_sparse_neighbor_conv_split(S, table, W, bias, out, workspace, act=SHC_ACT_RELU,
                                       stream=None) -> Prepared:
    K, Cin, Cout = W.shape
    n_max = min(S.numel() // Cin, table.numel() // K, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(table, "table", torch.int32), 0, K,
            _dev(W, "W", S.dtype, K * Cin * Cout), _opt_dev(bias, "bias", torch.float32, Cout),
            Cin, Cout, _dtype_code(S), act, _dev(out, "out", S.dtype), _dev(workspace, "workspace"),
            workspace.numel() * workspace.element_size(), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_split", args, 2, n_max,
                    (S, table, W, bias, out, workspace))


def prepare_sparse_neighbor_conv_packed(S, table, Wp, K, Cin, Cout, bias, out,
                                        act=SHC_ACT_RELU, stream=None) -> Prepared:
    """shc_sparse_neighbor_conv_packed with n_rows given per call."""
    n_max = min(S.numel() // Cin, table.numel() // K, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(table, "table", torch.int32), 0, K, _dev(Wp, "Wp"),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, _dtype_code(S), act,
            _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_packed", args, 2, n_max,
                    (S, table, Wp, bias, out))


def conv_packed_plan_bytes(n_rows: int, K: int, Cin: int, Cout: int,
                           dtype: int = SHC_BF16) -> int:
    """shc_conv_packed_plan_bytes: a packed-conv plan buffer for up to n_rows
    rows (0: the shape has no packed conv)."""
    return int(load().shc_conv_packed_plan_bytes(n_rows, K, Cin, Cout, dtype))


def build_conv_packed_plan(table: torch.Tensor, n_rows: int, K: int, Cin: int, Cout: int,
                           plan: torch.Tensor, stream=None):
    """shc_build_conv_packed_plan (bf16 shapes)."""
    args = [_dev(table, "table", torch.int32, K * n_rows), n_rows, K, Cin, Cout, SHC_BF16,
            _dev(plan, "plan"), plan.numel() * plan.element_size(), _stream(stream)]
    _check(load().shc_build_conv_packed_plan(*args), "shc_build_conv_packed_plan")


def sparse_neighbor_conv_packed_planned(S: torch.Tensor, plan: torch.Tensor, n_rows: int,
                                        Wp: torch.Tensor, K: int, Cin: int, Cout: int,
                                        bias: Optional[torch.Tensor], out: torch.Tensor,
                                        act: int = SHC_ACT_RELU, stream=None):
    """shc_sparse_neighbor_conv_packed_planned."""
    args = [_dev(S, "S", S.dtype, n_rows * Cin), _dev(plan, "plan"),
            plan.numel() * plan.element_size(), n_rows, K, _dev(Wp, "Wp"),
            _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout, _dtype_code(S), act,
            _dev(out, "out", S.dtype, n_rows * Cout), _stream(stream)]
    _check(load().shc_sparse_neighbor_conv_packed_planned(*args),
           "shc_sparse_neighbor_conv_packed_planned")


def prepare_build_conv_packed_plan(table, K, Cin, Cout, plan, stream=None) -> Prepared:
    """shc_build_conv_packed_plan with n_rows given per call."""
    args = [_dev(table, "table", torch.int32), 0, K, Cin, Cout, SHC_BF16, _dev(plan, "plan"),
            plan.numel() * plan.element_size(), _stream(stream)]
    return Prepared("shc_build_conv_packed_plan", args, 1, table.numel() // K, (table, plan))


def prepare_sparse_neighbor_conv_packed_planned(S, plan, Wp, K, Cin, Cout, bias, out,
                                                act=SHC_ACT_RELU, stream=None) -> Prepared:
    """shc_sparse_neighbor_conv_packed_planned with n_rows given per call."""
    n_max = min(S.numel() // Cin, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(plan, "plan"), plan.numel() * plan.element_size(), 0, K,
            _dev(Wp, "Wp"), _opt_dev(bias, "bias", torch.float32, Cout), Cin, Cout,
            _dtype_code(S), act, _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_packed_planned", args, 3, n_max,
                    (S, plan, Wp, bias, out))


def prepare_build_conv_plan(table, K, Cin, Cout, plan, dtype=SHC_BF16, stream=None) -> Prepared:
    """shc_build_conv_plan with n_rows given per call (table [K][n_rows] of
    the call's n_rows, plan sized for the largest n_rows called with)."""
    args = [_dev(table, "table", torch.int32), 0, K, Cin, Cout, dtype, _dev(plan, "plan"),
            plan.numel() * plan.element_size(), _stream(stream)]
    return Prepared("shc_build_conv_plan", args, 1, table.numel() // K, (table, plan))


def prepare_sparse_neighbor_conv_planned(S, plan, W, bias, out, act=SHC_ACT_RELU,
                                         stream=None) -> Prepared:
    K, Cin, Cout = W.shape
    n_max = min(S.numel() // Cin, out.numel() // Cout)
    args = [_dev(S, "S", S.dtype), _dev(plan, "plan"), plan.numel() * plan.element_size(), 0, K,
            _dev(W, "W", S.dtype, K * Cin * Cout), _opt_dev(bias, "bias", torch.float32, Cout),
            Cin, Cout, _dtype_code(S), act, _dev(out, "out", S.dtype), _stream(stream)]
    return Prepared("shc_sparse_neighbor_conv_planned", args, 3, n_max, (S, plan, W, bias, out))


def prepare_scatter(S, inv, coords, B, V, D, zero_fill=True, stream=None) -> Prepared:
    C = D.shape[-1]
    n_max = S.numel() // C if zero_fill else min(S.numel() // C, coords.numel() // 2)
    args = [_dev(S, "S", D.dtype), _dev(inv, "inv", torch.int32, B * V) if zero_fill else None,
            None if zero_fill else _dev(coords, "coords", torch.int32), 0, B, V, C,
            _dtype_code(D), 1 if zero_fill else 0, _dev(D, "D", D.dtype, B * V * C),
            _stream(stream)]
    return Prepared("shc_scatter", args, 3, n_max, (S, inv, coords, D))


def prepare_clear_inactive_rows(inv, B, V, D, stream=None) -> Prepared:
    C = D.shape[-1]
    args = [_dev(inv, "inv", torch.int32, B * V), B, V, C, _dtype_code(D),
            _dev(D, "D", D.dtype, B * V * C), _stream(stream)]
    return Prepared("shc_clear_inactive_rows", args, None, 0, (inv, D))


def prepare_segment_maxpool(S, row_ptr, B, P, empty_value=0.0, stream=None) -> Prepared:
    C = P.shape[-1]
    args = [_dev(S, "S", P.dtype), _dev(row_ptr, "row_ptr", torch.int32, B + 1), 0, B, C,
            _dtype_code(P), float(empty_value), _dev(P, "P", P.dtype, B * C), _stream(stream)]
    return Prepared("shc_segment_maxpool", args, 2, S.numel() // C, (S, row_ptr, P))
