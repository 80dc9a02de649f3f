"""Thin ctypes binding of libpfc (include/pfc.h): same names, marshalling only.

Every function takes plain integers for device pointers (e.g. a torch
tensor's ``data_ptr()``) and a stream handle (``torch.cuda.current_stream()
.cuda_stream``), and raises PfcError on a non-zero status.  All computation
happens in the HIP library; when the library is missing this module raises
on import instead of falling back to anything else.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpfc.so")

PFC_OK = 0
PFC_ERR_INVALID_ARG = 1
PFC_ERR_CAPACITY = 2
PFC_ERR_WORKSPACE = 3
PFC_ERR_UNSUPPORTED = 4
PFC_ERR_HIP = 5
PFC_ERR_SCRATCH = 6

PFC_F32, PFC_BF16, PFC_F16 = 0, 1, 2
PFC_MAX_BATCH = 8192
PFC_MAX_CLASSES = 1 << 30
PFC_NOALLOC_MAX_CLASSES = 1 << 21
PFC_COSFACE, PFC_ARCFACE = 0, 1

PFC_K_SAMPLE, PFC_K_PREP, PFC_K_FWD_GEMM, PFC_K_LSE = 0, 1, 2, 3
PFC_K_DX_GEMM, PFC_K_DX_FINAL, PFC_K_DW_UPDATE = 4, 5, 6
KERNEL_NAMES = {PFC_K_SAMPLE: "sample", PFC_K_PREP: "prep", PFC_K_FWD_GEMM: "fwd_gemm",
                PFC_K_LSE: "lse", PFC_K_DX_GEMM: "dx_gemm", PFC_K_DX_FINAL: "dx_final",
                PFC_K_DW_UPDATE: "dw_update"}

EXPORTS = ("pfc_workspace_bytes", "pfc_sample", "pfc_sample_noalloc", "pfc_forward_loss",
           "pfc_backward_update", "pfc_status_string", "pfc_timing_begin", "pfc_timing_end",
           "pfc_bank_stage", "pfc_bank_patch", "pfc_bank_writeback")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it first "
                      "(python -c 'import __graft_entry__ as g; g.build()')")

_lib = ctypes.CDLL(LIB_PATH)

_i64, _u64, _int = ctypes.c_int64, ctypes.c_uint64, ctypes.c_int
_sz, _dbl, _flt, _vp = ctypes.c_size_t, ctypes.c_double, ctypes.c_float, ctypes.c_void_p

_lib.pfc_workspace_bytes.argtypes = [_i64, _i64, _i64, _dbl, _int,
                                     ctypes.POINTER(_sz), ctypes.POINTER(_i64)]
_lib.pfc_workspace_bytes.restype = _int
_lib.pfc_sample.argtypes = [_vp, _i64, _i64, _i64, _dbl, _u64, _vp, _i64, _vp, _vp, _vp, _sz, _vp]
_lib.pfc_sample.restype = _int
_lib.pfc_sample_noalloc.argtypes = [_vp, _i64, _i64, _i64, _dbl, _u64, _vp, _i64, _vp, _vp, _vp]
_lib.pfc_sample_noalloc.restype = _int
_lib.pfc_forward_loss.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _i64, _vp, _vp, _i64, _vp,
                                  _int, _flt, _flt, _int, _flt, _vp, _vp, _vp, _sz, _vp]
_lib.pfc_forward_loss.restype = _int
_lib.pfc_backward_update.argtypes = [_vp, _int, _i64, _i64, _vp, _int, _vp, _vp, _i64, _vp, _vp,
                                     _i64, _vp, _int, _flt, _flt, _int, _vp, _flt, _flt, _vp,
                                     _vp, _sz, _vp]
_lib.pfc_backward_update.restype = _int
_lib.pfc_status_string.argtypes = [_int]
_lib.pfc_status_string.restype = ctypes.c_char_p
_lib.pfc_timing_begin.argtypes = [_int, _int]
_lib.pfc_timing_begin.restype = _int
_lib.pfc_timing_end.argtypes = [ctypes.POINTER(_dbl), ctypes.POINTER(_int)]
_lib.pfc_timing_end.restype = _int
_lib.pfc_bank_stage.argtypes = [_int, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _i64,
                                _vp, _vp, ctypes.c_int32, _vp, _vp]
_lib.pfc_bank_stage.restype = _int
_lib.pfc_bank_patch.argtypes = [_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _vp]
_lib.pfc_bank_patch.restype = _int
_lib.pfc_bank_writeback.argtypes = [_int, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _vp,
                                    ctypes.c_int32, _vp]
_lib.pfc_bank_writeback.restype = _int


class PfcError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: status {status} ({pfc_status_string(status)})")


def pfc_status_string(status):
    return _lib.pfc_status_string(int(status)).decode()


def _check(status, where):
    if status != PFC_OK:
        raise PfcError(status, where)


def pfc_workspace_bytes(B, d, C, r, compute_dtype):
    """Returns (workspace bytes, active_cap)."""
    nbytes, cap = _sz(0), _i64(0)
    _check(_lib.pfc_workspace_bytes(B, d, C, r, compute_dtype, ctypes.byref(nbytes),
                                    ctypes.byref(cap)), "pfc_workspace_bytes")
    return nbytes.value, cap.value


def pfc_sample(labels, B, C, class_offset, r, seed, active, active_cap, n_active,
               labels_mapped, ws, ws_bytes, stream):
    _check(_lib.pfc_sample(labels, B, C, class_offset, r, seed, active, active_cap, n_active,
                           labels_mapped, ws, ws_bytes, stream), "pfc_sample")


def pfc_sample_noalloc(labels, B, C, class_offset, r, seed, active, active_cap, n_active,
                       labels_mapped, stream):
    _check(_lib.pfc_sample_noalloc(labels, B, C, class_offset, r, seed, active, active_cap,
                                   n_active, labels_mapped, stream), "pfc_sample_noalloc")


def pfc_forward_loss(X, x_dtype, B, d, W, w_dtype, C, active, n_active, active_cap,
                     labels_mapped, compute_dtype, s, m, margin, tau, loss, row_lse, ws, ws_bytes,
                     stream):
    _check(_lib.pfc_forward_loss(X, x_dtype, B, d, W, w_dtype, C, active, n_active, active_cap,
                                 labels_mapped, compute_dtype, s, m, margin, tau, loss, row_lse,
                                 ws, ws_bytes, stream), "pfc_forward_loss")


def pfc_backward_update(X, x_dtype, B, d, W, w_dtype, W_master, momentum, C, active, n_active,
                        active_cap, labels_mapped, compute_dtype, s, m, margin, row_lse, lr, mu,
                        dX, ws, ws_bytes, stream):
    _check(_lib.pfc_backward_update(X, x_dtype, B, d, W, w_dtype, W_master, momentum, C, active,
                                    n_active, active_cap, labels_mapped, compute_dtype, s, m,
                                    margin, row_lse, lr, mu, dX, ws, ws_bytes, stream),
           "pfc_backward_update")


def pfc_timing_begin(kernel, max_launches):
    _check(_lib.pfc_timing_begin(kernel, max_launches), "pfc_timing_begin")


def pfc_timing_end():
    """Returns (total milliseconds, number of bracketed launches)."""
    ms, n = _dbl(0.0), _int(0)
    _check(_lib.pfc_timing_end(ctypes.byref(ms), ctypes.byref(n)), "pfc_timing_end")
    return ms.value, n.value


def _bank_arrays(src, dst, row_bytes):
    """Host arrays of the per-array pointers and row sizes of a bank copy
    (equal-length sequences of ints); kept alive by the caller's frame."""
    n = len(src)
    if len(dst) != n or len(row_bytes) != n:
        raise ValueError("bank copy: pointer and row-size lists of different lengths")
    return (n, (ctypes.c_void_p * max(n, 1))(*src), (ctypes.c_void_p * max(n, 1))(*dst),
            (ctypes.c_int64 * max(n, 1))(*row_bytes))


def pfc_bank_stage(banks, slots, row_bytes, C, next_active, next_n, prev_active, prev_n,
                   prev2_active, prev2_n, active_cap, bank_version, row_version, version, stale,
                   stream):
    n, b, s, rb = _bank_arrays(banks, slots, row_bytes)
    _check(_lib.pfc_bank_stage(n, b, s, rb, C, next_active, next_n, prev_active, prev_n,
                               prev2_active, prev2_n, active_cap, bank_version, row_version,
                               version, stale, stream), "pfc_bank_stage")


def pfc_bank_patch(prev_slots, next_slots, row_bytes, prev_active, prev_n, next_active, next_n,
                   active_cap, stream):
    n, p, q, rb = _bank_arrays(prev_slots, next_slots, row_bytes)
    _check(_lib.pfc_bank_patch(n, p, q, rb, prev_active, prev_n, next_active, next_n,
                               active_cap, stream), "pfc_bank_patch")


def pfc_bank_writeback(slots, banks, row_bytes, active, n_active, next_active, next_n,
                       active_cap, C, bank_version, version, stream):
    n, s, b, rb = _bank_arrays(slots, banks, row_bytes)
    _check(_lib.pfc_bank_writeback(n, s, b, rb, active, n_active, next_active, next_n,
                                   active_cap, C, bank_version, version, stream),
           "pfc_bank_writeback")
