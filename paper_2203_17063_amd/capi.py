"""Thin ctypes binding of libecc.so (the C ABI in include/libecc.h).

Functions carry the C names and only marshal arguments: device buffers may be
given as torch tensors (their ``data_ptr()``) or raw integer addresses, host
arrays as numpy arrays.  Every non-OK status raises :class:`EccError`.  All
computation happens in the HIP kernels of libecc.so; if the library is not
built, loading fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libecc.so")

ECC_OK, ECC_ERR_ARG, ECC_ERR_OVERLAP, ECC_ERR_RANGE = 0, 1, 2, 3
ECC_ERR_ALLOC, ECC_ERR_DEVICE, ECC_ERR_STATE = 4, 5, 6
ECC_UNBOUNDED = 0x7FFFFFFF
ECC_NORM_L1, ECC_NORM_L2 = 1, 2
ECC_KIND_JACOBI, ECC_KIND_POWER = 0, 1
ECC_TIMING_ASSEMBLE, ECC_TIMING_ALLREDUCE, ECC_TIMING_SWEEP, ECC_TIMING_NORM = 0, 1, 2, 3
ECC_TIMING_MF_GRAD, ECC_TIMING_MF_STEP, ECC_TIMING_KINDS = 4, 5, 6
ECC_THRESHOLD_DATA, ECC_THRESHOLD_PROCS = 0, 1
ECC_LAYOUT_STREAM, ECC_LAYOUT_SORTED, ECC_LAYOUT_SHORT, ECC_LAYOUT_RANGES = 0, 1, 2, 3
ECC_SCHEDULE_AUTO, ECC_SCHEDULE_STATIC, ECC_SCHEDULE_QUEUE, ECC_SCHEDULE_SINGLE = 0, 1, 2, 3
ECC_COMPACT_AUTO, ECC_COMPACT_NONE = 0, 1
ECC_FORM_GENERAL, ECC_FORM_COLUMN_VALUES, ECC_FORM_DIAGONALS = 0, 1, 2
ECC_MAX_DIAGONALS = 8
ECC_SCRATCH_DOUBLES = 1 << 20
ECC_GATHER_CHUNK = 2048

STATUS_NAMES = {0: "ECC_OK", 1: "ECC_ERR_ARG", 2: "ECC_ERR_OVERLAP", 3: "ECC_ERR_RANGE",
                4: "ECC_ERR_ALLOC", 5: "ECC_ERR_DEVICE", 6: "ECC_ERR_STATE"}


class EccError(RuntimeError):
    def __init__(self, status: int, message: str):
        self.status = status
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, str(status)), message))


class ecc_csr_t(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64), ("n_cols", ctypes.c_int64), ("nnz", ctypes.c_int64),
                ("d_row_ptr", ctypes.c_void_p), ("d_col", ctypes.c_void_p),
                ("d_val", ctypes.c_void_p)]


class ecc_matrix_opts_t(ctypes.Structure):
    _fields_ = [("range_bytes", ctypes.c_int64), ("tile_rows", ctypes.c_int64),
                ("schedule", ctypes.c_int32), ("compact", ctypes.c_int32)]


_lib = None

# (name, restype, argtypes)
_VP, _I32, _I64, _D = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
_SIGS = [
    ("ecc_abi_version", _I32, []),
    ("ecc_last_error", ctypes.c_char_p, []),
    ("ecc_status_string", ctypes.c_char_p, [ctypes.c_int]),
    ("ecc_plan_validate", ctypes.c_int, [_I32, _VP, _VP, _I32]),
    ("ecc_plan_create", ctypes.c_int, [_I32, _VP, _VP, _I32, _VP, ctypes.POINTER(_VP)]),
    ("ecc_plan_destroy", ctypes.c_int, [_VP]),
    ("ecc_plan_reset", ctypes.c_int, [_VP]),
    ("ecc_plan_set_stream", ctypes.c_int, [_VP, _VP]),
    ("ecc_plan_stats", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP]),
    ("ecc_plan_set_timing", ctypes.c_int, [_VP, _I32]),
    ("ecc_plan_timing", ctypes.c_int, [_VP, _I32, _VP, _VP, _I32]),
    ("ecc_allgatherv_assemble", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_allgatherv_assemble_packed", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_allreduce_partial", ctypes.c_int, [_VP, _I64, _VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_matrix_create", ctypes.c_int, [_VP, ctypes.POINTER(ecc_csr_t), _I32, ctypes.POINTER(_VP)]),
    ("ecc_matrix_create_ex", ctypes.c_int, [_VP, ctypes.POINTER(ecc_csr_t), _I32,
                                            ctypes.POINTER(ecc_matrix_opts_t),
                                            ctypes.POINTER(_VP)]),
    ("ecc_matrix_destroy", ctypes.c_int, [_VP]),
    ("ecc_matrix_tiling", ctypes.c_int, [_VP, _VP, _VP]),
    ("ecc_matrix_schedule", ctypes.c_int, [_VP, _VP]),
    ("ecc_matrix_form", ctypes.c_int, [_VP, _VP, _VP, _VP]),
    ("ecc_partials_size", _I64, [_VP]),
    ("ecc_matrix_layout", ctypes.c_int, [_VP, _VP, _VP]),
    ("ecc_iterate_jacobi", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_iterate_spmv", ctypes.c_int, [_VP, _VP, _D, _D, _VP, _VP, _VP, _VP]),
    ("ecc_residual", ctypes.c_int, [_VP, _VP, _I64, _I32, _VP, _VP]),
    ("ecc_iterate_jacobi_noalloc", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_stream_copy", ctypes.c_int, [_VP, _VP, _I64, _VP]),
    ("ecc_gather_probe", ctypes.c_int, [_VP, _I64, _VP, _I64, _VP, _I64, _VP]),
    ("ecc_hypercube_create", ctypes.c_int, [_I32, _I64, _I32, _VP, ctypes.POINTER(_VP)]),
    ("ecc_hypercube_destroy", ctypes.c_int, [_VP]),
    ("ecc_hypercube_reset", ctypes.c_int, [_VP]),
    ("ecc_allreduce_ssp", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_hypercube_stats", ctypes.c_int, [_VP, _VP, _VP, _VP, _VP]),
    ("ecc_bcast_threshold", ctypes.c_int, [_I32, _I32, _I64, _D, _VP, _VP, _VP, _VP]),
    ("ecc_reduce_threshold", ctypes.c_int, [_I32, _I32, _I64, _D, _I32, _VP, _VP, _VP, _VP,
                                            _VP]),
    ("ecc_allreduce_drop", ctypes.c_int, [_I32, _I64, _VP, _VP, _VP, _VP, _VP]),
    ("ecc_mf_create", ctypes.c_int, [_I32, _I32, _I32, _I32, _I32, _I64, _VP, _VP, _VP,
                                     ctypes.POINTER(_VP)]),
    ("ecc_mf_destroy", ctypes.c_int, [_VP]),
    ("ecc_mf_iterate", ctypes.c_int, [_VP, _VP, _D, _D, _VP, _VP, _VP, _VP, _VP, _VP, _VP,
                                      _VP]),
    ("ecc_mf_error", ctypes.c_int, [_VP, _VP, _VP, _VP]),
    ("ecc_solve", ctypes.c_int, [_VP, _VP, _VP, _D, _D, _VP, _VP, _VP, _VP, _I32, _D, _VP, _VP,
                                 _VP, _VP]),
]

EXPORTED = [s[0] for s in _SIGS]


def lib():
    """Load libecc.so (built in-tree by ``__graft_entry__.build()``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libecc.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in _SIGS:
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(x):
    """Address of a device/host buffer: torch tensor, numpy array, int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _check(status: int):
    if status != ECC_OK:
        raise EccError(status, lib().ecc_last_error().decode())


def _host_i64(a):
    if a is None:
        return None
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int64))
    return arr


# ----------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ----------------------------------------------------------------------------

def ecc_abi_version() -> int:
    return int(lib().ecc_abi_version())


def ecc_last_error() -> str:
    return lib().ecc_last_error().decode()


def ecc_plan_validate(P, counts=None, displs=None, max_staleness=0) -> int:
    """Returns the status code (does not raise)."""
    c, d = _host_i64(counts), _host_i64(displs)
    return int(lib().ecc_plan_validate(P, _ptr(c), _ptr(d), max_staleness))


def ecc_plan_create(P, counts, displs, max_staleness, stream=None) -> int:
    c, d = _host_i64(counts), _host_i64(displs)
    out = _VP()
    _check(lib().ecc_plan_create(P, _ptr(c), _ptr(d), max_staleness, stream, ctypes.byref(out)))
    return out.value


def ecc_plan_destroy(plan):
    _check(lib().ecc_plan_destroy(plan))


def ecc_plan_reset(plan):
    _check(lib().ecc_plan_reset(plan))


def ecc_plan_set_stream(plan, stream):
    _check(lib().ecc_plan_set_stream(plan, stream))


def ecc_plan_stats(plan, P: int):
    """Returns (clock, forced_total, version[P], age[P])."""
    clock = ctypes.c_int64()
    forced = ctypes.c_int64()
    ver = np.empty(P, dtype=np.int32)
    age = np.empty(P, dtype=np.int32)
    _check(lib().ecc_plan_stats(plan, ctypes.addressof(clock), ctypes.addressof(forced),
                                _ptr(ver), _ptr(age)))
    return clock.value, forced.value, ver, age


def ecc_plan_set_timing(plan, enable: bool):
    _check(lib().ecc_plan_set_timing(plan, 1 if enable else 0))


def ecc_plan_timing(plan, kernel: int, reset: bool = False):
    """Returns (total_ms, launches) of the launches of `kernel` timed so far."""
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check(lib().ecc_plan_timing(plan, kernel, ctypes.addressof(ms), ctypes.addressof(n),
                                 1 if reset else 0))
    return ms.value, n.value


def ecc_allgatherv_assemble(plan, d_send, d_recv, d_arrived, d_eff_out=None, d_age_out=None):
    _check(lib().ecc_allgatherv_assemble(plan, _ptr(d_send), _ptr(d_recv), _ptr(d_arrived),
                                         _ptr(d_eff_out), _ptr(d_age_out)))


def ecc_allgatherv_assemble_packed(plan, d_send_base, d_recv, d_arrived, d_eff_out=None,
                                   d_age_out=None):
    _check(lib().ecc_allgatherv_assemble_packed(plan, _ptr(d_send_base), _ptr(d_recv),
                                                _ptr(d_arrived), _ptr(d_eff_out),
                                                _ptr(d_age_out)))


def ecc_allreduce_partial(plan, m, d_fresh, d_slots, d_result, d_arrived, d_eff_out=None,
                          d_result_clock=None):
    _check(lib().ecc_allreduce_partial(plan, m, _ptr(d_fresh), _ptr(d_slots), _ptr(d_result),
                                       _ptr(d_arrived), _ptr(d_eff_out), _ptr(d_result_clock)))


def make_csr(n_rows, n_cols, nnz, d_row_ptr, d_col, d_val) -> ecc_csr_t:
    return ecc_csr_t(n_rows, n_cols, nnz, _ptr(d_row_ptr), _ptr(d_col), _ptr(d_val))


def ecc_matrix_create(plan, csr: ecc_csr_t, kind: int) -> int:
    out = _VP()
    _check(lib().ecc_matrix_create(plan, ctypes.byref(csr), kind, ctypes.byref(out)))
    return out.value


def ecc_matrix_create_ex(plan, csr: ecc_csr_t, kind: int, range_bytes: int = 0,
                         tile_rows: int = 0, schedule: int = 0, compact: int = 0) -> int:
    out = _VP()
    opts = ecc_matrix_opts_t(range_bytes, tile_rows, schedule, compact)
    _check(lib().ecc_matrix_create_ex(plan, ctypes.byref(csr), kind, ctypes.byref(opts),
                                      ctypes.byref(out)))
    return out.value


def ecc_matrix_tiling(mat):
    """(plane rows, tile rows) of a short-layout matrix; (0, 0) in row order."""
    plane, tile = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().ecc_matrix_tiling(mat, ctypes.byref(plane), ctypes.byref(tile)))
    return plane.value, tile.value


def ecc_matrix_schedule(mat) -> int:
    sch = ctypes.c_int32(0)
    _check(lib().ecc_matrix_schedule(mat, ctypes.byref(sch)))
    return sch.value


def ecc_matrix_form(mat):
    """(form, diagonal offsets): ECC_FORM_* and, for the diagonal form, the
    offsets col - row in increasing order (else an empty list)."""
    form, nd = ctypes.c_int32(0), ctypes.c_int32(0)
    offs = (ctypes.c_int32 * ECC_MAX_DIAGONALS)()
    _check(lib().ecc_matrix_form(mat, ctypes.byref(form), ctypes.byref(nd), offs))
    return form.value, list(offs[:nd.value])


def ecc_matrix_destroy(mat):
    _check(lib().ecc_matrix_destroy(mat))


def ecc_partials_size(mat) -> int:
    return int(lib().ecc_partials_size(mat))


def ecc_matrix_layout(mat):
    """(layout, entries held per row) of a matrix handle."""
    layout, slots = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().ecc_matrix_layout(mat, ctypes.byref(layout), ctypes.byref(slots)))
    return layout.value, slots.value


def ecc_iterate_jacobi(plan, mat, d_b, d_x_own, d_x_hat, d_x_next, d_partials):
    _check(lib().ecc_iterate_jacobi(plan, mat, _ptr(d_b), _ptr(d_x_own), _ptr(d_x_hat),
                                    _ptr(d_x_next), _ptr(d_partials)))


def ecc_iterate_jacobi_noalloc(plan, mat, d_b, d_x_own, d_x_hat, d_x_next, d_rho):
    _check(lib().ecc_iterate_jacobi_noalloc(plan, mat, _ptr(d_b), _ptr(d_x_own), _ptr(d_x_hat),
                                            _ptr(d_x_next), _ptr(d_rho)))


def ecc_iterate_spmv(plan, mat, alpha, beta, d_x_own, d_x_hat, d_x_next, d_partials):
    _check(lib().ecc_iterate_spmv(plan, mat, alpha, beta, _ptr(d_x_own), _ptr(d_x_hat),
                                  _ptr(d_x_next), _ptr(d_partials)))


def ecc_residual(plan, d_partials, n_partials, norm, h_out=True, d_out=None):
    """Returns the norm when h_out is true (synchronising), else None."""
    h = ctypes.c_double()
    _check(lib().ecc_residual(plan, _ptr(d_partials), n_partials, norm,
                              ctypes.addressof(h) if h_out else None, _ptr(d_out)))
    return h.value if h_out else None


def ecc_solve(plan, mat, d_b, alpha, beta, d_x, d_x_tmp, d_x_hat, d_mask, T, tol, d_rho,
              d_eff_hist=None, d_age_hist=None) -> int:
    iters = ctypes.c_int32()
    _check(lib().ecc_solve(plan, mat, _ptr(d_b), alpha, beta, _ptr(d_x), _ptr(d_x_tmp),
                           _ptr(d_x_hat), _ptr(d_mask), T, tol, _ptr(d_rho), _ptr(d_eff_hist),
                           _ptr(d_age_hist), ctypes.addressof(iters)))
    return iters.value


def ecc_stream_copy(d_dst, d_src, n, stream=None):
    _check(lib().ecc_stream_copy(_ptr(d_dst), _ptr(d_src), n, stream))


def ecc_gather_probe(d_idx, n, d_x, n_x, d_out, n_out, stream=None):
    _check(lib().ecc_gather_probe(_ptr(d_idx), n, _ptr(d_x), n_x, _ptr(d_out), n_out, stream))


def ecc_hypercube_create(P, m, slack, stream=None) -> int:
    out = _VP()
    _check(lib().ecc_hypercube_create(P, m, slack, stream, ctypes.byref(out)))
    return out.value


def ecc_hypercube_destroy(h):
    _check(lib().ecc_hypercube_destroy(h))


def ecc_hypercube_reset(h):
    _check(lib().ecc_hypercube_reset(h))


def ecc_allreduce_ssp(h, d_contrib, d_delivered, d_result, d_result_clock=None, d_outcome=None):
    _check(lib().ecc_allreduce_ssp(h, _ptr(d_contrib), _ptr(d_delivered), _ptr(d_result),
                                   _ptr(d_result_clock), _ptr(d_outcome)))


def ecc_hypercube_stats(h, P: int):
    """Returns (clock, waits_total, slot_clock[P][d], waits[P][d])."""
    d = P.bit_length() - 1
    clock = ctypes.c_int64()
    waits = ctypes.c_uint64()
    clk = np.empty((P, d), dtype=np.int32)
    w = np.empty((P, d), dtype=np.uint64)
    _check(lib().ecc_hypercube_stats(h, ctypes.addressof(clock), ctypes.addressof(waits),
                                     _ptr(clk), _ptr(w)))
    return clock.value, waits.value, clk, w


def ecc_bcast_threshold(P, root, m, theta, d_src, d_dst, stream=None) -> int:
    """Returns the number of elements delivered."""
    k = ctypes.c_int64()
    _check(lib().ecc_bcast_threshold(P, root, m, theta, _ptr(d_src), _ptr(d_dst),
                                     ctypes.addressof(k), stream))
    return k.value


def ecc_reduce_threshold(P, root, m, theta, mode, d_src, d_result, stream=None):
    """Returns (elements reduced, processes involved)."""
    k = ctypes.c_int64()
    n = ctypes.c_int32()
    _check(lib().ecc_reduce_threshold(P, root, m, theta, mode, _ptr(d_src), _ptr(d_result),
                                      ctypes.addressof(k), ctypes.addressof(n), stream))
    return k.value, n.value


def ecc_allreduce_drop(P, m, d_fresh, d_arrived, d_result, d_count=None, stream=None):
    _check(lib().ecc_allreduce_drop(P, m, _ptr(d_fresh), _ptr(d_arrived), _ptr(d_result),
                                    _ptr(d_count), stream))


def ecc_mf_create(n_users, n_items, rank, P, K, N, d_users, d_items, d_ratings) -> int:
    out = _VP()
    _check(lib().ecc_mf_create(n_users, n_items, rank, P, K, N, _ptr(d_users), _ptr(d_items),
                               _ptr(d_ratings), ctypes.byref(out)))
    return out.value


def ecc_mf_destroy(h):
    _check(lib().ecc_mf_destroy(h))


def ecc_mf_iterate(h, plan, eta, lam, d_W, d_grads, d_slots, d_G, d_arrived, d_batch, d_rmse,
                   d_eff_out=None):
    _check(lib().ecc_mf_iterate(h, plan, eta, lam, _ptr(d_W), _ptr(d_grads), _ptr(d_slots),
                                _ptr(d_G), _ptr(d_arrived), _ptr(d_batch), _ptr(d_rmse),
                                _ptr(d_eff_out)))


def ecc_mf_error(h, d_W, d_rmse, hip_stream=None):
    _check(lib().ecc_mf_error(h, _ptr(d_W), _ptr(d_rmse), hip_stream))
