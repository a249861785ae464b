"""Python binding of libspccl.so, the gfx950 Pici hot path (SpCCL, arXiv 2607.04676).

Argument marshalling only: every step runs in the HIP library.  Functions keep
the C names of include/spccl.h and take torch tensors for device buffers (their
data pointers and byte sizes are passed through) and an optional torch stream
(default: the current stream).  A nonzero status raises SpcclError.  There is
no fallback: if the library is missing, importing this package fails.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspccl.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(or python paper_2607_04676_amd/build.py)")

_lib = ctypes.CDLL(LIB_PATH)

SPCCL_OK = 0
STATUS_NAMES = {0: "OK", 1: "ERR_INVALID_ARG", 2: "ERR_CAPACITY", 3: "ERR_UNSUPPORTED",
                4: "ERR_CORRUPT_STREAM", 5: "ERR_WORKSPACE", 6: "ERR_HIP", 7: "ERR_TIMEOUT"}
SPCCL_F32, SPCCL_BF16 = 0, 1
SPCCL_FMT_DENSE, SPCCL_FMT_PICI, SPCCL_FMT_COO = 0, 1, 2
SPCCL_ARRAY, SPCCL_STREAM = 0, 1
HEADER_BYTES = 48
NNZ_UNKNOWN = (1 << 64) - 1

# every symbol the C header declares
EXPORTS = ("spccl_num_tiles", "spccl_pici_bytes", "spccl_stream_bound", "spccl_workspace_bytes",
           "spccl_workspace_min_bytes",
           "spccl_workspace_init", "spccl_compress", "spccl_decompress", "spccl_encode_dense",
           "spccl_reduce", "spccl_gather_expand", "spccl_copy_message", "spccl_read_header",
           "spccl_read_status", "spccl_status_string", "spccl_vr_scratch_bytes",
           "spccl_vr_reduce_scatter", "spccl_vr_all_gather", "spccl_vr_all_reduce",
           "spccl_slice_count", "spccl_slice_bytes", "spccl_compress_sliced", "spccl_decompress_sliced",
           "spccl_reduce_sliced", "spccl_copy_sliced", "spccl_coo_bytes", "spccl_message_bound",
           "spccl_compress_coo", "spccl_slice_tracker_bytes", "spccl_compress_sliced_tracked",
           "spccl_reduce_sliced_tracked", "spccl_vr_sliced_scratch_bytes", "spccl_vr_reduce_scatter_sliced",
           "spccl_vr_all_gather_sliced", "spccl_vr_all_reduce_sliced", "spccl_compress_static",
           "spccl_set_single_pass_limit")


class spccl_operand_t(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("fmt", ctypes.c_int32), ("ptr", ctypes.c_void_p),
                ("bytes", ctypes.c_uint64)]


class spccl_header_t(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("format", ctypes.c_uint16), ("dtype", ctypes.c_uint16),
                ("n", ctypes.c_uint64), ("nnz", ctypes.c_uint64), ("off_I", ctypes.c_uint64),
                ("off_A", ctypes.c_uint64), ("total_bytes", ctypes.c_uint64)]


class spccl_policy_t(ctypes.Structure):
    _fields_ = [("intra_thresh", ctypes.c_double), ("inter_thresh", ctypes.c_double),
                ("ag_thresh", ctypes.c_double), ("ranks_per_node", ctypes.c_int32),
                ("adaptive", ctypes.c_int32), ("sparse_fmt", ctypes.c_int32)]


class spccl_trace_t(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int32), ("rank", ctypes.c_int32), ("fmt", ctypes.c_int32),
                ("measured", ctypes.c_int32), ("bytes", ctypes.c_uint64), ("nnz", ctypes.c_uint64),
                ("sigma", ctypes.c_double)]


_u64, _i32, _vp = ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p
_sigs = {
    "spccl_num_tiles": (_u64, [_u64]),
    "spccl_pici_bytes": (_u64, [_u64, _i32, _u64]),
    "spccl_stream_bound": (_u64, [_u64, _i32]),
    "spccl_workspace_bytes": (_u64, [_u64, _i32]),
    "spccl_workspace_min_bytes": (_u64, [_u64, _i32]),
    "spccl_workspace_init": (_i32, [_vp, _u64, _vp]),
    "spccl_set_single_pass_limit": (ctypes.c_uint32, [ctypes.c_uint32]),
    "spccl_compress": (_i32, [_vp, _u64, _i32, _vp, _u64, _vp, _u64, _vp]),
    "spccl_compress_coo": (_i32, [_vp, _u64, _i32, _vp, _u64, _vp, _u64, _vp]),
    "spccl_compress_static": (_i32, [_vp, _u64, _i32, _vp, _u64, _vp]),
    "spccl_coo_bytes": (_u64, [_i32, _u64]),
    "spccl_message_bound": (_u64, [_u64, _i32, _i32]),
    "spccl_decompress": (_i32, [_vp, _u64, _vp, _u64, _i32, _vp, _u64, _vp]),
    "spccl_encode_dense": (_i32, [_vp, _u64, _i32, _vp, _u64, _vp]),
    "spccl_reduce": (_i32, [spccl_operand_t, spccl_operand_t, spccl_operand_t, _u64, _i32, _vp, _u64, _vp]),
    "spccl_gather_expand": (_i32, [ctypes.POINTER(spccl_operand_t), _i32, _u64, _i32, _vp, _u64, _vp, _u64,
                                   _vp]),
    "spccl_copy_message": (_i32, [_vp, _u64, _vp, _u64, _vp, _u64, _vp]),
    "spccl_read_header": (_i32, [_vp, ctypes.POINTER(spccl_header_t), _vp]),
    "spccl_read_status": (_i32, [_vp, _i32, _vp]),
    "spccl_status_string": (ctypes.c_char_p, [_i32]),
    "spccl_vr_scratch_bytes": (_u64, [_i32, _u64, _i32]),
    "spccl_vr_reduce_scatter": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32,
                                       ctypes.POINTER(spccl_policy_t), _vp, _u64, ctypes.POINTER(spccl_trace_t),
                                       _vp]),
    "spccl_vr_all_gather": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32,
                                   ctypes.POINTER(spccl_policy_t), _vp, _u64, ctypes.POINTER(spccl_trace_t), _vp]),
    "spccl_vr_all_reduce": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32,
                                   ctypes.POINTER(spccl_policy_t), _vp, _u64, ctypes.POINTER(spccl_trace_t),
                                   _vp]),
    "spccl_slice_count": (_u64, [_u64]),
    "spccl_slice_bytes": (_u64, [_i32]),
    "spccl_compress_sliced": (_i32, [_vp, _u64, _i32, ctypes.c_double, _vp, _u64, _vp, _u64, _vp]),
    "spccl_decompress_sliced": (_i32, [_vp, _u64, _vp, _u64, _i32, _vp, _u64, _vp]),
    "spccl_reduce_sliced": (_i32, [_vp, _vp, _u64, _vp, _u64, _i32, ctypes.c_double, _u64, _i32, _vp, _u64, _vp]),
    "spccl_copy_sliced": (_i32, [_vp, _u64, _vp, _u64, _u64, _i32, _vp, _u64, _vp]),
    "spccl_slice_tracker_bytes": (_u64, [_u64]),
    "spccl_compress_sliced_tracked": (_i32, [_vp, _u64, _i32, ctypes.c_double, _vp, _u64, _vp, _u64, _vp, _vp,
                                             _u64, _vp]),
    "spccl_reduce_sliced_tracked": (_i32, [_vp, _vp, _u64, _vp, _u64, ctypes.c_double, _vp, _u64, _vp, _u64, _i32,
                                           _vp, _u64, _vp]),
    "spccl_vr_sliced_scratch_bytes": (_u64, [_i32, _u64, _i32]),
    "spccl_vr_reduce_scatter_sliced": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32,
                                              ctypes.POINTER(spccl_policy_t), _vp, _u64, _vp, _vp]),
    "spccl_vr_all_gather_sliced": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32, _vp, _u64,
                                          _vp, _vp]),
    "spccl_vr_all_reduce_sliced": (_i32, [ctypes.POINTER(_vp), ctypes.POINTER(_vp), _i32, _u64, _i32,
                                          ctypes.POINTER(spccl_policy_t), _vp, _u64, _vp, _vp, _vp]),
}
for _name, (_res, _args) in _sigs.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


class SpcclError(RuntimeError):
    def __init__(self, status: int, what: str):
        msg = _lib.spccl_status_string(status).decode()
        super().__init__(f"{what}: {STATUS_NAMES.get(status, status)} ({msg})")
        self.status = status


def _check(st: int, what: str) -> None:
    if st != SPCCL_OK:
        raise SpcclError(st, what)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return SPCCL_F32
    if t.dtype in (torch.bfloat16, torch.int16, torch.uint16):
        return SPCCL_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def operand(t: torch.Tensor, kind: int = SPCCL_ARRAY, fmt: int = SPCCL_FMT_DENSE) -> spccl_operand_t:
    """The C operand of a device tensor.  It holds a reference to the tensor,
    so an operand made from a temporary keeps that memory alive as long as
    the operand itself."""
    o = spccl_operand_t(kind, fmt, t.data_ptr(), _nbytes(t))
    o._tensor = t
    return o


# ---- sizes --------------------------------------------------------------------------

def spccl_num_tiles(n: int) -> int:
    return _lib.spccl_num_tiles(n)


def spccl_pici_bytes(n: int, dtype: int, nnz: int) -> int:
    return _lib.spccl_pici_bytes(n, dtype, nnz)


def spccl_stream_bound(n: int, dtype: int) -> int:
    return _lib.spccl_stream_bound(n, dtype)


def spccl_workspace_bytes(n: int, dtype: int) -> int:
    return _lib.spccl_workspace_bytes(n, dtype)


def spccl_workspace_min_bytes(n: int, dtype: int) -> int:
    return _lib.spccl_workspace_min_bytes(n, dtype)


def spccl_set_single_pass_limit(max_partitions: int) -> int:
    """Upper bound (in 16384-element partitions) on the Pici outputs written in
    one launch with a full workspace (0: always two passes; default 2**32 - 1,
    the library's own limits); returns the previous bound."""
    return _lib.spccl_set_single_pass_limit(max_partitions)


def spccl_coo_bytes(dtype: int, nnz: int) -> int:
    return _lib.spccl_coo_bytes(dtype, nnz)


def spccl_message_bound(n: int, dtype: int, fmt: int) -> int:
    return _lib.spccl_message_bound(n, dtype, fmt)


def spccl_vr_scratch_bytes(P: int, msg_elems: int, dtype: int) -> int:
    return _lib.spccl_vr_scratch_bytes(P, msg_elems, dtype)


# ---- entry points ------------------------------------------------------------------

def spccl_workspace_init(ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_workspace_init(ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_workspace_init")


def spccl_compress(dense: torch.Tensor, out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_compress(dense.data_ptr(), dense.numel(), _dt(dense), out.data_ptr(), _nbytes(out),
                               ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_compress")


def spccl_compress_static(dense: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    """spccl_compress without a workspace (its scratch is the library's own
    static device array; n <= SPCCL_STATIC_MAX_ELEMS)."""
    _check(_lib.spccl_compress_static(dense.data_ptr(), dense.numel(), _dt(dense), out.data_ptr(), _nbytes(out),
                                      _stream(stream)), "spccl_compress_static")


SPCCL_STATIC_MAX_ELEMS = 1 << 28


def spccl_compress_coo(dense: torch.Tensor, out: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_compress_coo(dense.data_ptr(), dense.numel(), _dt(dense), out.data_ptr(), _nbytes(out),
                                   ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_compress_coo")


def spccl_decompress(msg: torch.Tensor, dense: torch.Tensor, ws: torch.Tensor, stream=None,
                     msg_bytes: int | None = None) -> None:
    _check(_lib.spccl_decompress(msg.data_ptr(), _nbytes(msg) if msg_bytes is None else msg_bytes,
                                 dense.data_ptr(), dense.numel(), _dt(dense), ws.data_ptr(), _nbytes(ws),
                                 _stream(stream)), "spccl_decompress")


def spccl_encode_dense(dense: torch.Tensor, out: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_encode_dense(dense.data_ptr(), dense.numel(), _dt(dense), out.data_ptr(), _nbytes(out),
                                   _stream(stream)), "spccl_encode_dense")


def spccl_reduce(a: spccl_operand_t, b: spccl_operand_t, out: spccl_operand_t, n: int, dtype: int,
                 ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_reduce(a, b, out, n, dtype, ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_reduce")


def spccl_gather_expand(parts: list, n_per_part: int, dtype: int, dense_out: torch.Tensor, ws: torch.Tensor,
                        stream=None) -> None:
    arr = (spccl_operand_t * len(parts))(*parts)
    _check(_lib.spccl_gather_expand(arr, len(parts), n_per_part, dtype, dense_out.data_ptr(), _nbytes(dense_out),
                                    ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_gather_expand")


def spccl_copy_message(src: torch.Tensor, dst: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_copy_message(src.data_ptr(), _nbytes(src), dst.data_ptr(), _nbytes(dst), ws.data_ptr(),
                                   _nbytes(ws), _stream(stream)), "spccl_copy_message")


def spccl_read_header(msg: torch.Tensor, stream=None) -> dict:
    h = spccl_header_t()
    _check(_lib.spccl_read_header(msg.data_ptr(), ctypes.byref(h), _stream(stream)), "spccl_read_header")
    return {f: getattr(h, f) for f, _ in spccl_header_t._fields_}


def spccl_read_status(ws: torch.Tensor, clear: bool = True, stream=None) -> int:
    return _lib.spccl_read_status(ws.data_ptr(), 1 if clear else 0, _stream(stream))


def spccl_status_string(status: int) -> str:
    return _lib.spccl_status_string(status).decode()


def _policy(policy) -> spccl_policy_t:
    if policy is None:
        return spccl_policy_t(0.6, 0.5, 0.1, 0, 1, SPCCL_FMT_PICI)
    if isinstance(policy, spccl_policy_t):
        return policy
    return spccl_policy_t(policy.intra_thresh, policy.inter_thresh, policy.ag_thresh, policy.ranks_per_node,
                          policy.adaptive, getattr(policy, "sparse_fmt", SPCCL_FMT_PICI))


def _ptrs(ts) -> ctypes.Array:
    return (ctypes.c_void_p * len(ts))(*[t.data_ptr() for t in ts])


def _trace(tr, count) -> list:
    return [(tr[i].step, tr[i].rank, tr[i].fmt, tr[i].measured, tr[i].bytes, tr[i].nnz, tr[i].sigma)
            for i in range(count)]


def spccl_vr_reduce_scatter(send: list, recv: list, scratch: torch.Tensor, policy=None, stream=None) -> list:
    P, n = len(send), send[0].numel()
    tr = (spccl_trace_t * max(1, P * (P - 1)))()
    pol = _policy(policy)
    _check(_lib.spccl_vr_reduce_scatter(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), ctypes.byref(pol),
                                        scratch.data_ptr(), _nbytes(scratch), tr, _stream(stream)),
           "spccl_vr_reduce_scatter")
    return _trace(tr, P * (P - 1))


def spccl_vr_all_gather(send: list, recv: list, scratch: torch.Tensor, policy=None, stream=None) -> list:
    P, n = len(send), send[0].numel()
    tr = (spccl_trace_t * P)()
    pol = _policy(policy)
    _check(_lib.spccl_vr_all_gather(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), ctypes.byref(pol),
                                    scratch.data_ptr(), _nbytes(scratch), tr, _stream(stream)), "spccl_vr_all_gather")
    return _trace(tr, P)


def spccl_vr_all_reduce(send: list, recv: list, scratch: torch.Tensor, policy=None, stream=None) -> list:
    P, n = len(send), send[0].numel()
    tr = (spccl_trace_t * (P * (P - 1) + P))()
    pol = _policy(policy)
    _check(_lib.spccl_vr_all_reduce(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), ctypes.byref(pol),
                                    scratch.data_ptr(), _nbytes(scratch), tr, _stream(stream)),
           "spccl_vr_all_reduce")
    return _trace(tr, P * (P - 1) + P)


# ---- sliced streams -----------------------------------------------------------------

SPCCL_SLICE_ELEMS = 16384


def spccl_slice_count(n: int) -> int:
    return _lib.spccl_slice_count(n)


def spccl_slice_bytes(dtype: int) -> int:
    return _lib.spccl_slice_bytes(dtype)


def spccl_compress_sliced(dense: torch.Tensor, out: torch.Tensor, ws: torch.Tensor, dense_thresh: float = -1.0,
                          stream=None) -> None:
    _check(_lib.spccl_compress_sliced(dense.data_ptr(), dense.numel(), _dt(dense), float(dense_thresh),
                                      out.data_ptr(), _nbytes(out), ws.data_ptr(), _nbytes(ws), _stream(stream)),
           "spccl_compress_sliced")


def spccl_decompress_sliced(inp: torch.Tensor, dense: torch.Tensor, ws: torch.Tensor, stream=None) -> None:
    _check(_lib.spccl_decompress_sliced(inp.data_ptr(), _nbytes(inp), dense.data_ptr(), dense.numel(), _dt(dense),
                                        ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_decompress_sliced")


def spccl_reduce_sliced(a: torch.Tensor, b: torch.Tensor, out: torch.Tensor, ws: torch.Tensor, out_sliced: bool,
                        dense_thresh: float = -1.0, stream=None) -> None:
    """out = a (dense) (+) b (sliced stream); out is a sliced stream or a dense array."""
    _check(_lib.spccl_reduce_sliced(a.data_ptr(), b.data_ptr(), _nbytes(b), out.data_ptr(), _nbytes(out),
                                    1 if out_sliced else 0, float(dense_thresh), a.numel(), _dt(a), ws.data_ptr(),
                                    _nbytes(ws), _stream(stream)), "spccl_reduce_sliced")


def spccl_copy_sliced(src: torch.Tensor, dst: torch.Tensor, n: int, dtype: int, ws: torch.Tensor,
                      stream=None) -> None:
    _check(_lib.spccl_copy_sliced(src.data_ptr(), _nbytes(src), dst.data_ptr(), _nbytes(dst), n, dtype,
                                  ws.data_ptr(), _nbytes(ws), _stream(stream)), "spccl_copy_sliced")


def spccl_slice_tracker_bytes(n: int) -> int:
    return _lib.spccl_slice_tracker_bytes(n)


def _ptr_or_null(t) -> int | None:
    return None if t is None else t.data_ptr()


def spccl_compress_sliced_tracked(dense: torch.Tensor, out: torch.Tensor, tracker: torch.Tensor, ws: torch.Tensor,
                                  tau: float, fmt_out: torch.Tensor | None = None, stream=None) -> None:
    _check(_lib.spccl_compress_sliced_tracked(dense.data_ptr(), dense.numel(), _dt(dense), float(tau),
                                              out.data_ptr(), _nbytes(out), tracker.data_ptr(), _nbytes(tracker),
                                              _ptr_or_null(fmt_out), ws.data_ptr(), _nbytes(ws), _stream(stream)),
           "spccl_compress_sliced_tracked")


def spccl_reduce_sliced_tracked(a: torch.Tensor, b: torch.Tensor, out: torch.Tensor, tracker: torch.Tensor,
                                ws: torch.Tensor, tau: float, fmt_out: torch.Tensor | None = None,
                                stream=None) -> None:
    _check(_lib.spccl_reduce_sliced_tracked(a.data_ptr(), b.data_ptr(), _nbytes(b), out.data_ptr(), _nbytes(out),
                                            float(tau), tracker.data_ptr(), _nbytes(tracker), _ptr_or_null(fmt_out),
                                            a.numel(), _dt(a), ws.data_ptr(), _nbytes(ws), _stream(stream)),
           "spccl_reduce_sliced_tracked")


def spccl_vr_sliced_scratch_bytes(P: int, msg_elems: int, dtype: int) -> int:
    return _lib.spccl_vr_sliced_scratch_bytes(P, msg_elems, dtype)


def spccl_vr_reduce_scatter_sliced(send: list, recv: list, scratch: torch.Tensor, policy=None, stream=None):
    """Returns the per-slice formats sent, shape (P-1, P, S)."""
    import numpy as np
    P, n = len(send), send[0].numel()
    S = spccl_slice_count(n // P)
    fm = np.zeros(max(1, (P - 1) * P * S), dtype=np.uint8)
    pol = _policy(policy)
    _check(_lib.spccl_vr_reduce_scatter_sliced(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), ctypes.byref(pol),
                                               scratch.data_ptr(), _nbytes(scratch), fm.ctypes.data,
                                               _stream(stream)), "spccl_vr_reduce_scatter_sliced")
    return fm[:(P - 1) * P * S].reshape(max(P - 1, 0), P, S)


def spccl_vr_all_gather_sliced(send: list, recv: list, scratch: torch.Tensor, stream=None):
    """Returns the per-slice formats sent, shape (P, S)."""
    import numpy as np
    P, n = len(send), send[0].numel()
    S = spccl_slice_count(n)
    fm = np.zeros(max(1, P * S), dtype=np.uint8)
    _check(_lib.spccl_vr_all_gather_sliced(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), scratch.data_ptr(),
                                           _nbytes(scratch), fm.ctypes.data, _stream(stream)),
           "spccl_vr_all_gather_sliced")
    return fm[:P * S].reshape(P, S)


def spccl_vr_all_reduce_sliced(send: list, recv: list, scratch: torch.Tensor, policy=None, stream=None):
    """Returns the per-slice formats (reduce-scatter (P-1, P, S), all-gather (P, S))."""
    import numpy as np
    P, n = len(send), send[0].numel()
    S = spccl_slice_count(n // P)
    frs = np.zeros(max(1, (P - 1) * P * S), dtype=np.uint8)
    fag = np.zeros(max(1, P * S), dtype=np.uint8)
    pol = _policy(policy)
    _check(_lib.spccl_vr_all_reduce_sliced(_ptrs(send), _ptrs(recv), P, n, _dt(send[0]), ctypes.byref(pol),
                                           scratch.data_ptr(), _nbytes(scratch), frs.ctypes.data, fag.ctypes.data,
                                           _stream(stream)), "spccl_vr_all_reduce_sliced")
    return frs[:(P - 1) * P * S].reshape(max(P - 1, 0), P, S), fag[:P * S].reshape(P, S)


def alloc_sliced(n: int, dtype: int, device="cuda") -> torch.Tensor:
    """A uint8 buffer with every slot of an n-element sliced stream."""
    return torch.empty(max(spccl_slice_count(n) * spccl_slice_bytes(dtype), 16), dtype=torch.uint8, device=device)


# ---- tensor helpers (allocation stays with the caller; these only size buffers) -----

def alloc_stream(n: int, dtype: int, device="cuda", fmt: int = SPCCL_FMT_PICI) -> torch.Tensor:
    """A uint8 buffer able to hold any n-element message of format fmt (or dense)."""
    return torch.empty(spccl_message_bound(n, dtype, fmt), dtype=torch.uint8, device=device)


def alloc_workspace(n: int, dtype: int, device="cuda", stream=None, minimal: bool = False) -> torch.Tensor:
    """A zeroed workspace for messages of up to n elements.  minimal=True
    sizes it for the one-launch kernels only (no per-partition slots)."""
    need = spccl_workspace_min_bytes(n, dtype) if minimal else spccl_workspace_bytes(n, dtype)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    spccl_workspace_init(ws, stream)
    return ws
