"""CPU oracle for the Pici hot path -- TEST INFRASTRUCTURE ONLY.

A thin ctypes wrapper over ``pici_oracle.c`` (plain single-threaded C, built
with gcc).  Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline
leg of ``bench.py`` may import this package; the GPU library never does, and
the two share no code.

The C file cites the paper passage each function follows: Sec. III-B and
Alg. 1 (format, compression), Sec. III-C (decompression), Sec. IV-B (where
compression and reduction happen in the ring collectives), Sec. IV-C with
Eq. 7 (the adaptive dense switch), Sec. V-B (the 48-byte header), and
Sec. II-B with Sec. IV-D (the flat COO format and its collectives).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pici_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

F32, BF16 = 0, 1
FMT_DENSE, FMT_PICI, FMT_COO = 0, 1, 2
ARRAY, STREAM = 0, 1
OK, ERR_INVALID_ARG, ERR_CAPACITY, ERR_UNSUPPORTED, ERR_CORRUPT_STREAM = 0, 1, 2, 3, 4
NNZ_UNKNOWN = (1 << 64) - 1
HEADER_BYTES = 48


def build() -> str:
    """Compile the oracle with gcc (-O2, IEEE arithmetic, no OpenMP)."""
    tmp = _LIB + ".tmp"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-Wall", "-Wextra", "-fPIC", "-shared",
                           "-fno-fast-math", _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, _LIB)
    return _LIB


class _Policy(ctypes.Structure):
    _fields_ = [("intra_thresh", ctypes.c_double), ("inter_thresh", ctypes.c_double),
                ("ag_thresh", ctypes.c_double), ("ranks_per_node", ctypes.c_int),
                ("adaptive", ctypes.c_int), ("sparse_fmt", ctypes.c_int)]


class _Trace(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int32), ("rank", ctypes.c_int32), ("fmt", ctypes.c_int32),
                ("measured", ctypes.c_int32), ("bytes", ctypes.c_uint64), ("nnz", ctypes.c_uint64),
                ("sigma", ctypes.c_double)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        u64, vp, i32 = ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int
        for name in ("orc_num_tiles", "orc_off_I", "orc_off_A"):
            getattr(L, name).restype = u64
            getattr(L, name).argtypes = [u64]
        L.orc_pici_bytes.restype = u64
        L.orc_pici_bytes.argtypes = [u64, i32, u64]
        L.orc_dense_bytes.restype = u64
        L.orc_dense_bytes.argtypes = [u64, i32]
        L.orc_stream_bound.restype = u64
        L.orc_stream_bound.argtypes = [u64, i32]
        L.orc_coo_off_V.restype = u64
        L.orc_coo_off_V.argtypes = [u64]
        L.orc_coo_bytes.restype = u64
        L.orc_coo_bytes.argtypes = [i32, u64]
        L.orc_message_bound.restype = u64
        L.orc_message_bound.argtypes = [u64, i32, i32]
        L.orc_compress_coo.restype = i32
        L.orc_compress_coo.argtypes = [vp, u64, i32, vp, u64, ctypes.POINTER(u64)]
        L.orc_compress.restype = i32
        L.orc_compress.argtypes = [vp, u64, i32, vp, u64, ctypes.POINTER(u64)]
        L.orc_encode_dense.restype = i32
        L.orc_encode_dense.argtypes = [vp, u64, i32, vp, u64]
        L.orc_validate.restype = i32
        L.orc_validate.argtypes = [vp, u64, u64, i32]
        L.orc_decompress.restype = i32
        L.orc_decompress.argtypes = [vp, u64, vp, u64, i32]
        L.orc_oplus.restype = ctypes.c_uint32
        L.orc_oplus.argtypes = [ctypes.c_uint32, ctypes.c_uint32, i32]
        L.orc_reduce.restype = i32
        L.orc_reduce.argtypes = [i32, vp, u64, i32, vp, u64, i32, i32, vp, u64, u64, i32,
                                 ctypes.POINTER(u64)]
        L.orc_ring_reduce_scatter.restype = i32
        L.orc_ring_reduce_scatter.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32,
                                              ctypes.POINTER(_Policy), ctypes.POINTER(_Trace),
                                              ctypes.POINTER(ctypes.c_double),
                                              ctypes.POINTER(ctypes.c_double)]
        L.orc_ring_all_gather.restype = i32
        L.orc_ring_all_gather.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32, i32,
                                          ctypes.POINTER(_Trace)]
        L.orc_slice_count.restype = u64
        L.orc_slice_count.argtypes = [u64]
        L.orc_slice_bytes.restype = u64
        L.orc_slice_bytes.argtypes = [i32]
        L.orc_encode_sliced.restype = i32
        L.orc_encode_sliced.argtypes = [vp, u64, i32, ctypes.c_double, vp, u64]
        L.orc_decode_sliced.restype = i32
        L.orc_decode_sliced.argtypes = [vp, u64, vp, u64, i32]
        L.orc_reduce_sliced.restype = i32
        L.orc_reduce_sliced.argtypes = [vp, vp, u64, i32, ctypes.c_double, vp, u64, u64, i32]
        L.orc_ring_reduce_scatter_sliced.restype = i32
        L.orc_ring_reduce_scatter_sliced.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32,
                                                     ctypes.POINTER(_Policy), vp]
        L.orc_ring_all_reduce.restype = i32
        L.orc_ring_all_reduce.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32,
                                          ctypes.POINTER(_Policy), ctypes.POINTER(_Trace)]
        L.orc_ring_all_gather_sliced.restype = i32
        L.orc_ring_all_gather_sliced.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32, vp]
        L.orc_time_step.restype = i32
        L.orc_time_step.argtypes = [vp, vp, u64, u64, i32, vp, vp, vp, u64, vp, vp, i32,
                                    ctypes.POINTER(ctypes.c_double)]
        L.orc_ring_all_reduce_sliced.restype = i32
        L.orc_ring_all_reduce_sliced.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(vp), i32, u64, i32,
                                                 ctypes.POINTER(_Policy), vp, vp]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: oracle status {status}")
        self.status = status


def _check(st: int, what: str):
    if st != OK:
        raise OracleError(st, what)


def dtype_code(arr: np.ndarray) -> int:
    if arr.dtype == np.float32:
        return F32
    if arr.dtype == np.uint16:
        return BF16
    raise TypeError(f"unsupported dtype {arr.dtype}")


def elem_size(dtype: int) -> int:
    return 2 if dtype == BF16 else 4


def _np_dtype(dtype: int):
    return np.uint16 if dtype == BF16 else np.float32


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


# ---- sizes (Sec. III-B component sizes, Sec. V-B header) ----------------------

def num_tiles(n: int) -> int:
    return lib().orc_num_tiles(n)


def off_I(n: int) -> int:
    return lib().orc_off_I(n)


def off_A(n: int) -> int:
    return lib().orc_off_A(n)


def pici_bytes(n: int, dtype: int, nnz: int) -> int:
    return lib().orc_pici_bytes(n, dtype, nnz)


def dense_bytes(n: int, dtype: int) -> int:
    return lib().orc_dense_bytes(n, dtype)


def stream_bound(n: int, dtype: int) -> int:
    return lib().orc_stream_bound(n, dtype)


def coo_off_V(nnz: int) -> int:
    return lib().orc_coo_off_V(nnz)


def coo_bytes(dtype: int, nnz: int) -> int:
    """Exact size of a COO message with nnz nonzeros (header, J, pad, V)."""
    return lib().orc_coo_bytes(dtype, nnz)


def message_bound(n: int, dtype: int, fmt: int) -> int:
    """Worst-case size of an n-element message in format fmt (or dense)."""
    return lib().orc_message_bound(n, dtype, fmt)


# ---- codec ---------------------------------------------------------------------

def compress(dense: np.ndarray) -> tuple[np.ndarray, int]:
    """Pici message (uint8 array of exactly total_bytes) and nnz."""
    dense = np.ascontiguousarray(dense)
    dt = dtype_code(dense)
    n = dense.size
    cap = stream_bound(n, dt)
    buf = np.zeros(max(cap, 1), dtype=np.uint8)
    nnz = ctypes.c_uint64(0)
    _check(lib().orc_compress(_ptr(dense), n, dt, _ptr(buf), cap, ctypes.byref(nnz)), "compress")
    total = int(buf[40:48].view(np.uint64)[0])
    return buf[:total].copy(), nnz.value


def compress_coo(dense: np.ndarray) -> tuple[np.ndarray, int]:
    """COO message (uint8 array of exactly total_bytes) and nnz."""
    dense = np.ascontiguousarray(dense)
    dt = dtype_code(dense)
    n = dense.size
    cap = message_bound(n, dt, FMT_COO)
    buf = np.zeros(max(cap, 1), dtype=np.uint8)
    nnz = ctypes.c_uint64(0)
    _check(lib().orc_compress_coo(_ptr(dense), n, dt, _ptr(buf), cap, ctypes.byref(nnz)), "compress_coo")
    total = int(buf[40:48].view(np.uint64)[0])
    return buf[:total].copy(), nnz.value


def encode_dense(dense: np.ndarray) -> np.ndarray:
    dense = np.ascontiguousarray(dense)
    dt = dtype_code(dense)
    cap = dense_bytes(dense.size, dt)
    buf = np.zeros(cap, dtype=np.uint8)
    _check(lib().orc_encode_dense(_ptr(dense), dense.size, dt, _ptr(buf), cap), "encode_dense")
    return buf


def validate(stream: np.ndarray, n: int, dtype: int) -> int:
    stream = np.ascontiguousarray(stream, dtype=np.uint8)
    return lib().orc_validate(_ptr(stream), stream.size, n, dtype)


def decompress(stream: np.ndarray, n: int, dtype: int) -> np.ndarray:
    stream = np.ascontiguousarray(stream, dtype=np.uint8)
    out = np.empty(n, dtype=_np_dtype(dtype))
    _check(lib().orc_decompress(_ptr(stream), stream.size, _ptr(out), n, dtype), "decompress")
    return out


def oplus(a_bits: int, b_bits: int, dtype: int) -> int:
    """a (+) b on raw bit patterns (one element)."""
    return lib().orc_oplus(a_bits, b_bits, dtype)


@dataclass
class Operand:
    """A reduce operand: a dense array (kind ARRAY) or a message (kind STREAM)."""
    kind: int
    data: np.ndarray

    @staticmethod
    def array(a: np.ndarray) -> "Operand":
        return Operand(ARRAY, np.ascontiguousarray(a))

    @staticmethod
    def stream(s: np.ndarray) -> "Operand":
        return Operand(STREAM, np.ascontiguousarray(s, dtype=np.uint8))


def reduce(a: Operand, b: Operand, n: int, dtype: int, out_kind: int = ARRAY,
           out_fmt: int = FMT_DENSE):
    """out = a (+) b.  Returns a dense array, or (message, nnz) for a message output."""
    L = lib()
    if out_kind == ARRAY:
        out = np.empty(n, dtype=_np_dtype(dtype))
        cap = 0
    else:
        cap = message_bound(n, dtype, out_fmt)
        out = np.zeros(cap, dtype=np.uint8)
    nnz = ctypes.c_uint64(NNZ_UNKNOWN)
    st = L.orc_reduce(a.kind, _ptr(a.data), a.data.nbytes, b.kind, _ptr(b.data), b.data.nbytes,
                      out_kind, out_fmt, _ptr(out), cap, n, dtype, ctypes.byref(nnz))
    _check(st, "reduce")
    if out_kind == ARRAY:
        return out
    total = int(out[40:48].view(np.uint64)[0])
    return out[:total].copy(), nnz.value


# ---- ring collectives over virtual ranks (Sec. IV-A..C) --------------------------

@dataclass
class Policy:
    intra_thresh: float = 0.6
    inter_thresh: float = 0.5
    ag_thresh: float = 0.1
    ranks_per_node: int = 0      # 0: every link is intra-node
    adaptive: int = 1            # 0 never dense, 1 threshold rule, 2 always dense
    sparse_fmt: int = FMT_PICI   # format of sparse sends: Pici or COO

    @staticmethod
    def coo(**kw) -> "Policy":
        """COO sends with the paper's COO thresholds (Sec. IV-D): intra 0.8,
        inter 0.7, ag 0.5."""
        return Policy(**{"intra_thresh": 0.8, "inter_thresh": 0.7, "ag_thresh": 0.5, "sparse_fmt": FMT_COO, **kw})

    def c(self) -> _Policy:
        return _Policy(self.intra_thresh, self.inter_thresh, self.ag_thresh,
                       self.ranks_per_node, self.adaptive, self.sparse_fmt)


@dataclass(frozen=True)
class TraceEntry:
    step: int
    rank: int
    fmt: int
    measured: int
    bytes: int
    nnz: int
    sigma: float


def _trace_list(tr, count) -> list:
    return [TraceEntry(tr[i].step, tr[i].rank, tr[i].fmt, tr[i].measured, tr[i].bytes, tr[i].nnz,
                       tr[i].sigma) for i in range(count)]


def _ptr_array(arrays):
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def ring_reduce_scatter(sends: list, policy: Policy | None = None):
    """sends[r]: rank r's n-element input.  Returns (recv list of n/P arrays, trace)."""
    policy = policy or Policy()
    P = len(sends)
    sends = [np.ascontiguousarray(s) for s in sends]
    dt = dtype_code(sends[0])
    n = sends[0].size
    m = n // P
    recvs = [np.empty(m, dtype=sends[0].dtype) for _ in range(P)]
    ntr = P * (P - 1)
    tr = (_Trace * max(ntr, 1))()
    s0 = (ctypes.c_double * P)()
    sp = (ctypes.c_double * P)()
    pol = policy.c()
    st = lib().orc_ring_reduce_scatter(_ptr_array(sends), _ptr_array(recvs), P, n, dt,
                                       ctypes.byref(pol), tr, s0, sp)
    _check(st, "ring_reduce_scatter")
    return recvs, _trace_list(tr, ntr)


def ring_all_gather(parts: list, sparse_fmt: int = FMT_PICI):
    """parts[q]: rank q's n-element contribution.  Returns (P outputs of P*n, trace)."""
    P = len(parts)
    parts = [np.ascontiguousarray(p) for p in parts]
    dt = dtype_code(parts[0])
    n = parts[0].size
    outs = [np.empty(P * n, dtype=parts[0].dtype) for _ in range(P)]
    tr = (_Trace * P)()
    _check(lib().orc_ring_all_gather(_ptr_array(parts), _ptr_array(outs), P, n, dt, sparse_fmt, tr),
           "ring_all_gather")
    return outs, _trace_list(tr, P)


def ring_all_reduce(sends: list, policy: Policy | None = None):
    """Returns (P outputs of n elements, trace of P*(P-1) + P entries)."""
    policy = policy or Policy()
    P = len(sends)
    sends = [np.ascontiguousarray(s) for s in sends]
    dt = dtype_code(sends[0])
    n = sends[0].size
    outs = [np.empty(n, dtype=sends[0].dtype) for _ in range(P)]
    ntr = P * (P - 1) + P
    tr = (_Trace * ntr)()
    pol = policy.c()
    _check(lib().orc_ring_all_reduce(_ptr_array(sends), _ptr_array(outs), P, n, dt,
                                     ctypes.byref(pol), tr), "ring_all_reduce")
    return outs, _trace_list(tr, ntr)


def header(stream: np.ndarray) -> dict:
    """The header fields of a message (little-endian, Sec. V-B layout)."""
    s = np.ascontiguousarray(stream[:HEADER_BYTES], dtype=np.uint8)
    return {
        "magic": int(s[0:4].view(np.uint32)[0]),
        "format": int(s[4:6].view(np.uint16)[0]),
        "dtype": int(s[6:8].view(np.uint16)[0]),
        "n": int(s[8:16].view(np.uint64)[0]),
        "nnz": int(s[16:24].view(np.uint64)[0]),
        "off_I": int(s[24:32].view(np.uint64)[0]),
        "off_A": int(s[32:40].view(np.uint64)[0]),
        "total_bytes": int(s[40:48].view(np.uint64)[0]),
    }


# ---- sliced streams (Sec. III-B phase 2, Sec. V-B) --------------------------------

SLICE_ELEMS = 16384


def slice_count(n: int) -> int:
    return lib().orc_slice_count(n)


def slice_bytes(dtype: int) -> int:
    """Bytes of one slot: the worst-case message of a full slice."""
    return lib().orc_slice_bytes(dtype)


def slice_len(n: int, q: int) -> int:
    return min(SLICE_ELEMS, n - q * SLICE_ELEMS)


def encode_sliced(dense: np.ndarray, dense_thresh: float = -1.0) -> np.ndarray:
    """The sliced stream of a dense array: slot q holds slice q as a message,
    dense iff that slice's sparsity is <= dense_thresh.  Bytes of a slot past
    its message are zero here (the library leaves them unwritten)."""
    dense = np.ascontiguousarray(dense)
    n, dt = dense.size, dtype_code(dense)
    cap = slice_count(n) * slice_bytes(dt)
    out = np.zeros(max(cap, 1), dtype=np.uint8)
    _check(lib().orc_encode_sliced(_ptr(dense), n, dt, float(dense_thresh), _ptr(out), cap), "encode_sliced")
    return out[:cap]


def decode_sliced(stream: np.ndarray, n: int, dtype: int) -> np.ndarray:
    stream = np.ascontiguousarray(stream, dtype=np.uint8)
    out = np.empty(n, dtype=_np_dtype(dtype))
    _check(lib().orc_decode_sliced(_ptr(stream), stream.nbytes, _ptr(out), n, dtype), "decode_sliced")
    return out


def reduce_sliced(a: np.ndarray, b: np.ndarray, n: int, dtype: int, out_sliced: bool,
                  dense_thresh: float = -1.0) -> np.ndarray:
    """a (dense array) (+) b (sliced stream) -> dense array or sliced stream."""
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b, dtype=np.uint8)
    if out_sliced:
        cap = slice_count(n) * slice_bytes(dtype)
        out = np.zeros(max(cap, 1), dtype=np.uint8)
    else:
        cap = 0
        out = np.empty(n, dtype=_np_dtype(dtype))
    _check(lib().orc_reduce_sliced(_ptr(a), _ptr(b), b.nbytes, 1 if out_sliced else 0, float(dense_thresh),
                                   _ptr(out), cap, n, dtype), "reduce_sliced")
    return out[:cap] if out_sliced else out


def slot_messages(stream: np.ndarray, n: int, dtype: int) -> list:
    """The message bytes of every slot (header.total_bytes of each)."""
    slot = slice_bytes(dtype)
    out = []
    for q in range(slice_count(n)):
        m = stream[q * slot:(q + 1) * slot]
        out.append(m[:int(m[40:48].view(np.uint64)[0])])
    return out


def ring_all_gather_sliced(parts: list):
    """All-gather over sliced streams (every slice Pici).  Returns (P outputs
    of P*n, formats uint8[P, S])."""
    P = len(parts)
    parts = [np.ascontiguousarray(p) for p in parts]
    dt = dtype_code(parts[0])
    n = parts[0].size
    S = slice_count(n)
    outs = [np.empty(P * n, dtype=parts[0].dtype) for _ in range(P)]
    fm = np.zeros(max(1, P * S), dtype=np.uint8)
    _check(lib().orc_ring_all_gather_sliced(_ptr_array(parts), _ptr_array(outs), P, n, dt, _ptr(fm)),
           "ring_all_gather_sliced")
    return outs, fm[:P * S].reshape(P, S)


def ring_all_reduce_sliced(sends: list, policy: Policy | None = None):
    """All-reduce over sliced streams: the sliced reduce-scatter, then the
    all-gather with a per-slice dense switch.  Returns (P outputs of n,
    reduce-scatter formats uint8[P-1, P, S], all-gather formats uint8[P, S]),
    S = slices of a chunk."""
    policy = policy or Policy()
    P = len(sends)
    sends = [np.ascontiguousarray(s) for s in sends]
    dt = dtype_code(sends[0])
    n = sends[0].size
    S = slice_count(n // P)
    outs = [np.empty(n, dtype=sends[0].dtype) for _ in range(P)]
    frs = np.zeros(max(1, (P - 1) * P * S), dtype=np.uint8)
    fag = np.zeros(max(1, P * S), dtype=np.uint8)
    pol = policy.c()
    _check(lib().orc_ring_all_reduce_sliced(_ptr_array(sends), _ptr_array(outs), P, n, dt, ctypes.byref(pol),
                                            _ptr(frs), _ptr(fag)), "ring_all_reduce_sliced")
    return outs, frs[:(P - 1) * P * S].reshape(max(P - 1, 0), P, S), fag[:P * S].reshape(P, S)


def ring_reduce_scatter_sliced(sends: list, policy: Policy | None = None):
    """Ring reduce-scatter over sliced streams with per-slice decisions.
    Returns (recv list of n/P arrays, formats uint8[P-1, P, S]: the format of
    every slice sent at every step by every rank)."""
    policy = policy or Policy()
    P = len(sends)
    sends = [np.ascontiguousarray(s) for s in sends]
    dt = dtype_code(sends[0])
    n = sends[0].size
    m = n // P
    S = slice_count(m)
    recvs = [np.empty(m, dtype=sends[0].dtype) for _ in range(P)]
    fm = np.zeros(max(1, (P - 1) * P * S), dtype=np.uint8)
    pol = policy.c()
    _check(lib().orc_ring_reduce_scatter_sliced(_ptr_array(sends), _ptr_array(recvs), P, n, dt,
                                                ctypes.byref(pol), _ptr(fm)), "ring_reduce_scatter_sliced")
    return recvs, fm[:(P - 1) * P * S].reshape(max(P - 1, 0), P, S)


def time_step(a: np.ndarray, b_msg: np.ndarray, reps: int = 3) -> list:
    """The benchmark step's op sequence on the oracle, timed inside the C
    library (monotonic clock), reps times: compress, decompress, the three
    reductions (dense + Pici -> Pici, Pici + Pici -> Pici, dense + Pici ->
    dense) and a two-part expansion.  Returns each repetition's seconds."""
    a = np.ascontiguousarray(a)
    n, dt = a.size, dtype_code(a)
    cap = stream_bound(n, dt)
    s1, s2, s3 = (np.zeros(cap, dtype=np.uint8) for _ in range(3))
    d1, d2 = np.empty_like(a), np.empty_like(a)
    secs = (ctypes.c_double * reps)()
    _check(lib().orc_time_step(_ptr(a), _ptr(b_msg), b_msg.size, n, dt, _ptr(s1), _ptr(s2), _ptr(s3), cap,
                               _ptr(d1), _ptr(d2), reps, secs), "time_step")
    if not np.array_equal(d1.view(np.uint8), a.view(np.uint8)):
        raise OracleError(4, "time_step: round trip differs")
    return [secs[i] for i in range(reps)]
