"""CPU checks of the C ABI: the library loads, exports every function the
header declares, its host-side size arithmetic agrees with the oracle, and
host-detectable errors are returned before anything is launched (so these run
without a GPU)."""
import ctypes
import os
import re

import pytest

import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spccl.h")


@pytest.fixture(scope="module")
def S():
    import paper_2607_04676_amd as S
    return S


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(spccl_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_expected_entry_points():
    names = declared_functions()
    for must in ("spccl_compress", "spccl_decompress", "spccl_reduce", "spccl_gather_expand"):
        assert must in names


def test_library_exports_every_declared_symbol(S):
    lib = ctypes.CDLL(S.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(S.EXPORTS) == declared_functions()


def test_no_oracle_linkage(S):
    """The product library neither links nor names the oracle."""
    data = open(S.LIB_PATH, "rb").read()
    assert b"liboracle" not in data and b"orc_compress" not in data


@pytest.mark.parametrize("n", [0, 1, 4095, 4096, 4097, 1 << 20, (1 << 26) + 3])
@pytest.mark.parametrize("dt", [O.F32, O.BF16])
def test_sizes_agree_with_oracle(S, n, dt):
    assert S.spccl_num_tiles(n) == O.num_tiles(n)
    assert S.spccl_stream_bound(n, dt) == O.stream_bound(n, dt)
    for nnz in (0, 1, n // 3, n):
        assert S.spccl_pici_bytes(n, dt, nnz) == O.pici_bytes(n, dt, nnz)
    assert S.spccl_workspace_bytes(n, dt) >= 256 + 8


def test_bad_dtype_and_sizes_rejected_on_host(S):
    lib = S._lib
    assert S.spccl_stream_bound(10, 7) == 0
    assert lib.spccl_compress(None, 10, 7, None, 0, None, 0, None) == 3          # unsupported dtype
    assert lib.spccl_compress(None, 1 << 32, 0, None, 0, None, 0, None) == 3     # n >= 2^32
    assert lib.spccl_compress(None, 10, 0, None, 0, None, 0, None) == 1          # null pointers
    assert lib.spccl_compress(16, 10, 0, 32, 0, 64, 1 << 20, None) == 2          # capacity
    assert lib.spccl_compress(17, 10, 0, 32, 1 << 20, 64, 1 << 20, None) == 1    # misaligned input
    assert lib.spccl_compress(16, 10, 0, 1 << 20, 1 << 20, 64, 8, None) == 5     # workspace too small
    assert lib.spccl_copy_message(16, 8, 4096, 100, 8192, 256, None) == 2        # source smaller than a header
    assert S.spccl_status_string(4) == "corrupt message"


def test_reduce_operand_checks_on_host(S):
    lib = S._lib
    op = S.spccl_operand_t
    a = op(S.SPCCL_ARRAY, 0, 1 << 20, 4 * 100)
    b = op(S.SPCCL_STREAM, S.SPCCL_FMT_PICI, 2 << 20, 1000)
    ws = 4 << 20
    # a Pici output that overlaps an input
    out = op(S.SPCCL_STREAM, S.SPCCL_FMT_PICI, (1 << 20) + 16, 1 << 16)
    assert lib.spccl_reduce(a, b, out, 100, 0, ws, 1 << 12, None) == 1
    # an array output too small
    out = op(S.SPCCL_ARRAY, 0, 3 << 20, 4 * 99)
    assert lib.spccl_reduce(a, b, out, 100, 0, ws, 1 << 12, None) == 2
    # an unknown format
    bad = op(S.SPCCL_STREAM, 9, 2 << 20, 1000)
    assert lib.spccl_reduce(a, bad, op(S.SPCCL_ARRAY, 0, 3 << 20, 400), 100, 0, ws, 1 << 12, None) == 1


def test_vr_argument_checks_on_host(S):
    lib = S._lib
    P = 4
    ptrs = (ctypes.c_void_p * P)(*[(k + 1) << 24 for k in range(P)])
    outs = (ctypes.c_void_p * P)(*[(k + 9) << 24 for k in range(P)])
    pol = S.spccl_policy_t(0.6, 0.5, 0.1, 0, 1)
    # n not divisible by P
    assert lib.spccl_vr_reduce_scatter(ptrs, outs, P, 4097, 0, ctypes.byref(pol), 1 << 30, 1 << 30, None, None) == 1
    # scratch too small
    assert lib.spccl_vr_reduce_scatter(ptrs, outs, P, 4096, 0, ctypes.byref(pol), 1 << 30, 16, None, None) == 5
    need = S.spccl_vr_scratch_bytes(P, 1024, 0)
    assert need >= 3 * P * O.stream_bound(1024, O.F32)


def test_operand_keeps_its_tensor_alive(S):
    """An operand built from a temporary tensor holds it: the memory behind the
    operand's pointer is not released (and reused by the next allocation)
    while the operand is still in use."""
    import gc
    import weakref
    torch = pytest.importorskip("torch")
    t = torch.arange(8, dtype=torch.float32)
    ref = weakref.ref(t)
    op = S.operand(t)
    ptr = t.data_ptr()
    del t
    gc.collect()
    assert ref() is not None and op.ptr == ptr
    del op
    gc.collect()
    assert ref() is None
