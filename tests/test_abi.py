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


def _parts(S, P, n, bad=None, kind=None):
    """P fake device operands (dense arrays of n fp32 at distinct aligned
    addresses); part `bad` is made invalid in the way `kind` says."""
    op = S.spccl_operand_t
    ps = []
    for q in range(P):
        ptr, k, nbytes = (q + 1) << 24, S.SPCCL_ARRAY, 4 * n
        if q == bad:
            if kind == "misaligned":
                ptr += 2
            elif kind == "small":
                nbytes -= 4
            elif kind == "kind":
                k = 7
            elif kind == "overlap":
                ptr = 1 << 34                 # inside the output below
        ps.append(op(k, 0, ptr, nbytes))
    return (op * P)(*ps)


@pytest.mark.parametrize("kind,status", [("misaligned", 1), ("small", 2), ("kind", 1), ("overlap", 1)])
@pytest.mark.parametrize("bad", [0, 64, 100, 129])
def test_gather_expand_checks_every_part_before_any_launch(S, kind, status, bad):
    """A bad part in any 64-part launch chunk is reported before the first
    chunk is launched: without a GPU a launch would fail with ERR_HIP, so the
    part's own error code shows that nothing was launched."""
    P, n = 130, 4096
    parts = _parts(S, P, n, bad, kind)
    out = 1 << 34
    st = S._lib.spccl_gather_expand(parts, P, n, 0, out, P * n * 4, 1 << 40, 1 << 20, None)
    assert st == status


def _vr_call(S, which, send, recv, P, n, scratch, scratch_bytes):
    lib = S._lib
    pol = S.spccl_policy_t(0.6, 0.5, 0.1, 0, 1, 1)
    sp = (ctypes.c_void_p * P)(*send)
    rp = (ctypes.c_void_p * P)(*recv)
    if which == "rs":
        return lib.spccl_vr_reduce_scatter(sp, rp, P, n, 0, ctypes.byref(pol), scratch, scratch_bytes, None, None)
    if which == "ag":
        return lib.spccl_vr_all_gather(sp, rp, P, n, 0, ctypes.byref(pol), scratch, scratch_bytes, None, None)
    if which == "ar":
        return lib.spccl_vr_all_reduce(sp, rp, P, n, 0, ctypes.byref(pol), scratch, scratch_bytes, None, None)
    if which == "rs_sliced":
        return lib.spccl_vr_reduce_scatter_sliced(sp, rp, P, n, 0, ctypes.byref(pol), scratch, scratch_bytes, None,
                                                  None)
    if which == "ag_sliced":
        return lib.spccl_vr_all_gather_sliced(sp, rp, P, n, 0, scratch, scratch_bytes, None, None)
    return lib.spccl_vr_all_reduce_sliced(sp, rp, P, n, 0, ctypes.byref(pol), scratch, scratch_bytes, None, None,
                                          None)


def _scratch_bytes(S, which, P, n):
    m = n if which.startswith("ag") else n // P
    if which.endswith("sliced"):
        return S.spccl_vr_sliced_scratch_bytes(P, m, 0)
    return S.spccl_vr_scratch_bytes(P, m, 0)


GB = 1 << 30


@pytest.mark.parametrize("which", ["rs", "ag", "ar", "rs_sliced", "ag_sliced", "ar_sliced"])
def test_collectives_reject_overlapping_buffers_before_launch(S, which):
    """Overlaps between a rank's receive buffer and another rank's send or
    receive buffer, or between any buffer and the scratch, are rejected on the
    host (INVALID_ARG, where a launch without a GPU would give ERR_HIP)."""
    P, n = 4, 4 * 4096
    s = 4
    rb = n * s if which.startswith(("ag", "ar")) else n // P * s
    if which.startswith("ag"):
        rb = P * n * s
    send = [(1 + r) * GB for r in range(P)]
    recv = [(10 + r) * GB for r in range(P)]
    scratch, sb = 40 * GB, _scratch_bytes(S, which, P, n)
    cases = {
        "recv_in_other_send": (send, [send[1] + 256] + recv[1:], scratch),
        "recv_overlaps_recv": (send, [recv[0], recv[0] + rb // 2] + recv[2:], scratch),
        "recv_in_scratch": (send, recv[:3] + [scratch + 512], scratch),
        "send_in_scratch": ([scratch + 1024] + send[1:], recv, scratch),
    }
    for name, (sd, rv, sc) in cases.items():
        assert _vr_call(S, which, sd, rv, P, n, sc, sb) == 1, name


def test_collectives_in_place_layouts_pass_the_host_checks(S):
    """The in-place layouts the canonical rings handle -- recv[r] as chunk r
    of send[r] (reduce-scatter), send[r] at part r of recv[r] (all-gather) --
    pass the overlap checks; without a GPU the call then fails at its first
    launch (ERR_HIP), which shows the checks let it through.  Any other
    position inside the own buffer is rejected."""
    P, n, s = 4, 4 * 4096, 4
    m = n // P
    send = [(1 + r) * GB for r in range(P)]
    scratch = 40 * GB
    sb = _scratch_bytes(S, "rs", P, n)
    rs_in_place = [send[r] + r * m * s for r in range(P)]
    assert _vr_call(S, "rs", send, rs_in_place, P, n, scratch, sb) == 6
    shifted = [send[r] + ((r + 1) % P) * m * s for r in range(P)]
    assert _vr_call(S, "rs", send, shifted, P, n, scratch, sb) == 1
    recv = [(10 + 2 * r) * GB for r in range(P)]
    sb = _scratch_bytes(S, "ag", P, n)
    ag_in_place = [recv[r] + r * n * s for r in range(P)]
    assert _vr_call(S, "ag", ag_in_place, recv, P, n, scratch, sb) == 6
    shifted = [recv[r] + ((r + 1) % P) * n * s for r in range(P)]
    assert _vr_call(S, "ag", shifted, recv, P, n, scratch, sb) == 1


def test_single_pass_limit_is_a_process_wide_bound(S):
    """spccl_set_single_pass_limit returns the previous bound; the default is
    UINT32_MAX (the library's own one-launch limits); host-only, no launch."""
    first = S.spccl_set_single_pass_limit(0)
    try:
        assert first == 0xFFFFFFFF
        assert S.spccl_set_single_pass_limit(1024) == 0
        assert S.spccl_set_single_pass_limit(1024) == 1024
    finally:
        S.spccl_set_single_pass_limit(first)
    assert S.spccl_set_single_pass_limit(first) == first
