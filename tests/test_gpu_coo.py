"""GPU parity of the COO format (Sec. II-B: one flat 32-bit index and one
value per nonzero; Sec. IV-D: the paper's collectives run it beside Pici)
against the CPU oracle, through the C ABI: whole COO messages byte for byte,
dense outputs bit for bit, collective outputs and decision traces exactly.
Corrupt index arrays (out of order, repeated, past the array) must be
flagged without any access outside the message."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import assert_bytes_equal, bits, first_diff, log, to_dev, to_host_bits

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


def dt_code(dtype):
    return O.BF16 if dtype == W.BF16 else O.F32


def tdt(dtype):
    return torch.bfloat16 if dtype == W.BF16 else torch.float32


def make(n, nnz, seed, dtype, specials=False):
    a = W.sparse_array(n, nnz, seed, dtype)
    if specials and n:
        raw = bits(a)
        rng = np.random.default_rng(seed)
        for v in ([0x8000, 0x0001, 0x0080] if dtype == W.BF16 else [0x80000000, 0x00000001, 0x00800000]):
            raw[rng.integers(0, n)] = v
    return a


def gpu_compress_coo(S, a, ws=None):
    n, dt = a.size, dt_code(W.BF16 if a.dtype == np.uint16 else W.F32)
    ws = S.alloc_workspace(max(n, 1), dt) if ws is None else ws
    out = S.alloc_stream(n, dt, fmt=S.SPCCL_FMT_COO)
    out.fill_(0xA5)                  # junk: every byte up to total_bytes must be written
    S.spccl_compress_coo(to_dev(a), out, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    return out


SIZES = [0, 1, 63, 4095, 4096, 4097, 3 * 4096 + 77, 4 * 4096 + 1, 37 * 4096 + 123]
FRACS = [0.0, 0.01, 0.1, 0.5, 0.9, 1.0]


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", SIZES)
def test_compress_coo_matches_oracle(S, n, dtype):
    for k, frac in enumerate(FRACS):
        nnz = int(round(frac * n))
        log(f"coo compress n={n} dtype={dtype} nnz={nnz}")
        a = make(n, nnz, [60, n, k], dtype, specials=frac > 0)
        exp, exp_nnz = O.compress_coo(a)
        out = gpu_compress_coo(S, a)
        assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"coo compress n={n} frac={frac}")
        h = S.spccl_read_header(out)
        assert h["total_bytes"] == exp.size and h["nnz"] == exp_nnz and h["format"] == S.SPCCL_FMT_COO


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", [1, 4097, 3 * 4096 + 77, 37 * 4096 + 123])
def test_decompress_coo(S, n, dtype):
    dt = dt_code(dtype)
    ws = S.alloc_workspace(n, dt)
    out = torch.empty(n, dtype=tdt(dtype), device="cuda")
    for k, frac in enumerate([0.0, 0.05, 0.6, 1.0]):
        log(f"coo decompress n={n} dtype={dtype} frac={frac}")
        a = make(n, int(round(frac * n)), [61, n, k], dtype, specials=frac > 0)
        out.fill_(7.0)
        S.spccl_decompress(torch.from_numpy(O.compress_coo(a)[0]).cuda(), out, ws)
        torch.cuda.synchronize()
        assert S.spccl_read_status(ws) == 0
        got = to_host_bits(out)
        assert np.array_equal(got, bits(a)), first_diff(got, bits(a))


def _cancel(a, b, k, seed):
    both = np.flatnonzero((bits(a) != 0) & (bits(b) != 0))
    if both.size:
        pick = np.random.default_rng(seed).choice(both, size=min(k, both.size), replace=False)
        if a.dtype == np.uint16:
            b[pick] = a[pick] ^ np.uint16(0x8000)
        else:
            b[pick] = -a[pick]


KINDS = ["array", "coo", "dense_msg"]


def _oracle_operand(x, kind):
    if kind == "array":
        return O.Operand.array(x)
    if kind == "coo":
        return O.Operand.stream(O.compress_coo(x)[0])
    return O.Operand.stream(O.encode_dense(x))


def _gpu_operand(S, x, kind, keep):
    if kind == "array":
        t = to_dev(x)
        keep.append(t)
        return S.operand(t)
    msg = O.compress_coo(x)[0] if kind == "coo" else O.encode_dense(x)
    t = torch.from_numpy(msg).cuda()
    keep.append(t)
    return S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_COO if kind == "coo" else S.SPCCL_FMT_DENSE)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", [4097, 9 * 4096 + 333])
@pytest.mark.parametrize("ka", KINDS)
@pytest.mark.parametrize("kb", KINDS)
def test_reduce_coo_operand_kinds(S, n, dtype, ka, kb):
    if ka != "coo" and kb != "coo":
        pytest.skip("covered by the Pici reduce tests unless the output is COO")
    dt = dt_code(dtype)
    ws = S.alloc_workspace(n, dt)
    for k, (fa, fb) in enumerate([(0.02, 0.03), (0.5, 0.4), (0.9, 0.95)]):
        a = make(n, int(fa * n), [62, n, k, 0], dtype, specials=True)
        b = make(n, int(fb * n), [62, n, k, 1], dtype)
        _cancel(a, b, 25, k)
        keep = []
        ga, gb = _gpu_operand(S, a, ka, keep), _gpu_operand(S, b, kb, keep)
        oa, ob = _oracle_operand(a, ka), _oracle_operand(b, kb)
        for out_kind in ("array", "array_search", "coo", "dense_msg"):
            log(f"coo reduce n={n} {dtype} {ka}+{kb}->{out_kind} fill=({fa},{fb})")
            if out_kind.startswith("array"):
                # a full workspace builds a tile index of each COO operand; one
                # of only the control block makes the tiles search J instead
                wsk = ws if out_kind == "array" else torch.zeros(256, dtype=torch.uint8, device="cuda")
                out = torch.empty(n, dtype=tdt(dtype), device="cuda")
                out.fill_(9.0)
                S.spccl_reduce(ga, gb, S.operand(out), n, dt, wsk)
                torch.cuda.synchronize()
                exp = O.reduce(oa, ob, n, dt)
                got = to_host_bits(out)
                assert np.array_equal(got, bits(exp)), first_diff(got, bits(exp))
                assert S.spccl_read_status(wsk) == 0
            else:
                fmt = S.SPCCL_FMT_COO if out_kind == "coo" else S.SPCCL_FMT_DENSE
                out = S.alloc_stream(n, dt, fmt=S.SPCCL_FMT_COO)
                out.fill_(0x5A)
                S.spccl_reduce(ga, gb, S.operand(out, S.SPCCL_STREAM, fmt), n, dt, ws)
                torch.cuda.synchronize()
                exp, _ = O.reduce(oa, ob, n, dt, O.STREAM, O.FMT_COO if out_kind == "coo" else O.FMT_DENSE)
                assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"coo reduce {ka}+{kb}->{out_kind}")
            assert S.spccl_read_status(ws) == 0


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_dense_operands_into_coo(S, dtype):
    """dense (+) dense and dense alone into a COO message (the RS step of a
    collective whose incoming message was dense)."""
    n, dt = 5 * 4096 + 17, dt_code(dtype)
    a = make(n, n // 10, [63, 0], dtype, specials=True)
    b = make(n, n // 10, [63, 1], dtype)
    _cancel(a, b, 30, 3)
    ws = S.alloc_workspace(n, dt)
    out = S.alloc_stream(n, dt, fmt=S.SPCCL_FMT_COO)
    ta, tb = to_dev(a), to_dev(b)                  # both alive until the kernels have run
    S.spccl_reduce(S.operand(ta), S.operand(tb), S.operand(out, S.SPCCL_STREAM, S.SPCCL_FMT_COO), n, dt, ws)
    torch.cuda.synchronize()
    exp, _ = O.reduce(O.Operand.array(a), O.Operand.array(b), n, dt, O.STREAM, O.FMT_COO)
    assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, "dense+dense->coo")


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_reduce_in_place_coo(S, dtype):
    n, dt = 5 * 4096 + 17, dt_code(dtype)
    a = make(n, n // 20, [64, 0], dtype)
    b = make(n, n // 20, [64, 1], dtype)
    ws = S.alloc_workspace(n, dt)
    exp = O.reduce(O.Operand.array(a), O.Operand.stream(O.compress_coo(b)[0]), n, dt)
    ta = to_dev(a)
    tb = torch.from_numpy(O.compress_coo(b)[0]).cuda()
    S.spccl_reduce(S.operand(ta), S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_COO), S.operand(ta), n, dt, ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_host_bits(ta), bits(exp))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_gather_expand_with_coo_parts(S, dtype):
    dt = dt_code(dtype)
    n, P = 3 * 4096 + 50, 5
    parts = [make(n, (q + 1) * n // 12, [65, q], dtype, specials=True) for q in range(P)]
    keep, ops = [], []
    for q, x in enumerate(parts):
        kind = ["coo", "array", "dense_msg", "pici", "coo"][q]
        if kind == "pici":
            t = torch.from_numpy(O.compress(x)[0]).cuda()
            keep.append(t)
            ops.append(S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI))
        else:
            ops.append(_gpu_operand(S, x, kind, keep))
    ws = S.alloc_workspace(n, dt)
    out = torch.empty(P * n, dtype=tdt(dtype), device="cuda")
    out.fill_(1.0)
    S.spccl_gather_expand(ops, n, dt, out, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    assert np.array_equal(to_host_bits(out), bits(np.concatenate(parts)))


def _coo_with(msg, J=None):
    m = msg.copy()
    nnz = int(m[16:24].view(np.uint64)[0])
    if J is not None:
        m[48:48 + 4 * nnz] = np.asarray(J, dtype=np.uint32).view(np.uint8)
    return m


def test_corrupt_coo_flagged(S):
    n = 3 * 4096 + 100
    a = make(n, 300, [67], W.F32)
    msg, nnz = O.compress_coo(a)
    J = msg[48:48 + 4 * nnz].view(np.uint32).copy()
    ws = S.alloc_workspace(n, O.F32)
    small = torch.zeros(256, dtype=torch.uint8, device="cuda")       # the control block only: no tile index
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    dense_out = torch.empty(n, dtype=torch.float32, device="cuda")
    coo_out = S.alloc_stream(n, O.F32, fmt=S.SPCCL_FMT_COO)
    swapped = J.copy(); swapped[[10, 11]] = swapped[[11, 10]]                # out of order inside a tile
    across = J.copy(); across[[5, nnz - 5]] = across[[nnz - 5, 5]]           # entries swapped across tiles
    dup = J.copy(); dup[20] = dup[19]                                        # repeated index
    past = J.copy(); past[-1] = n + 3                                        # past the array, last tile
    huge = J.copy(); huge[-1] = 0xFFFFFFF0                                   # far past the array
    first = J.copy(); first[0] = 4096 * 2 + 1                                # first entry belongs to a later tile
    cases = {"swapped": swapped, "across": across, "dup": dup, "past": past, "huge": huge, "first": first}
    for name, Jb in cases.items():
        bad = _coo_with(msg, Jb)
        assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM, name
        tb = torch.from_numpy(bad).cuda()
        log(f"corrupt coo {name}: decompress")
        S.spccl_decompress(tb, out, ws)
        assert S.spccl_read_status(ws, clear=True) == 4, name
        log(f"corrupt coo {name}: dense + coo -> dense (tile index, then search)")
        for wsk in (ws, small):
            S.spccl_reduce(S.operand(to_dev(a)), S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_COO),
                           S.operand(dense_out), n, O.F32, wsk)
            assert S.spccl_read_status(wsk, clear=True) == 4, name
        log(f"corrupt coo {name}: coo + dense -> coo")
        S.spccl_reduce(S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_COO), S.operand(to_dev(a)),
                       S.operand(coo_out, S.SPCCL_STREAM, S.SPCCL_FMT_COO), n, O.F32, ws)
        assert S.spccl_read_status(ws, clear=True) == 4, name
    # header offsets that disagree with nnz
    bad = msg.copy(); bad[32] ^= 16
    S.spccl_decompress(torch.from_numpy(bad).cuda(), out, ws)
    assert S.spccl_read_status(ws, clear=True) == 4
    # truncated capacity
    S.spccl_decompress(torch.from_numpy(msg).cuda(), out, ws, msg_bytes=msg.size - 4)
    assert S.spccl_read_status(ws, clear=True) == 4
    # the workspace still works
    got = gpu_compress_coo(S, a, ws)[:msg.size].cpu().numpy()
    assert_bytes_equal(got, msg, "after errors")


def test_coo_tile_index_gaps_and_zigzag(S):
    """The tile index leaves runs of more than 64 empty tiles to the search
    of J, and a corrupt J that jumps back and forth costs a bounded pass."""
    n = 300 * 4096 + 123
    ws = S.alloc_workspace(n, O.F32)
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    a = make(n, 2000, [70], W.F32)
    for name, keep in (("first and last tiles", lambda i: (i < 3 * 4096) | (i >= 290 * 4096)),
                       ("one entry in the middle", lambda i: i == 150 * 4096 + 7),
                       ("no entries", lambda i: i < 0)):
        b = make(n, 5000, [71], W.F32)
        b[~keep(np.arange(n))] = 0
        msg, _ = O.compress_coo(b)
        log(f"coo index gaps: {name}")
        S.spccl_reduce(S.operand(to_dev(a)), S.operand(torch.from_numpy(msg).cuda(), S.SPCCL_STREAM,
                       S.SPCCL_FMT_COO), S.operand(out), n, O.F32, ws)
        torch.cuda.synchronize()
        assert S.spccl_read_status(ws, clear=True) == 0, name
        exp = O.reduce(O.Operand.array(a), O.Operand.stream(msg), n, O.F32)
        assert np.array_equal(to_host_bits(out), bits(exp)), name
    b = make(n, 4096, [72], W.F32)
    msg, nnz = O.compress_coo(b)
    J = msg[48:48 + 4 * nnz].view(np.uint32).copy()
    J[1::2] = n - 1 - np.arange(J[1::2].size, dtype=np.uint32)      # every other entry jumps to the end
    bad = _coo_with(msg, J)
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM
    log("coo index zigzag")
    S.spccl_reduce(S.operand(to_dev(a)), S.operand(torch.from_numpy(bad).cuda(), S.SPCCL_STREAM, S.SPCCL_FMT_COO),
                   S.operand(out), n, O.F32, ws)
    assert S.spccl_read_status(ws, clear=True) == 4


def test_coo_host_errors(S):
    n = 4096
    a = to_dev(make(n, 10, [68], W.F32))
    ws = S.alloc_workspace(n, O.F32)
    small_ws = S.alloc_workspace(n, O.F32, minimal=True)
    out = S.alloc_stream(n, O.F32, fmt=S.SPCCL_FMT_COO)
    with pytest.raises(S.SpcclError) as e:                       # the COO sink needs its slots
        S.spccl_compress_coo(a, out, small_ws)
    assert e.value.status == 5
    with pytest.raises(S.SpcclError) as e:                       # capacity below the COO worst case
        S.spccl_compress_coo(a, S.alloc_stream(n, O.F32), ws)
    assert e.value.status == 2
    pici = torch.from_numpy(O.compress(make(n, 10, [69], W.F32))[0]).cuda()
    coo = torch.from_numpy(O.compress_coo(make(n, 10, [69], W.F32))[0]).cuda()
    with pytest.raises(S.SpcclError) as e:                       # Pici and COO do not meet
        S.spccl_reduce(S.operand(pici, S.SPCCL_STREAM, S.SPCCL_FMT_PICI),
                       S.operand(coo, S.SPCCL_STREAM, S.SPCCL_FMT_COO), S.operand(torch.empty_like(a)), n, O.F32, ws)
    assert e.value.status == 3
    with pytest.raises(S.SpcclError) as e:
        S.spccl_reduce(S.operand(a), S.operand(coo, S.SPCCL_STREAM, S.SPCCL_FMT_COO),
                       S.operand(S.alloc_stream(n, O.F32), S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert e.value.status == 3
    assert S.spccl_coo_bytes(O.F32, 7) == O.coo_bytes(O.F32, 7)
    for fmt in (0, 1, 2):
        assert S.spccl_message_bound(n, O.F32, fmt) == O.message_bound(n, O.F32, fmt)


# ---- collectives with COO sends (Sec. IV-D) ---------------------------------------------------

def run_rs(S, sends, policy):
    P, n = len(sends), sends[0].size
    m = n // P
    dt = O.dtype_code(sends[0])
    ts = [to_dev(x) for x in sends]
    outs = [torch.empty(m, dtype=torch.bfloat16 if dt else torch.float32, device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, m, dt), dtype=torch.uint8, device="cuda")
    tr = S.spccl_vr_reduce_scatter(ts, outs, scratch, policy)
    return [to_host_bits(o) for o in outs], tr


def trace_tuple(e):
    return (e.step, e.rank, e.fmt, e.measured, e.bytes, e.nnz, e.sigma)


def check_trace(gpu_tr, orc_tr):
    assert len(gpu_tr) == len(orc_tr)
    for g, o in zip(gpu_tr, orc_tr):
        assert g == trace_tuple(o), f"gpu {g} vs oracle {trace_tuple(o)}"


POLICIES = {
    "coo": O.Policy.coo(),
    "coo_never_dense": O.Policy.coo(adaptive=0),
    "coo_always_dense": O.Policy.coo(adaptive=2),
    "coo_two_nodes": O.Policy.coo(ranks_per_node=2),
}


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("pol", list(POLICIES))
def test_reduce_scatter_coo_matches_oracle(S, dtype, P, pol):
    m = 2 * 4096 + 123
    frac = [0.3, 0.02, 0.15][P % 3]
    sends = [W.sparse_array(P * m, int(frac * P * m), [70, P, r], dtype) for r in range(P)]
    log(f"coo rs P={P} dtype={dtype} policy={pol}")
    got, gtr = run_rs(S, sends, POLICIES[pol])
    exp, otr = O.ring_reduce_scatter(sends, POLICIES[pol])
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r])), f"rank {r}: {first_diff(got[r], bits(exp[r]))}"
    check_trace(gtr, otr)


def test_reduce_scatter_coo_decision_trace_hand_computed(S):
    """COO thresholds on the digit inputs: steps 0-1 COO (0.9, 0.81), steps
    2-6 dense (Sec. IV-C, IV-D)."""
    from test_oracle_coo import _digit_sparsity_inputs
    P, m = 8, 10000
    sends = _digit_sparsity_inputs(P, m, 4)
    got, gtr = run_rs(S, sends, O.Policy.coo())
    exp, otr = O.ring_reduce_scatter(sends, O.Policy.coo())
    check_trace(gtr, otr)
    assert [g[2] for g in gtr if g[1] == 0] == [2, 2, 0, 0, 0, 0, 0]
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r]))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 2, 5])
def test_all_gather_coo_matches_oracle(S, dtype, P):
    n = 3 * 4096 + 11
    parts = [W.sparse_array(n, (r + 1) * n // 40, [71, P, r], dtype) for r in range(P)]
    dt = O.dtype_code(parts[0])
    log(f"coo ag P={P} dtype={dtype}")
    ts = [to_dev(x) for x in parts]
    outs = [torch.empty(P * n, dtype=tdt(dtype), device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, n, dt), dtype=torch.uint8, device="cuda")
    gtr = S.spccl_vr_all_gather(ts, outs, scratch, O.Policy.coo())
    exp, otr = O.ring_all_gather(parts, O.FMT_COO)
    cat = bits(np.concatenate(parts))
    for r in range(P):
        assert np.array_equal(to_host_bits(outs[r]), cat)
    check_trace(gtr, otr)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 4, 8])
@pytest.mark.parametrize("pol", ["coo", "coo_never_dense", "coo_always_dense"])
def test_all_reduce_coo_matches_oracle(S, dtype, P, pol):
    m = 4096 + 77
    sends = [W.sparse_array(P * m, P * m // 6, [72, P, r], dtype) for r in range(P)]
    dt = O.dtype_code(sends[0])
    log(f"coo ar P={P} dtype={dtype} policy={pol}")
    ts = [to_dev(x) for x in sends]
    outs = [torch.empty(P * m, dtype=tdt(dtype), device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, m, dt), dtype=torch.uint8, device="cuda")
    gtr = S.spccl_vr_all_reduce(ts, outs, scratch, POLICIES[pol])
    exp, otr = O.ring_all_reduce(sends, POLICIES[pol])
    for r in range(P):
        got = to_host_bits(outs[r])
        assert np.array_equal(got, bits(exp[r])), f"rank {r}: {first_diff(got, bits(exp[r]))}"
    check_trace(gtr, otr)


@pytest.mark.slow
@pytest.mark.parametrize("permille", [500, 990])
def test_config2_coo_codec(S, permille):
    """The 256 MiB codec array in COO: compress, decompress (2 tiles per
    wave) and a 2-part gather of the message (4 tiles per wave: each wave's
    entry range is searched once and its tiles' boundaries inside it)."""
    n = W.CFG2_N
    log(f"cfg2 coo sigma={permille / 1000} generate")
    a = W.cfg2(permille, 0)
    ws = S.alloc_workspace(n, O.F32)
    log(f"cfg2 coo sigma={permille / 1000} compress")
    out = gpu_compress_coo(S, a, ws)
    exp, nnz = O.compress_coo(a)
    assert nnz == W.nnz_for(n, permille)
    assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"cfg2 coo compress {permille}")
    del exp
    one = torch.empty(n, dtype=torch.float32, device="cuda")
    log(f"cfg2 coo sigma={permille / 1000} decompress")
    S.spccl_decompress(out, one, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    assert np.array_equal(to_host_bits(one), bits(a)), "cfg2 coo decompress"
    del one
    back = torch.empty(2 * n, dtype=torch.float32, device="cuda")
    log(f"cfg2 coo sigma={permille / 1000} gather 2 parts")
    op = S.operand(out, S.SPCCL_STREAM, S.SPCCL_FMT_COO)
    S.spccl_gather_expand([op, op], n, O.F32, back, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    got = to_host_bits(back)
    assert np.array_equal(got[:n], bits(a)) and np.array_equal(got[n:], bits(a)), "cfg2 coo round trip"
