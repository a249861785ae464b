"""GPU parity of the codec, the reduction and the expand kernels against the
CPU oracle, through the C ABI.  Whole messages (header, B, I, pad, A) are
compared byte for byte: the format is exact, and the reductions add in a fixed
order, so every output must be bit-identical."""
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


def make(n, nnz, seed, dtype, specials=False):
    a = W.sparse_array(n, nnz, seed, dtype)
    if specials and n:
        raw = bits(a)
        rng = np.random.default_rng(seed)
        sp = [0x8000, 0x0001, 0x0080] if dtype == W.BF16 else [0x80000000, 0x00000001, 0x00800000]
        for v in sp:
            raw[rng.integers(0, n)] = v
    return a


@pytest.fixture(params=["two_pass", "single_pass"])
def ws_mode(request, S):
    """Full workspace with the count + place passes forced at every size (the
    library otherwise writes small outputs in one pass), or a minimal workspace
    (single-pass look-back)."""
    if request.param != "two_pass":
        yield request.param
        return
    prev = S.spccl_set_single_pass_limit(0)
    try:
        yield request.param
    finally:
        S.spccl_set_single_pass_limit(prev)


def gpu_compress(S, a, ws=None, minimal=False):
    n, dt = a.size, dt_code(W.BF16 if a.dtype == np.uint16 else W.F32)
    ws = S.alloc_workspace(max(n, 1), dt, minimal=minimal) if ws is None else ws
    out = S.alloc_stream(n, dt)
    out.fill_(0xA5)                  # junk: every byte up to total_bytes must be written
    S.spccl_compress(to_dev(a), out, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    return out


SIZES = [0, 1, 63, 64, 4095, 4096, 4097, 3 * 4096 + 77, 4 * 4096, 4 * 4096 + 1, 37 * 4096 + 123]
FRACS = [0.0, 0.01, 0.1, 0.5, 0.7, 1.0]


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", SIZES)
def test_compress_matches_oracle(S, n, dtype, ws_mode):
    for k, frac in enumerate(FRACS):
        nnz = int(round(frac * n))
        log(f"compress n={n} dtype={dtype} nnz={nnz} {ws_mode}")
        a = make(n, nnz, [20, n, k], dtype, specials=frac > 0)
        exp, exp_nnz = O.compress(a)
        out = gpu_compress(S, a, minimal=ws_mode == "single_pass")
        got = out[:exp.size].cpu().numpy()
        assert_bytes_equal(got, exp, f"compress n={n} frac={frac}")
        assert S.spccl_read_header(out)["total_bytes"] == exp.size


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_compress_dense_tiles_two_pass(S, dtype, ws_mode):
    """Tiles with more than 2048 nonzeros (fp32) take the two-half staging path."""
    n = 9 * 4096 + 5
    a = make(n, n - 300, [21], dtype, specials=True)       # nearly all present
    exp, _ = O.compress(a)
    got = gpu_compress(S, a, minimal=ws_mode == "single_pass")[:exp.size].cpu().numpy()
    assert_bytes_equal(got, exp, "dense tiles")


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", [1, 4097, 3 * 4096 + 77, 37 * 4096 + 123])
def test_decompress_round_trip(S, n, dtype):
    dt = dt_code(dtype)
    for k, frac in enumerate([0.0, 0.05, 0.6, 1.0]):
        log(f"decompress n={n} dtype={dtype} frac={frac}")
        a = make(n, int(round(frac * n)), [22, n, k], dtype, specials=frac > 0)
        msg, _ = O.compress(a)
        dmsg = torch.from_numpy(msg).cuda()
        ws = S.alloc_workspace(n, dt)
        out = torch.empty(n, dtype=torch.bfloat16 if dtype == W.BF16 else torch.float32, device="cuda")
        out.fill_(7.0)
        S.spccl_decompress(dmsg, out, ws)
        torch.cuda.synchronize()
        assert S.spccl_read_status(ws) == 0
        assert np.array_equal(to_host_bits(out), bits(a)), first_diff(to_host_bits(out), bits(a))
        # a dense message expands to its values as well
        dm = torch.from_numpy(O.encode_dense(a)).cuda()
        out.fill_(3.0)
        S.spccl_decompress(dm, out, ws)
        torch.cuda.synchronize()
        assert np.array_equal(to_host_bits(out), bits(a))


def _cancel(a, b, k, seed):
    """Make k overlapping positions of b cancel a exactly."""
    both = np.flatnonzero((bits(a) != 0) & (bits(b) != 0))
    if both.size:
        pick = np.random.default_rng(seed).choice(both, size=min(k, both.size), replace=False)
        if a.dtype == np.uint16:
            b[pick] = a[pick] ^ np.uint16(0x8000)
        else:
            b[pick] = -a[pick]


KINDS = ["array", "pici", "dense_msg"]


def _oracle_operand(x, kind):
    if kind == "array":
        return O.Operand.array(x)
    if kind == "pici":
        return O.Operand.stream(O.compress(x)[0])
    return O.Operand.stream(O.encode_dense(x))


def _gpu_operand(S, x, kind, keep):
    if kind == "array":
        t = to_dev(x)
        keep.append(t)
        return S.operand(t)
    msg = O.compress(x)[0] if kind == "pici" else O.encode_dense(x)
    t = torch.from_numpy(msg).cuda()
    keep.append(t)
    fmt = S.SPCCL_FMT_PICI if kind == "pici" else S.SPCCL_FMT_DENSE
    return S.operand(t, S.SPCCL_STREAM, fmt)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("n", [4097, 9 * 4096 + 333])
@pytest.mark.parametrize("ka", KINDS)
@pytest.mark.parametrize("kb", KINDS)
def test_reduce_all_operand_kinds(S, n, dtype, ka, kb, ws_mode):
    dt = dt_code(dtype)
    for k, (fa, fb) in enumerate([(0.02, 0.03), (0.5, 0.4), (0.9, 0.95)]):
        a = make(n, int(fa * n), [23, n, k, 0], dtype, specials=True)
        b = make(n, int(fb * n), [23, n, k, 1], dtype)
        _cancel(a, b, 25, k)
        ws = S.alloc_workspace(n, dt, minimal=ws_mode == "single_pass")
        keep = []
        ga, gb = _gpu_operand(S, a, ka, keep), _gpu_operand(S, b, kb, keep)
        oa, ob = _oracle_operand(a, ka), _oracle_operand(b, kb)
        for out_kind in ("array", "pici", "dense_msg"):
            log(f"reduce n={n} {dtype} {ka}+{kb}->{out_kind} fill=({fa},{fb})")
            if out_kind == "array":
                out = torch.empty(n, dtype=torch.bfloat16 if dtype == W.BF16 else torch.float32, device="cuda")
                out.fill_(9.0)
                S.spccl_reduce(ga, gb, S.operand(out), n, dt, ws)
                torch.cuda.synchronize()
                exp = O.reduce(oa, ob, n, dt)
                got = to_host_bits(out)
                assert np.array_equal(got, bits(exp)), first_diff(got, bits(exp))
            else:
                fmt = S.SPCCL_FMT_PICI if out_kind == "pici" else S.SPCCL_FMT_DENSE
                out = S.alloc_stream(n, dt)
                out.fill_(0x5A)
                S.spccl_reduce(ga, gb, S.operand(out, S.SPCCL_STREAM, fmt), n, dt, ws)
                torch.cuda.synchronize()
                exp, _ = O.reduce(oa, ob, n, dt, O.STREAM, O.FMT_PICI if out_kind == "pici" else O.FMT_DENSE)
                assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"reduce {ka}+{kb}->{out_kind}")
            assert S.spccl_read_status(ws) == 0


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_reduce_in_place(S, dtype):
    n = 5 * 4096 + 17
    dt = dt_code(dtype)
    a = make(n, n // 20, [24, 0], dtype)
    b = make(n, n // 20, [24, 1], dtype)
    ws = S.alloc_workspace(n, dt)
    exp = O.reduce(O.Operand.array(a), O.Operand.stream(O.compress(b)[0]), n, dt)
    ta = to_dev(a)
    tb = torch.from_numpy(O.compress(b)[0]).cuda()
    S.spccl_reduce(S.operand(ta), S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), S.operand(ta), n, dt, ws)
    torch.cuda.synchronize()
    assert np.array_equal(to_host_bits(ta), bits(exp))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_gather_expand_mixed_parts(S, dtype):
    dt = dt_code(dtype)
    n, P = 3 * 4096 + 50, 5
    parts = [make(n, (q + 1) * n // 12, [25, q], dtype, specials=True) for q in range(P)]
    keep, ops = [], []
    for q, x in enumerate(parts):
        kind = ["pici", "array", "dense_msg", "pici", "pici"][q]
        ops.append(_gpu_operand(S, x, kind, keep))
    ws = S.alloc_workspace(n, dt)
    out = torch.empty(P * n, dtype=torch.bfloat16 if dtype == W.BF16 else torch.float32, device="cuda")
    out.fill_(1.0)
    S.spccl_gather_expand(ops, n, dt, out, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    assert np.array_equal(to_host_bits(out), bits(np.concatenate(parts)))


def test_copy_message_device_sized(S):
    n = 5000
    a = make(n, 100, [26], W.F32)
    msg = O.compress(a)[0]
    src = torch.zeros(O.stream_bound(n, O.F32), dtype=torch.uint8, device="cuda")
    src[:msg.size] = torch.from_numpy(msg).cuda()
    dst = torch.full((O.stream_bound(n, O.F32),), 0x77, dtype=torch.uint8, device="cuda")
    ws = S.alloc_workspace(n, O.F32)
    S.spccl_copy_message(src, dst, ws)
    torch.cuda.synchronize()
    got = dst.cpu().numpy()
    assert np.array_equal(got[:msg.size], msg)
    assert (got[msg.size:] == 0x77).all()          # nothing past total_bytes


def test_workspace_reused_across_calls_and_sizes(S, ws_mode):
    """The look-back words carry a per-call epoch: one workspace serves many
    consecutive calls of different sizes without being cleared."""
    ws = S.alloc_workspace(64 * 4096, O.F32, minimal=ws_mode == "single_pass")
    for k, n in enumerate([64 * 4096, 4096, 13 * 4096 + 1, 64 * 4096, 0, 5, 40 * 4096 + 9, 64 * 4096]):
        log(f"ws reuse call {k} n={n}")
        a = make(n, n // 7, [27, k], W.F32)
        exp, _ = O.compress(a)
        got = gpu_compress(S, a, ws)[:exp.size].cpu().numpy()
        assert_bytes_equal(got, exp, f"reuse call {k}")


def test_corrupt_messages_flagged(S):
    n = 3 * 4096
    a = make(n, 500, [28], W.F32)
    msg = O.compress(a)[0]
    ws = S.alloc_workspace(n, O.F32)
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    cases = {"magic": (0, 0xFF), "n": (8, 0x01), "I": (O.off_I(n) + 4, 0x01)}
    for name, (pos, x) in cases.items():
        log(f"corrupt message: {name}")
        bad = msg.copy()
        bad[pos] ^= x
        S.spccl_decompress(torch.from_numpy(bad).cuda(), out, ws)
        assert S.spccl_read_status(ws, clear=True) == 4, name
    # truncated capacity: the header claims more bytes than the buffer holds
    S.spccl_decompress(torch.from_numpy(msg).cuda(), out, ws, msg_bytes=msg.size - 4)
    assert S.spccl_read_status(ws, clear=True) == 4
    # a Pici message passed where a dense one is declared (in a buffer that
    # could hold a dense message, so the host lets it through)
    tm = S.alloc_stream(n, O.F32)
    tm[:msg.size].copy_(torch.from_numpy(msg))
    so = S.alloc_stream(n, O.F32)
    S.spccl_reduce(S.operand(tm, S.SPCCL_STREAM, S.SPCCL_FMT_DENSE), S.operand(to_dev(a)),
                   S.operand(so, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert S.spccl_read_status(ws, clear=True) == 4
    # a buffer smaller than the smallest valid message of its declared format
    # is refused on the host
    with pytest.raises(S.SpcclError) as e:
        S.spccl_reduce(S.operand(tm[:100], S.SPCCL_STREAM, S.SPCCL_FMT_DENSE), S.operand(to_dev(a)),
                       S.operand(so, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert e.value.status == 2
    with pytest.raises(S.SpcclError) as e:
        S.spccl_reduce(S.operand(tm[:O.off_A(n) - 16], S.SPCCL_STREAM, S.SPCCL_FMT_PICI), S.operand(to_dev(a)),
                       S.operand(so, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert e.value.status == 2
    # and the workspace still works afterwards
    got = gpu_compress(S, a, ws)[:msg.size].cpu().numpy()
    assert_bytes_equal(got, msg, "after errors")


def test_bit_beyond_n_flagged(S):
    """A message whose counts agree with I but which sets a bit at a position
    >= n is corrupt (the oracle's decoder rejects it): every kernel that reads
    it flags the status and treats that tile as empty."""
    n = 3 * 4096 - 100                       # last tile: row 63 of every column lies beyond n
    a = make(n, 500, [31], W.F32)
    msg = O.compress(a)[0]
    t = 2
    B = msg[48:48 + 8 * 64 * 3].view(np.uint64).copy()
    col = next(c for c in range(64) if B[64 * t + c] != 0)
    w = int(B[64 * t + col])
    low = w & -w
    w = (w & ~low) | (1 << 63)               # same count: one bit moved past the end
    bad = msg.copy()
    bad[48 + 8 * (64 * t + col):48 + 8 * (64 * t + col) + 8] = np.array([w], dtype=np.uint64).view(np.uint8)
    with pytest.raises(O.OracleError):
        O.decompress(bad, n, O.F32)
    ws = S.alloc_workspace(n, O.F32)
    tb = torch.from_numpy(bad).cuda()
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    log("bit beyond n: decompress")
    S.spccl_decompress(tb, out, ws)
    assert S.spccl_read_status(ws, clear=True) == 4
    log("bit beyond n: pici + pici")
    so = S.alloc_stream(n, O.F32)
    good = torch.from_numpy(msg).cuda()
    S.spccl_reduce(S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), S.operand(good, S.SPCCL_STREAM, S.SPCCL_FMT_PICI),
                   S.operand(so, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert S.spccl_read_status(ws, clear=True) == 4
    log("bit beyond n: dense + pici")
    S.spccl_reduce(S.operand(to_dev(a)), S.operand(tb, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), S.operand(out), n, O.F32,
                   ws)
    assert S.spccl_read_status(ws, clear=True) == 4
    got = gpu_compress(S, a, ws)[:msg.size].cpu().numpy()
    assert_bytes_equal(got, msg, "after errors")


def test_host_errors_launch_nothing(S):
    n = 4096
    ws = S.alloc_workspace(n, O.F32)
    a = to_dev(make(n, 10, [29], W.F32))
    small = torch.empty(100, dtype=torch.uint8, device="cuda")
    with pytest.raises(S.SpcclError) as e:
        S.spccl_compress(a, small, ws)
    assert e.value.status == 2
    with pytest.raises(S.SpcclError) as e:
        S.spccl_compress(a, S.alloc_stream(n, O.F32), ws[:64])
    assert e.value.status == 5
    with pytest.raises(S.SpcclError) as e:            # a stream output may not alias an input
        S.spccl_reduce(S.operand(a), S.operand(a), S.operand(a, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), n, O.F32, ws)
    assert e.value.status in (1, 2)
