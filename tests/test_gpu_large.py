"""GPU parity at the edges of the ABI's range: one canonical message of more
than 2^28 elements (n < 2^32 is accepted, since I is 32-bit, Sec. III-B),
and gather-expands of more parts than one launch takes (the all-gather
receive side, Sec. IV-B).  Whole messages are compared byte for byte with the
oracle's."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import assert_bytes_equal, bits, log, to_dev, to_host_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


N_BIG = (1 << 28) + 4097          # 65,538 tiles: 16,385 partitions of 16,384 elements


@pytest.mark.slow
def test_message_above_2_28_elements(S):
    """compress, dense (+) Pici -> Pici (the reduce-scatter step) and
    Pici (+) Pici -> Pici of 268,439,553 fp32 elements at sparsity 0.99 with
    the full workspace, each in the library's default form (one launch for
    the dense sources) and in two passes: the global offsets of a message of
    more than 16384 partitions, against the oracle byte for byte."""
    n = N_BIG
    assert O.num_tiles(n) == 65538 and -(-O.num_tiles(n) // 4) == 16385
    log(f"large message: generating n={n}")
    a = W.sparse_array(n, W.nnz_for(n, 990), [30, 0, 0, 990], W.F32)
    b = W.sparse_array(n, W.nnz_for(n, 990), [30, 1, 0, 990], W.F32)
    exp_a, nnz_a = O.compress(a)
    exp_b, _ = O.compress(b)
    ws = S.alloc_workspace(n, O.F32)
    out = S.alloc_stream(n, O.F32)
    ta = to_dev(a)
    forms = (("default", 0xFFFFFFFF), ("two passes", 0))
    prev = S.spccl_set_single_pass_limit(0xFFFFFFFF)
    try:
        for form, bound in forms:
            S.spccl_set_single_pass_limit(bound)
            log(f"large message: compress n={n} nnz={nnz_a} ({form})")
            out.fill_(0xA5)
            S.spccl_compress(ta, out, ws)
            torch.cuda.synchronize()
            assert S.spccl_read_status(ws) == 0
            assert_bytes_equal(out[:exp_a.size].cpu().numpy(), exp_a, f"compress above 2^28 ({form})")
            assert S.spccl_read_header(out)["total_bytes"] == exp_a.size

        mb = S.alloc_stream(n, O.F32)
        mb[:exp_b.size].copy_(torch.from_numpy(exp_b))
        pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
        exp_r, _ = O.reduce(O.Operand.array(a), O.Operand.stream(exp_b), n, O.F32, O.STREAM, O.FMT_PICI)
        red = S.alloc_stream(n, O.F32)
        for form, bound in forms:
            S.spccl_set_single_pass_limit(bound)
            log(f"large message: dense (+) Pici -> Pici ({form})")
            red.fill_(0x5A)
            S.spccl_reduce(S.operand(ta), pici(mb), pici(red), n, O.F32, ws)
            torch.cuda.synchronize()
            assert S.spccl_read_status(ws) == 0
            assert_bytes_equal(red[:exp_r.size].cpu().numpy(), exp_r, f"dense (+) Pici above 2^28 ({form})")

        del ta
        exp_pp, _ = O.reduce(O.Operand.stream(exp_a), O.Operand.stream(exp_b), n, O.F32, O.STREAM, O.FMT_PICI)
        for form, bound in forms:
            S.spccl_set_single_pass_limit(bound)
            log(f"large message: Pici (+) Pici -> Pici ({form})")
            red.fill_(0x3C)
            S.spccl_reduce(pici(out), pici(mb), pici(red), n, O.F32, ws)
            torch.cuda.synchronize()
            assert S.spccl_read_status(ws) == 0
            assert_bytes_equal(red[:exp_pp.size].cpu().numpy(), exp_pp, f"Pici (+) Pici above 2^28 ({form})")
    finally:
        S.spccl_set_single_pass_limit(prev)


def _part(S, x, kind, keep):
    """Part x as a device operand of the given kind, from the oracle's encodings."""
    if kind == "array":
        t = to_dev(x)
        keep.append(t)
        return S.operand(t), x
    if kind == "pici":
        msg = O.compress(x)[0]
    elif kind == "coo":
        msg = O.compress_coo(x)[0]
    else:
        msg = O.encode_dense(x)
    t = torch.from_numpy(msg).cuda()
    keep.append(t)
    dt = O.BF16 if x.dtype == np.uint16 else O.F32
    return S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI), O.decompress(msg, x.size, dt)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [65, 130])
def test_gather_expand_past_one_launch(S, P, dtype):
    """More than 64 parts (one launch takes 64): mixed Pici, COO, dense-message
    and array parts of different densities, against the concatenation of the
    oracle's expansions of the same parts."""
    dt = O.BF16 if dtype == W.BF16 else O.F32
    n = 2 * 4096 + 37
    kinds = ["pici", "coo", "array", "dense_msg", "pici"]
    keep, ops, exp = [], [], []
    log(f"gather-expand of {P} parts, {dtype}")
    for q in range(P):
        x = W.sparse_array(n, [0, 5, n // 100, n // 10, n // 2, n][q % 6], [31, P, q], dtype)
        op, e = _part(S, x, kinds[q % len(kinds)], keep)
        ops.append(op)
        exp.append(bits(e))
    ws = S.alloc_workspace(n, dt)
    out = torch.empty(P * n, dtype=torch.bfloat16 if dtype == W.BF16 else torch.float32, device="cuda")
    out.fill_(1.0)
    S.spccl_gather_expand(ops, n, dt, out, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    got = to_host_bits(out)
    want = np.concatenate(exp)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, f"{bad.size} elements differ, first in part {int(bad[0]) // n}"
