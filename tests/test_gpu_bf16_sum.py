"""GPU parity of the bf16 (+) on its hard cases (Sec. IV-B reduces bf16 data;
the sum is the correctly rounded bfloat16 of the exact sum, absent elements
being the identity): ties to even, subnormals, overflow to infinity, exact
cancellations and -0.0, plus random finite bit patterns over the whole
exponent range, through every kernel that adds (dense (+) dense, dense (+)
Pici with a dense or a Pici result, Pici (+) Pici), against the oracle bit
for bit."""
import numpy as np
import pytest

import oracle as O
from helpers import assert_bytes_equal, bits, first_diff, log, to_dev, to_host_bits

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


# (a, b) bit patterns and what makes each hard
PAIRS = [
    (0x3F80, 0x3B80),   # 1 + 2^-8: halfway between 1 and 1 + 2^-7, to even (1)
    (0x3F81, 0x3B80),   # (1 + 2^-7) + 2^-8: halfway, to even (1 + 2^-6)
    (0xBF80, 0xBB80),   # the negative tie
    (0x4380, 0x3F80),   # 256 + 1: halfway between 256 and 258, to even (256)
    (0x4381, 0x3F80),   # 258 + 1: halfway between 258 and 260, to even (260)
    (0x4B80, 0x3F80),   # 2^24 + 1: far below half a unit, stays 2^24
    (0x0001, 0x0001),   # two smallest subnormals
    (0x007F, 0x0001),   # largest subnormal + smallest: the smallest normal
    (0x0080, 0x8001),   # smallest normal - smallest subnormal: a subnormal
    (0x0001, 0x8001),   # subnormals that cancel exactly: absent
    (0x3F80, 0xBF80),   # 1 - 1: absent
    (0x7F7F, 0x7F7F),   # largest finite twice: +inf
    (0x7F7F, 0x7B00),   # largest + half its unit: halfway, to even (+inf)
    (0x7F7F, 0x7A80),   # largest + a quarter of its unit: stays the largest
    (0xFF7F, 0xFB00),   # the same below zero: -inf
    (0x8000, 0x8000),   # -0.0 + -0.0 = -0.0, present
    (0x8000, 0x3F80),   # -0.0 + 1 = 1
    (0x8000, 0x0000),   # -0.0 with b absent: -0.0 kept
    (0x0000, 0x8000),   # a absent, b -0.0: kept
]


def operands(n, seed, sparse_b):
    rng = np.random.default_rng(seed)
    a = rng.integers(0, 1 << 16, n, dtype=np.uint32).astype(np.uint16)
    b = rng.integers(0, 1 << 16, n, dtype=np.uint32).astype(np.uint16)
    for x in (a, b):                             # finite patterns only (NaN is outside the contract)
        bad = (x & 0x7F80) == 0x7F80
        x[bad] &= 0x807F
        x[rng.random(n) < 0.3] = 0               # absent elements on both sides
    if sparse_b:                                 # a sparse Pici side (the sparse merge paths)
        b[rng.random(n) < 0.99] = 0
    pos = rng.choice(n, size=4 * len(PAIRS), replace=False)
    for k, p in enumerate(pos):
        a[p], b[p] = PAIRS[k % len(PAIRS)]
    return a, b


@pytest.mark.parametrize("sparse_b", [False, True], ids=["dense_b", "sparse_b"])
@pytest.mark.parametrize("n", [4096 + 5, 5 * 4096 + 123])
def test_bf16_sum_hard_cases(S, n, sparse_b):
    a, b = operands(n, 77 + n, sparse_b)
    dt = O.BF16
    ws = S.alloc_workspace(n, dt)
    ma, mb = O.compress(a)[0], O.compress(b)[0]
    ta, tb = to_dev(a), to_dev(b)
    pa, pb = torch.from_numpy(ma).cuda(), torch.from_numpy(mb).cuda()
    pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    oa, ob = O.Operand.array(a), O.Operand.array(b)
    exp_dense = O.reduce(oa, ob, n, dt)

    for name, ga, gb in (("dense+dense", S.operand(ta), S.operand(tb)),
                         ("dense+pici", S.operand(ta), pici(pb)),
                         ("pici+pici", pici(pa), pici(pb))):
        log(f"bf16 sum n={n} sparse_b={sparse_b} {name} -> array")
        out = torch.empty(n, dtype=torch.bfloat16, device="cuda")
        out.fill_(3.0)
        S.spccl_reduce(ga, gb, S.operand(out), n, dt, ws)
        torch.cuda.synchronize()
        got = to_host_bits(out)
        assert np.array_equal(got, bits(exp_dense)), f"{name}: {first_diff(got, bits(exp_dense))}"

    exp_msg, _ = O.reduce(oa, ob, n, dt, O.STREAM, O.FMT_PICI)
    for name, ga, gb in (("dense+pici", S.operand(ta), pici(pb)), ("pici+pici", pici(pa), pici(pb)),
                         ("dense+dense", S.operand(ta), S.operand(tb))):
        log(f"bf16 sum n={n} sparse_b={sparse_b} {name} -> pici")
        red = S.alloc_stream(n, dt)
        red.fill_(0x5A)
        S.spccl_reduce(ga, gb, pici(red), n, dt, ws)
        torch.cuda.synchronize()
        assert_bytes_equal(red[:exp_msg.size].cpu().numpy(), exp_msg, f"bf16 {name} -> pici")
    assert S.spccl_read_status(ws) == 0
