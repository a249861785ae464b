"""GPU parity of the virtual-rank ring collectives (reduce-scatter, all-gather,
all-reduce over P buffers on one device) against the oracle's ring: outputs
bit for bit, and the per-step send decisions (format, bytes, nonzeros,
tracked sparsity) exactly."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import bits, first_diff, log, to_dev, to_host_bits

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


@pytest.fixture(params=["one_launch", "two_passes"])
def passes(request, S):
    """The ring steps' Pici outputs in the library's default form (one launch
    with the two-level look-back) or forced onto the count and place passes."""
    if request.param == "one_launch":
        yield request.param
        return
    prev = S.spccl_set_single_pass_limit(0)
    try:
        yield request.param
    finally:
        S.spccl_set_single_pass_limit(prev)


def tdt(x):
    return torch.bfloat16 if x.dtype == np.uint16 else torch.float32


def run_rs(S, sends, policy):
    P, n = len(sends), sends[0].size
    m = n // P
    dt = O.dtype_code(sends[0])
    ts = [to_dev(x) for x in sends]
    outs = [torch.empty(m, dtype=tdt(sends[0]), device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, m, dt), dtype=torch.uint8, device="cuda")
    tr = S.spccl_vr_reduce_scatter(ts, outs, scratch, policy)
    return [to_host_bits(o) for o in outs], tr


def run_ar(S, sends, policy):
    P, n = len(sends), sends[0].size
    dt = O.dtype_code(sends[0])
    ts = [to_dev(x) for x in sends]
    outs = [torch.empty(n, dtype=tdt(sends[0]), device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, n // P, dt), dtype=torch.uint8, device="cuda")
    tr = S.spccl_vr_all_reduce(ts, outs, scratch, policy)
    return [to_host_bits(o) for o in outs], tr


def trace_tuple(e):
    return (e.step, e.rank, e.fmt, e.measured, e.bytes, e.nnz, e.sigma)


def check_trace(gpu_tr, orc_tr):
    assert len(gpu_tr) == len(orc_tr)
    for g, o in zip(gpu_tr, orc_tr):
        assert g == trace_tuple(o), f"gpu {g} vs oracle {trace_tuple(o)}"


POLICIES = {
    "default": O.Policy(),
    "never_dense": O.Policy(adaptive=0),
    "always_dense": O.Policy(adaptive=2),
    "two_nodes": O.Policy(ranks_per_node=2),
}


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("pol", list(POLICIES))
def test_reduce_scatter_matches_oracle(S, dtype, P, pol, passes):
    m = 2 * 4096 + 123
    frac = [0.3, 0.02, 0.15][P % 3]
    sends = [W.sparse_array(P * m, int(frac * P * m), [40, P, r], dtype) for r in range(P)]
    log(f"rs P={P} dtype={dtype} policy={pol} {passes}")
    got, gtr = run_rs(S, sends, POLICIES[pol])
    exp, otr = O.ring_reduce_scatter(sends, POLICIES[pol])
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r])), f"rank {r}: {first_diff(got[r], bits(exp[r]))}"
    check_trace(gtr, otr)


def test_reduce_scatter_decision_trace_hand_computed(S):
    """The digit-supported inputs whose measured sparsity after k ranks is
    exactly 0.9^k: steps 0-3 Pici, 4-6 dense (Sec. IV-C, Eq. 7)."""
    from test_oracle_pins import _digit_sparsity_inputs
    P, m = 8, 10000
    sends = _digit_sparsity_inputs(P, m, 4)
    got, gtr = run_rs(S, sends, O.Policy())
    exp, otr = O.ring_reduce_scatter(sends, O.Policy())
    check_trace(gtr, otr)
    assert [g[2] for g in gtr if g[1] == 0] == [1, 1, 1, 1, 0, 0, 0]
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r]))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 2, 5])
def test_all_gather_matches_oracle(S, dtype, P, passes):
    n = 3 * 4096 + 11
    parts = [W.sparse_array(n, (r + 1) * n // 40, [41, P, r], dtype) for r in range(P)]
    dt = O.dtype_code(parts[0])
    log(f"ag P={P} dtype={dtype} {passes}")
    ts = [to_dev(x) for x in parts]
    outs = [torch.empty(P * n, dtype=tdt(parts[0]), device="cuda") for _ in range(P)]
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P, n, dt), dtype=torch.uint8, device="cuda")
    gtr = S.spccl_vr_all_gather(ts, outs, scratch)
    exp, otr = O.ring_all_gather(parts)
    cat = bits(np.concatenate(parts))
    for r in range(P):
        assert np.array_equal(to_host_bits(outs[r]), cat)
    check_trace(gtr, otr)


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("P", [1, 4, 8])
@pytest.mark.parametrize("pol", ["default", "never_dense", "always_dense"])
def test_all_reduce_matches_oracle(S, dtype, P, pol, passes):
    m = 4096 + 77
    sends = [W.sparse_array(P * m, P * m // 6, [42, P, r], dtype) for r in range(P)]
    log(f"ar P={P} dtype={dtype} policy={pol} {passes}")
    got, gtr = run_ar(S, sends, POLICIES[pol])
    exp, otr = O.ring_all_reduce(sends, POLICIES[pol])
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r])), f"rank {r}: {first_diff(got[r], bits(exp[r]))}"
        assert np.array_equal(got[r], got[0])
    check_trace(gtr, otr)


def test_all_reduce_phase_aware_both_formats(S):
    """Per-rank densities straddle ag_thresh, so the all-gather mixes dense and
    Pici messages; the result must not depend on the mix."""
    P, m = 4, 4096
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            stride = 4 if c % 2 == 0 else 64                # chunks 0, 2 denser, 1, 3 sparser
            x[c * m:(c + 1) * m][((r - c) % P)::stride] = np.float32(1 + r)
        sends.append(x)
    pol = O.Policy(ag_thresh=0.4)                           # transition estimates 0.484 / 0.316
    got, gtr = run_ar(S, sends, pol)
    exp, otr = O.ring_all_reduce(sends, pol)
    check_trace(gtr, otr)
    assert {g[2] for g in gtr[P * (P - 1):]} == {0, 1}
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r]))


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("m", [1, 80, 102, 700])
@pytest.mark.parametrize("pol", ["never_dense", "default", "coo"])
def test_short_chunks(S, dtype, m, pol):
    """Chunks of a few hundred elements and less, where a Pici message (the
    column words and offsets of a whole tile) is larger than a COO one: the
    message buffers hold either, and results and traces match the oracle."""
    P = 5
    policy = O.Policy.coo(adaptive=0) if pol == "coo" else POLICIES[pol]
    sends = [W.sparse_array(P * m, [0, P * m, P * m // 3, 1, P * m // 10][r], [41, r, m], dtype) for r in range(P)]
    log(f"short chunks m={m} dtype={dtype} policy={pol}")
    got, gtr = run_rs(S, sends, policy)
    exp, otr = O.ring_reduce_scatter(sends, policy)
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r])), f"rs rank {r}: {first_diff(got[r], bits(exp[r]))}"
    check_trace(gtr, otr)
    got, gtr = run_ar(S, sends, policy)
    exp, otr = O.ring_all_reduce(sends, policy)
    for r in range(P):
        assert np.array_equal(got[r], bits(exp[r])), f"ar rank {r}: {first_diff(got[r], bits(exp[r]))}"
    check_trace(gtr, otr)
