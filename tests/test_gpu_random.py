"""Seeded random parity cases: sizes from one element to several hundred
thousand (partial tiles and slices), densities from empty to full, both
dtypes, exact cancellations, and every producer and reduce form -- canonical
Pici, COO and sliced -- against the oracle, bit for bit."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import bits, first_diff, log, to_dev, to_host_bits

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

DENSITIES = [0.0, 0.001, 0.01, 0.1, 0.5, 1.0]


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


def case(i):
    rng = np.random.default_rng([91, i])
    dtype = [W.F32, W.BF16][int(rng.integers(2))]
    n = int([rng.integers(1, 5000), rng.integers(1, 70000), rng.integers(1, 400000)][int(rng.integers(3))])
    fa, fb = float(rng.choice(DENSITIES)), float(rng.choice(DENSITIES))
    a = W.sparse_array(n, int(round(fa * n)), [91, i, 0], dtype)
    b = W.sparse_array(n, int(round(fb * n)), [91, i, 1], dtype)
    if rng.integers(3) == 0:                       # b holds -a at a quarter of a's places: exact cancellations
        ia = np.flatnonzero(bits(a) != 0)
        if ia.size:
            pick = rng.choice(ia, size=max(1, ia.size // 4), replace=False)
            bits(b)[pick] = bits(a)[pick] ^ (0x8000 if dtype == W.BF16 else 0x80000000)
    return dtype, n, fa, fb, a, b


@pytest.mark.parametrize("i", range(24))
def test_random_case(S, i):
    dtype, n, fa, fb, a, b = case(i)
    dt = O.F32 if dtype == W.F32 else O.BF16
    log(f"random case {i}: n={n} {dtype} densities {fa} {fb}")
    ws = S.alloc_workspace(n, dt)
    tdt = torch.float32 if dt == O.F32 else torch.bfloat16
    P = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    C = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_COO)
    exp = O.reduce(O.Operand.array(a), O.Operand.array(b), n, dt)
    da, db = to_dev(a), to_dev(b)
    out = torch.empty(n, dtype=tdt, device="cuda")

    ma, mb, mo = S.alloc_stream(n, dt), S.alloc_stream(n, dt), S.alloc_stream(n, dt)
    S.spccl_compress(da, ma, ws)
    S.spccl_compress(db, mb, ws)
    for x, m in ((a, ma), (b, mb)):
        e = O.compress(x)[0]
        assert np.array_equal(m[:e.size].cpu().numpy(), e), "compress"
    e_sum = O.compress(exp)[0]
    for name, oa, ob in (("Pici+Pici", P(ma), P(mb)), ("dense+Pici", S.operand(da), P(mb)),
                         ("Pici+dense", P(ma), S.operand(db))):
        S.spccl_reduce(oa, ob, P(mo), n, dt, ws)
        assert np.array_equal(mo[:e_sum.size].cpu().numpy(), e_sum), name + " -> Pici"
        S.spccl_reduce(oa, ob, S.operand(out), n, dt, ws)
        got = to_host_bits(out)
        assert np.array_equal(got, bits(exp)), name + " -> dense: " + first_diff(got, bits(exp))

    ca, cb, co = (S.alloc_stream(n, dt, fmt=S.SPCCL_FMT_COO) for _ in range(3))
    S.spccl_compress_coo(da, ca, ws)
    S.spccl_compress_coo(db, cb, ws)
    e = O.compress_coo(a)[0]
    assert np.array_equal(ca[:e.size].cpu().numpy(), e), "compress_coo"
    e_sum = O.compress_coo(exp)[0]
    for name, oa, ob in (("COO+COO", C(ca), C(cb)), ("dense+COO", S.operand(da), C(cb)),
                         ("COO+dense", C(ca), S.operand(db))):
        S.spccl_reduce(oa, ob, C(co), n, dt, ws)
        assert np.array_equal(co[:e_sum.size].cpu().numpy(), e_sum), name + " -> COO"
        S.spccl_reduce(oa, ob, S.operand(out), n, dt, ws)
        got = to_host_bits(out)
        assert np.array_equal(got, bits(exp)), name + " -> dense: " + first_diff(got, bits(exp))

    sa, sb, so = S.alloc_sliced(n, dt), S.alloc_sliced(n, dt), S.alloc_sliced(n, dt)
    S.spccl_compress_sliced(da, sa, ws, 0.6)
    S.spccl_compress_sliced(db, sb, ws, 0.6)
    S.spccl_decompress_sliced(sa, out, ws)
    assert np.array_equal(to_host_bits(out), bits(a)), "sliced round trip"
    S.spccl_reduce_sliced(da, sb, so, ws, True, 0.6)
    S.spccl_decompress_sliced(so, out, ws)
    got = to_host_bits(out)
    assert np.array_equal(got, bits(exp)), "sliced reduce: " + first_diff(got, bits(exp))
    assert S.spccl_read_status(ws) == 0


@pytest.mark.parametrize("i", range(12))
def test_random_collectives(S, i):
    """Seeded random ring collectives: P from 1 to 8 (and 33, past the
    32-rank launch batching of the sliced ring), chunks from one element,
    mixed densities, random thresholds, node sizes and send formats; the
    canonical reduce-scatter, all-gather and all-reduce, and for Pici with the
    threshold rule the sliced ones, against the oracle's rings."""
    rng = np.random.default_rng([95, i])
    dtype = [W.F32, W.BF16][int(rng.integers(2))]
    dt = O.F32 if dtype == W.F32 else O.BF16
    P = 33 if i == 11 else int(rng.integers(1, 9))
    m = int([rng.integers(1, 300), rng.integers(1, 20000)][int(rng.integers(2))])
    n = P * m
    if rng.integers(4) == 0 and P <= 8:
        pol = O.Policy.coo(ranks_per_node=int(rng.integers(0, P + 1)))
    else:
        pol = O.Policy(intra_thresh=float(rng.choice([0.0, 0.6, 0.9])), inter_thresh=float(rng.choice([0.0, 0.5, 1.0])),
                       ag_thresh=float(rng.choice([0.0, 0.1, 0.9])), ranks_per_node=int(rng.integers(0, P + 1)),
                       adaptive=1 if P > 8 else int(rng.integers(0, 3)))
    fr = [float(rng.choice([0.0, 0.001, 0.01, 0.1, 0.3, 1.0])) for _ in range(P)]
    sends = [W.sparse_array(n, int(round(f * n)), [95, i, r], dtype) for r, f in enumerate(fr)]
    log(f"random collectives {i}: P={P} m={m} {dtype} {pol}")
    ds = [to_dev(x) for x in sends]
    tdt = torch.float32 if dt == O.F32 else torch.bfloat16
    same = lambda got, exp: all(np.array_equal(to_host_bits(g), bits(e)) for g, e in zip(got, exp))
    # format decisions never change values (Sec. IV-C), so the traces --
    # format, bytes, nonzeros and tracked sparsity of every send -- are
    # compared as well: a wrong decision, threshold or link rule shows there
    tup = lambda e: (e.step, e.rank, e.fmt, e.measured, e.bytes, e.nnz, e.sigma)
    scr = torch.empty(S.spccl_vr_scratch_bytes(P, m, dt), dtype=torch.uint8, device="cuda")
    rv = [torch.empty(m, dtype=tdt, device="cuda") for _ in range(P)]
    av = [torch.empty(n, dtype=tdt, device="cuda") for _ in range(P)]
    gtr = S.spccl_vr_reduce_scatter(ds, rv, scr, pol)
    exp, otr = O.ring_reduce_scatter(sends, pol)
    assert same(rv, exp), "reduce-scatter"
    assert gtr == [tup(e) for e in otr], "reduce-scatter trace"
    gtr = S.spccl_vr_all_reduce(ds, av, scr, pol)
    exp, otr = O.ring_all_reduce(sends, pol)
    assert same(av, exp), "all-reduce"
    assert gtr == [tup(e) for e in otr], "all-reduce trace"
    parts = [d[:m] for d in ds]
    gtr = S.spccl_vr_all_gather(parts, av, scr, pol)
    exp, otr = O.ring_all_gather([x[:m] for x in sends], pol.sparse_fmt)
    assert same(av, exp), "all-gather"
    assert gtr == [tup(e) for e in otr], "all-gather trace"
    if pol.sparse_fmt == O.FMT_PICI and pol.adaptive == 1:
        ssc = torch.empty(S.spccl_vr_sliced_scratch_bytes(P, n, dt), dtype=torch.uint8, device="cuda")
        gfm = S.spccl_vr_reduce_scatter_sliced(ds, rv, ssc, pol)
        exp, ofm = O.ring_reduce_scatter_sliced(sends, pol)
        assert same(rv, exp), "sliced reduce-scatter"
        assert np.array_equal(gfm, ofm), "sliced reduce-scatter formats"
        grs, gag = S.spccl_vr_all_reduce_sliced(ds, av, ssc, pol)
        exp, ors, oag = O.ring_all_reduce_sliced(sends, pol)
        assert same(av, exp), "sliced all-reduce"
        assert np.array_equal(grs, ors) and np.array_equal(gag, oag), "sliced all-reduce formats"
        ssg = torch.empty(S.spccl_vr_sliced_scratch_bytes(P, m, dt), dtype=torch.uint8, device="cuda")
        gfm = S.spccl_vr_all_gather_sliced(parts, av, ssg)
        exp, ofm = O.ring_all_gather_sliced([x[:m] for x in sends])
        assert same(av, exp), "sliced all-gather"
        assert np.array_equal(gfm, ofm), "sliced all-gather formats"
