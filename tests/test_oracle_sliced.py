"""Pins of the oracle's sliced streams (one message per slice of 16384
elements, block-local prefix sums; Sec. III-B phase 2 and Sec. V-B) against
what the format and numpy fix independently: round trips, per-slot headers
and closed-form sizes, a hand-computed format decision at the threshold, and
the reduction checked against numpy's IEEE add."""
import numpy as np
import pytest

import oracle as O
import workloads as W

S = O.SLICE_ELEMS
SIZES = [1, 4097, S, S + 1, 3 * S + 777]


def _bits(x):
    return x.view(np.uint32) if x.dtype == np.float32 else x.view(np.uint16)


def _with_specials(x, seed):
    raw = _bits(x).copy()
    rng = np.random.default_rng(seed)
    sp = [0x8000, 0x0001] if x.dtype == np.uint16 else [0x80000000, 0x00000001]
    for v in sp:
        raw[rng.integers(0, x.size)] = v
    return raw.view(x.dtype)


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("thresh", [-1.0, 0.6, 1.0])
def test_round_trip_and_slot_headers(n, dtype, thresh):
    dt = O.F32 if dtype == W.F32 else O.BF16
    x = _with_specials(W.sparse_array(n, max(1, n // 50), [40, n], dtype), n)
    stream = O.encode_sliced(x, thresh)
    assert stream.size == O.slice_count(n) * O.slice_bytes(dt)
    assert O.slice_count(n) == -(-n // S)
    assert np.array_equal(_bits(O.decode_sliced(stream, n, dt)), _bits(x))
    for q, msg in enumerate(O.slot_messages(stream, n, dt)):
        part = _bits(x[q * S:(q + 1) * S])
        m, nnz = part.size, int(np.count_nonzero(part))
        h = O.header(msg)
        assert h["n"] == m
        dense = (m - nnz) / m <= thresh
        if dense:
            assert h["format"] == O.FMT_DENSE and msg.size == 48 + m * O.elem_size(dt)
            assert np.array_equal(msg[48:].view(part.dtype), part)
        else:
            assert h["format"] == O.FMT_PICI and h["nnz"] == nnz
            assert msg.size == O.pici_bytes(m, dt, nnz)              # closed-form size


def test_threshold_decision_hand_computed():
    """A full slice with 6554 nonzeros has sparsity 9830/16384 = 0.5999755859375,
    <= 0.6, so it goes dense; with 6553 nonzeros, 9831/16384 = 0.60003662109375,
    it stays Pici.  The test is inclusive."""
    for nnz, fmt in ((6554, O.FMT_DENSE), (6553, O.FMT_PICI)):
        x = W.sparse_array(S, nnz, [41, nnz], W.F32)
        msg = O.slot_messages(O.encode_sliced(x, 0.6), S, O.F32)[0]
        assert O.header(msg)["format"] == fmt
    x = W.sparse_array(S, 6554, [41, 6554], W.F32)
    assert O.header(O.slot_messages(O.encode_sliced(x, 0.5999755859375), S, O.F32)[0])["format"] == O.FMT_DENSE
    assert O.header(O.slot_messages(O.encode_sliced(x, 0.5999755859374), S, O.F32)[0])["format"] == O.FMT_PICI


def test_slots_are_independent_messages():
    """Slice q is its own message: changing elements of one slice changes that
    slot only, and a Pici slot decodes alone to its slice."""
    n = 3 * S + 100
    x = W.sparse_array(n, 800, [42], W.F32)
    a = O.slot_messages(O.encode_sliced(x), n, O.F32)
    y = x.copy()
    y[S + 5] = np.float32(3.0)
    b = O.slot_messages(O.encode_sliced(y), n, O.F32)
    assert [np.array_equal(p, q) for p, q in zip(a, b)] == [True, False, True, True]
    for q, msg in enumerate(a):
        m = O.slice_len(n, q)
        assert np.array_equal(O.decompress(msg, m, O.F32).view(np.uint32), x[q * S:q * S + m].view(np.uint32))


def _np_oplus_f32(x, y):
    with np.errstate(over="ignore"):
        s = x + y
    return np.where(y.view(np.uint32) == 0, x, np.where(x.view(np.uint32) == 0, y, s))


@pytest.mark.parametrize("n", [4097, 2 * S + 333])
@pytest.mark.parametrize("thresh", [-1.0, 0.6, 1.0])
def test_reduce_sliced_matches_numpy(n, thresh):
    a = W.sparse_array(n, n // 3, [43, 0], W.F32)
    b = W.sparse_array(n, n // 40, [43, 1], W.F32)
    hit = np.flatnonzero((a != 0) & (b != 0))
    b[hit[:5]] = -a[hit[:5]]                                 # exact cancellations drop
    sb = O.encode_sliced(b, thresh)
    want = _np_oplus_f32(a, b)
    got = O.reduce_sliced(a, sb, n, O.F32, out_sliced=False)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    so = O.reduce_sliced(a, sb, n, O.F32, out_sliced=True, dense_thresh=thresh)
    assert np.array_equal(O.decode_sliced(so, n, O.F32).view(np.uint32), want.view(np.uint32))
    for q, msg in enumerate(O.slot_messages(so, n, O.F32)):
        part = want[q * S:(q + 1) * S].view(np.uint32)
        m, nnz = part.size, int(np.count_nonzero(part))
        assert O.header(msg)["format"] == (O.FMT_DENSE if (m - nnz) / m <= thresh else O.FMT_PICI)


# ---- ring reduce-scatter over sliced streams, per-slice decisions --------------------------------

@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("adaptive", [0, 1, 2])
def test_sliced_ring_values_equal_the_plain_ring(P, adaptive):
    m = 2 * O.SLICE_ELEMS + 777
    sends = [W.sparse_array(P * m, P * m // 8, [80, P, r], W.BF16) for r in range(P)]
    got, fm = O.ring_reduce_scatter_sliced(sends, O.Policy(adaptive=adaptive))
    exp, _ = O.ring_reduce_scatter(sends, O.Policy(adaptive=adaptive))
    for r in range(P):
        assert np.array_equal(got[r], exp[r])
    if P > 1 and adaptive != 1:
        assert (fm == (O.FMT_DENSE if adaptive == 2 else O.FMT_PICI)).all()


def test_sliced_ring_decides_per_slice():
    """Chunk = one full slice + one slice of 10,000 elements.  Slice 0: rank
    j-th in the fold order holds the residue j-1 mod 100 (disjoint), so its
    sparsity after k contributions is 1 - k/100 and never reaches 0.6.  Slice
    1: the digit supports of the canonical pin (sparsity 0.9^k exactly), so
    with tau = 0.6 it is sent as Pici at steps 0-3 and dense at steps 4-6
    (0.59049 after extrapolation).  Each slice follows its own tracker."""
    P, L0, L1 = 8, O.SLICE_ELEMS, 10000
    m = L0 + L1
    idx0, idx1 = np.arange(L0), np.arange(L1)
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            j = (r - c) % P or P
            base = c * m
            x[base:base + L0][idx0 % 100 == (j - 1)] = 1.0
            x[base + L0:base + m][(idx1 // 10 ** ((j - 1) % 4)) % 10 == 0] = 1.0
        sends.append(x)
    got, fm = O.ring_reduce_scatter_sliced(sends, O.Policy())
    assert (fm[:, :, 0] == O.FMT_PICI).all()
    for r in range(P):
        assert fm[:, r, 1].tolist() == [1, 1, 1, 1, 0, 0, 0]
    exp, _ = O.ring_reduce_scatter(sends, O.Policy(adaptive=0))
    for r in range(P):
        assert np.array_equal(got[r], exp[r])


@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_sliced_all_gather_equals_the_plain_all_gather(P, dtype):
    """Formats never change values: the sliced all-gather delivers every
    part exactly as the plain ring all-gather does, and every slice is Pici
    (a standalone all-gather does not densify, Sec. IV-C)."""
    n = 2 * S + 555
    parts = [W.sparse_array(n, [40, 3000, n // 3][r % 3], [91, P, r], dtype) for r in range(P)]
    got, fm = O.ring_all_gather_sliced(parts)
    exp, _ = O.ring_all_gather(parts)
    for r in range(P):
        assert np.array_equal(_bits(got[r]), _bits(exp[r])), r
        for q in range(P):
            assert np.array_equal(_bits(got[r][q * n:(q + 1) * n]), _bits(parts[q])), (r, q)
    assert fm.shape == (P, O.slice_count(n)) and (fm == O.FMT_PICI).all()


@pytest.mark.parametrize("P", [1, 2, 3, 8])
@pytest.mark.parametrize("adaptive", [0, 1, 2])
def test_sliced_all_reduce_values_equal_the_plain_ring(P, adaptive):
    """Every rank ends with the full left-fold (Sec. IV-B): the plain ring
    all-reduce's values on every rank, whatever the formats."""
    m = S + 4097
    sends = [W.sparse_array(P * m, int(0.05 * P * m), [92, P, r]) for r in range(P)]
    pol = O.Policy(adaptive=adaptive)
    got, frs, fag = O.ring_all_reduce_sliced(sends, pol)
    exp, _ = O.ring_all_reduce(sends, pol)
    for r in range(P):
        assert np.array_equal(_bits(got[r]), _bits(exp[r])), r
        assert np.array_equal(_bits(got[r]), _bits(got[0])), r
    if P > 1:
        assert frs.shape == (P - 1, P, O.slice_count(m)) and fag.shape == (P, O.slice_count(m))
        if adaptive == 0:
            assert (frs == O.FMT_PICI).all() and (fag == O.FMT_PICI).all()
        if adaptive == 2:
            assert (frs == O.FMT_DENSE).all() and (fag == O.FMT_DENSE).all()


def test_sliced_all_reduce_transition_per_slice():
    """Hand-computed decisions (Sec. IV-C, per slice).  Each chunk has two
    slices.  Slice 0: every rank holds 1 in 100 of it at its own residue, so
    its sparsity stays near 0.99 - 0.93 and it is Pici everywhere; at the
    transition est = sigma_prev * sigma0 ~ 0.92 > 0.1: Pici.  Slice 1: 30%
    nonzeros (sigma0 = 0.7 > 0.6: Pici at step 0), then est = 0.7^(k+1) <=
    0.6: dense at steps 1-6 (tracking the estimate), and at the transition
    est = 0.7^7 * 0.7 = 0.0576 <= 0.1: dense."""
    P, L0, L1 = 8, O.SLICE_ELEMS, 10000
    m = L0 + L1
    idx0, idx1 = np.arange(L0), np.arange(L1)
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            j = (r - c) % P or P
            base = c * m
            x[base:base + L0][idx0 % 100 == (j - 1)] = 1.0
            x[base + L0:base + m][(idx1 + 7 * j) % 10 < 3] = 1.0
        sends.append(x)
    got, frs, fag = O.ring_all_reduce_sliced(sends, O.Policy())
    assert (frs[:, :, 0] == O.FMT_PICI).all()
    for r in range(P):
        assert frs[:, r, 1].tolist() == [1, 0, 0, 0, 0, 0, 0]
    assert fag[:, 0].tolist() == [O.FMT_PICI] * P
    assert fag[:, 1].tolist() == [O.FMT_DENSE] * P
    exp, _ = O.ring_all_reduce(sends, O.Policy(adaptive=0))
    for r in range(P):
        assert np.array_equal(got[r], exp[r])
