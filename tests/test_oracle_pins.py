"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test checks the oracle against something other than itself: closed-form
sizes (Sec. III-B, Eq. 4), special cases that reduce to textbook routines
(all-zero, all-present = per-tile transpose, single nonzero), hand-derived
fixtures under tests/golden/, IEEE arithmetic as numpy performs it, the
fixed ring order, and hand-computed decision traces (Sec. IV-C, Eq. 7).
"""
import functools
import os

import numpy as np
import pytest

import oracle as O
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32_from_bits(bits):
    return np.array(bits, dtype=np.uint32).view(np.float32)


def parse_stream(stream, n, dtype):
    """Split a Pici message into B, I, A with plain numpy views."""
    h = O.header(stream)
    T = -(-n // 4096)
    B = stream[48:48 + 512 * T].view(np.uint64)
    I = stream[h["off_I"]:h["off_I"] + 4 * (T + 1)].view(np.uint32)
    A = stream[h["off_A"]:h["total_bytes"]].view(np.uint16 if dtype == O.BF16 else np.uint32)
    return h, B, I, A


# ---- sizes: Sec. III-B component sizes and Eq. 4 --------------------------------

def test_sizes_config1_closed_form():
    n, nnz = 1 << 20, 10486
    T = 256
    assert O.num_tiles(n) == T
    # |B| = 512 T bytes, |I| = 4 (T + 1), |A| = 4 nnz
    assert O.off_I(n) - 48 == 131072
    assert O.off_A(n) == 132160           # 48 + 131072 + 1028 = 132148 -> 16-byte boundary
    assert O.pici_bytes(n, O.F32, nnz) == 174104
    assert O.pici_bytes(n, O.F32, nnz) - 48 - 12 == 174044   # paper payload (no header, no pad)


@pytest.mark.parametrize("n", [4096, 1 << 20, 1 << 26])
@pytest.mark.parametrize("sigma_permille", [0, 500, 900, 990, 999, 1000])
def test_eq4_payload_formula_exact(n, sigma_permille):
    """Payload = 4n(1 - sigma + omega) with omega = 1/32 + 1/4096 + 1/n (n multiple of 4096)."""
    nnz = W.nnz_for(n, sigma_permille)
    payload = 512 * (n // 4096) + 4 * (n // 4096 + 1) + 4 * nnz
    from fractions import Fraction as Fr
    sigma = Fr(n - nnz, n)
    omega = Fr(1, 32) + Fr(1, 4096) + Fr(1, n)
    assert Fr(payload) == 4 * n * (1 - sigma + omega)
    # the paper's rounded omega = 0.0315 (3.125% bit vector + ~0.78% of it for I)
    assert abs(float(omega) - 0.0315) < 5e-5 + 1.0 / n
    assert Fr(4 * (n // 4096 + 1), 512 * (n // 4096)) - Fr(1, 128) == Fr(1, 128 * (n // 4096))
    # oracle agrees with the component sum
    assert O.pici_bytes(n, O.F32, nnz) == O.off_A(n) + 4 * nnz


@pytest.mark.parametrize("n,T", [(0, 0), (1, 1), (63, 1), (64, 1), (4095, 1), (4096, 1),
                                 (4097, 2), (8192, 2)])
def test_tile_count_and_empty(n, T):
    assert O.num_tiles(n) == T
    d = np.zeros(n, dtype=np.float32)
    s, nnz = O.compress(d)
    h, B, I, A = parse_stream(s, n, O.F32)
    assert nnz == 0 and B.size == 64 * T and not B.any()
    assert I.tolist() == [0] * (T + 1) and A.size == 0
    assert h["total_bytes"] == O.off_A(n) == s.size
    if n == 0:
        assert s.size == 64


def test_stream_bound_worst_case():
    for n in (0, 1, 4097, 1 << 20):
        for dt in (O.F32, O.BF16):
            assert O.stream_bound(n, dt) == O.off_A(n) + n * O.elem_size(dt)
            assert O.stream_bound(n, dt) >= O.dense_bytes(n, dt)


# ---- special cases ------------------------------------------------------------------

@pytest.mark.parametrize("n", [4096, 3 * 4096])
def test_all_present_is_per_tile_transpose(n):
    rng = np.random.default_rng(11)
    d = (rng.random(n, dtype=np.float32) + 0.5).astype(np.float32)   # all nonzero
    s, nnz = O.compress(d)
    h, B, I, A = parse_stream(s, n, O.F32)
    T = n // 4096
    assert nnz == n
    assert (B == np.uint64(0xFFFFFFFFFFFFFFFF)).all()
    assert I.tolist() == [4096 * t for t in range(T + 1)]
    expect = d.reshape(T, 64, 64).transpose(0, 2, 1).ravel()
    assert np.array_equal(A, expect.view(np.uint32))


@pytest.mark.parametrize("p", [0, 1, 63, 64, 4095, 4096, 4097, 8191, 12287])
def test_single_nonzero_closed_form(p):
    n = 3 * 4096
    d = np.zeros(n, dtype=np.float32)
    d[p] = -2.5
    s, nnz = O.compress(d)
    h, B, I, A = parse_stream(s, n, O.F32)
    word, bit = (p // 4096) * 64 + p % 64, (p % 4096) // 64
    expectB = np.zeros(64 * 3, dtype=np.uint64)
    expectB[word] = np.uint64(1) << np.uint64(bit)
    assert np.array_equal(B, expectB)
    assert I.tolist() == [0 if t <= p // 4096 else 1 for t in range(4)]
    assert A.tolist() == [int(np.float32(-2.5).view(np.uint32))]


def test_golden_two_tiles():
    path = os.path.join(GOLDEN, "two_tiles_f32.txt")
    n, xs, Bw, I_exp, A_exp, fields = None, [], {}, None, None, {}
    for line in open(path):
        t = line.split("#")[0].split()
        if not t:
            continue
        if t[0] == "n":
            n = int(t[1])
        elif t[0] == "x":
            xs.append((int(t[1]), int(t[2], 16)))
        elif t[0] == "B":
            Bw[int(t[1])] = int(t[2], 16)
        elif t[0] == "I":
            I_exp = [int(v) for v in t[1:]]
        elif t[0] == "A":
            A_exp = [int(v, 16) for v in t[1:]]
        elif t[0] in ("off_I", "off_A", "total"):
            fields[t[0]] = int(t[1])
    d = np.zeros(n, dtype=np.uint32)
    for i, bits in xs:
        d[i] = bits
    s, nnz = O.compress(d.view(np.float32))
    h, B, I, A = parse_stream(s, n, O.F32)
    expectB = np.zeros(B.size, dtype=np.uint64)
    for k, v in Bw.items():
        expectB[k] = v
    assert np.array_equal(B, expectB)
    assert I.tolist() == I_exp
    assert A.tolist() == A_exp
    assert (h["off_I"], h["off_A"], h["total_bytes"]) == (fields["off_I"], fields["off_A"], fields["total"])
    assert h["magic"] == 0x49434950 and h["format"] == O.FMT_PICI and h["nnz"] == len(A_exp)
    assert bytes(s[0:4]) == b"PICI"
    assert not s[h["off_I"] + 12:h["off_A"]].any()          # pad bytes are zero


# ---- round trip and invariants ---------------------------------------------------------

@pytest.mark.parametrize("n", [1, 63, 64, 65, 4095, 4096, 4097, 8192, 3 * 4096 + 77])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_round_trip_bitwise_with_specials(n, dtype):
    rng = np.random.default_rng(n)
    d = W.sparse_array(n, n // 3, [99, n], dtype)
    raw = d.view(np.uint16 if dtype == W.BF16 else np.uint32)
    # plant -0.0, subnormals and a NaN payload at random positions
    specials = [0x8000, 0x0001, 0x7FC1] if dtype == W.BF16 else [0x80000000, 0x00000001, 0x7FC00001]
    for v in specials:
        raw[rng.integers(0, n)] = v
    s, nnz = O.compress(d)
    dt = O.dtype_code(d)
    assert nnz == int(np.count_nonzero(raw))
    h, B, I, A = parse_stream(s, n, dt)
    # popcount(B) == nnz == I[T]; I non-decreasing with steps <= 4096
    pc = sum(bin(int(w)).count("1") for w in B)
    assert pc == nnz == I[-1] == h["nnz"]
    assert I[0] == 0 and (np.diff(I.astype(np.int64)) >= 0).all() and (np.diff(I.astype(np.int64)) <= 4096).all()
    back = O.decompress(s, n, dt)
    assert np.array_equal(back.view(raw.dtype), raw)
    assert O.validate(s, n, dt) == O.OK


def test_numpy_vectorised_cross_check():
    """An independent vectorised statement of the layout: pad to whole tiles,
    view as (T, 64 rows, 64 cols), transpose to column-major, mask."""
    for n in (4096 * 5, 4096 * 2 + 1000):
        d = W.sparse_array(n, n // 10, [98, n], W.F32)
        s, nnz = O.compress(d)
        h, B, I, A = parse_stream(s, n, O.F32)
        T = -(-n // 4096)
        pad = np.zeros(T * 4096, dtype=np.uint32)
        pad[:n] = d.view(np.uint32)
        cols = pad.reshape(T, 64, 64).transpose(0, 2, 1)          # [t, c, r]
        mask = cols != 0
        words = (mask.astype(np.uint64) << np.arange(64, dtype=np.uint64)).sum(axis=2, dtype=np.uint64)
        assert np.array_equal(B, words.ravel())
        assert np.array_equal(A, cols[mask])
        assert np.array_equal(I, np.concatenate([[0], np.cumsum(mask.sum(axis=(1, 2)))]))


# ---- reduction (+) -------------------------------------------------------------------------

def _golden_oplus():
    for line in open(os.path.join(GOLDEN, "oplus_cases.txt")):
        t = line.split("#")[0].split()
        if t:
            yield t[0], int(t[1], 16), int(t[2], 16), int(t[3], 16), int(t[4])


@pytest.mark.parametrize("case", list(_golden_oplus()))
def test_oplus_hand_cases(case):
    dt_name, a, b, expect, present = case
    dt = O.F32 if dt_name == "f32" else O.BF16
    assert O.oplus(a, b, dt) == expect
    assert O.oplus(b, a, dt) == expect                 # commutative
    # through the array reduction and a Pici output: presence follows the sum's bits
    npdt = np.uint32 if dt == O.F32 else np.uint16
    A = np.array([a], dtype=npdt)
    Bv = np.array([b], dtype=npdt)
    view = (lambda x: x.view(np.float32)) if dt == O.F32 else (lambda x: x)
    out = O.reduce(O.Operand.array(view(A)), O.Operand.array(view(Bv)), 1, dt)
    assert int(out.view(npdt)[0]) == expect
    s, nnz = O.reduce(O.Operand.array(view(A)), O.Operand.array(view(Bv)), 1, dt, O.STREAM, O.FMT_PICI)
    assert nnz == present


def test_oplus_fp32_matches_numpy_ieee_add():
    rng = np.random.default_rng(5)
    a = (rng.standard_normal(20000) * np.exp2(rng.integers(-140, 120, 20000))).astype(np.float32)
    b = (rng.standard_normal(20000) * np.exp2(rng.integers(-140, 120, 20000))).astype(np.float32)
    a[::7] = 0.0
    b[::5] = 0.0
    b[3::11] = -a[3::11]                                   # exact cancellations
    out = O.reduce(O.Operand.array(a), O.Operand.array(b), a.size, O.F32)
    with np.errstate(over="ignore"):
        s = a + b                                          # numpy: IEEE binary32, nearest-even
    expect = np.where(b.view(np.uint32) == 0, a, np.where(a.view(np.uint32) == 0, b, s))
    assert np.array_equal(out.view(np.uint32), expect.view(np.uint32))


def test_oplus_bf16_matches_fp32_then_round():
    """The oracle rounds the exact sum once (via double); adding in fp32 and
    rounding to bfloat16 afterwards must agree (24 >= 2*8 + 2 bits)."""
    rng = np.random.default_rng(6)
    f = lambda k: (rng.standard_normal(k) * np.exp2(rng.integers(-130, 120, k))).astype(np.float32)
    a = W._bf16_bits_from_f32(f(30000))
    b = W._bf16_bits_from_f32(f(30000))
    b[1::9] = a[1::9] ^ 0x8000                             # exact cancellations
    a[::13] = 0
    out = O.reduce(O.Operand.array(a), O.Operand.array(b), a.size, O.BF16)
    fa = (a.astype(np.uint32) << 16).view(np.float32)
    fb = (b.astype(np.uint32) << 16).view(np.float32)
    with np.errstate(over="ignore"):
        s = W._bf16_bits_from_f32(fa + fb)
    expect = np.where(b == 0, a, np.where(a == 0, b, s))
    finite = ((fa + fb) != np.inf) & ((fa + fb) != -np.inf)
    assert np.array_equal(out[finite], expect[finite])


def test_fill_in_count():
    n = 4096 * 2 + 300
    a = W.sparse_array(n, 900, [7, 0], W.F32)
    b = W.sparse_array(n, 700, [7, 1], W.F32)
    both = np.flatnonzero((a != 0) & (b != 0))
    b[both[:3]] = -a[both[:3]]                             # three exact cancellations
    s, nnz = O.reduce(O.Operand.array(a), O.Operand.array(b), n, O.F32, O.STREAM, O.FMT_PICI)
    union = int(np.count_nonzero((a.view(np.uint32) != 0) | (b.view(np.uint32) != 0)))
    assert nnz == union - 3
    # every operand-kind combination agrees bit for bit
    sa, _ = O.compress(a)
    sb, _ = O.compress(b)
    ref = O.reduce(O.Operand.array(a), O.Operand.array(b), n, O.F32)
    for x in (O.Operand.array(a), O.Operand.stream(sa), O.Operand.stream(O.encode_dense(a))):
        for y in (O.Operand.array(b), O.Operand.stream(sb)):
            assert np.array_equal(O.reduce(x, y, n, O.F32).view(np.uint32), ref.view(np.uint32))
            s2, nnz2 = O.reduce(x, y, n, O.F32, O.STREAM, O.FMT_PICI)
            assert np.array_equal(s2, s) and nnz2 == nnz


# ---- ring collectives --------------------------------------------------------------------------

def _np_oplus(x, y):
    with np.errstate(over="ignore"):
        s = x + y
    return np.where(y.view(np.uint32) == 0, x, np.where(x.view(np.uint32) == 0, y, s))


@pytest.mark.parametrize("P", [2, 3, 4, 8])
@pytest.mark.parametrize("adaptive", [0, 1, 2])
def test_reduce_scatter_fixed_ring_order(P, adaptive):
    m = 4096 + 100
    sends = [(W.sparse_array(P * m, P * m // 2, [8, P, r], W.F32) * np.float32(10.0 ** (r % 3)))
             for r in range(P)]
    recvs, trace = O.ring_reduce_scatter(sends, O.Policy(adaptive=adaptive))
    for j in range(P):
        order = [(j + k) % P for k in range(1, P)] + [j]
        expect = functools.reduce(_np_oplus, [sends[r][j * m:(j + 1) * m] for r in order])
        assert np.array_equal(recvs[j].view(np.uint32), expect.view(np.uint32))
    assert len(trace) == P * (P - 1)
    fmts = {e.fmt for e in trace}
    if adaptive == 0:
        assert fmts == {O.FMT_PICI}
    if adaptive == 2:
        assert fmts == {O.FMT_DENSE}


def test_ring_order_is_observable():
    """Sensitivity: a different fold order changes the bits, so the order test can fail."""
    x = [np.float32(1e8), np.float32(1.0), np.float32(-1e8)]
    arr = [np.array([v], dtype=np.float32) for v in x]
    fwd = functools.reduce(_np_oplus, arr)
    swapped = functools.reduce(_np_oplus, [arr[0], arr[2], arr[1]])
    assert fwd[0] != swapped[0]
    # and the oracle's RS output on P=3 follows the ring order (j+1, j+2, j)
    P, m = 3, 1
    sends = [np.array([x[(r - 1) % 3]] * 3, dtype=np.float32) for r in range(P)]
    recvs, _ = O.ring_reduce_scatter(sends, O.Policy(adaptive=0))
    for j in range(P):
        expect = functools.reduce(_np_oplus, [sends[r][j:j + 1] for r in ((j + 1) % 3, (j + 2) % 3, j)])
        assert recvs[j].view(np.uint32)[0] == expect.view(np.uint32)[0]


def test_formats_never_change_values():
    P, m = 4, 3000
    sends = [W.sparse_array(P * m, 400, [9, r], W.BF16) for r in range(P)]
    outs = [O.ring_all_reduce(sends, O.Policy(adaptive=a))[0] for a in (0, 1, 2)]
    for o in outs[1:]:
        for r in range(P):
            assert np.array_equal(o[r], outs[0][r])
    for r in range(1, P):
        assert np.array_equal(outs[0][r], outs[0][0])     # every rank's result is identical


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("m", [1, 80, 102, 700])
def test_formats_never_change_values_short_chunks(dtype, m):
    """Short chunks, where a Pici message is larger than a COO one: every
    policy and send format gives the same all-reduce."""
    P = 5
    sends = [W.sparse_array(P * m, [0, P * m, P * m // 3, 1, P * m // 10][r], [10, r, m], dtype) for r in range(P)]
    pols = [O.Policy(adaptive=a) for a in (0, 1, 2)] + [O.Policy.coo(), O.Policy.coo(adaptive=0)]
    outs = [O.ring_all_reduce(sends, p)[0] for p in pols]
    for o in outs[1:]:
        for r in range(P):
            assert np.array_equal(o[r], outs[0][r])
    red, _ = O.ring_reduce_scatter(sends, O.Policy(adaptive=2))
    assert np.array_equal(outs[0][0], np.concatenate(red))


def test_all_gather_is_concatenation():
    P, n = 5, 4096 + 7
    parts = [W.sparse_array(n, n // 4, [10, r], W.BF16) for r in range(P)]
    outs, trace = O.ring_all_gather(parts)
    cat = np.concatenate(parts)
    for o in outs:
        assert np.array_equal(o, cat)
    assert [e.fmt for e in trace] == [O.FMT_PICI] * P
    assert [e.nnz for e in trace] == [n // 4] * P


def _digit_sparsity_inputs(P, m, digits):
    """Rank r's support on chunk c is {i : decimal digit j of i is 0}, j = the
    position of r in chunk c's fold order (1..P), so the union of the first k
    contributions has exactly m (1 - 0.9^k) elements for k <= digits."""
    idx = np.arange(m)
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            j = (r - c) % P or P                           # 1..P in fold order
            d = (j - 1) % digits
            sup = (idx // 10 ** d) % 10 == 0
            x[c * m:(c + 1) * m][sup] = 1.0
        sends.append(x)
    return sends


def test_decision_trace_hand_computed():
    """sigma0 = 0.9, tau = 0.6, P = 8 (Sec. IV-C): measured sparsity after k
    contributions is exactly 0.9^k; steps 0-3 send Pici (0.9, 0.81, 0.729,
    0.6561), step 4 extrapolates 0.6561 * 0.9 = 0.59049 <= 0.6 and sends dense,
    steps 5-6 keep extrapolating through dense sends (0.531441, 0.4782969)."""
    P, m = 8, 10000
    sends = _digit_sparsity_inputs(P, m, 4)
    recvs, trace = O.ring_reduce_scatter(sends, O.Policy())
    dense_b = 48 + 4 * m
    offA = O.off_A(m)
    expect_sig = [0.9, 0.81, 0.729, 0.6561, 0.59049, 0.531441, 0.4782969]
    for e in trace:
        s = e.step
        assert e.sigma == pytest.approx(expect_sig[s], rel=1e-12)
        if s <= 3:
            nnz = m - 9 ** (s + 1) * 10 ** (4 - (s + 1))
            assert (e.fmt, e.measured, e.nnz, e.bytes) == (O.FMT_PICI, 1, nnz, offA + 4 * nnz)
        else:
            assert (e.fmt, e.measured, e.nnz, e.bytes) == (O.FMT_DENSE, 0, O.NNZ_UNKNOWN, dense_b)


def test_decision_threshold_inclusive_and_link_aware():
    """sigma0 = 0.75 exactly; step-1 estimate 0.75 * 0.75 = 0.5625 exactly.
    tau = 0.5625 sends dense (<= is inclusive), tau just below keeps Pici.
    With ranks_per_node = 4 the links 3->4 and 7->0 use inter_thresh 0.5, so
    those two ranks keep Pici at step 1 while intra links (0.6) go dense."""
    P, m = 8, 4096
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            off = ((r - c) % P) % 4                      # 4 disjoint quarter supports
            x[c * m:(c + 1) * m][off::4] = 1.0
        sends.append(x)
    _, tr = O.ring_reduce_scatter(sends, O.Policy(intra_thresh=0.5625, inter_thresh=0.5625))
    step1 = [e for e in tr if e.step == 1]
    assert all(e.sigma == 0.5625 and e.fmt == O.FMT_DENSE for e in step1)
    _, tr = O.ring_reduce_scatter(sends, O.Policy(intra_thresh=0.5624, inter_thresh=0.5624))
    assert all(e.fmt == O.FMT_PICI for e in tr if e.step == 1)
    _, tr = O.ring_reduce_scatter(sends, O.Policy(ranks_per_node=4))
    fm = {e.rank: e.fmt for e in tr if e.step == 1}
    assert [r for r in range(P) if fm[r] == O.FMT_PICI] == [3, 7]
    assert all(e.fmt == O.FMT_PICI and e.sigma == 0.75 for e in tr if e.step == 0)


def test_all_reduce_phase_aware_switch():
    """At the RS -> AG transition each rank gathers densely iff
    sigma_prev * sigma0 <= ag_thresh."""
    P, m = 4, 4096
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            x[c * m:(c + 1) * m][((r - c) % P)::8] = 2.0   # sigma0 = 7/8 on every chunk
        sends.append(x)
    outs, tr = O.ring_all_reduce(sends, O.Policy())
    ag = tr[P * (P - 1):]
    # RS: sigma after k contributions is 1 - k/8 (disjoint supports): 0.875, 0.75, 0.625
    # tracked after the last send (step 2, Pici since 0.875*0.75=0.65625 > 0.6): 0.625
    # transition estimate 0.625 * 0.875 = 0.546875 > 0.1 -> Pici all-gather
    assert [e.fmt for e in tr[:P * (P - 1)]] == [O.FMT_PICI] * (P * (P - 1))
    assert all(e.fmt == O.FMT_PICI and e.sigma == 0.546875 and e.step == P - 1 for e in ag)
    assert all(e.nnz == m // 2 for e in ag)               # 4 of 8 residues present after the fold
    outs2, tr2 = O.ring_all_reduce(sends, O.Policy(ag_thresh=0.546875))
    assert all(e.fmt == O.FMT_DENSE and e.nnz == O.NNZ_UNKNOWN for e in tr2[P * (P - 1):])
    for r in range(P):
        assert np.array_equal(outs[r], outs2[r]) and np.array_equal(outs[r], outs[0])


def test_eq7_expected_fill_in_statistical():
    """Independent uniform supports: sparsity after k contributions ~ sigma0^k (Eq. 7)."""
    P, m = 8, 50000
    sends = [W.sparse_array(P * m, P * m // 10, [12, r], W.F32) for r in range(P)]
    _, tr = O.ring_reduce_scatter(sends, O.Policy(adaptive=0))
    for e in tr:
        k = e.step + 1
        p = 0.9 ** k
        sd = np.sqrt(p * (1 - p) / m)
        assert abs(e.sigma - p) < 4 * sd + 1e-3


# ---- validation -------------------------------------------------------------------------------

def test_validate_rejects_corruption():
    n = 4096 + 5
    d = W.sparse_array(n, 50, [13], W.F32)
    s, nnz = O.compress(d)
    assert O.validate(s, n, O.F32) == O.OK
    bad = s.copy(); bad[0] ^= 1
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM              # magic
    assert O.validate(s, n + 1, O.F32) == O.ERR_CORRUPT_STREAM            # n mismatch
    assert O.validate(s, n, O.BF16) == O.ERR_CORRUPT_STREAM               # dtype mismatch
    assert O.validate(s[:-1], n, O.F32) == O.ERR_CORRUPT_STREAM           # truncated
    bad = s.copy(); bad[48] ^= 0x10                                       # B disagrees with I
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM
    with pytest.raises(O.OracleError):
        O.decompress(bad, n, O.F32)


# bf16 sums whose correctly rounded results were worked out by hand from the
# bit patterns (8 significant bits; subnormal spacing 2^-133; overflow to
# infinity), each a case a plausible rounding mistake gets wrong
BF16_SUMS = [
    (0x3F80, 0x3B80, 0x3F80),   # 1 + 2^-8, halfway: to even, 1
    (0x3F81, 0x3B80, 0x3F82),   # (1 + 2^-7) + 2^-8, halfway: to even, 1 + 2^-6
    (0xBF80, 0xBB80, 0xBF80),   # the negative tie
    (0x4380, 0x3F80, 0x4380),   # 256 + 1, halfway: 256
    (0x4381, 0x3F80, 0x4382),   # 258 + 1, halfway: 260
    (0x4B80, 0x3F80, 0x4B80),   # 2^24 + 1: 2^24
    (0x0001, 0x0001, 0x0002),   # subnormals add exactly
    (0x007F, 0x0001, 0x0080),   # into the smallest normal
    (0x0080, 0x8001, 0x007F),   # back into the subnormals
    (0x0001, 0x8001, 0x0000),   # exact cancellation: absent
    (0x7F7F, 0x7F7F, 0x7F80),   # overflow: +inf
    (0x7F7F, 0x7B00, 0x7F80),   # largest + half its unit, halfway: to even, +inf
    (0x7F7F, 0x7A80, 0x7F7F),   # largest + a quarter unit: unchanged
    (0xFF7F, 0xFB00, 0xFF80),   # -inf
    (0x8000, 0x8000, 0x8000),   # -0 + -0 = -0
    (0x8000, 0x3F80, 0x3F80),   # -0 + 1 = 1
    (0x8000, 0x0000, 0x8000),   # absent operand: -0 kept
    (0x0000, 0x8000, 0x8000),
]


@pytest.mark.parametrize("a,b,want", BF16_SUMS)
def test_oracle_bf16_sum_hand_values(a, b, want):
    assert O.oplus(a, b, O.BF16) == want
    assert O.oplus(b, a, O.BF16) == want
