"""Pins of the oracle's COO format (Sec. II-B: the one-dimensional variant,
one flat 32-bit index per nonzero plus its value; Sec. IV-D: COO in the same
collectives, with its own thresholds).  CPU only.

What fixes the oracle here, independently of its own code:
  * numpy's flatnonzero is the definition of the index list (J) and fancy
    indexing of the values (V);
  * the paper's size statements: 32-bit indices and 32-bit values, COO as
    large as dense at 50% sparsity, COO smaller than a format with m bytes of
    sparsity-independent metadata iff 4 nnz < m, BV (1 bit per element) ahead
    of COO below 96.875% sparsity;
  * decision traces worked out by hand with the COO thresholds 0.8 / 0.7 / 0.5.
"""
import numpy as np
import pytest

import oracle as O
import workloads as W


def _coo_parts(msg):
    """(J, V bytes, header) of a COO message, parsed by hand from the layout."""
    h = O.header(msg)
    nnz = h["nnz"]
    J = msg[48:48 + 4 * nnz].view(np.uint32)
    V = msg[h["off_A"]:h["total_bytes"]]
    return J, V, h


def _bits(a):
    return a.view(np.uint16) if a.dtype == np.uint16 else a.view(np.uint32)


@pytest.mark.parametrize("n", [1, 63, 4096, 4097, 3 * 4096 + 77])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_coo_is_flatnonzero(n, dtype):
    x = W.sparse_array(n, max(1, n // 7), [21, n], dtype)
    msg, nnz = O.compress_coo(x)
    J, V, h = _coo_parts(msg)
    b = _bits(x)
    assert h["format"] == O.FMT_COO and h["n"] == n and h["nnz"] == nnz
    assert np.array_equal(J, np.flatnonzero(b != 0).astype(np.uint32))
    s = 2 if dtype == W.BF16 else 4
    assert np.array_equal(V.view(b.dtype), b[J])
    assert h["off_I"] == 48 and h["off_A"] == (48 + 4 * nnz + 15) // 16 * 16
    assert h["total_bytes"] == msg.size == O.coo_bytes(O.dtype_code(x), nnz) == h["off_A"] + s * nnz
    assert np.all(msg[48 + 4 * nnz:h["off_A"]] == 0)                   # pad bytes are zero


@pytest.mark.parametrize("n", [1, 64, 4097, 8192])
@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_coo_round_trip_bitwise_with_specials(n, dtype):
    x = W.sparse_array(n, n // 3, [22, n], dtype)
    b = _bits(x)
    special = [0x80000000, 0x00000001, 0x7FC00001] if dtype == W.F32 else [0x8000, 0x0001, 0x7FC1]
    for k, v in enumerate(special):
        if k < n:
            b[(k * 997) % n] = v                                      # -0.0, a subnormal, a NaN payload
    msg, nnz = O.compress_coo(x)
    assert nnz == int(np.count_nonzero(b))
    back = O.decompress(msg, n, O.dtype_code(x))
    assert np.array_equal(_bits(back), b)


def test_coo_edge_cases():
    z = W.empty(5000, W.F32)
    msg, nnz = O.compress_coo(z)                                        # sigma = 1
    assert nnz == 0 and msg.size == 48 and O.header(msg)["off_A"] == 48
    assert np.array_equal(O.decompress(msg, 5000, O.F32), z)
    msg, nnz = O.compress_coo(np.zeros(0, dtype=np.float32))            # n = 0
    assert nnz == 0 and msg.size == 48
    full = np.arange(1, 4098, dtype=np.float32)                         # sigma = 0: J = 0..n-1
    J, V, _ = _coo_parts(O.compress_coo(full)[0])
    assert np.array_equal(J, np.arange(4097, dtype=np.uint32))
    assert np.array_equal(V.view(np.float32), full)
    for p in (0, 1, 4095, 4096, 12345):                                 # one nonzero at p
        x = np.zeros(12346, dtype=np.float32)
        x[p] = -3.5
        J, V, h = _coo_parts(O.compress_coo(x)[0])
        assert J.tolist() == [p] and V.view(np.float32).tolist() == [-3.5] and h["total_bytes"] == 64 + 4


def test_coo_equals_dense_at_half_sparsity():
    """Sec. II-B: at 50% sparsity COO needs as much space as dense (32-bit
    index and value per nonzero vs 32 bits per element)."""
    n = 1 << 16
    x = W.sparse_array(n, n // 2, [23], W.F32)
    msg, nnz = O.compress_coo(x)
    assert nnz == n // 2
    idx_and_vals = 4 * nnz + 4 * nnz
    assert idx_and_vals == 4 * n == O.dense_bytes(n, O.F32) - 48
    pad = O.header(msg)["off_A"] - 48 - 4 * nnz
    assert msg.size == 48 + pad + idx_and_vals


def test_coo_versus_sparsity_independent_metadata():
    """Sec. II-B: COO uses less space than a format with m bytes of metadata
    iff 4 nnz < m.  Pici's metadata for T tiles is m = 512 T + 4 (T + 1)
    (Sec. III-B), so with n = 8 tiles the sizes tie at nnz = 129 T + 1."""
    T = 8
    n = 4096 * T
    m_pici = 512 * T + 4 * (T + 1)
    tie = 129 * T + 1
    assert 4 * tie == m_pici
    for nnz, cmp in ((tie - 1, -1), (tie, 0), (tie + 1, 1)):
        x = W.sparse_array(n, nnz, [24, nnz], W.F32)
        coo, k1 = O.compress_coo(x)
        pici, k2 = O.compress(x)
        assert k1 == k2 == nnz
        coo_payload = 4 * nnz + 4 * nnz                                   # J + V
        pici_payload = (O.off_I(n) - 48) + 4 * (T + 1) + 4 * nnz          # B + I + A
        assert coo.size == O.header(coo)["off_A"] + 4 * nnz
        assert pici.size == O.off_A(n) + 4 * nnz
        assert np.sign(coo_payload - pici_payload) == cmp


def test_bv_ahead_of_coo_below_96875_permille():
    """Sec. II-B: a plain bit vector (1 bit per element) is smaller than COO's
    indices below 96.875% sparsity; Pici's B is exactly that bit vector, so
    |B| == |J| at nnz = n / 32."""
    n = 4096 * 4
    nnz = n // 32
    assert 1 - nnz / n == 0.96875
    x = W.sparse_array(n, nnz, [25], W.F32)
    coo, _ = O.compress_coo(x)
    assert O.off_I(n) - 48 == 4 * O.header(coo)["nnz"]


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_coo_operands_reduce_like_any_format(dtype):
    """Formats carry values, they do not change them: a (+) b is the same
    whatever the operands' and output's formats."""
    n = 2 * 4096 + 999
    dt = O.BF16 if dtype == W.BF16 else O.F32
    a = W.sparse_array(n, n // 9, [26, 0], dtype)
    b = W.sparse_array(n, n // 9, [26, 1], dtype)
    both = np.flatnonzero(_bits(a) != 0)[:40]
    _bits(b)[both[:20]] = _bits(a)[both[:20]] ^ (0x80000000 if dt == O.F32 else 0x8000)   # exact cancellations
    _bits(b)[both[20:]] = _bits(a)[both[20:]]                                            # overlaps that add
    ref = O.reduce(O.Operand.array(a), O.Operand.array(b), n, dt)
    ops_a = [O.Operand.array(a), O.Operand.stream(O.compress(a)[0]), O.Operand.stream(O.compress_coo(a)[0])]
    ops_b = [O.Operand.array(b), O.Operand.stream(O.compress(b)[0]), O.Operand.stream(O.compress_coo(b)[0])]
    for oa in ops_a:
        for ob in ops_b:
            got = O.reduce(oa, ob, n, dt)
            assert np.array_equal(_bits(got), _bits(ref))
            assert np.count_nonzero(_bits(got)[both[:20]]) == 0
            msg, nnz = O.reduce(oa, ob, n, dt, O.STREAM, O.FMT_COO)
            exp, enz = O.compress_coo(ref)
            assert nnz == enz and np.array_equal(msg, exp)


def test_coo_reduce_cancellation_drops_the_index():
    a = np.zeros(100, dtype=np.float32)
    b = np.zeros(100, dtype=np.float32)
    a[[3, 10, 50]] = [1.5, 2.0, -4.0]
    b[[10, 50, 99]] = [-2.0, 1.0, 7.0]
    msg, nnz = O.reduce(O.Operand.stream(O.compress_coo(a)[0]), O.Operand.stream(O.compress_coo(b)[0]),
                        100, O.F32, O.STREAM, O.FMT_COO)
    J, V, _ = _coo_parts(msg)
    assert J.tolist() == [3, 50, 99] and V.view(np.float32).tolist() == [1.5, -3.0, 7.0]


def test_coo_validate_rejects_corruption():
    n = 5000
    x = W.sparse_array(n, 40, [27], W.F32)
    s, nnz = O.compress_coo(x)
    assert O.validate(s, n, O.F32) == O.OK
    bad = s.copy(); bad[48:52] = s[52:56]                                    # J[0] == J[1]: not increasing
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM
    bad = s.copy(); bad[48 + 4 * (nnz - 1):48 + 4 * nnz] = np.array([n], np.uint32).view(np.uint8)
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM                 # index past the array
    bad = s.copy(); bad[32] ^= 16                                            # off_V moved
    assert O.validate(bad, n, O.F32) == O.ERR_CORRUPT_STREAM
    assert O.validate(s[:-1], n, O.F32) == O.ERR_CORRUPT_STREAM              # truncated
    with pytest.raises(O.OracleError):
        O.decompress(s[:-1], n, O.F32)


# ---- COO in the collectives (Sec. IV-D) -------------------------------------------------------

def test_coo_collectives_give_the_same_values():
    P, m = 4, 3000
    sends = [W.sparse_array(P * m, 500, [28, r], W.F32) for r in range(P)]
    ref, _ = O.ring_all_reduce(sends, O.Policy(adaptive=0))
    for pol in (O.Policy.coo(adaptive=0), O.Policy.coo(), O.Policy.coo(adaptive=2)):
        outs, tr = O.ring_all_reduce(sends, pol)
        for r in range(P):
            assert np.array_equal(outs[r].view(np.uint32), ref[r].view(np.uint32))
        assert {e.fmt for e in tr} <= {O.FMT_DENSE, O.FMT_COO}
    outs, tr = O.ring_all_gather(sends, O.FMT_COO)
    cat = np.concatenate(sends)
    assert all(np.array_equal(o, cat) for o in outs)
    assert [e.fmt for e in tr] == [O.FMT_COO] * P
    assert [e.bytes for e in tr] == [O.coo_bytes(O.F32, 500)] * P


def _digit_sparsity_inputs(P, m, digits):
    """Rank r's support on chunk c: {i : decimal digit j of i is 0}, j the
    position of r in chunk c's fold order, so k contributions leave exactly
    m 0.9^k zeros (k <= digits)."""
    idx = np.arange(m)
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            j = (r - c) % P or P
            sup = (idx // 10 ** ((j - 1) % digits)) % 10 == 0
            x[c * m:(c + 1) * m][sup] = 1.0
        sends.append(x)
    return sends


def test_coo_decision_trace_hand_computed():
    """COO thresholds (Sec. IV-D): intra 0.8.  sigma0 = 0.9 > 0.8 sends COO;
    step 1 estimates 0.81 > 0.8, reduces into COO and measures 0.81; step 2
    estimates 0.729 <= 0.8 and goes dense, and steps 3-6 extrapolate through
    dense sends (0.6561, 0.59049, 0.531441, 0.4782969).  Pici's 0.6 on the
    same inputs keeps four sparse steps."""
    P, m = 8, 10000
    sends = _digit_sparsity_inputs(P, m, 4)
    _, tr = O.ring_reduce_scatter(sends, O.Policy.coo())
    sig = [0.9, 0.81, 0.729, 0.6561, 0.59049, 0.531441, 0.4782969]
    for e in tr:
        assert e.sigma == pytest.approx(sig[e.step], rel=1e-12)
        if e.step <= 1:
            nnz = m - 9 ** (e.step + 1) * 10 ** (4 - (e.step + 1))
            assert (e.fmt, e.measured, e.nnz, e.bytes) == (O.FMT_COO, 1, nnz, O.coo_bytes(O.F32, nnz))
        else:
            assert (e.fmt, e.measured, e.nnz, e.bytes) == (O.FMT_DENSE, 0, O.NNZ_UNKNOWN, 48 + 4 * m)
    _, tr = O.ring_reduce_scatter(sends, O.Policy())
    assert [e.fmt for e in tr if e.rank == 0] == [O.FMT_PICI] * 4 + [O.FMT_DENSE] * 3


def test_coo_all_reduce_transition_and_inter_links():
    """sigma0 = 7/8 on every chunk (disjoint residues mod 8).  COO RS: step 0
    COO (0.875 > 0.8); step 1 estimate 0.765625 <= 0.8 -> dense; step 2
    estimate 0.669921875 -> dense.  Transition estimate 0.586181640625 > 0.5
    -> COO all-gather; with ag_thresh at exactly that value -> dense.  Links
    3->4 and 7->0 are inter-node with ranks_per_node = 4: tau 0.7 keeps COO
    at step 1 there (0.765625 > 0.7)."""
    P, m = 4, 4096
    sends = []
    for r in range(P):
        x = np.zeros(P * m, dtype=np.float32)
        for c in range(P):
            x[c * m:(c + 1) * m][((r - c) % P)::8] = 2.0
        sends.append(x)
    outs, tr = O.ring_all_reduce(sends, O.Policy.coo())
    rs, ag = tr[:P * (P - 1)], tr[P * (P - 1):]
    assert [e.fmt for e in rs] == [O.FMT_COO] * P + [O.FMT_DENSE] * (2 * P)
    assert [e.sigma for e in rs[P:2 * P]] == [0.765625] * P
    assert [e.sigma for e in rs[2 * P:]] == [0.669921875] * P
    assert all(e.fmt == O.FMT_COO and e.sigma == 0.586181640625 and e.nnz == m // 2 for e in ag)
    outs2, tr2 = O.ring_all_reduce(sends, O.Policy.coo(ag_thresh=0.586181640625))
    assert all(e.fmt == O.FMT_DENSE for e in tr2[P * (P - 1):])
    for r in range(P):
        assert np.array_equal(outs[r], outs2[r]) and np.array_equal(outs[r], outs[0])
    P8 = 8
    sends8 = []
    for r in range(P8):
        x = np.zeros(P8 * m, dtype=np.float32)
        for c in range(P8):
            x[c * m:(c + 1) * m][((r - c) % P8)::8] = 2.0
        sends8.append(x)
    _, tr = O.ring_reduce_scatter(sends8, O.Policy.coo(ranks_per_node=4))
    fm = {e.rank: e.fmt for e in tr if e.step == 1}
    assert [r for r in range(P8) if fm[r] == O.FMT_COO] == [3, 7]
