"""Pici (+) Pici -> Pici (Sec. IV-B, fill-in as in Sec. I) against the
oracle byte for byte, on inputs built so that every staging path of the
first pass runs: partitions whose values fit the stage in one round, tiles
that fit it one at a time (the output buffer is written out between tiles),
tiles too dense for it (column groups), mixes of these inside one partition
and a ragged last partition; with exact cancellations and with zero values
stored in A (they read as absent); fp32 and bf16, both workspace sizes."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import assert_bytes_equal, bits, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


# per-tile densities, cycled: sparse tiles (a partition stages at once),
# ~0.1 tiles (one tile at a time, the buffer fills), dense tiles (groups)
PATTERNS = {
    "sparse": [0.002, 0.01, 0.0, 0.03],
    "tilewise": [0.1, 0.12, 0.09, 0.11],
    "dense": [0.6, 1.0, 0.3, 0.8],
    "mixed": [0.01, 0.1, 0.7, 0.0, 0.12, 1.0, 0.002, 0.2, 0.05, 0.3, 0.11, 0.5],
}


def tiled(n, pattern, seed, dtype):
    """n elements; tile t has density pattern[t % len(pattern)]."""
    out = W.empty(n, dtype)
    for t in range(-(-n // 4096)):
        lo, hi = 4096 * t, min(n, 4096 * (t + 1))
        out[lo:hi] = W.sparse_array(hi - lo, int(round(pattern[t % len(pattern)] * (hi - lo))), [60, seed, t], dtype)
    return out


def plant_cancellations(a, b, k, seed):
    both = np.flatnonzero((bits(a) != 0) & (bits(b) != 0))
    if both.size:
        pick = np.random.default_rng(seed).choice(both, size=min(k, both.size), replace=False)
        if a.dtype == np.uint16:
            b[pick] = a[pick] ^ np.uint16(0x8000)
        else:
            b[pick] = -a[pick]


def plant_zeros(msg, n, dt, k, seed):
    """Zero k stored values of a Pici message (bits set, value all-zero)."""
    h = O.header(msg)
    s = 2 if dt == O.BF16 else 4
    if h["nnz"] == 0:
        return msg
    msg = msg.copy()
    for i in np.random.default_rng(seed).choice(h["nnz"], size=min(k, h["nnz"]), replace=False):
        msg[O.off_A(n) + s * int(i): O.off_A(n) + s * (int(i) + 1)] = 0
    return msg


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("pa,pb", [("sparse", "sparse"), ("tilewise", "tilewise"), ("dense", "sparse"),
                                   ("mixed", "tilewise"), ("mixed", "dense")])
@pytest.mark.parametrize("case", ["plain", "cancel", "stored_zero"])
def test_pici_pici_paths(S, dtype, pa, pb, case, ws_mode):
    dt = O.BF16 if dtype == W.BF16 else O.F32
    n = 13 * 4096 + 1234                      # four partitions, the last one ragged
    a = tiled(n, PATTERNS[pa], 1, dtype)
    b = tiled(n, PATTERNS[pb], 2, dtype)
    if case == "cancel":
        plant_cancellations(a, b, 200, 3)
    ma, mb = O.compress(a)[0], O.compress(b)[0]
    if case == "stored_zero":
        ma, mb = plant_zeros(ma, n, dt, 40, 4), plant_zeros(mb, n, dt, 40, 5)
    exp, _ = O.reduce(O.Operand.stream(ma), O.Operand.stream(mb), n, dt, O.STREAM, O.FMT_PICI)
    log(f"pici+pici n={n} {dtype} {pa}+{pb} {case} {ws_mode}")
    ws = S.alloc_workspace(n, dt, minimal=ws_mode == "single_pass")
    ga, gb = torch.from_numpy(ma).cuda(), torch.from_numpy(mb).cuda()
    out = S.alloc_stream(n, dt)
    out.fill_(0x5A)
    pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    S.spccl_reduce(pici(ga), pici(gb), pici(out), n, dt, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"pici+pici {pa}+{pb} {case}")


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
