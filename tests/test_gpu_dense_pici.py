"""Dense (+) Pici -> Pici (Sec. IV-B, reduction with fill-in as in Sec. I)
against the oracle byte for byte, on tiles built around the choices the sink
makes per tile: how many Pici values a column holds (up to six are merged
sparsely, more take the row-wise merge), the union of both operands against
the LDS stage (at the limit the sparse merge runs, one past it the row-wise
one), exact cancellations where both operands are present, stored zeros in
the Pici values (they read as absent and send the tile to the row-wise
merge), tiles with too many values to be read early, empty operands and a
ragged last tile; fp32 and bf16, both operand orders, both workspace sizes."""
import numpy as np
import pytest

import oracle as O
import workloads as W
from helpers import assert_bytes_equal, bits, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TILE = 4096
EARLY = 512          # Pici values of a tile read before its dense rows finish
STAGE = {W.F32: 1792, W.BF16: 3584}     # output values one wave stages at once


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_04676_amd as S
    return S


def values(rng, k, dtype):
    """k nonzero values (raw bits nonzero) of the dtype."""
    x = rng.standard_normal(k).astype(np.float32)
    if dtype == W.BF16:
        b = (x.view(np.uint32) >> 16).astype(np.uint16)
        b[b == 0] = 0x3F80
        return b
    x[x.view(np.uint32) == 0] = 1.0
    return x


def per_column(rng, counts):
    """Positions inside a tile: counts[c] distinct rows of column c."""
    pos = [64 * rng.choice(64, size=k, replace=False) + c for c, k in enumerate(counts) if k]
    return np.sort(np.concatenate(pos)) if pos else np.zeros(0, np.int64)


# Each spec builds one tile: (name, Pici values per column, dense density).
# "edge" puts one Pici value in each column, on rows the dense operand leaves
# empty, and fills the dense operand so that both together are `stage - EARLY
# + d` values: d = 0 is the largest union the sparse merge takes.
SPECS = [("cols", 0, 0.01), ("cols", 1, 0.01), ("cols", 5, 0.02), ("cols", 6, 0.01), ("cols", 7, 0.01),
         ("cols", 6, 0.3), ("mixed", None, 0.05), ("edge", 0, None), ("edge", 1, None), ("cols", 10, 0.01),
         ("cols", 3, 0.0), ("cols", 0, 0.5), ("cols", 2, 1.0)]


def build(n, dtype, seed):
    rng = np.random.default_rng(seed)
    a, b = W.empty(n, dtype), W.empty(n, dtype)
    for t in range(-(-n // TILE)):
        lo, hi = TILE * t, min(n, TILE * (t + 1))
        name, k, da = SPECS[t % len(SPECS)]
        if name == "edge":
            pb = 64 * rng.integers(0, 64, size=64) + np.arange(64)
            free = np.setdiff1d(np.arange(TILE), pb)
            pa = rng.choice(free, size=STAGE[dtype] - EARLY - 64 + k, replace=False)
        else:
            counts = rng.integers(0, 9, size=64) if name == "mixed" else np.full(64, k)
            pb = per_column(rng, counts)
            pa = rng.choice(TILE, size=int(round(da * TILE)), replace=False)
        pa, pb = pa[pa < hi - lo], pb[pb < hi - lo]
        a[lo + pa] = values(rng, pa.size, dtype)
        b[lo + pb] = values(rng, pb.size, dtype)
    return a, b


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


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
@pytest.mark.parametrize("order", ["dense_pici", "pici_dense"])
@pytest.mark.parametrize("case", ["plain", "cancel", "stored_zero"])
def test_dense_pici_paths(S, dtype, order, case, ws_mode):
    dt = O.BF16 if dtype == W.BF16 else O.F32
    n = (2 * len(SPECS) + 2) * TILE + 1234    # every spec twice and more, then a ragged tile
    a, b = build(n, dtype, 11)
    if case == "cancel":
        plant_cancellations(a, b, 300, 12)
    mb = O.compress(b)[0]
    if case == "stored_zero":
        mb = plant_zeros(mb, n, dt, 40, 13)
    oa, ob = O.Operand.array(a), O.Operand.stream(mb)
    first, second = (oa, ob) if order == "dense_pici" else (ob, oa)
    exp, _ = O.reduce(first, second, n, dt, O.STREAM, O.FMT_PICI)
    log(f"dense+pici n={n} {dtype} {order} {case} {ws_mode}")
    ws = S.alloc_workspace(n, dt, minimal=ws_mode == "single_pass")
    ga = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()
    if dtype == W.BF16:
        ga = ga.view(torch.bfloat16)
    gb = torch.from_numpy(mb).cuda()
    out = S.alloc_stream(n, dt)
    out.fill_(0x5A)
    pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    x, y = (S.operand(ga), pici(gb)) if order == "dense_pici" else (pici(gb), S.operand(ga))
    S.spccl_reduce(x, y, pici(out), n, dt, ws)
    torch.cuda.synchronize()
    assert S.spccl_read_status(ws) == 0
    assert_bytes_equal(out[:exp.size].cpu().numpy(), exp, f"dense+pici {order} {case}")
