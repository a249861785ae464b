"""The threshold model (Sec. IV-C, the sweep of Fig. "rs_threshold_slice"
modelled): its decision replay must be the collectives' rule (checked against
the oracle's ring on inputs whose measured sparsity after k contributions is
exactly sigma0^k), its message sizes the closed forms, its link term the
Hockney model (Eq. 1, Eq. 6), and its sweep must land where the cost model
forces it to in limiting cases.  CPU only."""
import math

import numpy as np
import pytest

import oracle as O
from test_oracle_coo import _digit_sparsity_inputs

T = pytest.importorskip("paper_2607_04676_amd.tuner")


@pytest.mark.parametrize("pol", [O.Policy(), O.Policy(intra_thresh=0.7), O.Policy.coo(),
                                 O.Policy(ranks_per_node=2, inter_thresh=0.7), O.Policy(adaptive=0),
                                 O.Policy(adaptive=2)])
def test_replay_matches_the_oracle_ring(pol):
    P, m = 8, 10000
    sends = _digit_sparsity_inputs(P, m, 4)            # measured sparsity after k ranks: 0.9^k (k <= 4)
    _, tr = O.ring_reduce_scatter(sends, pol)
    tp = T.Policy(pol.intra_thresh, pol.inter_thresh, pol.ag_thresh, pol.ranks_per_node, pol.adaptive,
                  pol.sparse_fmt)
    fmts, tracked, _, _, _ = T.replay_rs(P, 0.9, tp)
    for e in tr:
        if e.step >= 4 and e.fmt != O.FMT_DENSE:
            continue                                   # past 4 contributions the digit supports stop being 0.9^k
        assert fmts[e.step][e.rank] == e.fmt, (e.step, e.rank)
        assert tracked[e.step][e.rank] == pytest.approx(e.sigma, rel=1e-12)


def test_message_sizes_are_the_closed_forms():
    m = 4 * 4096 + 5
    for sg in (0.0, 0.5, 0.9, 0.99, 1.0):
        nnz = int(round((1 - sg) * m))
        assert T.message_bytes(m, 4, T.FMT_PICI, sg) == O.pici_bytes(m, O.F32, nnz)
        assert T.message_bytes(m, 4, T.FMT_COO, sg) == O.coo_bytes(O.F32, nnz)
        assert T.message_bytes(m, 2, T.FMT_DENSE, sg) == O.dense_bytes(m, O.BF16)


def test_all_gather_is_eq6_without_kernel_costs():
    """With free kernels the sparse ring all-gather is (p-1)(alpha + beta n'/p)
    with n' the Pici payload (Eq. 4-6; here with the exact omega)."""
    P, m, s, sg = 8, 1 << 20, 4, 0.95
    link = T.Link(alpha_us=2.5, GBs=100.0)
    free = T.KernelModel.constant(1e12)
    got = T.ag_time_us(P, m, s, sg, T.FMT_PICI, free, T.Policy(), link, link)
    n_prime = T.message_bytes(m, s, T.FMT_PICI, sg)
    assert got == pytest.approx((P - 1) * (2.5 + n_prime / 100e3), rel=1e-9)


def test_free_kernels_never_switch_to_dense():
    """If compression cost nothing (T_comp = T_decomp = 0) only message size
    would matter (Sec. IV-C), and Pici is smaller than dense above about
    3.15% sparsity: the best reduce-scatter threshold is 0 (never dense)."""
    free = T.KernelModel.constant(1e12)
    tab = T.sweep_rs(8, (512 << 20) // 4 // 8, 4, 0.9, free, 0)
    best = min(tab, key=tab.get)
    assert best[0] == 0.0
    assert tab[(0.0, 0.0)] < tab[(1.0, 1.0)]


def test_expensive_compression_goes_dense_at_once():
    """Sparse kernels far slower than the link: the all-dense ring wins, so
    the best thresholds are those at or above sigma0 = 0.9 (dense from step
    0; the test is inclusive)."""
    slow = T.KernelModel.constant(1.0)               # 1 GB/s sparse kernels
    slow.ops["copy"] = T.OpCurve([0.0], [1e9])       # but plain copies and dense adds are free
    slow.ops["dense_dense"] = T.OpCurve([0.0], [1e9])
    tab = T.sweep_rs(8, 1 << 22, 4, 0.9, slow, 0)
    best = min(tab, key=tab.get)
    assert best[0] >= 0.9 and tab[best] == tab[(1.0, 1.0)]
    assert tab[(0.8, 0.8)] > tab[(0.9, 0.9)]


def test_recommend_is_a_grid_point_and_reports_the_paper_pair():
    km = T.KernelModel.constant(4000.0, fixed_us=4.0)
    rec = T.recommend(km, workloads=[(16, 512, 0.95), (32, 2048, 0.99)])
    assert rec["intra_thresh"] in T.GRID and rec["inter_thresh"] in T.GRID and rec["ag_thresh"] in T.GRID
    assert rec["geomean_slowdown_vs_best"] >= 1.0
    assert rec["paper_pair_geomean_slowdown"] >= rec["geomean_slowdown_vs_best"]
    for w in rec["workloads"]:
        assert w["best_us"] <= w["paper_us"] and w["best_us"] <= w["dense_us"] + 1e-9


@pytest.mark.parametrize("s,m,adaptive,launches", [(4, 1 << 16, 1, 43), (4, 1 << 16, 0, 23), (4, 1 << 16, 2, 24),
                                                     (2, 1 << 16, 1, 43), (2, 2049 * 16384, 1, 56),
                                                     (2, 2049 * 16384, 0, 30), (2, 2049 * 16384, 2, 25)])
def test_one_gpu_ring_launches_follow_the_policy(s, m, adaptive, launches):
    """The one-GPU ring issues, per step, a decide and a copy, then for each
    input format the policy allows a Pici sink (a sparse send: one launch, or
    a count and a place pass for bf16 messages above 2048 partitions) and a
    dense sink (a dense send or the last step); step 0 compresses, decides
    and, if dense sends are allowed, encodes them."""
    km = T.KernelModel.constant(4000.0)
    got = T.vr_rs_time_us(8, m, s, 0.99, T.Policy(adaptive=adaptive), km, 3.0)
    assert got["launches"] == launches
    assert got["launch_us"] == pytest.approx(3.0 * launches)


def test_one_gpu_ring_bytes_are_every_rank_summed():
    """Never dense, every op at one bandwidth: the bytes term is the sum over
    ranks and steps of compress (dense chunk + message), the copy of each
    received message (read and write) and the reduction (dense chunk, the
    received message, and the sent message or the dense output at the last
    step), with the message at sigma0^(k+1) after k + 1 contributions."""
    P, m, s, sg, GBs = 4, 3 * 4096 + 17, 4, 0.95, 2000.0
    km = T.KernelModel.constant(GBs)
    pici = lambda x: T.message_bytes(m, s, T.FMT_PICI, x)
    total = P * (m * s + pici(sg))
    for step in range(1, P):
        inb = pici(sg ** step)
        total += P * 2 * inb
        total += P * ((2 * m * s + inb) if step == P - 1 else (m * s + inb + pici(sg ** (step + 1))))
    got = T.vr_rs_time_us(P, m, s, sg, T.Policy(adaptive=0), km, 0.0)
    assert got["bytes_us"] == pytest.approx(total / (GBs * 1e3), rel=1e-12)


def test_recommend_reports_the_tied_region():
    km = T.KernelModel.constant(4000.0, fixed_us=4.0)
    rec = T.recommend(km, workloads=[(16, 512, 0.95), (32, 2048, 0.99)])
    ties = rec["ties"]
    assert ties["pairs"] >= 1
    assert ties["intra"][0] <= rec["intra_thresh"] <= ties["intra"][1]
    assert ties["inter"][0] <= rec["inter_thresh"] <= ties["inter"][1]
    assert ties["ag"][0] <= rec["ag_thresh"] <= ties["ag"][1]
