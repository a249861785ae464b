"""Threshold model for the adaptive dense switch of the ring collectives on
MI355X (Sec. IV-C; the sweep behind Fig. "rs_threshold_slice", modelled).

The paper picks its thresholds (Pici: intra 0.6, inter 0.5, ag 0.1; COO:
0.8 / 0.7 / 0.5) by sweeping them at steps of 0.1 on its own machine.  One
GPU cannot run a real ring, so this module replays the collectives' decision
rule on a cost model of every ring step and sweeps the thresholds the same
way:

* the decision rule is the collectives' own (Sec. IV-C, Eq. 7): step 0
  measures the sparsity sigma0 of the first chunk and sends dense iff
  sigma0 <= tau(link); a later step estimates sigma_prev * sigma0 and either
  reduces to a dense message (tracking the estimate) or reduces and
  compresses (tracking the measured sparsity); at the all-reduce transition
  the gather is dense iff sigma_prev * sigma0 <= ag_thresh;
* the sparsity a step really sees after k + 1 independent uniform
  contributions is sigma0^(k+1) (the expectation Eq. 7 extrapolates);
* a message costs alpha + bytes / bandwidth on its link (the Hockney model,
  Eq. 1), with one (alpha, bandwidth) per link kind;
* a kernel costs fixed + algorithmic bytes / bandwidth, where the bandwidth
  is interpolated in sparsity from times measured on this GPU (bench.py
  measures them; `KernelModel.from_bench` reads its JSON line).

Message sizes are exact (Sec. III-B components, the 48-byte header of
Sec. V-B, the 16-byte pad before the values; COO: a 32-bit index and a value
per nonzero, Sec. II-B).  The step time of a synchronous ring is the slowest
rank's compute plus send.  Nothing here runs on the GPU.
"""
from __future__ import annotations

import argparse
import json
import math
from dataclasses import dataclass, field

FMT_DENSE, FMT_PICI, FMT_COO = 0, 1, 2
HEADER = 48
GRID = [round(0.1 * k, 1) for k in range(11)]          # thresholds swept at steps of 0.1
TIE = 0.005             # geomean slowdowns within 0.5% of the best count as ties


def _align16(x: int) -> int:
    return (x + 15) // 16 * 16


def message_bytes(m: int, s: int, fmt: int, sigma: float) -> int:
    """Bytes of an m-element message of element size s at sparsity sigma."""
    if fmt == FMT_DENSE:
        return HEADER + m * s
    nnz = int(round((1.0 - sigma) * m))
    if fmt == FMT_COO:
        return _align16(HEADER + 4 * nnz) + nnz * s
    T = (m + 4095) // 4096
    return _align16(HEADER + 512 * T + 4 * (T + 1)) + nnz * s


@dataclass
class Link:
    """Hockney link (Eq. 1): a message of n bytes takes alpha + n / bandwidth."""
    alpha_us: float
    GBs: float

    def time_us(self, nbytes: float) -> float:
        return self.alpha_us + nbytes / (self.GBs * 1e3)


# One ring hop uses one link.  Within an 8-GPU MI355X node a hop is one
# xGMI link (about 153 GB/s); between nodes, one NIC (a 400 Gb/s NIC, about
# 50 GB/s).  Startup latencies are typical collective-library values.
XGMI = Link(alpha_us=3.0, GBs=153.0)
NIC = Link(alpha_us=8.0, GBs=50.0)


@dataclass
class OpCurve:
    """Achieved bandwidth of one kernel op (algorithmic bytes / time) at
    measured sparsities; interpolated linearly in sparsity, held flat past
    the ends, plus a fixed cost per launch."""
    sigmas: list
    GBs: list
    fixed_us: float = 0.0

    def bandwidth(self, sigma: float) -> float:
        xs, ys = self.sigmas, self.GBs
        if sigma <= xs[0]:
            return ys[0]
        if sigma >= xs[-1]:
            return ys[-1]
        for i in range(len(xs) - 1):
            if xs[i] <= sigma <= xs[i + 1]:
                f = (sigma - xs[i]) / (xs[i + 1] - xs[i])
                return ys[i] + f * (ys[i + 1] - ys[i])
        return ys[-1]

    def time_us(self, nbytes: float, sigma: float) -> float:
        return self.fixed_us + nbytes / (self.bandwidth(sigma) * 1e3)


@dataclass
class KernelModel:
    """Per-op curves: compress (dense -> sparse), expand (sparse -> dense),
    to_sparse (dense (+) sparse -> sparse), to_dense (dense (+) sparse ->
    dense), dense_dense (dense (+) dense -> dense), copy (a dense message)."""
    ops: dict = field(default_factory=dict)

    def time_us(self, op: str, nbytes: float, sigma: float) -> float:
        return self.ops[op].time_us(nbytes, sigma)

    @staticmethod
    def constant(GBs: float, fixed_us: float = 0.0) -> "KernelModel":
        names = ("compress", "expand", "to_sparse", "to_dense", "dense_dense", "copy")
        return KernelModel({k: OpCurve([0.0], [GBs], fixed_us) for k in names})

    @staticmethod
    def from_ops(ops: dict, dense_ops: dict, copy_GBs: float, fixed_us: float = 0.0) -> "KernelModel":
        """Curves from isolated per-op times on the 256 MiB fp32 array:
        ops["c2.f32.<permille>.<op>"] = [median us, algorithmic bytes, ...]
        (the bench record's roofline table)."""
        names = {"compress": "compress", "expand": "decompress", "to_sparse": "reduce_dense_pici_to_pici",
                 "to_dense": "reduce_dense_pici_to_dense"}
        points = {k: [] for k in names}
        for key, val in ops.items():
            parts = key.split(".")
            if len(parts) != 4 or parts[0] != "c2" or parts[1] != "f32":
                continue
            for k, op in names.items():
                if parts[3] == op:
                    points[k].append((int(parts[2]) / 1000.0, val[1] / (val[0] * 1e-6) / 1e9))
        curves = {}
        for k, pts in points.items():
            pts.sort()
            curves[k] = OpCurve([p[0] for p in pts], [p[1] for p in pts], fixed_us)
        for k in ("dense_dense", "copy"):
            g = dense_ops.get(k, {}).get("achieved_GBs") or copy_GBs
            curves[k] = OpCurve([0.0], [g], fixed_us)
        return KernelModel(curves)

    @staticmethod
    def from_bench(rec: dict, fmt: int = FMT_PICI, fixed_us: float = 4.0) -> "KernelModel":
        """Curves from a bench.py JSON line: its per-op table at the headline
        sparsity and at the swept ones (each entry: ms and algorithmic
        bytes), and its dense-op timings."""
        names = {"compress": "compress", "expand": "decompress", "to_sparse": "reduce_dense_pici_to_pici",
                 "to_dense": "reduce_dense_pici_to_dense"}
        points = {k: [] for k in names}
        tables = [(float(rec["config"]["sigma"]), rec["kernels"])]
        for sg, ent in rec.get("sweep", {}).items():
            tables.append((float(sg), ent["kernels"]))
        for sigma, table in tables:
            for k, op in names.items():
                e = table.get(op)
                if e and e.get("algorithmic_bytes"):
                    points[k].append((sigma, e["algorithmic_bytes"] / (e["ms"] * 1e-3) / 1e9))
        ops = {}
        for k, pts in points.items():
            pts.sort()
            ops[k] = OpCurve([p[0] for p in pts], [p[1] for p in pts], fixed_us)
        dense = rec.get("dense_ops", {})
        for k in ("dense_dense", "copy"):
            g = dense.get(k, {}).get("achieved_GBs") or rec["copy_ceiling"]["GBs"]
            ops[k] = OpCurve([0.0], [g], fixed_us)
        return KernelModel(ops)


@dataclass
class Policy:
    intra_thresh: float = 0.6
    inter_thresh: float = 0.5
    ag_thresh: float = 0.1
    ranks_per_node: int = 0
    adaptive: int = 1
    sparse_fmt: int = FMT_PICI


def link_is_inter(pol: Policy, r: int, P: int) -> bool:
    rpn = pol.ranks_per_node if pol.ranks_per_node > 0 else P
    return (r + 1) % rpn == 0 and rpn < P


def _dense(pol: Policy, sigma: float, tau: float) -> bool:
    if pol.adaptive == 0:
        return False
    if pol.adaptive == 2:
        return True
    return sigma <= tau


def replay_rs(P: int, sigma0: float, pol: Policy):
    """Formats the ring reduce-scatter sends and the sparsity each rank
    tracks, step by step, when every chunk starts at sparsity sigma0 and the
    supports are independent (true sparsity after k + 1 contributions:
    sigma0^(k+1)).  Returns (fmt[step][rank], sigma_tracked[step][rank],
    true_sigma[step], each rank's tracked sparsity after its last send, each
    rank's sigma0)."""
    fmts, tracked, true = [], [], []
    s0 = [sigma0] * P
    sp = [sigma0] * P
    row, trow = [], []
    for r in range(P):
        tau = pol.inter_thresh if link_is_inter(pol, r, P) else pol.intra_thresh
        row.append(FMT_DENSE if _dense(pol, s0[r], tau) else pol.sparse_fmt)
        trow.append(sp[r])
    fmts.append(row)
    tracked.append(trow)
    true.append(sigma0)
    for step in range(1, P - 1):
        row, trow = [], []
        meas = sigma0 ** (step + 1)
        for r in range(P):
            tau = pol.inter_thresh if link_is_inter(pol, r, P) else pol.intra_thresh
            est = sp[r] * s0[r]
            if _dense(pol, est, tau):
                row.append(FMT_DENSE)
                sp[r] = est
            else:
                row.append(pol.sparse_fmt)
                sp[r] = meas
            trow.append(sp[r])
        fmts.append(row)
        tracked.append(trow)
        true.append(meas)
    return fmts, tracked, true, sp, s0


def _link(pol: Policy, r: int, P: int, intra: Link, inter: Link) -> Link:
    return inter if link_is_inter(pol, r, P) else intra


def rs_time_us(P: int, m: int, s: int, sigma0: float, pol: Policy, km: KernelModel,
               intra: Link = XGMI, inter: Link = NIC) -> float:
    """Modelled time of a ring reduce-scatter whose ranks hold P chunks of m
    elements, each at sparsity sigma0."""
    if P == 1:
        return 0.0
    fmts, _, true, _, _ = replay_rs(P, sigma0, pol)
    dense_chunk = m * s
    total = 0.0
    # step 0: compress (and, if the rank goes dense, wrap the chunk as a dense message)
    worst = 0.0
    for r in range(P):
        mb = message_bytes(m, s, pol.sparse_fmt, sigma0)
        t = km.time_us("compress", dense_chunk + mb, sigma0)
        if fmts[0][r] == FMT_DENSE:
            t += km.time_us("copy", 2 * dense_chunk, sigma0)
        out = message_bytes(m, s, fmts[0][r], sigma0)
        t += _link(pol, r, P, intra, inter).time_us(out)
        worst = max(worst, t)
    total += worst
    for step in range(1, P):
        worst = 0.0
        sig_in = true[step - 1]
        sig_out = sigma0 ** (step + 1)
        for r in range(P):
            fin = fmts[step - 1][(r - 1) % P]
            in_b = message_bytes(m, s, fin, sig_in)
            last = step == P - 1
            fout = FMT_DENSE if last else fmts[step][r]
            if fout == FMT_DENSE:
                op = "dense_dense" if fin == FMT_DENSE else "to_dense"
                t = km.time_us(op, dense_chunk + in_b + dense_chunk, sig_in)
            else:
                out_b = message_bytes(m, s, fout, sig_out)
                t = km.time_us("to_sparse", dense_chunk + in_b + out_b, sig_out)
            if not last:
                t += _link(pol, r, P, intra, inter).time_us(message_bytes(m, s, fout, sig_out))
            worst = max(worst, t)
        total += worst
    return total


def pici_sink_launches(m: int, s: int) -> int:
    """Launches of one batched Pici-producing ring step: one (offsets found in
    the same launch) for fp32 messages and bf16 ones of up to 2048 partitions
    of 16384 elements, else a count and a place pass."""
    return 1 if s == 4 or -(-m // 16384) <= 2048 else 2


def vr_rs_time_us(P: int, m: int, s: int, sigma0: float, pol: Policy, km: KernelModel, launch_us: float) -> dict:
    """The same reduce-scatter on one GPU with P virtual ranks and free
    links, as the library runs it: every kernel of a ring step is one
    launch for all ranks, with the format decisions made on the device
    between launches, so a step costs the sum over ranks of its algorithmic
    bytes at the op's bandwidth plus launch_us per launch.  Launches per
    step: a decide and a copy of the received messages, then for each input
    format that can occur a Pici sink (a Pici send: pici_sink_launches) and a
    dense sink (a dense send, or the last step's output); step 0 compresses
    (a Pici sink), decides and, if the policy allows dense sends, encodes them.
    Returns the total and its two terms (us) and the launch count."""
    if P == 1:
        return {"total_us": 0.0, "bytes_us": 0.0, "launch_us": 0.0, "launches": 0}
    can_dense, can_sparse = pol.adaptive != 0, pol.adaptive != 2
    bw = lambda op, sg: km.ops[op].bandwidth(sg) * 1e3        # bytes per us
    fmts, _, true, _, _ = replay_rs(P, sigma0, pol)
    dense_chunk = m * s
    bytes_us = 0.0
    sink = pici_sink_launches(m, s)
    launches = sink + 1 + (1 if can_dense else 0)
    for r in range(P):
        bytes_us += (dense_chunk + message_bytes(m, s, pol.sparse_fmt, sigma0)) / bw("compress", sigma0)
        if fmts[0][r] == FMT_DENSE:
            bytes_us += (2 * dense_chunk) / bw("copy", sigma0)
    for step in range(1, P):
        last = step == P - 1
        launches += 2
        for fin_ok in (can_sparse, can_dense):
            if fin_ok:
                launches += (sink if (not last and can_sparse) else 0) + (1 if (last or can_dense) else 0)
        sig_in, sig_out = true[step - 1], sigma0 ** (step + 1)
        for r in range(P):
            fin = fmts[step - 1][(r - 1) % P]
            in_b = message_bytes(m, s, fin, sig_in)
            bytes_us += 2 * in_b / bw("copy", sig_in)
            fout = FMT_DENSE if last else fmts[step][r]
            if fout == FMT_DENSE:
                op = "dense_dense" if fin == FMT_DENSE else "to_dense"
                bytes_us += (2 * dense_chunk + in_b) / bw(op, sig_in)
            else:
                bytes_us += (dense_chunk + in_b + message_bytes(m, s, fout, sig_out)) / bw("to_sparse", sig_out)
    return {"total_us": bytes_us + launches * launch_us, "bytes_us": bytes_us, "launch_us": launches * launch_us,
            "launches": launches}


def ag_time_us(P: int, m: int, s: int, sigma: float, fmt: int, km: KernelModel,
               pol: Policy | None = None, intra: Link = XGMI, inter: Link = NIC) -> float:
    """Modelled ring all-gather of P parts of m elements at sparsity sigma
    sent in format fmt: encode once, P - 1 forwarding steps, each received
    part expanded (Eq. 4-6 with the kernel costs measured here)."""
    pol = pol or Policy()
    if P == 1:
        return 0.0
    mb = message_bytes(m, s, fmt, sigma)
    enc = km.time_us("copy", 2 * m * s, sigma) if fmt == FMT_DENSE else km.time_us("compress", m * s + mb, sigma)
    exp = km.time_us("copy", 2 * m * s, sigma) if fmt == FMT_DENSE else km.time_us("expand", mb + m * s, sigma)
    hop = max(_link(pol, r, P, intra, inter).time_us(mb) for r in range(P))
    return enc + (P - 1) * (hop + exp)


def ar_time_us(P: int, m: int, s: int, sigma0: float, pol: Policy, km: KernelModel,
               intra: Link = XGMI, inter: Link = NIC) -> float:
    """Ring all-reduce = reduce-scatter, then the phase-aware transition and
    an all-gather of the reduced chunks (Sec. IV-B, IV-C)."""
    t = rs_time_us(P, m, s, sigma0, pol, km, intra, inter)
    if P == 1:
        return t
    _, _, _, sp, s0 = replay_rs(P, sigma0, pol)
    est = sp[0] * s0[0]
    dense = pol.adaptive == 2 or (pol.adaptive == 1 and est <= pol.ag_thresh)
    sig_final = sigma0 ** P
    return t + ag_time_us(P, m, s, sig_final, FMT_DENSE if dense else pol.sparse_fmt, km, pol, intra, inter)


def dense_rs_time_us(P: int, m: int, s: int, km: KernelModel, intra: Link = XGMI, inter: Link = NIC,
                     ranks_per_node: int = 0) -> float:
    """The all-dense ring (every message dense: the NCCL-style baseline)."""
    return rs_time_us(P, m, s, 0.0, Policy(adaptive=2, ranks_per_node=ranks_per_node), km, intra, inter)


def sweep_rs(P: int, m: int, s: int, sigma0: float, km: KernelModel, ranks_per_node: int,
             sparse_fmt: int = FMT_PICI, intra: Link = XGMI, inter: Link = NIC) -> dict:
    """Modelled reduce-scatter time for every (intra, inter) pair of the
    grid; the paper's Fig. "rs_threshold_slice" for this machine model."""
    out = {}
    for ti in GRID:
        for te in GRID:
            pol = Policy(ti, te, 0.1, ranks_per_node, 1, sparse_fmt)
            out[(ti, te)] = rs_time_us(P, m, s, sigma0, pol, km, intra, inter)
    return out


def recommend(km: KernelModel, workloads=None, sparse_fmt: int = FMT_PICI, intra: Link = XGMI,
              inter: Link = NIC) -> dict:
    """Threshold pair (and ag threshold) that is best overall across the
    workloads: the one with the smallest geometric-mean slowdown against
    each workload's own best pair, as the paper picks pairs that are
    "generally strong" across GPU counts and sizes."""
    if workloads is None:
        workloads = [(P, mib, sg) for P in (16, 32) for mib in (512, 2048) for sg in (0.9, 0.95, 0.99)]
    s = 4
    logs = {pair: 0.0 for pair in ((a, b) for a in GRID for b in GRID)}
    per = []
    for P, mib, sg in workloads:
        m = (mib << 20) // s // P
        tab = sweep_rs(P, m, s, sg, km, 8, sparse_fmt, intra, inter)
        best = min(tab.values())
        for pair, t in tab.items():
            logs[pair] += math.log(t / best)
        bp = min(tab, key=tab.get)
        per.append({"P": P, "MiB": mib, "sigma0": sg, "best": bp, "best_us": round(best, 2),
                    "dense_us": round(dense_rs_time_us(P, m, s, km, intra, inter, 8), 2),
                    "paper_us": round(tab[(0.6, 0.5) if sparse_fmt == FMT_PICI else (0.8, 0.7)], 2)})
    pair = min(logs, key=logs.get)
    # pairs within TIE of the best geomean slowdown: the optimum is often a
    # plateau, and the single pick is then a tie-break (lowest thresholds)
    tied = sorted(q for q in logs if logs[q] <= logs[pair] + math.log1p(TIE))
    # ag threshold: best for the all-reduce at the chosen pair
    ag_logs = {g: 0.0 for g in GRID}
    for P, mib, sg in workloads:
        m = (mib << 20) // s // P
        times = {g: ar_time_us(P, m, s, sg, Policy(pair[0], pair[1], g, 8, 1, sparse_fmt), km, intra, inter)
                 for g in GRID}
        best = min(times.values())
        for g, t in times.items():
            ag_logs[g] += math.log(t / best)
    ag = min(ag_logs, key=ag_logs.get)
    n = len(workloads)
    ag_tied = sorted(g for g in ag_logs if ag_logs[g] <= ag_logs[ag] + math.log1p(TIE))
    return {"intra_thresh": pair[0], "inter_thresh": pair[1], "ag_thresh": ag,
            "ties": {"within": TIE, "pairs": len(tied),
                     "intra": [min(q[0] for q in tied), max(q[0] for q in tied)],
                     "inter": [min(q[1] for q in tied), max(q[1] for q in tied)],
                     "ag": [ag_tied[0], ag_tied[-1]]},
            "geomean_slowdown_vs_best": round(math.exp(logs[pair] / n), 4),
            "paper_pair_geomean_slowdown": round(math.exp(logs[(0.6, 0.5) if sparse_fmt == FMT_PICI
                                                           else (0.8, 0.7)] / n), 4),
            "workloads": per,
            "links": {"intra": vars(intra), "inter": vars(inter)}}


def main():
    ap = argparse.ArgumentParser(description="modelled threshold sweep from a bench.py JSON line")
    ap.add_argument("bench_json")
    args = ap.parse_args()
    rec = json.loads(open(args.bench_json).read().strip().splitlines()[-1])
    print(json.dumps(recommend(KernelModel.from_bench(rec)), indent=1))


if __name__ == "__main__":
    main()
