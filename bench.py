"""Throughput of the Pici hot path on one MI355X.

Headline workload (``value``): the codec sweep array -- 67,108,864 fp32
elements (256 MiB) with uniformly random nonzero positions and N(0,1) values
-- at sparsity 0.99.  Inputs are resident in HBM before timing; four copies
of each operand rotate between steps so the 256 MB Infinity Cache cannot
serve a step's dense input.  One step is one pass of the whole hot path:

  compress(a)                     dense -> Pici (count pass, then place pass)
  send                            device-sized copy of the message
  decompress(received)            Pici -> dense
  reduce a (+) Pici(b)            the reduce-scatter step with fill-in; its
                                  output is a Pici message, or a dense one
                                  when the adaptive switch says so
  switch_header                   that message's header is copied to pinned
                                  host memory right behind the reduce; the
                                  host applies Eq. 7 (estimate = tracked
                                  sparsity x sigma0 <= 0.6 -> the next step's
                                  reduce sends dense) while the GPU runs on
  reduce Pici(a) (+) Pici(b) -> Pici
  reduce a (+) Pici(b) -> dense   the last reduce-scatter step
  gather_expand of two messages   the all-gather receive side

value = dense-equivalent bytes of the step (n*s per codec op, 2*n*s per
reduce, parts*n*s per gather) / step time over the timed steps.

Per-op fractions of the HBM roofline: every op of every workload is also
timed on its own ("isolated": median over repetitions, each after 512 MiB of
scratch writes so no cache holds its operands) and priced by its algorithmic
bytes (dense bytes read or written plus message bytes read or written)
against 8 TB/s.  The table covers the sparsities 0.9 and 0.99 of the 256 MiB
array in fp32 and bf16, the 1,048,576-element pair, each step of the P = 8
reduce-scatter ring on one chunk, and the bf16 all-gather's compression and
8-part expansion; it is printed inside ``roofline`` as ``ops`` (key ->
[median us, algorithmic bytes, fraction]).  The collectives themselves
(reduce-scatter, all-gather, all-reduce; canonical and sliced) are timed as
whole calls.  --full-out writes the complete record (step-sequence op
times, sweeps, sliced and COO forms, the threshold model) to a file.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "dense-equivalent GB/s (and % of HBM peak) for Pici compress/decompress/reduce"

# ops that launch exactly one kernel, and that kernel's name in profiles
SINGLE_KERNEL_OPS = {
    "decompress": "k_gather<F32, 2>",
    "reduce_dense_pici_to_dense": "k_to_dense<F32, 1, 2>",
    "gather_expand": "k_gather<F32, 2>",
    "send": "k_copy_message",
}
TAU_INTRA = 0.6          # the paper's intra-node threshold for Pici (Sec. IV-C)


def kernel_source_digest() -> str:
    import hashlib
    src = os.path.join(ROOT, "paper_2607_04676_amd", "csrc", "spccl_kernels.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]


def traffic_for(op: str):
    """HBM bytes per launch of an op's kernel from rocprofv3 FETCH_SIZE and
    WRITE_SIZE counters (profiles/traffic.json, already scaled by the plain
    copy calibration), provided they were taken on the current kernel source;
    otherwise null."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    ent = rec.get("ops", {}).get(op)
    if ent is None or rec.get("kernel_source_sha256_16") != kernel_source_digest():
        return None
    return ent.get("hbm_bytes_per_launch")


def _ensure_built():
    lib = os.path.join(ROOT, "paper_2607_04676_amd", "libspccl.so")
    if not os.path.exists(lib):
        import __graft_entry__
        __graft_entry__.build()


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def frac_of(alg_bytes, us):
    return round(alg_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)


class Isolator:
    """Times ops on their own: before every repetition 512 MiB of scratch is
    written (untimed), so neither the Infinity Cache nor the L2 holds the op's
    operands and the op pays for that write-back as a cold launch would."""

    def __init__(self, torch, reps, warm=5):
        self.torch, self.reps, self.warm = torch, reps, warm
        self.junk = torch.empty(1 << 27, dtype=torch.float32, device="cuda")

    def time(self, f):
        torch = self.torch
        ts = []
        for r in range(self.warm + self.reps):
            self.junk.fill_(float(r))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            f()
            e1.record()
            e1.synchronize()
            if r >= self.warm:
                ts.append(e0.elapsed_time(e1) * 1e3)
        return float(np.median(ts)), float(min(ts)), float(max(ts))

    def table(self, ops, alg):
        """ops: [(name, launch)], alg: {name: algorithmic bytes} (after one run)."""
        out = {}
        for nm, f in ops:
            med, lo, hi = self.time(f)
            out[nm] = {"median_us": round(med, 2), "min_us": round(lo, 2), "max_us": round(hi, 2),
                       "reps": self.reps, "algorithmic_bytes": alg[nm], "frac_of_hbm_peak": frac_of(alg[nm], med)}
        return out


def _host(t):
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _dev(a):
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


class Runner:
    """Device buffers and the per-op launch closures of the step on the
    256 MiB array at one sparsity (fp32, or bf16 of the same byte size)."""

    def __init__(self, S, torch, n, permille, copies, bf16=False):
        import workloads as W
        self.S, self.torch, self.n, self.bf16 = S, torch, n, bf16
        self.dt = S.SPCCL_BF16 if bf16 else S.SPCCL_F32
        self.s = 2 if bf16 else 4
        t0 = time.time()
        if bf16:
            a = W.sparse_array(n, W.nnz_for(n, permille), [2, 0, 1, permille], W.BF16)
            b = W.sparse_array(n, W.nnz_for(n, permille), [2, 1, 1, permille], W.BF16)
        else:
            a, b = W.cfg2(permille, 0, n), W.cfg2(permille, 1, n)
        self.host_a, self.host_b = a, b
        _log(f"generated sigma={permille / 1000} {'bf16' if bf16 else 'fp32'} inputs in {time.time() - t0:.1f}s")
        ta, tb = _dev(a), _dev(b)
        self.a = [ta] + [ta.clone() for _ in range(copies - 1)]
        self.b = [tb] + [tb.clone() for _ in range(copies - 1)]
        self.ws = S.alloc_workspace(n, self.dt, "cuda")
        bound = S.spccl_stream_bound(n, self.dt)
        mk = lambda: torch.empty(bound, dtype=torch.uint8, device="cuda")
        self.msg_b = [mk() for _ in range(copies)]
        for k in range(copies):
            S.spccl_compress(self.b[k], self.msg_b[k], self.ws)
        self.msg_a, self.recv, self.red_p, self.red_pp = mk(), mk(), mk(), mk()
        edt = torch.bfloat16 if bf16 else torch.float32
        self.dense_out = torch.empty(n, dtype=edt, device="cuda")
        self.red_d = torch.empty(n, dtype=edt, device="cuda")
        self.gather_out = torch.empty(2 * n, dtype=edt, device="cuda")
        torch.cuda.synchronize()
        hb = S.spccl_read_header(self.msg_b[0])
        self.nnz_b, self.bytes_b = hb["nnz"], hb["total_bytes"]
        # adaptive switch state (Sec. IV-C): the first send compresses the
        # rank's chunk and measures sigma0, which is also the tracked sparsity
        # the first reduce-scatter step's estimate starts from
        S.spccl_compress(self.a[0], self.msg_a, self.ws)
        ha = S.spccl_read_header(self.msg_a)
        self.sigma0 = self.sigma_prev = (n - ha["nnz"]) / n
        self.next_dense = self.sigma_prev * self.sigma0 <= TAU_INTRA
        if self.next_dense:
            self.sigma_prev *= self.sigma0
        self.switch_log = []
        self.hdr_host = torch.empty(48, dtype=torch.uint8, pin_memory=True)
        self.hdr_ev = torch.cuda.Event()

    def ops(self, k):
        """(name, launch, dense-equivalent bytes) of one step on copy k."""
        S, n, s, dt = self.S, self.n, self.s, self.dt
        a, b, mb, ws = self.a[k], self.b[k], self.msg_b[k], self.ws
        P, D, A = S.SPCCL_FMT_PICI, S.SPCCL_FMT_DENSE, S.SPCCL_STREAM
        msg = lambda t, f=P: S.operand(t, A, f)
        rs_fmt = D if self.next_dense else P
        rs_name = "reduce_dense_pici_to_dense_msg" if self.next_dense else "reduce_dense_pici_to_pici"
        return [
            ("compress", lambda: S.spccl_compress(a, self.msg_a, ws), n * s),
            ("send", lambda: S.spccl_copy_message(self.msg_a, self.recv, ws), 0),
            ("decompress", lambda: S.spccl_decompress(self.recv, self.dense_out, ws), n * s),
            (rs_name, lambda: S.spccl_reduce(S.operand(a), msg(mb), msg(self.red_p, rs_fmt), n, dt, ws), 2 * n * s),
            ("switch_header", self.fetch_header, 0),
            ("reduce_pici_pici_to_pici", lambda: S.spccl_reduce(msg(self.msg_a), msg(mb), msg(self.red_pp), n, dt, ws),
             2 * n * s),
            ("reduce_dense_pici_to_dense", lambda: S.spccl_reduce(S.operand(a), msg(mb), S.operand(self.red_d), n,
                                                                  dt, ws), 2 * n * s),
            ("gather_expand", lambda: S.spccl_gather_expand([msg(self.recv), msg(self.red_p)], n, dt,
                                                            self.gather_out, ws), 2 * n * s),
        ]

    def fetch_header(self):
        """Queue the copy of the reduce-scatter step's 48-byte header to
        pinned host memory right behind the reduce that writes it."""
        self.hdr_host.copy_(self.red_p[:48], non_blocking=True)
        self.hdr_ev.record()

    def decide(self):
        """The adaptive switch (Sec. IV-C) for the next step's reduce: a Pici
        message's header gives the measured sparsity, which becomes the tracked
        one; the estimate sigma_prev * sigma0 (Eq. 7) <= 0.6 sends the next
        message dense, and a dense send tracks the estimate.  Waits for the
        header copy only, not for the ops queued after it."""
        self.hdr_ev.synchronize()
        h = self.hdr_host.numpy()
        assert int(h[:4].view(np.uint32)[0]) == 0x49434950
        if int(h[4:6].view(np.uint16)[0]) == self.S.SPCCL_FMT_PICI:
            nnz = int(h[16:24].view(np.uint64)[0])
            self.sigma_prev = (self.n - nnz) / self.n
        est = self.sigma_prev * self.sigma0
        self.next_dense = est <= TAU_INTRA
        if self.next_dense:
            self.sigma_prev = est
        self.switch_log.append("dense" if self.next_dense else "pici")

    def algorithmic_bytes(self):
        """Bytes each op must move at minimum (reads + writes), per launch."""
        S, n, s = self.S, self.n, self.s
        self.torch.cuda.synchronize()
        ba = S.spccl_read_header(self.msg_a)["total_bytes"]
        bp = S.spccl_read_header(self.red_p)["total_bytes"]
        bpp = S.spccl_read_header(self.red_pp)["total_bytes"]
        bb = self.bytes_b
        return {
            "compress": n * s + ba,
            "send": 2 * ba,
            "decompress": ba + n * s,
            "reduce_dense_pici_to_pici": n * s + bb + bp,
            "reduce_dense_pici_to_dense_msg": n * s + bb + 48 + n * s,
            "reduce_pici_pici_to_pici": ba + bb + bpp,
            "reduce_dense_pici_to_dense": n * s + bb + n * s,
            "gather_expand": ba + bp + 2 * n * s,
            "switch_header": 48,
        }

    def isolated_ops(self):
        """The five target ops on copy 0, each a fresh call (R3's output Pici)."""
        S, n, dt, ws = self.S, self.n, self.dt, self.ws
        a, mb = self.a[0], self.msg_b[0]
        msg = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
        return [
            ("compress", lambda: S.spccl_compress(a, self.msg_a, ws)),
            ("decompress", lambda: S.spccl_decompress(self.msg_a, self.dense_out, ws)),
            ("reduce_dense_pici_to_pici", lambda: S.spccl_reduce(S.operand(a), msg(mb), msg(self.red_p), n, dt, ws)),
            ("reduce_pici_pici_to_pici", lambda: S.spccl_reduce(msg(self.msg_a), msg(mb), msg(self.red_pp), n, dt,
                                                                ws)),
            ("reduce_dense_pici_to_dense", lambda: S.spccl_reduce(S.operand(a), msg(mb), S.operand(self.red_d), n, dt,
                                                                  ws)),
            ("gather_expand", lambda: S.spccl_gather_expand([msg(self.msg_a), msg(self.red_p)], n, dt,
                                                            self.gather_out, ws)),
        ]

    def calibration_copy(self):
        """One large plain copy of known size (a dense message of the input:
        48 + N*s bytes read and written) for scaling HBM byte counters."""
        S, torch = self.S, self.torch
        big = torch.empty(S.spccl_stream_bound(self.n, self.dt), dtype=torch.uint8, device="cuda")
        big2 = torch.empty_like(big)
        S.spccl_encode_dense(self.a[0], big)
        S.spccl_copy_message(big, big2, self.ws)
        torch.cuda.synchronize()
        return 48 + self.n * self.s

    def check_parity(self):
        """Sampled parity against the oracle: the compressed message of a, whole."""
        import oracle as O
        exp, _ = O.compress(self.host_a)
        got = self.msg_a[:exp.size].cpu().numpy()
        return bool(np.array_equal(got, exp))


class SlicedRunner:
    """The in-collective form of the same ops (Sec. III-B phase 2, Sec. V-B):
    sliced streams, one message per 16384-element slice with its own
    block-local prefix sums and its own format decision, on the arrays of R."""

    def __init__(self, R, dense_thresh=0.6):
        S, torch = R.S, R.torch
        self.R, self.S, self.torch, self.n, self.ws = R, S, torch, R.n, R.ws
        self.thresh = dense_thresh
        self.slot = S.spccl_slice_bytes(R.dt)
        self.nslices = S.spccl_slice_count(R.n)
        mk = lambda: S.alloc_sliced(R.n, R.dt)
        self.sb = [mk() for _ in R.b]
        for k, b in enumerate(R.b):
            S.spccl_compress_sliced(b, self.sb[k], R.ws, self.thresh)
        self.sa, self.recv, self.red = mk(), mk(), mk()
        torch.cuda.synchronize()

    def ops(self, k):
        S, R, n, s = self.S, self.R, self.n, self.R.s
        a, sb, ws, th = R.a[k], self.sb[k], R.ws, self.thresh
        return [
            ("compress_sliced", lambda: S.spccl_compress_sliced(a, self.sa, ws, th), n * s),
            ("send_sliced", lambda: S.spccl_copy_sliced(self.sa, self.recv, n, R.dt, ws), 0),
            ("decompress_sliced", lambda: S.spccl_decompress_sliced(self.recv, R.dense_out, ws), n * s),
            ("reduce_dense_sliced_to_sliced", lambda: S.spccl_reduce_sliced(a, sb, self.red, ws, True, th), 2 * n * s),
            ("reduce_dense_sliced_to_dense", lambda: S.spccl_reduce_sliced(a, sb, R.red_d, ws, False, th), 2 * n * s),
        ]

    def decide(self):
        pass

    def stream_bytes(self, buf):
        """Sum of the slots' message sizes (header.total_bytes of each slot)."""
        h = buf[: self.nslices * self.slot].view(self.nslices, self.slot)[:, :48].cpu().numpy()
        return int(h[:, 40:48].copy().view(np.uint64).sum())

    def algorithmic_bytes(self):
        n, s = self.n, self.R.s
        self.torch.cuda.synchronize()
        ba, bb, bo = self.stream_bytes(self.sa), self.stream_bytes(self.sb[0]), self.stream_bytes(self.red)
        return {
            "compress_sliced": n * s + ba,
            "send_sliced": 2 * ba,
            "decompress_sliced": ba + n * s,
            "reduce_dense_sliced_to_sliced": n * s + bb + bo,
            "reduce_dense_sliced_to_dense": 2 * n * s + bb,
        }

    def check_parity(self):
        """Sampled parity against the oracle: the first and last slices of the
        compressed stream of a, each message whole."""
        import oracle as O
        ok = True
        for q in (0, self.nslices - 1):
            lo = q * O.SLICE_ELEMS
            x = self.R.host_a[lo: lo + O.SLICE_ELEMS]
            exp = O.slot_messages(O.encode_sliced(x, self.thresh), x.size, O.F32)[0]
            got = self.sa[q * self.slot: q * self.slot + exp.size].cpu().numpy()
            ok = ok and bool(np.array_equal(got, exp))
        return ok


class CooRunner:
    """The same ops with COO messages (Sec. II-B format; Sec. IV-D runs it
    beside Pici): compress, send, decompress, the reduce-scatter step
    dense (+) COO -> COO, and dense (+) COO -> dense, on the arrays of R."""

    def __init__(self, R):
        S, torch = R.S, R.torch
        self.R, self.S, self.torch, self.n, self.ws = R, S, torch, R.n, R.ws
        mk = lambda: S.alloc_stream(R.n, R.dt, fmt=S.SPCCL_FMT_COO)
        self.cb = [mk() for _ in R.b]
        for k, b in enumerate(R.b):
            S.spccl_compress_coo(b, self.cb[k], R.ws)
        self.ca, self.recv, self.red = mk(), mk(), mk()
        torch.cuda.synchronize()

    def ops(self, k):
        S, R, n, s = self.S, self.R, self.n, self.R.s
        a, cb, ws, dt = R.a[k], self.cb[k], R.ws, R.dt
        msg = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_COO)
        return [
            ("compress_coo", lambda: S.spccl_compress_coo(a, self.ca, ws), n * s),
            ("send_coo", lambda: S.spccl_copy_message(self.ca, self.recv, ws), 0),
            ("decompress_coo", lambda: S.spccl_decompress(self.recv, R.dense_out, ws), n * s),
            ("reduce_dense_coo_to_coo", lambda: S.spccl_reduce(S.operand(a), msg(cb), msg(self.red), n, dt, ws),
             2 * n * s),
            ("reduce_dense_coo_to_dense", lambda: S.spccl_reduce(S.operand(a), msg(cb), S.operand(R.red_d), n, dt,
                                                                 ws), 2 * n * s),
        ]

    def decide(self):
        pass

    def algorithmic_bytes(self):
        S, n, s = self.S, self.n, self.R.s
        self.torch.cuda.synchronize()
        ba = S.spccl_read_header(self.ca)["total_bytes"]
        bb = S.spccl_read_header(self.cb[0])["total_bytes"]
        bo = S.spccl_read_header(self.red)["total_bytes"]
        return {
            "compress_coo": n * s + ba,
            "send_coo": 2 * ba,
            "decompress_coo": ba + n * s,
            "reduce_dense_coo_to_coo": n * s + bb + bo,
            "reduce_dense_coo_to_dense": 2 * n * s + bb,
        }

    def check_parity(self):
        """Sampled parity against the oracle: the COO message of a, whole."""
        import oracle as O
        exp, _ = O.compress_coo(self.R.host_a)
        return bool(np.array_equal(self.ca[:exp.size].cpu().numpy(), exp))


def run_steps(R, steps, copies, bracket):
    """steps steps of the op sequence; ops named in bracket are each wrapped in
    a pair of HIP events on the current stream.  Returns (total ms, wall s,
    {op: mean ms}, dense-equivalent bytes)."""
    torch = R.torch
    ev = {}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start_all = torch.cuda.Event(enable_timing=True)
    end_all = torch.cuda.Event(enable_timing=True)
    start_all.record()
    dense_eq = 0
    for k in range(steps):
        for nm, f, deq in R.ops(k % copies):
            if nm in bracket:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                f()
                e1.record()
                ev.setdefault(nm, []).append((e0, e1))
            else:
                f()
            dense_eq += deq
        R.decide()
    end_all.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start_all.elapsed_time(end_all)
    per = {nm: float(np.mean([a.elapsed_time(b) for a, b in v])) for nm, v in ev.items()}
    st = R.S.spccl_read_status(R.ws)
    if st != 0:
        raise RuntimeError(f"device status {st} after timing")
    return total_ms, wall, per, dense_eq


def time_steps(R, steps, warmup, copies):
    """Warm-up, a per-op breakdown pass (every op bracketed), then the timed
    steps with only the roofline op bracketed.  Returns (total ms, wall s,
    per-op ms from the breakdown, dense-equivalent bytes, roofline op, its ms
    in the timed region)."""
    for w in range(warmup):
        for _, f, _ in R.ops(w % copies):
            f()
        R.decide()
    names = set()
    for k in range(copies):
        names |= {op[0] for op in R.ops(k)} | {"reduce_dense_pici_to_pici", "reduce_dense_pici_to_dense_msg"}
    _, _, per, _ = run_steps(R, max(3, steps // 3), copies, names)
    dom = max((k for k in per if k in SINGLE_KERNEL_OPS), key=lambda k: per[k])
    total_ms, wall, timed, dense_eq = run_steps(R, steps, copies, {dom})
    return total_ms, wall, per, dense_eq, dom, timed[dom]


def run_once(R):
    """Run the isolated ops once (so every output message is the one they
    time) and return their algorithmic bytes."""
    for _, f in R.isolated_ops():
        f()
    return R.algorithmic_bytes()


def op_table(per, alg):
    out = {}
    for nm, ms in per.items():
        gbs = alg[nm] / (ms / 1e3) / 1e9
        out[nm] = {"ms": round(ms, 5), "algorithmic_bytes": alg[nm], "achieved_GBs": round(gbs, 1),
                   "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
    return out


def time_cfg1(S, torch, iso):
    """The 1,048,576-element fp32 pair at 0.99 (seeds 0 and 1): compress,
    decompress, Pici (+) Pici -> Pici, dense (+) Pici -> dense; each op's
    result checked byte for byte against the oracle."""
    import oracle as O
    import workloads as W
    a, b = W.cfg1()
    n, F = a.size, S.SPCCL_F32
    ta, tb = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    ws = S.alloc_workspace(n, F)
    ma, mb, mo = (S.alloc_stream(n, F) for _ in range(3))
    back = torch.empty(n, dtype=torch.float32, device="cuda")
    dn = torch.empty(n, dtype=torch.float32, device="cuda")
    msg = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    S.spccl_compress(tb, mb, ws)
    ops = [("compress", lambda: S.spccl_compress(ta, ma, ws)),
           ("decompress", lambda: S.spccl_decompress(ma, back, ws)),
           ("reduce_pici_pici_to_pici", lambda: S.spccl_reduce(msg(ma), msg(mb), msg(mo), n, F, ws)),
           ("reduce_dense_pici_to_dense", lambda: S.spccl_reduce(S.operand(ta), msg(mb), S.operand(dn), n, F, ws))]
    for _, f in ops:
        f()
    torch.cuda.synchronize()
    ea, _ = O.compress(a)
    eb, _ = O.compress(b)
    epp, _ = O.reduce(O.Operand.stream(ea), O.Operand.stream(eb), n, O.F32, O.STREAM, O.FMT_PICI)
    edn = O.reduce(O.Operand.array(a), O.Operand.stream(eb), n, O.F32)
    parity = (np.array_equal(ma[:ea.size].cpu().numpy(), ea) and np.array_equal(mo[:epp.size].cpu().numpy(), epp)
              and np.array_equal(back.cpu().numpy().view(np.uint32), a.view(np.uint32))
              and np.array_equal(dn.cpu().numpy().view(np.uint32), edn.view(np.uint32)))
    alg = {"compress": 4 * n + ea.size, "decompress": ea.size + 4 * n,
           "reduce_pici_pici_to_pici": ea.size + eb.size + epp.size, "reduce_dense_pici_to_dense": 8 * n + eb.size}
    res = iso.table(ops, alg)
    del ta, tb, ws, ma, mb, mo, back, dn
    return res, bool(parity)


def time_cfg3_steps(S, torch, iso):
    """The P = 8 x 33,554,432 fp32 reduce-scatter at 0.99, step by step on one
    chunk (chunk 0, m = 4,194,304): the ring folds X_1, X_2, ..., X_7 and last
    X_0 into it, so step s (1 <= s <= 6) reduces the received message of s
    contributions with X_{s+1}'s chunk into a Pici message of s + 1 (the fused
    step), and step 7 reduces the message of 7 with X_0's chunk into the dense
    result.  Each step is timed on its own; its first message and the step-1
    result are checked against the oracle."""
    import oracle as O
    import workloads as W
    P, m, F = W.CFG3_P, W.CFG3_N // W.CFG3_P, S.SPCCL_F32
    chunks = [W.cfg3_rank(r)[:m].copy() for r in range(P)]
    dev = [torch.from_numpy(c).cuda() for c in chunks]
    ws = S.alloc_workspace(m, F)
    msgs = [S.alloc_stream(m, F) for _ in range(P)]
    out = torch.empty(m, dtype=torch.float32, device="cuda")
    pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    S.spccl_compress(dev[1], msgs[1], ws)
    ops, alg = [], {}
    for s in range(1, P):
        own = dev[(s + 1) % P]
        if s < P - 1:
            f = (lambda i=s, o=own: S.spccl_reduce(pici(msgs[i]), S.operand(o), pici(msgs[i + 1]), m, F, ws))
        else:
            f = (lambda i=s, o=own: S.spccl_reduce(pici(msgs[i]), S.operand(o), S.operand(out), m, F, ws))
        f()
        torch.cuda.synchronize()
        bin_ = S.spccl_read_header(msgs[s])["total_bytes"]
        bout = S.spccl_read_header(msgs[s + 1])["total_bytes"] if s < P - 1 else 4 * m
        nm = f"step{s}"
        ops.append((nm, f))
        alg[nm] = bin_ + 4 * m + bout
    e1, _ = O.compress(chunks[1])
    e2, _ = O.reduce(O.Operand.stream(e1), O.Operand.array(chunks[2]), m, O.F32, O.STREAM, O.FMT_PICI)
    parity = (np.array_equal(msgs[1][:e1.size].cpu().numpy(), e1)
              and np.array_equal(msgs[2][:e2.size].cpu().numpy(), e2))
    res = iso.table(ops, alg)
    for s in range(1, P):
        res[f"step{s}"]["message_in_bytes"] = int(S.spccl_read_header(msgs[s])["total_bytes"])
    del dev, ws, msgs, out
    return res, bool(parity)


def time_cfg4_ops(S, torch, iso):
    """The P = 8 x 16,777,216 bf16 all-gather at 0.999: compression of one
    rank's part, and the 8-part expansion of all ranks' messages into the
    134,217,728-element output; rank 0's message and the expanded output
    (whole) checked against the oracle."""
    import oracle as O
    import workloads as W
    P, n, B = W.CFG4_P, W.CFG4_N, S.SPCCL_BF16
    parts = [W.cfg4_rank(r) for r in range(P)]
    dev = [_dev(x) for x in parts]
    ws = S.alloc_workspace(n, B)
    msgs = [S.alloc_stream(n, B) for _ in range(P)]
    for r in range(P):
        S.spccl_compress(dev[r], msgs[r], ws)
    out = torch.empty(P * n, dtype=torch.bfloat16, device="cuda")
    pici = lambda t: S.operand(t, S.SPCCL_STREAM, S.SPCCL_FMT_PICI)
    ops = [("compress_rank", lambda: S.spccl_compress(dev[0], msgs[0], ws)),
           ("gather_expand_8", lambda: S.spccl_gather_expand([pici(m) for m in msgs], n, B, out, ws))]
    for _, f in ops:
        f()
    torch.cuda.synchronize()
    sizes = [S.spccl_read_header(mm)["total_bytes"] for mm in msgs]
    e0, _ = O.compress(parts[0])
    parity = (np.array_equal(msgs[0][:e0.size].cpu().numpy(), e0)
              and np.array_equal(_host(out), np.concatenate(parts)))
    alg = {"compress_rank": 2 * n + sizes[0], "gather_expand_8": sum(sizes) + 2 * P * n}
    res = iso.table(ops, alg)
    del dev, ws, msgs, out
    return res, bool(parity)


def time_collectives(S, torch, with_cfg5=True, reps=3):
    """Whole collectives, wall time per call (each call synchronizes the
    stream itself): the P = 8 x 33,554,432 fp32 reduce-scatter at 0.99, the
    P = 8 x 16,777,216 bf16 all-gather at 0.999, and the all-reduce of the
    8 x 268,435,456 fp32 pruned-gradient-like buffers (64 segments, sparsity
    U[0.5, 0.99], 70% shared positions) -- each in its canonical form (one
    global message per rank and step, decided on the device from the
    headers) and its sliced form (per-slice decisions on the device); and
    the canonical reduce-scatter on one tile per rank (its launch cost)."""
    import workloads as W

    def timed(f, *args, times=reps):
        f(*args)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(times):
            f(*args)
        torch.cuda.synchronize()
        return round((time.perf_counter() - t0) / times * 1e3, 3)

    res = {}
    P, m, F = W.CFG3_P, W.CFG3_N // W.CFG3_P, S.SPCCL_F32
    sends = [torch.from_numpy(W.cfg3_rank(r)).cuda() for r in range(P)]
    outs = [torch.empty(m, dtype=torch.float32, device="cuda") for _ in range(P)]
    sc = torch.empty(S.spccl_vr_scratch_bytes(P, m, F), dtype=torch.uint8, device="cuda")
    res["rs_canonical_ms"] = timed(S.spccl_vr_reduce_scatter, sends, outs, sc)
    del sc
    # the same ring on one tile per rank: its bytes are negligible, so its
    # time per launch is the launch cost of this sequence (the tuner check)
    mt = 4096
    tiny = [torch.from_numpy(W.sparse_array(P * mt, W.nnz_for(P * mt, 990), [3, r, 1, 990])).cuda()
            for r in range(P)]
    touts = [torch.empty(mt, dtype=torch.float32, device="cuda") for _ in range(P)]
    tsc = torch.empty(S.spccl_vr_scratch_bytes(P, mt, F), dtype=torch.uint8, device="cuda")
    res["rs_one_tile_ms"] = timed(S.spccl_vr_reduce_scatter, tiny, touts, tsc, times=20)
    del tiny, touts, tsc
    sc = torch.empty(S.spccl_vr_sliced_scratch_bytes(P, m, F), dtype=torch.uint8, device="cuda")
    res["rs_sliced_ms"] = timed(S.spccl_vr_reduce_scatter_sliced, sends, outs, sc)
    del sc, sends, outs
    torch.cuda.empty_cache()
    P4, n4, B = W.CFG4_P, W.CFG4_N, S.SPCCL_BF16
    parts = [_dev(W.cfg4_rank(r)) for r in range(P4)]
    outs = [torch.empty(P4 * n4, dtype=torch.bfloat16, device="cuda") for _ in range(P4)]
    sc = torch.empty(S.spccl_vr_scratch_bytes(P4, n4, B), dtype=torch.uint8, device="cuda")
    res["ag_canonical_ms"] = timed(S.spccl_vr_all_gather, parts, outs, sc)
    del sc
    sc = torch.empty(S.spccl_vr_sliced_scratch_bytes(P4, n4, B), dtype=torch.uint8, device="cuda")
    res["ag_sliced_ms"] = timed(S.spccl_vr_all_gather_sliced, parts, outs, sc)
    del sc, parts, outs
    torch.cuda.empty_cache()
    if with_cfg5:
        t0 = time.time()
        plan = W.cfg5_plan()
        P5 = W.CFG5_P
        n5 = plan.n
        host = np.empty(n5, dtype=np.float32)
        sends = []
        for r in range(P5):
            W.cfg5_rank(plan, r, host)
            sends.append(torch.from_numpy(host).cuda())
        _log(f"all-reduce inputs generated in {time.time() - t0:.1f}s")
        outs = [torch.empty(n5, dtype=torch.float32, device="cuda") for _ in range(P5)]
        m5 = n5 // P5
        sc = torch.empty(S.spccl_vr_scratch_bytes(P5, m5, F), dtype=torch.uint8, device="cuda")
        res["ar_canonical_ms"] = timed(S.spccl_vr_all_reduce, sends, outs, sc, times=1)
        del sc
        sc = torch.empty(S.spccl_vr_sliced_scratch_bytes(P5, m5, F), dtype=torch.uint8, device="cuda")
        res["ar_sliced_ms"] = timed(S.spccl_vr_all_reduce_sliced, sends, outs, sc, times=1)
        del sc, sends, outs
        torch.cuda.empty_cache()
    return res


def tuner_check(ops_tab, dense_ops, copy_GBs, coll, tolerance=0.25):
    """The threshold model's kernel-cost term against the measured ring: the
    P = 8 x 33,554,432 fp32 reduce-scatter at 0.99 predicted on one GPU with
    free links (algorithmic bytes of every rank at the isolated 256 MiB op
    bandwidths, plus a per-launch cost calibrated on the same ring with one
    tile per rank), next to its measured wall time."""
    import workloads as W
    from paper_2607_04676_amd import tuner
    km = tuner.KernelModel.from_ops(ops_tab, dense_ops, copy_GBs)
    P, m, pol = W.CFG3_P, W.CFG3_N // W.CFG3_P, tuner.Policy()
    one = tuner.vr_rs_time_us(P, 4096, 4, 0.99, pol, km, 0.0)
    launch_us = max(0.0, (coll["rs_one_tile_ms"] * 1e3 - one["bytes_us"]) / one["launches"])
    pred = tuner.vr_rs_time_us(P, m, 4, 0.99, pol, km, launch_us)
    ratio = pred["total_us"] / 1e3 / coll["rs_canonical_ms"]
    return {"predicted_ms": round(pred["total_us"] / 1e3, 3), "measured_ms": coll["rs_canonical_ms"],
            "ratio": round(ratio, 3), "bytes_ms": round(pred["bytes_us"] / 1e3, 3), "launches": pred["launches"],
            "launch_us": round(launch_us, 2), "tolerance": tolerance, "within": abs(ratio - 1.0) <= tolerance}


def time_dense_ops(S, torch, n, reps=10):
    """The dense ops of the ring's dense steps (for the threshold model):
    dense (+) dense -> dense array, and wrapping an array as a dense message
    (a plain copy), each priced by its algorithmic bytes."""
    F = S.SPCCL_F32
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.ones(n, dtype=torch.float32, device="cuda")
    z = torch.empty(n, dtype=torch.float32, device="cuda")
    msg = torch.empty(S.spccl_stream_bound(n, F), dtype=torch.uint8, device="cuda")
    ws = S.alloc_workspace(16, F)
    ops = {"dense_dense": (lambda: S.spccl_reduce(S.operand(x), S.operand(y), S.operand(z), n, F, ws), 3 * n * 4),
           "copy": (lambda: S.spccl_encode_dense(x, msg), 2 * n * 4 + 48)}
    res = {}
    for nm, (f, nbytes) in ops.items():
        for _ in range(3):
            f()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            f()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[nm] = {"ms": round(ms, 5), "algorithmic_bytes": nbytes, "achieved_GBs": round(nbytes / (ms / 1e3) / 1e9, 1)}
    del x, y, z, msg
    torch.cuda.empty_cache()
    return res


def copy_ceiling(torch, n, reps=20):
    """Achievable HBM rate on this device for reference: back-to-back plain
    device copies of n fp32 elements (n*4 bytes read and written each), so
    each copy also pays for the previous one's write-back."""
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    torch.cuda.empty_cache()
    return {"GBs": round(2 * n * 4 / (ms / 1e3) / 1e9, 1), "bytes_per_copy": 2 * n * 4, "ms_per_copy": round(ms, 5),
            "what": "torch device copy of 256 MiB fp32, back to back"}


def cpu_baseline(permille, n):
    """The oracle (single thread, pinned to one core) on the headline
    workload: the step's op sequence (compress, decompress, the three
    reductions, a two-part expansion) on the whole 256 MiB array, timed inside
    the oracle's C library with the monotonic clock; the median of 3
    repetitions."""
    import oracle as O
    import workloads as W
    try:
        os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
    except (AttributeError, OSError):
        pass
    a, b = W.cfg2(permille, 0, n), W.cfg2(permille, 1, n)
    mb, _ = O.compress(b)
    secs = O.time_step(a, mb, reps=3)
    med = float(np.median(secs))
    dense_eq = (1 + 1 + 2 + 2 + 2 + 2) * n * 4
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(dense_eq / med / 1e9, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole {n}-element fp32 array at sigma={permille / 1000}: the step's op sequence "
                      f"(compress, decompress, 3 reductions, 2-part expansion; {dense_eq} dense-equivalent bytes), "
                      f"median of 3 reps ({', '.join(f'{x:.2f}' for x in secs)} s) timed in C, one thread pinned to "
                      f"one core; host cpu {cpu_model}, {os.cpu_count()} logical cpus"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--n", type=int, default=1 << 26)
    ap.add_argument("--permille", type=int, default=990)
    ap.add_argument("--sweep", default="500,900,999", help="other sparsities (permille) to report; '' for none")
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calib", action="store_true", help="also run one large plain copy (counter calibration)")
    ap.add_argument("--iso-reps", type=int, default=30,
                    help="repetitions of each op timed on its own; 0 skips them (profiling runs)")
    ap.add_argument("--no-collectives", dest="collectives", action="store_false",
                    help="skip the whole-collective timings")
    ap.add_argument("--no-allreduce", dest="allreduce", action="store_false",
                    help="skip the 8 x 1 GiB all-reduce (its inputs take about a minute to generate)")
    ap.add_argument("--extras", action="store_true", help="also time the sliced and COO forms and the sweep")
    ap.add_argument("--full-out", default="", help="write the complete record (JSON) to this file")
    ap.add_argument("--profile-bf16", type=int, default=0, metavar="PERMILLE",
                    help="profiling run: only the bf16 ops of the 256 MiB array at this sparsity, three "
                         "calls each (for per-kernel counters), then the parity check; no timing")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build emulates P ranks on one device); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    _ensure_built()
    import torch
    import paper_2607_04676_amd as S

    if args.profile_bf16:
        Rb = Runner(S, torch, args.n * 2, args.profile_bf16, 1, bf16=True)
        names = ("compress", "decompress", "reduce_dense_pici_to_pici", "reduce_dense_pici_to_dense")
        alg = run_once(Rb)
        for _ in range(3):
            for nm, f in Rb.isolated_ops():
                if nm in names:
                    f()
        torch.cuda.synchronize()
        print(json.dumps({"profile": f"bf16 ops, {args.n * 2:,} elements, sigma={args.profile_bf16 / 1000}",
                          "algorithmic_bytes": {k: alg[k] for k in names}, "parity": Rb.check_parity()}))
        return

    torch.cuda.init()
    _log(f"device: {torch.cuda.get_device_name(0)}")
    full = {}
    ops_tab = {}                      # the per-op roofline table: key -> [median us, algorithmic bytes, frac]
    parity = {}

    def put(prefix, table):
        for nm, e in table.items():
            ops_tab[f"{prefix}.{nm}"] = [e["median_us"], e["algorithmic_bytes"], e["frac_of_hbm_peak"]]

    # ---- the headline step --------------------------------------------------
    R = Runner(S, torch, args.n, args.permille, args.copies)
    total_ms, wall, per, dense_eq, dom, dom_ms = time_steps(R, args.steps, args.warmup, args.copies)
    _log(f"timed {args.steps} steps: {total_ms / args.steps:.4f} ms per step")
    alg = R.algorithmic_bytes()
    parity["c2.f32.990"] = R.check_parity()
    calib = R.calibration_copy() if args.calib else None
    ms_per_step = total_ms / args.steps
    value = dense_eq / (total_ms / 1e3) / 1e9
    dgbs = alg[dom] / (dom_ms / 1e3) / 1e9
    roof = {"bound": "hbm", "achieved": round(dgbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dgbs / HBM_PEAK_GBS, 4), "traffic": traffic_for(dom),
            "kernel": SINGLE_KERNEL_OPS[dom], "op": dom, "algorithmic_bytes_per_launch": alg[dom],
            "avg_launch_ms": round(dom_ms, 5)}
    full["step_ops"] = op_table(per, alg)
    full["switch"] = {"sigma0": R.sigma0, "decisions": R.switch_log[-args.steps:]}
    iso = Isolator(torch, args.iso_reps) if args.iso_reps > 0 else None
    if iso:
        t = iso.table(R.isolated_ops(), run_once(R))
        full["isolated.c2.f32.990"] = t
        put("c2.f32.990", t)
    extras = {}
    if args.extras:
        SR = SlicedRunner(R)
        for w in range(2):
            for _, f, _ in SR.ops(w % args.copies):
                f()
        _, _, per_s, _ = run_steps(SR, max(5, args.steps // 3), args.copies, {op[0] for op in SR.ops(0)})
        extras["sliced"] = {"parity": SR.check_parity(), "kernels": op_table(per_s, SR.algorithmic_bytes())}
        del SR
        CR = CooRunner(R)
        for w in range(2):
            for _, f, _ in CR.ops(w % args.copies):
                f()
        _, _, per_c, _ = run_steps(CR, max(5, args.steps // 3), args.copies, {op[0] for op in CR.ops(0)})
        extras["coo"] = {"parity": CR.check_parity(), "kernels": op_table(per_c, CR.algorithmic_bytes())}
        del CR
    del R
    torch.cuda.empty_cache()
    ceiling = copy_ceiling(torch, args.n)

    # ---- the other sparsities and bf16 of the 256 MiB array ------------------
    sweep = {}
    sweep_pm = [int(x) for x in args.sweep.split(",") if x.strip()] if (args.extras or iso) else []
    for pm in sweep_pm:
        if pm != 900 and not args.extras:
            continue
        Rs = Runner(S, torch, args.n, pm, 2)
        t_ms, _, p_s, deq, _, _ = time_steps(Rs, max(5, args.steps // 3), 2, 2)
        ent = {"dense_equiv_GBs": round(deq / (t_ms / 1e3) / 1e9, 1), "kernels": op_table(p_s, Rs.algorithmic_bytes())}
        parity[f"c2.f32.{pm}"] = Rs.check_parity()
        if iso:
            t = iso.table(Rs.isolated_ops(), run_once(Rs))
            ent["isolated"] = t
            put(f"c2.f32.{pm}", t)
        sweep[str(pm / 1000)] = ent
        del Rs
        torch.cuda.empty_cache()
    if iso:
        for pm in (990, 900):
            Rb = Runner(S, torch, args.n * 2, pm, 1, bf16=True)
            t = iso.table([op for op in Rb.isolated_ops() if op[0] in ("compress", "decompress",
                                                                       "reduce_dense_pici_to_pici",
                                                                       "reduce_dense_pici_to_dense")],
                          run_once(Rb))
            full[f"isolated.c2.bf16.{pm}"] = t
            put(f"c2.bf16.{pm}", t)
            if pm == 990:
                parity["c2.bf16.990"] = Rb.check_parity()
            del Rb
            torch.cuda.empty_cache()
        _log("timing the 1,048,576-element pair")
        t, parity["c1"] = time_cfg1(S, torch, iso)
        full["isolated.c1"] = t
        put("c1", t)
        _log("timing the reduce-scatter ring steps")
        t, parity["c3.steps"] = time_cfg3_steps(S, torch, iso)
        full["isolated.c3"] = t
        put("c3", t)
        _log("timing the all-gather parts")
        t, parity["c4"] = time_cfg4_ops(S, torch, iso)
        full["isolated.c4"] = t
        put("c4", t)
        torch.cuda.empty_cache()
    if args.collectives:
        _log("timing the collectives")
    collectives = time_collectives(S, torch, args.allreduce) if args.collectives else None
    dense_ops = time_dense_ops(S, torch, args.n)
    cpu = None
    if not args.no_cpu:
        _log("timing the CPU oracle")
        cpu = cpu_baseline(args.permille, args.n)
    check = None
    if iso and collectives:
        check = tuner_check(ops_tab, dense_ops, ceiling["GBs"], collectives)
    if iso:
        roof["ops"] = ops_tab
        roof["ops_key"] = ("config.dtype.sparsity(permille).op -> [isolated median us, algorithmic bytes, "
                           "fraction of 8 TB/s]; c1 = 1,048,576 fp32 pair, c2 = 256 MiB array, c3.stepS = "
                           "reduce-scatter ring step S on one 4,194,304-element chunk, c4 = bf16 all-gather parts")
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"codec sweep array: {args.n:,} fp32 elements ({args.n * 4 >> 20} MiB), "
                               f"sigma={args.permille / 1000}, uniform random nonzero positions, N(0,1) values; "
                               "step = compress, send, decompress, 3 reductions, gather-expand, adaptive switch",
                   "n": args.n, "sigma": args.permille / 1000, "parallelism": "1 GPU (virtual ranks)"},
        "roofline": roof, "cpu_baseline": cpu, "copy_ceiling_GBs": ceiling["GBs"], "collectives_ms": collectives,
        "parity_vs_oracle": parity, "wall_s_timed": round(wall, 3), "calibration_copy_bytes": calib,
        "tuner_check": check,
    }
    full.update({"line": out, "copy_ceiling": ceiling, "dense_ops": dense_ops, "sweep": sweep, **extras,
                 "kernels": full["step_ops"]})
    if sweep and args.extras:
        # thresholds for this machine from the modelled sweep (Sec. IV-C),
        # with the kernel costs just measured
        from paper_2607_04676_amd import tuner
        rec = dict(full)
        rec["config"] = out["config"]
        res = tuner.recommend(tuner.KernelModel.from_bench(rec))
        full["thresholds"] = {k: res[k] for k in res if k != "table"}
    if args.full_out:
        with open(args.full_out, "w") as f:
            json.dump(full, f, indent=1)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
