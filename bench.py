"""Throughput of the Pici hot path on one MI355X.

Workload: the codec sweep array -- 67,108,864 fp32 elements (256 MiB) with
uniformly random nonzero positions and N(0,1) values -- at sparsity 99% (the
headline), with 50 / 90 / 99.9% reported as a sweep.  Inputs are resident in
HBM before timing; four copies of each operand rotate between steps so the
256 MB Infinity Cache cannot serve a step's dense input.

One step is one pass of the whole hot path over one batch:
  compress(a)                     dense -> Pici (count pass, then place pass)
  send                            device-sized copy of the message
  decompress(received)            Pici -> dense
  reduce a (+) Pici(b) -> Pici    fused reduce-scatter step with fill-in
  reduce Pici(a) (+) Pici(b) -> Pici
  reduce a (+) Pici(b) -> dense   last reduce-scatter step
  gather_expand of the two        all-gather receive side
  adaptive switch                 the fused step's header (nonzero count) is
                                  copied to pinned host memory as soon as that
                                  reduce ends (op "switch_header"); the host
                                  waits for that copy only, then applies Eq. 7
                                  against the 0.6 threshold while the GPU runs
                                  the rest

value = dense-equivalent bytes of the step (N*s per codec op, 2*N*s per
reduce, P*N*s per gather) / step time over K timed steps.  Inside the timed
region only the roofline kernel's op is bracketed by HIP events (each event
pair costs the stream a few microseconds).  A separate pass of the same steps,
before the timed region, brackets every op with events for the per-op table
("kernels"), each priced by its algorithmic bytes (dense bytes read or written
plus message bytes read or written) against 8 TB/s.  With a full workspace
the Pici-producing ops launch two kernels (count pass, place pass); the
roofline entry is the single-kernel op with the largest time share, so its
event time is one kernel's duration and matches the rocprofv3 summary.

Each op is also timed on its own ("isolated": median, min and max over 50
repetitions, each after 512 MiB of scratch writes), at the headline sparsity,
in the sliced form and at each swept sparsity.

Reported beside the step (not part of value): the same ops in the
in-collective sliced form ("sliced") and in COO ("coo"), per op; the dense
ops of dense ring steps ("dense_ops"); the emulated reduce-scatter of the
P = 8 x 33,554,432 workload in its canonical and device-decided sliced forms
("collectives"); and the thresholds the modelled sweep picks for this GPU
from the kernel costs just measured ("thresholds").
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


class Runner:
    """Device buffers and the per-op launch closures for one sparsity."""

    def __init__(self, S, torch, n, permille, copies):
        import workloads as W
        self.S, self.torch, self.n = S, torch, n
        dt = S.SPCCL_F32
        self.s = 4
        t0 = time.time()
        a = W.cfg2(permille, 0, n)
        b = W.cfg2(permille, 1, n)
        self.host_a, self.host_b = a, b
        _log(f"generated sigma={permille / 1000} inputs in {time.time() - t0:.1f}s")
        dev = "cuda"
        ta, tb = torch.from_numpy(a).to(dev), torch.from_numpy(b).to(dev)
        self.a = [ta] + [ta.clone() for _ in range(copies - 1)]
        self.b = [tb] + [tb.clone() for _ in range(copies - 1)]
        self.ws = S.alloc_workspace(n, dt, dev)
        bound = S.spccl_stream_bound(n, dt)
        mk = lambda: torch.empty(bound, dtype=torch.uint8, device=dev)
        self.msg_b = [mk() for _ in range(copies)]
        for k in range(copies):
            S.spccl_compress(self.b[k], self.msg_b[k], self.ws)
        self.msg_a, self.recv, self.red_p, self.red_pp = mk(), mk(), mk(), mk()
        self.dense_out = torch.empty(n, dtype=torch.float32, device=dev)
        self.red_d = torch.empty(n, dtype=torch.float32, device=dev)
        self.gather_out = torch.empty(2 * n, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        hb = S.spccl_read_header(self.msg_b[0])
        self.nnz_b, self.bytes_b = hb["nnz"], hb["total_bytes"]
        self.sigma0 = None
        self.hdr_host = torch.empty(48, dtype=torch.uint8, pin_memory=True)
        self.hdr_ev = torch.cuda.Event()

    def ops(self, k):
        """(name, launch, dense-equivalent bytes) of one step on copy k."""
        S, n, s = self.S, self.n, self.s
        a, b, mb, ws = self.a[k], self.b[k], self.msg_b[k], self.ws
        F, P, D, A = S.SPCCL_F32, S.SPCCL_FMT_PICI, S.SPCCL_FMT_DENSE, S.SPCCL_STREAM
        msg = lambda t, f=P: S.operand(t, A, f)
        return [
            ("compress", lambda: S.spccl_compress(a, self.msg_a, ws), n * s),
            ("send", lambda: S.spccl_copy_message(self.msg_a, self.recv, ws), 0),
            ("decompress", lambda: S.spccl_decompress(self.recv, self.dense_out, ws), n * s),
            ("reduce_dense_pici_to_pici", lambda: S.spccl_reduce(S.operand(a), msg(mb), msg(self.red_p), n, F, ws),
             2 * n * s),
            ("switch_header", self.fetch_header, 0),
            ("reduce_pici_pici_to_pici", lambda: S.spccl_reduce(msg(self.msg_a), msg(mb), msg(self.red_pp), n, F, ws),
             2 * n * s),
            ("reduce_dense_pici_to_dense", lambda: S.spccl_reduce(S.operand(a), msg(mb), S.operand(self.red_d), n,
                                                                  F, ws), 2 * n * s),
            ("gather_expand", lambda: S.spccl_gather_expand([msg(self.recv), msg(self.red_p)], n, F,
                                                            self.gather_out, ws), 2 * n * s),
        ]

    def fetch_header(self):
        """Queue the copy of the fused step's 48-byte header to pinned host
        memory right behind the reduce that writes it."""
        self.hdr_host.copy_(self.red_p[:48], non_blocking=True)
        self.hdr_ev.record()

    def decide(self):
        """Adaptive switch for the next send (Sec. IV-C): measured sparsity of
        the fused step's output against the extrapolation rule.  Waits for the
        header copy only, not for the ops queued after it."""
        self.hdr_ev.synchronize()
        h = self.hdr_host.numpy()
        assert int(h[:4].view(np.uint32)[0]) == 0x49434950 and int(h[4:6].view(np.uint16)[0]) == 1
        nnz = int(h[16:24].view(np.uint64)[0])
        sigma = (self.n - nnz) / self.n
        if self.sigma0 is None:
            self.sigma0 = sigma
        return sigma * self.sigma0 <= 0.6

    def algorithmic_bytes(self):
        """Bytes each kernel must move at minimum (reads + writes), per launch."""
        S, n, s = self.S, self.n, self.s
        torch = self.torch
        torch.cuda.synchronize()
        ba = S.spccl_read_header(self.msg_a)["total_bytes"]
        bp = S.spccl_read_header(self.red_p)["total_bytes"]
        bpp = S.spccl_read_header(self.red_pp)["total_bytes"]
        bb = self.bytes_b
        return {
            "compress": n * s + ba,
            "send": 2 * ba,
            "decompress": ba + n * s,
            "reduce_dense_pici_to_pici": n * s + bb + bp,
            "reduce_pici_pici_to_pici": ba + bb + bpp,
            "reduce_dense_pici_to_dense": n * s + bb + n * s,
            "gather_expand": ba + bp + 2 * n * s,
            "switch_header": 48,
        }

    def calibration_copy(self):
        """One large plain copy of known size (a dense message of the input:
        48 + N*s bytes read and written) for scaling HBM byte counters."""
        S, torch = self.S, self.torch
        big = torch.empty(S.spccl_stream_bound(self.n, S.SPCCL_F32), dtype=torch.uint8, device="cuda")
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
        self.slot = S.spccl_slice_bytes(S.SPCCL_F32)
        self.nslices = S.spccl_slice_count(R.n)
        mk = lambda: S.alloc_sliced(R.n, S.SPCCL_F32)
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
            ("send_sliced", lambda: S.spccl_copy_sliced(self.sa, self.recv, n, S.SPCCL_F32, ws), 0),
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
        F = S.SPCCL_F32
        mk = lambda: S.alloc_stream(R.n, F, fmt=S.SPCCL_FMT_COO)
        self.cb = [mk() for _ in R.b]
        for k, b in enumerate(R.b):
            S.spccl_compress_coo(b, self.cb[k], R.ws)
        self.ca, self.recv, self.red = mk(), mk(), mk()
        torch.cuda.synchronize()

    def ops(self, k):
        S, R, n, s = self.S, self.R, self.n, self.R.s
        a, cb, ws = R.a[k], self.cb[k], R.ws
        F, C = S.SPCCL_F32, S.SPCCL_FMT_COO
        msg = lambda t: S.operand(t, S.SPCCL_STREAM, C)
        return [
            ("compress_coo", lambda: S.spccl_compress_coo(a, self.ca, ws), n * s),
            ("send_coo", lambda: S.spccl_copy_message(self.ca, self.recv, ws), 0),
            ("decompress_coo", lambda: S.spccl_decompress(self.recv, R.dense_out, ws), n * s),
            ("reduce_dense_coo_to_coo", lambda: S.spccl_reduce(S.operand(a), msg(cb), msg(self.red), n, F, ws),
             2 * n * s),
            ("reduce_dense_coo_to_dense", lambda: S.spccl_reduce(S.operand(a), msg(cb), S.operand(R.red_d), n, F, ws),
             2 * n * s),
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
    ev = {nm: [] for nm in bracket}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start_all = torch.cuda.Event(enable_timing=True)
    end_all = torch.cuda.Event(enable_timing=True)
    start_all.record()
    dense_eq = 0
    for k in range(steps):
        for nm, f, deq in R.ops(k % copies):
            if nm in ev:
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                f()
                e1.record()
                ev[nm].append((e0, e1))
            else:
                f()
            dense_eq += deq
        R.decide()
    end_all.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = start_all.elapsed_time(end_all)
    per = {nm: float(np.mean([a.elapsed_time(b) for a, b in ev[nm]])) for nm in bracket}
    st = R.S.spccl_read_status(R.ws)
    if st != 0:
        raise RuntimeError(f"device status {st} after timing")
    return total_ms, wall, per, dense_eq


def time_steps(R, steps, warmup, copies):
    """Warm-up, a per-op breakdown pass (every op bracketed), then the timed
    steps with only the roofline op bracketed.  Returns (total ms, wall s,
    per-op ms from the breakdown, dense-equivalent bytes, roofline op, its ms
    in the timed region)."""
    names = [op[0] for op in R.ops(0)]
    for w in range(warmup):
        for _, f, _ in R.ops(w % copies):
            f()
        R.decide()
    _, _, per, _ = run_steps(R, max(3, steps // 3), copies, names)
    dom = max((k for k in per if k in SINGLE_KERNEL_OPS), key=lambda k: per[k])
    total_ms, wall, timed, dense_eq = run_steps(R, steps, copies, [dom])
    return total_ms, wall, per, dense_eq, dom, timed[dom]


def time_isolated(R, reps=50, warm=5):
    """Each op of a runner on its own: before every repetition 512 MiB of
    scratch is written (untimed), so neither the Infinity Cache nor the L2
    holds the op's operands and the op pays for that write-back as a cold
    launch would; the op is bracketed by HIP events.  Median, min and max
    over reps, in microseconds, and the median's fraction of 8 TB/s by
    algorithmic bytes."""
    torch = R.torch
    junk = torch.empty(1 << 27, dtype=torch.float32, device="cuda")
    alg = R.algorithmic_bytes()
    res = {}
    for nm, f, _ in R.ops(0):
        if nm == "switch_header":
            continue
        ts = []
        for r in range(warm + reps):
            junk.fill_(float(r))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            f()
            e1.record()
            e1.synchronize()
            if r >= warm:
                ts.append(e0.elapsed_time(e1) * 1e3)
        med = float(np.median(ts))
        res[nm] = {"median_us": round(med, 2), "min_us": round(min(ts), 2), "max_us": round(max(ts), 2),
                   "reps": reps, "algorithmic_bytes": alg[nm],
                   "frac_of_hbm_peak": round(alg[nm] / (med * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    del junk
    return res


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


def time_collectives(S, torch, reps=3):
    """The emulated reduce-scatter of the P = 8 x 33,554,432 fp32 workload at
    99%: the canonical ring (one global message per step, the host reads the
    step's headers to decide) and the sliced ring (per-slice decisions on
    the device, one synchronisation at the end); and the all-gather of the
    P = 8 x 16,777,216 bf16 workload at 99.9% in both forms.  Wall time per
    collective, each call synchronizing the stream itself."""
    import workloads as W
    P, m = W.CFG3_P, W.CFG3_N // W.CFG3_P
    F = S.SPCCL_F32
    sends = [torch.from_numpy(W.cfg3_rank(r)).cuda() for r in range(P)]
    outs = [torch.empty(m, dtype=torch.float32, device="cuda") for _ in range(P)]
    res = {"workload": f"reduce-scatter, P = {P} x {W.CFG3_N:,} fp32, sigma = 0.99"}
    runs = {
        "canonical_ring_ms": (torch.empty(S.spccl_vr_scratch_bytes(P, m, F), dtype=torch.uint8, device="cuda"),
                              S.spccl_vr_reduce_scatter),
        "sliced_ring_device_decisions_ms": (torch.empty(S.spccl_vr_sliced_scratch_bytes(P, m, F), dtype=torch.uint8,
                                                        device="cuda"), S.spccl_vr_reduce_scatter_sliced),
    }
    def timed(f, *args):
        f(*args)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            f(*args)
        torch.cuda.synchronize()
        return round((time.perf_counter() - t0) / reps * 1e3, 3)

    for nm, (scratch, f) in runs.items():
        res[nm] = timed(f, sends, outs, scratch)
        del scratch
    del sends, outs
    torch.cuda.empty_cache()
    # the all-gather workload: P = 8 x 16,777,216 bf16 at 99.9%
    P4, n4, B = W.CFG4_P, W.CFG4_N, S.SPCCL_BF16
    parts = [torch.from_numpy(W.cfg4_rank(r).view(np.int16)).cuda().view(torch.bfloat16) for r in range(P4)]
    outs = [torch.empty(P4 * n4, dtype=torch.bfloat16, device="cuda") for _ in range(P4)]
    ag = {"workload": f"all-gather, P = {P4} x {n4:,} bf16, sigma = 0.999"}
    scratch = torch.empty(S.spccl_vr_scratch_bytes(P4, n4, B), dtype=torch.uint8, device="cuda")
    ag["canonical_ring_ms"] = timed(S.spccl_vr_all_gather, parts, outs, scratch)
    del scratch
    scratch = torch.empty(S.spccl_vr_sliced_scratch_bytes(P4, n4, B), dtype=torch.uint8, device="cuda")
    ag["sliced_ring_ms"] = timed(S.spccl_vr_all_gather_sliced, parts, outs, scratch)
    del scratch, parts, outs
    torch.cuda.empty_cache()
    res["all_gather"] = ag
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


def cpu_baseline(permille, n_full, budget_s):
    """The oracle (single thread, pinned to one core) on a bounded sample of
    the same workload: the same op sequence on the first n_sample elements."""
    import oracle as O
    import workloads as W
    try:
        os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
    except (AttributeError, OSError):
        pass
    n = n_full // 16
    a = W.cfg2(permille, 0, n_full)[:n].copy()
    b = W.cfg2(permille, 1, n_full)[:n].copy()
    s = 4
    mb, _ = O.compress(b)
    done_bytes, t_total, reps = 0, 0.0, 0
    while t_total < budget_s and reps < 50:
        t0 = time.perf_counter()
        ma, _ = O.compress(a)
        back = O.decompress(ma, n, O.F32)
        O.reduce(O.Operand.array(a), O.Operand.stream(mb), n, O.F32, O.STREAM, O.FMT_PICI)
        O.reduce(O.Operand.stream(ma), O.Operand.stream(mb), n, O.F32, O.STREAM, O.FMT_PICI)
        O.reduce(O.Operand.array(a), O.Operand.stream(mb), n, O.F32)
        O.decompress(ma, n, O.F32)
        O.decompress(mb, n, O.F32)
        t_total += time.perf_counter() - t0
        done_bytes += (2 + 3 * 2 + 2) * n * s
        reps += 1
        assert np.array_equal(back.view(np.uint32), a.view(np.uint32))
    cpu_model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": done_bytes / t_total / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"first {n} of {n_full} elements (1/16) at sigma={permille / 1000}, the step's op sequence "
                      f"x{reps} in {t_total:.1f} s, single thread pinned to one core; host cpu: {cpu_model}, "
                      f"{os.cpu_count()} logical cpus"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--n", type=int, default=1 << 26)
    ap.add_argument("--permille", type=int, default=990)
    ap.add_argument("--sweep", default="500,900,999", help="other sparsities (permille) to report; '' for none")
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--calib", action="store_true", help="also run one large plain copy (counter calibration)")
    ap.add_argument("--iso-reps", type=int, default=50,
                    help="repetitions of each op timed on its own; 0 skips them (profiling runs)")
    ap.add_argument("--no-collectives", dest="collectives", action="store_false",
                    help="skip timing the emulated reduce-scatter collectives")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (this build emulates P ranks on one device); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    _ensure_built()
    import torch
    import paper_2607_04676_amd as S

    torch.cuda.init()
    _log(f"device: {torch.cuda.get_device_name(0)}")
    R = Runner(S, torch, args.n, args.permille, args.copies)
    total_ms, wall, per, dense_eq, dom, dom_ms = time_steps(R, args.steps, args.warmup, args.copies)
    alg = R.algorithmic_bytes()
    parity = R.check_parity()
    calib = R.calibration_copy() if args.calib else None
    ms_per_step = total_ms / args.steps
    value = dense_eq / (total_ms / 1e3) / 1e9
    kernels = {}
    for nm, ms in per.items():
        gbs = alg[nm] / (ms / 1e3) / 1e9
        kernels[nm] = {"ms": round(ms, 5), "algorithmic_bytes": alg[nm], "achieved_GBs": round(gbs, 1),
                       "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
    # the roofline entry is the single-kernel op with the largest share of the
    # step, so its event time is one kernel's duration (the Pici-producing ops
    # launch a count pass and a place pass and are reported under "kernels");
    # its duration is the mean over the timed steps
    dgbs = alg[dom] / (dom_ms / 1e3) / 1e9
    roof = {"bound": "hbm", "kernel": SINGLE_KERNEL_OPS[dom], "op": dom, "achieved": round(dgbs, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(dgbs / HBM_PEAK_GBS, 4),
            "traffic": traffic_for(dom),
            "algorithmic_bytes_per_launch": alg[dom], "avg_launch_ms": round(dom_ms, 5)}
    isolated = time_isolated(R, args.iso_reps) if args.iso_reps > 0 else None
    # the in-collective (sliced) form of the codec and reduce ops, per op
    SR = SlicedRunner(R)
    for w in range(2):
        for _, f, _ in SR.ops(w % args.copies):
            f()
    _, _, per_s, _ = run_steps(SR, max(5, args.steps // 3), args.copies, [op[0] for op in SR.ops(0)])
    alg_s = SR.algorithmic_bytes()
    sliced = {"slice_elems": 16384, "dense_thresh": SR.thresh, "parity_compress_vs_oracle": SR.check_parity(),
              "kernels": {}, "isolated": time_isolated(SR, args.iso_reps) if args.iso_reps > 0 else None}
    for nm, ms in per_s.items():
        gbs = alg_s[nm] / (ms / 1e3) / 1e9
        sliced["kernels"][nm] = {"ms": round(ms, 5), "algorithmic_bytes": alg_s[nm], "achieved_GBs": round(gbs, 1),
                                 "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
    del SR
    # the COO form of the codec and reduce ops
    CR = CooRunner(R)
    for w in range(2):
        for _, f, _ in CR.ops(w % args.copies):
            f()
    _, _, per_c, _ = run_steps(CR, max(5, args.steps // 3), args.copies, [op[0] for op in CR.ops(0)])
    alg_c = CR.algorithmic_bytes()
    coo = {"parity_compress_vs_oracle": CR.check_parity(), "kernels": {}}
    for nm, ms in per_c.items():
        gbs = alg_c[nm] / (ms / 1e3) / 1e9
        coo["kernels"][nm] = {"ms": round(ms, 5), "algorithmic_bytes": alg_c[nm], "achieved_GBs": round(gbs, 1),
                              "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)}
    del CR
    sweep = {}
    del R
    torch.cuda.empty_cache()
    ceiling = copy_ceiling(torch, args.n)
    for pm in [int(x) for x in args.sweep.split(",") if x.strip()]:
        Rs = Runner(S, torch, args.n, pm, args.copies)
        t_ms, _, p_s, deq, _, _ = time_steps(Rs, max(5, args.steps // 3), 2, args.copies)
        a_s = Rs.algorithmic_bytes()
        sweep[str(pm / 1000)] = {
            "dense_equiv_GBs": round(deq / (t_ms / 1e3) / 1e9, 1),
            "kernels": {nm: {"ms": round(ms, 5), "algorithmic_bytes": a_s[nm],
                             "frac_of_hbm_peak": round(a_s[nm] / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4)}
                        for nm, ms in p_s.items()},
            "parity_compress": Rs.check_parity(),
            "isolated": time_isolated(Rs, args.iso_reps) if args.iso_reps > 0 else None,
        }
        del Rs
        torch.cuda.empty_cache()
    dense_ops = time_dense_ops(S, torch, args.n)
    collectives = time_collectives(S, torch) if args.collectives else None
    cpu = None
    if not args.no_cpu:
        _log("timing the CPU oracle")
        cpu = cpu_baseline(args.permille, args.n, args.cpu_budget)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"codec sweep array: {args.n:,} fp32 elements ({args.n * 4 >> 20} MiB), "
                               f"sigma={args.permille / 1000}, uniform random nonzero positions, N(0,1) values; "
                               "step = compress, send, decompress, 3 reduce variants, gather-expand, adaptive switch",
                   "n": args.n, "sigma": args.permille / 1000, "parallelism": "1 GPU (virtual ranks)"},
        "roofline": roof, "cpu_baseline": cpu, "copy_ceiling": ceiling, "kernels": kernels, "isolated": isolated,
        "sliced": sliced,
        "coo": coo, "sweep": sweep, "dense_ops": dense_ops, "collectives": collectives,
        "parity_compress_vs_oracle": parity, "wall_s_timed": round(wall, 3),
        "calibration_copy_bytes": calib,
    }
    if sweep:
        # thresholds for this machine from the modelled sweep (Sec. IV-C),
        # with the kernel costs just measured
        from paper_2607_04676_amd import tuner
        rec = tuner.recommend(tuner.KernelModel.from_bench(out))
        out["thresholds"] = {k: rec[k] for k in ("intra_thresh", "inter_thresh", "ag_thresh",
                                                  "geomean_slowdown_vs_best", "paper_pair_geomean_slowdown")}
    print(json.dumps(out))


if __name__ == "__main__":
    main()
