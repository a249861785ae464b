"""Shared helpers of the GPU tests: host <-> device transfer of the seeded
inputs and byte-level comparison against the oracle."""
import os
import sys
import time

import numpy as np


# a folder for a progress log (SPCCL_PROGRESS_DIR; none by default)
_PROGRESS = os.environ.get("SPCCL_PROGRESS_DIR", "")


def log(msg: str) -> None:
    """Name the case before a GPU step (flushed, so it survives a crash); the
    line also goes to progress.log in SPCCL_PROGRESS_DIR when that is set, so a
    long test shows progress while pytest captures its output."""
    line = f"[gpu-case] {time.strftime('%H:%M:%S')} {msg}"
    print(line, file=sys.stderr, flush=True)
    if _PROGRESS and os.path.isdir(_PROGRESS):
        with open(os.path.join(_PROGRESS, "progress.log"), "a") as f:
            f.write(line + "\n")


def to_dev(arr: np.ndarray):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def to_host_bits(t) -> np.ndarray:
    """Raw bit patterns of a device tensor (uint32 for fp32, uint16 for bf16, uint8 for bytes)."""
    import torch
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    if t.dtype == torch.float32:
        return t.cpu().numpy().view(np.uint32)
    return t.cpu().numpy()


def bits(arr: np.ndarray) -> np.ndarray:
    return arr.view(np.uint16) if arr.dtype == np.uint16 else arr.view(np.uint32)


def assert_bytes_equal(got: np.ndarray, exp: np.ndarray, what: str) -> None:
    if got.shape == exp.shape and np.array_equal(got, exp):
        return
    n = min(got.size, exp.size)
    diff = np.flatnonzero(got[:n] != exp[:n])
    first = int(diff[0]) if diff.size else n
    raise AssertionError(f"{what}: sizes {got.size} vs {exp.size}, {diff.size} differing bytes, first at {first}")


def first_diff(got: np.ndarray, exp: np.ndarray) -> str:
    d = np.flatnonzero(got != exp)
    if d.size == 0:
        return "equal"
    i = int(d[0])
    return f"{d.size} differ, first at {i}: got {got[i]:#x} expected {exp[i]:#x}"
