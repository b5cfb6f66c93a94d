"""Helpers for the GPU parity tests: device transfer of uint64 residue arrays
(stored in int64 tensors) and a flushed progress line before each GPU step."""
import sys

import numpy as np
import pytest
import torch


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def to_dev(a: np.ndarray) -> torch.Tensor:
    a = np.ascontiguousarray(a, dtype=np.uint64)
    return torch.from_numpy(a.view(np.int64)).cuda()


def to_host(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.cpu().numpy().view(np.uint64)


def step(msg: str):
    print(f"[gpu-step] {msg}", flush=True)
    sys.stdout.flush()


def first_mismatch(got: np.ndarray, want: np.ndarray) -> str:
    bad = np.argwhere(got != want)
    if len(bad) == 0:
        return "equal"
    i = tuple(bad[0])
    return f"{len(bad)} mismatches, first at {i}: got {got[i]} want {want[i]}"
