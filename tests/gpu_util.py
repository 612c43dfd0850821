"""Helpers shared by the GPU parity tests (not collected as tests)."""
import sys

import numpy as np
import pytest
import torch


def announce(msg: str):
    """Name the case before any GPU work, so a failure that ends the run is attributable."""
    sys.stdout.write(f"[gpu-case] {msg}\n")
    sys.stdout.flush()


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")


def u16(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def u8(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().view(torch.uint8).cpu().numpy()


def f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().contiguous().cpu().numpy().astype(np.float32)


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def assert_codes_equal(got: np.ndarray, want: np.ndarray, what: str):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        idx = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} mismatches; first at {idx}: "
                             f"got {got[idx]!r} want {want[idx]!r}")


def assert_scales_equal(got: np.ndarray, want: np.ndarray, what: str):
    assert_codes_equal(np.ascontiguousarray(got).view(np.uint32), np.ascontiguousarray(want).view(np.uint32),
                       what + " (scale bits)")
