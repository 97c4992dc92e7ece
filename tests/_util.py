"""Helpers shared by the tests: moving generator arrays to and from the GPU,
oracle-side conversions and the tolerance checks."""

import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def ensure_built():
    """Build libpolestar.so only when it is missing."""
    from paper_2607_14107_amd import build, polestar
    if not os.path.exists(polestar.LIB_PATH):
        build.build(verbose=False)
    return polestar.lib()


def to_dev(x: np.ndarray, dtype: str):
    """A generator array (bf16 bits or fp32) -> GPU tensor of the run dtype."""
    import torch
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint16).view(np.int16))
        return t.view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def from_dev(t) -> np.ndarray:
    """GPU tensor -> numpy (bf16 as uint16 bits)."""
    import torch
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def bits_of(values: np.ndarray, dtype: str) -> np.ndarray:
    """float64 values exactly representable in the run dtype -> stored array."""
    v = np.asarray(values, dtype=np.float64).astype(np.float32)
    if dtype == "bf16":
        u = v.view(np.uint32)
        assert np.all((u & 0xFFFF) == 0), "value not representable in bf16"
        return (u >> 16).astype(np.uint16)
    return v


RTOL = {"fp32": 1e-4, "bf16": 2e-2}


def assert_rows_close(got: np.ndarray, want: np.ndarray, rtol: float, what: str):
    """Row-normwise check over the last axis: max|g - o| <= rtol * max|o|."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    err = np.abs(got - want).max(axis=-1)
    scale = np.abs(want).max(axis=-1)
    bad = err > rtol * scale
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} rows off, first {tuple(idx)}: "
                             f"err {err[tuple(idx)]:.3e} vs scale {scale[tuple(idx)]:.3e}")


def assert_drift_close(got: np.ndarray, want: np.ndarray, rtol: float = 1e-4, floor: float = 1e-7):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    tol = np.maximum(rtol * np.abs(want), rtol * floor)
    err = np.abs(got - want)
    small = np.abs(want) < floor
    ok = np.where(small, err <= floor, err <= tol)
    if not ok.all():
        i = np.argwhere(~ok)[0]
        raise AssertionError(f"drift off at {tuple(i)}: got {got[tuple(i)]:.9e} want {want[tuple(i)]:.9e} "
                             f"({(~ok).sum()} entries; max rel {np.max(err / np.maximum(np.abs(want), floor)):.2e})")
