"""Shared helpers for the GPU parity tests: device copies of seeded inputs, oracle
inputs from the same draws, and the tolerance checks.

Tolerances (written here once, used by every parity test):
  level map            bit-exact
  forward, fp32        |gpu - ref| <= 1e-6 + 1e-5 |ref|  elementwise
  backward, fp32       |gpu - ref| <= 1e-4 * S  elementwise, S = A^T|g| (the sum of the
                       absolute contributions, from the oracle), and
                       ||gpu - ref||_2 <= 1e-4 ||ref||_2
  bf16 inputs          forward |gpu - ref| <= 1e-2 |ref| + 1e-4; backward as fp32 with 1e-2
"""
from __future__ import annotations

import sys

import numpy as np

import oracle
from paper_1906_07155_amd import workloads as W

FWD_F32 = (1e-6, 1e-5)
BWD_F32 = 1e-4
FWD_BF16 = (1e-4, 1e-2)
BWD_BF16 = 1e-2


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    return torch


def to_device(arr: np.ndarray, dtype: str, layout: str = "cl"):
    """NCHW numpy array (float32, or uint16 bf16 bits) -> device tensor."""
    torch = torch_mod()
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).cuda().view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()
    if layout == "cl":
        t = t.contiguous(memory_format=torch.channels_last)
    return t


def as_f64(arr: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return W.bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


def from_device(t) -> np.ndarray:
    torch = torch_mod()
    if t.dtype == torch.bfloat16:
        return W.bf16_bits_to_f32(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                                  ).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def check_fwd(got: np.ndarray, ref: np.ndarray, bf16: bool, what: str) -> float:
    atol, rtol = FWD_BF16 if bf16 else FWD_F32
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if got.size == 0:
        return 0.0
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    assert not bad.any(), "%s: %d elements out of tolerance, worst %g at %s (got %g ref %g)" % (
        what, int(bad.sum()), float(err.max()), np.unravel_index(int(err.argmax()), err.shape),
        float(got.flat[int(err.argmax())]), float(ref.flat[int(err.argmax())]))
    return float(err.max())


def check_bwd(got: np.ndarray, ref: np.ndarray, absref: np.ndarray, bf16: bool,
              what: str) -> float:
    tol = BWD_BF16 if bf16 else BWD_F32
    err = np.abs(got - ref)
    bad = err > tol * absref + 1e-30
    assert not bad.any(), "%s: %d elements out of tolerance, worst excess %g" % (
        what, int(bad.sum()), float((err - tol * absref).max()))
    nref = np.linalg.norm(ref)
    assert np.linalg.norm(got - ref) <= tol * max(nref, 1e-30), what + " normwise"
    return float(np.linalg.norm(got - ref) / max(nref, 1e-30))


class Case:
    """Device and oracle views of one seeded workload."""

    def __init__(self, wl: W.Workload, layout: str = "cl", feats=None, rois=None):
        torch = torch_mod()
        self.wl = wl
        self.feats_np = feats if feats is not None else wl.features()
        self.rois = rois if rois is not None else wl.rois()
        self.K = self.rois.shape[0]
        self.shapes = [f.shape for f in self.feats_np]
        self.scales = list(wl.scales)
        self.feats = [to_device(f, wl.feat_dtype, layout) for f in self.feats_np]
        self.rois_dev = torch.from_numpy(self.rois).cuda()
        self.bf16 = wl.feat_dtype == "bf16"

    def oracle_levels(self) -> np.ndarray:
        return oracle.level_map(self.rois, len(self.shapes), self.wl.finest_scale)
