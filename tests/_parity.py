"""Helpers for the GPU parity tests: upload seeded inputs, run the library,
run the oracle, and compare with the tolerances of the correctness bar.

Bar (per the benchmark spec's tolerance, staged as below):
  * ternary codes / packed words and integer sums: bit-exact;
  * quantised activations: at most 1 LSB apart in at most 0.1% of entries
    (both sides take the rounding decision in fp32 from an fp64 row sum, so 0
    differences are expected);
  * a_scale, w_scale: within 1e-6 relative (bit-exact expected);
  * y: rows whose q match exactly: |dy| <= 1e-3 |y_ref| per element, and
    y == 0 exactly where the integer sum is 0; rows with LSB flips:
    max|dy| <= 1e-3 max|y_ref| over the row.
"""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import workloads

Q_FLIP_BUDGET = 1e-3
Y_REL_TOL = 1e-3


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev() -> torch.device:
    return torch.device("cuda:0")


def to_dev_x(x_dev_form: np.ndarray) -> torch.Tensor:
    """float32 array -> float32 tensor; uint16 bf16 bits -> bfloat16 tensor."""
    if x_dev_form.dtype == np.float32:
        return torch.from_numpy(np.ascontiguousarray(x_dev_form)).to(dev())
    t = torch.from_numpy(np.ascontiguousarray(x_dev_form).view(np.int16)).to(dev())
    return t.view(torch.bfloat16)


def packed_to_np(Wp: torch.Tensor) -> np.ndarray:
    return Wp.cpu().numpy().view(np.uint32)


def np_to_packed(words: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(words, np.uint32).view(np.int32)).to(dev())


def compare_q(q_gpu: np.ndarray, q_ref: np.ndarray) -> tuple[np.ndarray, float]:
    """Returns (rows with any difference, fraction of differing entries)."""
    d = np.abs(q_gpu.astype(np.int16) - q_ref.astype(np.int16))
    assert d.max(initial=0) <= 1, f"q differs by {d.max()} LSB"
    frac = float((d > 0).mean()) if d.size else 0.0
    assert frac <= Q_FLIP_BUDGET, f"q differs in {frac:.2e} of entries"
    return np.nonzero(d.any(axis=1))[0], frac


def compare_y(y_gpu: np.ndarray, y_ref: np.ndarray, acc_ref: np.ndarray,
              flip_rows_mask: np.ndarray | None = None) -> float:
    """Per-element relative check (exact zero where acc is 0); rows flagged in
    flip_rows_mask use the row-norm bound.  Returns the max relative error."""
    y_gpu = y_gpu.astype(np.float64)
    y_ref = y_ref.astype(np.float64)
    err = np.abs(y_gpu - y_ref)
    ok_rows = np.ones(y_ref.shape[0], bool) if flip_rows_mask is None else ~flip_rows_mask
    zero = acc_ref == 0
    assert (y_gpu[ok_rows][zero[ok_rows]] == 0).all(), "nonzero output where the ternary sum is 0"
    nz = ~zero & ok_rows[:, None]
    rel = err[nz] / np.abs(y_ref[nz]) if nz.any() else np.zeros(1)
    worst = float(rel.max(initial=0.0))
    assert worst <= Y_REL_TOL, f"max rel error {worst:.3e}"
    if flip_rows_mask is not None and flip_rows_mask.any():
        for m in np.nonzero(flip_rows_mask)[0]:
            bound = Y_REL_TOL * np.abs(y_ref[m]).max(initial=0.0)
            assert err[m].max(initial=0.0) <= bound + 1e-30
    return worst


class Case:
    """One seeded problem: host arrays, oracle results, device tensors."""

    def __init__(self, x_dev_form, x_f32, gamma, W, name=""):
        self.name = name
        self.x_dev_form = x_dev_form
        self.x_f32 = x_f32
        self.gamma = gamma
        self.W = W
        self.M, self.K = x_f32.shape
        self.N = W.shape[0]

    @classmethod
    def from_workload(cls, w: workloads.Workload, M: int | None = None):
        xd, xf = workloads.make_x(w, M)
        g = workloads.make_gamma(w)
        W = workloads.make_w(w)
        return cls(xd, xf, None if w.gamma_kind == "ones" else g, W, w.name)

    # -- oracle side --------------------------------------------------------
    def oracle_weights(self):
        self.t, self.ws_ref = oracle.weight_quant(self.W)
        self.words_ref = oracle.pack(self.t)

    def oracle_act(self):
        self.q_ref, self.a_ref = oracle.rmsnorm_act_quant(self.x_f32, self.gamma)

    # -- device side --------------------------------------------------------
    def upload(self):
        self.x_d = to_dev_x(self.x_dev_form)
        self.g_d = None if self.gamma is None else torch.from_numpy(self.gamma).to(dev())
        self.W_d = torch.from_numpy(self.W).to(dev())
