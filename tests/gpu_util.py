"""Helpers for the GPU tests: move generator batches to the device and compare with the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

from paper_2606_00535_amd import workload as W

# Attention tolerance of the contract: max-abs error against the fp64 oracle, bf16 in / fp32 accumulate.
ATTN_TOL_BF16 = 2e-2
# fp32 inputs, fp32 arithmetic throughout (exp2 approximations, reassociation): far below this.
ATTN_TOL_F32 = 1e-5
# lse is computed from fp32 scores whatever the input type.
LSE_TOL = 2e-3

# Attention entropy of a row (nats), absolute.  The kernel's scores are fp32 sums of exact products of the bf16
# inputs (the matrix cores multiply bf16 exactly and accumulate in fp32), so each differs from the oracle's fp64
# score by rounding only: for these N(0,1) inputs a few 1e-7 in log2 units.  H = -sum p ln p moves by at most
# 2 ln(n) times the largest score error (ln n <= 9 here), and the fp32 sums of p and p*(z - m) add a few units of
# 2^-24 relative.  Every tested shape stays under 2e-6; 1e-5 is that with margin, and a relative error of 1e-4
# in H (5e-4 absolute at H ~ 5) fails it.
ENTROPY_TOL = 1e-5

# Visual-token importance (Eq. 2), relative, plus an absolute floor for the exact zeros.  Each term is
# 2^(s c - lse2) with an fp32 score and the attention call's fp32 log-sum-exp: a few 1e-6 in the exponent, so a
# few 1e-6 relative per term; the fp32 sums over <= 8192 rows and the heads add less.  3e-5 is that with
# margin, and a relative error of 1e-4 fails it.
IMPORTANCE_REL_TOL = 3e-5
IMPORTANCE_ABS_TOL = 1e-9


def entropy_error(got, ref):
    """(largest absolute error, whether it is within ENTROPY_TOL)."""
    err = float(np.max(np.abs(np.asarray(got, np.float64) - np.asarray(ref, np.float64)))) if np.size(ref) else 0.0
    return err, err <= ENTROPY_TOL


def importance_error(got, ref):
    """(largest relative error, whether every entry is within IMPORTANCE_REL_TOL * |ref| + IMPORTANCE_ABS_TOL)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    rel = float(np.max(err / (np.abs(ref) + 1e-30))) if err.size else 0.0
    return rel, bool(np.all(err <= IMPORTANCE_REL_TOL * np.abs(ref) + IMPORTANCE_ABS_TOL))


def note(*msg):
    print(*msg, flush=True)
    sys.stdout.flush()


def device():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a HIP device")
    return torch.device("cuda", 0)


def to_dev(a: np.ndarray, dev, bf16: bool = False) -> torch.Tensor:
    if bf16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def layer_tensors(batch: W.Batch, li: int, dev):
    bf = batch.wl.dtype == "bf16"
    q = to_dev(batch.q[li], dev, bf)
    k = to_dev(batch.k_cache[li], dev, bf)
    v = to_dev(batch.v_cache[li], dev, bf)
    kv = to_dev(batch.kv_len, dev)
    par = to_dev(batch.parent, dev)
    return q, k, v, kv, par


def f32(a: np.ndarray) -> np.ndarray:
    return W.bf16_bits_to_f32(a) if a.dtype == np.uint16 else a


def attn_errors(out: torch.Tensor, ref: np.ndarray):
    o = out.float().cpu().numpy().astype(np.float64)
    err = np.abs(o - ref)
    return float(err.max()), float((err / (np.abs(ref) + 1e-3)).max()), o


def dense_bits_of(t: torch.Tensor) -> np.ndarray:
    return t.cpu().view(torch.int16).numpy().view(np.uint16) if t.dtype == torch.bfloat16 else t.cpu().numpy()
