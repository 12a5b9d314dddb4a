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
