"""dreams_tree_verify_attn_noalloc (the allocation-free entry point) against dreams_tree_verify_attn, through the
C ABI: the same kernels, so the outputs and lse must agree bit for bit -- and with the fp64 oracle within the
attention bound -- on two calls in a row, the second with a smaller input (the library's scratch array keeps
the first call's contents)."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from gpu_util import ATTN_TOL_BF16, LSE_TOL, device, f32, layer_tensors, note
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu


def _call_noalloc(q, k, v, kv, par, num_splits, max_kv_len):
    desc = dreams.attn_desc(q, k, num_splits=num_splits, max_kv_len=max_kv_len)
    out = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
    st = dreams.lib().dreams_tree_verify_attn_noalloc(
        ctypes.byref(desc), ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
        ctypes.c_void_p(v.data_ptr()), ctypes.c_void_p(kv.data_ptr()), ctypes.c_void_p(par.data_ptr()), None,
        ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(lse.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, dreams.lib().dreams_last_error_message().decode()
    return out, lse, dreams.tree_verify_attn_splits(desc)


def _check_against(batch, q, k, v, kv, par, out, lse, splits, label):
    # the workspace entry point on the same inputs and split count: identical bits
    o2, l2 = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits, max_kv_len=batch.wl.max_kv_len)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), o2.view(torch.int16)), label
    assert torch.equal(lse, l2), label
    # and the oracle, within the contract's bound
    v32 = f32(batch.v_cache[0])
    ref, lref = oracle.tree_attn(f32(batch.q[0]), f32(batch.k_cache[0]), v32, batch.kv_len, batch.parent,
                                 batch.scale, batch.wl.num_kv_heads)
    err = float(np.abs(out.float().cpu().numpy() - ref).max())
    lerr = float(np.abs(lse.cpu().numpy() - lref).max())
    note("%s: splits=%d max_abs=%.3e lse=%.2e" % (label, splits, err, lerr))
    assert err <= ATTN_TOL_BF16 and lerr <= LSE_TOL, label


@pytest.mark.parametrize("splits", [8, 3, 1])
def test_noalloc_matches_workspace_call_twice(splits):
    dev = device()
    big = W.Workload(name="noalloc_big", batch=2, num_q_heads=8, num_kv_heads=4, head_dim=128, dtype="bf16",
                     num_layers=1, kv_len=1500, image_tokens=0, num_nodes=60, depth=6, max_branch=4, vocab=64,
                     agree=0.7, seed=21)
    small = W.Workload(name="noalloc_small", batch=1, num_q_heads=4, num_kv_heads=2, head_dim=64, dtype="bf16",
                       num_layers=1, kv_len=400, image_tokens=0, num_nodes=16, depth=4, max_branch=3, vocab=64,
                       agree=0.7, seed=22)
    for wl in (big, small):   # the second call is smaller than the first
        batch = W.make_batch(wl, with_logits=False)
        q, k, v, kv, par = layer_tensors(batch, 0, dev)
        note("noalloc %s splits=%d" % (wl.name, splits))
        out, lse, s = _call_noalloc(q, k, v, kv, par, splits, wl.max_kv_len)
        torch.cuda.synchronize()
        _check_against(batch, q, k, v, kv, par, out, lse, s, "noalloc %s" % wl.name)


def test_noalloc_rejects_shape_beyond_scratch():
    dev = device()
    q = torch.zeros((64, 32, 128, 128), dtype=torch.bfloat16, device=dev)
    k = torch.zeros((64, 32, 256, 128), dtype=torch.bfloat16, device=dev)
    desc = dreams.attn_desc(q, k, num_splits=2)
    need = dreams.tree_verify_attn_workspace_size(desc)
    assert need > 16 << 20
    kv = torch.zeros(64, dtype=torch.int32, device=dev)
    par = torch.zeros((64, 128), dtype=torch.int32, device=dev)
    st = dreams.lib().dreams_tree_verify_attn_noalloc(
        ctypes.byref(desc), ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()),
        ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(kv.data_ptr()), ctypes.c_void_p(par.data_ptr()), None,
        ctypes.c_void_p(q.data_ptr()), None, None)
    assert st == dreams.DREAMS_ERR_UNSUPPORTED
    assert b"scratch" in dreams.lib().dreams_last_error_message()
