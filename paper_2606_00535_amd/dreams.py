"""Python binding of libdreams.so (C ABI in include/dreams.h).

Argument marshalling only: every step runs in the library's HIP kernels.  PyTorch supplies device memory
and the current stream.  The library must be built (``python -m paper_2606_00535_amd.build``); if it is
missing every call raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
import threading
from typing import Optional, Tuple

import torch

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdreams.so")

DREAMS_OK, DREAMS_ERR_INVALID_ARG, DREAMS_ERR_UNSUPPORTED, DREAMS_ERR_WORKSPACE, DREAMS_ERR_HIP = 0, -1, -2, -3, -4
DREAMS_ERR_DEVICE = -5
DREAMS_F32, DREAMS_BF16 = 0, 1

# every symbol include/dreams.h declares
EXPORTS = (
    "dreams_tree_verify_attn_workspace_size", "dreams_tree_verify_attn", "dreams_tree_accept_workspace_size",
    "dreams_tree_accept", "dreams_kv_commit", "dreams_status_string", "dreams_last_error_message",
    "dreams_check_tree_host", "dreams_stream_read", "dreams_tree_verify_attn_entropy", "dreams_attn_entropy_mean",
    "dreams_attn_entropy_select", "dreams_visual_importance_workspace_size", "dreams_visual_importance",
    "dreams_visual_topk", "dreams_visual_gather", "dreams_tree_accept_sampled_workspace_size",
    "dreams_tree_accept_sampled", "dreams_tree_accept_lm_head_workspace_size", "dreams_tree_accept_lm_head",
    "dreams_workspace_status", "dreams_tree_verify_attn_splits", "dreams_tree_verify_attn_noalloc",
    "dreams_set_wait_limit", "dreams_prefill_attn_stats", "dreams_prefill_attn_entropy_mean",
    "dreams_prefill_visual_importance",
)


class DreamsError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__("%s (status %d)" % (message, status))
        self.status = status


class AttnDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_nodes", ctypes.c_int32), ("cache_capacity", ctypes.c_int32),
                ("max_kv_len", ctypes.c_int32), ("num_splits", ctypes.c_int32), ("dtype", ctypes.c_int),
                ("scale", ctypes.c_float)]


class PrefillDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("num_rows", ctypes.c_int32), ("cache_capacity", ctypes.c_int32),
                ("scale", ctypes.c_float)]


_lib = None
_lib_lock = threading.Lock()


def library_path() -> str:
    return LIBRARY


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        with _lib_lock:
            if _lib is None:
                if not os.path.exists(LIBRARY):
                    raise RuntimeError("libdreams.so is not built (run: python -m paper_2606_00535_amd.build)")
                L = ctypes.CDLL(LIBRARY)
                P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
                L.dreams_tree_verify_attn_workspace_size.argtypes = [ctypes.POINTER(AttnDesc), ctypes.POINTER(SZ)]
                L.dreams_tree_verify_attn.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, P, P, P, P, P, SZ, P]
                L.dreams_tree_accept_workspace_size.argtypes = [I32, I32, I32, ctypes.POINTER(SZ)]
                L.dreams_tree_accept.argtypes = [I32, I32, I32, P, P, P, P, P, P, P, P, SZ, P]
                L.dreams_kv_commit.argtypes = [I32, ctypes.c_int64, I32, I32, I32, I32, ctypes.c_int, P, P, P, P, P,
                                               I32, P, P]
                L.dreams_status_string.argtypes = [ctypes.c_int]
                L.dreams_status_string.restype = ctypes.c_char_p
                L.dreams_last_error_message.argtypes = []
                L.dreams_last_error_message.restype = ctypes.c_char_p
                L.dreams_check_tree_host.argtypes = [P, I32]
                L.dreams_stream_read.argtypes = [P, SZ, P, P]
                L.dreams_tree_verify_attn_entropy.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, P, P, P, P, P, P,
                                                              SZ, P]
                L.dreams_attn_entropy_mean.argtypes = [ctypes.c_int64, P, P, P]
                L.dreams_attn_entropy_select.argtypes = [I32, P, P, P]
                L.dreams_visual_importance_workspace_size.argtypes = [I32, I32, I32, ctypes.POINTER(SZ)]
                L.dreams_visual_importance.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, I32, I32, P, P, SZ, P]
                L.dreams_visual_topk.argtypes = [I32, I32, I32, P, P, P]
                L.dreams_tree_accept_sampled_workspace_size.argtypes = [I32, I32, I32, ctypes.POINTER(SZ)]
                L.dreams_tree_accept_sampled.argtypes = [I32, I32, I32, ctypes.c_double, P, P, P, P, P, P, P, P, P,
                                                         SZ, P]
                L.dreams_tree_accept_lm_head_workspace_size.argtypes = [I32, I32, I32, I32, ctypes.POINTER(SZ)]
                L.dreams_tree_accept_lm_head.argtypes = [I32, I32, I32, I32, P, P, P, P, P, P, P, P, P, SZ, P]
                L.dreams_visual_gather.argtypes = [I32, I32, I32, I32, ctypes.c_int, P, P, I32, P, I32, P, P, P]
                L.dreams_workspace_status.argtypes = [P, SZ, P]
                L.dreams_set_wait_limit.argtypes = [ctypes.c_double]
                L.dreams_tree_verify_attn_noalloc.argtypes = [ctypes.POINTER(AttnDesc), P, P, P, P, P, P, P, P, P]
                L.dreams_tree_verify_attn_splits.argtypes = [ctypes.POINTER(AttnDesc), ctypes.POINTER(I32)]
                L.dreams_prefill_attn_stats.argtypes = [ctypes.POINTER(PrefillDesc), P, P, P, P, P, P]
                L.dreams_prefill_attn_entropy_mean.argtypes = [I32, I32, I32, P, P, P, P]
                L.dreams_prefill_visual_importance.argtypes = [ctypes.POINTER(PrefillDesc), P, P, P, P, I32, I32, P, P,
                                                               SZ, P]
                for f in ("dreams_tree_verify_attn_workspace_size", "dreams_tree_verify_attn",
                          "dreams_tree_accept_workspace_size", "dreams_tree_accept", "dreams_kv_commit",
                          "dreams_check_tree_host", "dreams_stream_read", "dreams_tree_verify_attn_entropy",
                          "dreams_attn_entropy_mean", "dreams_attn_entropy_select",
                          "dreams_visual_importance_workspace_size", "dreams_visual_importance", "dreams_visual_topk",
                          "dreams_visual_gather", "dreams_workspace_status", "dreams_tree_verify_attn_splits",
                          "dreams_tree_verify_attn_noalloc", "dreams_set_wait_limit", "dreams_prefill_attn_stats",
                          "dreams_prefill_attn_entropy_mean", "dreams_prefill_visual_importance"):
                    getattr(L, f).restype = ctypes.c_int
                _lib = L
    return _lib


def _check(status: int):
    if status != DREAMS_OK:
        msg = lib().dreams_last_error_message().decode() or lib().dreams_status_string(status).decode()
        raise DreamsError(status, msg)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _need(t: torch.Tensor, name: str, dtype, device=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if ndim is not None and t.dim() != ndim:
        raise ValueError("%s must have %d dimensions" % (name, ndim))


# Workspaces: one per (device, stream, verb), zero-filled when created and left zero by every call.
_ws = {}
_ws_lock = threading.Lock()


def _workspace(kind: str, nbytes: int, device: torch.device, stream) -> Optional[torch.Tensor]:
    if nbytes == 0:
        return None
    key = (kind, device.index, stream.value if stream.value else 0)
    with _ws_lock:
        t = _ws.get(key)
        if t is None or t.numel() < nbytes:
            t = torch.zeros(nbytes, dtype=torch.uint8, device=device)
            _ws[key] = t
        return t


def attn_desc(q: torch.Tensor, k_cache: torch.Tensor, num_splits: int = 0, max_kv_len: int = 0,
              scale: Optional[float] = None) -> AttnDesc:
    B, Hq, T, D = q.shape
    Hkv, S_cap = k_cache.shape[1], k_cache.shape[2]
    dtype = DREAMS_BF16 if q.dtype == torch.bfloat16 else DREAMS_F32
    return AttnDesc(B, Hq, Hkv, D, T, S_cap, max_kv_len, num_splits, dtype,
                    1.0 / math.sqrt(D) if scale is None else float(scale))


def tree_verify_attn_workspace_size(desc: AttnDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dreams_tree_verify_attn_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def tree_verify_attn_splits(desc: AttnDesc) -> int:
    """dreams_tree_verify_attn_splits: pieces of the key axis the library uses for `desc`."""
    n = ctypes.c_int32(0)
    _check(lib().dreams_tree_verify_attn_splits(ctypes.byref(desc), ctypes.byref(n)))
    return n.value


def workspace_status(workspace: torch.Tensor, stream=None) -> None:
    """dreams_workspace_status: raises DreamsError (DREAMS_ERR_DEVICE) if a kernel flagged a failure in
    `workspace` since the last check; clears the flags."""
    _need(workspace, "workspace", torch.uint8, workspace.device)
    _check(lib().dreams_workspace_status(_ptr(workspace), workspace.numel(), _stream(stream)))


def set_wait_limit(seconds: float) -> None:
    """dreams_set_wait_limit: bound on every in-kernel wait for another workgroup (default 0.2 s)."""
    _check(lib().dreams_set_wait_limit(float(seconds)))


def cached_workspaces():
    """The workspaces the binding created (one per device, stream and verb)."""
    with _ws_lock:
        return list(_ws.values())


def tree_verify_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
                     parent: Optional[torch.Tensor] = None, tree_mask: Optional[torch.Tensor] = None,
                     scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                     lse: Optional[torch.Tensor] = None, with_lse: bool = True, max_kv_len: int = 0,
                     num_splits: int = 0, workspace: Optional[torch.Tensor] = None,
                     stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """dreams_tree_verify_attn.  q [B,Hq,T,D]; k_cache/v_cache [B,Hkv,S_cap,D] (bf16 or fp32, same as q);
    kv_len [B] int32; parent [B,T] int32 or tree_mask [B,T,ceil(T/64)] int64 (bit patterns).
    Returns (out [B,Hq,T,D], lse [B,Hq,T] float32 or None)."""
    out, lse, _ = _verify_attn(q, k_cache, v_cache, kv_len, parent, tree_mask, scale, out, lse, with_lse,
                               max_kv_len, num_splits, workspace, stream, None)
    return out, lse


def tree_verify_attn_entropy(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
                             parent: Optional[torch.Tensor] = None, tree_mask: Optional[torch.Tensor] = None,
                             scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                             lse: Optional[torch.Tensor] = None, with_lse: bool = True,
                             entropy: Optional[torch.Tensor] = None, max_kv_len: int = 0, num_splits: int = 0,
                             workspace: Optional[torch.Tensor] = None, stream=None):
    """dreams_tree_verify_attn_entropy: as tree_verify_attn, plus every row's attention entropy (nats).
    Returns (out, lse or None, entropy [B,Hq,T] float32)."""
    B, Hq, T, _ = q.shape
    if entropy is None:
        entropy = torch.empty((B, Hq, T), dtype=torch.float32, device=q.device)
    else:
        _need(entropy, "entropy", torch.float32, q.device)
        if tuple(entropy.shape) != (B, Hq, T):
            raise ValueError("entropy must be [B, Hq, T]")
    return _verify_attn(q, k_cache, v_cache, kv_len, parent, tree_mask, scale, out, lse, with_lse, max_kv_len,
                        num_splits, workspace, stream, entropy)


def attn_entropy_mean(entropy: torch.Tensor, ae: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dreams_attn_entropy_mean: AE of one layer from its row entropies (any shape).  Returns a [1] float32."""
    _need(entropy, "entropy", torch.float32, entropy.device)
    if ae is None:
        ae = torch.empty(1, dtype=torch.float32, device=entropy.device)
    _check(lib().dreams_attn_entropy_mean(entropy.numel(), _ptr(entropy), _ptr(ae), _stream(stream)))
    return ae


def attn_entropy_select(ae: torch.Tensor, best: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dreams_attn_entropy_select: the distillation layer from per-layer AE [NL].  Returns a [1] int32."""
    _need(ae, "ae", torch.float32, ae.device, 1)
    if best is None:
        best = torch.empty(1, dtype=torch.int32, device=ae.device)
    _check(lib().dreams_attn_entropy_select(ae.numel(), _ptr(ae), _ptr(best), _stream(stream)))
    return best


VISUAL_MAX_TOKENS = 8192


def visual_importance_workspace_size(batch: int, num_kv_heads: int, vis_count: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dreams_visual_importance_workspace_size(batch, num_kv_heads, vis_count, ctypes.byref(n)))
    return n.value


def visual_importance(q: torch.Tensor, k_cache: torch.Tensor, kv_len: torch.Tensor, lse: torch.Tensor,
                      vis_begin: int, vis_count: int, scale: Optional[float] = None,
                      importance: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                      stream=None) -> torch.Tensor:
    """dreams_visual_importance (Eq. 2): q [B,Hq,T,D] and k_cache [B,Hkv,S_cap,D] bf16, kv_len [B] int32, lse
    [B,Hq,T] float32 from the attention call on the same rows.  Returns importance [B, vis_count] float32."""
    dev = q.device
    _need(q, "q", torch.bfloat16, dev, 4)
    _need(k_cache, "k_cache", torch.bfloat16, dev, 4)
    _need(kv_len, "kv_len", torch.int32, dev, 1)
    _need(lse, "lse", torch.float32, dev, 3)
    B, Hq, T, D = q.shape
    desc = attn_desc(q, k_cache, 0, 0, scale)
    if importance is None:
        importance = torch.empty((B, vis_count), dtype=torch.float32, device=dev)
    else:
        _need(importance, "importance", torch.float32, dev)
    nbytes = visual_importance_workspace_size(B, k_cache.shape[1], vis_count)
    st = _stream(stream)
    if workspace is None:
        workspace = _workspace("visual", nbytes, dev, st)
    _check(lib().dreams_visual_importance(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(kv_len), _ptr(lse),
                                          vis_begin, vis_count, _ptr(importance), _ptr(workspace),
                                          0 if workspace is None else workspace.numel() * workspace.element_size(),
                                          st))
    return importance


def prefill_desc(q: torch.Tensor, k_cache: torch.Tensor, scale: Optional[float] = None) -> PrefillDesc:
    B, Hq, N, D = q.shape
    return PrefillDesc(B, Hq, k_cache.shape[1], D, N, k_cache.shape[2],
                       float(1.0 / math.sqrt(D) if scale is None else scale))


def prefill_attn_stats(q: torch.Tensor, k_cache: torch.Tensor, prompt_len: torch.Tensor, scale: Optional[float] = None,
                       lse: Optional[torch.Tensor] = None, entropy: Optional[torch.Tensor] = None,
                       with_lse: bool = True, with_entropy: bool = True, stream=None):
    """dreams_prefill_attn_stats: the causal attention of a prompt's own rows (row i sees slots 0..i).  q
    [B,Hq,N,D] and k_cache [B,Hkv,S_cap,D] bf16, prompt_len [B] int32.  Returns (lse, entropy), each [B,Hq,N]
    float32 or None."""
    dev = q.device
    _need(q, "q", torch.bfloat16, dev, 4)
    _need(k_cache, "k_cache", torch.bfloat16, dev, 4)
    _need(prompt_len, "prompt_len", torch.int32, dev, 1)
    B, Hq, N, D = q.shape
    if with_lse and lse is None:
        lse = torch.empty((B, Hq, N), dtype=torch.float32, device=dev)
    if with_entropy and entropy is None:
        entropy = torch.empty((B, Hq, N), dtype=torch.float32, device=dev)
    for t, nm in ((lse, "lse"), (entropy, "entropy")):
        if t is not None:
            _need(t, nm, torch.float32, dev, 3)
    desc = prefill_desc(q, k_cache, scale)
    _check(lib().dreams_prefill_attn_stats(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(prompt_len), _ptr(lse),
                                           _ptr(entropy), _stream(stream)))
    return lse, entropy


def prefill_attn_entropy_mean(entropy: torch.Tensor, prompt_len: torch.Tensor, ae: Optional[torch.Tensor] = None,
                              stream=None) -> torch.Tensor:
    """dreams_prefill_attn_entropy_mean: AE of one layer over prompts from entropy [B,Hq,N].  Returns [1] float32."""
    _need(entropy, "entropy", torch.float32, entropy.device, 3)
    _need(prompt_len, "prompt_len", torch.int32, entropy.device, 1)
    if ae is None:
        ae = torch.empty(1, dtype=torch.float32, device=entropy.device)
    B, Hq, N = entropy.shape
    _check(lib().dreams_prefill_attn_entropy_mean(B, Hq, N, _ptr(entropy), _ptr(prompt_len), _ptr(ae),
                                                  _stream(stream)))
    return ae


def prefill_visual_importance(q: torch.Tensor, k_cache: torch.Tensor, prompt_len: torch.Tensor, lse: torch.Tensor,
                              vis_begin: int, vis_count: int, scale: Optional[float] = None,
                              importance: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                              stream=None) -> torch.Tensor:
    """dreams_prefill_visual_importance (Eq. 2 over the prompt's causal attention): lse [B,Hq,N] from
    prefill_attn_stats.  Returns importance [B, vis_count] float32."""
    dev = q.device
    _need(q, "q", torch.bfloat16, dev, 4)
    _need(k_cache, "k_cache", torch.bfloat16, dev, 4)
    _need(prompt_len, "prompt_len", torch.int32, dev, 1)
    _need(lse, "lse", torch.float32, dev, 3)
    B = q.shape[0]
    if importance is None:
        importance = torch.empty((B, vis_count), dtype=torch.float32, device=dev)
    else:
        _need(importance, "importance", torch.float32, dev)
    nbytes = visual_importance_workspace_size(B, k_cache.shape[1], vis_count)
    st = _stream(stream)
    if workspace is None:
        workspace = _workspace("visual", nbytes, dev, st)
    desc = prefill_desc(q, k_cache, scale)
    _check(lib().dreams_prefill_visual_importance(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(prompt_len),
                                                  _ptr(lse), vis_begin, vis_count, _ptr(importance), _ptr(workspace),
                                                  0 if workspace is None else workspace.numel() * workspace.element_size(),
                                                  st))
    return importance


def visual_topk(importance: torch.Tensor, keep_count: int, keep: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """dreams_visual_topk: importance [B, n] float32 -> keep [B, keep_count] int32 (increasing token order)."""
    _need(importance, "importance", torch.float32, importance.device, 2)
    B, n = importance.shape
    if keep is None:
        keep = torch.empty((B, keep_count), dtype=torch.int32, device=importance.device)
    else:
        _need(keep, "keep", torch.int32, importance.device, 2)
    _check(lib().dreams_visual_topk(B, n, keep_count, _ptr(importance), _ptr(keep), _stream(stream)))
    return keep


def visual_gather(k_cache: torch.Tensor, v_cache: torch.Tensor, vis_begin: int, keep: torch.Tensor,
                  k_out: Optional[torch.Tensor] = None, v_out: Optional[torch.Tensor] = None, stream=None):
    """dreams_visual_gather: the kept visual tokens' K/V rows -> (k_out, v_out) [B, Hkv, keep_count, D]."""
    dt = k_cache.dtype
    dev = k_cache.device
    _need(k_cache, "k_cache", dt, dev, 4)
    _need(v_cache, "v_cache", dt, dev, 4)
    _need(keep, "keep", torch.int32, dev, 2)
    B, Hkv, S, D = k_cache.shape
    r = keep.shape[1]
    if k_out is None:
        k_out = torch.empty((B, Hkv, r, D), dtype=dt, device=dev)
    if v_out is None:
        v_out = torch.empty((B, Hkv, r, D), dtype=dt, device=dev)
    _check(lib().dreams_visual_gather(B, Hkv, D, S, DREAMS_BF16 if dt == torch.bfloat16 else DREAMS_F32,
                                      _ptr(k_cache), _ptr(v_cache), vis_begin, _ptr(keep), r, _ptr(k_out),
                                      _ptr(v_out), _stream(stream)))
    return k_out, v_out


def _verify_attn(q, k_cache, v_cache, kv_len, parent, tree_mask, scale, out, lse, with_lse, max_kv_len, num_splits,
                 workspace, stream, entropy):
    dt = q.dtype
    if dt not in (torch.bfloat16, torch.float32):
        raise TypeError("q must be bfloat16 or float32")
    dev = q.device
    _need(q, "q", dt, dev, 4)
    _need(k_cache, "k_cache", dt, dev, 4)
    _need(v_cache, "v_cache", dt, dev, 4)
    _need(kv_len, "kv_len", torch.int32, dev, 1)
    if k_cache.shape != v_cache.shape:
        raise ValueError("k_cache and v_cache shapes differ")
    B, Hq, T, D = q.shape
    if k_cache.shape[0] != B or k_cache.shape[3] != D or kv_len.shape[0] != B:
        raise ValueError("batch / head_dim mismatch between q, caches and kv_len")
    if parent is not None:
        _need(parent, "parent", torch.int32, dev, 2)
        if tuple(parent.shape) != (B, T):
            raise ValueError("parent must be [B, T]")
    if tree_mask is not None:
        _need(tree_mask, "tree_mask", torch.int64, dev, 3)
        if tuple(tree_mask.shape) != (B, T, (T + 63) // 64):
            raise ValueError("tree_mask must be [B, T, ceil(T/64)]")
    desc = attn_desc(q, k_cache, num_splits, max_kv_len, scale)
    if out is None:
        out = torch.empty_like(q)
    else:
        _need(out, "out", dt, dev)
        if out.shape != q.shape:
            raise ValueError("out must have q's shape")
    if lse is None and with_lse:
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    elif lse is not None:
        _need(lse, "lse", torch.float32, dev)
        if tuple(lse.shape) != (B, Hq, T):
            raise ValueError("lse must be [B, Hq, T]")
    st = _stream(stream)
    nbytes = tree_verify_attn_workspace_size(desc)
    if workspace is None:
        workspace = _workspace("attn", nbytes, dev, st)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if entropy is None:
        _check(lib().dreams_tree_verify_attn(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kv_len),
                                             _ptr(parent), _ptr(tree_mask), _ptr(out), _ptr(lse), _ptr(workspace),
                                             ws_bytes, st))
    else:
        _check(lib().dreams_tree_verify_attn_entropy(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                     _ptr(kv_len), _ptr(parent), _ptr(tree_mask), _ptr(out), _ptr(lse),
                                                     _ptr(entropy), _ptr(workspace), ws_bytes, st))
    return out, lse, entropy


def tree_verify_attn_noalloc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
                             parent: Optional[torch.Tensor] = None, tree_mask: Optional[torch.Tensor] = None,
                             scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                             lse: Optional[torch.Tensor] = None, with_lse: bool = True, max_kv_len: int = 0,
                             num_splits: int = 0, stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """dreams_tree_verify_attn_noalloc: tree_verify_attn without a workspace (the library's fixed scratch array
    instead).  `out` and `lse` may be passed in so that nothing is allocated here either."""
    dt = q.dtype
    if dt not in (torch.bfloat16, torch.float32):
        raise TypeError("q must be bfloat16 or float32")
    dev = q.device
    for t, name in ((q, "q"), (k_cache, "k_cache"), (v_cache, "v_cache")):
        _need(t, name, dt, dev, 4)
    _need(kv_len, "kv_len", torch.int32, dev, 1)
    if parent is not None:
        _need(parent, "parent", torch.int32, dev, 2)
    if tree_mask is not None:
        _need(tree_mask, "tree_mask", torch.int64, dev, 3)
    B, Hq, T, D = q.shape
    desc = attn_desc(q, k_cache, num_splits, max_kv_len, scale)
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", dt, dev)
    if out.shape != q.shape:
        raise ValueError("out must have q's shape")
    if lse is None and with_lse:
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
        if tuple(lse.shape) != (B, Hq, T):
            raise ValueError("lse must be [B, Hq, T]")
    _check(lib().dreams_tree_verify_attn_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                 _ptr(kv_len), _ptr(parent), _ptr(tree_mask), _ptr(out), _ptr(lse),
                                                 _stream(stream)))
    return out, lse


def tree_accept_workspace_size(batch: int, num_nodes: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dreams_tree_accept_workspace_size(batch, num_nodes, vocab, ctypes.byref(n)))
    return n.value


def tree_accept(target_logits: torch.Tensor, draft_tokens: torch.Tensor, parent: torch.Tensor,
                want_target_argmax: bool = False, outputs=None, workspace: Optional[torch.Tensor] = None,
                stream=None):
    """dreams_tree_accept.  target_logits [B,T,V] float32, draft_tokens / parent [B,T] int32.
    Returns (accept_len [B], accept_path [B,T], next_token [B], target_argmax [B,T] or None), all int32.
    `outputs` may pass preallocated (accept_len, accept_path, next_token, target_argmax-or-None)."""
    dev = target_logits.device
    _need(target_logits, "target_logits", torch.float32, dev, 3)
    B, T, V = target_logits.shape
    _need(draft_tokens, "draft_tokens", torch.int32, dev, 2)
    _need(parent, "parent", torch.int32, dev, 2)
    if tuple(draft_tokens.shape) != (B, T) or tuple(parent.shape) != (B, T):
        raise ValueError("draft_tokens and parent must be [B, T]")
    if outputs is None:
        alen = torch.empty(B, dtype=torch.int32, device=dev)
        path = torch.empty((B, T), dtype=torch.int32, device=dev)
        nxt = torch.empty(B, dtype=torch.int32, device=dev)
        am = torch.empty((B, T), dtype=torch.int32, device=dev) if want_target_argmax else None
    else:
        alen, path, nxt, am = outputs
        for t, nm, shp in ((alen, "accept_len", (B,)), (path, "accept_path", (B, T)), (nxt, "next_token", (B,))):
            _need(t, nm, torch.int32, dev)
            if tuple(t.shape) != shp:
                raise ValueError("%s has the wrong shape" % nm)
        if am is not None:
            _need(am, "target_argmax", torch.int32, dev)
    st = _stream(stream)
    nbytes = tree_accept_workspace_size(B, T, V)
    if workspace is None:
        workspace = _workspace("accept", nbytes, dev, st)
    _check(lib().dreams_tree_accept(B, T, V, _ptr(target_logits), _ptr(draft_tokens), _ptr(parent), _ptr(alen),
                                    _ptr(path), _ptr(nxt), _ptr(am), _ptr(workspace),
                                    0 if workspace is None else workspace.numel(), st))
    return alen, path, nxt, am


def tree_accept_sampled_workspace_size(batch: int, num_nodes: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dreams_tree_accept_sampled_workspace_size(batch, num_nodes, vocab, ctypes.byref(n)))
    return n.value


def tree_accept_sampled(target_logits: torch.Tensor, draft_logits: torch.Tensor, draft_tokens: torch.Tensor,
                        parent: torch.Tensor, uniforms: torch.Tensor, temperature: float = 1.0, outputs=None,
                        workspace: Optional[torch.Tensor] = None, stream=None):
    """dreams_tree_accept_sampled.  target_logits / draft_logits [B,T,V] float32, draft_tokens / parent [B,T]
    int32, uniforms [B,T] float32 in [0, 1).  Returns (accept_len [B], accept_path [B,T], next_token [B]), int32.
    `outputs` may pass preallocated (accept_len, accept_path, next_token)."""
    dev = target_logits.device
    _need(target_logits, "target_logits", torch.float32, dev, 3)
    B, T, V = target_logits.shape
    _need(draft_logits, "draft_logits", torch.float32, dev, 3)
    if tuple(draft_logits.shape) != (B, T, V):
        raise ValueError("draft_logits must have the shape of target_logits")
    _need(draft_tokens, "draft_tokens", torch.int32, dev, 2)
    _need(parent, "parent", torch.int32, dev, 2)
    _need(uniforms, "uniforms", torch.float32, dev, 2)
    if tuple(draft_tokens.shape) != (B, T) or tuple(parent.shape) != (B, T) or tuple(uniforms.shape) != (B, T):
        raise ValueError("draft_tokens, parent and uniforms must be [B, T]")
    if outputs is None:
        alen = torch.empty(B, dtype=torch.int32, device=dev)
        path = torch.empty((B, T), dtype=torch.int32, device=dev)
        nxt = torch.empty(B, dtype=torch.int32, device=dev)
    else:
        alen, path, nxt = outputs
        for t, nm, shp in ((alen, "accept_len", (B,)), (path, "accept_path", (B, T)), (nxt, "next_token", (B,))):
            _need(t, nm, torch.int32, dev)
            if tuple(t.shape) != shp:
                raise ValueError("%s has the wrong shape" % nm)
    st = _stream(stream)
    nbytes = tree_accept_sampled_workspace_size(B, T, V)
    if workspace is None:
        workspace = _workspace("accept_sampled", nbytes, dev, st)
    _check(lib().dreams_tree_accept_sampled(B, T, V, float(temperature), _ptr(target_logits), _ptr(draft_logits),
                                            _ptr(draft_tokens), _ptr(parent), _ptr(uniforms), _ptr(alen),
                                            _ptr(path), _ptr(nxt), _ptr(workspace),
                                            0 if workspace is None else workspace.numel(), st))
    return alen, path, nxt


def tree_accept_lm_head_workspace_size(batch: int, num_nodes: int, hidden: int, vocab: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().dreams_tree_accept_lm_head_workspace_size(batch, num_nodes, hidden, vocab, ctypes.byref(n)))
    return n.value


def tree_accept_lm_head(hidden_states: torch.Tensor, lm_weight: torch.Tensor, draft_tokens: torch.Tensor,
                        parent: torch.Tensor, want_target_argmax: bool = False, outputs=None,
                        workspace: Optional[torch.Tensor] = None, stream=None):
    """dreams_tree_accept_lm_head.  hidden_states [B,T,H] bfloat16, lm_weight [V,H] bfloat16, draft_tokens /
    parent [B,T] int32.  Returns (accept_len [B], accept_path [B,T], next_token [B], target_argmax [B,T] or
    None), all int32.  `outputs` may pass preallocated (accept_len, accept_path, next_token, target_argmax)."""
    dev = hidden_states.device
    _need(hidden_states, "hidden_states", torch.bfloat16, dev, 3)
    B, T, H = hidden_states.shape
    _need(lm_weight, "lm_weight", torch.bfloat16, dev, 2)
    V = lm_weight.shape[0]
    if lm_weight.shape[1] != H:
        raise ValueError("lm_weight must be [V, H] with the hidden size of hidden_states")
    _need(draft_tokens, "draft_tokens", torch.int32, dev, 2)
    _need(parent, "parent", torch.int32, dev, 2)
    if tuple(draft_tokens.shape) != (B, T) or tuple(parent.shape) != (B, T):
        raise ValueError("draft_tokens and parent must be [B, T]")
    if outputs is None:
        alen = torch.empty(B, dtype=torch.int32, device=dev)
        path = torch.empty((B, T), dtype=torch.int32, device=dev)
        nxt = torch.empty(B, dtype=torch.int32, device=dev)
        am = torch.empty((B, T), dtype=torch.int32, device=dev) if want_target_argmax else None
    else:
        alen, path, nxt, am = outputs
        for t, nm, shp in ((alen, "accept_len", (B,)), (path, "accept_path", (B, T)), (nxt, "next_token", (B,))):
            _need(t, nm, torch.int32, dev)
            if tuple(t.shape) != shp:
                raise ValueError("%s has the wrong shape" % nm)
        if am is not None:
            _need(am, "target_argmax", torch.int32, dev)
    st = _stream(stream)
    nbytes = tree_accept_lm_head_workspace_size(B, T, H, V)
    if workspace is None:
        workspace = _workspace("accept_lm_head", nbytes, dev, st)
    _check(lib().dreams_tree_accept_lm_head(B, T, H, V, _ptr(hidden_states), _ptr(lm_weight), _ptr(draft_tokens),
                                            _ptr(parent), _ptr(alen), _ptr(path), _ptr(nxt), _ptr(am),
                                            _ptr(workspace), 0 if workspace is None else workspace.numel(), st))
    return alen, path, nxt, am


def kv_commit(k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len_in: torch.Tensor, accept_path: torch.Tensor,
              accept_len: torch.Tensor, kv_len_out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dreams_kv_commit, in place on k_cache / v_cache of shape [NL, B, Hkv, S_cap, D] (or [B, Hkv, S_cap, D]
    for one layer).  Returns kv_len_out [B] int32."""
    dt = k_cache.dtype
    if dt not in (torch.bfloat16, torch.float32):
        raise TypeError("caches must be bfloat16 or float32")
    dev = k_cache.device
    _need(k_cache, "k_cache", dt, dev)
    _need(v_cache, "v_cache", dt, dev)
    if k_cache.shape != v_cache.shape or k_cache.dim() not in (4, 5):
        raise ValueError("caches must share a [NL,]B,Hkv,S_cap,D shape")
    shp = k_cache.shape if k_cache.dim() == 5 else (1,) + tuple(k_cache.shape)
    NL, B, Hkv, S_cap, D = shp
    _need(kv_len_in, "kv_len_in", torch.int32, dev, 1)
    _need(accept_path, "accept_path", torch.int32, dev, 2)
    _need(accept_len, "accept_len", torch.int32, dev, 1)
    if kv_len_out is None:
        kv_len_out = torch.empty(B, dtype=torch.int32, device=dev)
    _need(kv_len_out, "kv_len_out", torch.int32, dev, 1)
    if kv_len_in.shape[0] != B or accept_len.shape[0] != B or accept_path.shape[0] != B or kv_len_out.shape[0] != B:
        raise ValueError("length / path arrays must have the cache's batch size")
    _check(lib().dreams_kv_commit(NL, B * Hkv * S_cap * D, B, Hkv, D, S_cap,
                                  DREAMS_BF16 if dt == torch.bfloat16 else DREAMS_F32, _ptr(k_cache), _ptr(v_cache),
                                  _ptr(kv_len_in), _ptr(accept_path), _ptr(accept_len), accept_path.shape[1],
                                  _ptr(kv_len_out), _stream(stream)))
    return kv_len_out


def check_tree_host(parent) -> None:
    """dreams_check_tree_host on a host int32 array; raises DreamsError if it is not a valid parent array."""
    import numpy as np
    p = np.ascontiguousarray(parent, dtype=np.int32)
    _check(lib().dreams_check_tree_host(p.ctypes.data_as(ctypes.c_void_p), int(p.shape[0])))


STREAM_READ_SINK_WORDS = 2048


def stream_read(src: torch.Tensor, sink: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dreams_stream_read: one plain read of every byte of `src` (a contiguous device tensor whose size is a
    multiple of 16 bytes), for measuring read bandwidth.  Returns the sink words."""
    if not src.is_contiguous():
        raise ValueError("src must be contiguous")
    if sink is None:
        sink = torch.empty(STREAM_READ_SINK_WORDS, dtype=torch.int32, device=src.device)
    _check(lib().dreams_stream_read(_ptr(src), src.numel() * src.element_size(), _ptr(sink), _stream(stream)))
    return sink
