"""CPU oracle for the tree-verification step -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the package smoke check and the benchmark's CPU-baseline leg may import this package.
The product (the HIP library and its Python binding) never imports, links or calls it.

Thin ctypes wrapper over ``oracle.c`` (plain C, fp64 accumulation; that file states what each function
computes and which passage of the paper it follows), plus a few plain numpy definitions at the end of this
file (the layer mean and choice of the attention entropy, the LM head's logits in fp64, the greedy rule on
given per-node tokens).  The shared library is built with gcc by :func:`build` -- no hipcc, no header shared
with the HIP path.  :class:`Oracle` can also wrap a differently built copy of
the source (the mutation tests compile copies with planted mistakes to show that the pins catch them).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_DIR = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_DIR, "oracle.c")
LIBRARY = os.path.join(_DIR, "liboracle.so")


def compile_source(src_path: str, lib_path: str) -> str:
    """Compile an oracle C source with gcc -O2 (no fast-math) and OpenMP into a shared library."""
    tmp = lib_path + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
                           "-o", tmp, src_path, "-lm"])
    os.replace(tmp, lib_path)
    return lib_path


def build(force: bool = True) -> str:
    """Build liboracle.so next to oracle.c."""
    if force or not os.path.exists(LIBRARY):
        compile_source(SOURCE, LIBRARY)
    return LIBRARY


class OracleError(RuntimeError):
    pass


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return None if a is None else np.ascontiguousarray(a, dtype=dtype)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError("%s failed with code %d" % (what, rc))


class Oracle:
    """The oracle's entry points over one built library."""

    def __init__(self, lib_path: str):
        lib = ctypes.CDLL(lib_path)
        P, I = ctypes.c_void_p, ctypes.c_int
        lib.oracle_tree_attn.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, P, P, P, P, P]
        lib.oracle_tree_attn_rows.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, P, P, P, I, P, P, P]
        lib.oracle_tree_accept.argtypes = [I, I, I, P, P, P, P, P, P, P]
        lib.oracle_kv_commit.argtypes = [I, ctypes.c_int64, I, I, I, I, I, P, P, P, P, P, I, P]
        lib.oracle_tree_attn_entropy.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, P, P, P]
        lib.oracle_tree_accept_sampled.argtypes = [I, I, I, ctypes.c_double, P, P, P, P, P, P, P, P]
        lib.oracle_tree_accept_sampled.restype = ctypes.c_int
        lib.oracle_visual_importance.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, P, P, I, I, P]
        lib.oracle_visual_topk.argtypes = [I, I, I, P, P]
        lib.oracle_visual_gather.argtypes = [I, I, I, I, I, P, P, I, P, I, P, P]
        lib.oracle_prefill_attn_stats.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, P, P]
        lib.oracle_prefill_visual_importance.argtypes = [I, I, I, I, I, I, ctypes.c_double, P, P, P, I, I, P]
        for f in (lib.oracle_tree_attn, lib.oracle_tree_attn_rows, lib.oracle_tree_accept, lib.oracle_kv_commit,
                  lib.oracle_tree_attn_entropy, lib.oracle_visual_importance, lib.oracle_visual_topk,
                  lib.oracle_visual_gather, lib.oracle_prefill_attn_stats, lib.oracle_prefill_visual_importance):
            f.restype = ctypes.c_int
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        lib.oracle_set_num_threads.argtypes = [I]
        lib.oracle_set_num_threads.restype = None
        self.lib = lib
        self.path = lib_path

    def num_threads(self) -> int:
        return int(self.lib.oracle_num_threads())

    def set_num_threads(self, n: int) -> None:
        self.lib.oracle_set_num_threads(int(n))

    def tree_attn(self, q, k_cache, v_cache, kv_len, parent, scale: float, num_kv_heads: int,
                  tree_mask=None, with_lse: bool = True):
        """q [B,Hq,T,D]; k/v [B,Hkv,S_cap,D] (fp32 values); kv_len [B]; parent [B,T] (or None together with
        tree_mask [B,T,ceil(T/64)] uint64).  Returns (out [B,Hq,T,D] float64, lse [B,Hq,T] float64)."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        v_cache = _c(v_cache, np.float32)
        B, Hq, T, D = q.shape
        S_cap = k_cache.shape[2]
        assert k_cache.shape == (B, num_kv_heads, S_cap, D) and v_cache.shape == k_cache.shape
        kv_len = _c(kv_len, np.int32)
        parent = _c(parent, np.int32)
        tree_mask = _c(tree_mask, np.uint64)
        out = np.empty((B, Hq, T, D), dtype=np.float64)
        lse = np.empty((B, Hq, T), dtype=np.float64) if with_lse else None
        rc = self.lib.oracle_tree_attn(B, Hq, num_kv_heads, T, D, S_cap, float(scale), _p(q), _p(k_cache),
                                       _p(v_cache), _p(kv_len), _p(parent), _p(tree_mask), _p(out), _p(lse))
        _check(rc, "oracle_tree_attn")
        return out, lse

    def tree_attn_rows(self, q, k_cache, v_cache, kv_len, parent, scale: float, num_kv_heads: int, rows,
                       tree_mask=None):
        """Selected rows only: rows is an [n, 3] array of (b, h, i).  Returns (out [n, D], lse [n])."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        v_cache = _c(v_cache, np.float32)
        B, Hq, T, D = q.shape
        S_cap = k_cache.shape[2]
        rows = _c(rows, np.int32).reshape(-1, 3)
        kv_len = _c(kv_len, np.int32)
        parent = _c(parent, np.int32)
        tree_mask = _c(tree_mask, np.uint64)
        out = np.empty((rows.shape[0], D), dtype=np.float64)
        lse = np.empty(rows.shape[0], dtype=np.float64)
        rc = self.lib.oracle_tree_attn_rows(B, Hq, num_kv_heads, T, D, S_cap, float(scale), _p(q),
                                            _p(k_cache), _p(v_cache), _p(kv_len), _p(parent), _p(tree_mask),
                                            rows.shape[0], _p(rows), _p(out), _p(lse))
        _check(rc, "oracle_tree_attn_rows")
        return out, lse

    def tree_attn_entropy(self, q, k_cache, kv_len, parent, scale: float, num_kv_heads: int, tree_mask=None):
        """Attention entropy (nats) of every row, [B,Hq,T] float64: -sum_j A_ij log A_ij over the row's visible
        slots (the per-row term of the paper's average attention entropy AE, Section 3.2)."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        B, Hq, T, D = q.shape
        S_cap = k_cache.shape[2]
        assert k_cache.shape == (B, num_kv_heads, S_cap, D)
        ent = np.empty((B, Hq, T), dtype=np.float64)
        rc = self.lib.oracle_tree_attn_entropy(B, Hq, num_kv_heads, T, D, S_cap, float(scale), _p(q), _p(k_cache),
                                               _p(_c(kv_len, np.int32)), _p(_c(parent, np.int32)),
                                               _p(_c(tree_mask, np.uint64)), _p(ent))
        _check(rc, "oracle_tree_attn_entropy")
        return ent

    def visual_importance(self, q, k_cache, kv_len, parent, scale: float, num_kv_heads: int, vis_begin: int,
                          vis_count: int, tree_mask=None):
        """Importance of visual tokens vis_begin.. (Eq. 2, Section 3.1): [B, vis_count] float64."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        B, Hq, T, D = q.shape
        S_cap = k_cache.shape[2]
        assert k_cache.shape == (B, num_kv_heads, S_cap, D)
        imp = np.empty((B, vis_count), dtype=np.float64)
        rc = self.lib.oracle_visual_importance(B, Hq, num_kv_heads, T, D, S_cap, float(scale), _p(q), _p(k_cache),
                                               _p(_c(kv_len, np.int32)), _p(_c(parent, np.int32)),
                                               _p(_c(tree_mask, np.uint64)), int(vis_begin), int(vis_count), _p(imp))
        _check(rc, "oracle_visual_importance")
        return imp

    def prefill_attn_stats(self, q, k_cache, prompt_len, scale: float, num_kv_heads: int):
        """Causal attention of a prompt's own rows (row i sees slots 0..i): (lse, entropy), each [B, Hq, N]
        float64; rows at or past prompt_len[b] get -inf and 0."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        B, Hq, N, D = q.shape
        S_cap = k_cache.shape[2]
        assert k_cache.shape == (B, num_kv_heads, S_cap, D)
        lse = np.empty((B, Hq, N), dtype=np.float64)
        ent = np.empty((B, Hq, N), dtype=np.float64)
        rc = self.lib.oracle_prefill_attn_stats(B, Hq, num_kv_heads, N, D, S_cap, float(scale), _p(q), _p(k_cache),
                                                _p(_c(prompt_len, np.int32)), _p(lse), _p(ent))
        _check(rc, "oracle_prefill_attn_stats")
        return lse, ent

    def prefill_visual_importance(self, q, k_cache, prompt_len, scale: float, num_kv_heads: int, vis_begin: int,
                                  vis_count: int):
        """Eq. 2 over a prompt's causal attention: [B, vis_count] float64."""
        q = _c(q, np.float32)
        k_cache = _c(k_cache, np.float32)
        B, Hq, N, D = q.shape
        S_cap = k_cache.shape[2]
        assert k_cache.shape == (B, num_kv_heads, S_cap, D)
        imp = np.empty((B, vis_count), dtype=np.float64)
        rc = self.lib.oracle_prefill_visual_importance(B, Hq, num_kv_heads, N, D, S_cap, float(scale), _p(q),
                                                       _p(k_cache), _p(_c(prompt_len, np.int32)), int(vis_begin),
                                                       int(vis_count), _p(imp))
        _check(rc, "oracle_prefill_visual_importance")
        return imp

    def visual_topk(self, importance, r: int):
        """Indices of the r most important tokens per sequence (ties: smaller index), increasing: [B, r]."""
        imp = _c(importance, np.float32)
        B, n = imp.shape
        keep = np.empty((B, r), dtype=np.int32)
        _check(self.lib.oracle_visual_topk(B, n, int(r), _p(imp), _p(keep)), "oracle_visual_topk")
        return keep

    def visual_gather(self, k_cache, v_cache, vis_begin: int, keep):
        """k_cache/v_cache [B, Hkv, S_cap, D] (uint16 bf16 bits or float32) -> (k_out, v_out) [B, Hkv, r, D]."""
        assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous and k_cache.shape == v_cache.shape
        B, Hkv, S_cap, D = k_cache.shape
        keep = _c(keep, np.int32)
        r = keep.shape[1]
        ko = np.empty((B, Hkv, r, D), dtype=k_cache.dtype)
        vo = np.empty_like(ko)
        _check(self.lib.oracle_visual_gather(B, Hkv, D, S_cap, k_cache.dtype.itemsize, _p(k_cache), _p(v_cache),
                                             int(vis_begin), _p(keep), r, _p(ko), _p(vo)), "oracle_visual_gather")
        return ko, vo

    def tree_accept_sampled(self, target_logits, draft_logits, tokens, parent, uniforms, temperature: float):
        """Sampled tree acceptance.  Returns (accept_len [B], accept_path [B,T], next_token [B]), int32."""
        tl = _c(target_logits, np.float32)
        B, T, V = tl.shape
        dl = _c(draft_logits, np.float32)
        assert dl.shape == tl.shape
        alen = np.empty(B, dtype=np.int32)
        path = np.empty((B, T), dtype=np.int32)
        nxt = np.empty(B, dtype=np.int32)
        rc = self.lib.oracle_tree_accept_sampled(B, T, V, float(temperature), _p(tl), _p(dl),
                                                 _p(_c(tokens, np.int32)), _p(_c(parent, np.int32)),
                                                 _p(_c(uniforms, np.float32)), _p(alen), _p(path), _p(nxt))
        _check(rc, "oracle_tree_accept_sampled")
        return alen, path, nxt

    def tree_accept(self, logits, tokens, parent):
        """Returns (accept_len [B], accept_path [B,T], next_token [B], target_argmax [B,T]), all int32."""
        logits = _c(logits, np.float32)
        B, T, V = logits.shape
        tokens = _c(tokens, np.int32)
        parent = _c(parent, np.int32)
        alen = np.empty(B, dtype=np.int32)
        path = np.empty((B, T), dtype=np.int32)
        nxt = np.empty(B, dtype=np.int32)
        am = np.empty((B, T), dtype=np.int32)
        rc = self.lib.oracle_tree_accept(B, T, V, _p(logits), _p(tokens), _p(parent), _p(alen), _p(path),
                                         _p(nxt), _p(am))
        _check(rc, "oracle_tree_accept")
        return alen, path, nxt, am

    def kv_commit(self, k_cache: np.ndarray, v_cache: np.ndarray, kv_len_in, accept_path, accept_len):
        """In place on k_cache / v_cache of shape [NL, B, Hkv, S_cap, D] (uint16 bf16 bits or float32).
        Returns kv_len_out [B]."""
        assert k_cache.flags.c_contiguous and v_cache.flags.c_contiguous and k_cache.shape == v_cache.shape
        NL, B, Hkv, S_cap, D = k_cache.shape
        accept_path = _c(accept_path, np.int32)
        out = np.empty(B, dtype=np.int32)
        rc = self.lib.oracle_kv_commit(NL, B * Hkv * S_cap * D, B, Hkv, D, S_cap, k_cache.dtype.itemsize,
                                       _p(k_cache), _p(v_cache), _p(_c(kv_len_in, np.int32)), _p(accept_path),
                                       _p(_c(accept_len, np.int32)), accept_path.shape[1], _p(out))
        _check(rc, "oracle_kv_commit")
        return out


_default: Optional[Oracle] = None


def default() -> Oracle:
    global _default
    if _default is None:
        if not os.path.exists(LIBRARY):
            build(force=False)
        _default = Oracle(LIBRARY)
    return _default


def num_threads() -> int:
    return default().num_threads()


def set_num_threads(n: int) -> None:
    default().set_num_threads(n)


def tree_attn(*a, **kw):
    return default().tree_attn(*a, **kw)


def tree_attn_rows(*a, **kw):
    return default().tree_attn_rows(*a, **kw)


def tree_accept(*a, **kw):
    return default().tree_accept(*a, **kw)


def kv_commit(*a, **kw):
    return default().kv_commit(*a, **kw)


def tree_attn_entropy(*a, **kw):
    return default().tree_attn_entropy(*a, **kw)


def tree_accept_sampled(*a, **kw):
    return default().tree_accept_sampled(*a, **kw)


def visual_importance(*a, **kw):
    return default().visual_importance(*a, **kw)


def visual_topk(*a, **kw):
    return default().visual_topk(*a, **kw)


def visual_gather(*a, **kw):
    return default().visual_gather(*a, **kw)


def prefill_attn_stats(*a, **kw):
    return default().prefill_attn_stats(*a, **kw)


def prefill_visual_importance(*a, **kw):
    return default().prefill_visual_importance(*a, **kw)


def prefill_attn_entropy_mean(entropy, prompt_len) -> float:
    """AE of one layer over prompts (Section 3.2): the mean of the entropies of the prompt rows i < n_b of every
    head and sequence (entropy [B, Hq, N]), summed in fp64."""
    e = np.asarray(entropy, dtype=np.float64)
    n = np.asarray(prompt_len, dtype=np.int64)
    total, count = 0.0, 0
    for b in range(e.shape[0]):
        total += float(e[b, :, :n[b]].sum())
        count += e.shape[1] * int(n[b])
    if count == 0:
        raise OracleError("prefill_attn_entropy_mean of no rows")
    return total / count


def attn_entropy_mean(entropy) -> float:
    """AE of one layer (Section 3.2): the mean of its rows' attention entropies (rows of every head and
    sequence alike), summed in fp64."""
    e = np.asarray(entropy, dtype=np.float64).ravel()
    if e.size == 0:
        raise OracleError("attn_entropy_mean of no rows")
    return float(e.sum() / e.size)


def attn_entropy_select(ae) -> int:
    """The distillation layer of Section 3.2: the layer l minimising AE(l) + |AE(l) - AE(l-1)|.  Only layers
    with a predecessor are candidates (the change is undefined for the first), so l runs over 1..NL-1; the
    scores are formed in fp32 from fp32 AE values and ties go to the smallest l."""
    ae = np.asarray(ae, dtype=np.float32).ravel()
    if ae.size < 2:
        raise OracleError("attn_entropy_select needs at least two layers")
    best, best_score = -1, None
    for l in range(1, ae.size):
        score = np.float32(ae[l] + np.float32(abs(np.float32(ae[l] - ae[l - 1]))))
        if best_score is None or score < best_score:
            best, best_score = l, score
    return best


def lm_head_logits(hidden_bits, weight_bits) -> np.ndarray:
    """The target's logits from its final hidden states and its LM head (Section 2, "Speculative decoding":
    the target's token at a position is the argmax of these): logit[..., v] = sum_k hidden[..., k] *
    weight[v, k].  Inputs are bfloat16 bit patterns (uint16), decoded exactly; products and sums in fp64, the
    one library step being numpy's matrix product.  hidden_bits [..., H], weight_bits [V, H] -> fp64 [..., V]."""
    def decode(bits):
        b = np.ascontiguousarray(bits, dtype=np.uint16)
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    h = decode(hidden_bits)
    w = decode(weight_bits)
    return h @ w.T


def tree_accept_from_argmax(target_argmax, tokens, parent):
    """The greedy rule (oracle_tree_accept) on given per-node target tokens: one-hot logits at those tokens.
    target_argmax, tokens, parent [B, T] int -> (accept_len, accept_path, next_token)."""
    am = np.asarray(target_argmax, dtype=np.int64)
    B, T = am.shape
    V = int(max(am.max(initial=0), np.asarray(tokens).max(initial=0))) + 1
    onehot = np.zeros((B, T, V), dtype=np.float32)
    np.put_along_axis(onehot, am[:, :, None], 1.0, axis=2)
    alen, path, nxt, _ = default().tree_accept(onehot, tokens, parent)
    return alen, path, nxt
