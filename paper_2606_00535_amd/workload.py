"""Seeded synthetic inputs for the tree-verification workloads.

This module only *draws* inputs: tree topologies, prefix lengths, queries, keys, values, target logits and
draft tokens.  It contains none of the verification arithmetic (no attention, no acceptance, no commit), so
both the HIP path and the CPU oracle can be fed from it without sharing any of the method's code.

The generator looks at a logit row in two places, both of which only shape the *distribution* of inputs and never
produce an expected value: it plants draft tokens that agree with their parent's target argmax with a given
probability (the agreement model of the greedy workloads; ``numpy.argmax``), and, for sampled acceptance, it
draws each child's token from the draft's distribution at its parent with the Gumbel-max trick (the argmax of
the logits over the temperature plus Gumbel noise).

Shapes follow the paper's target models (LLaVA-v1.6-Vicuna-7B/13B: 32/40 heads, head_dim 128, vocabulary
32000, 2880 "anyres" image tokens held in the KV cache beside the text tokens; the paper's Section 2,
"Vision-Language Models", notes that every visual token is attended at each decoding step).  None of the
paper's benchmark data is available, so seeded Gaussian tensors of those shapes stand in for it.

Seeding: every tensor of every (layer, sequence) comes from its own PCG64 stream,
``SeedSequence(seed, spawn_key=(layer, b, tensor_id))``, so any subset can be regenerated independently.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Optional, Sequence, Tuple

import numpy as np

# tensor ids for the per-(layer, b) substreams
_T_TOPOLOGY, _T_AGREE, _T_LEN, _T_LOGITS, _T_TOKENS = 0, 1, 2, 3, 4
_T_Q, _T_KPRE, _T_VPRE, _T_KTREE, _T_VTREE = 10, 11, 12, 13, 14
_T_VARIANT = 20
_T_DRAFT, _T_DRAFT_TOKENS, _T_UNIFORMS = 30, 31, 32
_T_PROMPT_Q, _T_PROMPT_K = 40, 41


@dataclass(frozen=True)
class Workload:
    """One synthetic tree-verification workload.

    kv_len: fixed committed prefix length L, or a (lo, hi) pair for per-sequence lengths drawn uniformly
    from the integers lo..hi.  agree: draft-agreement probability, or a (lo, hi) pair for a per-sequence
    probability drawn uniformly.  q_std: standard deviation of the query entries.
    """
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str              # "f32" or "bf16"
    num_layers: int
    kv_len: object          # int or (lo, hi)
    image_tokens: int
    num_nodes: int
    depth: int
    max_branch: int
    vocab: int
    agree: object           # float or (lo, hi)
    q_std: float = 1.0
    logit_std: float = 3.0
    commit: bool = False
    seed: int = 0

    @property
    def max_kv_len(self) -> int:
        return self.kv_len[1] if isinstance(self.kv_len, tuple) else int(self.kv_len)

    @property
    def cache_capacity(self) -> int:
        n = self.max_kv_len + self.num_nodes
        return (n + 63) // 64 * 64

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads the build is measured and checked on.
WORKLOADS = {
    # 1 layer, 4 heads, head_dim 64, fp32; 576 image + 64 text tokens; 16-node depth-4 tree, branching <= 3.
    "tiny": Workload("tiny", 1, 4, 4, 64, "f32", 1, 640, 576, 16, 4, 3, 1000, 0.7,
                     q_std=1.0 / 8.0, seed=0),
    # LLaVA-1.6-7B-shaped single layer: 32 heads x 128, bf16, 2880 image + 256 text tokens, 60-node depth-6 tree.
    "llava7b_layer": Workload("llava7b_layer", 1, 32, 32, 128, "bf16", 1, 3136, 2880, 60, 6, 4, 32000, 0.7,
                              seed=1),
    # LLaVA-1.6-7B-shaped full verify pass: 32 layers, batch 4, prefix lengths U{2900..4096}, then commit.
    "llava7b_full": Workload("llava7b_full", 4, 32, 32, 128, "bf16", 32, (2900, 4096), 2880, 60, 6, 4, 32000,
                             0.7, commit=True, seed=2),
    # LLaVA-1.6-13B-shaped layer: 40 heads, batch 8, 2880 image + 1216 text, agreement U[0.5, 0.9] per sequence.
    "llava13b_layer": Workload("llava13b_layer", 8, 40, 40, 128, "bf16", 1, 4096, 2880, 60, 6, 4, 32000,
                               (0.5, 0.9), seed=3),
    # Synthetic GQA long-context: 28 query heads over 4 KV heads, batch 16, 6400 image + 1792 text tokens,
    # 128-node depth-8 trees with branching <= 6, vocabulary 152064.
    "gqa_long": Workload("gqa_long", 16, 28, 4, 128, "bf16", 1, 8192, 6400, 128, 8, 6, 152064, 0.7, seed=4),
}


def rng_for(seed: int, layer: int, b: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(layer, b, tensor_id))))


# ----------------------------------------------------------------------------------------------- bf16 helpers
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (round to nearest, ties to even); returns the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------------------------------------------- topology
def random_tree(rng: np.random.Generator, num_nodes: int, depth: int, max_branch: int) -> np.ndarray:
    """Draft-token tree as a parent array in breadth-first order (parent[0] = -1, parent[i] < i).

    A spine of `depth` nodes below the root fixes the tree depth exactly; each remaining node attaches to a
    node drawn uniformly among those with depth < `depth` and fewer than `max_branch` children.  Nodes are
    then relabelled breadth-first, children in creation order.
    """
    if num_nodes < 1:
        raise ValueError("a tree needs at least the root")
    depth = min(depth, num_nodes - 1)
    par, dep, nch = [-1], [0], [0]
    for d in range(1, depth + 1):
        par.append(d - 1)
        dep.append(d)
        nch.append(0)
        nch[d - 1] += 1
    while len(par) < num_nodes:
        elig = [i for i in range(len(par)) if dep[i] < depth and nch[i] < max_branch]
        if not elig:
            raise ValueError("tree capacity exhausted for the requested depth / branching")
        p = elig[int(rng.integers(len(elig)))]
        par.append(p)
        dep.append(dep[p] + 1)
        nch.append(0)
        nch[p] += 1
    children = [[] for _ in par]
    for i in range(1, len(par)):
        children[par[i]].append(i)
    order, head = [0], 0
    while head < len(order):
        order.extend(children[order[head]])
        head += 1
    new_id = {old: new for new, old in enumerate(order)}
    out = np.empty(num_nodes, dtype=np.int32)
    for old in order:
        out[new_id[old]] = -1 if par[old] < 0 else new_id[par[old]]
    return out


def chain_tree(num_nodes: int) -> np.ndarray:
    return np.arange(-1, num_nodes - 1, dtype=np.int32)


def star_tree(num_nodes: int) -> np.ndarray:
    p = np.zeros(num_nodes, dtype=np.int32)
    p[0] = -1
    return p


# ------------------------------------------------------------------------------------------------ the batch
@dataclass
class Batch:
    """All inputs of one verify step.  Arrays are numpy; bf16 tensors are stored as uint16 bit patterns.

    q:        [NL, B, Hq, T, D]
    k_cache:  [NL, B, Hkv, S_cap, D]   slots [0, L_b) = committed prefix, [L_b, L_b+T) = the tree's own K/V
    v_cache:  same
    kv_len:   [B] int32   committed prefix length L_b
    parent:   [B, T] int32
    logits:   [B, T, V] float32  target logits at every tree node
    tokens:   [B, T] int32       draft token of every node (tokens[b, 0] is the already-emitted root token)
    """
    wl: Workload
    q: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    kv_len: np.ndarray
    parent: np.ndarray
    logits: Optional[np.ndarray]
    tokens: Optional[np.ndarray]
    agree_p: np.ndarray

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.wl.head_dim))

    def as_f32(self, name: str) -> np.ndarray:
        a = getattr(self, name)
        return bf16_bits_to_f32(a) if a.dtype == np.uint16 else a


def _draw(rng: np.random.Generator, shape, std: float, dtype: str) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x) if dtype == "bf16" else x


def make_batch(wl: Workload, *, layers: Optional[Sequence[int]] = None, with_logits: bool = True,
               parents: Optional[np.ndarray] = None, kv_lens: Optional[Sequence[int]] = None) -> Batch:
    """Draw one verify step of workload `wl`.

    layers: subset of layer indices to materialise (default all); the arrays then hold only those layers,
            in the given order, drawn from exactly the streams the full set would use.
    parents / kv_lens: override the drawn topology / prefix lengths (used by invariant tests).
    """
    B, T, D = wl.batch, wl.num_nodes, wl.head_dim
    layers = list(range(wl.num_layers)) if layers is None else list(layers)
    S = wl.cache_capacity
    parent = np.empty((B, T), dtype=np.int32)
    kv_len = np.empty(B, dtype=np.int32)
    agree_p = np.empty(B, dtype=np.float64)
    for b in range(B):
        parent[b] = random_tree(rng_for(wl.seed, 0, b, _T_TOPOLOGY), T, wl.depth, wl.max_branch) \
            if parents is None else np.asarray(parents[b], dtype=np.int32)
        if isinstance(wl.agree, tuple):
            agree_p[b] = rng_for(wl.seed, 0, b, _T_AGREE).uniform(wl.agree[0], wl.agree[1])
        else:
            agree_p[b] = float(wl.agree)
        if kv_lens is not None:
            kv_len[b] = int(kv_lens[b])
        elif isinstance(wl.kv_len, tuple):
            kv_len[b] = int(rng_for(wl.seed, 0, b, _T_LEN).integers(wl.kv_len[0], wl.kv_len[1] + 1))
        else:
            kv_len[b] = int(wl.kv_len)
    if int(kv_len.max(initial=0)) + T > S:
        S = (int(kv_len.max()) + T + 63) // 64 * 64

    logits = tokens = None
    if with_logits:
        V = wl.vocab
        logits = np.empty((B, T, V), dtype=np.float32)
        tokens = np.empty((B, T), dtype=np.int32)
        for b in range(B):
            logits[b] = rng_for(wl.seed, 0, b, _T_LOGITS).standard_normal((T, V), dtype=np.float32)
            logits[b] *= np.float32(wl.logit_std)
            am = np.argmax(logits[b], axis=1)          # agreement model only (see module docstring)
            r = rng_for(wl.seed, 0, b, _T_TOKENS)
            uni = r.integers(0, V, size=T)
            hit = r.random(T) < agree_p[b]
            tokens[b, 0] = uni[0]
            for i in range(1, T):
                tokens[b, i] = am[parent[b, i]] if hit[i] else uni[i]

    edt = np.uint16 if wl.dtype == "bf16" else np.float32
    NLs = len(layers)
    q = np.empty((NLs, B, wl.num_q_heads, T, D), dtype=edt)
    kc = np.zeros((NLs, B, wl.num_kv_heads, S, D), dtype=edt)
    vc = np.zeros((NLs, B, wl.num_kv_heads, S, D), dtype=edt)
    Hkv = wl.num_kv_heads
    for li, layer in enumerate(layers):
        for b in range(B):
            L = int(kv_len[b])
            q[li, b] = _draw(rng_for(wl.seed, layer, b, _T_Q), (wl.num_q_heads, T, D), wl.q_std, wl.dtype)
            kc[li, b, :, :L] = _draw(rng_for(wl.seed, layer, b, _T_KPRE), (Hkv, L, D), 1.0, wl.dtype)
            vc[li, b, :, :L] = _draw(rng_for(wl.seed, layer, b, _T_VPRE), (Hkv, L, D), 1.0, wl.dtype)
            kc[li, b, :, L:L + T] = _draw(rng_for(wl.seed, layer, b, _T_KTREE), (Hkv, T, D), 1.0, wl.dtype)
            vc[li, b, :, L:L + T] = _draw(rng_for(wl.seed, layer, b, _T_VTREE), (Hkv, T, D), 1.0, wl.dtype)
    return Batch(wl, q, kc, vc, kv_len, parent, logits, tokens, agree_p)


# ------------------------------------------------------------------------------------- harder input variants
def make_tree_dominant(batch: Batch, logit_boost: float = 8.0, seed: int = 99) -> Batch:
    """Mask-sensitive variant: every tree key gets a shared direction u added, and every query gets u too,
    scaled so the tree keys' scores exceed the prefix keys' by about `logit_boost`.  The visible tree keys
    then carry most of the softmax mass, so including a non-ancestor or dropping an ancestor changes the
    output by O(1) instead of by the ~0.2% a plain Gaussian input would show."""
    wl = batch.wl
    D = wl.head_dim
    r = rng_for(seed, 0, 0, _T_VARIANT)
    u = r.standard_normal(D)
    u /= np.linalg.norm(u)
    # scale * (a*u).(c*u) = scale * a * c = logit_boost, with a = c
    a = np.sqrt(logit_boost * np.sqrt(D))
    q = batch.as_f32("q").copy()
    k = batch.as_f32("k_cache").copy()
    q += (a * u).astype(np.float32)
    for b in range(wl.batch):
        L = int(batch.kv_len[b])
        k[:, b, :, L:L + wl.num_nodes] += (a * u).astype(np.float32)
    conv = f32_to_bf16_bits if wl.dtype == "bf16" else (lambda x: x.astype(np.float32))
    return dataclasses.replace(batch, q=conv(q), k_cache=conv(k))


def make_sharp(batch: Batch, q_gain: float = 4.0) -> Batch:
    """Sharp-softmax variant: queries multiplied by `q_gain` (logit std grows by the same factor)."""
    q = batch.as_f32("q") * np.float32(q_gain)
    conv = f32_to_bf16_bits if batch.wl.dtype == "bf16" else (lambda x: x.astype(np.float32))
    return dataclasses.replace(batch, q=conv(q))


def tree_depths_for_generator_checks(parent: np.ndarray) -> np.ndarray:
    """Depth of each node (used only to check the generator's own output: spine depth, branching)."""
    d = np.zeros(len(parent), dtype=np.int32)
    for i in range(1, len(parent)):
        d[i] = d[parent[i]] + 1
    return d


# ------------------------------------------------------------------------------------- sampled acceptance
@dataclass
class SampledInputs:
    """Inputs of sampled acceptance for one verify step.

    target_logits, draft_logits: [B, T, V] float32; tokens, parent: [B, T] int32; uniforms: [B, T] float32 in
    [0, 1) (entry 0 draws the emitted token, entry c decides child c); temperature: the one both were drawn for.
    """
    target_logits: np.ndarray
    draft_logits: np.ndarray
    tokens: np.ndarray
    parent: np.ndarray
    uniforms: np.ndarray
    temperature: float


def make_sampled(wl: Workload, *, temperature: float = 1.0, draft_noise: float = 1.0,
                 parents: Optional[np.ndarray] = None, target_logits: Optional[np.ndarray] = None) -> SampledInputs:
    """Draw sampled-acceptance inputs for workload `wl`.

    Target logits are those of make_batch (N(0, logit_std), same streams) unless given; the draft's logits are
    the target's plus N(0, draft_noise) noise (a draft that approximates the target); every child's token is a
    sample of softmax(draft_logits[parent] / temperature), drawn by the Gumbel-max trick; the root's token is
    uniform.  Uniforms are float32 in [0, 1).
    """
    B, T, V = wl.batch, wl.num_nodes, wl.vocab
    parent = np.empty((B, T), dtype=np.int32)
    for b in range(B):
        parent[b] = random_tree(rng_for(wl.seed, 0, b, _T_TOPOLOGY), T, wl.depth, wl.max_branch) \
            if parents is None else np.asarray(parents[b], dtype=np.int32)
    tl = np.empty((B, T, V), dtype=np.float32) if target_logits is None else np.asarray(target_logits, np.float32)
    dl = np.empty((B, T, V), dtype=np.float32)
    tokens = np.empty((B, T), dtype=np.int32)
    uniforms = np.empty((B, T), dtype=np.float32)
    for b in range(B):
        if target_logits is None:
            tl[b] = rng_for(wl.seed, 0, b, _T_LOGITS).standard_normal((T, V), dtype=np.float32)
            tl[b] *= np.float32(wl.logit_std)
        noise = rng_for(wl.seed, 0, b, _T_DRAFT).standard_normal((T, V), dtype=np.float32)
        dl[b] = tl[b] + np.float32(draft_noise) * noise
        r = rng_for(wl.seed, 0, b, _T_DRAFT_TOKENS)
        tokens[b, 0] = r.integers(0, V)
        for i in range(1, T):
            with np.errstate(divide="ignore"):   # a uniform of exactly 0 gives -inf noise: never drawn
                g = -np.log(-np.log(r.random(V, dtype=np.float32)))
            tokens[b, i] = int(np.argmax(dl[b, parent[b, i]] / np.float32(temperature) + g))
        uniforms[b] = rng_for(wl.seed, 0, b, _T_UNIFORMS).random(T, dtype=np.float32)
    return SampledInputs(tl, dl, tokens, parent, uniforms, float(temperature))


# ------------------------------------------------------------------------------------------- prompt (prefill)
@dataclasses.dataclass
class Prompt:
    """A prefilling pass's query and key rows: q [B, Hq, N, D] and k_cache [B, Hkv, S_cap, D] (bf16 bits), the
    prompt of sequence b in rows / slots 0..prompt_len[b]-1 (the rest of q is drawn too, the rest of the cache
    is zero), and the visual-token window [vis_begin, vis_begin + vis_count) inside it."""
    q: np.ndarray
    k_cache: np.ndarray
    prompt_len: np.ndarray
    vis_begin: int
    vis_count: int
    num_kv_heads: int

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.q.shape[3]))


def make_prompt(batch: int, num_q_heads: int, num_kv_heads: int, head_dim: int, prompt_lens: Sequence[int],
                vis_begin: int, vis_count: int, *, num_rows: Optional[int] = None, cache_capacity: Optional[int] = None,
                q_std: float = 1.0, seed: int = 0) -> Prompt:
    """Seeded N(0, q_std^2) queries and N(0, 1) keys of every prompt position, rounded to bf16, one stream per
    (sequence, tensor).  num_rows defaults to the longest prompt, cache_capacity to num_rows rounded up to 64."""
    lens = np.asarray(prompt_lens, dtype=np.int32)
    N = int(num_rows if num_rows is not None else max(1, int(lens.max(initial=1))))
    S = int(cache_capacity if cache_capacity is not None else (N + 63) // 64 * 64)
    q = np.empty((batch, num_q_heads, N, head_dim), dtype=np.uint16)
    k = np.zeros((batch, num_kv_heads, S, head_dim), dtype=np.uint16)
    for b in range(batch):
        q[b] = _draw(rng_for(seed, 0, b, _T_PROMPT_Q), (num_q_heads, N, head_dim), q_std, "bf16")
        n = int(min(max(lens[b], 0), N))
        k[b, :, :n] = _draw(rng_for(seed, 0, b, _T_PROMPT_K), (num_kv_heads, n, head_dim), 1.0, "bf16")
    return Prompt(q, k, lens, int(vis_begin), int(vis_count), int(num_kv_heads))
