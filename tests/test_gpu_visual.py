"""GPU parity of target-aware visual-token selection (Eq. 2 importance, top-r, K/V gather) against the CPU
oracle on the same seeded inputs.

Importance tolerance (gpu_util.IMPORTANCE_REL_TOL, 3e-5 relative, plus 1e-9 absolute for the zeros): each term
A = 2^(s*c - lse2) comes from an fp32 score (a 128-term fp32 dot product of the same bf16 values the oracle widens
to fp64) and the attention call's fp32 log-sum-exp; both errors are a few 1e-6 in the exponent, i.e. a relative
error of a few 1e-6 per term, and the fp32 sums over <= 8192 rows add less.  The tests report the observed
maximum.
Top-r is bit-exact on the same fp32 importances; end to end, where two candidates are closer than the
tolerance, any valid choice between them is accepted.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import IMPORTANCE_ABS_TOL as ABS_TOL, IMPORTANCE_REL_TOL as REL_TOL, device, f32, layer_tensors, note
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def small_wl(**kw):
    base = dict(name="small", batch=2, num_q_heads=4, num_kv_heads=2, head_dim=128, dtype="bf16", num_layers=1,
                kv_len=300, image_tokens=0, num_nodes=16, depth=4, max_branch=3, vocab=64, agree=0.7, seed=31)
    base.update(kw)
    return W.Workload(**base)


def gpu_importance(batch, dev, vis_begin, vis_count, splits=0):
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits)
    imp = dreams.visual_importance(q, k, kv, lse, vis_begin, vis_count)
    torch.cuda.synchronize()
    return imp.cpu().numpy().astype(np.float64)


def oracle_importance(batch, vis_begin, vis_count):
    return oracle.visual_importance(f32(batch.q[0]), f32(batch.k_cache[0]), batch.kv_len, batch.parent, batch.scale,
                                    batch.wl.num_kv_heads, vis_begin, vis_count)


CASES = [  # (D, Hq, Hkv, T, L, vis_begin, vis_count): the second sequence's prefix is 37 shorter
    (128, 4, 2, 16, 300, 0, 300),      # the first sequence's whole prefix; the tail is past the second's
    (128, 32, 32, 60, 700, 20, 600),   # MHA, a window inside the prefix
    (128, 28, 4, 128, 500, 0, 450),    # GQA, 7 heads per KV head, 128 nodes
    (64, 8, 8, 33, 257, 1, 255),       # head_dim 64, ragged 64-token blocks
    (128, 2, 1, 1, 90, 0, 120),        # one node; tokens past both prefixes have importance 0
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "D%d_Hq%d_Hkv%d_T%d_L%d_v%d+%d" % c)
def test_importance_parity(dev, case):
    D, Hq, Hkv, T, L, v0, nv = case
    wl = small_wl(head_dim=D, num_q_heads=Hq, num_kv_heads=Hkv, num_nodes=T, depth=min(6, T - 1) if T > 1 else 0,
                  max_branch=3 if T > 1 else 1, kv_len=L)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[L, L - 37])
    note("importance %s" % (case,))
    got = gpu_importance(batch, dev, v0, nv)
    ref = oracle_importance(batch, v0, nv)
    err = np.abs(got - ref)
    rel = float(np.max(err / (np.abs(ref) + 1e-30)))
    note("importance %s: max rel %.3e, max abs %.3e, sum %.4f" % (case, rel, float(err.max()), float(ref[0].sum())))
    assert np.all(err <= REL_TOL * np.abs(ref) + ABS_TOL)
    for b in range(2):
        assert np.all(got[b, max(0, int(batch.kv_len[b]) - v0):] == 0.0)


def test_importance_repeat_and_counters_left_zero(dev):
    wl = small_wl(num_q_heads=12, num_kv_heads=4, num_nodes=40, depth=5, max_branch=4, kv_len=900, batch=3)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    nbytes = dreams.visual_importance_workspace_size(3, 4, 850)
    ws = torch.zeros(nbytes, dtype=torch.uint8, device=dev)
    first = None
    for rep in range(4):
        imp = dreams.visual_importance(q, k, kv, lse, 40, 850, workspace=ws)
        torch.cuda.synchronize()
        cur = imp.cpu().numpy()
        if first is None:
            first = cur
        else:
            assert np.array_equal(cur, first), rep   # heads summed in a fixed order: bit-identical repeats
    assert nbytes == 65536 + 3 * 4 * 850 * 4
    assert not ws[:65536].cpu().numpy().any()
    # a workspace shared with calls of other shapes (and other verbs) stays valid: the counter region has a
    # fixed size, so partial sums of a larger call never land where a later call keeps its counters
    dreams.visual_importance(q, k, kv, lse, 0, 940)
    again = dreams.visual_importance(q, k, kv, lse, 40, 850)
    torch.cuda.synchronize()
    assert np.array_equal(again.cpu().numpy(), first)


def test_topk_bit_exact_with_ties(dev):
    rng = np.random.default_rng(7)
    for n in (1, 2, 63, 64, 65, 1000, 2880, 4097, 8192):
        vals = (rng.integers(0, 40, size=(3, n)) / 8.0).astype(np.float32)   # many exact ties
        for r in sorted({1, n, max(1, n // 5), max(1, n - 1)}):
            keep = dreams.visual_topk(torch.from_numpy(vals).to(dev), r)
            torch.cuda.synchronize()
            ref = oracle.visual_topk(vals, r)
            assert np.array_equal(keep.cpu().numpy(), ref), (n, r)
    note("top-r: bit-exact on tied values, n up to 8192")


def test_gather_bit_exact(dev):
    rng = np.random.default_rng(8)
    for dt, D in ((torch.bfloat16, 128), (torch.bfloat16, 64), (torch.float32, 64)):
        B, Hkv, S, v0, r = 3, 4, 500, 17, 77
        npdt = np.uint16 if dt == torch.bfloat16 else np.float32
        if dt == torch.bfloat16:
            kc = rng.integers(0, 65536, size=(B, Hkv, S, D), dtype=np.uint16)
            vc = rng.integers(0, 65536, size=(B, Hkv, S, D), dtype=np.uint16)
            kt = torch.from_numpy(kc.view(np.int16)).to(dev).view(torch.bfloat16)
            vt = torch.from_numpy(vc.view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            kc = rng.standard_normal((B, Hkv, S, D)).astype(npdt)
            vc = rng.standard_normal((B, Hkv, S, D)).astype(npdt)
            kt, vt = torch.from_numpy(kc).to(dev), torch.from_numpy(vc).to(dev)
        keep = np.sort(np.stack([rng.choice(S - v0, r, replace=False) for _ in range(B)]), axis=1).astype(np.int32)
        ko, vo = dreams.visual_gather(kt, vt, v0, torch.from_numpy(keep).to(dev))
        torch.cuda.synchronize()
        rk, rv = oracle.visual_gather(kc, vc, v0, keep)
        if dt == torch.bfloat16:
            gk, gv = ko.cpu().view(torch.int16).numpy().view(np.uint16), vo.cpu().view(torch.int16).numpy().view(np.uint16)
        else:
            gk, gv = ko.cpu().numpy(), vo.cpu().numpy()
        assert np.array_equal(gk.view(np.uint8), rk.view(np.uint8)) and np.array_equal(gv.view(np.uint8), rv.view(np.uint8))


def check_selection(keep, ref_imp, r):
    """keep (device choice) against the oracle's importances: identical to the oracle's own choice unless the
    r-th and (r+1)-th candidates are within the tolerance, and in any case no kept token is clearly below a
    dropped one."""
    n = ref_imp.shape[0]
    ref_keep = oracle.visual_topk(ref_imp[None].astype(np.float32), r)[0]
    order = np.lexsort((np.arange(n), -ref_imp))
    tol = 2 * (REL_TOL * np.abs(ref_imp).max() + ABS_TOL)
    if r < n and ref_imp[order[r - 1]] - ref_imp[order[r]] > tol:
        assert np.array_equal(keep, ref_keep)
    dropped = np.setdiff1d(np.arange(n), keep)
    if len(dropped):
        assert ref_imp[keep].min() >= ref_imp[dropped].max() - tol
    return int(np.sum(keep != ref_keep))


def test_selection_end_to_end(dev):
    wl = small_wl(num_q_heads=8, num_kv_heads=8, num_nodes=60, depth=6, max_branch=4, kv_len=1200)
    batch = W.make_batch(wl, with_logits=False)
    v0, nv, r = 50, 1100, 220
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    imp = dreams.visual_importance(q, k, kv, lse, v0, nv)
    keep = dreams.visual_topk(imp, r)
    ko, vo = dreams.visual_gather(k, v, v0, keep)
    torch.cuda.synchronize()
    ref_imp = oracle_importance(batch, v0, nv)
    keep_h = keep.cpu().numpy()
    diffs = [check_selection(keep_h[b], ref_imp[b], r) for b in range(wl.batch)]
    kb = k.cpu().view(torch.int16).numpy()
    gk = ko.cpu().view(torch.int16).numpy()
    for b in range(wl.batch):
        assert np.array_equal(gk[b], kb[b][:, v0 + keep_h[b]])
    note("end to end: keep differs from the oracle's choice in %s places (near-ties only)" % diffs)


def test_importance_full_size(dev):
    # llava7b_layer: the 2880 image tokens of the 3136-token prefix, every head and node; keep 576
    wl = W.WORKLOADS["llava7b_layer"]
    batch = W.make_batch(wl, with_logits=False, layers=[0])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, lse = dreams.tree_verify_attn(q, k, v, kv, par, max_kv_len=wl.max_kv_len)
    imp = dreams.visual_importance(q, k, kv, lse, 0, wl.image_tokens)
    keep = dreams.visual_topk(imp, 576)
    torch.cuda.synchronize()
    ref = oracle_importance(batch, 0, wl.image_tokens)
    got = imp.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    note("llava7b_layer importance: max rel %.3e" % float(np.max(err / np.abs(ref))))
    assert np.all(err <= REL_TOL * np.abs(ref) + ABS_TOL)
    d = check_selection(keep.cpu().numpy()[0], ref[0], 576)
    note("llava7b_layer keep 576 of 2880: %d differences from the oracle (near-ties)" % d)
