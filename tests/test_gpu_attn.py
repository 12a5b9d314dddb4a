"""GPU parity of dreams_tree_verify_attn against the fp64 CPU oracle, on the same seeded inputs.

Bars: the contract (max-abs <= 2e-2 for bf16 in / fp32 accumulate; 1e-5 for the fp32 path) and a tighter
bound derived from the bf16 path's arithmetic.  The probabilities are rounded to bf16 once before the value
product and the output is rounded to bf16 once (unit roundoff u = 2^-8: bf16 keeps 8 significant bits),
everything else is fp32, so per element
    |out - ref| <= u * (sum_j p_j |v_j| / sum_j p_j + |ref|)     (+ fp32 noise),
and the first term is exactly the oracle's output on |V|.  With the key axis in several pieces, each piece's
output (a weighted mean of its V rows, so at most its share of sum p|v| / sum p) is rounded to bf16 once more
before the fp32 merge, which adds the first term once more:
    |out - ref| <= u * (2 sum_j p_j |v_j| / sum_j p_j + |ref|).
The tests allow 1.02x the bound that applies to the call plus 1e-6.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import ATTN_TOL_BF16, ATTN_TOL_F32, LSE_TOL, attn_errors, device, f32, layer_tensors, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu


def bf16_bound(absref, ref, splits=1):
    return 1.02 * 2.0 ** -8 * ((2 if splits > 1 else 1) * absref + np.abs(ref)) + 1e-6


def splits_of(q, k, num_splits=0, max_kv_len=0):
    return dreams.tree_verify_attn_splits(dreams.attn_desc(q, k, num_splits=num_splits, max_kv_len=max_kv_len))


def oracle_layer(batch, li, abs_v=False, parent=None, mask=None):
    v = f32(batch.v_cache[li])
    return oracle.tree_attn(f32(batch.q[li]), f32(batch.k_cache[li]), np.abs(v) if abs_v else v, batch.kv_len,
                            batch.parent if parent is None and mask is None else parent, batch.scale,
                            batch.wl.num_kv_heads, tree_mask=mask)


def check_bf16(out, lse, batch, li, label, ref=None, absref=None, mask=None, splits=1):
    if ref is None:
        ref = oracle_layer(batch, li, mask=mask)
    if absref is None:
        absref = oracle_layer(batch, li, abs_v=True, mask=mask)[0]
    o_ref, l_ref = ref
    mx, _, o = attn_errors(out, o_ref)
    bound = bf16_bound(absref, o_ref, splits)
    worst = float(np.max(np.abs(o - o_ref) / bound))
    lerr = float(np.nanmax(np.abs(lse.cpu().numpy() - l_ref))) if lse is not None else 0.0
    note("%s: splits=%d max_abs=%.3e (contract %.0e) worst/bound=%.3f lse_err=%.2e"
         % (label, splits, mx, ATTN_TOL_BF16, worst, lerr))
    assert mx <= ATTN_TOL_BF16, label
    assert worst <= 1.0, label
    assert lerr <= LSE_TOL, label
    return o


def small_wl(**kw):
    base = dict(name="small", batch=2, num_q_heads=4, num_kv_heads=2, head_dim=128, dtype="bf16", num_layers=1,
                kv_len=300, image_tokens=0, num_nodes=16, depth=4, max_branch=3, vocab=64, agree=0.7, seed=11)
    base.update(kw)
    return W.Workload(**base)


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def test_tiny_fp32(dev):
    batch = W.make_batch(W.WORKLOADS["tiny"], with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("tiny fp32: B=1 Hq=4 D=64 L=640 T=16")
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    torch.cuda.synchronize()
    ref, lref = oracle_layer(batch, 0)
    err = float(np.abs(out.cpu().numpy() - ref).max())
    lerr = float(np.abs(lse.cpu().numpy() - lref).max())
    note("tiny fp32 max_abs=%.3e lse=%.3e" % (err, lerr))
    assert err <= ATTN_TOL_F32 and lerr <= 1e-4


@pytest.mark.parametrize("variant", ["plain", "sharp", "tree_dominant"])
def test_tiny_fp32_variants(dev, variant):
    batch = W.make_batch(W.WORKLOADS["tiny"], with_logits=False)
    batch = {"plain": batch, "sharp": W.make_sharp(batch, 32.0), "tree_dominant": W.make_tree_dominant(batch)}[variant]
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    out, _ = dreams.tree_verify_attn(q, k, v, kv, par)
    ref, _ = oracle_layer(batch, 0)
    err = float(np.abs(out.cpu().numpy() - ref).max())
    note("tiny fp32 %s max_abs=%.3e" % (variant, err))
    assert err <= ATTN_TOL_F32



F32_CASES = [  # (D, Hq, Hkv, T, depth, branch, L, mask input, empty row)
    (128, 4, 2, 100, 8, 6, 300, False, False),    # head_dim 128, GQA, T > 64 (second ancestor word)
    (64, 2, 1, 33, 5, 3, 0, True, True),          # empty prefix, mask input with an all-zero row
    (128, 3, 3, 1, 0, 1, 1000, False, False),     # single node, more keys than a row's threads
    (64, 6, 2, 60, 6, 4, 1300, False, False),     # head_dim 64, several rounds of keys per thread
]


@pytest.mark.parametrize("case", F32_CASES, ids=lambda c: "D%d_Hq%d_Hkv%d_T%d_L%d_mask%d" % (c[0], c[1], c[2], c[3], c[6], c[7]))
def test_fp32_path(dev, case):
    # the fp32 kernel over shapes beyond the tiny workload: every row against the oracle
    from pins import ancestor_closure, mask_bits_from_closure
    D, Hq, Hkv, T, depth, br, L, use_mask, empty_row = case
    wl = small_wl(head_dim=D, num_q_heads=Hq, num_kv_heads=Hkv, num_nodes=T, depth=depth, max_branch=br,
                  kv_len=L, dtype="f32")
    batch = W.make_batch(wl, with_logits=False, kv_lens=[L, max(0, L - 37)])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("fp32 path %s" % (case,))
    bits = None
    if use_mask:
        bits = np.stack([mask_bits_from_closure(ancestor_closure(batch.parent[b])) for b in range(wl.batch)])
        if empty_row:
            bits[:, T // 2] = 0
        out, lse = dreams.tree_verify_attn(q, k, v, kv, None, tree_mask=to_dev(bits.view(np.int64), dev))
    else:
        out, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    torch.cuda.synchronize()
    ref, lref = oracle.tree_attn(f32(batch.q[0]), f32(batch.k_cache[0]), f32(batch.v_cache[0]), batch.kv_len,
                                 None if use_mask else batch.parent, batch.scale, Hkv, tree_mask=bits)
    o = out.cpu().numpy()
    l = lse.cpu().numpy()
    live = np.isfinite(lref)
    assert np.array_equal(np.isfinite(l), live)
    err = float(np.abs(o - ref).max())
    lerr = float(np.abs(l[live] - lref[live]).max()) if live.any() else 0.0
    note("  max_abs=%.3e lse=%.3e" % (err, lerr))
    assert err <= ATTN_TOL_F32 and lerr <= 1e-4


CASES = [  # (D, Hq, Hkv, T, depth, branch, L, splits)
    (128, 4, 2, 16, 4, 3, 300, 0),
    (128, 4, 2, 16, 4, 3, 300, 1),
    (128, 4, 2, 16, 4, 3, 300, 3),
    (128, 2, 2, 60, 6, 4, 1000, 0),
    (128, 2, 2, 60, 6, 4, 1000, 7),
    (128, 3, 1, 60, 6, 4, 77, 2),      # G=3: 180 rows -> 3 row groups, ragged
    (64, 4, 4, 16, 4, 3, 513, 0),
    (64, 2, 1, 100, 8, 6, 130, 4),     # T > 64: second mask word
    (128, 2, 2, 1, 0, 1, 250, 0),      # single node = decode step
    (128, 2, 2, 33, 5, 3, 0, 0),       # empty prefix: tree keys only
    (128, 2, 2, 33, 5, 3, 0, 2),
    (128, 7, 1, 128, 8, 6, 700, 0),    # GQA 7 x 128 rows = 7 row groups of 128, deepest tree
    (128, 2, 2, 9, 3, 3, 400, 3),      # 9 rows: 16-row workgroups, four key groups
    (64, 4, 2, 16, 4, 3, 333, 2),      # 32 rows, head_dim 64
    (64, 2, 2, 60, 6, 4, 900, 0),      # 64 rows, head_dim 64
    # long pieces: the ring wraps several times in every row configuration
    (128, 2, 2, 9, 3, 3, 2100, 1),     # 16 rows
    (128, 4, 2, 16, 4, 3, 2100, 1),    # 32 rows
    (128, 2, 2, 60, 6, 4, 3000, 2),    # 64 rows
    (128, 4, 2, 60, 6, 4, 2000, 1),    # 128 rows
    (128, 3, 1, 60, 6, 4, 2000, 1),    # 128-row workgroups, 2 row groups (180 rows)
    (64, 2, 2, 60, 6, 4, 3000, 1),     # 64 rows, head_dim 64
    (64, 4, 2, 60, 6, 4, 2000, 1),     # 128 rows, head_dim 64
    # more (sequence, KV head) sets than compute units: 16- and 32-row workgroups in several rounds (short
    # prefixes, so one piece each: the key-axis pieces of these shapes are covered below)
    (128, 320, 320, 9, 3, 3, 200, 0),  # 16 rows, 640 sets
    (128, 320, 160, 16, 4, 3, 200, 0), # 32 rows (G=2), 320 sets
    (64, 300, 300, 16, 4, 3, 200, 0),  # 16 rows, head_dim 64
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "D%d_Hq%d_Hkv%d_T%d_L%d_S%d" % (c[0], c[1], c[2], c[3], c[6], c[7]))
@pytest.mark.parametrize("variant", ["plain", "tree_dominant"])
def test_bf16_parity(dev, case, variant):
    D, Hq, Hkv, T, depth, br, L, splits = case
    wl = small_wl(head_dim=D, num_q_heads=Hq, num_kv_heads=Hkv, num_nodes=T, depth=depth, max_branch=br, kv_len=L)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[L, max(0, L - 37)])
    if variant == "tree_dominant":
        batch = W.make_tree_dominant(batch)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("bf16 %s %s" % (variant, case))
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits)
    torch.cuda.synchronize()
    check_bf16(out, lse, batch, 0, "bf16 %s %s" % (variant, case), splits=splits_of(q, k, splits))


# More workgroups than the 256 compute units, several pieces per row set: the last piece of each set to arrive
# merges it while other sets still stream (every row configuration, D = 64 and 128).
FUSED_CASES = [  # (D, Hq, Hkv, T, depth, branch, L, splits): grid = 8*ceil(2*Hkv/8) * splits * row_groups
    (128, 64, 64, 16, 4, 3, 400, 4),   # 16-row workgroups (4 waves): 512 workgroups
    (64, 48, 48, 60, 6, 4, 700, 3),    # 64 rows, head_dim 64: 288
    (128, 64, 32, 60, 6, 4, 600, 5),   # G=2, 128 rows: 320
    (128, 84, 12, 128, 8, 6, 500, 3),  # G=7, 128-row workgroups, 7 row groups: 504
    (128, 320, 320, 9, 3, 3, 900, 3),  # 16-row workgroups, 3 pieces: 1920
    (64, 320, 160, 16, 4, 3, 800, 2),  # 32-row workgroups, head_dim 64: 640
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=lambda c: "D%d_Hq%d_Hkv%d_T%d_L%d_S%d" % (c[0], c[1], c[2], c[3], c[6], c[7]))
def test_many_workgroups(dev, case):
    D, Hq, Hkv, T, depth, br, L, splits = case
    wl = small_wl(head_dim=D, num_q_heads=Hq, num_kv_heads=Hkv, num_nodes=T, depth=depth, max_branch=br, kv_len=L)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[L, max(0, L - 37)])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    desc = dreams.attn_desc(q, k, num_splits=splits)
    ws = torch.zeros(dreams.tree_verify_attn_workspace_size(desc), dtype=torch.uint8, device=dev)
    note("many workgroups %s" % (case,))
    ref = oracle_layer(batch, 0)
    absref = oracle_layer(batch, 0, abs_v=True)[0]
    first = None
    for rep in range(3):
        out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits, workspace=ws)
        torch.cuda.synchronize()
        cur = out.view(torch.int16).cpu().numpy()
        if first is None:
            check_bf16(out, lse, batch, 0, "many workgroups %s" % (case,), ref, absref, splits=splits)
            first = cur
        else:
            assert np.array_equal(cur, first), rep   # same result on every call
    assert not ws[:65536].cpu().numpy().any()       # counters left zero
    dreams.workspace_status(ws)                      # no failure flagged


@pytest.mark.parametrize("scale", [-0.07, 0.0, 0.31])
def test_scale_sign_and_zero(dev, scale):
    # the kernel folds |scale| into the exponent and flips the queries' sign for a negative scale
    wl = small_wl(num_nodes=60, depth=6, max_branch=4, kv_len=500)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("scale %g" % scale)
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, scale=scale, num_splits=2)
    splits = splits_of(q, k, 2)
    torch.cuda.synchronize()
    v32 = f32(batch.v_cache[0])
    args = (f32(batch.q[0]), f32(batch.k_cache[0]))
    ref = oracle.tree_attn(*args, v32, batch.kv_len, batch.parent, scale, wl.num_kv_heads)
    absref = oracle.tree_attn(*args, np.abs(v32), batch.kv_len, batch.parent, scale, wl.num_kv_heads)[0]
    check_bf16(out, lse, batch, 0, "scale %g" % scale, ref, absref, splits=splits)


def test_split_sweep_agrees(dev):
    wl = small_wl(num_q_heads=2, num_kv_heads=2, num_nodes=60, depth=6, max_branch=4, kv_len=1500)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    ref = oracle_layer(batch, 0)
    absref = oracle_layer(batch, 0, abs_v=True)[0]
    outs = []
    for s in (1, 2, 8, 24, 32, 4096):
        note("split sweep S=%d" % s)
        out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=s)
        torch.cuda.synchronize()
        outs.append(check_bf16(out, lse, batch, 0, "split %d" % s, ref, absref, splits=splits_of(q, k, s)))
    for o in outs[1:]:
        assert np.max(np.abs(o - outs[0])) <= 3 * 2.0 ** -8 * (np.abs(outs[0]).max() + 1)


def test_repeat_is_bitwise_identical(dev):
    wl = small_wl(num_q_heads=4, num_kv_heads=4, num_nodes=60, depth=6, max_branch=4, kv_len=2000)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    first = None
    for rep in range(5):
        out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=8)
        torch.cuda.synchronize()
        cur = (out.view(torch.int16).cpu().numpy(), lse.cpu().numpy())
        if first is None:
            first = cur
        else:
            assert np.array_equal(cur[0], first[0]) and np.array_equal(cur[1], first[1]), rep


def test_workspace_left_zero(dev):
    wl = small_wl(num_nodes=60, depth=6, max_branch=4, kv_len=900)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    desc = dreams.attn_desc(q, k, num_splits=5)
    n = dreams.tree_verify_attn_workspace_size(desc)
    ws = torch.zeros(n, dtype=torch.uint8, device=dev)
    for _ in range(3):
        dreams.tree_verify_attn(q, k, v, kv, par, num_splits=5, workspace=ws)
    torch.cuda.synchronize()
    cnt = ws[:65536].cpu().numpy()          # the arrival counters open every workspace
    assert not cnt.any()
    dreams.workspace_status(ws)


def test_nonancestor_perturbation_bitwise(dev):
    wl = small_wl(num_q_heads=2, num_kv_heads=2, num_nodes=60, depth=6, max_branch=4, kv_len=700, batch=1)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=3)
    parent = batch.parent[0]
    anc = [set() for _ in range(60)]
    for i in range(60):
        j = i
        while j >= 0:
            anc[i].add(j)
            j = parent[j]
    rng = np.random.default_rng(5)
    for i in rng.choice(60, size=6, replace=False):
        k2, v2 = k.clone(), v.clone()
        others = [j for j in range(60) if j not in anc[i]]
        idx = torch.tensor([700 + j for j in others], device=dev)
        k2[0][:, idx] = torch.randn_like(k2[0][:, idx]) * 3
        v2[0][:, idx] = torch.randn_like(v2[0][:, idx]) * 3
        out2, lse2 = dreams.tree_verify_attn(q, k2, v2, kv, par, num_splits=3)
        torch.cuda.synchronize()
        assert torch.equal(out2[0, :, i].view(torch.int16), out[0, :, i].view(torch.int16)), int(i)
        assert torch.equal(lse2[0, :, i], lse[0, :, i]), int(i)


@pytest.mark.parametrize("hq,hkv,t", [(2, 2, 60), (4, 2, 60), (3, 1, 60), (4, 2, 16)],
                         ids=["64rows", "128rows", "128rows_2groups", "32rows"])
def test_garbage_past_sequence_end_bitwise(dev, hq, hkv, t):
    # cache slots at or past L_b + T are not part of the problem: infinities and NaNs there change nothing
    wl = small_wl(num_q_heads=hq, num_kv_heads=hkv, num_nodes=t, depth=4, max_branch=4, kv_len=500)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[500, 437])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("garbage past end %s" % ((hq, hkv, t),))
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=2, max_kv_len=500)
    k2, v2 = k.clone(), v.clone()
    for b, L in enumerate(batch.kv_len):
        n = int(L) + t
        k2[b, :, n:] = float("nan")
        v2[b, :, n:] = float("inf")
        k2[b, :, n + 1::3] = float("-inf")
        v2[b, :, n + 1::3] = float("nan")
    out2, lse2 = dreams.tree_verify_attn(q, k2, v2, kv, par, num_splits=2, max_kv_len=500)
    torch.cuda.synchronize()
    assert torch.equal(out2.view(torch.int16), out.view(torch.int16))
    assert torch.equal(lse2, lse)


def test_mask_input_matches_parent_and_empty_rows(dev):
    from pins import ancestor_closure, mask_bits_from_closure
    wl = small_wl(num_q_heads=2, num_kv_heads=1, num_nodes=100, depth=8, max_branch=6, kv_len=400)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    bits = np.stack([mask_bits_from_closure(ancestor_closure(batch.parent[b])) for b in range(2)])
    mask = to_dev(bits.view(np.int64), dev)
    o1, l1 = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=2)
    o2, l2 = dreams.tree_verify_attn(q, k, v, kv, None, tree_mask=mask, num_splits=2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)) and torch.equal(l1, l2)
    # empty prefix and an all-zero mask row: nothing visible -> zeros and lse = -inf, like the oracle
    bits2 = bits.copy()
    bits2[:, 5] = 0
    kv0 = torch.zeros(2, dtype=torch.int32, device=dev)
    o3, l3 = dreams.tree_verify_attn(q, k, v, kv0, None, tree_mask=to_dev(bits2.view(np.int64), dev), num_splits=2)
    torch.cuda.synchronize()
    assert torch.all(o3[:, :, 5] == 0) and torch.all(torch.isneginf(l3[:, :, 5]))
    ref, lref = oracle.tree_attn(f32(batch.q[0]), f32(batch.k_cache[0]), f32(batch.v_cache[0]),
                                 np.zeros(2, np.int32), None, batch.scale, 1, tree_mask=bits2)
    o3n = o3.float().cpu().numpy()
    ok = np.isfinite(lref)
    assert np.max(np.abs(o3n - ref)) <= ATTN_TOL_BF16 and np.max(np.abs(l3.cpu().numpy()[ok] - lref[ok])) <= LSE_TOL



@pytest.mark.parametrize("splits", [2, 4, 7])
def test_pieces_cut_per_sequence_length(dev, splits):
    # several sequences of very different lengths (one with no prefix): each sequence's key axis is cut into
    # pieces of its own length, so a short sequence has short or empty pieces; every row against the oracle
    wl = small_wl(num_q_heads=4, num_kv_heads=2, num_nodes=60, depth=6, max_branch=4, kv_len=2600, batch=3)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[0, 2600, 45])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("pieces per sequence length, splits=%d" % splits)
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits)
    torch.cuda.synchronize()
    check_bf16(out, lse, batch, 0, "pieces per sequence length S=%d" % splits, splits=splits_of(q, k, splits))

def test_kv_len_clamped_into_cache(dev):
    # a prefix length past the capacity is clamped to S_cap - T: same result as that length, no stray access
    wl = small_wl(num_nodes=16, kv_len=300)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    S = batch.k_cache.shape[3]
    big = torch.tensor([S + 1000, 10 ** 9], dtype=torch.int32, device=dev)
    clamp = torch.tensor([S - 16, S - 16], dtype=torch.int32, device=dev)
    o1, _ = dreams.tree_verify_attn(q, k, v, big, par, num_splits=2)
    o2, _ = dreams.tree_verify_attn(q, k, v, clamp, par, num_splits=2)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


def test_batch_zero_is_noop(dev):
    q = torch.empty((0, 2, 4, 128), dtype=torch.bfloat16, device=dev)
    k = torch.empty((0, 2, 64, 128), dtype=torch.bfloat16, device=dev)
    kv = torch.empty(0, dtype=torch.int32, device=dev)
    par = torch.empty((0, 4), dtype=torch.int32, device=dev)
    out, lse = dreams.tree_verify_attn(q, k, k, kv, par)
    torch.cuda.synchronize()
    assert out.shape == q.shape


# ------------------------------------------------------------------------- full-size shapes
def test_llava7b_layer_full_parity(dev):
    batch = W.make_batch(W.WORKLOADS["llava7b_layer"], with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("llava7b_layer: B=1 Hq=32 D=128 L=3136 T=60 (auto splits)")
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    torch.cuda.synchronize()
    splits = splits_of(q, k)
    check_bf16(out, lse, batch, 0, "llava7b_layer", splits=splits)
    bdom = W.make_tree_dominant(batch)
    q, k, v, kv, par = layer_tensors(bdom, 0, dev)
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par)
    torch.cuda.synchronize()
    check_bf16(out, lse, bdom, 0, "llava7b_layer tree_dominant", splits=splits)


def sampled_rows(rng, B, Hq, T, n):
    rows = np.stack([rng.integers(0, B, n), rng.integers(0, Hq, n), rng.integers(0, T, n)], axis=1).astype(np.int32)
    rows[:4] = [[0, 0, 0], [B - 1, Hq - 1, T - 1], [0, Hq - 1, T // 2], [B - 1, 0, 1 % T]]
    return rows


@pytest.mark.parametrize("name,layers", [("llava7b_full", [0, 15, 31]), ("llava13b_layer", [0]), ("gqa_long", [0])])
def test_full_size_sampled_rows(dev, name, layers):
    wl = W.WORKLOADS[name]
    batch = W.make_batch(wl, layers=layers, with_logits=False)
    rng = np.random.default_rng(3)
    for li, layer in enumerate(layers):
        q, k, v, kv, par = layer_tensors(batch, li, dev)
        note("%s layer %d: sampled rows (auto splits)" % (name, layer))
        out, lse = dreams.tree_verify_attn(q, k, v, kv, par, max_kv_len=wl.max_kv_len)
        torch.cuda.synchronize()
        rows = sampled_rows(rng, wl.batch, wl.num_q_heads, wl.num_nodes, 96)
        args = (f32(batch.q[li]), f32(batch.k_cache[li]))
        ref, lref = oracle.tree_attn_rows(*args, f32(batch.v_cache[li]), batch.kv_len, batch.parent, batch.scale,
                                          wl.num_kv_heads, rows)
        absref, _ = oracle.tree_attn_rows(*args, np.abs(f32(batch.v_cache[li])), batch.kv_len, batch.parent,
                                          batch.scale, wl.num_kv_heads, rows)
        o = out.float().cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]].astype(np.float64)
        l = lse.cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
        mx = float(np.abs(o - ref).max())
        worst = float(np.max(np.abs(o - ref) / bf16_bound(absref, ref, splits_of(q, k, 0, wl.max_kv_len))))
        note("  max_abs=%.3e worst/bound=%.3f lse=%.2e" % (mx, worst, float(np.abs(l - lref).max())))
        assert mx <= ATTN_TOL_BF16 and worst <= 1.0 and float(np.abs(l - lref).max()) <= LSE_TOL
        # property at any size: every output row is a convex combination of V rows -> bounded by max |V|
        assert float(out.float().abs().max()) <= float(v.float().abs().max()) * (1 + 2 ** -7)


# ------------------------------------------------------------------------- graph replay
@pytest.mark.parametrize("name", ["small", "llava7b_layer"])
def test_graph_replay_matches_eager(dev, name):
    # Several pieces per row set under HIP-graph replay: a graph's kernels start their round-robin over the XCDs
    # at another XCD than direct launches do, and the merge must not depend on which.  Each replay (with eager
    # work of other grid sizes between replays) must equal the direct call bit for bit, leave the counters zero
    # and set no failure flag; the direct call is held to the oracle.
    if name == "small":
        wl = small_wl(num_q_heads=4, num_kv_heads=2, num_nodes=60, depth=6, max_branch=4, kv_len=2000)
        splits_req = 5
    else:
        wl = W.WORKLOADS[name]
        splits_req = 0
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    desc = dreams.attn_desc(q, k, num_splits=splits_req)
    splits = dreams.tree_verify_attn_splits(desc)
    assert splits > 1
    ws = torch.zeros(dreams.tree_verify_attn_workspace_size(desc), dtype=torch.uint8, device=dev)
    note("%s: graph replay, splits=%d" % (name, splits))
    out_e, lse_e, ent_e = dreams.tree_verify_attn_entropy(q, k, v, kv, par, num_splits=splits_req, workspace=ws)
    torch.cuda.synchronize()
    dreams.workspace_status(ws)
    check_bf16(out_e, lse_e, batch, 0, "%s direct" % name, splits=splits)
    out_g, lse_g, ent_g = torch.empty_like(out_e), torch.empty_like(lse_e), torch.empty_like(ent_e)
    out_p = torch.empty_like(out_e)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        dreams.tree_verify_attn(q, k, v, kv, par, out=out_p, with_lse=False, num_splits=splits_req, workspace=ws)
        dreams.tree_verify_attn_entropy(q, k, v, kv, par, out=out_g, lse=lse_g, entropy=ent_g,
                                        num_splits=splits_req, workspace=ws)
    filler = torch.zeros(7 * 64 + 3, device=dev)
    for rep in range(4):
        for t in (out_g, out_p):
            t.fill_(float("nan"))
        filler.add_(1.0)
        g.replay()
        torch.cuda.synchronize()
        dreams.workspace_status(ws)
        assert np.array_equal(out_g.view(torch.int16).cpu().numpy(), out_e.view(torch.int16).cpu().numpy()), rep
        assert np.array_equal(out_p.view(torch.int16).cpu().numpy(), out_e.view(torch.int16).cpu().numpy()), rep
        assert np.array_equal(lse_g.cpu().numpy(), lse_e.cpu().numpy()), rep
        assert np.array_equal(ent_g.cpu().numpy(), ent_e.cpu().numpy()), rep
    assert not ws[:65536].cpu().numpy().any()
