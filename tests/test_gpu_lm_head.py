"""GPU parity of dreams_tree_accept_lm_head (the LM head fused with greedy acceptance) against the oracle.

The oracle forms the logits in fp64 from the same bf16 operands; the kernel accumulates in fp32, so a row's
argmax is compared exactly wherever the oracle's maximum beats every other entry by more than both entries'
fp32 error bounds (1e-5 * sum_k |h_k w_k| each, far above what a 4096-deep fp32 sum can lose), and otherwise
must be an entry within those bounds of the maximum.  Accepted lengths, paths and bonus tokens must then equal
the greedy rule applied to the kernel's per-node tokens, bit for bit."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import device, note
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu
REL = 1e-5


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def bf16_bits(x):
    return W.f32_to_bf16_bits(np.asarray(x, dtype=np.float32))


def draw(rng, B, T, H, V, w_std=0.02):
    hid = bf16_bits(rng.standard_normal((B, T, H), dtype=np.float32))
    wt = bf16_bits(rng.standard_normal((V, H), dtype=np.float32) * np.float32(w_std))
    return hid, wt


def to_bf16_dev(bits, dev):
    return torch.from_numpy(bits.view(np.int16)).to(dev).view(torch.bfloat16)


def expected_argmax(hid, wt, rows=None):
    """(oracle argmax, fp64 logits, per-entry bounds) for the given flat rows (all by default)."""
    H = hid.shape[-1]
    flat = hid.reshape(-1, H)
    if rows is not None:
        flat = flat[rows]
    logits = oracle.lm_head_logits(flat, wt)
    mag = np.abs(W.bf16_bits_to_f32(flat).astype(np.float64)) @ np.abs(W.bf16_bits_to_f32(wt).astype(np.float64)).T
    return logits.argmax(axis=1), logits, REL * mag + 1e-30


def check_argmax(gpu_am, logits, bound, label):
    """Exact where the oracle's row maximum is unambiguous, within the bounds elsewhere; returns the number of
    ambiguous rows."""
    ref = logits.argmax(axis=1)
    r = np.arange(len(ref))
    m1 = logits[r, ref]
    gap_ok = logits < (m1 - bound[r, ref])[:, None] - bound
    gap_ok[r, ref] = True
    unambiguous = gap_ok.all(axis=1)
    assert np.array_equal(gpu_am[unambiguous], ref[unambiguous]), label
    amb = ~unambiguous
    if amb.any():
        g = gpu_am[amb]
        assert np.all(logits[amb][np.arange(amb.sum()), g] >= m1[amb] - bound[amb][np.arange(amb.sum()), g]
                      - bound[r[amb], ref[amb]]), label
    return int(amb.sum())


def plant_tokens(rng, am, parent, p=0.7, V=None):
    B, T = am.shape
    agree = am[np.arange(B)[:, None], np.maximum(parent, 0)]
    return np.where(rng.random((B, T)) < p, agree, rng.integers(0, V, (B, T))).astype(np.int32)


def run_case(dev, rng, B, T, H, V, label, w_std=0.02, depth=5, branch=4):
    hid, wt = draw(rng, B, T, H, V, w_std)
    parent = np.stack([W.random_tree(rng, T, min(depth, T - 1), branch) for _ in range(B)]) if T > 1 \
        else np.full((B, 1), -1, np.int32)
    ref_am, logits, bound = expected_argmax(hid, wt)
    tokens = plant_tokens(rng, ref_am.reshape(B, T), parent, V=V)
    alen, path, nxt, am = dreams.tree_accept_lm_head(to_bf16_dev(hid, dev), to_bf16_dev(wt, dev),
                                                      torch.from_numpy(tokens).to(dev),
                                                      torch.from_numpy(parent).to(dev), want_target_argmax=True)
    torch.cuda.synchronize()
    gam = am.cpu().numpy()
    amb = check_argmax(gam.reshape(-1), logits, bound, label)
    ea, ep, en = oracle.tree_accept_from_argmax(gam, tokens, parent)
    note("%s: B=%d T=%d H=%d V=%d, ambiguous rows %d, accepted mean %.2f" % (label, B, T, H, V, amb,
                                                                            float(ea.mean())))
    assert np.array_equal(alen.cpu().numpy(), ea) and np.array_equal(path.cpu().numpy(), ep), label
    assert np.array_equal(nxt.cpu().numpy(), en), label
    return amb


def test_llava7b_shape(dev):
    """LLaVA-1.6-7B's LM head (hidden 4096, vocabulary 32000) over a 60-node tree."""
    assert run_case(dev, np.random.default_rng(1), 1, 60, 4096, 32000, "llava7b") <= 1


@pytest.mark.parametrize("B,T,H,V", [(1, 1, 256, 1), (1, 16, 256, 1000), (2, 60, 512, 4099), (3, 7, 768, 65),
                                     (4, 128, 1024, 2048), (1, 64, 256, 64), (5, 13, 512, 12345),
                                     (3, 60, 768, 5000)])
def test_ragged_shapes(dev, B, T, H, V):
    """Rows and vocabularies that are not multiples of the tiles (one 64-row tile up to 64 rows, 128 x 256 up to
    128, 256 x 256 beyond), a single node, a vocabulary of one."""
    run_case(dev, np.random.default_rng(B * 1000 + T), B, T, H, V, "B=%d T=%d H=%d V=%d" % (B, T, H, V))


def test_ties_go_to_the_smallest_index(dev):
    """Duplicated weight rows give bit-identical logits; the maximum is planted on such a pair (and across
    tiles), and the smaller vocabulary index must win."""
    rng = np.random.default_rng(3)
    B, T, H, V = 2, 20, 512, 300
    hid, wt = draw(rng, B, T, H, V)
    h32 = W.bf16_bits_to_f32(hid).reshape(-1, H)
    for row in range(B * T):
        v1, v2 = sorted(rng.choice(V, size=2, replace=False))
        big = bf16_bits(np.sign(h32[row]) * 0.5)
        wt[v1] = big
        wt[v2] = big
    # every row now has its own planted pair; rows see the other rows' pairs too, so the winner is whichever
    # pair aligns best with the row -- compare against the oracle's first maximum directly
    parent = np.stack([W.random_tree(rng, T, 4, 3) for _ in range(B)])
    ref_am, logits, bound = expected_argmax(hid, wt)
    tokens = plant_tokens(rng, ref_am.reshape(B, T), parent, V=V)
    _, _, _, am = dreams.tree_accept_lm_head(to_bf16_dev(hid, dev), to_bf16_dev(wt, dev),
                                             torch.from_numpy(tokens).to(dev), torch.from_numpy(parent).to(dev),
                                             want_target_argmax=True)
    torch.cuda.synchronize()
    gam = am.cpu().numpy().reshape(-1)
    r = np.arange(B * T)
    ties = (logits == logits[r, ref_am][:, None]).sum(axis=1) > 1
    assert ties.sum() >= B * T // 2
    np.testing.assert_array_equal(gam, ref_am)


def test_large_batch_sampled_rows(dev):
    """The gqa_long shape (16 sequences of 128 nodes, hidden 3584, vocabulary 152064): the oracle checks 96
    sampled rows' argmax; every sequence's path must follow the greedy rule on the kernel's tokens."""
    rng = np.random.default_rng(4)
    B, T, H, V = 16, 128, 3584, 152064
    hid, wt = draw(rng, B, T, H, V)
    parent = np.stack([W.random_tree(rng, T, 8, 6) for _ in range(B)])
    rows = np.sort(rng.choice(B * T, size=96, replace=False))
    ref_am, logits, bound = expected_argmax(hid, wt, rows)
    tokens = rng.integers(0, V, (B, T)).astype(np.int32)
    flat = tokens.reshape(-1)
    alen, path, nxt, am = dreams.tree_accept_lm_head(to_bf16_dev(hid, dev), to_bf16_dev(wt, dev),
                                                      torch.from_numpy(tokens).to(dev),
                                                      torch.from_numpy(parent).to(dev), want_target_argmax=True)
    torch.cuda.synchronize()
    gam = am.cpu().numpy()
    amb = check_argmax(gam.reshape(-1)[rows], logits, bound, "gqa rows")
    note("gqa_long LM head: ambiguous sampled rows %d" % amb)
    # tokens planted from the kernel's own argmax so that paths are long; the rule must hold on them
    tokens2 = plant_tokens(rng, gam, parent, V=V)
    alen, path, nxt, am2 = dreams.tree_accept_lm_head(to_bf16_dev(hid, dev), to_bf16_dev(wt, dev),
                                                       torch.from_numpy(tokens2).to(dev),
                                                       torch.from_numpy(parent).to(dev), want_target_argmax=True)
    torch.cuda.synchronize()
    assert np.array_equal(am2.cpu().numpy(), gam)          # repeatable
    ea, ep, en = oracle.tree_accept_from_argmax(gam, tokens2, parent)
    assert np.array_equal(alen.cpu().numpy(), ea) and np.array_equal(path.cpu().numpy(), ep)
    assert np.array_equal(nxt.cpu().numpy(), en)
    assert flat.size == B * T


def test_matches_accept_on_materialised_logits(dev):
    """The same logits written out by torch (fp32 matmul on the device) and fed to dreams_tree_accept give the
    same per-node tokens wherever torch's logits and the kernel's agree on an unambiguous maximum."""
    rng = np.random.default_rng(5)
    B, T, H, V = 2, 60, 1024, 8000
    hid, wt = draw(rng, B, T, H, V)
    parent = np.stack([W.random_tree(rng, T, 6, 4) for _ in range(B)])
    ref_am, logits, bound = expected_argmax(hid, wt)
    tokens = plant_tokens(rng, ref_am.reshape(B, T), parent, V=V)
    hd, wd = to_bf16_dev(hid, dev), to_bf16_dev(wt, dev)
    tk, pr = torch.from_numpy(tokens).to(dev), torch.from_numpy(parent).to(dev)
    out_f = dreams.tree_accept_lm_head(hd, wd, tk, pr, want_target_argmax=True)
    lg = (hd.float().reshape(B * T, H) @ wd.float().t().contiguous()).reshape(B, T, V).contiguous()
    out_l = dreams.tree_accept(lg, tk, pr, want_target_argmax=True)
    torch.cuda.synchronize()
    amb = check_argmax(out_l[3].cpu().numpy().reshape(-1), logits, bound, "materialised")
    if amb == 0:
        for x, y in zip(out_f, out_l):
            assert torch.equal(x, y)


def test_workspace_reuse(dev):
    """One workspace for calls of several shapes, repeated: identical results."""
    n = max(dreams.tree_accept_lm_head_workspace_size(4, 128, 1024, 9000), 1 << 20)
    ws = torch.zeros(n, dtype=torch.uint8, device=dev)
    rng = np.random.default_rng(6)
    for B, T, H, V in [(4, 128, 1024, 9000), (1, 5, 256, 77), (2, 60, 512, 4099)]:
        hid, wt = draw(rng, B, T, H, V)
        parent = np.stack([W.random_tree(rng, T, min(T - 1, 5), 4) for _ in range(B)])
        tokens = rng.integers(0, V, (B, T)).astype(np.int32)
        args = (to_bf16_dev(hid, dev), to_bf16_dev(wt, dev), torch.from_numpy(tokens).to(dev),
                torch.from_numpy(parent).to(dev))
        a1 = dreams.tree_accept_lm_head(*args, want_target_argmax=True, workspace=ws)
        a1 = [t.clone() for t in a1]
        a2 = dreams.tree_accept_lm_head(*args, want_target_argmax=True, workspace=ws)
        torch.cuda.synchronize()
        for x, y in zip(a1, a2):
            assert torch.equal(x, y)
        ref_am, logits, bound = expected_argmax(hid, wt)
        check_argmax(a1[3].cpu().numpy().reshape(-1), logits, bound, str((B, T, H, V)))
