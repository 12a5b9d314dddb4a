"""GPU parity of the prefill statistics (a prompt's own causal attention, where the paper reads Eq. 2 and AE):
per-row log-sum-exp and entropy, the layer's AE over prompt rows, and Eq. 2 visual-token importance, against the
CPU oracle on the same seeded inputs.

Tolerances.  The scores are fp32 sums of exact products of the bf16 inputs, as in the verification call, so the
entropy bound (gpu_util.ENTROPY_TOL, 1e-5 absolute) and the importance bound (gpu_util.IMPORTANCE_REL_TOL, 3e-5
relative) carry over: rows here see up to 3136 keys, fewer than the 8192 those bounds were derived for.  lse is
log of an fp32 sum of <= 3136 terms 2^(z - m) <= 1 plus the reference m: the same few 1e-6 as the entropy's
log-sum term, plus the fp32 rounding of the reference m itself (2^-24 relative, which matters for the sharp rows'
large scores): held to LSE_PREFILL_TOL = 1e-5 plus 2^-22 |lse|.  AE is the fp64 mean of the kernel's own fp32 entropies, so it
must equal that mean (recomputed here in fp64) to one fp32 rounding, and the oracle's AE to ENTROPY_TOL.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import ENTROPY_TOL, device, importance_error, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu

LSE_PREFILL_TOL = 1e-5


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def run_gpu(p: W.Prompt, dev):
    q = to_dev(p.q, dev, True)
    k = to_dev(p.k_cache, dev, True)
    pl = to_dev(p.prompt_len, dev)
    lse, ent = dreams.prefill_attn_stats(q, k, pl)
    ae = dreams.prefill_attn_entropy_mean(ent, pl)
    imp = dreams.prefill_visual_importance(q, k, pl, lse, p.vis_begin, p.vis_count)
    torch.cuda.synchronize()
    return (lse.cpu().numpy().astype(np.float64), ent.cpu().numpy().astype(np.float64), float(ae.cpu()[0]),
            imp.cpu().numpy().astype(np.float64), ent.cpu().numpy())


def run_oracle(p: W.Prompt):
    qf, kf = W.bf16_bits_to_f32(p.q), W.bf16_bits_to_f32(p.k_cache)
    lse, ent = oracle.prefill_attn_stats(qf, kf, p.prompt_len, p.scale, p.num_kv_heads)
    imp = oracle.prefill_visual_importance(qf, kf, p.prompt_len, p.scale, p.num_kv_heads, p.vis_begin, p.vis_count)
    return lse, ent, imp


def check(p: W.Prompt, dev, label):
    glse, gent, gae, gimp, gent32 = run_gpu(p, dev)
    rlse, rent, rimp = run_oracle(p)
    live = np.isfinite(rlse)
    assert np.array_equal(np.isfinite(glse), live), "rows past the prompt must have lse = -inf"
    assert np.all(gent[~live] == 0.0)
    lerr = float(np.max(np.abs(glse[live] - rlse[live]))) if live.any() else 0.0
    lok = bool(np.all(np.abs(glse[live] - rlse[live]) <= LSE_PREFILL_TOL + 2.0 ** -22 * np.abs(rlse[live])))
    eerr = float(np.max(np.abs(gent - rent)))
    rel, ok = importance_error(gimp, rimp)
    n = np.clip(p.prompt_len, 0, p.q.shape[2])
    ae_fp64 = float(gent32.astype(np.float64).sum() / (p.q.shape[1] * n.sum())) if n.sum() > 0 else 0.0
    ae_ref = oracle.prefill_attn_entropy_mean(rent, p.prompt_len) if n.sum() > 0 else 0.0
    note("%s: lse max-abs %.2e, entropy max-abs %.2e, importance max-rel %.2e, AE %.6f (oracle %.6f)"
         % (label, lerr, eerr, rel, gae, ae_ref))
    assert lok
    assert eerr <= ENTROPY_TOL
    assert ok
    assert abs(gae - ae_fp64) <= 2.0 ** -23 * max(abs(ae_fp64), 1e-30)
    assert abs(gae - ae_ref) <= ENTROPY_TOL
    return gimp, rimp


CASES = [  # (B, Hq, Hkv, D, prompt lengths, vis_begin, vis_count)
    (2, 4, 2, 128, (300, 170), 20, 200),      # GQA pairs; the window runs past the second prompt
    (1, 8, 2, 64, (257,), 0, 257),            # head_dim 64, ragged 256-row and 16-key blocks
    (3, 2, 2, 128, (1, 65, 300), 0, 64),      # a one-token prompt (entropy 0), a 65-token one
    (1, 32, 32, 128, (700,), 35, 600),        # the LLaVA head layout
]


@pytest.mark.parametrize("case", CASES, ids=[str(c[:5]) for c in CASES])
def test_prefill_parity(dev, case):
    B, Hq, Hkv, D, lens, vb, vc = case
    p = W.make_prompt(B, Hq, Hkv, D, lens, vb, vc, seed=61)
    check(p, dev, "prefill %s" % (case,))


def test_prefill_empty_prompt(dev):
    # a sequence with no prompt: every row -inf / 0, importance 0, and it does not count in AE
    p = W.make_prompt(2, 4, 4, 128, (0, 90), 0, 80, num_rows=96, seed=62)
    gimp, _ = check(p, dev, "prefill with an empty prompt")
    assert np.all(gimp[0] == 0.0)


def test_prefill_sharp_rows(dev):
    # large queries: rows dominated by one key (entropy near 0, lse far from log n)
    p = W.make_prompt(1, 4, 4, 128, (400,), 10, 300, q_std=6.0, seed=63)
    check(p, dev, "prefill, sharp rows")


def test_prefill_llava7b_prompt(dev):
    # the LLaVA-1.6-7B prompt shape: 3136 tokens, 2880 of them visual (after a 40-token system text), 8 of the 32
    # heads (the oracle's cost); every row and every visual token compared
    p = W.make_prompt(1, 8, 8, 128, (3136,), 40, 2880, seed=64)
    check(p, dev, "prefill, LLaVA-7B prompt (8 heads)")


def test_prefill_repeatable_and_counters_clear(dev):
    p = W.make_prompt(2, 4, 2, 128, (300, 170), 20, 200, seed=65)
    q, k, pl = to_dev(p.q, dev, True), to_dev(p.k_cache, dev, True), to_dev(p.prompt_len, dev)
    ws = torch.zeros(dreams.visual_importance_workspace_size(2, 2, 200), dtype=torch.uint8, device=dev)
    outs = []
    for _ in range(3):
        lse, ent = dreams.prefill_attn_stats(q, k, pl)
        imp = dreams.prefill_visual_importance(q, k, pl, lse, 20, 200, workspace=ws)
        torch.cuda.synchronize()
        outs.append((lse.cpu().numpy(), ent.cpu().numpy(), imp.cpu().numpy()))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    assert not ws[:65536 - 128].cpu().numpy().any()
