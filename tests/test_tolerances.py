"""The GPU tests' derived tolerances for the attention entropy and the visual-token importance are tight enough
to see a regression: the oracle's own values pass, and the same values off by a relative 1e-4 fail.  (CPU only:
the references come from the oracle on a small seeded case.)"""
import numpy as np

import oracle
from gpu_util import entropy_error, f32, importance_error
from paper_2606_00535_amd import workload as W


def small_case():
    wl = W.Workload(name="tol", batch=2, num_q_heads=4, num_kv_heads=2, head_dim=64, dtype="bf16", num_layers=1,
                    kv_len=300, image_tokens=0, num_nodes=16, depth=4, max_branch=3, vocab=64, agree=0.7, seed=41)
    return W.make_batch(wl, with_logits=False)


def test_entropy_tolerance_catches_a_1e4_relative_error():
    b = small_case()
    ref = oracle.tree_attn_entropy(f32(b.q[0]), f32(b.k_cache[0]), b.kv_len, b.parent, b.scale, 2)
    assert ref.min() > 1.0                      # rows of a few hundred keys: H of several nats
    assert entropy_error(ref.astype(np.float32), ref)[1]      # the oracle rounded to fp32 passes
    assert not entropy_error(ref * (1 + 1e-4), ref)[1]
    assert not entropy_error(ref + 2e-5, ref)[1]


def test_importance_tolerance_catches_a_1e4_relative_error():
    b = small_case()
    ref = oracle.visual_importance(f32(b.q[0]), f32(b.k_cache[0]), b.kv_len, b.parent, b.scale, 2, 10, 200)
    assert ref.max() > 0
    assert importance_error(ref.astype(np.float32), ref)[1]
    assert not importance_error(ref * (1 + 1e-4), ref)[1]
    bumped = ref.copy()
    bumped[0, np.argmax(ref[0])] *= 1 + 5e-5
    assert not importance_error(bumped, ref)[1]
