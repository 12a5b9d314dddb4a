"""The seeded input generator produces what the workloads describe (topology, lengths, agreement, dtype)."""
import numpy as np
import pytest

from paper_2606_00535_amd import workload as W


@pytest.mark.parametrize("T,depth,branch", [(16, 4, 3), (60, 6, 4), (128, 8, 6), (1, 0, 1), (7, 6, 1)])
def test_random_tree_shape(T, depth, branch):
    for seed in range(20):
        p = W.random_tree(W.rng_for(seed, 0, 0, 0), T, depth, branch)
        assert p[0] == -1 and all(0 <= p[i] < i for i in range(1, T))
        d = W.tree_depths_for_generator_checks(p)
        assert d.max(initial=0) == min(depth, T - 1)
        counts = np.bincount(p[1:], minlength=T) if T > 1 else np.zeros(1)
        assert counts.max(initial=0) <= branch
        assert np.all(np.diff(d) >= 0)            # breadth-first numbering: depths never decrease


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e-39, 65504.0], dtype=np.float32)
    bits = W.f32_to_bf16_bits(x)
    back = W.bf16_bits_to_f32(bits)
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even mantissa (1.0); 1 + 3*2^-8 -> 1 + 2^-6 (even)
    assert back[0] == 1.0 and back[1] == 1.0 and back[2] == 1.015625 and back[3] == -2.5
    import torch
    rng = np.random.default_rng(0)
    y = np.concatenate([x, rng.standard_normal(10000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 10000)])
    ref = torch.from_numpy(y.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.f32_to_bf16_bits(y.astype(np.float32)), ref)


def test_tiny_batch_and_agreement():
    wl = W.WORKLOADS["tiny"]
    b = W.make_batch(wl)
    assert b.q.shape == (1, 1, 4, 16, 64) and b.q.dtype == np.float32
    assert b.k_cache.shape == (1, 1, 4, wl.cache_capacity, 64)
    assert int(b.kv_len[0]) == 640
    assert abs(float(b.q.std()) - 1 / 8) < 0.01
    # slots past L+T stay zero
    assert np.all(b.k_cache[..., 640 + 16:, :] == 0)
    b2 = W.make_batch(wl)
    assert np.array_equal(b.q, b2.q) and np.array_equal(b.tokens, b2.tokens)


def test_agreement_rate_and_ragged_lengths():
    wl = W.WORKLOADS["llava7b_full"].replace(num_layers=1, vocab=64, num_q_heads=2, num_kv_heads=2, head_dim=16)
    wl = wl.replace(batch=64)
    b = W.make_batch(wl)
    assert np.all((b.kv_len >= 2900) & (b.kv_len <= 4096))
    am = np.argmax(b.logits, axis=2)
    agree = [b.tokens[s, i] == am[s, b.parent[s, i]] for s in range(64) for i in range(1, 60)]
    p_eff = 0.7 + 0.3 / 64
    assert abs(np.mean(agree) - p_eff) < 4 * np.sqrt(p_eff * (1 - p_eff) / len(agree))


def test_layer_subset_matches_full_draw():
    wl = W.WORKLOADS["llava7b_full"].replace(num_layers=4, batch=2, num_q_heads=2, num_kv_heads=2, head_dim=16,
                                             vocab=32)
    full = W.make_batch(wl, with_logits=False)
    sub = W.make_batch(wl, layers=[3, 1], with_logits=False)
    assert np.array_equal(sub.q[0], full.q[3]) and np.array_equal(sub.k_cache[1], full.k_cache[1])


def test_variants_keep_shape():
    wl = W.WORKLOADS["tiny"]
    b = W.make_batch(wl, with_logits=False)
    d = W.make_tree_dominant(b)
    s = W.make_sharp(b)
    assert d.q.shape == b.q.shape and s.q.shape == b.q.shape and d.k_cache.dtype == b.k_cache.dtype
