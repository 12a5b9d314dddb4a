"""GPU parity of dreams_tree_accept against the CPU oracle: bit-exact accepted lengths, paths, bonus tokens
and per-node target argmax, on the workloads' seeded inputs and on tie-heavy tiny vocabularies."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import device, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def run_and_compare(dev, logits, tokens, parent, label, logits_dev=None):
    lg = to_dev(logits, dev) if logits_dev is None else logits_dev
    alen, path, nxt, am = dreams.tree_accept(lg, to_dev(tokens, dev), to_dev(parent, dev), want_target_argmax=True)
    torch.cuda.synchronize()
    ra, rp, rn, ram = oracle.tree_accept(logits, tokens, parent)
    ga, gp, gn, gam = alen.cpu().numpy(), path.cpu().numpy(), nxt.cpu().numpy(), am.cpu().numpy()
    note("%s: accepted mean %.3f, mismatching rows: len %d path %d next %d argmax %d" % (
        label, float(ra.mean()), int((ga != ra).sum()), int((gp != rp).any(axis=1).sum()), int((gn != rn).sum()),
        int((gam != ram).sum())))
    assert np.array_equal(gam, ram), label
    assert np.array_equal(ga, ra) and np.array_equal(gp, rp) and np.array_equal(gn, rn), label
    return ra


@pytest.mark.parametrize("name", ["tiny", "llava7b_layer", "llava7b_full", "llava13b_layer", "gqa_long"])
def test_workload_parity(dev, name):
    wl = W.WORKLOADS[name].replace(num_layers=1)
    batch = W.make_batch(wl, layers=[], with_logits=True)
    note("%s: B=%d T=%d V=%d" % (name, wl.batch, wl.num_nodes, wl.vocab))
    ra = run_and_compare(dev, batch.logits, batch.tokens, batch.parent, name)
    assert np.all((ra >= 0) & (ra <= wl.depth))


@pytest.mark.parametrize("V", [1, 2, 3, 4, 7, 4096, 4099, 40003])
def test_ties_and_ragged_vocab(dev, V):
    rng = np.random.default_rng(V)
    B, T = 64, 20
    parent = np.stack([W.random_tree(rng, T, 5, 4) for _ in range(B)])
    vals = np.array([-1.0, -0.0, 0.0, 0.5, 1.0], dtype=np.float32)
    logits = rng.choice(vals, size=(B, T, V)).astype(np.float32)
    am = np.argmax(logits, axis=2)
    tokens = np.where(rng.random((B, T)) < 0.8, am[np.arange(B)[:, None], np.maximum(parent, 0)],
                      rng.integers(0, V, (B, T))).astype(np.int32)
    run_and_compare(dev, logits, tokens, parent, "ties V=%d" % V)


def test_misaligned_logits_scalar_path(dev):
    rng = np.random.default_rng(9)
    B, T, V = 3, 16, 1000
    parent = np.stack([W.random_tree(rng, T, 4, 3) for _ in range(B)])
    logits = rng.standard_normal((B, T, V)).astype(np.float32)
    tokens = rng.integers(0, V, (B, T)).astype(np.int32)
    big = torch.zeros(B * T * V + 1, dtype=torch.float32, device=dev)
    big[1:] = to_dev(logits.reshape(-1), dev)
    view = big[1:].view(B, T, V)          # 4-byte aligned, not 16-byte aligned
    run_and_compare(dev, logits, tokens, parent, "misaligned", logits_dev=view)


def test_extreme_cases(dev):
    rng = np.random.default_rng(10)
    B, T, V = 8, 128, 777
    parent = np.stack([W.random_tree(rng, T, 8, 6) for _ in range(B)])
    logits = rng.standard_normal((B, T, V)).astype(np.float32) * 3
    am = np.argmax(logits, axis=2)
    agree = am[np.arange(B)[:, None], np.maximum(parent, 0)].astype(np.int32)
    run_and_compare(dev, logits, agree, parent, "all agree")
    run_and_compare(dev, logits, (agree + 1) % V, parent, "none agree")
    chain = np.tile(W.chain_tree(T), (B, 1))
    run_and_compare(dev, logits, am[np.arange(B)[:, None], np.maximum(chain, 0)].astype(np.int32), chain, "chain")
    one = np.full((B, 1), -1, np.int32)
    run_and_compare(dev, logits[:, :1], agree[:, :1], one, "single node")


def test_one_workspace_serves_every_shape(dev):
    """Calls of different shapes (and both verbs) one after another on a single workspace."""
    n = max(dreams.tree_accept_workspace_size(16, 128, 152064), 1 << 22)
    ws = torch.zeros(n, dtype=torch.uint8, device=dev)
    rng = np.random.default_rng(12)
    for B, T, V in [(16, 128, 5000), (3, 7, 11), (1, 60, 32000), (8, 20, 4099), (2, 128, 3)]:
        parent = np.stack([W.random_tree(rng, T, min(T - 1, 6), 6) for _ in range(B)])
        logits = rng.standard_normal((B, T, V)).astype(np.float32)
        tokens = rng.integers(0, V, (B, T)).astype(np.int32)
        alen, path, nxt, am = dreams.tree_accept(to_dev(logits, dev), to_dev(tokens, dev), to_dev(parent, dev),
                                                 want_target_argmax=True, workspace=ws)
        torch.cuda.synchronize()
        ra, rp, rn, ram = oracle.tree_accept(logits, tokens, parent)
        assert np.array_equal(am.cpu().numpy(), ram) and np.array_equal(path.cpu().numpy(), rp), (B, T, V)
        assert np.array_equal(alen.cpu().numpy(), ra) and np.array_equal(nxt.cpu().numpy(), rn), (B, T, V)
    assert not ws[:65536].any()


def test_workspace_reuse_and_repeat(dev):
    wl = W.WORKLOADS["llava7b_layer"].replace(batch=4)
    batch = W.make_batch(wl, layers=[], with_logits=True)
    lg, tk, pr = to_dev(batch.logits, dev), to_dev(batch.tokens, dev), to_dev(batch.parent, dev)
    n = dreams.tree_accept_workspace_size(4, 60, 32000)
    ws = torch.zeros(n, dtype=torch.uint8, device=dev)
    outs = [dreams.tree_accept(lg, tk, pr, want_target_argmax=True, workspace=ws) for _ in range(4)]
    torch.cuda.synchronize()
    assert not ws[:65536].any()          # the arrival counters are back to zero
    for o in outs[1:]:
        for x, y in zip(o, outs[0]):
            assert torch.equal(x, y)
