"""GPU parity of the attention entropy (dreams_tree_verify_attn_entropy) and of the layer-level AE mean and
distillation-layer choice, against the CPU oracle on the same seeded inputs.

Tolerance of the row entropy (gpu_util.ENTROPY_TOL, 1e-5 absolute).  The kernel forms the scores in fp32 from
the same bf16 inputs the oracle widens to fp64, and sums p and p*(z - m) in fp32.  An error d in the scores
moves H = -sum p ln p by at most d * sum_j p_j |ln p_j + H| <= d * 2 ln n, and the fp32 sums add a relative
error of a few units of 2^-24 per term to l and to e/l (|e/l| <= ln n / ln 2 in log2 units).  The matrix cores
multiply the bf16 entries exactly and accumulate in fp32, so d is a few 1e-7 here; the tests report the observed
maximum (under 2e-6 on every shape).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import ENTROPY_TOL as ENT_TOL, f32, layer_tensors, note, device
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
                kv_len=300, image_tokens=0, num_nodes=16, depth=4, max_branch=3, vocab=64, agree=0.7, seed=21)
    base.update(kw)
    return W.Workload(**base)


def oracle_entropy(batch, li=0, parent=None, mask=None, k=None):
    return oracle.tree_attn_entropy(f32(batch.q[li]), f32(batch.k_cache[li]) if k is None else k, batch.kv_len,
                                    batch.parent if parent is None and mask is None else parent, batch.scale,
                                    batch.wl.num_kv_heads, tree_mask=mask)


# every bf16 row configuration, one and several pieces, both merges, D = 64 and 128
CASES = [  # (D, Hq, Hkv, T, depth, branch, L, splits)
    (128, 4, 2, 16, 4, 3, 300, 1),      # 32 rows, one piece
    (128, 4, 2, 16, 4, 3, 300, 3),      # 32 rows, merge kernel
    (128, 2, 2, 9, 3, 3, 400, 3),       # 16 rows (4 waves, 4 key groups)
    (128, 2, 2, 60, 6, 4, 1000, 7),     # 64 rows (2 key groups)
    (128, 4, 2, 60, 6, 4, 2000, 1),     # 128 rows, long piece
    (128, 7, 1, 128, 8, 6, 700, 2),     # 128-row workgroups (two 16-row blocks per wave), GQA
    (64, 2, 1, 100, 8, 6, 130, 4),      # head_dim 64, T > 64
    (64, 4, 4, 16, 4, 3, 513, 0),       # head_dim 64, library's choice
    (128, 2, 2, 33, 5, 3, 0, 2),        # empty prefix
    (128, 64, 64, 16, 4, 3, 400, 4),    # merge inside the launch (512 workgroups)
    (64, 48, 48, 60, 6, 4, 700, 3),     # merge inside the launch, head_dim 64
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "D%d_Hq%d_Hkv%d_T%d_L%d_S%d" % (c[0], c[1], c[2], c[3], c[6], c[7]))
def test_entropy_parity(dev, case):
    D, Hq, Hkv, T, depth, br, L, splits = case
    wl = small_wl(head_dim=D, num_q_heads=Hq, num_kv_heads=Hkv, num_nodes=T, depth=depth, max_branch=br, kv_len=L)
    batch = W.make_batch(wl, with_logits=False, kv_lens=[L, max(0, L - 37)])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    note("entropy %s" % (case,))
    out, lse, ent = dreams.tree_verify_attn_entropy(q, k, v, kv, par, num_splits=splits)
    out0, lse0 = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=splits)
    torch.cuda.synchronize()
    # the entropy term leaves the attention output and lse bit for bit as they are without it
    assert torch.equal(out.view(torch.int16), out0.view(torch.int16)) and torch.equal(lse, lse0)
    ref = oracle_entropy(batch)
    err = float(np.abs(ent.cpu().numpy().astype(np.float64) - ref).max())
    note("entropy %s: max_abs=%.3e (tol %.0e), H in [%.3f, %.3f]" % (case, err, ENT_TOL, ref.min(), ref.max()))
    assert err <= ENT_TOL


def test_entropy_uniform_rows(dev):
    # equal keys: every row's attention is uniform over its n visible slots, H = ln n
    wl = small_wl(num_nodes=60, depth=6, max_branch=4, kv_len=777)
    batch = W.make_batch(wl, with_logits=False)
    batch.k_cache[0][...] = batch.k_cache[0][:, :, :1]
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, _, ent = dreams.tree_verify_attn_entropy(q, k, v, kv, par, num_splits=3)
    torch.cuda.synchronize()
    ref = oracle_entropy(batch)
    got = ent.cpu().numpy().astype(np.float64)
    for b in range(wl.batch):
        depth = np.zeros(wl.num_nodes, np.int64)
        for i in range(1, wl.num_nodes):
            depth[i] = depth[batch.parent[b, i]] + 1
        n = batch.kv_len[b] + depth + 1
        assert np.max(np.abs(ref[b] - np.log(n)[None, :])) <= 1e-12
        assert np.max(np.abs(got[b] - np.log(n)[None, :])) <= ENT_TOL
    note("uniform rows: max_abs=%.3e" % float(np.abs(got - ref).max()))


def test_entropy_nonancestor_keys_bitwise(dev):
    wl = small_wl(num_q_heads=2, num_kv_heads=2, num_nodes=60, depth=6, max_branch=4, kv_len=700, batch=1)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, _, e0 = dreams.tree_verify_attn_entropy(q, k, v, kv, par, num_splits=3)
    e0 = e0.cpu().numpy()
    parent = batch.parent[0]
    L = int(batch.kv_len[0])
    for j in (5, 37, 59):
        anc = set()
        for i in range(60):
            x = i
            while x >= 0:
                if x == j:
                    anc.add(i)
                x = parent[x] if x > 0 else -1
        k2 = k.clone()
        k2[0, :, L + j] = k2[0, :, L + j] * 2.0 + 1.0
        _, _, e1 = dreams.tree_verify_attn_entropy(q, k2, v, kv, par, num_splits=3)
        e1 = e1.cpu().numpy()
        for i in range(60):
            if i in anc:
                assert np.all(e1[0, :, i] != e0[0, :, i]), (j, i)
            else:
                assert np.array_equal(e1[0, :, i], e0[0, :, i]), (j, i)


def test_entropy_tree_mask_input(dev):
    # an explicit mask: the ancestor closure with arbitrary extra bits in some rows, and (empty prefix) one
    # row that sees nothing, whose entropy is 0
    from pins import ancestor_closure, mask_bits_from_closure
    wl = small_wl(num_nodes=100, depth=8, max_branch=6, kv_len=333, head_dim=64)
    batch = W.make_batch(wl, with_logits=False)
    rng = np.random.default_rng(9)
    bits = np.stack([mask_bits_from_closure(ancestor_closure(batch.parent[b])) for b in range(2)])
    bits[:, 10:20] |= rng.integers(0, 2 ** 62, size=bits[:, 10:20].shape, dtype=np.int64).astype(np.uint64)
    bits[:, 7] = 0
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    m = torch.from_numpy(bits.view(np.int64)).to(dev)
    for kvlen in (batch.kv_len, np.zeros(2, np.int32)):
        _, _, ent = dreams.tree_verify_attn_entropy(q, k, v, torch.from_numpy(kvlen).to(dev), None, tree_mask=m,
                                                    num_splits=2)
        torch.cuda.synchronize()
        ref = oracle.tree_attn_entropy(f32(batch.q[0]), f32(batch.k_cache[0]), kvlen, None, batch.scale,
                                       wl.num_kv_heads, tree_mask=bits)
        got = ent.cpu().numpy().astype(np.float64)
        err = float(np.abs(got - ref).max())
        note("tree mask, prefix %d: max_abs=%.3e" % (int(kvlen[0]), err))
        assert err <= ENT_TOL
        if kvlen[0] == 0:
            assert np.all(got[:, :, 7] == 0.0)


def test_entropy_fp32_path(dev):
    batch = W.make_batch(W.WORKLOADS["tiny"], with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, _, ent = dreams.tree_verify_attn_entropy(q, k, v, kv, par)
    torch.cuda.synchronize()
    ref = oracle_entropy(batch)
    err = float(np.abs(ent.cpu().numpy().astype(np.float64) - ref).max())
    note("fp32 path: max_abs=%.3e" % err)
    assert err <= 1e-4


@pytest.mark.parametrize("name", ["llava7b_layer"])
def test_entropy_full_size(dev, name):
    wl = W.WORKLOADS[name]
    batch = W.make_batch(wl, with_logits=False, layers=[0])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    _, _, ent = dreams.tree_verify_attn_entropy(q, k, v, kv, par, max_kv_len=wl.max_kv_len)
    torch.cuda.synchronize()
    ref = oracle_entropy(batch)
    err = float(np.abs(ent.cpu().numpy().astype(np.float64) - ref).max())
    note("%s: every row, max_abs=%.3e, H in [%.3f, %.3f]" % (name, err, ref.min(), ref.max()))
    assert err <= ENT_TOL


def test_layer_mean_and_choice(dev):
    rng = np.random.default_rng(5)
    for count in (1, 7, 256, 1000, 3 * 32 * 60, 123457):
        e = rng.uniform(0.0, 9.0, count).astype(np.float32)
        got = float(dreams.attn_entropy_mean(torch.from_numpy(e).to(dev)).cpu()[0])
        ref = oracle.attn_entropy_mean(e)
        assert abs(got - ref) <= 2 ** -23 * abs(ref), (count, got, ref)
    cases = [rng.uniform(0.0, 8.0, n).astype(np.float32) for n in (2, 3, 5, 32, 40)]
    cases += [np.array([5.0, 4.0, 4.5, 1.0, 1.5], np.float32), np.array([2.0, 2.0, 2.0], np.float32),
              np.array([4.0, 4.0, 0.5], np.float32), np.round(rng.uniform(0, 4, 24) * 2) / 2]
    for ae in cases:
        ae = np.asarray(ae, np.float32)
        got = int(dreams.attn_entropy_select(torch.from_numpy(ae).to(dev)).cpu()[0])
        assert got == oracle.attn_entropy_select(ae), ae


def test_layer_choice_from_the_layers_of_a_model(dev):
    # the whole chain on a 4-layer model: per-layer entropies, AE per layer on the device, then the choice
    wl = small_wl(num_layers=4, num_nodes=60, depth=6, max_branch=4, kv_len=500, seed=23)
    batch = W.make_batch(wl, with_logits=False)
    ae_dev = torch.empty(wl.num_layers, dtype=torch.float32, device=dev)
    ae_ref = []
    for li in range(wl.num_layers):
        q, k, v, kv, par = layer_tensors(batch, li, dev)
        _, _, ent = dreams.tree_verify_attn_entropy(q, k, v, kv, par, num_splits=2)
        dreams.attn_entropy_mean(ent, ae=ae_dev[li:li + 1])
        ae_ref.append(oracle.attn_entropy_mean(oracle_entropy(batch, li)))
    best = int(dreams.attn_entropy_select(ae_dev).cpu()[0])
    got = ae_dev.cpu().numpy()
    note("AE per layer: device %s, oracle %s, choice %d" % (np.round(got, 5), np.round(ae_ref, 5), best))
    assert np.max(np.abs(got - np.array(ae_ref))) <= ENT_TOL
    assert best == oracle.attn_entropy_select(got)
