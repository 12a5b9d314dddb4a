"""GPU parity of dreams_kv_commit against the CPU oracle (bit-exact caches and lengths), and of the whole
verify step: tree attention, acceptance, commit, then one decode step over the committed cache."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import ATTN_TOL_BF16, LSE_TOL, dense_bits_of, device, f32, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_commit_aliasing_paths(dev, dtype):
    rng = np.random.default_rng(1)
    NL, B, Hkv, S, D, T = 3, 4, 2, 96, 128, 9
    npdt = np.uint16 if dtype == "bf16" else np.float32
    if dtype == "bf16":
        k = rng.integers(0, 65535, size=(NL, B, Hkv, S, D)).astype(np.uint16)
        v = rng.integers(0, 65535, size=(NL, B, Hkv, S, D)).astype(np.uint16)
    else:
        k = rng.standard_normal((NL, B, Hkv, S, D)).astype(np.float32)
        v = rng.standard_normal((NL, B, Hkv, S, D)).astype(np.float32)
    paths = [[0, 2, 5, 7], [0], [0, 1, 4], [0, 2, 3, 5, 6, 8]]
    kv_in = np.array([10, 0, 33, 54], np.int32)
    alen = np.array([len(p) - 1 for p in paths], np.int32)
    path = np.full((B, T), -1, np.int32)
    for b, p in enumerate(paths):
        path[b, :len(p)] = p
    kd, vd = to_dev(k, dev, dtype == "bf16"), to_dev(v, dev, dtype == "bf16")
    out = dreams.kv_commit(kd, vd, to_dev(kv_in, dev), to_dev(path, dev), to_dev(alen, dev))
    torch.cuda.synchronize()
    ref_len = oracle.kv_commit(k, v, kv_in, path, alen)
    assert np.array_equal(out.cpu().numpy(), ref_len)
    assert np.array_equal(dense_bits_of(kd).astype(npdt), k) and np.array_equal(dense_bits_of(vd).astype(npdt), v)


def test_commit_skips_invalid_entries(dev):
    NL, B, Hkv, S, D = 1, 2, 1, 64, 64
    k = torch.arange(NL * B * Hkv * S * D, dtype=torch.float32, device=dev).view(NL, B, Hkv, S, D)
    v = -k.clone()
    k0, v0 = k.clone(), v.clone()
    path = torch.tensor([[0, 0, 3, -1], [0, 70, 2, -1]], dtype=torch.int32, device=dev)   # k=1: src<k; src past cache
    alen = torch.tensor([2, 2], dtype=torch.int32, device=dev)
    kv_in = torch.tensor([5, 0], dtype=torch.int32, device=dev)
    out = dreams.kv_commit(k, v, kv_in, path, alen)
    torch.cuda.synchronize()
    e = k0.clone()
    e[0, 0, 0, 5 + 2] = k0[0, 0, 0, 5 + 3]
    e[0, 1, 0, 0 + 2] = k0[0, 1, 0, 0 + 2]
    assert torch.equal(k, e) and torch.equal(v, -e)
    assert out.tolist() == [8, 3]


def test_full_step_llava7b_full_layers(dev):
    """Verify attention on a layer subset of the 32-layer workload, acceptance, commit of every layer's cache,
    then a single-node decode over the committed cache must reproduce the accepted leaf's tree row."""
    wl = W.WORKLOADS["llava7b_full"]
    layers = [0, 31]
    batch = W.make_batch(wl, layers=layers, with_logits=True)
    kc = to_dev(batch.k_cache, dev, True)
    vc = to_dev(batch.v_cache, dev, True)
    kv = to_dev(batch.kv_len, dev)
    par = to_dev(batch.parent, dev)
    q = to_dev(batch.q, dev, True)
    outs = []
    for li in range(len(layers)):
        note("full step layer %d" % layers[li])
        o, l = dreams.tree_verify_attn(q[li], kc[li], vc[li], kv, par, max_kv_len=wl.max_kv_len)
        outs.append((o, l))
    alen, path, nxt, _ = dreams.tree_accept(to_dev(batch.logits, dev), to_dev(batch.tokens, dev), par)
    kv_out = dreams.kv_commit(kc, vc, kv, path, alen)
    torch.cuda.synchronize()
    ra, rp, rn, _ = oracle.tree_accept(batch.logits, batch.tokens, batch.parent)
    assert np.array_equal(alen.cpu().numpy(), ra) and np.array_equal(path.cpu().numpy(), rp)
    assert np.array_equal(nxt.cpu().numpy(), rn)
    kref, vref = batch.k_cache.copy(), batch.v_cache.copy()
    lref = oracle.kv_commit(kref, vref, batch.kv_len, rp, ra)
    assert np.array_equal(kv_out.cpu().numpy(), lref)
    assert np.array_equal(dense_bits_of(kc), kref) and np.array_equal(dense_bits_of(vc), vref)
    # composition: decode of the last accepted node's query over the committed cache
    for li in range(len(layers)):
        for b in range(wl.batch):
            last = int(rp[b, ra[b]])
            qd = q[li][b:b + 1, :, last:last + 1].contiguous()
            one = torch.full((1, 1), -1, dtype=torch.int32, device=dev)
            Lb = int(batch.kv_len[b]) + int(ra[b])
            od, ld = dreams.tree_verify_attn(qd, kc[li][b:b + 1], vc[li][b:b + 1],
                                             torch.tensor([Lb], dtype=torch.int32, device=dev), one)
            torch.cuda.synchronize()
            ot, lt = outs[li][0][b, :, last].float(), outs[li][1][b, :, last]
            assert float((od[0, :, 0].float() - ot).abs().max()) <= ATTN_TOL_BF16
            assert float((ld[0, :, 0] - lt).abs().max()) <= LSE_TOL


@pytest.mark.gpu
def test_stream_read_touches_every_word_once(dev):
    # the XOR of the sink words is the XOR of every word read: each 16-byte piece is read exactly once
    g = torch.Generator().manual_seed(3)
    for n_words in (4, 4 * 1000, 4 * (1 << 20) + 4 * 77):
        x = torch.randint(-2 ** 31, 2 ** 31 - 1, (n_words,), generator=g, dtype=torch.int64).to(torch.int32)
        sink = dreams.stream_read(x.to(dev))
        torch.cuda.synchronize()
        want = int(np.bitwise_xor.reduce(x.numpy().view(np.uint32)))
        got = int(np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)))
        assert got == want, n_words
