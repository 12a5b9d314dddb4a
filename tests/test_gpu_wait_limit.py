"""A bounded wait that gives up is reported, not silent: with the wait limit forced to 0 from the host
(dreams_set_wait_limit), the waits inside sampled acceptance and the attention merge give up at once, every
kernel still exits normally, and dreams_workspace_status reports DREAMS_ERR_DEVICE; with the default limit
restored, the same calls give the oracle's results and a clean status."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import ATTN_TOL_BF16, device, f32, layer_tensors, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture
def dev():
    d = device()
    dreams.lib()
    yield d
    dreams.set_wait_limit(0.2)


def test_sampled_wait_gives_up_and_is_reported(dev):
    wl = W.Workload(name="wait", batch=2, num_q_heads=2, num_kv_heads=2, head_dim=64, dtype="bf16", num_layers=1,
                    kv_len=64, image_tokens=0, num_nodes=40, depth=6, max_branch=4, vocab=20000, agree=0.7, seed=51)
    smp = W.make_sampled(wl)
    tl, dl = to_dev(smp.target_logits, dev), to_dev(smp.draft_logits, dev)
    tok, par, uni = to_dev(smp.tokens, dev), to_dev(smp.parent, dev), to_dev(smp.uniforms, dev)
    B, T, V = smp.target_logits.shape
    ws = torch.zeros(dreams.tree_accept_sampled_workspace_size(B, T, V), dtype=torch.uint8, device=dev)
    dreams.set_wait_limit(0.0)
    note("sampled acceptance with every wait giving up at once")
    dreams.tree_accept_sampled(tl, dl, tok, par, uni, smp.temperature, workspace=ws)
    torch.cuda.synchronize()
    with pytest.raises(dreams.DreamsError) as ei:
        dreams.workspace_status(ws)
    assert ei.value.status == dreams.DREAMS_ERR_DEVICE and "gave up" in str(ei.value)
    dreams.workspace_status(ws)                # the flag was cleared by the read
    words = ws[:65536 - 128].view(torch.int32).cpu().numpy()
    nz = np.nonzero(words)[0]
    note("non-zero counter words after the call: %d %s %s" % (len(nz), nz[:16].tolist(), words[nz[:16]].tolist()))
    assert len(nz) == 0                        # and the arrival words are back at zero
    dreams.set_wait_limit(0.2)
    alen, path, nxt = dreams.tree_accept_sampled(tl, dl, tok, par, uni, smp.temperature, workspace=ws)
    torch.cuda.synchronize()
    dreams.workspace_status(ws)
    ref = oracle.tree_accept_sampled(smp.target_logits, smp.draft_logits, smp.tokens, smp.parent, smp.uniforms,
                                     smp.temperature)
    assert np.array_equal(alen.cpu().numpy(), ref[0]) and np.array_equal(path.cpu().numpy(), ref[1])
    assert np.array_equal(nxt.cpu().numpy(), ref[2])


def test_attention_merge_wait_gives_up_and_is_reported(dev):
    # 8 pieces per row set in one round: merging workgroups wait for the pieces
    wl = W.Workload(name="wait_attn", batch=2, num_q_heads=4, num_kv_heads=2, head_dim=128, dtype="bf16",
                    num_layers=1, kv_len=2000, image_tokens=0, num_nodes=60, depth=6, max_branch=4, vocab=64,
                    agree=0.7, seed=52)
    batch = W.make_batch(wl, with_logits=False)
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    desc = dreams.attn_desc(q, k, num_splits=8)
    ws = torch.zeros(dreams.tree_verify_attn_workspace_size(desc), dtype=torch.uint8, device=dev)
    dreams.set_wait_limit(0.0)
    note("attention merge with every wait giving up at once")
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=8, workspace=ws)
    torch.cuda.synchronize()
    with pytest.raises(dreams.DreamsError) as ei:
        dreams.workspace_status(ws)
    assert ei.value.status == dreams.DREAMS_ERR_DEVICE
    # the pieces that had not arrived leave their counts behind: clear the counter region before reuse
    ws[:65536].zero_()
    dreams.set_wait_limit(0.2)
    out, lse = dreams.tree_verify_attn(q, k, v, kv, par, num_splits=8, workspace=ws)
    torch.cuda.synchronize()
    dreams.workspace_status(ws)
    ref, _ = oracle.tree_attn(f32(batch.q[0]), f32(batch.k_cache[0]), f32(batch.v_cache[0]), batch.kv_len,
                              batch.parent, batch.scale, wl.num_kv_heads)
    assert float(np.abs(out.float().cpu().numpy() - ref).max()) <= ATTN_TOL_BF16
    assert not ws[:65536].cpu().numpy().any()
