"""Every verb under HIP-graph replay (the KV commit, which moves the cache in place, from a restored cache).

A graph's kernels start their round-robin over the XCDs at another XCD than direct launches do, and every
cross-workgroup hand-off here (arrival counters, pieces merged in the same launch) must not depend on which.
Each verb is called eagerly, then captured into a graph that writes fresh output tensors; every replay, with
eager work of other grid sizes and the program's own synchronisations between replays, must equal the eager
call bit for bit, leave the counters zero and set no failure flag.  The eager results themselves are held to
the oracle by the verbs' own parity tests on the same kinds of inputs."""
import numpy as np
import pytest
import torch

from gpu_util import device, layer_tensors, note, to_dev
from paper_2606_00535_amd import dreams
from paper_2606_00535_amd import workload as W

pytestmark = pytest.mark.gpu
REPLAYS = 3


@pytest.fixture(scope="module")
def dev():
    d = device()
    dreams.lib()
    return d


def bits(t):
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    elif t.dtype == torch.float32:
        t = t.view(torch.int32)
    return t.cpu().numpy()


def spoil(t):
    if t.dtype in (torch.float32, torch.bfloat16):
        t.fill_(float("nan"))
    else:
        t.fill_(-7)


def replay_matches_eager(dev, call, eager_outs, workspaces, label):
    """Captures call(outs) into a graph writing fresh tensors shaped like eager_outs, replays it REPLAYS times
    and compares each replay with eager_outs bit for bit."""
    torch.cuda.synchronize()
    for ws in workspaces:
        dreams.workspace_status(ws)
    ref = [bits(t) for t in eager_outs]
    outs = [torch.empty_like(t) for t in eager_outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(outs)
    filler = torch.zeros(5 * 64 + 1, device=dev)
    for rep in range(REPLAYS):
        for t in outs:
            spoil(t)
        filler.add_(1.0)
        g.replay()
        torch.cuda.synchronize()
        for ws in workspaces:
            dreams.workspace_status(ws)
        for i, (t, r) in enumerate(zip(outs, ref)):
            assert np.array_equal(bits(t), r), "%s: output %d differs on replay %d" % (label, i, rep)
    note("%s: %d replays equal the eager call" % (label, REPLAYS))


def random_tree(rng, B, T, depth, branch):
    return np.stack([W.random_tree(rng, T, depth, branch) for _ in range(B)]) if T > 1 \
        else np.full((B, 1), -1, np.int32)


@pytest.mark.parametrize("B,T,V", [(1, 60, 32000), (4, 128, 4099)])
def test_tree_accept(dev, B, T, V):
    rng = np.random.default_rng(71)
    par = random_tree(rng, B, T, 6, 4)
    logits = (rng.standard_normal((B, T, V)) * 3).astype(np.float32)
    am = logits.argmax(axis=2)
    tok = np.where(rng.random((B, T)) < 0.7, am[np.arange(B)[:, None], np.maximum(par, 0)],
                   rng.integers(0, V, (B, T))).astype(np.int32)
    tl, tk, pr = to_dev(logits, dev), to_dev(tok, dev), to_dev(par, dev)
    ws = torch.zeros(dreams.tree_accept_workspace_size(B, T, V), dtype=torch.uint8, device=dev)
    eager = dreams.tree_accept(tl, tk, pr, want_target_argmax=True, workspace=ws)
    note("greedy B=%d T=%d V=%d: accepted %s" % (B, T, V, eager[0].cpu().numpy()))
    replay_matches_eager(dev, lambda o: dreams.tree_accept(tl, tk, pr, outputs=tuple(o), workspace=ws),
                         list(eager), [ws], "tree_accept")


@pytest.mark.parametrize("B,T,V,sub", [(1, 60, 32000, 1), (4, 128, 65536, 4)],
                         ids=["row_pieces", "split_pieces"])
def test_tree_accept_sampled(dev, B, T, V, sub):
    # 1x60x32000 takes pieces of 4096 entries per row; 4x128x65536 is past the workgroup count where pieces of
    # 8192 entries in four parts take over
    g = torch.Generator(device=dev)
    g.manual_seed(72)
    rng = np.random.default_rng(72)
    par_h = random_tree(rng, B, T, 8, 4)
    pr = to_dev(par_h, dev)
    tl = torch.randn((B, T, V), generator=g, device=dev) * 3
    dl = tl + torch.randn((B, T, V), generator=g, device=dev)
    tau = 0.8
    rows = dl[torch.arange(B, device=dev)[:, None], pr.clamp(min=0).long()].reshape(B * T, V)
    tk = torch.multinomial(torch.softmax(rows / tau, dim=1), 1, generator=g).reshape(B, T).to(torch.int32)
    uni = torch.rand((B, T), generator=g, device=dev)
    ws = torch.zeros(dreams.tree_accept_sampled_workspace_size(B, T, V), dtype=torch.uint8, device=dev)
    eager = dreams.tree_accept_sampled(tl, dl, tk, pr, uni, tau, workspace=ws)
    note("sampled B=%d T=%d V=%d: accepted %s" % (B, T, V, eager[0].cpu().numpy()))
    replay_matches_eager(dev, lambda o: dreams.tree_accept_sampled(tl, dl, tk, pr, uni, tau, outputs=tuple(o),
                                                                   workspace=ws),
                         list(eager), [ws], "tree_accept_sampled (%d parts a piece)" % sub)


def test_tree_accept_lm_head(dev):
    # the LLaVA-1.6-7B head (hidden 4096, vocabulary 32000) over a 60-node tree, two sequences
    B, T, H, V = 2, 60, 4096, 32000
    g = torch.Generator(device=dev)
    g.manual_seed(73)
    hid = torch.randn((B, T, H), generator=g, device=dev).to(torch.bfloat16)
    wt = (torch.randn((V, H), generator=g, device=dev) * 0.02).to(torch.bfloat16)
    rng = np.random.default_rng(73)
    pr = to_dev(random_tree(rng, B, T, 6, 4), dev)
    tk = torch.randint(0, V, (B, T), generator=g, device=dev, dtype=torch.int32)
    ws = torch.zeros(dreams.tree_accept_lm_head_workspace_size(B, T, H, V), dtype=torch.uint8, device=dev)
    _, _, _, am = dreams.tree_accept_lm_head(hid, wt, tk, pr, want_target_argmax=True, workspace=ws)
    # draft tokens that follow the head's own choices, so that paths grow past the root
    tk = torch.where(torch.rand((B, T), generator=g, device=dev) < 0.7,
                     torch.gather(am, 1, pr.clamp(min=0).long()), tk).contiguous()
    eager = dreams.tree_accept_lm_head(hid, wt, tk, pr, want_target_argmax=True, workspace=ws)
    note("lm head: accepted %s" % eager[0].cpu().numpy())
    replay_matches_eager(dev, lambda o: dreams.tree_accept_lm_head(hid, wt, tk, pr, outputs=tuple(o), workspace=ws),
                         list(eager), [ws], "tree_accept_lm_head")


def test_verify_statistics_and_selection(dev):
    # one graph for the statistics read from the verify rows: attention with entropy, the layer's AE and the
    # layer choice, Eq. 2 importance over the 2880 image tokens, keep 576, gather their K/V (llava7b_layer)
    wl = W.WORKLOADS["llava7b_layer"]
    batch = W.make_batch(wl, with_logits=False, layers=[0])
    q, k, v, kv, par = layer_tensors(batch, 0, dev)
    vb, vc, r = 0, wl.image_tokens, 576
    ws_a = torch.zeros(dreams.tree_verify_attn_workspace_size(dreams.attn_desc(q, k)), dtype=torch.uint8,
                       device=dev)
    ws_v = torch.zeros(dreams.visual_importance_workspace_size(q.shape[0], k.shape[1], vc), dtype=torch.uint8,
                       device=dev)
    ae = torch.tensor([9.0, 0.0, 7.5], device=dev)   # per-layer AE; this layer's goes in the middle

    def chain(o):
        out, lse, ent, ae0, best, imp, keep, ko, vo = o
        dreams.tree_verify_attn_entropy(q, k, v, kv, par, out=out, lse=lse, entropy=ent, workspace=ws_a)
        dreams.attn_entropy_mean(ent, ae=ae0)
        dreams.attn_entropy_mean(ent, ae=ae[1:2])
        dreams.attn_entropy_select(ae, best=best)
        dreams.visual_importance(q, k, kv, lse, vb, vc, importance=imp, workspace=ws_v)
        dreams.visual_topk(imp, r, keep=keep)
        dreams.visual_gather(k, v, vb, keep, k_out=ko, v_out=vo)

    B, Hq, T, D = q.shape
    eager = [torch.empty((B, Hq, T, D), dtype=torch.bfloat16, device=dev),
             torch.empty((B, Hq, T), device=dev), torch.empty((B, Hq, T), device=dev),
             torch.empty(1, device=dev), torch.empty(1, dtype=torch.int32, device=dev),
             torch.empty((B, vc), device=dev), torch.empty((B, r), dtype=torch.int32, device=dev),
             torch.empty((B, k.shape[1], r, D), dtype=torch.bfloat16, device=dev),
             torch.empty((B, k.shape[1], r, D), dtype=torch.bfloat16, device=dev)]
    chain(eager)
    torch.cuda.synchronize()
    note("verify statistics: AE %.4f, layer %d" % (float(eager[3].cpu()[0]), int(eager[4].cpu()[0])))
    replay_matches_eager(dev, chain, eager, [ws_a, ws_v], "verify statistics and selection")


def test_prefill_statistics(dev):
    # the prompt-side statistics in one graph: causal LSE and entropy, the layer's AE and Eq. 2 importance, on
    # two ragged prompts
    p = W.make_prompt(2, 8, 4, 128, (1500, 1137), 40, 1000, seed=74)
    q, k, pl = to_dev(p.q, dev, True), to_dev(p.k_cache, dev, True), to_dev(p.prompt_len, dev)
    ws = torch.zeros(dreams.visual_importance_workspace_size(2, 4, 1000), dtype=torch.uint8, device=dev)

    def chain(o):
        lse, ent, ae, imp = o
        dreams.prefill_attn_stats(q, k, pl, lse=lse, entropy=ent)
        dreams.prefill_attn_entropy_mean(ent, pl, ae=ae)
        dreams.prefill_visual_importance(q, k, pl, lse, 40, 1000, importance=imp, workspace=ws)

    B, Hq, N, _ = q.shape
    eager = [torch.empty((B, Hq, N), device=dev), torch.empty((B, Hq, N), device=dev), torch.empty(1, device=dev),
             torch.empty((B, 1000), device=dev)]
    chain(eager)
    replay_matches_eager(dev, chain, eager, [ws], "prefill statistics")


def test_accept_then_commit(dev):
    # the end of a verify step in one graph: greedy acceptance, then the accepted path's K/V moved into place in
    # every layer; the cache is restored between replays (the commit is in place, so a replay is a repeat only
    # from the same cache)
    NL, B, Hkv, S_cap, D, T, V = 4, 2, 8, 1024, 128, 60, 4099
    rng = np.random.default_rng(75)
    g = torch.Generator(device=dev)
    g.manual_seed(75)
    kv = to_dev(np.array([700, 650], np.int32), dev)
    par_h = random_tree(rng, B, T, 6, 4)
    logits = (rng.standard_normal((B, T, V)) * 3).astype(np.float32)
    am = logits.argmax(axis=2)
    tok = np.where(rng.random((B, T)) < 0.8, am[np.arange(B)[:, None], np.maximum(par_h, 0)],
                   rng.integers(0, V, (B, T))).astype(np.int32)
    tl, tk, pr = to_dev(logits, dev), to_dev(tok, dev), to_dev(par_h, dev)
    k0 = torch.randn((NL, B, Hkv, S_cap, D), generator=g, device=dev).to(torch.bfloat16)
    v0 = torch.randn((NL, B, Hkv, S_cap, D), generator=g, device=dev).to(torch.bfloat16)
    ws = torch.zeros(dreams.tree_accept_workspace_size(B, T, V), dtype=torch.uint8, device=dev)
    kc, vc = k0.clone(), v0.clone()

    def chain(o):
        alen, path, nxt, kv_out = o
        dreams.tree_accept(tl, tk, pr, outputs=(alen, path, nxt, None), workspace=ws)
        dreams.kv_commit(kc, vc, kv, path, alen, kv_len_out=kv_out)

    eager = [torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, T), dtype=torch.int32, device=dev),
             torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, dtype=torch.int32, device=dev)]
    chain(eager)
    torch.cuda.synchronize()
    dreams.workspace_status(ws)
    note("accept then commit: accepted %s, lengths %s" % (eager[0].cpu().numpy(), eager[3].cpu().numpy()))
    k_ref, v_ref = bits(kc), bits(vc)
    ref = [bits(t) for t in eager]
    outs = [torch.empty_like(t) for t in eager]
    kc.copy_(k0)
    vc.copy_(v0)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        chain(outs)
    for rep in range(REPLAYS):
        kc.copy_(k0)
        vc.copy_(v0)
        for t in outs:
            spoil(t)
        graph.replay()
        torch.cuda.synchronize()
        dreams.workspace_status(ws)
        for i, (t, r) in enumerate(zip(outs, ref)):
            assert np.array_equal(bits(t), r), "output %d differs on replay %d" % (i, rep)
        assert np.array_equal(bits(kc), k_ref) and np.array_equal(bits(vc), v_ref), "cache differs on replay %d" % rep
    note("accept then commit: %d replays equal the eager call" % REPLAYS)
