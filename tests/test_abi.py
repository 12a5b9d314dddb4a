"""C ABI of libdreams.so on the CPU: the library loads, exports every symbol include/dreams.h declares, and
rejects bad host-visible arguments (with a message) before anything is enqueued.  No kernel runs here."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dreams.h")


@pytest.fixture(scope="module")
def D():
    from paper_2606_00535_amd import dreams
    if not os.path.exists(dreams.LIBRARY):
        from paper_2606_00535_amd import build
        build.build()
    return dreams


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(dreams_\w+)\s*\(", text, re.M)))


def test_header_and_binding_agree(D):
    assert declared_functions() == sorted(D.EXPORTS)


def test_every_declared_symbol_is_exported(D):
    out = subprocess.run(["nm", "-D", "--defined-only", D.LIBRARY], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT\s+(dreams_\w+)$", out, re.M))
    missing = set(declared_functions()) - exported
    assert not missing, missing
    lib = D.lib()
    for name in declared_functions():
        assert getattr(lib, name) is not None


def test_header_compiles_as_c():
    r = subprocess.run(["gcc", "-std=c99", "-fsyntax-only", "-Wall", "-Werror", "-I/opt/rocm/include",
                        "-D__HIP_PLATFORM_AMD__", "-x", "c", "-"], input='#include "%s"\nint main(void){return 0;}\n'
                       % HEADER, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _desc(D, **kw):
    base = dict(batch=1, num_q_heads=32, num_kv_heads=32, head_dim=128, num_nodes=60, cache_capacity=3200,
                max_kv_len=0, num_splits=8, dtype=D.DREAMS_BF16, scale=0.088)
    base.update(kw)
    return D.AttnDesc(**base)


def _ws(D, desc):
    n = ctypes.c_size_t(123)
    st = D.lib().dreams_tree_verify_attn_workspace_size(ctypes.byref(desc), ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), -1), (dict(num_q_heads=0), -1), (dict(num_kv_heads=0), -1),
    (dict(num_q_heads=30, num_kv_heads=4), -1), (dict(head_dim=96), -2), (dict(num_nodes=0), -1),
    (dict(num_nodes=129), -1), (dict(cache_capacity=59), -1), (dict(max_kv_len=3141), -1),
    (dict(max_kv_len=-5), -1), (dict(num_splits=-1), -1), (dict(num_splits=5000), -1), (dict(dtype=7), -1),
    (dict(scale=float("inf")), -1), (dict(scale=float("nan")), -1),
])
def test_attn_desc_rejected(D, kw, status):
    st, _ = _ws(D, _desc(D, **kw))
    assert st == status
    assert D.lib().dreams_last_error_message().decode() != ""


def test_attn_workspace_size_formula(D):
    # explicit split count: no device query needed; counters, partial accumulators, (m, l) and the entropy
    # terms, each 256-aligned
    desc = _desc(D, num_splits=8)
    st, n = _ws(D, desc)
    assert st == 0
    rows = 32 * 1 * 8 * 64
    up = lambda x: (x + 255) // 256 * 256
    # bf16 partial outputs, fp32 (max, sum) and entropy terms
    assert n == 65536 + up(rows * 128 * 2) + up(rows * 2 * 4) + up(rows * 4)
    assert D.lib().dreams_last_error_message().decode() == ""
    s = ctypes.c_int32(0)
    assert D.lib().dreams_tree_verify_attn_splits(ctypes.byref(desc), ctypes.byref(s)) == 0 and s.value == 8
    assert D.lib().dreams_tree_verify_attn_splits(ctypes.byref(_desc(D, num_splits=4000)), ctypes.byref(s)) == 0
    assert s.value == 25
    assert D.lib().dreams_tree_verify_attn_splits(ctypes.byref(_desc(D, num_splits=3, dtype=D.DREAMS_F32)),
                                                  ctypes.byref(s)) == 0 and s.value == 1
    assert _ws(D, _desc(D, num_splits=1))[1] == 0
    assert _ws(D, _desc(D, dtype=D.DREAMS_F32, num_splits=4))[1] == 0
    # a request above one piece per 128 keys (3200 slots -> 25) or above 32 pieces is reduced
    assert _ws(D, _desc(D, num_splits=4000)) == _ws(D, _desc(D, num_splits=32))
    assert _ws(D, _desc(D, num_splits=20, cache_capacity=640)) == _ws(D, _desc(D, num_splits=10, cache_capacity=640))


def test_attn_call_rejections(D):
    lib = D.lib()
    desc = _desc(D, num_splits=1)
    fake = ctypes.c_void_p(0x100000)
    # batch 0: nothing to do, nothing enqueued
    assert lib.dreams_tree_verify_attn(ctypes.byref(_desc(D, batch=0)), None, None, None, None, None, None, None,
                                       None, None, 0, None) == 0
    assert lib.dreams_tree_verify_attn(ctypes.byref(desc), None, fake, fake, fake, fake, None, fake, None, None, 0,
                                       None) == -1
    assert lib.dreams_tree_verify_attn(ctypes.byref(desc), fake, fake, fake, fake, None, None, fake, None, None, 0,
                                       None) == -1
    assert "parent or tree_mask" in lib.dreams_last_error_message().decode()
    mis = ctypes.c_void_p(0x100002)
    assert lib.dreams_tree_verify_attn(ctypes.byref(desc), mis, fake, fake, fake, fake, None, fake, None, None, 0,
                                       None) == -1
    desc8 = _desc(D, num_splits=8)
    assert lib.dreams_tree_verify_attn(ctypes.byref(desc8), fake, fake, fake, fake, fake, None, fake, None, None, 0,
                                       None) == -3
    assert lib.dreams_tree_verify_attn(ctypes.byref(desc8), fake, fake, fake, fake, fake, None, fake, None, fake, 16,
                                       None) == -3
    assert "needed" in lib.dreams_last_error_message().decode()
    assert lib.dreams_tree_verify_attn(None, fake, fake, fake, fake, fake, None, fake, None, None, 0, None) == -1


def test_accept_rejections_and_sizes(D):
    lib = D.lib()
    n = ctypes.c_size_t(0)
    assert lib.dreams_tree_accept_workspace_size(1, 60, 32000, ctypes.byref(n)) == 0 and n.value > 65536
    assert lib.dreams_tree_accept_workspace_size(1, 0, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_workspace_size(1, 129, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_workspace_size(1, 60, 0, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_workspace_size(-1, 60, 10, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_workspace_size(1, 60, 10, None) == -1
    fake = ctypes.c_void_p(0x100000)
    assert lib.dreams_tree_accept(0, 60, 10, None, None, None, None, None, None, None, None, 0, None) == 0
    assert lib.dreams_tree_accept(1, 60, 10, fake, fake, None, fake, fake, fake, None, fake, 1 << 20, None) == -1
    assert lib.dreams_tree_accept(1, 60, 10, fake, fake, fake, fake, fake, fake, None, None, 0, None) == -3


def test_commit_rejections(D):
    lib = D.lib()
    fake = ctypes.c_void_p(0x100000)
    other = ctypes.c_void_p(0x200000)
    args = lambda **kw: dict(dict(NL=2, stride=4 * 2 * 64 * 128, B=4, Hkv=2, Dh=128, S=64, dt=D.DREAMS_BF16,
                                  k=fake, v=fake, lin=fake, path=fake, alen=fake, ps=60, lout=other), **kw)

    def call(a):
        return lib.dreams_kv_commit(a["NL"], a["stride"], a["B"], a["Hkv"], a["Dh"], a["S"], a["dt"], a["k"], a["v"],
                                    a["lin"], a["path"], a["alen"], a["ps"], a["lout"], None)
    assert call(args(NL=0)) == -1
    assert call(args(Dh=4)) == -2                       # 8-byte rows are not a multiple of 16 bytes
    assert call(args(Dh=256, dt=D.DREAMS_F32)) == -2    # 1 KiB rows
    assert call(args(stride=100)) == -1                 # layers would overlap
    assert call(args(lout=fake)) == -1                  # kv_len_out aliases kv_len_in
    assert "overlap" in lib.dreams_last_error_message().decode()
    assert call(args(k=None)) == -1
    assert call(args(dt=5)) == -1
    assert call(args(B=0)) == 0


def test_check_tree_host(D):
    D.check_tree_host(np.array([-1, 0, 0, 1, 2], np.int32))
    D.check_tree_host(np.array([-1], np.int32))
    for bad in ([0, 0], [-1, 1], [-1, 0, 3], [-1, -1], [-1, 0, -2]):
        with pytest.raises(D.DreamsError):
            D.check_tree_host(np.array(bad, np.int32))


def test_status_strings(D):
    lib = D.lib()
    for s in (0, -1, -2, -3, -4, -5):
        assert lib.dreams_status_string(s).decode().startswith("DREAMS_")
    assert b"unknown" in lib.dreams_status_string(42)


def test_wait_limit_range(D):
    lib = D.lib()
    for bad in (-1.0, 61.0, float("nan")):
        assert lib.dreams_set_wait_limit(bad) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_set_wait_limit(0.2) == 0


def test_workspace_status_rejects_bad_arguments(D):
    lib = D.lib()
    assert lib.dreams_workspace_status(None, 65536, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_workspace_status(ctypes.c_void_p(4096 + 16), 65536, None) == D.DREAMS_ERR_WORKSPACE
    assert lib.dreams_workspace_status(ctypes.c_void_p(4096), 65535, None) == D.DREAMS_ERR_WORKSPACE
    assert lib.dreams_last_error_message().decode() != ""


def test_stream_read_rejects_bad_arguments(D):
    lib = D.lib()
    fake = ctypes.c_void_p(4096)   # never dereferenced: validation fails before any launch
    assert lib.dreams_stream_read(fake, 17, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_stream_read(ctypes.c_void_p(4100), 64, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_stream_read(None, 64, fake, None) == D.DREAMS_ERR_INVALID_ARG


def test_entropy_entry_points_reject_bad_arguments(D):
    lib = D.lib()
    fake = ctypes.c_void_p(0x100000)
    desc = _desc(D, num_splits=1)
    # the entropy output is required (before anything else is looked at)
    assert lib.dreams_tree_verify_attn_entropy(ctypes.byref(desc), fake, fake, fake, fake, fake, None, fake, None,
                                               None, None, 0, None) == D.DREAMS_ERR_INVALID_ARG
    assert "entropy" in lib.dreams_last_error_message().decode()
    assert lib.dreams_tree_verify_attn_entropy(ctypes.byref(desc), fake, fake, fake, fake, fake, None, fake, None,
                                               ctypes.c_void_p(0x100002), None, 0, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_attn_entropy_mean(0, fake, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_attn_entropy_mean(10, None, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_attn_entropy_select(1, fake, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_attn_entropy_select(4, fake, None, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_attn_entropy_select(4, ctypes.c_void_p(0x100001), fake, None) == D.DREAMS_ERR_INVALID_ARG


def test_prefill_entry_points_reject_bad_arguments(D):
    lib = D.lib()
    fake = ctypes.c_void_p(0x100000)
    ok = dict(batch=2, num_q_heads=8, num_kv_heads=2, head_dim=128, num_rows=300, cache_capacity=320, scale=0.088)

    def pdesc(**kw):
        d = dict(ok)
        d.update(kw)
        return D.PrefillDesc(**d)

    def stats(desc, q=fake, k=fake, pl=fake, lse=fake, ent=fake):
        return lib.dreams_prefill_attn_stats(ctypes.byref(desc), q, k, pl, lse, ent, None)

    assert lib.dreams_prefill_attn_stats(None, fake, fake, fake, fake, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(num_q_heads=6, num_kv_heads=4)) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(head_dim=96)) == D.DREAMS_ERR_UNSUPPORTED
    assert stats(pdesc(num_rows=0)) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(cache_capacity=299)) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(scale=float("inf"))) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(), q=None) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(), pl=ctypes.c_void_p(0x100002)) == D.DREAMS_ERR_INVALID_ARG
    assert stats(pdesc(batch=0)) == D.DREAMS_OK                    # nothing to do, nothing launched
    assert stats(pdesc(), lse=None, ent=None) == D.DREAMS_OK       # no output asked for
    assert lib.dreams_prefill_attn_entropy_mean(0, 8, 300, fake, fake, fake, None) == D.DREAMS_ERR_INVALID_ARG
    assert lib.dreams_prefill_attn_entropy_mean(2, 8, 300, fake, None, fake, None) == D.DREAMS_ERR_INVALID_ARG

    def imp(desc, vb, vc, ws=fake, nbytes=1 << 24, lse=fake):
        return lib.dreams_prefill_visual_importance(ctypes.byref(desc), fake, fake, fake, lse, vb, vc, fake, ws,
                                                    nbytes, None)

    assert imp(pdesc(), 0, 301) == D.DREAMS_ERR_INVALID_ARG      # past the prompt rows
    assert imp(pdesc(), -1, 10) == D.DREAMS_ERR_INVALID_ARG
    assert imp(pdesc(), 0, 0) == D.DREAMS_ERR_INVALID_ARG
    assert imp(pdesc(), 0, 300, lse=None) == D.DREAMS_ERR_INVALID_ARG
    assert imp(pdesc(), 0, 300, ws=None) == D.DREAMS_ERR_WORKSPACE
    assert imp(pdesc(), 0, 300, nbytes=65536) == D.DREAMS_ERR_WORKSPACE
    assert imp(pdesc(), 0, 300, ws=ctypes.c_void_p(0x100040)) == D.DREAMS_ERR_WORKSPACE


def test_sampled_accept_rejections_and_sizes(D):
    lib = D.lib()
    n = ctypes.c_size_t(0)

    def r256(x):
        return (x + 255) // 256 * 256

    for B, T, V in [(1, 60, 32000), (16, 128, 152064), (3, 1, 1), (2, 7, 2049)]:
        assert lib.dreams_tree_accept_sampled_workspace_size(B, T, V, ctypes.byref(n)) == 0
        rows, chunks = B * T, (V + 4095) // 4096
        if rows * chunks > 4096:           # large pieces
            chunks = (V + 8191) // 8192
        assert n.value == 65536 + r256(rows * chunks * 32) + r256(rows * chunks * 8) + r256(rows * 8)
    assert lib.dreams_tree_accept_sampled_workspace_size(0, 60, 32000, ctypes.byref(n)) == 0 and n.value == 0
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 0, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 129, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 60, 0, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 60, (1 << 21) + 1, ctypes.byref(n)) == 0   # large
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 60, (1 << 23) + 1, ctypes.byref(n)) == -2
    assert lib.dreams_tree_accept_sampled_workspace_size(31, 128, 100, ctypes.byref(n)) == 0
    assert lib.dreams_tree_accept_sampled_workspace_size(32, 128, 100, ctypes.byref(n)) == -2    # counters
    assert lib.dreams_tree_accept_sampled_workspace_size(1, 60, 10, None) == -1
    fake = ctypes.c_void_p(0x100000)
    f = lib.dreams_tree_accept_sampled
    assert f(0, 60, 10, 1.0, None, None, None, None, None, None, None, None, None, 0, None) == 0
    for tau in (0.0, -1.0, float("inf"), float("nan")):
        assert f(1, 60, 10, tau, fake, fake, fake, fake, fake, fake, fake, fake, fake, 1 << 20, None) == -1
        assert b"temperature" in lib.dreams_last_error_message()
    assert f(1, 60, 10, 1.0, fake, None, fake, fake, fake, fake, fake, fake, fake, 1 << 20, None) == -1
    assert f(1, 60, 10, 1.0, fake, fake, fake, fake, fake, fake, fake, fake, None, 0, None) == -3
    assert f(1, 60, 10, 1.0, fake, fake, fake, fake, fake, fake, fake, fake, fake, 100, None) == -3


def test_lm_head_accept_rejections_and_sizes(D):
    lib = D.lib()
    n = ctypes.c_size_t(0)

    def r256(x):
        return (x + 255) // 256 * 256

    for B, T, H, V in [(1, 60, 4096, 32000), (16, 128, 3584, 152064), (2, 7, 256, 1)]:
        assert lib.dreams_tree_accept_lm_head_workspace_size(B, T, H, V, ctypes.byref(n)) == 0
        tile = 128 if B * T <= 64 else 256         # one 64-row tile by 128 entries, else 128 x 256 tiles
        tiles = (V + tile - 1) // tile
        assert n.value == 65536 + 2 * r256(B * T * tiles * 4)
    assert lib.dreams_tree_accept_lm_head_workspace_size(0, 60, 4096, 32000, ctypes.byref(n)) == 0 and n.value == 0
    assert lib.dreams_tree_accept_lm_head_workspace_size(1, 60, 4000, 32000, ctypes.byref(n)) == -2   # H % 256
    assert lib.dreams_tree_accept_lm_head_workspace_size(1, 60, 0, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_lm_head_workspace_size(1, 129, 4096, 32000, ctypes.byref(n)) == -1
    assert lib.dreams_tree_accept_lm_head_workspace_size(1, 60, 4096, 0, ctypes.byref(n)) == -1
    fake, odd = ctypes.c_void_p(0x100000), ctypes.c_void_p(0x100008)
    f = lib.dreams_tree_accept_lm_head
    assert f(0, 60, 4096, 100, None, None, None, None, None, None, None, None, None, 0, None) == 0
    assert f(1, 60, 4096, 100, fake, None, fake, fake, fake, fake, fake, None, fake, 1 << 24, None) == -1
    assert f(1, 60, 4096, 100, odd, fake, fake, fake, fake, fake, fake, None, fake, 1 << 24, None) == -1   # align
    assert f(1, 60, 4096, 100, fake, fake, fake, fake, fake, fake, fake, None, None, 0, None) == -3
    assert f(1, 60, 4096, 100, fake, fake, fake, fake, fake, fake, fake, None, fake, 100, None) == -3


def test_bindings_reject_bad_tensors_before_any_launch(D):
    """The Python bindings of the newer verbs check dtypes, devices and shapes on the host (no GPU needed)."""
    import torch
    f32 = torch.zeros((1, 2, 8), dtype=torch.float32)
    i32 = torch.zeros((1, 2), dtype=torch.int32)
    u32 = torch.zeros((1, 2), dtype=torch.float32)
    with pytest.raises(ValueError):        # host tensors
        D.tree_accept_sampled(f32, f32, i32, i32, u32, 1.0)
    with pytest.raises(TypeError):         # wrong dtype
        D.tree_accept_sampled(f32.double(), f32, i32, i32, u32, 1.0)
    bf = torch.zeros((1, 2, 256), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        D.tree_accept_lm_head(bf, torch.zeros((10, 256), dtype=torch.bfloat16), i32, i32)
    with pytest.raises(TypeError):
        D.tree_accept_lm_head(bf.float(), torch.zeros((10, 256), dtype=torch.bfloat16), i32, i32)
