"""The allocation-free decode attention (static device scratch) against the
entry point with a caller workspace, through the C ABI: two calls in a row on
one GPU, the second with a smaller input, each bit-identical to the
workspace entry point's output (the two share their kernels); a call whose
scratch need exceeds the static array is refused before any launch."""
import numpy as np
import pytest

import gpu_harness as H
from oracle import qsvd_oracle as O
from paper_2510_16292_amd import binding as B
from paper_2510_16292_amd import prep
from workloads import configs, gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()


def _layer(L, seed):
    g = np.random.default_rng(seed)
    A = g.standard_normal((L.d, L.r)) / np.sqrt(L.d)
    Bm = g.standard_normal((L.r, L.N)) / np.sqrt(L.r)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
    return ol, B.DeviceLayer(prep.quantize_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0))


def _cache(wl, fmt, lengths, cap):
    """A device cache holding seeded synthetic latent rows at the given lengths."""
    L = wl.layer
    batch = len(lengths)
    dc = B.DeviceCache(fmt, batch, cap, L.r, lengths)
    rows = gen.latent_rows(wl, batch, cap)
    if fmt == B.QSVD_CACHE_F16:
        dc.data.copy_(H.dev(rows))
    else:
        data = np.zeros((batch, cap, L.r), np.int8)
        scale = np.zeros((batch, cap), np.float32)
        for b in range(batch):
            codes, sc = O.quantize_act(rows[b], 8)
            data[b], scale[b] = codes, sc
        dc.data.copy_(H.dev(data))
        dc.scale.copy_(H.dev(scale))
    return dc


def _both(dl, dc, q, q_len=1):
    """Output of the workspace entry point and of the allocation-free one."""
    want = H.host(H.decode_attention(dl, dc, q, B.QSVD_ATTN_AUTO, q_len=q_len))
    out = H.torch().empty_like(q)
    B.check(B.qsvd_latent_decode_attention_noalloc(dl.c, dc.c, B.ptr(q), q_len, B.QSVD_ATTN_AUTO, 0.0, B.ptr(out),
                                                   B.stream_handle()))
    return H.host(out), want


def test_noalloc_matches_workspace_entry_twice_second_smaller():
    assert B.qsvd_noalloc_scratch_bytes() == 32 << 20
    # call 1: LLaVA-7B-shaped width (32 heads x 128, r = 1536), fp16 cache,
    # 16 ragged sequences up to 2000 tokens (25 MB of scratch)
    L1 = configs.LayerShape(d=256, n_q_heads=32, n_kv_heads=32, head_dim=128, r=1536)
    wl1 = configs.Workload(97, "noalloc-a", L1, "gaussian", 8, 0, 8, B.QSVD_CACHE_F16)
    ol1, dl1 = _layer(L1, 9100)
    lengths1 = [1 + (137 * b) % 2000 for b in range(16)]
    dc1 = _cache(wl1, B.QSVD_CACHE_F16, lengths1, 2000)
    need1 = B.qsvd_decode_workspace_size(dl1.c, dc1.c, 1, B.QSVD_ATTN_AUTO)
    assert 0 < need1 <= B.qsvd_noalloc_scratch_bytes()
    q1 = H.dev(gen.random_rows(91, (16, L1.n_q_heads * L1.head_dim), 1.0))
    H.say(f"noalloc call 1: batch 16, r 1536, fp16 cache, scratch need {need1} B")
    got, want = _both(dl1, dc1, q1)
    assert np.all(np.isfinite(want.astype(np.float32)))
    assert np.array_equal(got.view(np.uint16), want.view(np.uint16))
    # call 2, smaller: grouped heads 28 / 4, r = 1024, int8 cache, 3 sequences
    L2 = configs.LayerShape(d=256, n_q_heads=28, n_kv_heads=4, head_dim=128, r=1024)
    wl2 = configs.Workload(98, "noalloc-b", L2, "gaussian", 8, 0, 8, B.QSVD_CACHE_I8)
    ol2, dl2 = _layer(L2, 9200)
    lengths2 = [5, 300, 77]
    dc2 = _cache(wl2, B.QSVD_CACHE_I8, lengths2, 320)
    need2 = B.qsvd_decode_workspace_size(dl2.c, dc2.c, 1, B.QSVD_ATTN_AUTO)
    assert 0 < need2 < need1
    q2 = H.dev(gen.random_rows(92, (3, L2.n_q_heads * L2.head_dim), 1.0))
    H.say(f"noalloc call 2: batch 3, r 1024, int8 cache, scratch need {need2} B")
    got2, want2 = _both(dl2, dc2, q2)
    assert np.array_equal(got2.view(np.uint16), want2.view(np.uint16))
    # the first shape again after the smaller call: the same bits
    got3, _ = _both(dl1, dc1, q1)
    assert np.array_equal(got3.view(np.uint16), want.view(np.uint16))


def test_noalloc_refuses_more_than_the_static_scratch():
    L = configs.LayerShape(d=256, n_q_heads=40, n_kv_heads=40, head_dim=128, r=3072)
    _, dl = _layer(L, 9300)
    c = B.QsvdCache(B.QSVD_CACHE_F16, 64, 4096, 3072, 0x100000, 0, 0x100000, 4096, 0)
    assert B.qsvd_decode_workspace_size(dl.c, c, 1, B.QSVD_ATTN_AUTO) > B.qsvd_noalloc_scratch_bytes()
    out = H.torch().empty((64, L.n_q_heads * L.head_dim), dtype=H.torch().float16, device="cuda")
    st = B.qsvd_latent_decode_attention_noalloc(dl.c, c, B.ptr(out), 1, B.QSVD_ATTN_AUTO, 0.0, B.ptr(out),
                                                B.stream_handle())
    assert st == B.QSVD_ERR_WORKSPACE, B.last_error()
    assert "static" in B.last_error()
