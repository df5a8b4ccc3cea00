"""A whole decode step (quantize, Q-only projection, append, absorbed
attention) captured once as a graph and replayed: every replay must equal the
eager step bit for bit, with eager work and synchronizations between the
replays.  The library allocates nothing and issues no memsets, so its calls
are capturable; launch grids follow the cache's host max_len, which both
sides hold at the final length."""
import numpy as np
import pytest

import gpu_harness as H
from paper_2510_16292_amd import binding as B
from paper_2510_16292_amd import prep
from workloads import configs, gen

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fmt", [B.QSVD_CACHE_F16, B.QSVD_CACHE_I8], ids=["f16", "i8"])
def test_decode_step_graph_replays_match_eager(fmt):
    torch = H.torch()
    wl = configs.get(1)
    L = wl.layer
    pl = prep.prepare_from_weight(gen.weight_matrix(wl), L.r, L.n_q_heads, L.n_kv_heads, L.head_dim)
    dl = B.DeviceLayer(pl)
    prior, steps = [10, 37], 4
    batch, cap = len(prior), max(prior) + steps + 2
    final = max(prior) + steps

    def make_cache():
        dc = B.DeviceCache(fmt, batch, cap, L.r, prior)
        if fmt == B.QSVD_CACHE_F16:
            dc.data.copy_(H.dev(gen.latent_rows(wl, batch, cap)))
        else:
            codes, scales = gen.latent_codes(wl, batch, cap)
            dc.data.copy_(H.dev(codes))
            dc.scale.copy_(H.dev(scales))
        return dc

    ce, cg = make_cache(), make_cache()
    x = H.dev(gen.decode_activations(wl, 0, batch=batch))
    nq = L.n_q_heads * L.head_dim

    def buffers():
        return dict(xq=torch.empty((batch, L.d), dtype=torch.int8, device="cuda"),
                    sx=torch.empty((batch,), dtype=torch.float32, device="cuda"),
                    c_h=torch.empty((batch, L.r), dtype=torch.float16, device="cuda"),
                    cq=torch.empty((batch, L.r), dtype=torch.int8, device="cuda"),
                    sc=torch.empty((batch,), dtype=torch.float32, device="cuda"),
                    q=torch.empty((batch, nq), dtype=torch.float16, device="cuda"),
                    out=torch.empty((batch, nq), dtype=torch.float16, device="cuda"))

    be, bg = buffers(), buffers()
    wsb = B.qsvd_decode_workspace_size(dl.c, ce.c, 1, B.QSVD_ATTN_ABSORBED)
    wse = torch.empty((wsb,), dtype=torch.uint8, device="cuda")
    wsg = torch.empty((wsb,), dtype=torch.uint8, device="cuda")
    P = B.ptr

    def step(dc, b, ws, s):
        f16 = fmt == B.QSVD_CACHE_F16
        B.check(B.qsvd_quantize_act(P(x), batch, L.d, L.d, 8, 1.0, P(b["xq"]), P(b["sx"]), s))
        B.check(B.qsvd_lowrank_qkv_prefill(dl.c, P(b["xq"]), P(b["sx"]), batch, 8, B.QSVD_OUT_Q, P(b["c_h"]),
                                           P(b["cq"]), P(b["sc"]), P(b["q"]), 0, 0, 0, 0, 0, 0, s))
        B.check(B.qsvd_latent_cache_append(dc.c, P(b["c_h"]) if f16 else 0, 0 if f16 else P(b["cq"]),
                                           0 if f16 else P(b["sc"]), 1, s))
        B.check(B.qsvd_latent_decode_attention(dl.c, dc.c, P(b["q"]), 1, B.QSVD_ATTN_ABSORBED, 0.0, P(b["out"]),
                                               P(ws), wsb, s))

    # eager reference outputs, launch configuration held at the final length
    eager = []
    for _ in range(steps):
        ce.c.max_len = final - 1
        step(ce, be, wse, B.stream_handle())
        torch.cuda.synchronize()
        eager.append(H.host(be["out"]).copy())
    H.say(f"graph capture fmt={fmt}")
    cg.c.max_len = final - 1
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(cg, bg, wsg, B.stream_handle())
    assert int(H.host(cg.seq_len).max()) == max(prior), "capture must not run the step"
    for i in range(steps):
        g.replay()
        torch.cuda.synchronize()
        got = H.host(bg["out"])
        assert np.array_equal(got.view(np.uint16), eager[i].view(np.uint16)), f"replay {i}"
        # unrelated eager work between replays
        B.check(B.qsvd_latent_decode_attention(dl.c, ce.c, P(be["q"]), 1, B.QSVD_ATTN_ABSORBED, 0.0,
                                               P(be["out"]), P(wse), wsb, B.stream_handle()))
        torch.cuda.synchronize()
    assert np.array_equal(H.host(cg.seq_len), H.host(ce.seq_len))
    assert np.array_equal(H.host(cg.data).view(np.uint8), H.host(ce.data).view(np.uint8))
    if fmt != B.QSVD_CACHE_F16:
        assert np.array_equal(H.host(cg.scale).view(np.uint32), H.host(ce.scale).view(np.uint32))
    del g
