"""Small helpers for the GPU tests: upload seeded inputs, call the C ABI
through the binding, download results.  No arithmetic of the method here."""
import sys

import numpy as np

from paper_2510_16292_amd import binding as B


def torch():
    import torch as _t
    return _t


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a):
    t = torch()
    return t.from_numpy(np.ascontiguousarray(a)).to("cuda")


def host(t):
    torch().cuda.synchronize()
    return t.detach().cpu().numpy()


def empty(shape, dtype):
    t = torch()
    return t.empty(shape, dtype=dtype, device="cuda")


def quantize_act(x_np, bits=8, clip=1.0, K=None):
    """x_np fp16 [M][ld]; quantizes the first K columns (default all).
    Returns (xq bytes [M][K or K/2], sx [M])."""
    t = torch()
    M, ld = x_np.shape
    K = ld if K is None else K
    x = dev(x_np)
    width = K if bits == 8 else K // 2
    xq = t.empty((M, width), dtype=t.uint8, device="cuda")
    sx = t.empty((M,), dtype=t.float32, device="cuda")
    B.check(B.qsvd_quantize_act(B.ptr(x), M, K, ld, bits, clip, B.ptr(xq), B.ptr(sx), B.stream_handle()))
    return host(xq), host(sx)


def quantize_act_rotated(x_np, signs_np, block, bits=8, clip=1.0):
    """Q(X H1^T) on the device: x_np fp16 [M][K], signs_np int8 [K] or None.
    Returns (xq bytes [M][K or K/2], sx [M])."""
    t = torch()
    M, K = x_np.shape
    x = dev(x_np)
    sg = dev(signs_np) if signs_np is not None else None
    xq = t.empty((M, K if bits == 8 else K // 2), dtype=t.uint8, device="cuda")
    sx = t.empty((M,), dtype=t.float32, device="cuda")
    B.check(B.qsvd_quantize_act_rotated(B.ptr(x), M, K, K, bits, clip, B.ptr(sg), block, B.ptr(xq), B.ptr(sx),
                                        B.stream_handle()))
    return host(xq), host(sx)


class Prefill:
    """Device buffers for one projection call of M tokens."""

    def __init__(self, dl, M, mask=7, debug=True, abits=8):
        t = torch()
        self.dl, self.M, self.mask, self.abits = dl, M, mask, abits
        nq, nkv, r, N = dl.n_q_heads * dl.head_dim, dl.n_kv_heads * dl.head_dim, dl.r, dl.N
        per = 1 if abits == 8 else 2           # codes per byte
        self.xq = t.empty((M, dl.d // per), dtype=t.int8 if abits == 8 else t.uint8, device="cuda")
        self.sx = t.empty((M,), dtype=t.float32, device="cuda")
        self.c_h = t.empty((M, r), dtype=t.float16, device="cuda")
        self.cq = t.empty((M, r // per), dtype=t.int8 if abits == 8 else t.uint8, device="cuda")
        self.sc = t.empty((M,), dtype=t.float32, device="cuda")
        self.q = t.empty((M, nq), dtype=t.float16, device="cuda")
        self.k = t.empty((M, nkv), dtype=t.float16, device="cuda")
        self.v = t.empty((M, nkv), dtype=t.float16, device="cuda")
        self.acc_xa = t.empty((M, r), dtype=t.int32, device="cuda") if debug else None
        self.acc_cb = t.empty((M, N), dtype=t.int32, device="cuda") if debug else None
        self.ws_bytes = B.qsvd_prefill_workspace_size(dl.c, M, mask)
        self.ws = t.empty((max(self.ws_bytes, 1),), dtype=t.uint8, device="cuda")

    def run(self, x, signs=None, block=0):
        """x: device fp16 [M][d]; with block > 0 the activations are rotated
        online (device int8 signs [d] or None) before quantization."""
        s = B.stream_handle()
        if block:
            B.check(B.qsvd_quantize_act_rotated(B.ptr(x), self.M, self.dl.d, self.dl.d, self.abits, 1.0, B.ptr(signs),
                                                block, B.ptr(self.xq), B.ptr(self.sx), s))
        else:
            B.check(B.qsvd_quantize_act(B.ptr(x), self.M, self.dl.d, self.dl.d, self.abits, 1.0, B.ptr(self.xq),
                                        B.ptr(self.sx), s))
        B.check(B.qsvd_lowrank_qkv_prefill(self.dl.c, B.ptr(self.xq), B.ptr(self.sx), self.M, self.abits, self.mask,
                                           B.ptr(self.c_h), B.ptr(self.cq), B.ptr(self.sc), B.ptr(self.q),
                                           B.ptr(self.k), B.ptr(self.v), B.ptr(self.acc_xa), B.ptr(self.acc_cb),
                                           B.ptr(self.ws), self.ws_bytes, s))
        return self

    def result(self):
        out = dict(xq=host(self.xq), sx=host(self.sx), C_h=host(self.c_h), cq=host(self.cq), sc=host(self.sc))
        if self.mask & B.QSVD_OUT_Q:
            out["Q"] = host(self.q)
        if self.mask & B.QSVD_OUT_K:
            out["K"] = host(self.k)
        if self.mask & B.QSVD_OUT_V:
            out["V"] = host(self.v)
        if self.acc_xa is not None:
            out["acc_xa"], out["acc_cb"] = host(self.acc_xa), host(self.acc_cb)
        return out


def decode_attention(dl, dc, q_dev, mode, sm_scale=0.0, q_len=1, rope_theta=None):
    """q_dev: [batch, q_len, Hq*head_dim] (or [batch, Hq*head_dim] for q_len 1).
    With rope_theta, the rotary variant (reconstruct form only)."""
    t = torch()
    out = t.empty_like(q_dev)
    ws_mode = B.QSVD_ATTN_RECONSTRUCT if rope_theta else mode
    ws_bytes = B.qsvd_decode_workspace_size(dl.c, dc.c, q_len, ws_mode)
    ws = t.empty((max(ws_bytes, 1),), dtype=t.uint8, device="cuda")
    if rope_theta:
        B.check(B.qsvd_latent_decode_attention_rope(dl.c, dc.c, B.ptr(q_dev), q_len, mode, sm_scale, rope_theta,
                                                    B.ptr(out), B.ptr(ws), ws_bytes, B.stream_handle()))
    else:
        B.check(B.qsvd_latent_decode_attention(dl.c, dc.c, B.ptr(q_dev), q_len, mode, sm_scale, B.ptr(out),
                                               B.ptr(ws), ws_bytes, B.stream_handle()))
    return out


def append(dc, c_h=None, cq=None, sc=None, n_new=1):
    B.check(B.qsvd_latent_cache_append(dc.c, B.ptr(c_h), B.ptr(cq), B.ptr(sc), n_new, B.stream_handle()))


def close_enough(got, want, max_abs=2e-2, rel_l2=5e-3):
    """Floating-point outputs against the oracle: every element within
    max_abs * (1 + |want|) -- max_abs itself on outputs of unit scale; the fp16
    roundings of the attention path (the absorbed query, the chunk partials,
    the merged latent output, the output) are relative, so on larger outputs
    the bound grows with the value -- and the whole within relative L2 error
    rel_l2.  Returns (ok, (max-abs error, relative L2, rms of want, max
    scaled error))."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    err = np.abs(got - want)
    scaled = err / (1.0 + np.abs(want))
    rel = np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30)
    return scaled.max() <= max_abs and rel <= rel_l2, (float(err.max()), float(rel), float(np.sqrt(np.mean(want ** 2))),
                                                       float(scaled.max()))


def prefill_attention(q_dev, k_dev, v_dev, lengths, n_q_heads, n_kv_heads, head_dim, max_seqlen=None, sm_scale=0.0,
                      rope_theta=None):
    """Causal prefill attention of sequences back to back (lengths) over the
    device Q, K, V rows (rotary with rope_theta); returns the device output."""
    t = torch()
    cu = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    cu_d = dev(cu)
    out = t.empty_like(q_dev)
    ms = max(lengths) if max_seqlen is None else max_seqlen
    if rope_theta:
        B.check(B.qsvd_prefill_attention_rope(B.ptr(q_dev), B.ptr(k_dev), B.ptr(v_dev), len(lengths), B.ptr(cu_d), ms,
                                              n_q_heads, n_kv_heads, head_dim, sm_scale, rope_theta, B.ptr(out),
                                              B.stream_handle()))
    else:
        B.check(B.qsvd_prefill_attention(B.ptr(q_dev), B.ptr(k_dev), B.ptr(v_dev), len(lengths), B.ptr(cu_d), ms,
                                         n_q_heads, n_kv_heads, head_dim, sm_scale, B.ptr(out), B.stream_handle()))
    t.cuda.synchronize()
    return out
