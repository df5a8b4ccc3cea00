"""ctypes binding of libqsvd.so (include/qsvd.h): argument marshalling only.

The functions named like the C entry points take raw pointers (ints) and
return the status code.  The small helpers below them (:class:`DeviceLayer`,
:class:`DeviceCache`, :func:`check`) hold the torch device tensors that back
the C structs and turn a non-OK status into an exception.  Every step of the
hot path runs in the HIP library; nothing here computes.
"""
import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "_lib", "libqsvd.so")

QSVD_OK, QSVD_ERR_INVALID_ARG, QSVD_ERR_UNSUPPORTED, QSVD_ERR_CAPACITY, QSVD_ERR_WORKSPACE, QSVD_ERR_HIP = range(6)
QSVD_CACHE_F16, QSVD_CACHE_I8, QSVD_CACHE_I4 = 0, 1, 2
QSVD_ATTN_AUTO, QSVD_ATTN_ABSORBED, QSVD_ATTN_RECONSTRUCT = 0, 1, 2
QSVD_OUT_Q, QSVD_OUT_K, QSVD_OUT_V = 1, 2, 4

EXPORTED = [
    "qsvd_quantize_act", "qsvd_quantize_act_rotated", "qsvd_lowrank_qkv_prefill", "qsvd_prefill_workspace_size",
    "qsvd_latent_cache_append", "qsvd_decode_project_append", "qsvd_prefill_attention",
    "qsvd_prefill_attention_rope",
    "qsvd_latent_decode_attention",
    "qsvd_latent_decode_attention_rope",
    "qsvd_decode_workspace_size", "qsvd_latent_decode_attention_noalloc", "qsvd_noalloc_scratch_bytes",
    "qsvd_status_string", "qsvd_last_error", "qsvd_profile_enable", "qsvd_profile_reset",
    "qsvd_profile_read",
]


class QsvdLayer(ctypes.Structure):
    _fields_ = [
        ("d", ctypes.c_int32), ("r", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("w_bits", ctypes.c_int32),
        ("w_group", ctypes.c_int32), ("a_t", ctypes.c_void_p), ("s_a", ctypes.c_void_p),
        ("b_t", ctypes.c_void_p), ("s_b", ctypes.c_void_p),
    ]


class QsvdCache(ctypes.Structure):
    _fields_ = [
        ("fmt", ctypes.c_int32), ("batch", ctypes.c_int32), ("capacity", ctypes.c_int32),
        ("r", ctypes.c_int32), ("data", ctypes.c_void_p), ("scale", ctypes.c_void_p),
        ("seq_len", ctypes.c_void_p), ("max_len", ctypes.c_int32), ("overflow", ctypes.c_void_p),
    ]


class QsvdError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{status_string(status)} ({status}): {message}")
        self.status = status


_lib = None


def lib():
    """The loaded library; raises if it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2510_16292_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, U32, SZ, F = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                    ctypes.c_size_t, ctypes.c_float)
        LP, CP = ctypes.POINTER(QsvdLayer), ctypes.POINTER(QsvdCache)
        sig = {
            "qsvd_quantize_act": (I32, [P, I64, I32, I64, I32, F, P, P, P]),
            "qsvd_quantize_act_rotated": (I32, [P, I64, I32, I64, I32, F, P, I32, P, P, P]),
            "qsvd_lowrank_qkv_prefill": (I32, [LP, P, P, I64, I32, U32, P, P, P, P, P, P, P, P, P, SZ, P]),
            "qsvd_prefill_workspace_size": (SZ, [LP, I64, U32]),
            "qsvd_latent_cache_append": (I32, [CP, P, P, P, I32, P]),
            "qsvd_decode_project_append": (I32, [LP, CP, P, I64, I32, F, P, P, P, P, P, P, P]),
            "qsvd_prefill_attention": (I32, [P, P, P, I32, P, I32, I32, I32, I32, F, P, P]),
            "qsvd_prefill_attention_rope": (I32, [P, P, P, I32, P, I32, I32, I32, I32, F, F, P, P]),
            "qsvd_latent_decode_attention": (I32, [LP, CP, P, I32, I32, F, P, P, SZ, P]),
            "qsvd_latent_decode_attention_rope": (I32, [LP, CP, P, I32, I32, F, F, P, P, SZ, P]),
            "qsvd_decode_workspace_size": (SZ, [LP, CP, I32, I32]),
            "qsvd_latent_decode_attention_noalloc": (I32, [LP, CP, P, I32, I32, F, P, P]),
            "qsvd_noalloc_scratch_bytes": (SZ, []),
            "qsvd_status_string": (ctypes.c_char_p, [I32]),
            "qsvd_last_error": (ctypes.c_char_p, []),
            "qsvd_profile_enable": (I32, [I32, ctypes.c_char_p]),
            "qsvd_profile_reset": (I32, []),
            "qsvd_profile_read": (I32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64)]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


# ---------------------------------------------------------------- raw entry points

def qsvd_quantize_act(x, M, K, ldx, bits, clip, xq, sx, stream):
    return lib().qsvd_quantize_act(x, M, K, ldx, bits, clip, xq, sx, stream)


def qsvd_quantize_act_rotated(x, M, K, ldx, bits, clip, signs, block, xq, sx, stream):
    return lib().qsvd_quantize_act_rotated(x, M, K, ldx, bits, clip, signs, block, xq, sx, stream)


def qsvd_lowrank_qkv_prefill(layer, xq, sx, M, act_bits, out_mask, c_h, cq, sc, q, k, v,
                             dbg_acc_xa, dbg_acc_cb, ws, ws_bytes, stream):
    return lib().qsvd_lowrank_qkv_prefill(ctypes.byref(layer), xq, sx, M, act_bits, out_mask, c_h, cq, sc,
                                          q, k, v, dbg_acc_xa, dbg_acc_cb, ws, ws_bytes, stream)


def qsvd_prefill_workspace_size(layer, M, out_mask):
    return lib().qsvd_prefill_workspace_size(ctypes.byref(layer), M, out_mask)


def qsvd_latent_cache_append(cache, c_h, cq, sc, n_new, stream):
    return lib().qsvd_latent_cache_append(ctypes.byref(cache), c_h, cq, sc, n_new, stream)


def qsvd_decode_project_append(layer, cache, x, ldx, act_bits, clip, xq, sx, c_h, cq, sc, q, stream):
    return lib().qsvd_decode_project_append(ctypes.byref(layer), ctypes.byref(cache), x, ldx, act_bits, clip, xq, sx,
                                            c_h, cq, sc, q, stream)


def qsvd_prefill_attention(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads, head_dim, sm_scale, out,
                           stream):
    return lib().qsvd_prefill_attention(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads, head_dim,
                                        sm_scale, out, stream)


def qsvd_prefill_attention_rope(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads, head_dim, sm_scale,
                                rope_theta, out, stream):
    return lib().qsvd_prefill_attention_rope(q, k, v, batch, cu_seqlens, max_seqlen, n_q_heads, n_kv_heads,
                                             head_dim, sm_scale, rope_theta, out, stream)


def qsvd_latent_decode_attention(layer, cache, q, q_len, mode, sm_scale, out, ws, ws_bytes, stream):
    return lib().qsvd_latent_decode_attention(ctypes.byref(layer), ctypes.byref(cache), q, q_len, mode,
                                              sm_scale, out, ws, ws_bytes, stream)


def qsvd_latent_decode_attention_rope(layer, cache, q, q_len, mode, sm_scale, rope_theta, out, ws, ws_bytes,
                                      stream):
    return lib().qsvd_latent_decode_attention_rope(ctypes.byref(layer), ctypes.byref(cache), q, q_len, mode,
                                                   sm_scale, rope_theta, out, ws, ws_bytes, stream)


def qsvd_latent_decode_attention_noalloc(layer, cache, q, q_len, mode, sm_scale, out, stream):
    return lib().qsvd_latent_decode_attention_noalloc(ctypes.byref(layer), ctypes.byref(cache), q, q_len, mode,
                                                      sm_scale, out, stream)


def qsvd_noalloc_scratch_bytes():
    return lib().qsvd_noalloc_scratch_bytes()


def qsvd_decode_workspace_size(layer, cache, q_len, mode):
    return lib().qsvd_decode_workspace_size(ctypes.byref(layer), ctypes.byref(cache), q_len, mode)


def status_string(status):
    return lib().qsvd_status_string(status).decode()


def last_error():
    return lib().qsvd_last_error().decode()


def profile_enable(on, filter=None):
    return lib().qsvd_profile_enable(1 if on else 0, None if filter is None else filter.encode())


def profile_reset():
    return lib().qsvd_profile_reset()


def profile_read(name):
    ms, n = ctypes.c_double(), ctypes.c_int64()
    check(lib().qsvd_profile_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def check(status):
    if status != QSVD_OK:
        raise QsvdError(status, last_error())
    return status


# ---------------------------------------------------------------- torch-backed helpers

def ptr(t):
    return 0 if t is None else t.data_ptr()


def stream_handle(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


class DeviceLayer:
    """A prepared layer uploaded to the device; ``.c`` is the qsvd_layer struct."""

    def __init__(self, host, device="cuda"):
        import torch
        self.d, self.r = host.d, host.r
        self.n_q_heads, self.n_kv_heads, self.head_dim = host.n_q_heads, host.n_kv_heads, host.head_dim
        self.w_bits, self.w_group = host.w_bits, host.w_group
        self.a_t = torch.from_numpy(host.a_t).to(device)
        self.s_a = torch.from_numpy(host.s_a).to(device)
        self.b_t = torch.from_numpy(host.b_t).to(device)
        self.s_b = torch.from_numpy(host.s_b).to(device)
        self.c = QsvdLayer(self.d, self.r, self.n_q_heads, self.n_kv_heads, self.head_dim, self.w_bits,
                           self.w_group, ptr(self.a_t), ptr(self.s_a), ptr(self.b_t), ptr(self.s_b))

    @classmethod
    def from_device(cls, d, r, n_q_heads, n_kv_heads, head_dim, w_bits, w_group, a_t, s_a, b_t, s_b):
        """Wrap weight codes and scales already in device memory (same layouts
        as a prepared layer: a_t [r][d], s_a, b_t [N][r], s_b)."""
        self = cls.__new__(cls)
        self.d, self.r = d, r
        self.n_q_heads, self.n_kv_heads, self.head_dim = n_q_heads, n_kv_heads, head_dim
        self.w_bits, self.w_group = w_bits, w_group
        self.a_t, self.s_a, self.b_t, self.s_b = a_t, s_a, b_t, s_b
        self.c = QsvdLayer(d, r, n_q_heads, n_kv_heads, head_dim, w_bits, w_group, ptr(a_t), ptr(s_a), ptr(b_t),
                           ptr(s_b))
        return self

    @property
    def N(self):
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


class DeviceCache:
    """A latent cache in device memory; ``.c`` is the qsvd_cache struct.

    ``lengths`` initialises every seq_len[b] (ragged batches allowed); max_len
    is their maximum.  ``overflow`` is the device flag an append sets when it
    would run past capacity on the device."""

    def __init__(self, fmt, batch, capacity, r, lengths=None, device="cuda"):
        import torch
        self.fmt, self.batch, self.capacity, self.r = fmt, batch, capacity, r
        width = r if fmt != QSVD_CACHE_I4 else r // 2
        dtype = torch.float16 if fmt == QSVD_CACHE_F16 else (torch.int8 if fmt == QSVD_CACHE_I8 else torch.uint8)
        self.data = torch.zeros((batch, capacity, width), dtype=dtype, device=device)
        self.scale = None if fmt == QSVD_CACHE_F16 else torch.zeros((batch, capacity), dtype=torch.float32,
                                                                   device=device)
        lengths = [0] * batch if lengths is None else list(lengths)
        self.seq_len = torch.tensor(lengths, dtype=torch.int32, device=device)
        self.overflow = torch.zeros((1,), dtype=torch.int32, device=device)
        self.c = QsvdCache(fmt, batch, capacity, r, ptr(self.data), ptr(self.scale), ptr(self.seq_len),
                           max(lengths) if lengths else 0, ptr(self.overflow))

    @property
    def max_len(self):
        return self.c.max_len

    def snapshot(self):
        """Host copy of the cache state (rows, scales, lengths, host bound) from
        which a decode resumes; taken after the work queued on the current
        stream."""
        return dict(data=self.data.cpu(), scale=None if self.scale is None else self.scale.cpu(),
                    seq_len=self.seq_len.cpu(), max_len=int(self.c.max_len))

    def restore(self, snap):
        """Put a snapshot back (same format and shape), ordered on the current stream."""
        assert tuple(snap["data"].shape) == tuple(self.data.shape) and snap["data"].dtype == self.data.dtype
        self.data.copy_(snap["data"])
        if self.scale is not None:
            self.scale.copy_(snap["scale"])
        self.seq_len.copy_(snap["seq_len"])
        self.c.max_len = snap["max_len"]


def projection_evaluator(n_q_heads, n_kv_heads, head_dim, w_bits=8, w_group=0, a_bits=8):
    """A callable (A, B, X) -> the fp16 Q | K | V of the quantized projection of
    X through the layer built from W^d = A and W^u = B on the GPU (weights
    quantized by the offline stage, activations and latent by the library),
    for offline searches such as the beta search of ``prep.search_beta``."""
    import numpy as np
    import torch

    from . import prep

    def project(A, B, X):
        layer = DeviceLayer(prep.quantize_layer(A, B, n_q_heads, n_kv_heads, head_dim, w_bits, w_group))
        M, d = X.shape
        r, N = layer.r, layer.N
        per = 1 if a_bits == 8 else 2
        x = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float16)).cuda()
        xq = torch.empty((M, d // per), dtype=torch.uint8, device="cuda")
        sx = torch.empty((M,), dtype=torch.float32, device="cuda")
        c_h = torch.empty((M, r), dtype=torch.float16, device="cuda")
        cq = torch.empty((M, r // per), dtype=torch.uint8, device="cuda")
        sc = torch.empty((M,), dtype=torch.float32, device="cuda")
        nq, nkv = n_q_heads * head_dim, n_kv_heads * head_dim
        q = torch.empty((M, nq), dtype=torch.float16, device="cuda")
        k = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
        v = torch.empty((M, nkv), dtype=torch.float16, device="cuda")
        s = stream_handle()
        check(qsvd_quantize_act(ptr(x), M, d, d, a_bits, 1.0, ptr(xq), ptr(sx), s))
        check(qsvd_lowrank_qkv_prefill(layer.c, ptr(xq), ptr(sx), M, a_bits, 7, ptr(c_h), ptr(cq), ptr(sc),
                                       ptr(q), ptr(k), ptr(v), 0, 0, 0, 0, s))
        out = torch.cat([q, k, v], dim=1).cpu().numpy()
        del layer
        return out

    return project
