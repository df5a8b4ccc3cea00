"""The C ABI on the CPU: the library loads, exports what include/qsvd.h
declares, the ctypes structs match the C layout, and argument validation
returns the documented status before any GPU work (no GPU needed)."""
import ctypes
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

from paper_2510_16292_amd import binding as B
from paper_2510_16292_amd import prep
from workloads import configs, gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qsvd.h")

FAKE = 0x100000          # 16-byte-aligned non-NULL address that is never dereferenced on the host


@pytest.fixture(scope="module")
def lib():
    return B.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(qsvd_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_four_hot_path_calls():
    names = declared_functions()
    for n in ("qsvd_quantize_act", "qsvd_lowrank_qkv_prefill", "qsvd_latent_cache_append",
              "qsvd_latent_decode_attention"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", B.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\s[TW]\s+(qsvd_\w+)", out))
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    assert sorted(exported) == sorted(set(B.EXPORTED))


def test_struct_layout_matches_header():
    src = r"""
#include <stddef.h>
#include <stdio.h>
#include "qsvd.h"
#define F(T, f) printf(#T "." #f " %zu %zu\n", offsetof(T, f), sizeof(((T*)0)->f));
int main(void) {
  F(qsvd_layer, d) F(qsvd_layer, r) F(qsvd_layer, n_q_heads) F(qsvd_layer, n_kv_heads)
  F(qsvd_layer, head_dim) F(qsvd_layer, w_bits) F(qsvd_layer, w_group) F(qsvd_layer, a_t)
  F(qsvd_layer, s_a) F(qsvd_layer, b_t) F(qsvd_layer, s_b)
  F(qsvd_cache, fmt) F(qsvd_cache, batch) F(qsvd_cache, capacity) F(qsvd_cache, r)
  F(qsvd_cache, data) F(qsvd_cache, scale) F(qsvd_cache, seq_len) F(qsvd_cache, max_len)
  F(qsvd_cache, overflow)
  printf("sizeof.qsvd_layer %zu 0\nsizeof.qsvd_cache %zu 0\n", sizeof(qsvd_layer), sizeof(qsvd_cache));
  return 0;
}
"""
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "layout.c")
        exe = os.path.join(d, "layout")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), c, "-o", exe], check=True)
        lines = subprocess.run([exe], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {}
    for ln in lines:
        if ln.strip():
            k, off, size = ln.split()
            got[k] = (int(off), int(size))
    for cls, cname in ((B.QsvdLayer, "qsvd_layer"), (B.QsvdCache, "qsvd_cache")):
        for fname, ftype in cls._fields_:
            desc = getattr(cls, fname)
            assert got[f"{cname}.{fname}"] == (desc.offset, desc.size), (cname, fname)
        assert got[f"sizeof.{cname}"][0] == ctypes.sizeof(cls)


def layer_struct(**over):
    kw = dict(d=256, r=128, n_q_heads=4, n_kv_heads=4, head_dim=64, w_bits=8, w_group=0,
              a_t=FAKE, s_a=FAKE, b_t=FAKE, s_b=FAKE)
    kw.update(over)
    return B.QsvdLayer(**kw)


def cache_struct(**over):
    kw = dict(fmt=B.QSVD_CACHE_F16, batch=2, capacity=64, r=128, data=FAKE, scale=0, seq_len=FAKE, max_len=10)
    kw.update(over)
    return B.QsvdCache(**kw)


def test_status_strings(lib):
    assert B.status_string(B.QSVD_OK) == "ok"
    assert B.status_string(B.QSVD_ERR_CAPACITY) == "cache capacity exceeded"
    assert B.status_string(99) == "unknown status"


@pytest.mark.parametrize("args,status", [
    ((0, 4, 16, 16, 8, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),            # NULL x
    ((FAKE, 4, 16, 16, 3, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),         # bits
    ((FAKE, 4, 16, 16, 8, 0.0, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),         # clip
    ((FAKE, 4, 16, 16, 8, 1.5, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),         # clip
    ((FAKE, -1, 16, 16, 8, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),        # M < 0
    ((FAKE, 4, 16, 8, 8, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),          # ldx < K
    ((FAKE, 4, 12, 16, 8, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_UNSUPPORTED),         # K % 8
    ((FAKE + 2, 4, 16, 16, 8, 1.0, FAKE, FAKE, 0), B.QSVD_ERR_UNSUPPORTED),     # misaligned x
])
def test_quantize_act_validation(lib, args, status):
    assert B.qsvd_quantize_act(*args) == status


@pytest.mark.parametrize("args,status", [
    ((0, 4, 16, 16, 8, 1.0, 0, 16, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),        # NULL x
    ((FAKE, 4, 16, 16, 3, 1.0, 0, 16, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),     # bits
    ((FAKE, 4, 16, 16, 8, 0.0, 0, 16, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),     # clip
    ((FAKE, 4, 48, 48, 8, 1.0, 0, 32, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),     # block does not divide K
    ((FAKE, 4, 48, 48, 8, 1.0, 0, 24, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),     # block not a power of two
    ((FAKE, 4, 16, 16, 8, 1.0, 0, 4, FAKE, FAKE, 0), B.QSVD_ERR_INVALID_ARG),      # block < 8
    ((FAKE, 4, 32768, 32768, 8, 1.0, 0, 8, FAKE, FAKE, 0), B.QSVD_ERR_UNSUPPORTED),  # K too large
    ((FAKE, 4, 16, 16, 8, 1.0, FAKE + 4, 16, FAKE, FAKE, 0), B.QSVD_ERR_UNSUPPORTED),  # misaligned signs
    ((FAKE, 0, 16, 16, 8, 1.0, 0, 16, FAKE, FAKE, 0), B.QSVD_OK),                  # nothing to do
])
def test_quantize_act_rotated_validation(lib, args, status):
    assert B.qsvd_quantize_act_rotated(*args) == status
    assert B.last_error()


def _prefill(layer, M=16, act_bits=8, mask=7, ws=FAKE, ws_bytes=1 << 30, **ptrs):
    p = dict(xq=FAKE, sx=FAKE, c_h=FAKE, cq=FAKE, sc=FAKE, q=FAKE, k=FAKE, v=FAKE)
    p.update(ptrs)
    return B.qsvd_lowrank_qkv_prefill(layer, p["xq"], p["sx"], M, act_bits, mask, p["c_h"], p["cq"], p["sc"],
                                      p["q"], p["k"], p["v"], 0, 0, ws, ws_bytes, 0)


def test_prefill_validation(lib):
    assert B.lib().qsvd_lowrank_qkv_prefill(None, FAKE, FAKE, 4, 8, 7, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                            0, 0, FAKE, 1, 0) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(d=0)) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(n_q_heads=6, n_kv_heads=4)) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(a_t=0)) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(w_bits=6)) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(w_bits=4, w_group=0)) == B.QSVD_ERR_UNSUPPORTED
    assert _prefill(layer_struct(w_group=48)) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(d=200)) == B.QSVD_ERR_UNSUPPORTED
    assert _prefill(layer_struct(), M=-1) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(), mask=8) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(), act_bits=5) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(), mask=B.QSVD_OUT_K, k=0) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(), c_h=0) == B.QSVD_ERR_INVALID_ARG
    assert _prefill(layer_struct(), M=0) == B.QSVD_OK          # nothing to do, nothing launched
    assert B.lib().qsvd_lowrank_qkv_prefill(ctypes.byref(layer_struct()), FAKE, FAKE, 4, 4, 7, FAKE, FAKE, FAKE, FAKE,
                                            FAKE, FAKE, FAKE, 0, 0, 0, 0) == B.QSVD_ERR_UNSUPPORTED  # dumps: A8
    assert _prefill(layer_struct(w_bits=4, w_group=32)) == B.QSVD_ERR_UNSUPPORTED        # groups of 64 codes
    assert _prefill(layer_struct(w_bits=4, w_group=32), M=33) == B.QSVD_ERR_UNSUPPORTED
    assert _prefill(layer_struct(d=384, w_bits=4, w_group=192), M=33) == B.QSVD_ERR_INVALID_ARG  # 192 does not divide r
    g = layer_struct(w_bits=4, w_group=64)
    assert B.lib().qsvd_lowrank_qkv_prefill(ctypes.byref(g), FAKE, FAKE, 4, 8, 7, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                            FAKE, 0, 0, 0, 0) == B.QSVD_ERR_UNSUPPORTED   # no dumps with groups


def test_cache_append_validation(lib):
    c = cache_struct(max_len=60)
    assert B.qsvd_latent_cache_append(c, FAKE, 0, 0, 5, 0) == B.QSVD_ERR_CAPACITY
    assert c.max_len == 60
    assert B.qsvd_latent_cache_append(c, FAKE, 0, 0, 0, 0) == B.QSVD_OK
    assert B.qsvd_latent_cache_append(c, FAKE, 0, 0, -1, 0) == B.QSVD_ERR_INVALID_ARG
    assert B.qsvd_latent_cache_append(c, 0, 0, 0, 1, 0) == B.QSVD_ERR_INVALID_ARG
    ci = cache_struct(fmt=B.QSVD_CACHE_I8, scale=FAKE)
    assert B.qsvd_latent_cache_append(ci, FAKE, 0, FAKE, 1, 0) == B.QSVD_ERR_INVALID_ARG   # needs cq
    assert B.qsvd_latent_cache_append(cache_struct(fmt=B.QSVD_CACHE_I8), 0, FAKE, FAKE, 1, 0) == B.QSVD_ERR_INVALID_ARG
    assert B.qsvd_latent_cache_append(cache_struct(fmt=7), FAKE, 0, 0, 1, 0) == B.QSVD_ERR_INVALID_ARG
    assert B.qsvd_latent_cache_append(cache_struct(r=48), FAKE, 0, 0, 1, 0) == B.QSVD_ERR_UNSUPPORTED
    assert B.qsvd_latent_cache_append(cache_struct(max_len=65), FAKE, 0, 0, 1, 0) == B.QSVD_ERR_INVALID_ARG
    assert B.qsvd_latent_cache_append(cache_struct(seq_len=0), FAKE, 0, 0, 1, 0) == B.QSVD_ERR_INVALID_ARG


def test_decode_project_append_validation(lib):
    """Every case fails before a launch; the capacity error leaves max_len alone."""
    def call(layer=None, cache=None, ldx=256, bits=8, clip=1.0, ptrs=None):
        p = ptrs or [FAKE] * 6
        return B.qsvd_decode_project_append(layer or layer_struct(), cache or cache_struct(), FAKE, ldx, bits, clip,
                                            *p, 0)
    assert call(bits=5) == B.QSVD_ERR_INVALID_ARG
    assert call(clip=0.0) == B.QSVD_ERR_INVALID_ARG
    assert call(ldx=128) == B.QSVD_ERR_INVALID_ARG
    assert call(ptrs=[FAKE, FAKE, 0, FAKE, FAKE, FAKE]) == B.QSVD_ERR_INVALID_ARG
    assert call(cache=cache_struct(r=256)) == B.QSVD_ERR_INVALID_ARG
    assert call(cache=cache_struct(fmt=B.QSVD_CACHE_I8, scale=FAKE), bits=4) == B.QSVD_ERR_UNSUPPORTED
    assert call(cache=cache_struct(fmt=B.QSVD_CACHE_I4, scale=FAKE), bits=8) == B.QSVD_ERR_UNSUPPORTED
    full = cache_struct(max_len=64)
    assert call(cache=full) == B.QSVD_ERR_CAPACITY
    assert full.max_len == 64
    assert call(cache=cache_struct(batch=33)) == B.QSVD_ERR_UNSUPPORTED
    assert call(ldx=260) == B.QSVD_ERR_UNSUPPORTED


def test_prefill_attention_validation(lib):
    """Every case fails (or returns OK with nothing to do) before a launch."""
    def call(q=FAKE, k=FAKE, v=FAKE, batch=2, cu=FAKE, ms=64, hq=4, hkv=2, dh=64, sm=0.0, out=FAKE):
        return B.qsvd_prefill_attention(q, k, v, batch, cu, ms, hq, hkv, dh, sm, out, 0)
    assert call(batch=-1) == B.QSVD_ERR_INVALID_ARG
    assert call(ms=-1) == B.QSVD_ERR_INVALID_ARG
    assert call(hq=0) == B.QSVD_ERR_INVALID_ARG
    assert call(hq=6, hkv=4) == B.QSVD_ERR_INVALID_ARG
    assert call(sm=-1.0) == B.QSVD_ERR_INVALID_ARG
    assert call(sm=float("inf")) == B.QSVD_ERR_INVALID_ARG
    assert call(batch=0) == B.QSVD_OK
    assert call(ms=0) == B.QSVD_OK
    assert call(q=0) == B.QSVD_ERR_INVALID_ARG
    assert call(cu=0) == B.QSVD_ERR_INVALID_ARG
    assert call(dh=96) == B.QSVD_ERR_UNSUPPORTED
    assert call(dh=32) == B.QSVD_ERR_UNSUPPORTED
    assert call(out=FAKE + 8) == B.QSVD_ERR_UNSUPPORTED


def test_prefill_attention_rope_validation(lib):
    """The rotary prefill entry validates like the plain one, and refuses a
    rotary base that is not finite and > 1, all before any GPU work."""
    def call(q=FAKE, batch=2, ms=64, hq=4, hkv=2, dh=64, sm=0.0, theta=10000.0, out=FAKE):
        return B.qsvd_prefill_attention_rope(q, FAKE, FAKE, batch, FAKE, ms, hq, hkv, dh, sm, theta, out, 0)
    for theta in (0.0, 1.0, -5.0, float("inf"), float("nan")):
        assert call(theta=theta) == B.QSVD_ERR_INVALID_ARG, theta
        assert "rope_theta" in B.last_error()
    assert call(batch=-1) == B.QSVD_ERR_INVALID_ARG
    assert call(hq=6, hkv=4) == B.QSVD_ERR_INVALID_ARG
    assert call(sm=float("inf")) == B.QSVD_ERR_INVALID_ARG
    assert call(batch=0) == B.QSVD_OK
    assert call(ms=0) == B.QSVD_OK
    assert call(q=0) == B.QSVD_ERR_INVALID_ARG
    assert call(dh=96) == B.QSVD_ERR_UNSUPPORTED
    assert call(out=FAKE + 8) == B.QSVD_ERR_UNSUPPORTED


def test_noalloc_decode_validation(lib):
    """The allocation-free decode attention validates like the workspace entry
    point and refuses a call whose scratch need exceeds the static array, all
    before any GPU work."""
    assert B.qsvd_noalloc_scratch_bytes() == 32 << 20
    L, C = layer_struct(), cache_struct()
    call = lambda layer, cache, q_len=1, mode=0: B.qsvd_latent_decode_attention_noalloc(layer, cache, FAKE, q_len,
                                                                                      mode, 0.0, FAKE, 0)
    assert call(L, C, q_len=0) == B.QSVD_ERR_INVALID_ARG
    assert call(L, C, mode=3) == B.QSVD_ERR_INVALID_ARG
    assert call(L, cache_struct(r=256)) == B.QSVD_ERR_INVALID_ARG
    wide = layer_struct(d=5120, r=3072, n_q_heads=40, n_kv_heads=40, head_dim=128)
    big = cache_struct(batch=64, capacity=4096, r=3072, max_len=4096)
    assert B.qsvd_decode_workspace_size(wide, big, 1, B.QSVD_ATTN_AUTO) > B.qsvd_noalloc_scratch_bytes()
    assert call(wide, big) == B.QSVD_ERR_WORKSPACE
    assert "static" in B.last_error()


def _decode(layer, cache, q_len=1, mode=0, sm=0.0, ws=FAKE, ws_bytes=1 << 40, q=FAKE, out=FAKE):
    return B.qsvd_latent_decode_attention(layer, cache, q, q_len, mode, sm, out, ws, ws_bytes, 0)


def test_decode_validation(lib):
    L, C = layer_struct(), cache_struct()
    assert _decode(L, C, q_len=0) == B.QSVD_ERR_INVALID_ARG
    assert _decode(L, C, q_len=11) == B.QSVD_ERR_INVALID_ARG                  # more queries than cached tokens
    # the reconstruct form with q_len > 1 (the cache-mode flash kernel) needs head_dim 64 or 128
    need_q2 = B.qsvd_decode_workspace_size(L, C, 2, B.QSVD_ATTN_RECONSTRUCT)
    assert need_q2 == B.qsvd_decode_workspace_size(L, C, 1, B.QSVD_ATTN_RECONSTRUCT) > 0
    assert _decode(L, C, q_len=2, mode=B.QSVD_ATTN_RECONSTRUCT, ws_bytes=need_q2 - 1) == B.QSVD_ERR_WORKSPACE
    assert _decode(layer_struct(head_dim=32, n_q_heads=8, n_kv_heads=8), C, q_len=2,
                   mode=B.QSVD_ATTN_RECONSTRUCT) == B.QSVD_ERR_UNSUPPORTED
    assert B.qsvd_decode_workspace_size(layer_struct(head_dim=32, n_q_heads=8, n_kv_heads=8), C, 2,
                                        B.QSVD_ATTN_RECONSTRUCT) == 0
    assert _decode(L, cache_struct(batch=64, max_len=2000, capacity=4096), q_len=1025) == B.QSVD_ERR_UNSUPPORTED
    assert _decode(L, C, mode=3) == B.QSVD_ERR_INVALID_ARG
    assert _decode(L, C, sm=-1.0) == B.QSVD_ERR_INVALID_ARG
    assert _decode(L, C, q=0) == B.QSVD_ERR_INVALID_ARG
    assert _decode(L, cache_struct(r=256)) == B.QSVD_ERR_INVALID_ARG
    assert _decode(L, cache_struct(max_len=0)) == B.QSVD_ERR_INVALID_ARG
    assert _decode(layer_struct(n_q_heads=80, n_kv_heads=8, head_dim=64), C) == B.QSVD_ERR_UNSUPPORTED
    # more than 32 query heads: absorbed form with 16-head blocks (r a multiple
    # of 128), or the reconstruct form with its partials in two 32-head blocks
    wide = layer_struct(n_q_heads=40, n_kv_heads=8, head_dim=64)
    need_w = B.qsvd_decode_workspace_size(wide, C, 1, B.QSVD_ATTN_RECONSTRUCT)
    assert need_w > 0
    assert _decode(wide, C, mode=B.QSVD_ATTN_RECONSTRUCT, ws_bytes=need_w - 1) == B.QSVD_ERR_WORKSPACE
    # r 192 has no absorbed plan at 40 heads: AUTO takes the reconstruct form
    w192, c192 = layer_struct(n_q_heads=40, n_kv_heads=8, head_dim=64, r=192), cache_struct(r=192)
    assert _decode(w192, c192, mode=B.QSVD_ATTN_ABSORBED) == B.QSVD_ERR_UNSUPPORTED
    need192 = B.qsvd_decode_workspace_size(w192, c192, 1, B.QSVD_ATTN_AUTO)
    assert need192 == B.qsvd_decode_workspace_size(w192, c192, 1, B.QSVD_ATTN_RECONSTRUCT) > 0
    assert _decode(w192, c192, ws_bytes=need192 - 1) == B.QSVD_ERR_WORKSPACE
    assert _decode(layer_struct(r=3200), cache_struct(r=3200), mode=B.QSVD_ATTN_ABSORBED) == B.QSVD_ERR_UNSUPPORTED
    # three head blocks x 64 sequences x 400 queries exceed the grid's rows
    big = cache_struct(batch=64, max_len=2000, capacity=4096)
    assert _decode(wide, big, q_len=400) == B.QSVD_ERR_UNSUPPORTED
    assert B.qsvd_decode_workspace_size(wide, big, 400, B.QSVD_ATTN_ABSORBED) == 0
    assert B.qsvd_decode_workspace_size(wide, big, 300, B.QSVD_ATTN_ABSORBED) > 0
    assert _decode(wide, C, mode=B.QSVD_ATTN_ABSORBED, ws_bytes=B.qsvd_decode_workspace_size(wide, C, 1, 1) - 1) \
        == B.QSVD_ERR_WORKSPACE
    assert _decode(layer_struct(head_dim=48, n_q_heads=4), C) == B.QSVD_ERR_UNSUPPORTED
    assert _decode(L, cache_struct(batch=65)) == B.QSVD_ERR_UNSUPPORTED
    c4 = cache_struct(fmt=B.QSVD_CACHE_I4, scale=FAKE)       # int4 caches rebuild on the 4-bit products
    need4 = B.qsvd_decode_workspace_size(L, c4, 1, B.QSVD_ATTN_RECONSTRUCT)
    assert need4 > 0
    assert _decode(L, c4, mode=B.QSVD_ATTN_RECONSTRUCT, ws_bytes=need4 - 1) == B.QSVD_ERR_WORKSPACE
    assert _decode(layer_struct(r=192), cache_struct(r=192), mode=B.QSVD_ATTN_ABSORBED) == B.QSVD_ERR_UNSUPPORTED
    need = B.qsvd_decode_workspace_size(L, C, 1, B.QSVD_ATTN_ABSORBED)
    assert need > 0
    assert _decode(L, C, mode=B.QSVD_ATTN_ABSORBED, ws_bytes=need - 1) == B.QSVD_ERR_WORKSPACE
    need_r = B.qsvd_decode_workspace_size(L, C, 1, B.QSVD_ATTN_RECONSTRUCT)
    assert _decode(L, C, mode=B.QSVD_ATTN_RECONSTRUCT, ws_bytes=need_r - 1) == B.QSVD_ERR_WORKSPACE
    assert B.qsvd_decode_workspace_size(L, C, 0, 0) == 0
    # q_len > 1 (absorbed): one query row block per (sequence, query)
    need2 = B.qsvd_decode_workspace_size(L, C, 2, B.QSVD_ATTN_ABSORBED)
    assert need2 >= need
    assert _decode(L, C, q_len=2, mode=B.QSVD_ATTN_ABSORBED, ws_bytes=need2 - 1) == B.QSVD_ERR_WORKSPACE


def _decode_rope(layer, cache, theta=10000.0, q_len=1, mode=0, ws_bytes=1 << 40):
    return B.qsvd_latent_decode_attention_rope(layer, cache, FAKE, q_len, mode, 0.0, theta, FAKE, FAKE, ws_bytes, 0)


def test_decode_rope_validation(lib):
    """Every case fails before a launch.  Rotary layers run the form with the
    value side in latent space (ABSORBED, or AUTO where its 32-head plans
    apply; q_len 1) or the full rebuild (RECONSTRUCT; any q_len, head_dim 64
    or 128 above 1), with a base above 1; one workspace size (the
    reconstruct query) serves both."""
    L, C = layer_struct(), cache_struct()
    for theta in (0.0, -5.0, 1.0, float("inf"), float("nan")):
        assert _decode_rope(L, C, theta=theta) == B.QSVD_ERR_INVALID_ARG
    # latent-value form: 32-head plans only
    assert _decode_rope(layer_struct(r=192), cache_struct(r=192), mode=B.QSVD_ATTN_ABSORBED) == \
        B.QSVD_ERR_UNSUPPORTED
    wide = layer_struct(n_q_heads=40, n_kv_heads=8, head_dim=64)
    assert _decode_rope(wide, C, mode=B.QSVD_ATTN_ABSORBED) == B.QSVD_ERR_UNSUPPORTED
    need_w = B.qsvd_decode_workspace_size(wide, C, 1, B.QSVD_ATTN_RECONSTRUCT)
    assert _decode_rope(wide, C, ws_bytes=need_w - 1) == B.QSVD_ERR_WORKSPACE   # AUTO -> full rebuild, 40 heads
    assert _decode_rope(layer_struct(n_q_heads=80, n_kv_heads=8, head_dim=64), C) == B.QSVD_ERR_UNSUPPORTED
    for mode in (B.QSVD_ATTN_AUTO, B.QSVD_ATTN_ABSORBED, B.QSVD_ATTN_RECONSTRUCT):
        if mode == B.QSVD_ATTN_ABSORBED:          # the latent-value form: one query per sequence
            assert _decode_rope(L, C, q_len=2, mode=mode) == B.QSVD_ERR_UNSUPPORTED
        else:                                     # AUTO and RECONSTRUCT rebuild K and V for q_len > 1
            need2 = B.qsvd_decode_workspace_size(L, C, 2, B.QSVD_ATTN_RECONSTRUCT)
            assert _decode_rope(L, C, q_len=2, mode=mode, ws_bytes=need2 - 1) == B.QSVD_ERR_WORKSPACE
    assert _decode_rope(L, cache_struct(capacity=20000), mode=B.QSVD_ATTN_RECONSTRUCT) == B.QSVD_ERR_UNSUPPORTED
    assert _decode_rope(L, C, mode=3) == B.QSVD_ERR_INVALID_ARG
    for c in (C, cache_struct(fmt=B.QSVD_CACHE_I8, scale=FAKE), cache_struct(fmt=B.QSVD_CACHE_I4, scale=FAKE)):
        need = B.qsvd_decode_workspace_size(L, c, 1, B.QSVD_ATTN_RECONSTRUCT)
        assert need > 0
        for mode in (B.QSVD_ATTN_AUTO, B.QSVD_ATTN_ABSORBED, B.QSVD_ATTN_RECONSTRUCT):
            assert _decode_rope(L, c, mode=mode, ws_bytes=need - 1) == B.QSVD_ERR_WORKSPACE


def test_decode_workspace_sizes_cover_growth(lib):
    """The absorbed workspace depends on batch and rank, not on the current
    length, so one allocation serves every decode step up to capacity."""
    L = layer_struct(d=4096, r=1536, n_q_heads=32, n_kv_heads=32, head_dim=128)
    sizes = {B.qsvd_decode_workspace_size(L, cache_struct(batch=16, capacity=4352, r=1536, max_len=m), 1, 1)
             for m in (1, 100, 4096, 4352)}
    assert len(sizes) == 1
    a = B.qsvd_decode_workspace_size(L, cache_struct(batch=8, capacity=4352, r=1536, max_len=9), 1, 1)
    b = B.qsvd_decode_workspace_size(L, cache_struct(batch=16, capacity=4352, r=1536, max_len=9), 1, 1)
    assert b >= a


def test_profiler_off_by_default(lib):
    assert B.profile_read("latent_attn") == (0.0, 0)


def test_prep_matches_oracle_prep():
    """The product's offline stage produces the oracle's quantized weights bit for bit."""
    from oracle import qsvd_oracle as O
    wl = configs.get(1)
    L = wl.layer
    W = gen.weight_matrix(wl)
    A, Bm = O.factors_from_weight(W, L.r, wl.beta)
    for w_bits, w_group in ((8, 0), (4, 32), (4, 128)):
        P = prep.prepare_from_weight(W, L.r, L.n_q_heads, L.n_kv_heads, L.head_dim, wl.beta, w_bits, w_group)
        ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, w_bits, w_group)
        at = ol.Aq.T if w_bits == 8 else O.pack_int4(ol.Aq.T)
        bt = ol.Bq.T if w_bits == 8 else O.pack_int4(ol.Bq.T)
        assert np.array_equal(P.a_t.view(np.uint8), np.ascontiguousarray(at).view(np.uint8))
        assert np.array_equal(P.b_t.view(np.uint8), np.ascontiguousarray(bt).view(np.uint8))
        assert np.array_equal(P.s_a, ol.sA) and np.array_equal(P.s_b, ol.sB)
    # decaying-spectrum workload: factors known by construction
    wl4 = configs.Workload(91, "small_decay", configs.LayerShape(128, 4, 2, 32, 64), "decay", 4, 64, 8,
                           configs.CACHE_I8)
    U, s, V = gen.weight_factors(wl4)
    P = prep.prepare_from_svd(U, s, V, 4, 2, 32, 0.5, 4, 64)
    A4, B4 = O.split_beta(U, s, V.T, 0.5)
    ol = O.make_layer(A4, B4, 4, 2, 32, 4, 64)
    assert np.array_equal(P.a_t, O.pack_int4(np.ascontiguousarray(ol.Aq.T)))
    assert np.array_equal(P.b_t, O.pack_int4(np.ascontiguousarray(ol.Bq.T)))


@pytest.mark.parametrize("shape", [(256, 128, 4, 4, 64), (4096, 1536, 32, 32, 128), (3584, 1024, 28, 4, 128),
                                   (5120, 2048, 40, 40, 128)], ids=["tiny", "llava7b", "qwen2vl", "13b"])
def test_projection_needs_no_workspace(lib, shape):
    """The projection keeps every partial sum on chip (decode sizes reduce in
    LDS, prefill tiles accumulate in registers), so its workspace query is 0 for
    every size and output selection.  (An earlier split-contraction design wrote
    int32 partials to a workspace and once overflowed it on a Q-only call.)"""
    d, r, hq, hkv, dh = shape
    L = layer_struct(d=d, r=r, n_q_heads=hq, n_kv_heads=hkv, head_dim=dh)
    for M in (1, 8, 16, 31, 32, 33, 640, 2560):
        for mask in range(8):
            assert B.qsvd_prefill_workspace_size(L, M, mask) == 0


def test_prep_fold_input_rotation_matches_oracle_matrix():
    """The offline fold H1 W^d (fast transform, fp64) equals the oracle's explicit
    H1 times W^d."""
    from oracle import qsvd_oracle as O
    g = np.random.default_rng(5)
    for d in (256, 640):
        B = O.hadamard_block(d)
        s = O.rotation_signs(d, seed=d + 1)
        A = g.standard_normal((d, 48))
        assert np.allclose(prep.fold_input_rotation(A, s, B), O.rotation_matrix(s, B) @ A, rtol=0, atol=1e-12)
