"""HIP path against the oracle, element by element, through the C ABI.

Bit-exact: activation and latent codes and scales, the int32 accumulators,
the fp16 latent C and the fp16 Q/K/V (the epilogues follow the oracle's
rounding order), and every cache byte.  Toleranced: attention outputs,
max-abs 2e-2 and relative L2 1e-2 against the fp64 plain definition.
"""
import numpy as np
import pytest

import gpu_harness as H
from oracle import qsvd_oracle as O
from paper_2510_16292_amd import binding as B
from paper_2510_16292_amd import prep
from workloads import configs, gen

pytestmark = pytest.mark.gpu

MODES = [B.QSVD_ATTN_ABSORBED, B.QSVD_ATTN_RECONSTRUCT]
MODE_IDS = ["absorbed", "reconstruct"]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    B.lib()   # fails loudly if the HIP library is not built


# ------------------------------------------------------------------ layers

def _layers_from_weight(W, L, beta=0.5, w_bits=8, w_group=0):
    A, Bm = O.factors_from_weight(W, L.r, beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, w_bits, w_group)
    pl = prep.prepare_from_weight(W, L.r, L.n_q_heads, L.n_kv_heads, L.head_dim, beta, w_bits, w_group)
    return ol, B.DeviceLayer(pl)


@pytest.fixture(scope="module")
def tiny():
    wl = configs.get(1)
    ol, dl = _layers_from_weight(gen.weight_matrix(wl), wl.layer)
    return wl, ol, dl


@pytest.fixture(scope="module")
def gqa():
    """A small grouped-query layer: 8 query heads over 2 key/value heads."""
    L = configs.LayerShape(d=256, n_q_heads=8, n_kv_heads=2, head_dim=64, r=128)
    g = np.random.default_rng(77)
    W = (g.standard_normal((L.d, L.N)) * 0.02).astype(np.float32).astype(np.float64)
    ol, dl = _layers_from_weight(W, L)
    return L, ol, dl


@pytest.fixture(scope="module", params=[64, 128], ids=["g64", "g128"])
def tiny_w4(request):
    """The tiny layer with int4 weights, one scale per output channel and per
    group of 64 or 128 contraction rows (W4A8)."""
    wl = configs.get(1)
    ol, dl = _layers_from_weight(gen.weight_matrix(wl), wl.layer, w_bits=4, w_group=request.param)
    return wl, ol, dl


@pytest.fixture(scope="module")
def qwen():
    """Qwen2-VL-7B-shaped grouped-query layer: d=3584, 28 query / 4 key-value
    heads x 128, r=1024, int4 weights in groups of 128 (W4A8)."""
    wl = configs.get(4)
    L = wl.layer
    U, s, V = gen.weight_factors(wl)
    A, Bm = O.split_beta(U, s, V.T, wl.beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 4, 128)
    dl = B.DeviceLayer(prep.prepare_from_svd(U, s, V, L.n_q_heads, L.n_kv_heads, L.head_dim, wl.beta, 4, 128))
    return wl, ol, dl


@pytest.fixture(scope="module")
def llava():
    wl = configs.get(3)
    L = wl.layer
    U, s, V = gen.weight_factors(wl)
    A, Bm = O.split_beta(U, s, V.T, wl.beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
    dl = B.DeviceLayer(prep.prepare_from_svd(U, s, V, L.n_q_heads, L.n_kv_heads, L.head_dim, wl.beta))
    return wl, ol, dl


# ------------------------------------------------------------------ a1: quantizer

def _quant_cases():
    wl1, wl2 = configs.get(1), configs.get(2)
    ties = np.array([[127, 2.5, 3.5, -2.5, -0.5, 0.5, 1.5, -126.5]], np.float16)
    zero_and_ties = np.concatenate([np.zeros((1, 8), np.float16), ties, -ties])
    return [
        ("tiny-8bit", gen.prefill_activations(wl1), 8, 1.0, None),
        ("tiny-4bit", gen.prefill_activations(wl1), 4, 1.0, None),
        ("tiny-clip0.9", gen.prefill_activations(wl1), 8, 0.9, None),
        ("llava7b-prefill-2560x4096", gen.prefill_activations(wl2), 8, 1.0, None),
        ("K8", gen.random_rows(1, (5, 8), 3.0), 8, 1.0, None),
        ("K520-ragged", gen.random_rows(2, (7, 520), 1.0), 8, 1.0, None),
        ("M1", gen.random_rows(3, (1, 4096), 1.0), 8, 1.0, None),
        ("zero-and-ties", zero_and_ties, 8, 1.0, None),
        ("strided-ldx", gen.random_rows(4, (9, 264), 1.0), 8, 1.0, 256),
        ("4bit-strided", gen.random_rows(5, (9, 264), 1.0), 4, 1.0, 256),
    ]


@pytest.mark.parametrize("case", _quant_cases(), ids=lambda c: c[0])
def test_quantize_act_bitexact(case):
    name, x, bits, clip, K = case
    H.say(f"quantize_act {name} shape={x.shape} bits={bits}")
    xq, sx = H.quantize_act(x, bits, clip, K)
    xs = x if K is None else x[:, :K]
    q_ref, s_ref = O.quantize_act(xs, bits, clip)
    if bits == 4:
        q_ref = O.pack_int4(q_ref)
    assert np.array_equal(xq.view(np.uint8), q_ref.view(np.uint8))
    assert np.array_equal(sx.view(np.uint32), s_ref.view(np.uint32))


# ------------------------------------------------------------------ online H1 rotation + quantizer

def _rot_cases():
    wl1, wl2, wl4, wl5 = configs.get(1), configs.get(2), configs.get(4), configs.get(5)
    spike = np.zeros((2, 1024), np.float16)
    spike[0, 5], spike[1, 700] = 60000.0, -3.0
    spike4k = gen.random_rows(11, (3, 4096), 0.5)
    spike4k[0, 4095], spike4k[1, 0], spike4k[2, 2048] = 60000.0, -60000.0, 1000.0
    return [
        ("tiny-8bit", gen.prefill_activations(wl1), 8, None, 21),
        ("tiny-4bit", gen.prefill_activations(wl1), 4, None, 22),
        ("llava7b-2560x4096", gen.prefill_activations(wl2), 8, None, 23),
        ("qwen-640x3584-b512", gen.fill_activations(wl4, 640), 8, None, 24),
        ("13b-200x5120-b1024-4bit", gen.fill_activations(wl5, 200), 4, None, 25),
        ("K4096-b64", gen.random_rows(6, (37, 4096), 2.0), 8, 64, 26),
        ("K4096-b8", gen.random_rows(7, (5, 4096), 2.0), 8, 8, 27),
        ("K16384-b16384", gen.random_rows(8, (3, 16384), 1.0), 8, None, 28),
        ("no-signs", gen.random_rows(9, (11, 2048), 1.0), 8, None, None),
        ("zero-row-and-spikes", np.concatenate([np.zeros((1, 1024), np.float16), spike]), 8, None, 29),
        # K = B = 4096 (one wavefront per row): 4-bit codes, no signs with a zero row and spikes
        ("K4096-4bit", gen.random_rows(10, (9, 4096), 1.5), 4, None, 30),
        ("K4096-no-signs-zero-spike", np.concatenate([np.zeros((1, 4096), np.float16), spike4k]), 8, None, None),
    ]


@pytest.mark.parametrize("case", _rot_cases(), ids=lambda c: c[0])
def test_quantize_act_rotated_bitexact(case):
    """Q(X H1^T) with H1 = blockdiag(H_B) diag(s) / sqrt(B): codes and scales
    bit-exact against the oracle's stage-by-stage fp32 transform."""
    name, x, bits, block, seed = case
    K = x.shape[1]
    block = O.hadamard_block(K) if block is None else block
    signs = O.rotation_signs(K, seed) if seed is not None else None
    H.say(f"quantize_act_rotated {name} shape={x.shape} block={block} bits={bits}")
    xq, sx = H.quantize_act_rotated(x, signs, block, bits)
    q_ref, s_ref = O.quantize_act_rotated(x, signs if signs is not None else np.ones(K, np.int8), block, bits)
    if bits == 4:
        q_ref = O.pack_int4(q_ref)
    assert np.array_equal(sx.view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(xq.view(np.uint8), q_ref.view(np.uint8))


def test_prefill_with_online_rotation(tiny):
    """The tiny layer with H1 folded into W^d offline and X rotated online:
    every stored result bit-exact against the oracle, and the latent closer to
    the unquantized fp64 X W^d than without the rotation (outlier channels
    x20 spread over the block)."""
    wl, _, _ = tiny
    L = wl.layer
    A, Bm = O.factors_from_weight(gen.weight_matrix(wl), L.r, 0.5)
    blk = O.hadamard_block(L.d)
    s = O.rotation_signs(L.d, seed=31)
    A_rot = prep.fold_input_rotation(A, s, blk)
    ol = O.make_layer(A_rot, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
    dl = B.DeviceLayer(prep.quantize_layer(A_rot, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0))
    X = gen.prefill_activations(wl)
    H.say("prefill with online rotation, tiny layer")
    got = H.Prefill(dl, X.shape[0]).run(H.dev(X), signs=H.dev(s), block=blk).result()
    xq, sx = O.quantize_act_rotated(X, s, blk, 8)
    acc_xa, C_h = O.down_projection(ol, xq, sx)
    cq, sc = O.quantize_latent(C_h, 8)
    acc_cb, Q, K, V = O.up_projection(ol, cq, sc)
    assert np.array_equal(got["xq"], xq) and np.array_equal(got["sx"].view(np.uint32), sx.view(np.uint32))
    assert np.array_equal(got["acc_xa"], acc_xa)
    assert np.array_equal(got["C_h"].view(np.uint16), C_h.view(np.uint16))
    assert np.array_equal(got["acc_cb"], acc_cb)
    for key, ref in (("Q", Q), ("K", K), ("V", V)):
        assert np.array_equal(got[key].view(np.uint16), ref.view(np.uint16)), key
    exact = X.astype(np.float64) @ A
    plain = O.prefill(O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0), X, 8)["C_h"]
    e_rot = np.linalg.norm(got["C_h"].astype(np.float64) - exact) / np.linalg.norm(exact)
    e_plain = np.linalg.norm(plain.astype(np.float64) - exact) / np.linalg.norm(exact)
    H.say(f"  latent rel. error: rotated {e_rot:.3e}, plain {e_plain:.3e}")
    assert e_rot < e_plain


# ------------------------------------------------------------------ offline beta search on the GPU path

def test_beta_search_with_gpu_projection():
    """The beta line search (Eq. 14) scoring each beta with the GPU's quantized
    projection picks the same beta with the same squared errors as with the
    oracle's (the Q | K | V are bit-exact), on a layer with a decaying
    spectrum and outlier-heavy activations."""
    wl = configs.get(1)
    L = wl.layer
    g = np.random.default_rng(5)
    Q1, _ = np.linalg.qr(g.standard_normal((L.d, L.d)))
    Q2, _ = np.linalg.qr(g.standard_normal((L.N, L.d)))
    W = Q1 @ np.diag(0.5 * np.arange(1, L.d + 1) ** -0.7) @ Q2.T
    U, s, Vt = O.joint_svd(W)
    Ur, sr, Vtr = U[:, :L.r], s[:L.r], Vt[:L.r]
    X = gen.prefill_activations(wl)
    betas = [0.0, 0.2, 0.4, 0.5, 0.6, 0.8, 1.0]

    def oracle_proj(A, Bm, Xc):
        p = O.prefill(O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0), Xc, 8)
        return np.concatenate([p["Q"], p["K"], p["V"]], axis=1)

    H.say("beta search on the GPU projection")
    best, errs = prep.search_beta(Ur, sr, Vtr, X, betas, B.projection_evaluator(L.n_q_heads, L.n_kv_heads,
                                                                                L.head_dim))
    best_o, vals_o = O.beta_search(Ur, sr, Vtr, X, betas, oracle_proj)
    H.say(f"  beta {best}: errors {[round(e, 4) for e in errs]}")
    assert best == best_o
    assert np.array_equal(np.array(errs), np.array(vals_o))


# ------------------------------------------------------------------ a2-a4: projection

def _check_prefill(ol, got, X):
    ref = O.prefill(ol, X, 8)
    assert np.array_equal(got["xq"], ref["xq"])
    assert np.array_equal(got["sx"].view(np.uint32), ref["sx"].view(np.uint32))
    assert np.array_equal(got["acc_xa"], ref["acc_xa"])
    assert np.array_equal(got["C_h"].view(np.uint16), ref["C_h"].view(np.uint16))
    assert np.array_equal(got["cq"], ref["cq"])
    assert np.array_equal(got["sc"].view(np.uint32), ref["sc"].view(np.uint32))
    assert np.array_equal(got["acc_cb"], ref["acc_cb"])
    for key in ("Q", "K", "V"):
        if key in got:
            assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16)), key


@pytest.mark.parametrize("M", [1, 16, 31, 32, 33, 64, 200])
def test_prefill_bitexact_tiny(tiny, M):
    wl, ol, dl = tiny
    X = gen.fill_activations(wl, M)
    H.say(f"prefill tiny M={M}")
    got = H.Prefill(dl, M).run(H.dev(X)).result()
    _check_prefill(ol, got, X)


@pytest.mark.parametrize("M", [1, 16, 32])
def test_projection_bitexact_w4a8(tiny_w4, M):
    """Decode-size projection with int4 grouped weights: per-group fp32 sums in
    the definition's order make C, Q(C) and Q/K/V bit-exact."""
    wl, ol, dl = tiny_w4
    X = gen.fill_activations(wl, M)
    H.say(f"projection w4a8 group={dl.w_group} M={M}")
    got = H.Prefill(dl, M, debug=False).run(H.dev(X)).result()
    ref = O.prefill(ol, X, 8)
    for key in ("xq", "cq"):
        assert np.array_equal(got[key], ref[key]), key
    for key in ("sx", "sc"):
        assert np.array_equal(got[key].view(np.uint32), ref[key].view(np.uint32)), key
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16)), key


def test_projection_bitexact_llava7b_w4a8_g64_m32(llava):
    """The LLaVA-1.5-7B-shaped layer with int4 weights in groups of 64 and a
    32-token decode batch: 64 groups x 2 row blocks of int32 tiles (128 KB of
    LDS) in the down-projection, bit-exact against the oracle."""
    wl, _, _ = llava
    L = wl.layer
    U, s, V = gen.weight_factors(wl)
    A, Bm = O.split_beta(U, s, V.T, wl.beta)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, 4, 64)
    dl = B.DeviceLayer(prep.prepare_from_svd(U, s, V, L.n_q_heads, L.n_kv_heads, L.head_dim, wl.beta, 4, 64))
    X = gen.decode_activations(wl, 0, batch=32)
    H.say("projection llava7b w4a8 g64 M=32")
    got = H.Prefill(dl, 32, debug=False).run(H.dev(X)).result()
    ref = O.prefill(ol, X, 8)
    assert np.array_equal(got["cq"], ref["cq"])
    assert np.array_equal(got["sc"].view(np.uint32), ref["sc"].view(np.uint32))
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16)), key


@pytest.mark.parametrize("M", [1, 16, 32])
def test_projection_bitexact_w4a4(tiny_w4, M):
    """W4A4 decode-size projection: 4-bit per-token activation codes (two per
    byte) and 4-bit Q(C), int4 per-group weights; codes, scales, C and Q/K/V
    bit-exact against the oracle."""
    wl, ol, dl = tiny_w4
    X = gen.fill_activations(wl, M)
    H.say(f"projection w4a4 group={dl.w_group} M={M}")
    got = H.Prefill(dl, M, debug=False, abits=4).run(H.dev(X)).result()
    ref = O.prefill(ol, X, 4)
    assert np.array_equal(got["xq"].view(np.uint8), O.pack_int4(ref["xq"]))
    assert np.array_equal(got["cq"].view(np.uint8), O.pack_int4(ref["cq"]))
    for key in ("sx", "sc"):
        assert np.array_equal(got[key].view(np.uint32), ref[key].view(np.uint32)), key
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16)), key


def _check_mixed(ol, got, X, abits):
    ref = O.prefill(ol, X, abits)
    pack = (lambda c: c.view(np.uint8)) if abits == 8 else O.pack_int4
    assert np.array_equal(got["xq"].view(np.uint8), pack(ref["xq"]))
    assert np.array_equal(got["cq"].view(np.uint8), pack(ref["cq"]))
    for key in ("sx", "sc"):
        assert np.array_equal(got[key].view(np.uint32), ref[key].view(np.uint32)), key
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16)), key


@pytest.mark.parametrize("abits", [8, 4], ids=["a8", "a4"])
@pytest.mark.parametrize("M", [33, 64, 200])
def test_prefill_bitexact_w4(tiny_w4, M, abits):
    """Prefill-size projections with int4 per-group weights (groups of 64 or
    128) and 8- or 4-bit activations: the pipelined kernel widens int4 codes to
    int8 in registers and folds each group's exact int32 sum into fp32 in group
    order; everything bit-exact against the oracle, ragged row tiles."""
    wl, ol, dl = tiny_w4
    X = gen.fill_activations(wl, M)
    H.say(f"prefill w4a{abits} group={dl.w_group} M={M}")
    got = H.Prefill(dl, M, debug=False, abits=abits).run(H.dev(X)).result()
    _check_mixed(ol, got, X, abits)


def test_prefill_bitexact_w8a4_and_grouped_w8(tiny):
    """W8A4 with per-channel weights, and int8 weights with per-group scales,
    at 100 tokens."""
    wl, ol, dl = tiny
    X = gen.fill_activations(wl, 100)
    H.say("prefill w8a4 per-channel M=100")
    _check_mixed(ol, H.Prefill(dl, 100, debug=False, abits=4).run(H.dev(X)).result(), X, 4)
    ol8g, dl8g = _layers_from_weight(gen.weight_matrix(wl), wl.layer, w_bits=8, w_group=64)
    H.say("prefill w8a8 group 64 M=100")
    _check_mixed(ol8g, H.Prefill(dl8g, 100, debug=False).run(H.dev(X)).result(), X, 8)


def test_prefill_bitexact_qwen2vl_w4a8(qwen):
    """Qwen2-VL-shaped layer (d=3584, r=1024, N=4608, int4 groups of 128) over
    640 tokens, bit-exact."""
    wl, ol, dl = qwen
    X = gen.fill_activations(wl, 640)
    H.say("prefill qwen2vl w4a8 M=640")
    _check_mixed(ol, H.Prefill(dl, 640, debug=False).run(H.dev(X)).result(), X, 8)


def test_prefill_masks_leave_other_outputs(tiny):
    wl, ol, dl = tiny
    X = gen.fill_activations(wl, 40)
    for mask in (B.QSVD_OUT_Q, B.QSVD_OUT_K | B.QSVD_OUT_V):
        H.say(f"prefill mask={mask}")
        p = H.Prefill(dl, 40, mask=mask, debug=False)
        for t in (p.q, p.k, p.v):
            t.fill_(7.0)
        got = p.run(H.dev(X)).result()
        ref = O.prefill(ol, X, 8)
        for key, bit, t in (("Q", 1, p.q), ("K", 2, p.k), ("V", 4, p.v)):
            if mask & bit:
                assert np.array_equal(got[key].view(np.uint16), ref[key].view(np.uint16))
            else:
                assert bool((t == 7.0).all())


def test_prefill_bitexact_llava7b_full(llava):
    """The LLaVA-1.5-7B-shaped prefill at its full size: 4 x 640 tokens, d=4096, r=1536, N=12288."""
    wl, ol, dl = llava
    wl2 = configs.get(2)
    X = gen.prefill_activations(wl2)
    H.say(f"prefill llava7b M={X.shape[0]}")
    got = H.Prefill(dl, X.shape[0]).run(H.dev(X)).result()
    _check_prefill(ol, got, X)


@pytest.mark.parametrize("M", [2560, 2688, 2601], ids=["m2560", "m2688", "m2601"])
def test_prefill_bitexact_llava7b_production_tiles(llava, M):
    """The launch configuration the bench times: without accumulator dumps the
    up-projection (N=12288) runs on the 256 x 256-tile kernel in the per-XCD
    tile order.  M=2560 is the 4 x 640-token prefill (480 tiles, 60 per XCD);
    M=2688 adds a ragged last tile row (11 rows of tiles) and a last group of
    3 tile rows after the 8-row groups; M=2601 ends on a one-row tile row
    (loads clamped to the last row, stores masked)."""
    wl, ol, dl = llava
    X = gen.prefill_activations(configs.get(2), rows=M)
    H.say(f"prefill llava7b production tiles M={M}")
    got = H.Prefill(dl, M, debug=False).run(H.dev(X)).result()
    _check_mixed(ol, got, X, 8)


# ------------------------------------------------------------------ a3: cache append

@pytest.mark.parametrize("fmt", [B.QSVD_CACHE_F16, B.QSVD_CACHE_I8, B.QSVD_CACHE_I4], ids=["f16", "i8", "i4"])
def test_cache_append_bytes(tiny, fmt):
    wl, ol, dl = tiny
    bits = 4 if fmt == B.QSVD_CACHE_I4 else 8
    lengths = [0, 5, 17]
    batch, cap, r = 3, 32, wl.layer.r
    dc = B.DeviceCache(fmt, batch, cap, r, lengths)
    oc = O.LatentCache(fmt, batch, cap, r)
    oc.seq_len[:] = lengths
    for step, n_new in enumerate((3, 1, 6)):
        X = gen.fill_activations(wl, batch * n_new, layer=step)
        ref = O.prefill(ol, X, bits)
        H.say(f"cache append fmt={fmt} n_new={n_new}")
        c_h = H.dev(ref["C_h"])
        cq = H.dev(ref["cq"] if bits == 8 else O.pack_int4(ref["cq"]))
        sc = H.dev(ref["sc"])
        H.append(dc, c_h, cq, sc, n_new)
        for b in range(batch):
            oc.append(b, ref["C_h"][b * n_new:(b + 1) * n_new], ref["cq"][b * n_new:(b + 1) * n_new],
                      ref["sc"][b * n_new:(b + 1) * n_new])
    assert np.array_equal(H.host(dc.data).view(np.uint8), oc.data.view(np.uint8))
    if fmt != B.QSVD_CACHE_F16:
        assert np.array_equal(H.host(dc.scale).view(np.uint32), oc.scale.view(np.uint32))
    assert list(H.host(dc.seq_len)) == list(oc.seq_len)
    assert dc.max_len == 17 + 10
    with pytest.raises(B.QsvdError):
        H.append(dc, c_h, cq, sc, cap)


@pytest.mark.parametrize("n_new", [1, 17], ids=["fused", "two-launch"])
def test_cache_append_stops_at_capacity_on_device(tiny, n_new):
    """An append that the host check cannot see running past capacity (the
    host bound max_len lags the device lengths, as in a replayed graph) writes
    only the rows that fit, stops seq_len at capacity and raises the device
    overflow flag; sequences with room are appended as usual."""
    wl, ol, dl = tiny
    r = wl.layer.r
    cap = 4 if n_new == 1 else 18
    lengths = [cap, 2] if n_new == 1 else [3, 0]
    dc = B.DeviceCache(B.QSVD_CACHE_F16, 2, cap, r, lengths)
    before = gen.random_rows(61, (2, cap, r), 1.0)
    dc.data.copy_(H.dev(before))
    dc.c.max_len = 0                       # the host bound no longer covers the device lengths
    src = gen.random_rows(62, (2 * n_new, r), 1.0)
    H.say(f"cache append past capacity n_new={n_new}")
    H.append(dc, c_h=H.dev(src), n_new=n_new)
    got = H.host(dc.data)
    want = before.copy()
    for b, n0 in enumerate(lengths):
        k = max(0, min(n_new, cap - n0))
        want[b, n0:n0 + k] = src[b * n_new:b * n_new + k]
    assert np.array_equal(got.view(np.uint16), want.view(np.uint16))
    assert list(H.host(dc.seq_len)) == [min(n + n_new, cap) for n in lengths]
    assert int(H.host(dc.overflow)[0]) == 1
    # a later append that fits leaves the flag as the caller left it
    dc.overflow.zero_()
    dc.seq_len.fill_(0)
    dc.c.max_len = 0
    H.append(dc, c_h=H.dev(src), n_new=n_new)
    assert int(H.host(dc.overflow)[0]) == 0


@pytest.mark.parametrize("fmt", [B.QSVD_CACHE_F16, B.QSVD_CACHE_I8], ids=["f16", "i8"])
def test_cache_snapshot_resume(tiny, fmt):
    """Decode resumed from a snapshot of the device cache continues exactly as
    before: three steps, restore, the same three steps again give bit-identical
    outputs, cache bytes and lengths, in the original cache and in a fresh one."""
    wl, ol, dl = tiny
    r = wl.layer.r
    X = gen.prefill_activations(wl)[:40]
    dc = B.DeviceCache(fmt, 2, 48, r, [0, 0])
    pre = H.Prefill(dl, 40, mask=0, debug=False).run(H.dev(X))
    H.append(dc, pre.c_h, pre.cq, pre.sc, n_new=20)
    snap = dc.snapshot()
    steps = [gen.decode_activations(wl, t, batch=2) for t in range(3)]

    def run(cache):
        outs = []
        for xt in steps:
            p = H.Prefill(dl, 2, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
            H.append(cache, p.c_h, p.cq, p.sc, n_new=1)
            outs.append(H.host(H.decode_attention(dl, cache, p.q, B.QSVD_ATTN_AUTO)))
        return outs, H.host(cache.data), H.host(cache.seq_len)

    H.say(f"cache snapshot / resume fmt={fmt}")
    first = run(dc)
    for target in (dc, B.DeviceCache(fmt, 2, 48, r, [0, 0])):
        target.restore(snap)
        again = run(target)
        for a, b in zip(first[0], again[0]):
            assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
        assert np.array_equal(first[1].view(np.uint8), again[1].view(np.uint8))
        assert list(first[2]) == list(again[2]) == [23, 23]


# ------------------------------------------------------------------ f1: prefill attention over Q, K, V

def test_prefill_attention_flash_tiny_end_to_end(tiny):
    """Tiny layer (4 heads x 64): the 64 prefill tokens through the projection
    (Q, K, V bit-exact against the oracle), then causal attention over the
    projection's own rows, against the oracle's plain definition."""
    wl, ol, dl = tiny
    X = gen.prefill_activations(wl)
    ref = O.prefill(ol, X, 8)
    L = wl.layer
    H.say("prefill flash tiny")
    p = H.Prefill(dl, 64, mask=7, debug=False).run(H.dev(X))
    for name, t in (("Q", p.q), ("K", p.k), ("V", p.v)):
        assert np.array_equal(H.host(t).view(np.uint16), ref[name].view(np.uint16)), name
    out = H.host(H.prefill_attention(p.q, p.k, p.v, [64], L.n_q_heads, L.n_kv_heads, L.head_dim))
    want = O.prefill_attention(ref["Q"], ref["K"], ref["V"], [64], L.n_q_heads, L.n_kv_heads, L.head_dim)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    # the last row equals the latent-cache attention of the same query at that position
    oc = O.LatentCache(O.CACHE_F16, 1, 64, L.r)
    oc.append(0, ref["C_h"])
    last = O.attention_reference(ol, oc, ref["Q"][None, -1:], 1)[0, 0]
    assert np.abs(out[-1].astype(np.float64) - last).max() <= 2e-2


def _qkv(seed, M, hq, hkv, dh, scale=1.0):
    return (gen.random_rows(seed, (M, hq * dh), scale), gen.random_rows(seed + 1, (M, hkv * dh), scale),
            gen.random_rows(seed + 2, (M, hkv * dh), 1.0))


@pytest.mark.parametrize("shape,lengths", [
    ((8, 2, 64), [1, 45, 130]),          # grouped, ragged: one row, a partial tile, two query tiles
    ((4, 4, 128), [0, 200, 129, 1]),     # an empty sequence, tile edges at 128 + 1
    ((28, 4, 128), [640, 300]),          # Qwen2-VL-shaped grouping
], ids=["gqa8-2-dh64", "mha4-dh128-empty", "qwen28-4"])
def test_prefill_attention_flash_ragged(shape, lengths):
    """Causal prefill attention over seeded Q, K, V rows against the oracle,
    over ragged sequence lengths and grouped heads."""
    hq, hkv, dh = shape
    M = sum(lengths)
    Q, K, V = _qkv(300 + hq, M, hq, hkv, dh)
    H.say(f"prefill flash heads={hq}/{hkv} dh={dh} lengths={lengths}")
    out = H.host(H.prefill_attention(H.dev(Q), H.dev(K), H.dev(V), lengths, hq, hkv, dh))
    want = O.prefill_attention(Q, K, V, lengths, hq, hkv, dh)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


def test_prefill_attention_flash_llava7b_full():
    """The LLaVA-1.5-7B-shaped prompt batch at full size (4 x 640 tokens,
    32 heads x 128) in the bench's launch configuration, every output row
    against the oracle; then the same rows with ragged lengths (640, 640, 620,
    660) and a larger max_seqlen than any length; run twice bit-identically."""
    hq, hkv, dh = 32, 32, 128
    Q, K, V = _qkv(700, 2560, hq, hkv, dh)
    qd, kd, vd = H.dev(Q), H.dev(K), H.dev(V)
    for lengths, ms in (([640] * 4, 640), ([640, 640, 620, 660], 700)):
        H.say(f"prefill flash llava7b lengths={lengths} max_seqlen={ms}")
        out = H.host(H.prefill_attention(qd, kd, vd, lengths, hq, hkv, dh, max_seqlen=ms))
        want = O.prefill_attention(Q, K, V, lengths, hq, hkv, dh)
        ok, info = H.close_enough(out, want)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, info
    again = H.host(H.prefill_attention(qd, kd, vd, [640, 640, 620, 660], hq, hkv, dh, max_seqlen=700))
    assert np.array_equal(again.view(np.uint16), out.view(np.uint16))


def test_prefill_attention_flash_13b_two_sequences():
    """The 13B-shaped prompt (40 heads x 128, 704 = 576 + 128 tokens per
    sequence) on two of the batch's eight sequences, against the oracle, with
    queries scaled so that the softmax is peaked."""
    hq, hkv, dh = 40, 40, 128
    Q, K, V = _qkv(800, 1408, hq, hkv, dh, scale=2.0)
    H.say("prefill flash 13b two sequences")
    out = H.host(H.prefill_attention(H.dev(Q), H.dev(K), H.dev(V), [704, 704], hq, hkv, dh))
    want = O.prefill_attention(Q, K, V, [704, 704], hq, hkv, dh)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


# ------------------------------------------------------------------ f3 at q_len > 1: rotary prefill attention

def test_prefill_attention_rope_tiny_end_to_end(tiny):
    """Tiny layer (4 heads x 64): the projection's own Q, K, V through the
    rotary prefill attention against the oracle; its last row also against
    the oracle's rotary attention over the latent cache at that position,
    which a decode step continuing the prompt computes."""
    wl, ol, dl = tiny
    X = gen.prefill_activations(wl)
    ref = O.prefill(ol, X, 8)
    L = wl.layer
    H.say("prefill flash rope tiny")
    p = H.Prefill(dl, 64, mask=7, debug=False).run(H.dev(X))
    out = H.host(H.prefill_attention(p.q, p.k, p.v, [64], L.n_q_heads, L.n_kv_heads, L.head_dim, rope_theta=10000.0))
    want = O.prefill_attention(ref["Q"], ref["K"], ref["V"], [64], L.n_q_heads, L.n_kv_heads, L.head_dim,
                               rope_theta=10000.0)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    oc = O.LatentCache(O.CACHE_F16, 1, 64, L.r)
    oc.append(0, ref["C_h"])
    last = O.attention_reference(ol, oc, ref["Q"][None, -1:], 1, rope_theta=10000.0)[0, 0]
    assert np.abs(out[-1].astype(np.float64) - last).max() <= 2e-2
    plain = O.prefill_attention(ref["Q"], ref["K"], ref["V"], [64], L.n_q_heads, L.n_kv_heads, L.head_dim)
    assert not H.close_enough(out, plain)[0]


@pytest.mark.parametrize("shape,lengths,theta", [
    ((8, 2, 64), [1, 45, 130], 10000.0),          # grouped, ragged: one row, a partial tile, two query tiles
    ((4, 4, 128), [0, 200, 129, 1], 10000.0),     # an empty sequence, tile edges at 128 + 1
    ((28, 4, 128), [640, 300], 1e6),              # Qwen2-VL-shaped grouping, its rotary base
    ((8, 2, 128), [3000], 10000.0),               # positions up to 2999: thousands of turns per pair 0
], ids=["gqa8-2-dh64", "mha4-dh128-empty", "qwen28-4", "long3000"])
def test_prefill_attention_rope_ragged(shape, lengths, theta):
    """Rotary prefill attention over seeded Q, K, V rows against the oracle,
    over ragged lengths, grouped heads, two rotary bases and long positions."""
    hq, hkv, dh = shape
    M = sum(lengths)
    Q, K, V = _qkv(340 + hq, M, hq, hkv, dh)
    H.say(f"prefill flash rope heads={hq}/{hkv} dh={dh} lengths={lengths} theta={theta}")
    out = H.host(H.prefill_attention(H.dev(Q), H.dev(K), H.dev(V), lengths, hq, hkv, dh, rope_theta=theta))
    want = O.prefill_attention(Q, K, V, lengths, hq, hkv, dh, rope_theta=theta)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


def test_prefill_attention_rope_llava7b_full():
    """The LLaVA-1.5-7B-shaped prompt batch at full size (4 x 640 tokens,
    32 heads x 128, rotary base 10000) in the bench's launch configuration,
    every output row against the oracle, run twice bit-identically."""
    hq, hkv, dh = 32, 32, 128
    Q, K, V = _qkv(710, 2560, hq, hkv, dh)
    qd, kd, vd = H.dev(Q), H.dev(K), H.dev(V)
    H.say("prefill flash rope llava7b 4 x 640")
    out = H.host(H.prefill_attention(qd, kd, vd, [640] * 4, hq, hkv, dh, rope_theta=10000.0))
    want = O.prefill_attention(Q, K, V, [640] * 4, hq, hkv, dh, rope_theta=10000.0)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    again = H.host(H.prefill_attention(qd, kd, vd, [640] * 4, hq, hkv, dh, rope_theta=10000.0))
    assert np.array_equal(again.view(np.uint16), out.view(np.uint16))


def test_prefill_attention_rope_13b_two_sequences():
    """The 40-head 13B-shaped prompt (704 tokens per sequence) with rotary
    embeddings on two of the batch's eight sequences, against the oracle."""
    hq, hkv, dh = 40, 40, 128
    Q, K, V = _qkv(810, 1408, hq, hkv, dh, scale=2.0)
    H.say("prefill flash rope 13b two sequences")
    out = H.host(H.prefill_attention(H.dev(Q), H.dev(K), H.dev(V), [704, 704], hq, hkv, dh, rope_theta=10000.0))
    want = O.prefill_attention(Q, K, V, [704, 704], hq, hkv, dh, rope_theta=10000.0)
    ok, info = H.close_enough(out, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


def _layer_for(shape_id):
    """(layer shape, oracle layer, device layer, weight bits, group) of a decode projection case."""
    if shape_id == "tiny":
        wl = configs.get(1)
        ol, dl = _layers_from_weight(gen.weight_matrix(wl), wl.layer)
        return wl.layer, dl
    if shape_id == "llava7b":
        L = configs.LayerShape(d=4096, n_q_heads=32, n_kv_heads=32, head_dim=128, r=1536)
        return L, _random_factor_layer(L, 7007)[1]
    if shape_id == "qwen2vl":
        L = configs.LayerShape(d=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, r=1024)
        return L, _random_factor_layer(L, 7008, w_bits=4, w_group=128)[1]
    L = configs.LayerShape(d=5120, n_q_heads=40, n_kv_heads=40, head_dim=128, r=2048)
    return L, _random_factor_layer(L, 7009, w_bits=4, w_group=128)[1]


@pytest.mark.parametrize("shape_id,fmt,abits,batch,clip", [
    ("tiny", B.QSVD_CACHE_F16, 8, 1, 1.0),
    ("tiny", B.QSVD_CACHE_I8, 8, 3, 0.9),
    ("llava7b", B.QSVD_CACHE_F16, 8, 16, 1.0),       # the bench's decode step
    ("llava7b", B.QSVD_CACHE_I4, 4, 16, 1.0),
    ("qwen2vl", B.QSVD_CACHE_I8, 8, 32, 1.0),        # 32 rows: the quantizer as its own launch
    # d = 5120, wider than one wave's registers: 8 rows take two waves each
    # (each half read once), 3 and 5 rows four and three waves (uneven parts),
    # 16 rows one wave each (the row read twice)
    ("stack13b", B.QSVD_CACHE_I4, 4, 8, 1.0),
    ("stack13b", B.QSVD_CACHE_I8, 8, 3, 0.9),
    ("stack13b", B.QSVD_CACHE_F16, 4, 5, 1.0),
    ("stack13b", B.QSVD_CACHE_I8, 8, 16, 1.0),
], ids=["tiny-f16", "tiny-i8-clip", "llava7b-f16", "llava7b-i4", "qwen2vl-i8-w4", "13b-i4-w4a4", "13b-i8-b3",
        "13b-f16-a4-b5", "13b-i8-b16"])
def test_decode_project_append_equals_separate_calls(shape_id, fmt, abits, batch, clip):
    """The fused decode projection with its cache append leaves every output
    byte, cache byte and length exactly as quantize + projection (Q only) +
    append do, on two caches holding the same ragged rows."""
    torch = H.torch()
    L, dl = _layer_for(shape_id)
    per = 1 if abits == 8 else 2
    lengths = [(37 * b + 5) % 61 for b in range(batch)]
    cap = 64
    width = L.r if fmt != B.QSVD_CACHE_I4 else L.r // 2
    caches = [B.DeviceCache(fmt, batch, cap, L.r, lengths) for _ in range(2)]
    fill = gen.random_rows(900 + batch, (batch, cap, width), 1.0)
    for c in caches:
        if fmt == B.QSVD_CACHE_F16:
            c.data.copy_(H.dev(fill))
        else:
            c.data.copy_(H.dev(fill.view(np.uint16).astype(np.uint8)).view(c.data.dtype))
            c.scale.copy_(H.dev(np.abs(fill[:, :, 0]).astype(np.float32) + 0.01))
    X = gen.random_rows(950 + batch, (batch, L.d + 8), 1.0)
    X[:, 7] *= 30.0
    xd = H.dev(X)
    s = B.stream_handle()
    H.say(f"decode project+append {shape_id} fmt={fmt} a{abits} batch={batch}")
    outs = []
    for fused, c in ((False, caches[0]), (True, caches[1])):
        xq = torch.empty((batch, L.d // per), dtype=torch.uint8, device="cuda")
        sx = torch.empty((batch,), dtype=torch.float32, device="cuda")
        c_h = torch.empty((batch, L.r), dtype=torch.float16, device="cuda")
        cq = torch.empty((batch, L.r // per), dtype=torch.uint8, device="cuda")
        sc = torch.empty((batch,), dtype=torch.float32, device="cuda")
        q = torch.empty((batch, L.n_q), dtype=torch.float16, device="cuda")
        if fused:
            B.check(B.qsvd_decode_project_append(dl.c, c.c, B.ptr(xd), L.d + 8, abits, clip, B.ptr(xq), B.ptr(sx),
                                                 B.ptr(c_h), B.ptr(cq), B.ptr(sc), B.ptr(q), s))
        else:
            B.check(B.qsvd_quantize_act(B.ptr(xd), batch, L.d, L.d + 8, abits, clip, B.ptr(xq), B.ptr(sx), s))
            B.check(B.qsvd_lowrank_qkv_prefill(dl.c, B.ptr(xq), B.ptr(sx), batch, abits, B.QSVD_OUT_Q, B.ptr(c_h),
                                               B.ptr(cq), B.ptr(sc), B.ptr(q), 0, 0, 0, 0, 0, 0, s))
            if fmt == B.QSVD_CACHE_F16:
                H.append(c, c_h=c_h, n_new=1)
            else:
                H.append(c, cq=cq, sc=sc, n_new=1)
        outs.append({k: H.host(t).view(np.uint8).copy() for k, t in
                     (("xq", xq), ("sx", sx), ("c_h", c_h), ("cq", cq), ("sc", sc), ("q", q))})
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert np.array_equal(H.host(caches[0].data).view(np.uint8), H.host(caches[1].data).view(np.uint8))
    if fmt != B.QSVD_CACHE_F16:
        assert np.array_equal(H.host(caches[0].scale).view(np.uint32), H.host(caches[1].scale).view(np.uint32))
    assert list(H.host(caches[1].seq_len)) == [n + 1 for n in lengths]
    assert caches[0].max_len == caches[1].max_len == max(lengths) + 1
    assert int(H.host(caches[1].overflow)[0]) == 0


def test_decode_project_append_capacity_on_device(tiny):
    """A fused append the host bound cannot see running past capacity drops
    the row, stops seq_len at capacity and raises the overflow flag."""
    wl, ol, dl = tiny
    L = wl.layer
    torch = H.torch()
    dc = B.DeviceCache(B.QSVD_CACHE_I8, 2, 8, L.r, [8, 3])
    dc.c.max_len = 0
    before = H.host(dc.data).copy()
    x = H.dev(gen.random_rows(71, (2, L.d), 1.0))
    bufs = [torch.empty(shape, dtype=dt, device="cuda") for shape, dt in
            (((2, L.d), torch.int8), ((2,), torch.float32), ((2, L.r), torch.float16), ((2, L.r), torch.int8),
             ((2,), torch.float32), ((2, L.n_q), torch.float16))]
    B.check(B.qsvd_decode_project_append(dl.c, dc.c, B.ptr(x), L.d, 8, 1.0, *[B.ptr(t) for t in bufs],
                                         B.stream_handle()))
    got = H.host(dc.data)
    assert np.array_equal(got[0], before[0])
    assert np.array_equal(got[1, 3], H.host(bufs[3])[1])
    assert list(H.host(dc.seq_len)) == [8, 4]
    assert int(H.host(dc.overflow)[0]) == 1


# ------------------------------------------------------------------ a5-a7: decode attention

@pytest.mark.parametrize("mode", MODES, ids=MODE_IDS)
def test_decode_tiny_end_to_end(tiny, mode):
    """Tiny layer: 64 prefill tokens into an fp16 latent cache, then 16 decode
    steps of projection, append and attention, each against the oracle."""
    wl, ol, dl = tiny
    X = gen.prefill_activations(wl)
    oc = O.LatentCache(O.CACHE_F16, 1, 64 + wl.decode_steps, wl.layer.r)
    O.cache_append_prefill(oc, O.prefill(ol, X, 8), [64])
    dc = B.DeviceCache(B.QSVD_CACHE_F16, 1, 64 + wl.decode_steps, wl.layer.r, [0])
    pre = H.Prefill(dl, 64, mask=0, debug=False).run(H.dev(X))
    H.append(dc, pre.c_h, n_new=64)
    for t in range(wl.decode_steps):
        xt = gen.decode_activations(wl, t)
        ref = O.decode_step(ol, oc, xt, 8)
        H.say(f"decode tiny step={t} mode={mode}")
        p = H.Prefill(dl, 1, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
        H.append(dc, p.c_h, n_new=1)
        out = H.host(H.decode_attention(dl, dc, p.q, mode))
        assert np.array_equal(H.host(p.c_h).view(np.uint16), ref["C_h"].view(np.uint16))
        assert np.array_equal(H.host(p.q).view(np.uint16), ref["Q"].view(np.uint16))
        ok, info = H.close_enough(out, ref["out"])
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (t, info)


@pytest.mark.parametrize("mode", MODES, ids=MODE_IDS)
def test_decode_gqa_int8_ragged(gqa, mode):
    """Grouped queries (8 over 2), int8 latent cache with per-token scales,
    ragged lengths 1 / 45 / 130 across the batch, 3 decode steps."""
    L, ol, dl = gqa
    lengths = [1, 45, 130]
    batch, cap = 3, 140
    wl = configs.Workload(95, "gqa-test", L, "gaussian", 8, 0, 8, configs.CACHE_I8)
    codes, scales = gen.latent_codes(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_I8, batch, cap, L.r)
    dc = B.DeviceCache(B.QSVD_CACHE_I8, batch, cap, L.r, lengths)
    for b, n in enumerate(lengths):
        oc.append(b, None, codes[b, :n], scales[b, :n])
    dc.data.copy_(H.dev(np.where(np.arange(cap)[None, :, None] < np.array(lengths)[:, None, None], codes, 0)))
    dc.scale.copy_(H.dev(np.where(np.arange(cap)[None, :] < np.array(lengths)[:, None], scales, 0)))
    for t in range(3):
        xt = gen.decode_activations(wl, t, batch=batch)
        ref = O.decode_step(ol, oc, xt, 8)
        H.say(f"decode gqa int8 step={t} mode={mode}")
        p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
        H.append(dc, cq=p.cq, sc=p.sc, n_new=1)
        out = H.host(H.decode_attention(dl, dc, p.q, mode))
        assert np.array_equal(H.host(p.cq), ref["cq"])
        ok, info = H.close_enough(out, ref["out"])
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (t, info)
    assert np.array_equal(H.host(dc.data), oc.data)


@pytest.mark.parametrize("mode", MODES, ids=MODE_IDS)
def test_decode_llava7b_width_ragged(llava, mode):
    """LLaVA-1.5-7B-shaped layer (r=1536, 32 heads) over an fp16 latent cache
    with ragged lengths 1 / 33 / 290 / 1000 (one to many tiles and chunks)."""
    wl, ol, dl = llava
    lengths = [1, 33, 290, 1000]
    batch, cap = 4, 1008
    rows = gen.latent_rows(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_F16, batch, cap, wl.layer.r)
    for b, n in enumerate(lengths):
        oc.append(b, rows[b, :n])
    dc = B.DeviceCache(B.QSVD_CACHE_F16, batch, cap, wl.layer.r, lengths)
    dc.data.copy_(H.dev(oc.data))
    xt = gen.decode_activations(wl, 0, batch=batch)
    ref = O.decode_step(ol, oc, xt, 8)
    H.say(f"decode llava7b ragged mode={mode}")
    p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
    H.append(dc, p.c_h, n_new=1)
    out = H.host(H.decode_attention(dl, dc, p.q, mode))
    assert np.array_equal(H.host(p.q).view(np.uint16), ref["Q"].view(np.uint16))
    ok, info = H.close_enough(out, ref["out"])
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I8, O.CACHE_I4], ids=["f16", "i8", "i4"])
def test_decode_llava7b_width_odd_capacity_full(llava, fmt):
    """The 32-head r = 1536 attention reads its staged tiles in range-checked
    groups of 8 (fp16) or 16 (integer) rows that end at the chunk end: a
    capacity of 1001 rows (a multiple of neither), one sequence filling it,
    one ending two rows short, one of a single row and one of 17, in every
    cache format, against the oracle; a second call gives the same bytes."""
    wl, ol, dl = llava
    lengths = [1001, 999, 1, 17]
    oc, dc = _prefilled_caches(wl, fmt, lengths, 1001)
    g = np.random.default_rng(1001)
    q = (g.standard_normal((4, wl.layer.n_q_heads * wl.layer.head_dim)) * 2.0).astype(np.float16)
    H.say(f"decode llava7b width odd capacity fmt={fmt}")
    ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1)[:, 0, :]
    out = H.host(H.decode_attention(dl, dc, H.dev(q), B.QSVD_ATTN_ABSORBED))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    again = H.host(H.decode_attention(dl, dc, H.dev(q), B.QSVD_ATTN_ABSORBED))
    assert np.array_equal(out.view(np.uint16), again.view(np.uint16))


def test_decode_llava7b_full_size_sampled(llava):
    """The decode workload at its full size (16 sequences x 4096 cached tokens,
    fp16 latent cache of width 1536) in the launch configuration the bench
    times; every sequence against the oracle's absorbed form (pinned equal to
    the plain definition), two also against the plain definition."""
    wl, ol, dl = llava
    batch, L0, cap = 16, 4096, 4096 + 8
    rows = gen.latent_rows(wl, batch, cap)
    dc = B.DeviceCache(B.QSVD_CACHE_F16, batch, cap, wl.layer.r, [L0] * batch)
    dc.data.copy_(H.dev(rows))
    xt = gen.decode_activations(wl, 0, batch=batch)
    H.say("decode llava7b full size")
    p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
    H.append(dc, p.c_h, n_new=1)
    out = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    out2 = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    assert np.array_equal(out.view(np.uint16), out2.view(np.uint16)), "decode attention is not deterministic"
    assert np.all(np.isfinite(out.astype(np.float32)))
    for b in range(batch):
        for plain in ((False, True) if b in (0, 11) else (False,)):
            oc = O.LatentCache(O.CACHE_F16, 1, cap, wl.layer.r)
            oc.append(0, rows[b, :L0])
            ref = O.decode_step(ol, oc, xt[b:b + 1], 8, reference=plain)
            ok, info = H.close_enough(out[b:b + 1], ref["out"])
            H.say(f"  b={b} plain={plain} max-abs, rel-L2, rms = {info}")
            assert ok, (b, plain, info)


def test_decode_qwen2vl_w4a8_int8_cache_full_size(qwen):
    """The Qwen2-VL-7B-shaped decode workload at full size: 32 sequences x 8192
    cached tokens in an int8 latent cache with per-token scales, W4A8 projection
    of the new tokens, grouped-query absorbed attention; every sequence
    checked against the oracle's absorbed form (pinned equal to the plain
    definition), two also against the plain definition; all outputs finite,
    run twice bit-identically."""
    wl, ol, dl = qwen
    L = wl.layer
    batch, L0 = wl.decode_batch, wl.decode_ctx
    cap = L0 + 8
    codes, scales = gen.latent_codes(wl, batch, cap)
    dc = B.DeviceCache(B.QSVD_CACHE_I8, batch, cap, L.r, [L0] * batch)
    dc.data.copy_(H.dev(codes))
    dc.scale.copy_(H.dev(scales))
    xt = gen.decode_activations(wl, 0, batch=batch)
    H.say("decode qwen2vl w4a8 int8 cache full size")
    p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
    H.append(dc, cq=p.cq, sc=p.sc, n_new=1)
    out = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    out2 = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    assert np.array_equal(out.view(np.uint16), out2.view(np.uint16))
    assert np.all(np.isfinite(out.astype(np.float32)))
    for b in range(batch):
        for plain in ((False, True) if b in (0, 29) else (False,)):
            oc = O.LatentCache(O.CACHE_I8, 1, cap, L.r)
            oc.append(0, None, codes[b, :L0], scales[b, :L0])
            ref = O.decode_step(ol, oc, xt[b:b + 1], 8, reference=plain)
            assert np.array_equal(H.host(p.cq)[b:b + 1], ref["cq"])
            assert np.array_equal(H.host(p.q)[b:b + 1].view(np.uint16), ref["Q"].view(np.uint16))
            ok, info = H.close_enough(out[b:b + 1], ref["out"])
            H.say(f"  b={b} plain={plain} max-abs, rel-L2, rms = {info}")
            assert ok, (b, plain, info)


# ------------------------------------------------------------------ 13B-shaped stack layer at full size

@pytest.fixture(scope="module")
def stack13b():
    """One layer of the LLaVA-1.5-13B-shaped stack at its widest rank: d=5120,
    40 heads x 128, r=3072, int4 weights in groups of 128 (random factors:
    the stack's timing runs draw codes directly, parity needs a prepared
    layer)."""
    wl = configs.get(5)
    L = configs.LayerShape(d=5120, n_q_heads=40, n_kv_heads=40, head_dim=128, r=3072)
    ol, dl = _random_factor_layer(L, 13013, w_bits=4, w_group=128)
    return gen.with_rank(wl, 3072), L, ol, dl


def test_prefill_13b_w4a4_full_size_sampled(stack13b):
    """The stack's prefill at full size (8 x 704 = 5632 tokens, W4A4, the launch
    the bench times): sampled rows bit-exact against the oracle."""
    wl, L, ol, dl = stack13b
    X = gen.prefill_activations(wl)
    M = X.shape[0]
    H.say(f"prefill 13b w4a4 M={M} r={L.r}")
    got = H.Prefill(dl, M, debug=False, abits=4).run(H.dev(X)).result()
    rows = np.array([0, 1, 575, 703, 704, 2816, 4223, M - 1])
    ref = O.prefill(ol, X[rows], 4)
    assert np.array_equal(got["xq"][rows].view(np.uint8), O.pack_int4(ref["xq"]))
    assert np.array_equal(got["cq"][rows].view(np.uint8), O.pack_int4(ref["cq"]))
    for key in ("sx", "sc"):
        assert np.array_equal(got[key][rows].view(np.uint32), ref[key].view(np.uint32)), key
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key][rows].view(np.uint16), ref[key].view(np.uint16)), key
    for key in ("Q", "K", "V"):
        assert np.all(np.isfinite(got[key].astype(np.float32))), key


def test_decode_13b_int4_cache_full_size_sampled(stack13b):
    """The stack's decode at full size for its widest layer: batch 8 over 4096
    cached tokens in an int4 latent cache (r = 3072, three 128-column units per
    wave), W4A4 projection of the new tokens, 40 query heads in 16-head blocks;
    every sequence checked against the oracle's latent form (pinned equal to
    the plain definition), all outputs finite, run twice bit-identically."""
    wl, L, ol, dl = stack13b
    torch = H.torch()
    batch, L0 = wl.decode_batch, wl.decode_ctx
    cap = L0 + 4
    rows = gen.latent_rows(wl, batch, L0)
    data = np.zeros((batch, cap, L.r // 2), np.uint8)
    scale = np.zeros((batch, cap), np.float32)
    codes_of = {}
    for b in range(batch):
        codes, sc = O.quantize_act(rows[b], 4)
        data[b, :L0], scale[b, :L0] = O.pack_int4(codes), sc
        codes_of[b] = codes
    dc = B.DeviceCache(B.QSVD_CACHE_I4, batch, cap, L.r, [L0] * batch)
    dc.data.copy_(H.dev(data))
    dc.scale.copy_(H.dev(scale))
    xt = gen.decode_activations(wl, 0, batch=batch)
    H.say(f"decode 13b int4 cache full size r={L.r}")
    p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False, abits=4).run(H.dev(xt))
    cq4 = torch.empty((batch, L.r // 2), dtype=torch.uint8, device="cuda")
    sc4 = torch.empty((batch,), dtype=torch.float32, device="cuda")
    B.check(B.qsvd_quantize_act(B.ptr(p.c_h), batch, L.r, L.r, 4, 1.0, B.ptr(cq4), B.ptr(sc4), B.stream_handle()))
    H.append(dc, cq=cq4, sc=sc4, n_new=1)
    out = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    out2 = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    assert np.array_equal(out.view(np.uint16), out2.view(np.uint16))
    assert np.all(np.isfinite(out.astype(np.float32)))
    for b in range(batch):
        ref = O.prefill(ol, xt[b:b + 1], 4)
        assert np.array_equal(H.host(p.q)[b:b + 1].view(np.uint16), ref["Q"].view(np.uint16))
        q4, s4 = O.quantize_act(ref["C_h"], 4)
        oc = O.LatentCache(O.CACHE_I4, 1, cap, L.r)
        oc.append(0, None, codes_of[b], scale[b, :L0])
        oc.append(0, None, q4, s4)
        assert np.array_equal(H.host(dc.data)[b, :L0 + 1], oc.data[0, :L0 + 1])
        want = O.attention_absorbed(ol, oc, ref["Q"][:, None, :], 1)[:, 0, :]
        ok, info = H.close_enough(out[b:b + 1], want)
        H.say(f"  b={b} max-abs, rel-L2, rms = {info}")
        assert ok, (b, info)


@pytest.mark.parametrize("M,tile_rows", [(5632, (2816, 2944)), (5600, (5504, 5600))],
                         ids=["m5632-interior-tile-row", "m5600-ragged-last-tile-row"])
def test_prefill_13b_w4a4_whole_tile_rows(stack13b, M, tile_rows):
    """The stack's W4A4 prefill (d = 5120, r = 3072, N = 15360) checked over a
    whole 128-row tile row of the products: an interior one at the full
    8 x 704 = 5632 tokens, and the ragged last one (96 rows) at 5600 tokens;
    codes, scales, C and Q / K / V bit-exact against the oracle."""
    wl, L, ol, dl = stack13b
    X = gen.prefill_activations(wl)[:M]
    H.say(f"prefill 13b w4a4 M={M} rows {tile_rows}")
    got = H.Prefill(dl, M, debug=False, abits=4).run(H.dev(X)).result()
    rows = np.arange(*tile_rows)
    ref = O.prefill(ol, X[rows], 4)
    assert np.array_equal(got["xq"][rows].view(np.uint8), O.pack_int4(ref["xq"]))
    assert np.array_equal(got["cq"][rows].view(np.uint8), O.pack_int4(ref["cq"]))
    for key in ("sx", "sc"):
        assert np.array_equal(got[key][rows].view(np.uint32), ref[key].view(np.uint32)), key
    for key in ("C_h", "Q", "K", "V"):
        assert np.array_equal(got[key][rows].view(np.uint16), ref[key].view(np.uint16)), key


def test_decode_13b_int4_cache_rank_2048_plain_definition():
    """A mid-range layer of the stack (r = 2048, two 128-column units per wave,
    32-token tiles) at the full decode size (batch 8 over 4096 cached int4 rows,
    W4A4 projection, 40 heads in 16-head blocks), two sequences against the
    plain definition (K and V rebuilt from the cache, Eq. 5) rather than the
    latent form."""
    wl = gen.with_rank(configs.get(5), 2048)
    L = configs.LayerShape(d=5120, n_q_heads=40, n_kv_heads=40, head_dim=128, r=2048)
    ol, dl = _random_factor_layer(L, 12048, w_bits=4, w_group=128)
    torch = H.torch()
    batch, L0 = wl.decode_batch, wl.decode_ctx
    cap = L0 + 4
    rows = gen.latent_rows(wl, batch, L0)
    data = np.zeros((batch, cap, L.r // 2), np.uint8)
    scale = np.zeros((batch, cap), np.float32)
    codes_of = {}
    for b in range(batch):
        codes, sc = O.quantize_act(rows[b], 4)
        data[b, :L0], scale[b, :L0] = O.pack_int4(codes), sc
        if b in (2, 7):
            codes_of[b] = codes
    dc = B.DeviceCache(B.QSVD_CACHE_I4, batch, cap, L.r, [L0] * batch)
    dc.data.copy_(H.dev(data))
    dc.scale.copy_(H.dev(scale))
    xt = gen.decode_activations(wl, 3, batch=batch)
    H.say(f"decode 13b int4 cache r={L.r} against the plain definition")
    p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False, abits=4).run(H.dev(xt))
    cq4 = torch.empty((batch, L.r // 2), dtype=torch.uint8, device="cuda")
    sc4 = torch.empty((batch,), dtype=torch.float32, device="cuda")
    B.check(B.qsvd_quantize_act(B.ptr(p.c_h), batch, L.r, L.r, 4, 1.0, B.ptr(cq4), B.ptr(sc4), B.stream_handle()))
    H.append(dc, cq=cq4, sc=sc4, n_new=1)
    out = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
    assert np.all(np.isfinite(out.astype(np.float32)))
    for b in (2, 7):
        ref = O.prefill(ol, xt[b:b + 1], 4)
        assert np.array_equal(H.host(p.q)[b:b + 1].view(np.uint16), ref["Q"].view(np.uint16))
        q4, s4 = O.quantize_act(ref["C_h"], 4)
        oc = O.LatentCache(O.CACHE_I4, 1, cap, L.r)
        oc.append(0, None, codes_of[b], scale[b, :L0])
        oc.append(0, None, q4, s4)
        want = O.attention_reference(ol, oc, ref["Q"][:, None, :], 1)[:, 0, :]
        ok, info = H.close_enough(out[b:b + 1], want)
        H.say(f"  b={b} max-abs, rel-L2, rms = {info}")
        assert ok, (b, info)


# ------------------------------------------------------------------ prefill attention (q_len > 1)

def test_prefill_attention_tiny_causal(tiny):
    """The tiny layer's 64 prefill tokens attend causally over their own latent
    rows (queries = the last q_len = 64 cached positions), absorbed form,
    against the plain definition."""
    wl, ol, dl = tiny
    X = gen.prefill_activations(wl)
    M, nq = X.shape[0], wl.layer.n_q
    ref_proj = O.prefill(ol, X, 8)
    oc = O.LatentCache(O.CACHE_F16, 1, M, wl.layer.r)
    O.cache_append_prefill(oc, ref_proj, [M])
    ref = O.attention_reference(ol, oc, ref_proj["Q"].reshape(1, M, nq), M)
    dc = B.DeviceCache(B.QSVD_CACHE_F16, 1, M, wl.layer.r, [0])
    H.say("prefill attention tiny q_len=64")
    p = H.Prefill(dl, M, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(X))
    H.append(dc, p.c_h, n_new=M)
    assert np.array_equal(H.host(p.q).view(np.uint16), ref_proj["Q"].view(np.uint16))
    out = H.host(H.decode_attention(dl, dc, p.q.reshape(1, M, nq), B.QSVD_ATTN_ABSORBED, q_len=M))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    # the last query row is the decode query at the same position
    out1 = H.host(H.decode_attention(dl, dc, p.q[M - 1:], B.QSVD_ATTN_ABSORBED))
    ok, info = H.close_enough(out1[0], ref[0, M - 1])
    assert ok, info


def test_prefill_attention_gqa_int8_ragged(gqa):
    """Five new tokens per sequence (projected together, 15 rows) appended to
    int8 caches of ragged prior lengths 0 / 40 / 100, then attended causally
    with q_len = 5: grouped queries (8 over 2), absorbed form."""
    L, ol, dl = gqa
    prior, q_len, batch = [0, 40, 100], 5, 3
    cap = max(prior) + q_len
    wl = configs.Workload(95, "gqa-test", L, "gaussian", 8, 0, 8, configs.CACHE_I8)
    codes, scales = gen.latent_codes(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_I8, batch, cap, L.r)
    dc = B.DeviceCache(B.QSVD_CACHE_I8, batch, cap, L.r, prior)
    for b, n in enumerate(prior):
        if n:
            oc.append(b, None, codes[b, :n], scales[b, :n])
    dc.data.copy_(H.dev(np.where(np.arange(cap)[None, :, None] < np.array(prior)[:, None, None], codes, 0)))
    dc.scale.copy_(H.dev(np.where(np.arange(cap)[None, :] < np.array(prior)[:, None], scales, 0)))
    X = gen.decode_activations(wl, 7, batch=batch * q_len)
    ref_proj = O.prefill(ol, X, 8)
    for b in range(batch):
        rows = slice(b * q_len, (b + 1) * q_len)
        oc.append(b, None, ref_proj["cq"][rows], ref_proj["sc"][rows])
    nq = L.n_q_heads * L.head_dim
    ref = O.attention_reference(ol, oc, ref_proj["Q"].reshape(batch, q_len, nq), q_len)
    H.say("prefill attention gqa int8 ragged q_len=5")
    p = H.Prefill(dl, batch * q_len, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(X))
    H.append(dc, cq=p.cq, sc=p.sc, n_new=q_len)
    assert np.array_equal(H.host(dc.data), oc.data)
    out = H.host(H.decode_attention(dl, dc, p.q.reshape(batch, q_len, nq), B.QSVD_ATTN_AUTO, q_len=q_len))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


def test_prefill_attention_llava7b_chunked(llava):
    """LLaVA-shaped layer (r = 1536): four new tokens per sequence on top of
    fp16 caches of 300 / 1000 tokens, q_len = 4, several context chunks per
    query row; three query rows checked against the plain definition."""
    wl, ol, dl = llava
    L = wl.layer
    prior, q_len, batch = [300, 1000], 4, 2
    cap = max(prior) + q_len
    rows = gen.latent_rows(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_F16, batch, cap, L.r)
    dc = B.DeviceCache(B.QSVD_CACHE_F16, batch, cap, L.r, prior)
    for b, n in enumerate(prior):
        oc.append(b, rows[b, :n])
    dc.data.copy_(H.dev(np.where(np.arange(cap)[None, :, None] < np.array(prior)[:, None, None], rows, 0)))
    X = gen.decode_activations(wl, 3, batch=batch * q_len)
    ref_proj = O.prefill(ol, X, 8)
    for b in range(batch):
        oc.append(b, ref_proj["C_h"][b * q_len:(b + 1) * q_len])
    H.say("prefill attention llava7b q_len=4")
    p = H.Prefill(dl, batch * q_len, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(X))
    H.append(dc, p.c_h, n_new=q_len)
    nq = L.n_q
    out = H.host(H.decode_attention(dl, dc, p.q.reshape(batch, q_len, nq), B.QSVD_ATTN_ABSORBED, q_len=q_len))
    for b, i in ((0, 0), (1, 3), (1, 1)):
        ref = O.attention_reference(ol, oc, ref_proj["Q"].reshape(batch, q_len, nq), q_len, batches=[b])
        ok, info = H.close_enough(out[b, i], ref[b, i])
        H.say(f"  b={b} i={i} max-abs, rel-L2, rms = {info}")
        assert ok, (b, i, info)


def _random_factor_layer(L, seed, w_bits=8, w_group=0):
    """A layer straight from random factors A (d x r) ~ N(0, 1/d) and
    B (r x N) ~ N(0, 1/r), for wide shapes where an SVD would be slow (the
    attention only sees B and the latent rows)."""
    g = np.random.default_rng(seed)
    A = g.standard_normal((L.d, L.r)) / np.sqrt(L.d)
    Bm = g.standard_normal((L.r, L.N)) / np.sqrt(L.r)
    ol = O.make_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, w_bits, w_group)
    pl = prep.quantize_layer(A, Bm, L.n_q_heads, L.n_kv_heads, L.head_dim, w_bits, w_group)
    return ol, B.DeviceLayer(pl)


def _prefilled_caches(wl, fmt, prior, cap):
    """Oracle and device caches holding synthetic rows at the given lengths."""
    L = wl.layer
    batch = len(prior)
    oc = O.LatentCache(fmt, batch, cap, L.r)
    dc = B.DeviceCache(fmt, batch, cap, L.r, prior)
    rows = gen.latent_rows(wl, batch, cap)
    if fmt == O.CACHE_F16:
        for b, n in enumerate(prior):
            if n:
                oc.append(b, rows[b, :n])
        dc.data.copy_(H.dev(np.where(np.arange(cap)[None, :, None] < np.array(prior)[:, None, None], rows, 0)))
        return oc, dc
    bits = 4 if fmt == O.CACHE_I4 else 8
    data = np.zeros((batch, cap, L.r // 2 if bits == 4 else L.r), np.uint8)
    scale = np.zeros((batch, cap), np.float32)
    for b, n in enumerate(prior):
        if n:
            codes, sc = O.quantize_act(rows[b, :n], bits)
            oc.append(b, None, codes, sc)
            data[b, :n] = O.pack_int4(codes) if bits == 4 else codes.view(np.uint8)
            scale[b, :n] = sc
    dc.data.copy_(H.dev(data.view(np.int8) if bits == 8 else data))
    dc.scale.copy_(H.dev(scale))
    return oc, dc


def _append_new_rows(ol, dl, oc, dc, X, q_len):
    """Project X (batch * q_len rows, sequence-major) on both sides and append
    the new latent rows in the cache's format; returns (oracle Q, device Q)."""
    torch = H.torch()
    batch = dc.batch
    ref = O.prefill(ol, X, 8)
    p = H.Prefill(dl, X.shape[0], mask=B.QSVD_OUT_Q, debug=False).run(H.dev(X))
    if oc.fmt == O.CACHE_F16:
        new_o = [(ref["C_h"][b * q_len:(b + 1) * q_len],) for b in range(batch)]
        H.append(dc, c_h=p.c_h, n_new=q_len)
    elif oc.fmt == O.CACHE_I8:
        new_o = [(None, ref["cq"][b * q_len:(b + 1) * q_len], ref["sc"][b * q_len:(b + 1) * q_len])
                 for b in range(batch)]
        H.append(dc, cq=p.cq, sc=p.sc, n_new=q_len)
    else:
        q4, s4 = O.quantize_act(ref["C_h"], 4)
        new_o = [(None, q4[b * q_len:(b + 1) * q_len], s4[b * q_len:(b + 1) * q_len]) for b in range(batch)]
        r = oc.r
        cq4 = torch.empty((X.shape[0], r // 2), dtype=torch.uint8, device="cuda")
        sc4 = torch.empty((X.shape[0],), dtype=torch.float32, device="cuda")
        B.check(B.qsvd_quantize_act(B.ptr(p.c_h), X.shape[0], r, r, 4, 1.0, B.ptr(cq4), B.ptr(sc4),
                                    B.stream_handle()))
        H.append(dc, cq=cq4, sc=sc4, n_new=q_len)
    for b in range(batch):
        oc.append(b, *new_o[b])
    return ref["Q"], p.q


FMTS = [O.CACHE_F16, O.CACHE_I8, O.CACHE_I4]
FMT_IDS = ["f16", "i8", "i4"]


@pytest.mark.parametrize("fmt", FMTS, ids=FMT_IDS)
@pytest.mark.parametrize("r", [1152, 2176])
def test_decode_wide_heads(fmt, r):
    """40 query heads over 8 key/value heads (more than one 32-head block) at
    ranks 1152 and 2176 (128-column units that do not split evenly over the
    waves): the 16-head-block attention, ragged prior lengths 1 / 130 / 777,
    one decode step, every cache format."""
    L = configs.LayerShape(d=256, n_q_heads=40, n_kv_heads=8, head_dim=128, r=r)
    ol, dl = _random_factor_layer(L, 4000 + r)
    wl = configs.Workload(96, "wide-test", L, "gaussian", 8, 0, 8, fmt)
    prior = [1, 130, 777]
    oc, dc = _prefilled_caches(wl, fmt, prior, max(prior) + 1)
    X = gen.decode_activations(wl, 0, batch=len(prior))
    Qo, Qd = _append_new_rows(ol, dl, oc, dc, X, 1)
    ref = O.attention_reference(ol, oc, Qo[:, None, :], 1)[:, 0, :]
    H.say(f"decode wide heads fmt={fmt} r={r}")
    out = H.host(H.decode_attention(dl, dc, Qd, B.QSVD_ATTN_AUTO))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info
    assert np.array_equal(H.host(dc.data).view(np.uint8), oc.data.view(np.uint8))


@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I4], ids=["f16", "i4"])
def test_decode_rank_3072_and_2048(fmt):
    """The widest ranks of the 13B-shaped stack: r = 3072 with 40 heads (three
    128-column units per wave) and r = 2048 with 32 heads (more than a 32-head
    block's registers hold, so the 16-head variant also serves <= 32 heads)."""
    for heads, kv, r in ((40, 40, 3072), (32, 32, 2048)):
        L = configs.LayerShape(d=256, n_q_heads=heads, n_kv_heads=kv, head_dim=128, r=r)
        ol, dl = _random_factor_layer(L, 5000 + r)
        wl = configs.Workload(96, "wide-test", L, "gaussian", 8, 0, 8, fmt)
        prior = [600, 64]
        oc, dc = _prefilled_caches(wl, fmt, prior, max(prior) + 1)
        X = gen.decode_activations(wl, 1, batch=len(prior))
        Qo, Qd = _append_new_rows(ol, dl, oc, dc, X, 1)
        ref = O.attention_reference(ol, oc, Qo[:, None, :], 1)[:, 0, :]
        H.say(f"decode heads={heads} r={r} fmt={fmt}")
        out = H.host(H.decode_attention(dl, dc, Qd, B.QSVD_ATTN_AUTO))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (heads, r, info)


def test_prefill_attention_wide_int4(fmt=O.CACHE_I4):
    """q_len = 6 causal queries per sequence through the 16-head variant:
    40 heads, r = 1664, int4 cache, prior lengths 0 / 200."""
    L = configs.LayerShape(d=256, n_q_heads=40, n_kv_heads=40, head_dim=128, r=1664)
    ol, dl = _random_factor_layer(L, 6664)
    wl = configs.Workload(96, "wide-test", L, "gaussian", 8, 0, 8, fmt)
    prior, q_len = [0, 200], 6
    oc, dc = _prefilled_caches(wl, fmt, prior, max(prior) + q_len)
    X = gen.decode_activations(wl, 2, batch=len(prior) * q_len)
    Qo, Qd = _append_new_rows(ol, dl, oc, dc, X, q_len)
    nq = L.n_q_heads * L.head_dim
    ref = O.attention_reference(ol, oc, Qo.reshape(len(prior), q_len, nq), q_len)
    H.say("prefill attention wide int4 q_len=6")
    out = H.host(H.decode_attention(dl, dc, Qd.reshape(len(prior), q_len, nq), B.QSVD_ATTN_AUTO, q_len=q_len))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


def test_decode_gqa_int4_cache_ragged(gqa):
    """Int4 latent cache (4-bit per-token codes of C with fp32 scales, two codes
    per byte): ragged prior lengths 3 / 50 / 97 of synthetic rows, then 3 decode
    steps whose new rows are the device's 4-bit quantization of the projected C;
    grouped queries (8 over 2), absorbed form."""
    L, ol, dl = gqa
    prior, batch = [3, 50, 97], 3
    cap = max(prior) + 3
    wl = configs.Workload(95, "gqa-test", L, "gaussian", 8, 0, 8, configs.CACHE_I4)
    rows = gen.latent_rows(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_I4, batch, cap, L.r)
    data = np.zeros((batch, cap, L.r // 2), np.uint8)
    scale = np.zeros((batch, cap), np.float32)
    for b, n in enumerate(prior):
        codes, sc = O.quantize_act(rows[b, :n], 4)
        oc.append(b, None, codes, sc)
        data[b, :n], scale[b, :n] = O.pack_int4(codes), sc
    dc = B.DeviceCache(B.QSVD_CACHE_I4, batch, cap, L.r, prior)
    dc.data.copy_(H.dev(data))
    dc.scale.copy_(H.dev(scale))
    torch = H.torch()
    for t in range(3):
        xt = gen.decode_activations(wl, t, batch=batch)
        proj = O.prefill(ol, xt, 8)
        q4, s4 = O.quantize_act(proj["C_h"], 4)
        for b in range(batch):
            oc.append(b, None, q4[b:b + 1], s4[b:b + 1])
        ref = O.attention_reference(ol, oc, proj["Q"][:, None, :], 1)[:, 0, :]
        H.say(f"decode gqa int4 cache step={t}")
        p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
        cq4 = torch.empty((batch, L.r // 2), dtype=torch.uint8, device="cuda")
        sc4 = torch.empty((batch,), dtype=torch.float32, device="cuda")
        B.check(B.qsvd_quantize_act(B.ptr(p.c_h), batch, L.r, L.r, 4, 1.0, B.ptr(cq4), B.ptr(sc4),
                                    B.stream_handle()))
        H.append(dc, cq=cq4, sc=sc4, n_new=1)
        out = H.host(H.decode_attention(dl, dc, p.q, B.QSVD_ATTN_AUTO))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (t, info)
    assert np.array_equal(H.host(dc.data), oc.data)
    assert np.array_equal(H.host(dc.scale).view(np.uint32), oc.scale.view(np.uint32))


# ------------------------------------------------------------------ rotary position embedding

# Rotary layers: ABSORBED rebuilds and turns K^ for the scores and keeps the
# value side in latent space; RECONSTRUCT rebuilds K^ and V^.
ROPE_MODES = [B.QSVD_ATTN_ABSORBED, B.QSVD_ATTN_RECONSTRUCT]
ROPE_MODE_IDS = ["latent_v", "rebuild_kv"]


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
def test_decode_rope_tiny_end_to_end(tiny, mode):
    """Tiny layer with rotary embeddings: 64 prefill tokens into an fp16 latent
    cache, then 8 decode steps of projection, append and rotary attention (the
    rebuilt K rows and the query turned at their positions), each against the
    oracle's plain definition with the same base."""
    wl, ol, dl = tiny
    theta = 10000.0
    X = gen.prefill_activations(wl)
    oc = O.LatentCache(O.CACHE_F16, 1, 64 + 8, wl.layer.r)
    O.cache_append_prefill(oc, O.prefill(ol, X, 8), [64])
    dc = B.DeviceCache(B.QSVD_CACHE_F16, 1, 64 + 8, wl.layer.r, [0])
    pre = H.Prefill(dl, 64, mask=0, debug=False).run(H.dev(X))
    H.append(dc, pre.c_h, n_new=64)
    for t in range(8):
        xt = gen.decode_activations(wl, t)
        proj = O.decode_step(ol, oc, xt, 8)
        ref = O.attention_reference(ol, oc, proj["Q"][:, None, :], 1, rope_theta=theta)[:, 0, :]
        H.say(f"decode rope tiny step={t} mode={mode}")
        p = H.Prefill(dl, 1, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
        H.append(dc, p.c_h, n_new=1)
        out = H.host(H.decode_attention(dl, dc, p.q, mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (t, info)
        # the rotation changed the result: it is not the unrotated attention
        assert not H.close_enough(out, proj["out"], max_abs=1e-3, rel_l2=1e-3)[0]


def _gqa_cache(L, fmt, lengths, cap, codes_bits=8):
    """Ragged int8 or int4 latent cache of the small GQA layer (rows past each
    length hold the same synthetic distribution)."""
    wl = configs.Workload(95, "gqa-test", L, "gaussian", 8, 0, 8, fmt)
    batch = len(lengths)
    oc = O.LatentCache(fmt, batch, cap, L.r)
    dc = B.DeviceCache(fmt, batch, cap, L.r, lengths)
    if fmt == O.CACHE_I8:
        codes, scales = gen.latent_codes(wl, batch, cap)
        for b, n in enumerate(lengths):
            oc.append(b, None, codes[b, :n], scales[b, :n])
        dc.data.copy_(H.dev(codes))
        dc.scale.copy_(H.dev(scales))
    else:
        rows = gen.latent_rows(wl, batch, cap)
        data = np.zeros((batch, cap, L.r // 2), np.uint8)
        scale = np.zeros((batch, cap), np.float32)
        for b in range(batch):
            codes, sc = O.quantize_act(rows[b], 4)
            data[b], scale[b] = O.pack_int4(codes), sc
            oc.append(b, None, codes[:lengths[b]], sc[:lengths[b]])
        dc.data.copy_(H.dev(data))
        dc.scale.copy_(H.dev(scale))
    return wl, oc, dc


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
@pytest.mark.parametrize("theta", [1.0e4, 1.0e6], ids=["base1e4", "base1e6"])
def test_decode_rope_gqa_int8_ragged(gqa, theta, mode):
    """Grouped queries (8 over 2) over an int8 latent cache with ragged lengths
    1 / 45 / 130, 3 decode steps of rotary attention (the int8 rows rebuilt on
    the int8 matrix cores, then rotated)."""
    L, ol, dl = gqa
    wl, oc, dc = _gqa_cache(L, O.CACHE_I8, [1, 45, 130], 140)
    batch = 3
    for t in range(3):
        xt = gen.decode_activations(wl, t, batch=batch)
        proj = O.decode_step(ol, oc, xt, 8)
        ref = O.attention_reference(ol, oc, proj["Q"][:, None, :], 1, rope_theta=theta)[:, 0, :]
        H.say(f"decode rope gqa int8 step={t} theta={theta} mode={mode}")
        p = H.Prefill(dl, batch, mask=B.QSVD_OUT_Q, debug=False).run(H.dev(xt))
        H.append(dc, cq=p.cq, sc=p.sc, n_new=1)
        out = H.host(H.decode_attention(dl, dc, p.q, mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (t, info)


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
def test_decode_rope_and_reconstruct_gqa_int4_cache(gqa, mode):
    """Int4 latent cache (ragged 3 / 50 / 97): the rows rebuilt on the 4-bit
    activation products, attended without (RECONSTRUCT only) and with rotary
    embeddings."""
    L, ol, dl = gqa
    wl, oc, dc = _gqa_cache(L, O.CACHE_I4, [3, 50, 97], 100)
    g = np.random.default_rng(44)
    q = (g.standard_normal((3, L.n_q_heads * L.head_dim)) * 8.0).astype(np.float16)
    for theta in ((None, 1.0e4) if mode == B.QSVD_ATTN_RECONSTRUCT else (1.0e4,)):
        H.say(f"decode gqa int4 cache theta={theta} mode={mode}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=theta)[:, 0, :]
        out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (theta, info)


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
def test_decode_reconstruct_and_rope_qwen_w4_int8_cache(qwen, mode):
    """Qwen2-VL-7B-shaped layer (28 over 4 heads, r=1024, int4 weights in groups
    of 128) over an int8 latent cache with ragged lengths 7 / 300 / 1029: the
    rows rebuilt by the int4-weight product, attended without (RECONSTRUCT
    only) and with rotary embeddings (base 1e6)."""
    wl, ol, dl = qwen
    L = wl.layer
    lengths = [7, 300, 1029]
    batch, cap = 3, 1040
    codes, scales = gen.latent_codes(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_I8, batch, cap, L.r)
    for b, n in enumerate(lengths):
        oc.append(b, None, codes[b, :n], scales[b, :n])
    dc = B.DeviceCache(B.QSVD_CACHE_I8, batch, cap, L.r, lengths)
    dc.data.copy_(H.dev(codes))
    dc.scale.copy_(H.dev(scales))
    g = np.random.default_rng(2024)
    q = (g.standard_normal((batch, L.n_q_heads * L.head_dim)) * 2.0).astype(np.float16)
    q_dev = H.dev(q)
    for theta in ((None, 1.0e6) if mode == B.QSVD_ATTN_RECONSTRUCT else (1.0e6,)):
        H.say(f"decode qwen int8 cache theta={theta} mode={mode}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=theta)[:, 0, :]
        out = H.host(H.decode_attention(dl, dc, q_dev, mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (theta, info)


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
def test_decode_rope_long_positions(gqa, mode):
    """Positions up to the full rebuild's largest capacity (16384): one
    sequence filled to capacity and one to 9001 tokens of an int8 cache, a
    random query at the last position; the angles reach 16383 rad and are
    reduced in fp64 before the fp32 sine and cosine."""
    L, ol, dl = gqa
    wl, oc, dc = _gqa_cache(L, O.CACHE_I8, [16384, 9001], 16384)
    g = np.random.default_rng(16384)
    # queries large enough for a peaked softmax, so that a wrong angle moves the output
    q = (g.standard_normal((2, L.n_q_heads * L.head_dim)) * 20.0).astype(np.float16)
    for theta in (1.0e4, 5.0e5):
        H.say(f"decode rope long positions theta={theta} mode={mode}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=theta)[:, 0, :]
        out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (theta, info)


def test_decode_rope_latent_v_llava7b_width(llava):
    """LLaVA-1.5-7B-shaped layer (32 heads x 128, r=1536) over an fp16 latent
    cache with ragged lengths 1 / 290 / 1000: the latent-value rotary form
    (fp16 rows rebuilt on the fp16 matrix cores, one workgroup per 32 heads
    and chunk for the value side) against the oracle."""
    wl, ol, dl = llava
    L = wl.layer
    lengths = [1, 290, 1000]
    batch, cap = 3, 1008
    rows = gen.latent_rows(wl, batch, cap)
    oc = O.LatentCache(O.CACHE_F16, batch, cap, L.r)
    for b, n in enumerate(lengths):
        oc.append(b, rows[b, :n])
    dc = B.DeviceCache(B.QSVD_CACHE_F16, batch, cap, L.r, lengths)
    dc.data.copy_(H.dev(oc.data))
    g = np.random.default_rng(7)
    q = (g.standard_normal((batch, L.n_q_heads * L.head_dim)) * 2.0).astype(np.float16)
    for theta in (1.0e4,):
        H.say(f"decode rope llava7b width theta={theta}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=theta)[:, 0, :]
        for mode in ROPE_MODES:
            out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=theta))
            ok, info = H.close_enough(out, ref)
            H.say(f"  mode={mode} max-abs, rel-L2, rms = {info}")
            assert ok, (mode, info)
            again = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=theta))
            assert np.array_equal(out.view(np.uint16), again.view(np.uint16)), (mode, "not deterministic")


@pytest.mark.parametrize("shape", [(12, 4, 96), (32, 4, 32), (16, 16, 64), (32, 8, 128)],
                         ids=["g3_dh96", "g8_dh32", "mha_dh64", "g4_dh128"])
@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I8, O.CACHE_I4], ids=["f16", "i8", "i4"])
def test_decode_rope_head_dims(shape, fmt):
    """Rotary decode at the other head dimensions (96, 32, 64: 6, 2 and 4
    16-byte runs per half row) and group sizes on both sides of the MFMA /
    fp32 score split (3, 8, 1 and 4 query heads per key/value head; 32 over 8
    at dh = 128 stages the most query rows per workgroup), r = 512
    (64 latent columns per wave in the value half), every cache format,
    ragged lengths 2 / 77 / 300; both forms against the oracle."""
    Hq, Hkv, dh = shape
    L = configs.LayerShape(d=512, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=dh, r=512)
    ol, dl = _random_factor_layer(L, 900 + dh + Hq)
    wl = configs.Workload(96, "rope-dims", L, "gaussian", 8, 0, 8, fmt)
    oc, dc = _prefilled_caches(wl, fmt, [2, 77, 300], 304)
    g = np.random.default_rng(dh * 7 + Hq)
    q = (g.standard_normal((3, Hq * dh)) * 4.0).astype(np.float16)
    ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=1.0e4)[:, 0, :]
    for mode in ROPE_MODES:
        H.say(f"decode rope dims Hq={Hq} Hkv={Hkv} dh={dh} fmt={fmt} mode={mode}")
        out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=1.0e4))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (mode, info)


@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I8], ids=["f16", "i8"])
def test_decode_rope_latent_short_lengths(fmt):
    """The rotary latent-value form when the cached lengths are short against
    the capacity (3 / 17 / 40 of 304), so the key rebuild runs one product per
    sequence over its own rows (the scores come from the products' epilogue
    for these caches); GQA 4 query heads per key/value head at dh 128 and MHA
    at dh 64, against the oracle, run twice bit-identically."""
    for shape in ((32, 8, 128), (16, 16, 64)):
        Hq, Hkv, dh = shape
        L = configs.LayerShape(d=512, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=dh, r=512)
        ol, dl = _random_factor_layer(L, 1300 + dh + Hq)
        wl = configs.Workload(97, "rope-short", L, "gaussian", 8, 0, 8, fmt)
        oc, dc = _prefilled_caches(wl, fmt, [3, 17, 40], 304)
        g = np.random.default_rng(dh * 11 + Hq)
        q = (g.standard_normal((3, Hq * dh)) * 4.0).astype(np.float16)
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=1.0e4)[:, 0, :]
        H.say(f"decode rope latent short lengths Hq={Hq} Hkv={Hkv} dh={dh} fmt={fmt}")
        out = H.host(H.decode_attention(dl, dc, H.dev(q), B.QSVD_ATTN_ABSORBED, rope_theta=1.0e4))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (shape, info)
        again = H.host(H.decode_attention(dl, dc, H.dev(q), B.QSVD_ATTN_ABSORBED, rope_theta=1.0e4))
        assert np.array_equal(out.view(np.uint16), again.view(np.uint16)), (shape, "not deterministic")


def _check_qlen_block(out, ref, lengths, q_len):
    """Rows with a visible position against the oracle; rows whose position
    precedes the cache (a sequence shorter than the query block) are zeros."""
    for b, n in enumerate(lengths):
        for i in range(q_len):
            if n - q_len + i < 0:
                assert not np.any(out[b, i].astype(np.float32)), (b, i)
    keep = [(b, i) for b, n in enumerate(lengths) for i in range(q_len) if n - q_len + i >= 0]
    got = np.stack([out[b, i] for b, i in keep])
    want = np.stack([ref[b, i] for b, i in keep])
    ok, info = H.close_enough(got, want)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


@pytest.mark.parametrize("theta", [None, 1.0e4], ids=["plain", "rope"])
@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I8, O.CACHE_I4], ids=["f16", "i8", "i4"])
def test_decode_reconstruct_qlen_block(gqa, fmt, theta):
    """Several queries per sequence in the full-rebuild form (grouped heads
    8/2, dh 64): the last 5 positions of ragged caches 3 / 45 / 130 (the
    first sequence shorter than the block: its first two rows see nothing
    and are zeros), causal, with and without rotary embeddings (the rotary
    latent-value form takes one query, so AUTO rebuilds here), against the
    oracle."""
    L, ol, dl = gqa
    lengths, q_len = [3, 45, 130], 5
    wl = configs.Workload(99, "qlen-block", L, "gaussian", 8, 0, 8, fmt)
    oc, dc = _prefilled_caches(wl, fmt, lengths, 136)
    g = np.random.default_rng(55)
    q = (g.standard_normal((3, q_len, L.n_q_heads * L.head_dim)) * 4.0).astype(np.float16)
    ref = np.zeros(q.shape, np.float64)
    for b, n in enumerate(lengths):
        k = min(q_len, n)
        ref[b:b + 1, q_len - k:] = O.attention_reference(ol, oc, q.astype(np.float64)[:, q_len - k:], q_len=k,
                                                         batches=[b], rope_theta=theta)[b:b + 1]
    modes = [B.QSVD_ATTN_RECONSTRUCT] + ([B.QSVD_ATTN_AUTO] if theta else [])
    for mode in modes:
        H.say(f"decode q_len block fmt={fmt} theta={theta} mode={mode}")
        out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, q_len=q_len, rope_theta=theta))
        _check_qlen_block(out.reshape(q.shape), ref, lengths, q_len)


def test_decode_rope_qlen_llava7b_chunk(llava):
    """A 64-query chunk continuing two LLaVA-7B-shaped sequences (32 heads x
    128, r = 1536, fp16 cache of 200 and 1000 tokens) with rotary embeddings
    in the full-rebuild form, against the oracle; the plain form of the same
    block against the absorbed form's result."""
    wl, ol, dl = llava
    L = wl.layer
    lengths, q_len, cap = [200, 1000], 64, 1008
    rows = gen.latent_rows(wl, 2, cap)
    oc = O.LatentCache(O.CACHE_F16, 2, cap, L.r)
    for b, n in enumerate(lengths):
        oc.append(b, rows[b, :n])
    dc = B.DeviceCache(B.QSVD_CACHE_F16, 2, cap, L.r, lengths)
    dc.data.copy_(H.dev(oc.data))
    g = np.random.default_rng(64)
    q = (g.standard_normal((2, q_len, L.n_q_heads * L.head_dim)) * 2.0).astype(np.float16)
    q_dev = H.dev(q)
    H.say("decode rope q_len 64 llava7b")
    ref = O.attention_reference(ol, oc, q.astype(np.float64), q_len=q_len, rope_theta=1.0e4)
    out = H.host(H.decode_attention(dl, dc, q_dev, B.QSVD_ATTN_RECONSTRUCT, q_len=q_len, rope_theta=1.0e4))
    _check_qlen_block(out.reshape(q.shape), ref, lengths, q_len)
    again = H.host(H.decode_attention(dl, dc, q_dev, B.QSVD_ATTN_RECONSTRUCT, q_len=q_len, rope_theta=1.0e4))
    assert np.array_equal(out.view(np.uint16), again.view(np.uint16)), "not deterministic"
    H.say("decode plain q_len 64 llava7b: rebuild vs absorbed")
    rec = H.host(H.decode_attention(dl, dc, q_dev, B.QSVD_ATTN_RECONSTRUCT, q_len=q_len)).reshape(q.shape)
    ab = H.host(H.decode_attention(dl, dc, q_dev, B.QSVD_ATTN_ABSORBED, q_len=q_len)).reshape(q.shape)
    want = O.attention_reference(ol, oc, q.astype(np.float64), q_len=q_len)
    _check_qlen_block(rec, want, lengths, q_len)
    _check_qlen_block(ab, want, lengths, q_len)


@pytest.mark.parametrize("shape,r", [((40, 40, 128), 1024), ((40, 8, 64), 512), ((64, 64, 64), 512)],
                         ids=["mha40_dh128", "g5_40_dh64", "mha64_dh64"])
@pytest.mark.parametrize("fmt", [O.CACHE_F16, O.CACHE_I8, O.CACHE_I4], ids=["f16", "i8", "i4"])
def test_decode_reconstruct_wide_heads(shape, r, fmt):
    """More than 32 query heads in the full-rebuild form, whose partials go
    out in blocks of 32 heads: 40 heads x 128 (the 13B-shaped layer's heads),
    40 over 8 (a group of five straddles heads 30-34, across the blocks) and
    the 64-head maximum; ragged lengths 3 / 130 / 257 of every cache format,
    with rotary embeddings (AUTO also takes this form for them) and without,
    against the oracle."""
    Hq, Hkv, dh = shape
    L = configs.LayerShape(d=512, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=dh, r=r)
    ol, dl = _random_factor_layer(L, 1300 + Hq + Hkv + dh)
    wl = configs.Workload(97, "wide-heads", L, "gaussian", 8, 0, 8, fmt)
    oc, dc = _prefilled_caches(wl, fmt, [3, 130, 257], 264)
    g = np.random.default_rng(Hq * 11 + Hkv + dh)
    q = (g.standard_normal((3, Hq * dh)) * 4.0).astype(np.float16)
    q_dev = H.dev(q)
    for theta, mode in ((1.0e4, B.QSVD_ATTN_RECONSTRUCT), (1.0e4, B.QSVD_ATTN_AUTO), (None, B.QSVD_ATTN_RECONSTRUCT)):
        H.say(f"decode wide heads Hq={Hq} Hkv={Hkv} dh={dh} r={r} fmt={fmt} theta={theta} mode={mode}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=theta)[:, 0, :]
        out = H.host(H.decode_attention(dl, dc, q_dev, mode, rope_theta=theta))
        ok, info = H.close_enough(out, ref)
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (theta, mode, info)
        again = H.host(H.decode_attention(dl, dc, q_dev, mode, rope_theta=theta))
        assert np.array_equal(out.view(np.uint16), again.view(np.uint16)), (theta, mode, "not deterministic")


def test_decode_rope_13b_shape_full_rebuild():
    """The 13B-shaped layer at its size (40 heads x 128, r = 2048, int4
    weights in groups of 128) over an int4 latent cache of 8 sequences with
    the workload's prompt and decode lengths (704 tokens and more), rotary
    embeddings (base 1e4) in the full-rebuild form, every sequence against
    the oracle."""
    L = configs.LayerShape(d=5120, n_q_heads=40, n_kv_heads=40, head_dim=128, r=2048)
    ol, dl = _random_factor_layer(L, 1340, w_bits=4, w_group=128)
    wl = configs.Workload(98, "13b-rope", L, "gaussian", 4, 128, 4, O.CACHE_I4)
    lengths = [704, 705, 720, 740, 760, 800, 830, 832]
    oc, dc = _prefilled_caches(wl, O.CACHE_I4, lengths, 832)
    g = np.random.default_rng(5120)
    q = (g.standard_normal((8, 40 * 128)) * 2.0).astype(np.float16)
    H.say("decode rope 13b shape full rebuild")
    ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, rope_theta=1.0e4)[:, 0, :]
    out = H.host(H.decode_attention(dl, dc, H.dev(q), B.QSVD_ATTN_AUTO, rope_theta=1.0e4))
    ok, info = H.close_enough(out, ref)
    H.say(f"  max-abs, rel-L2, rms = {info}")
    assert ok, info


@pytest.mark.parametrize("mode", ROPE_MODES, ids=ROPE_MODE_IDS)
def test_decode_rope_empty_sequence(gqa, mode):
    """A sequence with nothing cached (length 0) beside ragged ones (33, 70):
    its output is zeros (no visible position), the others match the oracle;
    with and without rotary embeddings (the latter in the reconstruct form)."""
    L, ol, dl = gqa
    wl, oc, dc = _gqa_cache(L, O.CACHE_I8, [0, 33, 70], 72)
    g = np.random.default_rng(3)
    q = (g.standard_normal((3, L.n_q_heads * L.head_dim)) * 4.0).astype(np.float16)
    for theta in ((None, 1.0e4) if mode == B.QSVD_ATTN_RECONSTRUCT else (1.0e4,)):
        H.say(f"decode empty sequence theta={theta} mode={mode}")
        ref = O.attention_reference(ol, oc, q.astype(np.float64)[:, None, :], 1, batches=[1, 2],
                                    rope_theta=theta)[:, 0, :]
        out = H.host(H.decode_attention(dl, dc, H.dev(q), mode, rope_theta=theta))
        assert np.array_equal(out[0].view(np.uint16), np.zeros_like(out[0]).view(np.uint16))
        ok, info = H.close_enough(out[1:], ref[1:])
        H.say(f"  max-abs, rel-L2, rms = {info}")
        assert ok, (theta, info)
