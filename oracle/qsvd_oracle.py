"""QSVD oracle: a plain, slow, CPU-only definition of the latent-QKV hot path.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code
with the HIP library or its Python binding; the two meet only in the seeded
inputs of :mod:`workloads`.

What it computes (paper: "QSVD", arXiv 2510.16292):

* Offline stage -- joint SVD of the concatenated [W_q | W_k | W_v] (Section 3.1,
  Eq. 2), truncation to rank r, the beta split of Sigma between the down- and
  up-projection (Eq. 3-4), optional orthogonal rotations folded into the
  factors (Eq. 11), and round-to-nearest symmetric weight quantization
  (Section 4, experimental setup).
* Online stage -- per-token symmetric activation quantization (Section 4),
  the quantized down-projection C = Q(X) Q(W^d) (Eq. 12), the latent cache of
  C only (Section 3.1), the quantized up-projection Y' = Q(C) Q(W^u) (Eq. 11),
  and attention whose keys and values are recomputed from the cached latent,
  K = C W^u_k and V = C W^u_v (Eq. 5), for the current query.

Precision: fp64 for real arithmetic, exact integers for the quantized
products, and fp32/fp16 exactly where the stored formats require it (scales
are fp32, the latent and the projections are stored as fp16).  Every fp32
operation is one numpy float32 operation (IEEE round-to-nearest-even), so
the order written here is the order that is meant.

Readings of points the paper leaves open are listed in the repository's
design notes and repeated at each function.  Parity unpinned: nothing; every
function is checked by the CPU pin tests (closed forms, invariants, special
cases, brute force on tiny inputs).
"""
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

F32 = np.float32

CACHE_F16, CACHE_I8, CACHE_I4 = 0, 1, 2


def qmax(bits: int) -> int:
    """Largest code of a symmetric signed grid: 127 for 8 bits, 7 for 4 bits.

    Reading: "symmetric" quantization (Section 4) uses [-Qm, Qm]; -2^(b-1) is
    never produced.
    """
    return (1 << (bits - 1)) - 1


# --------------------------------------------------------------------------
# Offline stage
# --------------------------------------------------------------------------

def joint_svd(W: np.ndarray):
    """Thin SVD of the concatenated weight W = [W_q | W_k | W_v] (d x N), Eq. 2.

    Returns (U [d,n], sigma [n] descending, Vt [n,N]) with n = min(d, N).
    Singular vectors are only defined up to sign; the sign is fixed so that the
    entry of largest magnitude in each right singular vector is positive.
    """
    U, s, Vt = np.linalg.svd(np.asarray(W, dtype=np.float64), full_matrices=False)
    idx = np.argmax(np.abs(Vt), axis=1)
    sgn = np.sign(Vt[np.arange(Vt.shape[0]), idx])
    sgn[sgn == 0] = 1.0
    return U * sgn[None, :], s, Vt * sgn[:, None]


def split_beta(U_r: np.ndarray, sigma_r: np.ndarray, Vt_r: np.ndarray, beta: float):
    """Eq. 3: W^d = U_r Sigma_r^beta (d x r), W^u = Sigma_r^(1-beta) V_r^T (r x N)."""
    A = U_r * (sigma_r ** beta)[None, :]
    B = (sigma_r ** (1.0 - beta))[:, None] * Vt_r
    return A, B


def factors_from_weight(W: np.ndarray, r: int, beta: float):
    """Truncated joint SVD of W followed by the beta split (Eq. 2-4)."""
    U, s, Vt = joint_svd(W)
    return split_beta(U[:, :r], s[:r], Vt[:r, :], beta)


# --------------------------------------------------------------------------
# Offline rank allocation and beta (Section 3.2, Eq. 6-10, Appendix A; Eq. 14)
# --------------------------------------------------------------------------

def importance_naive(U: np.ndarray, s: np.ndarray, Vt: np.ndarray, grads, S_inv: np.ndarray = None) -> np.ndarray:
    """Importance score by its definition (Eq. 9): for every singular value,
    Delta W_i = sigma_i u_i v_i^T (Eq. 6), taken back to the weight space through
    S^{-1} when the SVD was of the whitened W S (Appendix A), and
    I_i = mean_n <Delta W_i, G^(n)>_F^2 with the first-order loss change of
    Eq. 8.  Builds every Delta W_i explicitly: tiny sizes only."""
    n = s.size
    out = np.zeros(n)
    for i in range(n):
        dW = s[i] * np.outer(U[:, i], Vt[i, :])
        if S_inv is not None:
            dW = dW @ S_inv
        out[i] = np.mean([np.sum(dW * G) ** 2 for G in grads])
    return out


def importance_scores(U: np.ndarray, s: np.ndarray, Vt: np.ndarray, grads, S_inv: np.ndarray = None) -> np.ndarray:
    """Eq. 10: I_i = mean_n sigma_i^2 [U^T G^(n) V]_(i,i)^2, or with whitening
    mean_n sigma_i^2 [U^T G^(n) S^{-T} V]_(i,i)^2 (Appendix A)."""
    V = Vt.T
    acc = np.zeros(s.size)
    for G in grads:
        Gw = G if S_inv is None else G @ S_inv.T
        acc += np.diag(U.T @ Gw @ V) ** 2
    return s ** 2 * acc / len(grads)


def allocate_ranks(scores, budget: int):
    """Global ranking across layers (Section 3.2): all singular values of all
    layers sorted by importance, the top `budget` kept.  Returns, per layer,
    the sorted indices of its kept singular values.  Reading: ties go to the
    lower (layer, index) pair."""
    entries = [(-float(v), l, i) for l, sc in enumerate(scores) for i, v in enumerate(sc)]
    entries.sort()
    kept = [[] for _ in scores]
    for _, l, i in entries[:budget]:
        kept[l].append(i)
    return [np.array(sorted(k), dtype=np.int64) for k in kept]


def beta_objective(A: np.ndarray, B: np.ndarray, X: np.ndarray, layer_fn) -> float:
    """Eq. 14's per-layer term: the sum over calibration rows d of
    ||Y_d - Y'_d||^2 (squared Euclidean norm, every output column), with
    Y = X W^d W^u in fp64 and Y' = `layer_fn(A, B, X)`, the quantized
    projection (the concatenated fp16 Q | K | V).

    Reading: the paper scores the self-attention block's output; here the
    score is taken on the block's quantized projection (the part of the block
    that beta changes), not on the attention that follows it."""
    Y = np.asarray(X, dtype=np.float64) @ A @ B
    Yq = np.asarray(layer_fn(A, B, X), dtype=np.float64)
    assert Yq.shape == Y.shape
    return float(np.sum((Y - Yq) ** 2))


def beta_search(U_r: np.ndarray, s_r: np.ndarray, Vt_r: np.ndarray, X: np.ndarray, betas, layer_fn):
    """Line search of Eq. 14 over a grid of beta: returns (best beta, the
    objective at every grid point).  Reading: the first minimum in grid order."""
    vals = []
    for b in betas:
        A, B = split_beta(U_r, s_r, Vt_r, b)
        vals.append(beta_objective(A, B, X, layer_fn))
    return betas[int(np.argmin(vals))], vals


def random_orthogonal(n: int, seed: int) -> np.ndarray:
    """A seeded orthogonal matrix (QR of a Gaussian) for the rotation pins."""
    g = np.random.default_rng(seed)
    q, rr = np.linalg.qr(g.standard_normal((n, n)))
    return q * np.sign(np.diag(rr))[None, :]


def fold_rotations(A: np.ndarray, B: np.ndarray, H1: np.ndarray, H2: np.ndarray):
    """Eq. 11: with orthogonal H1 (d x d) and H2 (r x r) the layer becomes
    Y = (X H1^T)(H1 W^d H2^T)(H2 W^u).  Returns (H1 A H2^T, H2 B)."""
    return H1 @ A @ H2.T, H2 @ B


def hadamard_block(d: int) -> int:
    """Block size of the randomized block Walsh-Hadamard rotation: the largest
    power of two dividing d (reading: the paper asks only for orthogonal
    H1, H2 in the QuaRot/DFRot style, Section 3.3)."""
    return d & -d


def rotation_signs(d: int, seed: int) -> np.ndarray:
    """A seeded +-1 diagonal (int8 [d]) of the randomized rotation."""
    g = np.random.default_rng(seed)
    return np.where(g.integers(0, 2, size=d) == 0, 1, -1).astype(np.int8)


def walsh_hadamard_rows(v: np.ndarray, block: int, dtype=F32) -> np.ndarray:
    """Unnormalized Walsh-Hadamard transform of every length-`block` segment
    of every row, v -> v H_block (Sylvester order), by the radix-2 stages
    h = 1, 2, 4, ..., block/2: (v_i, v_{i+h}) -> (v_i + v_{i+h}, v_i - v_{i+h})
    for every i whose bit h is clear, each sum rounded to `dtype`."""
    out = np.array(v, dtype=dtype, copy=True)
    M, K = out.shape
    assert K % block == 0 and block & (block - 1) == 0
    h = 1
    while h < block:
        w = out.reshape(M, K // (2 * h), 2, h)
        a = w[:, :, 0, :].copy()
        b = w[:, :, 1, :].copy()
        w[:, :, 0, :] = (a + b).astype(dtype)
        w[:, :, 1, :] = (a - b).astype(dtype)
        h *= 2
    return out


def rotation_matrix(signs: np.ndarray, block: int) -> np.ndarray:
    """H1 = blockdiag(H_B, ..., H_B) diag(signs) / sqrt(B) as an explicit fp64
    matrix (H_B the Sylvester Hadamard matrix), for the pins and for folding."""
    d = signs.size
    Hb = walsh_hadamard_rows(np.eye(block), block, np.float64)      # rows of H_B
    H = np.zeros((d, d))
    for k in range(d // block):
        H[k * block:(k + 1) * block, k * block:(k + 1) * block] = Hb
    return H * signs.astype(np.float64)[None, :] / np.sqrt(block)


def rotate_act(x: np.ndarray, signs: np.ndarray, block: int) -> np.ndarray:
    """Online rotation X H1^T of Eq. 11 / Q(X H1^T) of Eq. 12 for
    H1 = blockdiag(H_B) diag(signs) / sqrt(B): in fp32, x_i * s_i (exact), the
    Walsh-Hadamard stages of each block, then one product by fp32(1/sqrt(B))."""
    v = (np.asarray(x).astype(F32) * signs.astype(F32)[None, :]).astype(F32)
    y = walsh_hadamard_rows(v, block, F32)
    c = F32(1.0 / np.sqrt(float(block)))
    return (y * c).astype(F32)


def quantize_act_rotated(x: np.ndarray, signs: np.ndarray, block: int, bits: int, clip: float = 1.0):
    """Q(X H1^T): the rotated rows (fp32) through the per-token quantizer."""
    return quantize_act(rotate_act(x, signs, block), bits, clip)


def quantize_weight(W: np.ndarray, bits: int, group: int = 0, clip: float = 1.0):
    """Round-to-nearest symmetric weight quantization (Section 4 setup).

    ``W`` is (K x Nout) with K the contraction index.  group == 0 gives one
    scale per output column ("per-channel"); group > 0 gives one scale per
    output column and per block of ``group`` consecutive contraction rows.

    Reading: the scale is computed in fp64 as clip * max|w| / Qm and stored as
    fp32; codes are rint(w / s32) in fp64 (ties to even), clamped to
    [-Qm, Qm].  An all-zero column or group gets scale 1.  The learnable
    clipping ratio of the paper is a parameter here (1.0 by default).

    Returns (q int8 [K, Nout], s fp32 [Nout] or [K/group, Nout]).
    """
    W = np.asarray(W, dtype=np.float64)
    K, Nout = W.shape
    Qm = qmax(bits)
    if group == 0:
        amax = np.max(np.abs(W), axis=0)                       # [Nout]
        s = (clip * amax / Qm).astype(F32)
        s[amax == 0] = F32(1.0)
        q = np.rint(W / s.astype(np.float64)[None, :])
    else:
        assert K % group == 0
        G = K // group
        Wg = W.reshape(G, group, Nout)
        amax = np.max(np.abs(Wg), axis=1)                      # [G, Nout]
        s = (clip * amax / Qm).astype(F32)
        s[amax == 0] = F32(1.0)
        q = np.rint(Wg / s.astype(np.float64)[:, None, :]).reshape(K, Nout)
    q = np.clip(q, -Qm, Qm).astype(np.int8)
    return q, s


def dequantize_weight(q: np.ndarray, s: np.ndarray, group: int = 0) -> np.ndarray:
    """fp64 value s * q of a quantized (K x Nout) weight."""
    q = q.astype(np.float64)
    if group == 0:
        return q * s.astype(np.float64)[None, :]
    K, Nout = q.shape
    return (q.reshape(K // group, group, Nout) * s.astype(np.float64)[:, None, :]).reshape(K, Nout)


@dataclass
class Layer:
    """One attention layer after the offline stage.

    Aq [d, r] / sA: quantized down-projection W^d.  Bq [r, N] / sB: quantized
    up-projection [W^u_q | W^u_k | W^u_v].  A, B: the fp64 factors they came from.
    """
    d: int
    r: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    w_bits: int
    w_group: int
    Aq: np.ndarray
    sA: np.ndarray
    Bq: np.ndarray
    sB: np.ndarray
    A: Optional[np.ndarray] = None
    B: Optional[np.ndarray] = None

    @property
    def N(self):
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    def A_hat(self):
        return dequantize_weight(self.Aq, self.sA, self.w_group)

    def B_hat(self):
        return dequantize_weight(self.Bq, self.sB, self.w_group)


def make_layer(A: np.ndarray, B: np.ndarray, n_q_heads: int, n_kv_heads: int, head_dim: int,
               w_bits: int, w_group: int, clip: float = 1.0) -> Layer:
    """Quantize the factors A (d x r, contraction d) and B (r x N, contraction r)."""
    d, r = A.shape
    Aq, sA = quantize_weight(A, w_bits, w_group, clip)
    Bq, sB = quantize_weight(B, w_bits, w_group, clip)
    return Layer(d, r, n_q_heads, n_kv_heads, head_dim, w_bits, w_group, Aq, sA, Bq, sB, A, B)


# --------------------------------------------------------------------------
# Online stage
# --------------------------------------------------------------------------

def quantize_act(x: np.ndarray, bits: int, clip: float = 1.0):
    """Per-token symmetric quantization (Section 4 setup; Q(.) of Eq. 11-12).

    Per row, all in fp32: amax = max|x_i|; a = clip * amax; if a == 0 the row
    gets scale 1 and codes 0; else inv = Qm / a, s = a / Qm and
    q_i = clamp(rint(x_i * inv), -Qm, Qm) with ties to even.

    Returns (q int8 [M, K], s fp32 [M]).
    """
    xf = np.asarray(x).astype(F32)
    M = xf.shape[0]
    Qm = F32(qmax(bits))
    q = np.zeros(xf.shape, dtype=np.int8)
    s = np.ones(M, dtype=F32)
    for m in range(M):
        row = xf[m]
        a = F32(F32(clip) * np.max(np.abs(row))) if row.size else F32(0)
        if a == F32(0):
            continue
        inv = F32(Qm / a)
        s[m] = F32(a / Qm)
        prod = (row * inv).astype(F32)
        q[m] = np.clip(np.rint(prod), -Qm, Qm).astype(np.int8)
    return q, s


def int_matmul(aq: np.ndarray, bq: np.ndarray) -> np.ndarray:
    """Exact integer product of an int8 [M,K] and an int8 [K,N] matrix.

    fp64 BLAS is exact here: every partial sum is an integer below 2^53.
    """
    acc = aq.astype(np.float64) @ bq.astype(np.float64)
    assert np.all(np.abs(acc) < 2.0 ** 31), "int32 accumulator range exceeded"
    return acc.astype(np.int64)


def _scaled(acc: np.ndarray, s_row: np.ndarray, w_scale: np.ndarray, group: int, K: int,
            aq: np.ndarray, wq: np.ndarray) -> np.ndarray:
    """fp32 dequantization of an integer product, in this order:

    per-channel: y = (f32(acc) * s_row) * s_w
    per-group:   S = 0; for g: S = S + f32(acc_g) * s_w[g];  y = S * s_row
    """
    if group == 0:
        y = (acc.astype(F32) * s_row.astype(F32)[:, None]).astype(F32)
        return (y * w_scale.astype(F32)[None, :]).astype(F32)
    G = K // group
    S = np.zeros(acc.shape, dtype=F32)
    for g in range(G):
        acc_g = int_matmul(aq[:, g * group:(g + 1) * group], wq[g * group:(g + 1) * group, :])
        S = (S + (acc_g.astype(F32) * w_scale[g].astype(F32)[None, :]).astype(F32)).astype(F32)
    return (S * s_row.astype(F32)[:, None]).astype(F32)


def to_f16(y32: np.ndarray) -> np.ndarray:
    out = y32.astype(np.float16)
    assert np.all(np.isfinite(out)), "fp16 overflow in a stored result"
    return out


def down_projection(layer: Layer, xq: np.ndarray, sx: np.ndarray):
    """Latent C = Q(X) Q(W^d) (Eq. 12): the shared down-projection, done once
    for Q, K and V (Section 3.1).  Returns (acc int [M, r], C_h fp16 [M, r]).

    Reading: C is materialised once as fp16; the int32 accumulator is dequantized
    in fp32 as (acc * s_x) * s_A (per-group: sum over groups first).
    """
    acc = int_matmul(xq, layer.Aq)
    c32 = _scaled(acc, sx, layer.sA, layer.w_group, layer.d, xq, layer.Aq)
    return acc, to_f16(c32)


def quantize_latent(C_h: np.ndarray, bits: int):
    """Q(C) of Eq. 11: per-token symmetric quantization of the fp16 latent."""
    return quantize_act(C_h, bits, 1.0)


def up_projection(layer: Layer, cq: np.ndarray, sc: np.ndarray):
    """Y' = Q(C) Q(W^u) (Eq. 11): all of Q, K, V from the one latent.

    Returns (acc int [M, N], Q fp16 [M, n_q], K fp16 [M, n_kv], V fp16 [M, n_kv]).
    Columns are [Q heads | K heads | V heads], head h at columns h*head_dim...
    """
    acc = int_matmul(cq, layer.Bq)
    y32 = _scaled(acc, sc, layer.sB, layer.w_group, layer.r, cq, layer.Bq)
    y = to_f16(y32)
    nq = layer.n_q_heads * layer.head_dim
    nkv = layer.n_kv_heads * layer.head_dim
    return acc, y[:, :nq], y[:, nq:nq + nkv], y[:, nq + nkv:]


def prefill(layer: Layer, x: np.ndarray, a_bits: int, clip: float = 1.0) -> Dict[str, np.ndarray]:
    """The projection half of the hot path for a block of tokens."""
    xq, sx = quantize_act(x, a_bits, clip)
    acc_xa, C_h = down_projection(layer, xq, sx)
    cq, sc = quantize_latent(C_h, a_bits)
    acc_cb, Q, K, V = up_projection(layer, cq, sc)
    return dict(xq=xq, sx=sx, acc_xa=acc_xa, C_h=C_h, cq=cq, sc=sc, acc_cb=acc_cb, Q=Q, K=K, V=V)


# --------------------------------------------------------------------------
# Latent cache (Section 3.1: only C is buffered, eta = r L)
# --------------------------------------------------------------------------

def pack_int4(q: np.ndarray) -> np.ndarray:
    """Two's-complement nibbles, element 2i in the low nibble of byte i."""
    q = q.astype(np.int16)
    assert q.shape[-1] % 2 == 0 and np.all(np.abs(q) <= 8)
    lo = q[..., 0::2] & 0xF
    hi = q[..., 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(p: np.ndarray) -> np.ndarray:
    p = p.astype(np.int16)
    lo = p & 0xF
    hi = (p >> 4) & 0xF
    lo = np.where(lo >= 8, lo - 16, lo)
    hi = np.where(hi >= 8, hi - 16, hi)
    out = np.empty(p.shape[:-1] + (p.shape[-1] * 2,), dtype=np.int8)
    out[..., 0::2] = lo
    out[..., 1::2] = hi
    return out


class LatentCache:
    """Per-sequence rows of the latent C, stored as fp16, or as int8/int4 codes
    with one fp32 scale per token.

    Reading: an integer cache stores Q(C) exactly as fed to the up-projection;
    an fp16 cache stores the fp16 latent itself.
    """

    def __init__(self, fmt: int, batch: int, capacity: int, r: int):
        self.fmt, self.batch, self.capacity, self.r = fmt, batch, capacity, r
        if fmt == CACHE_F16:
            self.data = np.zeros((batch, capacity, r), dtype=np.float16)
        elif fmt == CACHE_I8:
            self.data = np.zeros((batch, capacity, r), dtype=np.int8)
        else:
            self.data = np.zeros((batch, capacity, r // 2), dtype=np.uint8)
        self.scale = np.zeros((batch, capacity), dtype=F32) if fmt != CACHE_F16 else None
        self.seq_len = np.zeros(batch, dtype=np.int32)
        self.elements_stored = 0

    def append(self, b: int, C_h: np.ndarray, cq: np.ndarray = None, sc: np.ndarray = None):
        n = C_h.shape[0] if C_h is not None else cq.shape[0]
        t0 = int(self.seq_len[b])
        assert t0 + n <= self.capacity, "latent cache capacity exceeded"
        if self.fmt == CACHE_F16:
            self.data[b, t0:t0 + n] = C_h
        elif self.fmt == CACHE_I8:
            self.data[b, t0:t0 + n] = cq
            self.scale[b, t0:t0 + n] = sc
        else:
            self.data[b, t0:t0 + n] = pack_int4(cq)
            self.scale[b, t0:t0 + n] = sc
        self.seq_len[b] += n
        self.elements_stored += n * self.r

    def rows(self, b: int) -> np.ndarray:
        """fp64 value of the stored latent rows [0, seq_len[b]) of sequence b."""
        L = int(self.seq_len[b])
        if self.fmt == CACHE_F16:
            return self.data[b, :L].astype(np.float64)
        codes = self.data[b, :L] if self.fmt == CACHE_I8 else unpack_int4(self.data[b, :L])
        return codes.astype(np.float64) * self.scale[b, :L].astype(np.float64)[:, None]


# --------------------------------------------------------------------------
# Attention over the latent cache
# --------------------------------------------------------------------------

def kv_group(h: int, n_q_heads: int, n_kv_heads: int) -> int:
    """Query head h reads key/value head floor(h * Hkv / Hq) (grouped-query reading)."""
    return (h * n_kv_heads) // n_q_heads


def _softmax(s: np.ndarray) -> np.ndarray:
    e = np.exp(s - np.max(s, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def rope(x: np.ndarray, positions: np.ndarray, theta: float, dh: int) -> np.ndarray:
    """Rotary position embedding of the head vectors of x [T, heads * dh] at
    the given positions (not in the paper, which has no position encoding;
    the variant for layers that apply it to q and k).  Reading: rotate-half
    pairs (j, j + dh/2) turned by the angle pos * theta^(-2j/dh), in fp64:
    (a, b) -> (a cos - b sin, b cos + a sin)."""
    x = np.asarray(x, dtype=np.float64)
    T, n = x.shape
    half = dh // 2
    inv = theta ** (-2.0 * np.arange(half) / dh)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]      # [T, half]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    for h in range(n // dh):
        a = x[:, h * dh:h * dh + half]
        b = x[:, h * dh + half:(h + 1) * dh]
        out[:, h * dh:h * dh + half] = a * c - b * s
        out[:, h * dh + half:(h + 1) * dh] = b * c + a * s
    return out


def attention_reference(layer: Layer, cache: LatentCache, q: np.ndarray, q_len: int = 1,
                        sm_scale: float = None, batches=None, heads=None, rope_theta: float = None) -> np.ndarray:
    """Plain definition: rebuild K = C W^u_k and V = C W^u_v from the cached
    latent (Eq. 5) and attend with the current queries (Section 3.1).

    q: [B, q_len, Hq*head_dim] (fp16 values).  The queries sit at the last
    q_len positions of each sequence and attend causally to positions
    [0, own position].  Reading: the softmax scale is 1/sqrt(head_dim); the
    latent is used as stored (dequantized), times the dequantized W^u.

    With rope_theta, q and every rebuilt K row are first rotated (:func:`rope`)
    at their positions; then K can no longer be folded into the query, which
    is why only this plain form takes it.

    Returns fp64 [B, q_len, Hq*head_dim] (rows/heads not requested are 0).
    """
    Hq, Hkv, dh = layer.n_q_heads, layer.n_kv_heads, layer.head_dim
    nq, nkv = Hq * dh, Hkv * dh
    sm = 1.0 / np.sqrt(dh) if not sm_scale else sm_scale
    Bh = layer.B_hat()
    Bk, Bv = Bh[:, nq:nq + nkv], Bh[:, nq + nkv:]
    q = np.asarray(q, dtype=np.float64).reshape(q.shape[0], q_len, nq)
    out = np.zeros_like(q)
    batches = range(cache.batch) if batches is None else batches
    heads = range(Hq) if heads is None else heads
    for b in batches:
        C = cache.rows(b)
        L = C.shape[0]
        K = C @ Bk                       # [L, Hkv*dh]
        V = C @ Bv
        qb = q[b]
        if rope_theta:
            K = rope(K, np.arange(L), rope_theta, dh)
            qb = rope(qb, np.arange(L - q_len, L), rope_theta, dh)
        for i in range(q_len):
            pos = L - q_len + i
            for h in heads:
                g = kv_group(h, Hq, Hkv)
                qh = qb[i, h * dh:(h + 1) * dh]
                s = (K[:pos + 1, g * dh:(g + 1) * dh] @ qh) * sm
                p = _softmax(s)
                out[b, i, h * dh:(h + 1) * dh] = p @ V[:pos + 1, g * dh:(g + 1) * dh]
    return out


def attention_absorbed(layer: Layer, cache: LatentCache, q: np.ndarray, q_len: int = 1,
                       sm_scale: float = None) -> np.ndarray:
    """Same attention with W^u_k folded into the query and W^u_v applied after
    the latent-space weighted sum (the latent-attention form the method is
    built on, Section 1 and 2.2).  s_t = (q W^u_k^T) . C_t ; o = (sum_t p_t C_t) W^u_v.
    Used to check :func:`attention_reference`; equal up to fp64 rounding."""
    Hq, Hkv, dh = layer.n_q_heads, layer.n_kv_heads, layer.head_dim
    nq, nkv = Hq * dh, Hkv * dh
    sm = 1.0 / np.sqrt(dh) if not sm_scale else sm_scale
    Bh = layer.B_hat()
    q = np.asarray(q, dtype=np.float64).reshape(q.shape[0], q_len, nq)
    out = np.zeros_like(q)
    for b in range(cache.batch):
        C = cache.rows(b)
        L = C.shape[0]
        for i in range(q_len):
            pos = L - q_len + i
            for h in range(Hq):
                g = kv_group(h, Hq, Hkv)
                Bk = Bh[:, nq + g * dh: nq + (g + 1) * dh]            # [r, dh]
                Bv = Bh[:, nq + nkv + g * dh: nq + nkv + (g + 1) * dh]
                q_lat = Bk @ q[b, i, h * dh:(h + 1) * dh]           # [r]
                p = _softmax((C[:pos + 1] @ q_lat) * sm)
                out[b, i, h * dh:(h + 1) * dh] = (p @ C[:pos + 1]) @ Bv
    return out


def prefill_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, lengths: List[int], n_q_heads: int,
                      n_kv_heads: int, head_dim: int, sm_scale: float = None,
                      rope_theta: float = None) -> np.ndarray:
    """Causal self-attention of a prefill block over its own projections.

    In prefill every token of the prompt has its keys and values at hand: the
    up-projection Y' = Q(C) Q(W^u) (Eq. 11) gives Q, K and V of all tokens at
    once (K = C W^u_k, V = C W^u_v, Eq. 5), and token i of a sequence attends
    to tokens 0..i of the same sequence.  Q [M, Hq*dh], K and V [M, Hkv*dh]
    are token-major with the sequences back to back (`lengths`); query head h
    reads key/value head floor(h * Hkv / Hq); softmax scale 1/sqrt(dh) unless
    given; fp64 throughout.  With rope_theta, the Q and K rows of a sequence
    are first rotated (:func:`rope`) at their positions 0..n-1 within it, as
    the decode form does over the cache.  Returns fp64 [M, Hq*dh]."""
    dh = head_dim
    sm = 1.0 / np.sqrt(dh) if not sm_scale else sm_scale
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    out = np.zeros_like(Q)
    t0 = 0
    for n in lengths:
        if n == 0:                                      # an empty sequence has no query rows
            continue
        Qs, Ks = Q[t0:t0 + n], K[t0:t0 + n]
        if rope_theta:
            Qs = rope(Qs, np.arange(n), rope_theta, dh)
            Ks = rope(Ks, np.arange(n), rope_theta, dh)
        for h in range(n_q_heads):
            g = kv_group(h, n_q_heads, n_kv_heads)
            qh = Qs[:, h * dh:(h + 1) * dh]
            kh = Ks[:, g * dh:(g + 1) * dh]
            vh = V[t0:t0 + n, g * dh:(g + 1) * dh]
            s = (qh @ kh.T) * sm
            s[np.triu_indices(n, 1)] = -np.inf          # query i sees keys 0..i
            out[t0:t0 + n, h * dh:(h + 1) * dh] = _softmax(s) @ vh
        t0 += n
    return out


def cache_snapshot(cache: LatentCache) -> Dict[str, np.ndarray]:
    """Copy of the cache state (rows, scales, lengths) from which a decode can
    resume."""
    snap = dict(data=cache.data.copy(), seq_len=cache.seq_len.copy())
    if cache.scale is not None:
        snap["scale"] = cache.scale.copy()
    return snap


def cache_restore(cache: LatentCache, snap: Dict[str, np.ndarray]):
    """Put a snapshot's state back into a cache of the same shape."""
    assert snap["data"].shape == cache.data.shape
    cache.data[...] = snap["data"]
    cache.seq_len[...] = snap["seq_len"]
    if cache.scale is not None:
        cache.scale[...] = snap["scale"]


def cache_append_prefill(cache: LatentCache, proj: Dict[str, np.ndarray], lengths: List[int]):
    """Append the latent rows of a prefill block (token-major, sequences back to
    back with the given lengths) to the cache."""
    t = 0
    for b, n in enumerate(lengths):
        cache.append(b, proj["C_h"][t:t + n], proj["cq"][t:t + n], proj["sc"][t:t + n])
        t += n


def decode_step(layer: Layer, cache: LatentCache, x_t: np.ndarray, a_bits: int,
                clip: float = 1.0, reference: bool = True) -> Dict[str, np.ndarray]:
    """One generated token per sequence (Section 3.1, decoding with l = 1):
    project the new token, append its latent, then attend with its query over
    every cached position including itself (append-then-attend reading)."""
    proj = prefill(layer, x_t, a_bits, clip)
    for b in range(x_t.shape[0]):
        cache.append(b, proj["C_h"][b:b + 1], proj["cq"][b:b + 1], proj["sc"][b:b + 1])
    q = proj["Q"][:, None, :]
    attn = attention_reference if reference else attention_absorbed
    proj["out"] = attn(layer, cache, q, 1)[:, 0, :]
    return proj


# --------------------------------------------------------------------------
# Hardware-cost model (Section 3.1) and the ratios R1, R2 (Eq. 15)
# --------------------------------------------------------------------------

class MacCounter:
    """Counts the multiply-accumulates the oracle's projections perform."""

    def __init__(self):
        self.macs = 0

    def matmul(self, a: np.ndarray, b: np.ndarray) -> np.ndarray:
        self.macs += a.shape[0] * a.shape[1] * b.shape[1]
        return a @ b


def projection_macs(layer: Layer, x: np.ndarray) -> int:
    """MACs of the fp64 projection X W^d then C [W^u_q | W^u_k | W^u_v],
    counted while computing it."""
    c = MacCounter()
    C = c.matmul(np.asarray(x, dtype=np.float64), layer.A)
    c.matmul(C, layer.B)
    return c.macs


def cost_ratios(r: int, E: int, w_bits: int = 16, kv_bits: int = 16):
    """R1 = alpha_qsvd / alpha_fp = 4 r E / 3 E^2 and R2 = eta_qsvd / eta_fp =
    r L / 2 L E (Section 3.1, Eq. 15), with the compressed weights and cache
    stored at w_bits and kv_bits against an fp16 original."""
    R1 = (4.0 * r * E) / (3.0 * E * E) * (w_bits / 16.0)
    R2 = (1.0 * r) / (2.0 * E) * (kv_bits / 16.0)
    return R1, R2
