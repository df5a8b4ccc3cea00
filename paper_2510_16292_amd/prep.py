"""Offline stage of QSVD: turn a layer's [W_q | W_k | W_v] into the quantized,
transposed factors the HIP library consumes.

This runs once per layer on the host before inference, as in the paper
(Section 3.1: joint SVD and truncation, Eq. 2-4; Section 3.3 / Section 4:
round-to-nearest symmetric weight quantization).  It is not part of the
per-token hot path.

Conventions (shared with the C ABI, include/qsvd.h):
  * Y = X W with W of shape d x N; W^d = U_r Sigma_r^beta (d x r) and
    W^u = Sigma_r^(1-beta) V_r^T (r x N).
  * Right singular vectors are sign-normalized: the entry of largest magnitude
    of each is positive (the left vector flips with it).
  * Weight codes are rint(w / s) in fp64 with the scale s = clip*max|w|/Qm
    rounded to fp32 (1 for an all-zero column or group), clamped to [-Qm, Qm];
    per output channel (w_group 0) or per output channel and per block of
    w_group contraction rows.
  * Device layout is transposed (contraction index contiguous): a_t [r][d],
    b_t [N][r]; int4 codes pack element 2i in the low nibble of byte i.
"""
from dataclasses import dataclass

import numpy as np


@dataclass
class PreparedLayer:
    d: int
    r: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    w_bits: int
    w_group: int
    a_t: np.ndarray     # int8 [r][d] or uint8 [r][d/2]
    s_a: np.ndarray     # fp32 [r] or [d/G][r]
    b_t: np.ndarray     # int8 [N][r] or uint8 [N][r/2]
    s_b: np.ndarray     # fp32 [N] or [r/G][N]

    @property
    def N(self):
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


def truncated_factors(W: np.ndarray, r: int, beta: float):
    """(W^d, W^u) of the rank-r joint SVD of W with Sigma split by beta."""
    U, s, Vt = np.linalg.svd(np.asarray(W, dtype=np.float64), full_matrices=False)
    lead = np.abs(Vt).argmax(axis=1)
    flip = np.where(Vt[np.arange(len(s)), lead] < 0, -1.0, 1.0)
    U, Vt = U * flip, Vt * flip[:, None]
    return factors_from_svd(U[:, :r], s[:r], Vt[:r].T, beta)


# ---------------------------------------------------------------------------
# Rank allocation by importance score and the beta search (Section 3.2,
# Eq. 10 and Appendix A; Eq. 14)
# ---------------------------------------------------------------------------

def importance_scores(U: np.ndarray, s: np.ndarray, Vt: np.ndarray, grads=None, factored=None,
                      S_inv: np.ndarray = None) -> np.ndarray:
    """Importance of every singular value (Eq. 10): mean over calibration
    samples of sigma_i^2 [U^T G V]_(i,i)^2, with G S^{-T} in place of G when the
    SVD was of a whitened W S (Appendix A).  Gradients come either explicitly
    (`grads`: d x N arrays) or factored as a linear layer's (X_n, dY_n) pairs,
    G_n = X_n^T dY_n, in which case [U^T G V]_(i,i) = sum_t (X_n U)[t,i]
    (dY_n S^{-T} V)[t,i] and no d x N gradient is formed."""
    V = np.asarray(Vt, dtype=np.float64).T
    U = np.asarray(U, dtype=np.float64)
    total, count = np.zeros(s.size), 0
    for G in grads or []:
        Gw = np.asarray(G, dtype=np.float64)
        if S_inv is not None:
            Gw = Gw @ S_inv.T
        total += np.einsum("ji,ji->i", U, Gw @ V) ** 2
        count += 1
    for Xn, dYn in factored or []:
        dYw = np.asarray(dYn, dtype=np.float64)
        if S_inv is not None:
            dYw = dYw @ S_inv.T
        total += np.einsum("ti,ti->i", np.asarray(Xn, dtype=np.float64) @ U, dYw @ V) ** 2
        count += 1
    return np.asarray(s, dtype=np.float64) ** 2 * total / max(count, 1)


def allocate_ranks(scores, budget: int):
    """Cross-layer rank selection (Section 3.2): every singular value of every
    layer ranked by importance, the `budget` highest kept (ties to the lower
    layer, then the lower index).  Returns each layer's kept indices, sorted."""
    layer = np.concatenate([np.full(len(sc), l) for l, sc in enumerate(scores)]) if scores else np.zeros(0)
    index = np.concatenate([np.arange(len(sc)) for sc in scores]) if scores else np.zeros(0)
    value = np.concatenate([np.asarray(sc, dtype=np.float64) for sc in scores]) if scores else np.zeros(0)
    order = np.lexsort((index, layer, -value))[:budget]
    return [np.sort(index[order][layer[order] == l]).astype(np.int64) for l in range(len(scores))]


def select_factors(U: np.ndarray, s: np.ndarray, Vt: np.ndarray, keep: np.ndarray, beta: float):
    """W^d, W^u of the kept singular triplets (any subset of indices), Eq. 3-4."""
    return factors_from_svd(U[:, keep], s[keep], np.asarray(Vt)[keep].T, beta)


def search_beta(U_r: np.ndarray, s_r: np.ndarray, Vt_r: np.ndarray, X: np.ndarray, betas, project):
    """Per-layer line search of Eq. 14 on the projection: for each beta of the
    grid, Y' = project(A, B, X) (the quantized Q | K | V of the layer built
    from W^d = U Sigma^beta, W^u = Sigma^(1 - beta) V^T) against the fp64
    Y = X W^d W^u; returns (the first beta with the least squared error, all
    errors)."""
    Xf = np.asarray(X, dtype=np.float64)
    errs = []
    for b in betas:
        A, B = factors_from_svd(U_r, s_r, np.asarray(Vt_r).T, b)
        errs.append(float(np.sum((Xf @ A @ B - np.asarray(project(A, B, X), dtype=np.float64)) ** 2)))
    return betas[int(np.argmin(errs))], errs


def fold_input_rotation(A: np.ndarray, signs: np.ndarray, block: int) -> np.ndarray:
    """H1 W^d for the online input rotation H1 = blockdiag(H_B) diag(signs) /
    sqrt(B) (Eq. 11), so that Q(X H1^T) Q(H1 W^d) replaces Q(X) Q(W^d): rows
    of W^d are multiplied by the signs, then every column goes through the
    block Walsh-Hadamard transform along its rows, in fp64."""
    A = np.asarray(A, dtype=np.float64) * np.asarray(signs, dtype=np.float64)[:, None]
    d, r = A.shape
    assert d % block == 0 and block & (block - 1) == 0
    out = A.reshape(d // block, block, r).copy()
    h = 1
    while h < block:
        v = out.reshape(d // block, block // (2 * h), 2, h, r)
        a, b = v[:, :, 0].copy(), v[:, :, 1].copy()
        v[:, :, 0], v[:, :, 1] = a + b, a - b
        h *= 2
    return out.reshape(d, r) / np.sqrt(block)


def factors_from_svd(U_r: np.ndarray, sigma_r: np.ndarray, V_r: np.ndarray, beta: float):
    """W^d = U_r diag(sigma^beta), W^u = diag(sigma^(1-beta)) V_r^T."""
    return U_r * np.power(sigma_r, beta), (V_r * np.power(sigma_r, 1.0 - beta)).T


def _quantize_t(Wt: np.ndarray, bits: int, group: int, clip: float):
    """Quantize a transposed weight Wt [Nout][K] along K; returns codes [Nout][K]
    and scales [Nout] or [K/group][Nout]."""
    qm = float((1 << (bits - 1)) - 1)
    n_out, K = Wt.shape
    if group:
        blocks = Wt.reshape(n_out, K // group, group)
        amax = np.abs(blocks).max(axis=2)                       # [Nout][G]
        scale = np.where(amax == 0, np.float32(1), (clip * amax / qm).astype(np.float32)).astype(np.float32)
        codes = np.rint(blocks / scale.astype(np.float64)[:, :, None]).reshape(n_out, K)
        scale = np.ascontiguousarray(scale.T)                    # [G][Nout]
    else:
        amax = np.abs(Wt).max(axis=1)
        scale = np.where(amax == 0, np.float32(1), (clip * amax / qm).astype(np.float32)).astype(np.float32)
        codes = np.rint(Wt / scale.astype(np.float64)[:, None])
    codes = np.clip(codes, -qm, qm).astype(np.int8)
    return codes, scale


def pack_int4_rows(codes: np.ndarray) -> np.ndarray:
    """Pack int8 codes in [-8, 7] two per byte along the last axis (even index low)."""
    c = codes.astype(np.uint8) & 0x0F
    return np.ascontiguousarray(c[..., 0::2] | (c[..., 1::2] << 4))


def quantize_layer(A: np.ndarray, B: np.ndarray, n_q_heads: int, n_kv_heads: int, head_dim: int,
                   w_bits: int = 8, w_group: int = 0, clip: float = 1.0) -> PreparedLayer:
    """Quantize W^d (d x r) and W^u (r x N) and lay them out for the device."""
    d, r = A.shape
    assert B.shape[0] == r and B.shape[1] == (n_q_heads + 2 * n_kv_heads) * head_dim
    a_codes, s_a = _quantize_t(np.ascontiguousarray(A.T), w_bits, w_group, clip)   # [r][d]
    b_codes, s_b = _quantize_t(np.ascontiguousarray(B.T), w_bits, w_group, clip)   # [N][r]
    if w_bits == 4:
        a_codes, b_codes = pack_int4_rows(a_codes), pack_int4_rows(b_codes)
    return PreparedLayer(d, r, n_q_heads, n_kv_heads, head_dim, w_bits, w_group,
                         np.ascontiguousarray(a_codes), s_a, np.ascontiguousarray(b_codes), s_b)


def prepare_from_weight(W, r, n_q_heads, n_kv_heads, head_dim, beta=0.5, w_bits=8, w_group=0, clip=1.0):
    A, B = truncated_factors(W, r, beta)
    return quantize_layer(A, B, n_q_heads, n_kv_heads, head_dim, w_bits, w_group, clip)


def prepare_from_svd(U_r, sigma_r, V_r, n_q_heads, n_kv_heads, head_dim, beta=0.5, w_bits=8, w_group=0,
                     clip=1.0):
    A, B = factors_from_svd(U_r, sigma_r, V_r, beta)
    return quantize_layer(A, B, n_q_heads, n_kv_heads, head_dim, w_bits, w_group, clip)
