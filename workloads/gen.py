"""Seeded random inputs: weights (or their known factors), activations, decode inputs.

Seeds are ``numpy.random.default_rng(16292 + 100*cfg + role + 1000*layer)``.
Roles: 0 weights, 1 prefill activations, 2 outlier channels, 3 synthetic
cache fill, 4+t decode input of step t, 99 per-layer ranks of a stack.

Nothing here belongs to the method: weights with a prescribed spectrum are
built as U diag(sigma) V^T from orthonormal factors (so for those workloads the
truncated SVD is known by construction), activations are Gaussian with a few
channel-wise outlier columns as described for the profiled activations in
Section 3.3.
"""
import numpy as np

from .configs import Workload

ROLE_W, ROLE_X, ROLE_OUTLIER, ROLE_FILL, ROLE_DECODE0 = 0, 1, 2, 3, 4
ROLE_RANKS = 99     # per-layer ranks of a stack (drawn once per workload, layer 0)


def stack_ranks(wl: Workload) -> list:
    """Per-layer ranks of a multi-layer stack, standing in for an importance-
    based rank allocation: multiples of 128 drawn uniformly in [1024, 3072]
    (multiples of the 128-element weight group, so every group along r is
    whole)."""
    g = rng_for(wl, ROLE_RANKS)
    return [int(128 * k) for k in g.integers(8, 25, size=wl.n_layers)]


def with_rank(wl: Workload, r: int) -> Workload:
    """The same workload with the layer rank replaced (one layer of a stack)."""
    from dataclasses import replace
    return replace(wl, layer=replace(wl.layer, r=int(r)))


def weight_codes_device(seed: int, rows: int, cols: int, bits: int, groups: int, device="cuda"):
    """Device-side weight codes and positive scales for timing-only stacks:
    codes [rows][cols] (int8, or int4 packed two per byte along cols, low
    nibble first) drawn as a rounded N(0, (qmax/3)^2) clipped to +-qmax, the
    spread round-to-nearest leaves for Gaussian weights; scales [groups][rows]
    fp32 around 0.02 / qmax (one row when groups is 1)."""
    import torch
    qm = (1 << (bits - 1)) - 1
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    z = torch.randn((rows, cols), generator=g, device=device) * (qm / 3.0)
    c = torch.clamp(torch.round(z), -qm, qm).to(torch.int8)
    if bits == 4:
        u = (c.to(torch.int16) & 0xF).to(torch.uint8)
        c = (u[:, 0::2] | (u[:, 1::2] << 4)).contiguous()
    s = (torch.rand((groups, rows), generator=g, device=device) * 0.5 + 0.75) * (0.02 / qm)
    return c, s.to(torch.float32).contiguous()


def rng_for(wl: Workload, role: int, layer: int = 0) -> np.random.Generator:
    return np.random.default_rng(16292 + 100 * wl.cfg_id + role + 1000 * layer)


def weight_matrix(wl: Workload, layer: int = 0) -> np.ndarray:
    """Concatenated [W_q | W_k | W_v] (d x N), iid N(0, w_std^2) rounded to fp32.

    Returned as float64 holding fp32 values.  Only for ``spectrum == "gaussian"``.
    """
    assert wl.spectrum == "gaussian"
    L = wl.layer
    g = rng_for(wl, ROLE_W, layer)
    w = (g.standard_normal((L.d, L.N)) * wl.w_std).astype(np.float32)
    return w.astype(np.float64)


def _orthonormal(g: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    q, r = np.linalg.qr(g.standard_normal((rows, cols)))
    return q * np.sign(np.diag(r))[None, :]


def spectrum(wl: Workload) -> np.ndarray:
    """sigma_i = sigma_1 * i^-decay_exp for i = 1..min(d, N); sigma_1 makes
    ||W||_F equal to that of an iid N(0, w_std^2) matrix of the same shape."""
    L = wl.layer
    n = min(L.d, L.N)
    i = np.arange(1, n + 1, dtype=np.float64)
    shape = i ** (-wl.decay_exp)
    sigma1 = wl.w_std * np.sqrt(L.d * L.N) / np.sqrt(np.sum(shape * shape))
    return sigma1 * shape


def weight_factors(wl: Workload, layer: int = 0, rank: int = None):
    """Leading ``rank`` singular triplets (U_r [d,r], sigma_r [r], V_r [N,r]) of a
    d x N weight with the decaying spectrum, known by construction.

    The full matrix would be U diag(sigma) V^T over all min(d, N) triplets; the
    trailing ones are orthogonal to these and are never needed by the hot path.
    """
    assert wl.spectrum == "decay"
    L = wl.layer
    rank = L.r if rank is None else rank
    g = rng_for(wl, ROLE_W, layer)
    U = _orthonormal(g, L.d, rank)
    V = _orthonormal(g, L.N, rank)
    return U, spectrum(wl)[:rank].copy(), V


def outlier_channels(wl: Workload, layer: int = 0) -> np.ndarray:
    g = rng_for(wl, ROLE_OUTLIER, layer)
    return np.sort(g.choice(wl.layer.d, size=wl.outlier_count, replace=False))


def _activation_rows(g: np.random.Generator, wl: Workload, rows: int, layer: int) -> np.ndarray:
    x = g.standard_normal((rows, wl.layer.d))
    x[:, outlier_channels(wl, layer)] *= wl.outlier_scale
    return x.astype(np.float16)


def prefill_activations(wl: Workload, layer: int = 0, rows: int = None) -> np.ndarray:
    """fp16 [prefill_M, d]: N(0,1) with the outlier channels scaled."""
    rows = wl.prefill_M if rows is None else rows
    return _activation_rows(rng_for(wl, ROLE_X, layer), wl, rows, layer)


def decode_activations(wl: Workload, step: int, layer: int = 0, batch: int = None) -> np.ndarray:
    """fp16 [batch, d]: a fresh seeded row per sequence for decode step ``step``."""
    batch = wl.decode_batch if batch is None else batch
    return _activation_rows(rng_for(wl, ROLE_DECODE0 + step, layer), wl, batch, layer)


def fill_activations(wl: Workload, rows: int, layer: int = 0) -> np.ndarray:
    """fp16 [rows, d] used to build a pre-filled latent cache."""
    return _activation_rows(rng_for(wl, ROLE_FILL, layer), wl, rows, layer)


def random_rows(seed: int, shape, scale: float = 1.0, dtype=np.float16) -> np.ndarray:
    """Plain N(0, scale^2) array for small edge-case tests."""
    g = np.random.default_rng(seed)
    return (g.standard_normal(shape) * scale).astype(dtype)


def latent_rows(wl: Workload, batch: int, length: int, layer: int = 0, seed_offset: int = 0) -> np.ndarray:
    """fp16 [batch, length, r] synthetic rows for a pre-filled fp16 latent
    cache: column j ~ N(0, sigma_j) for the decaying spectrum (unit variance
    for the Gaussian one), the magnitude of X W^d with beta = 1/2 and unit X."""
    g = rng_for(wl, ROLE_FILL + seed_offset, layer)
    r = wl.layer.r
    std = np.sqrt(spectrum(wl)[:r]) if wl.spectrum == "decay" else np.ones(r)
    rows = np.empty((batch, length, r), dtype=np.float16)
    for b in range(batch):
        rows[b] = (g.standard_normal((length, r)) * std[None, :]).astype(np.float16)
    return rows


def latent_codes(wl: Workload, batch: int, length: int, layer: int = 0, seed_offset: int = 0):
    """Synthetic int8 latent cache contents with the magnitudes of
    :func:`latent_rows`: codes in [-127, 127] whose column j spreads in
    proportion to sigma_j (column 0 at +127, so every row reaches the top code),
    and positive per-token fp32 scales around sigma_1 / 40, so code * scale has
    about the spread of the fp16 latent rows."""
    g = rng_for(wl, ROLE_FILL + seed_offset, layer)
    r = wl.layer.r
    std = np.sqrt(spectrum(wl)[:r]) if wl.spectrum == "decay" else np.ones(r)
    z = g.standard_normal((batch, length, r)) * (40.0 * std / std[0])[None, None, :]
    codes = np.clip(np.rint(z), -127, 127).astype(np.int8)
    codes[:, :, 0] = 127
    scales = (g.uniform(0.8, 1.25, (batch, length)) * (std[0] / 40.0)).astype(np.float32)
    return codes, scales


def latent_rows_device(wl: Workload, batch: int, length: int, seed: int, out=None, device="cuda"):
    """Device-side variant of :func:`latent_rows` for large pre-filled caches
    (torch's seeded generator on the GPU): fp16 [batch, length, r] with
    column j ~ N(0, sigma_j).  Writes into ``out[:, :length]`` if given."""
    import torch
    r = wl.layer.r
    std = np.sqrt(spectrum(wl)[:r]) if wl.spectrum == "decay" else np.ones(r)
    std_t = torch.tensor(std, dtype=torch.float32, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    if out is None:
        out = torch.empty((batch, length, r), dtype=torch.float16, device=device)
    for b in range(batch):
        out[b, :length] = (torch.randn((length, r), generator=g, device=device) * std_t).to(torch.float16)
    return out


def latent_codes_device(wl: Workload, batch: int, length: int, seed: int, codes=None, scales=None, device="cuda",
                        bits: int = 8):
    """Device-side variant of :func:`latent_codes` for large pre-filled integer
    caches (torch's seeded generator on the GPU): writes codes into
    ``codes[:, :length]`` (int8 [batch, >=length, r], or for bits 4 uint8
    [batch, >=length, r/2] with two codes per byte, low nibble first) and
    per-token scales into ``scales[:, :length]``.  Column j spreads in
    proportion to sigma_j with column 0 at the top code; the scales put
    code * scale at the magnitude of the fp16 latent rows."""
    import torch
    r = wl.layer.r
    qm = (1 << (bits - 1)) - 1
    spread = 40.0 * qm / 127.0
    std = np.sqrt(spectrum(wl)[:r]) if wl.spectrum == "decay" else np.ones(r)
    col = torch.tensor(spread * std / std[0], dtype=torch.float32, device=device)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    for b in range(batch):
        z = torch.randn((length, r), generator=g, device=device) * col
        c = torch.clamp(torch.round(z), -qm, qm).to(torch.int8)
        c[:, 0] = qm
        if bits == 4:
            u = (c.to(torch.int16) & 0xF).to(torch.uint8)
            codes[b, :length] = u[:, 0::2] | (u[:, 1::2] << 4)
        else:
            codes[b, :length] = c
        u = torch.rand((length,), generator=g, device=device) * 0.45 + 0.8
        scales[b, :length] = u * float(std[0] / spread)
