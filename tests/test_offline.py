"""Offline stage against the oracle (CPU): importance scores (Eq. 10, with
whitening and with factored linear-layer gradients), cross-layer rank
allocation, and the beta line search (Eq. 14) on synthetic layers."""
import numpy as np

from oracle import qsvd_oracle as O
from paper_2510_16292_amd import prep
from workloads import configs, gen


def _decaying_weight(d, N, slope, seed):
    g = np.random.default_rng(seed)
    Q1, _ = np.linalg.qr(g.standard_normal((d, d)))
    Q2, _ = np.linalg.qr(g.standard_normal((N, d)))
    return Q1 @ np.diag(0.5 * np.arange(1, d + 1) ** -slope) @ Q2.T


def _factored_grads(wl, d, N, n, seed):
    """Linear-layer gradients G = X^T dY: X the workload's outlier-heavy
    activations, dY ~ N(0, 1)."""
    g = np.random.default_rng(seed)
    pairs = []
    for t in range(n):
        X = gen.decode_activations(wl, t, batch=8).astype(np.float64)[:, :d]
        pairs.append((X, g.standard_normal((X.shape[0], N))))
    return pairs


def test_importance_scores_match_oracle():
    g = np.random.default_rng(1)
    d, N = 24, 40
    W = g.standard_normal((d, N))
    U, s, Vt = O.joint_svd(W)
    pairs = [(g.standard_normal((5, d)), g.standard_normal((5, N))) for _ in range(6)]
    grads = [x.T @ y for x, y in pairs]
    S_inv = np.linalg.inv(np.eye(N) + 0.2 * g.standard_normal((N, N)))
    for Si in (None, S_inv):
        ref = O.importance_scores(U, s, Vt, grads, Si)
        assert np.allclose(prep.importance_scores(U, s, Vt, grads=grads, S_inv=Si), ref, rtol=1e-12)
        assert np.allclose(prep.importance_scores(U, s, Vt, factored=pairs, S_inv=Si), ref, rtol=1e-12)


def test_allocate_ranks_matches_oracle_with_ties():
    g = np.random.default_rng(2)
    scores = [np.round(g.random(n) * 4) / 4 for n in (9, 5, 12, 1)]    # many ties
    total = sum(len(sc) for sc in scores)
    for k in range(total + 1):
        got, ref = prep.allocate_ranks(scores, k), O.allocate_ranks(scores, k)
        assert all(np.array_equal(a, b) for a, b in zip(got, ref)), k


def test_multilayer_allocation_follows_importance():
    """Four synthetic layers whose spectra decay at different rates: a global
    budget lands unevenly, and as the oracle allocates it."""
    wl = configs.get(1)
    d, N = 64, 96
    scores = []
    for l, slope in enumerate((0.3, 0.7, 1.2, 2.0)):
        U, s, Vt = O.joint_svd(_decaying_weight(d, N, slope, 10 + l))
        pairs = _factored_grads(wl, d, N, 4, 20 + l)
        sc = prep.importance_scores(U, s, Vt, factored=pairs)
        assert np.allclose(sc, O.importance_scores(U, s, Vt, [x.T @ y for x, y in pairs]), rtol=1e-10)
        scores.append(sc)
    kept = prep.allocate_ranks(scores, 96)
    ref = O.allocate_ranks(scores, 96)
    assert all(np.array_equal(a, b) for a, b in zip(kept, ref))
    ranks = [k.size for k in kept]
    assert sum(ranks) == 96 and ranks[0] > ranks[3]


def test_search_beta_matches_oracle():
    wl = configs.get(1)
    L = wl.layer
    U, s, Vt = O.joint_svd(_decaying_weight(L.d, L.N, 0.7, 5))
    Ur, sr, Vtr = U[:, :L.r], s[:L.r], Vt[:L.r]
    X = gen.prefill_activations(wl)[:24]
    betas = [0.0, 0.25, 0.5, 0.75, 1.0]

    def quant(A, B, Xc):
        lay = O.make_layer(A, B, L.n_q_heads, L.n_kv_heads, L.head_dim, 8, 0)
        p = O.prefill(lay, Xc, 8)
        return np.concatenate([p["Q"], p["K"], p["V"]], axis=1)

    best, errs = prep.search_beta(Ur, sr, Vtr, X, betas, quant)
    best_o, vals_o = O.beta_search(Ur, sr, Vtr, X, betas, quant)
    assert best == best_o
    assert np.allclose(errs, vals_o, rtol=1e-12)
