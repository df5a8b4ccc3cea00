"""Plant a plausible mistake in the oracle (CPU only) and check that a pin fails.

Each case monkeypatches one oracle function with a wrong variant; the listed
checks must raise.  This shows the pins can tell a correct oracle from a
subtly wrong one.
"""
import numpy as np
import pytest

import oracle_checks as C
from oracle import qsvd_oracle as O

_orig_split = O.split_beta
_orig_quant = O.quantize_act
_orig_scaled = O._scaled
_orig_pack = O.pack_int4
_orig_svd = O.joint_svd


def _split_sigma_both(U_r, s, Vt_r, beta):          # Sigma^beta on both sides
    return U_r * (s ** beta)[None, :], (s ** beta)[:, None] * Vt_r


def _split_truncate_wrong_end(U_r, s, Vt_r, beta):  # keeps the smallest values
    A, B = _orig_split(U_r, s, Vt_r, beta)
    return A[:, ::-1], B[::-1, :] * 0.999


def _quant_floor(x, bits, clip=1.0):                # truncation instead of RNE
    xf = np.asarray(x).astype(np.float32)
    Qm = np.float32(O.qmax(bits))
    a = np.max(np.abs(xf), axis=1)
    a[a == 0] = 1
    s = (a / Qm).astype(np.float32)
    q = np.clip(np.trunc(xf * (Qm / a)[:, None]), -Qm, Qm).astype(np.int8)
    return q, s


def _quant_divide(x, bits, clip=1.0):               # x / s instead of x * (Qm / a)
    xf = np.asarray(x).astype(np.float32)
    Qm = np.float32(O.qmax(bits))
    a = np.max(np.abs(xf), axis=1).astype(np.float32)
    s = (a / Qm).astype(np.float32)
    s[a == 0] = 1
    q = np.clip(np.rint(xf / s[:, None]), -Qm, Qm).astype(np.int8)
    return q, s


def _scaled_swapped(acc, s_row, w_scale, group, K, aq, wq):   # scales applied in the other order
    if group:
        return _orig_scaled(acc, s_row, w_scale, group, K, aq, wq)
    y = (acc.astype(np.float32) * w_scale.astype(np.float32)[None, :]).astype(np.float32)
    return (y * s_row.astype(np.float32)[:, None]).astype(np.float32)


def _scaled_in_f64(acc, s_row, w_scale, group, K, aq, wq):    # no fp32 rounding at all
    if group:
        return _orig_scaled(acc, s_row, w_scale, group, K, aq, wq)
    return (acc * s_row.astype(np.float64)[:, None] * w_scale.astype(np.float64)[None, :]).astype(np.float32)


def _pack_swapped(q):                                # high/low nibble swapped
    p = _orig_pack(q)
    return ((p >> 4) | (p << 4)).astype(np.uint8)


def _svd_no_sign_fix(W):
    U, s, Vt = np.linalg.svd(np.asarray(W, dtype=np.float64), full_matrices=False)
    return -U, s, -Vt


def _kv_group_modulo(h, hq, hkv):                    # interleaved instead of blocked groups
    return h % hkv


def _kv_group_off_by_one(h, hq, hkv):
    return min(hkv - 1, (h * hkv) // hq + (1 if h == 1 else 0))


_good_wht = O.walsh_hadamard_rows
_good_rotate = O.rotate_act


def _wht_sub_swapped(v, block, dtype=np.float32):       # (b - a) in the second output
    out = np.array(v, dtype=dtype, copy=True)
    M, K = out.shape
    h = 1
    while h < block:
        w = out.reshape(M, K // (2 * h), 2, h)
        a, b = w[:, :, 0, :].copy(), w[:, :, 1, :].copy()
        w[:, :, 0, :] = (a + b).astype(dtype)
        w[:, :, 1, :] = (b - a).astype(dtype)
        h *= 2
    return out


def _rotate_no_signs(x, signs, block):                  # random diagonal dropped
    return _good_rotate(x, np.ones_like(signs), block)


def _rotate_scale_by_b(x, signs, block):                # 1/B instead of 1/sqrt(B)
    return (_good_rotate(x, signs, block) * np.float32(1.0 / np.sqrt(block))).astype(np.float32)


def _importance_sigma_not_squared(U, s, Vt, grads, S_inv=None):   # sigma instead of sigma^2
    V = Vt.T
    acc = np.zeros(s.size)
    for G in grads:
        Gw = G if S_inv is None else G @ S_inv.T
        acc += np.diag(U.T @ Gw @ V) ** 2
    return s * acc / len(grads)


def _importance_whitening_untransposed(U, s, Vt, grads, S_inv=None):   # S^-1 where S^-T belongs
    V = Vt.T
    acc = np.zeros(s.size)
    for G in grads:
        Gw = G if S_inv is None else G @ S_inv
        acc += np.diag(U.T @ Gw @ V) ** 2
    return s ** 2 * acc / len(grads)


def _allocate_lowest(scores, budget):                   # keeps the least important
    entries = sorted((float(v), l, i) for l, sc in enumerate(scores) for i, v in enumerate(sc))
    kept = [[] for _ in scores]
    for _, l, i in entries[:budget]:
        kept[l].append(i)
    return [np.array(sorted(k), dtype=np.int64) for k in kept]


def _rope_freq_wrong(x, positions, theta, dh):            # theta^(-j/dh) instead of theta^(-2j/dh)
    x = np.asarray(x, dtype=np.float64)
    half = dh // 2
    ang = np.asarray(positions, dtype=np.float64)[:, None] * (theta ** (-1.0 * np.arange(half) / dh))[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    for h in range(x.shape[1] // dh):
        a, b = x[:, h * dh:h * dh + half], x[:, h * dh + half:(h + 1) * dh]
        out[:, h * dh:h * dh + half], out[:, h * dh + half:(h + 1) * dh] = a * c - b * s, b * c + a * s
    return out


def _rope_sign_wrong(x, positions, theta, dh):            # rotation the other way
    return _rope_freq_ok(x, -np.asarray(positions, dtype=np.float64), theta, dh)


_rope_freq_ok = O.rope
_good_prefill_attention = O.prefill_attention
_good_snapshot = O.cache_snapshot


def _beta_objective_norm_not_squared(A, B, X, layer_fn):   # ||Y - Y'|| instead of ||Y - Y'||^2
    Y = np.asarray(X, dtype=np.float64) @ A @ B
    return float(np.sqrt(np.sum((Y - np.asarray(layer_fn(A, B, X), np.float64)) ** 2)))


def _beta_objective_q_only(A, B, X, layer_fn):             # only the query third of the columns
    Y = np.asarray(X, dtype=np.float64) @ A @ B
    n = Y.shape[1] // 3
    return float(np.sum((Y - np.asarray(layer_fn(A, B, X), np.float64))[:, :n] ** 2))


def _prefill_attention_no_mask(Q, K, V, lengths, hq, hkv, dh, sm_scale=None):   # every token sees all
    sm = 1.0 / np.sqrt(dh)
    out = np.zeros(np.shape(Q))
    t0 = 0
    for n in lengths:
        for h in range(hq):
            g = O.kv_group(h, hq, hkv)
            s = (Q[t0:t0 + n, h * dh:(h + 1) * dh] @ K[t0:t0 + n, g * dh:(g + 1) * dh].T) * sm
            out[t0:t0 + n, h * dh:(h + 1) * dh] = O._softmax(s) @ V[t0:t0 + n, g * dh:(g + 1) * dh]
        t0 += n
    return out


def _prefill_attention_one_sequence(Q, K, V, lengths, hq, hkv, dh, sm_scale=None):   # sequences not separated
    return _good_prefill_attention(Q, K, V, [sum(lengths)], hq, hkv, dh, sm_scale)


def _prefill_attention_strict(Q, K, V, lengths, hq, hkv, dh, sm_scale=None):   # query i sees 0..i-1 (own key dropped)
    sm = 1.0 / np.sqrt(dh)
    out = np.zeros(np.shape(Q))
    t0 = 0
    for n in lengths:
        for h in range(hq):
            g = O.kv_group(h, hq, hkv)
            s = (Q[t0:t0 + n, h * dh:(h + 1) * dh] @ K[t0:t0 + n, g * dh:(g + 1) * dh].T) * sm
            s[np.triu_indices(n, 0)] = -np.inf
            s[0, 0] = 0.0
            out[t0:t0 + n, h * dh:(h + 1) * dh] = O._softmax(s) @ V[t0:t0 + n, g * dh:(g + 1) * dh]
        t0 += n
    return out


def _per_sequence_rope(x, lengths, theta, dh, reverse=False):
    out = np.array(x, dtype=np.float64)
    t0 = 0
    for n in lengths:
        pos = np.arange(n)[::-1] if reverse else np.arange(n)
        out[t0:t0 + n] = _rope_freq_ok(out[t0:t0 + n], pos, theta, dh)
        t0 += n
    return out


def _prefill_rope_rotates_v(Q, K, V, lengths, hq, hkv, dh, sm_scale=None, rope_theta=None):   # V turned too
    if rope_theta:
        V = _per_sequence_rope(V, lengths, rope_theta, dh)
    return _good_prefill_attention(Q, K, V, lengths, hq, hkv, dh, sm_scale, rope_theta)


def _prefill_rope_q_only(Q, K, V, lengths, hq, hkv, dh, sm_scale=None, rope_theta=None):   # keys left unturned
    if rope_theta:
        Q = _per_sequence_rope(Q, lengths, rope_theta, dh)
    return _good_prefill_attention(Q, K, V, lengths, hq, hkv, dh, sm_scale)


def _prefill_rope_reversed(Q, K, V, lengths, hq, hkv, dh, sm_scale=None, rope_theta=None):   # positions n-1..0
    if rope_theta:
        Q = _per_sequence_rope(Q, lengths, rope_theta, dh, reverse=True)
        K = _per_sequence_rope(K, lengths, rope_theta, dh, reverse=True)
    return _good_prefill_attention(Q, K, V, lengths, hq, hkv, dh, sm_scale)


def _prefill_rope_global_positions_reversed(Q, K, V, lengths, hq, hkv, dh, sm_scale=None, rope_theta=None):
    # positions counted over the whole block, last token first (only a constant
    # shift of all positions would leave the scores unchanged)
    if rope_theta:
        Q = _per_sequence_rope(Q, [sum(lengths)], rope_theta, dh, reverse=True)
        K = _per_sequence_rope(K, [sum(lengths)], rope_theta, dh, reverse=True)
    return _good_prefill_attention(Q, K, V, lengths, hq, hkv, dh, sm_scale)


def _snapshot_views(cache):                                  # no copy: later appends change it
    snap = dict(data=cache.data, seq_len=cache.seq_len)
    if cache.scale is not None:
        snap["scale"] = cache.scale
    return snap


MUTATIONS = [
    ("split_beta", _split_sigma_both, [C.check_full_rank_reconstruction, C.check_beta_and_rotation_invariance]),
    ("split_beta", _split_truncate_wrong_end, [C.check_eckart_young]),
    ("quantize_act", _quant_floor, [C.check_act_quant_exact, C.check_act_quant_properties]),
    ("quantize_act", _quant_divide, [C.check_act_quant_exact]),
    ("_scaled", _scaled_swapped, [C.check_projection_epilogues]),
    ("_scaled", _scaled_in_f64, [C.check_projection_epilogues]),
    ("pack_int4", _pack_swapped, [C.check_cache_append_and_int4]),
    ("joint_svd", _svd_no_sign_fix, [C.check_svd_factors]),
    ("kv_group", _kv_group_modulo, [C.check_full_rank_matches_textbook_attention]),
    ("kv_group", _kv_group_off_by_one, [C.check_full_rank_matches_textbook_attention]),
    ("walsh_hadamard_rows", _wht_sub_swapped, [C.check_rotation_matrix_and_transform]),
    ("rotate_act", _rotate_no_signs, [C.check_rotation_matrix_and_transform]),
    ("rotate_act", _rotate_scale_by_b, [C.check_rotation_matrix_and_transform]),
    ("importance_scores", _importance_sigma_not_squared, [C.check_importance_closed_form]),
    ("importance_scores", _importance_whitening_untransposed, [C.check_importance_closed_form]),
    ("allocate_ranks", _allocate_lowest, [C.check_rank_allocation]),
    ("rope", _rope_freq_wrong, [C.check_rope]),
    ("rope", _rope_sign_wrong, [C.check_rope]),
    ("beta_objective", _beta_objective_norm_not_squared, [C.check_beta_objective_value]),
    ("beta_objective", _beta_objective_q_only, [C.check_beta_objective_value]),
    ("prefill_attention", _prefill_attention_no_mask, [C.check_prefill_attention]),
    ("prefill_attention", _prefill_attention_one_sequence, [C.check_prefill_attention]),
    ("prefill_attention", _prefill_attention_strict, [C.check_prefill_attention]),
    ("kv_group", _kv_group_modulo, [C.check_prefill_attention]),
    ("prefill_attention", _prefill_rope_rotates_v, [C.check_prefill_attention_rope]),
    ("prefill_attention", _prefill_rope_q_only, [C.check_prefill_attention_rope]),
    ("prefill_attention", _prefill_rope_reversed, [C.check_prefill_attention_rope]),
    ("prefill_attention", _prefill_rope_global_positions_reversed, [C.check_prefill_attention_rope]),
    ("cache_snapshot", _snapshot_views, [C.check_cache_snapshot_resume]),
]


@pytest.mark.parametrize("name,bad,checks", MUTATIONS,
                         ids=[f"{m[0]}:{m[1].__name__}" for m in MUTATIONS])
def test_planted_mistake_is_caught(monkeypatch, name, bad, checks):
    monkeypatch.setattr(O, name, bad)
    for check in checks:
        with pytest.raises(AssertionError):
            check()
