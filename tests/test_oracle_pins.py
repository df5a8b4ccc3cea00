"""The oracle against what the paper and mathematics fix (CPU only)."""
import pytest

import oracle_checks as C

PINS = [
    C.check_full_rank_reconstruction,
    C.check_eckart_young,
    C.check_svd_factors,
    C.check_decay_spectrum_factors,
    C.check_beta_and_rotation_invariance,
    C.check_act_quant_exact,
    C.check_act_quant_properties,
    C.check_weight_quant,
    C.check_int_matmul,
    C.check_projection_epilogues,
    C.check_quantized_projection_accuracy,
    C.check_absorbed_equals_reference,
    C.check_full_rank_matches_textbook_attention,
    C.check_softmax_special_cases,
    C.check_causal_prefix_consistency,
    C.check_prefill_attention,
    C.check_cache_append_and_int4,
    C.check_cache_snapshot_resume,
    C.check_cost_model,
    C.check_printed_cost_ratios,
    C.check_rotation_matrix_and_transform,
    C.check_rotation_fold_and_error_reduction,
    C.check_importance_closed_form,
    C.check_rank_allocation,
    C.check_beta_objective_value,
    C.check_beta_search,
    C.check_rope,
    C.check_prefill_attention_rope,
]


@pytest.mark.parametrize("check", PINS, ids=[f.__name__ for f in PINS])
def test_pin(check):
    check()


def test_per_group_epilogue():
    C.check_projection_epilogues(w_bits=4, w_group=32, n_samples=60)
