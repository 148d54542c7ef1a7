"""The oracle against its pins (CPU only): values the paper prints, closed
forms, invariants, library routines and brute force on tiny inputs."""

import oracle
from oracle.attention import attend
import oracle_pins as P


def test_visible_sets():
    P.pin_visible_sets(oracle.visible_key_sets)


def test_attention_brute_force():
    P.pin_attention_brute_force(oracle.chunk_attention)


def test_attention_vs_sdpa():
    P.pin_attention_vs_sdpa(oracle.chunk_attention)


def test_softmax_rows_sum_to_one():
    P.pin_softmax_rows_sum_to_one(attend)


def test_local_equals_full_when_window_covers():
    P.pin_local_equals_full_when_window_covers(oracle.chunk_attention)


def test_single_visible_key():
    P.pin_single_visible_key(oracle.chunk_attention)


def test_zero_query_gives_mean():
    P.pin_zero_query_gives_mean(oracle.chunk_attention)


def test_dominant_logit():
    P.pin_dominant_logit(oracle.chunk_attention)


def test_key_permutation_invariance():
    P.pin_key_permutation_invariance(attend)


def test_merge_identity():
    P.pin_merge_identity(oracle.chunk_attention, oracle.lse_merge)


def test_bf16_round_matches_torch():
    P.pin_bf16_round_matches_torch(oracle.bf16_round)


def test_residual_rounding():
    P.pin_residual_rounding(oracle.residual)


def test_stats_chunking_and_psd():
    P.pin_stats_chunking_and_psd(oracle.Stats)


def test_solve_scalar_hand_example():
    P.pin_solve_scalar_hand_example(oracle.solve_modulation)


def test_solve_normal_equations():
    P.pin_solve_normal_equations(oracle.Stats, oracle.solve_modulation, oracle.lstsq_modulation,
                                 oracle.residual)


def test_solve_planted():
    P.pin_solve_planted(oracle.Stats, oracle.solve_modulation)


def test_solve_orthonormal():
    P.pin_solve_orthonormal(oracle.solve_modulation)


def test_not_spd():
    P.pin_not_spd(oracle.solve_modulation, oracle.NotSPD)


def test_feasibility():
    P.pin_feasibility(oracle.Stats, oracle.solve_modulation, oracle.feasibility,
                      oracle.feasibility_direct, oracle.residual)


def test_select_layers():
    P.pin_select_layers(oracle.select_layers)


def test_inject():
    P.pin_inject(oracle.inject, oracle.bf16_round)


def test_project():
    P.pin_project(oracle.project)


def test_quantize_rows():
    P.pin_quantize_rows(oracle.quantize_rows, oracle.dequantize_rows)


def test_project_w8a8():
    P.pin_project_w8a8(oracle.project_w8a8)


def test_evict_local():
    P.pin_evict_local(oracle.evict_local)


def test_local_history():
    P.pin_local_history(oracle.LocalHistory)


def test_kv_table():
    P.pin_kv_table(oracle.kv_retained_fraction)


def test_layer_budget():
    P.pin_layer_budget(oracle.n_local_layers)


def test_hyperparams():
    P.pin_hyperparams()
