"""The oracle against its pins (hand tables, closed forms, invariants,
brute force, exact rationals, library matmul, the paper's bit accounting)."""
import pytest

import oracle_pins as pins


def test_hand_cases_c_oracle(oracle_lib):
    pins.check_hand_cases_c()


def test_hand_cases_exact_rationals():
    pins.check_hand_cases_exact()


@pytest.mark.parametrize("m", [4, 6, 8])
@pytest.mark.parametrize("rnd", [0, 1])
@pytest.mark.parametrize("clamp", [0, 1])
def test_single_element_blocks_exhaustive(oracle_lib, m, rnd, clamp):
    pins.check_single_element_exhaustive(m, rnd, clamp)


def test_exponent_bracketing(oracle_lib):
    pins.check_exponent_bracketing()


def test_bruteforce_nearest(oracle_lib):
    pins.check_bruteforce_nearest()


def test_c_oracle_equals_exact_rationals(oracle_lib):
    pins.check_exact_agrees()


def test_symmetries(oracle_lib):
    pins.check_symmetries()


def test_round_trip_and_idempotence(oracle_lib):
    pins.check_round_trip()


def test_gemm_equals_dequantized_matmul(oracle_lib):
    pins.check_gemm_vs_dequantized_matmul()


def test_gemm_exact_rationals(oracle_lib):
    pins.check_gemm_exact_rationals()


def test_absbound_exact_rationals(oracle_lib):
    pins.check_absbound_exact_rationals()


def test_absbound_invariants(oracle_lib):
    pins.check_absbound_invariants()


def test_gemm_textbook_case(oracle_lib):
    pins.check_gemm_textbook_case()


def test_gemm_permutation_invariance(oracle_lib):
    pins.check_gemm_permutation_invariance()


def test_permutation_gather(oracle_lib):
    pins.check_permutation_gather()


def test_block_partials(oracle_lib):
    pins.check_block_partials()


def test_gemm_nan_propagation(oracle_lib):
    pins.check_gemm_nan()


def test_packed_layout(oracle_lib):
    pins.check_pack_layout()


def test_storage_accounting(oracle_lib):
    pins.check_storage_accounting()
