"""The analytic cost model against the closed forms and limits the paper
states for it (Sec. 4.1-4.3)."""
import math

import pytest

from paper_2606_19025_amd import costmodel as C


@pytest.mark.parametrize("M", [2, 4, 8, 16])
def test_full_replica_limit(M):
    # O_e = M: no migration ever, and the expert payload is the dense ring cost
    assert C.migration_factor(M, M, 1.0) == 0.0
    assert C.p_hit(M, M) == 1.0
    S = 1e9
    assert math.isclose(C.sparse_bytes(M, M, 1.0, S), C.dense_bytes(M, S))


@pytest.mark.parametrize("M", [2, 4, 8, 16])
def test_disjoint_partition_limit(M):
    # O_e = 1: no aggregation ring; nearly every reshuffle replaces the set
    assert C.ring_factor(1) == 0.0
    assert math.isclose(C.migration_factor(1, M, 1.0), 1 - 1 / M)
    assert C.sparse_bytes(1, M, 0.0, 5e8) == 0.0  # fixed placement: nothing moves


def test_probabilities_and_hand_example():
    M, O_e, N_e = 8, 2, 64
    assert C.local_experts(N_e, O_e, M) == 16
    assert math.isclose(C.p_hit(O_e, M) + C.p_miss(O_e, M), 1.0)
    assert C.ring_factor(2) == 1.0
    assert math.isclose(C.migration_factor(2, 8, 1.0), 0.75)
    assert math.isclose(C.sparse_bytes(2, 8, 1.0, 100.0), 175.0)
    assert math.isclose(C.sparse_bytes(2, 8, 1.0, 100.0, localadamw=True), 525.0)


def test_flops_per_token_limits():
    layers = [C.MoELayerCost(F_ffn=100.0, F_gate=10.0, N_e=64, k=2)] * 3
    full = 50.0 + 3 * (100.0 + 10.0)
    # full replica: every expert local, nothing skipped
    assert math.isclose(C.flops_per_token(50.0, layers, 8, 8), full)
    assert math.isclose(C.flops_per_token(50.0, layers, 8, 8, skip_token=True), full)
    # N_le >= k: the FFN term is unchanged, the router shrinks to N_le / N_e
    assert math.isclose(C.flops_per_token(50.0, layers, 2, 8), 50.0 + 3 * (100.0 + 2.5))
    # skip-token scales the FFN term by sigma_st = N_le / N_e
    assert math.isclose(C.flops_per_token(50.0, layers, 2, 8, skip_token=True),
                        50.0 + 3 * (25.0 + 2.5))
    # N_le < k: min(k, N_le) / k of the FFN
    one = [C.MoELayerCost(F_ffn=100.0, F_gate=10.0, N_e=8, k=2)]
    assert math.isclose(C.flops_per_token(0.0, one, 1, 8), 50.0 + 10.0 / 8)


def test_memory_bytes_per_token_and_time():
    assert C.BYTES_PER_PARAM == 18
    assert C.steady_state_memory(8e9, 1e9, 8, 8) == 9e9 * 18
    assert C.steady_state_memory(8e9, 1e9, 1, 8) == 2e9 * 18
    # BPT = B_site / (K B_l), B_l = B_g / M
    assert math.isclose(C.bytes_per_token(1e9, 32, 8 * 4096, 8), 1e9 / (32 * 4096))
    tc = C.t_comp(6e9, 8 * 4096, 8, 0.4, 2.5e15)
    assert math.isclose(tc, 6e9 * 4096 / 1e15)
    tm = C.t_comm(1e9, 2e9, 1.25e8, rho=0.5)
    assert math.isclose(tm, 12.0)
    # alpha = 1: communication fully overlapped, only compute remains
    assert math.isclose(C.t_total(1e9, 8, 4096, 32, tc, tm, alpha=1.0), 1e9 / (8 * 4096) * tc)
    assert C.t_total(1e9, 8, 4096, 32, tc, tm) > C.t_total(1e9, 8, 4096, 64, tc, tm)
