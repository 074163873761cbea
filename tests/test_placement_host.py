"""Host logic of the placement entry points (no GPU): the library's placement
and migration maps against the oracle's, and their argument checks."""
import numpy as np
import pytest

from oracle import moe_oracle as O
from paper_2606_19025_amd import binding as B


@pytest.fixture(scope="module")
def lib():
    return B.lib()


@pytest.mark.parametrize("N_e,O_e,M", [(64, 4, 8), (16, 1, 4), (16, 4, 4), (12, 2, 8), (8, 3, 6),
                                       (256, 2, 16)])
def test_placement_matches_oracle(lib, N_e, O_e, M):
    g = np.random.default_rng(N_e + 7 * O_e + 31 * M)
    for draw in range(5):
        ep = None if draw == 0 else g.permutation(N_e)
        wp = None if draw == 0 else g.permutation(M)
        assert np.array_equal(B.moe_gen_placement(N_e, O_e, M, ep, wp),
                              O.gen_placement(N_e, O_e, M, ep, wp))


def test_placement_rejects_bad_arguments(lib):
    with pytest.raises(B.MoeError):
        B.moe_gen_placement(10, 3, 4)  # 4 does not divide 30
    with pytest.raises(B.MoeError):
        B.moe_gen_placement(8, 5, 4)   # O_e > M
    with pytest.raises(B.MoeError):
        B.moe_gen_placement(8, 2, 4, expert_perm=[0, 1, 2, 3, 4, 5, 6, 6])


def test_migration_map_matches_oracle(lib):
    g = np.random.default_rng(5)
    for _ in range(20):
        prev = np.sort(g.choice(64, 16, replace=False))
        new = np.sort(g.choice(64, 16, replace=False))
        assert np.array_equal(B.moe_migration_map(prev, new), O.migration_map(prev, new))
    with pytest.raises(B.MoeError):
        B.moe_migration_map([1, 2], [3, 3])  # not strictly ascending


def test_warmup_lr_matches_oracle(lib):
    """The warm-up of experts new to a worker (Sec. 3.4; linear over W local
    steps from the restart of the expert's state) against the oracle's
    schedule, bit for bit, and its closed form."""
    g = np.random.default_rng(11)
    for W in (0, 1, 4, 32, 1000):
        steps = g.integers(0, 3 * max(W, 1) + 2, 64)
        for lr in (1e-3, 3e-4, 0.7):
            got = B.moe_warmup_lr(steps, lr, W)
            ref = np.array([lr * O.warmup_scale(int(s), W) for s in steps], np.float32)
            assert np.array_equal(got, ref), (W, lr)
    assert np.array_equal(B.moe_warmup_lr([0, 1, 2, 4, 9], 1.0, 4),
                          np.float32([0.0, 0.25, 0.5, 1.0, 1.0]))
    assert B.moe_warmup_lr([], 1e-3, 4).size == 0


def test_warmup_lr_rejects_bad_arguments(lib):
    with pytest.raises(B.MoeError):
        B.moe_warmup_lr([1, -1], 1e-3, 4)
    with pytest.raises(B.MoeError):
        B.moe_warmup_lr([1], float("nan"), 4)
