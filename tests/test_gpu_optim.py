"""GPU parity of the optimiser entry points (through the C ABI) against the
oracle: bit-exact fp32 for AdamW, the outer Nesterov step and the replica-group
mean, on ragged sizes and at the fine-grained workload's full parameter count
of its resident experts; the bf16 working copy is the nearest-even rounding of
the fp32 result."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_19025_amd import binding as B
from paper_2606_19025_amd import inputs as I

from .parity_helpers import say

pytestmark = pytest.mark.gpu


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def rne_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16).float().numpy()


@pytest.mark.parametrize("n,wd", [(1, 0.0), (4099, 0.0), (1_000_003, 0.1)])
def test_adamw_bit_exact(gpu_lib, n, wd):
    say(f"[optim] adamw n={n} wd={wd}")
    g = np.random.default_rng(n)
    theta = (g.standard_normal(n) * 0.02).astype(np.float32)
    th_d, m_d, v_d = dev(theta), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    lp = torch.full((n,), float("nan"), dtype=torch.bfloat16, device="cuda")
    th, m, v = theta, np.zeros(n, np.float32), np.zeros(n, np.float32)
    for t in range(1, 4):
        grad = (g.standard_normal(n) * 0.1).astype(np.float32)
        B.moe_adamw_step(th_d, dev(grad), m_d, v_d, n, t, 0.01, 0.9, 0.95, 1e-8, wd, lp)
        th, m, v = O.adamw_step(th, grad, m, v, t, 0.01, 0.9, 0.95, 1e-8, wd)
        torch.cuda.synchronize()
        assert np.array_equal(th_d.cpu().numpy(), th), f"theta differs at step {t}"
        assert np.array_equal(m_d.cpu().numpy(), m) and np.array_equal(v_d.cpu().numpy(), v)
        assert np.array_equal(lp.float().cpu().numpy(), rne_bf16(th))


@pytest.mark.parametrize("n", [3, 4096, 777_777])
def test_outer_nesterov_bit_exact(gpu_lib, n):
    say(f"[optim] outer nesterov n={n}")
    g = np.random.default_rng(n + 1)
    start = (g.standard_normal(n) * 0.02).astype(np.float32)
    s_d, now_d = dev(start), dev(start + 1.0)
    b_d = torch.zeros(n, device="cuda")
    lp = torch.full((n,), float("nan"), dtype=torch.bfloat16, device="cuda")
    th, b = start, np.zeros(n, np.float32)
    for _ in range(3):
        delta = (g.standard_normal(n) * 1e-3).astype(np.float32)
        B.moe_outer_nesterov(s_d, now_d, dev(delta), b_d, n, 0.7, 0.9, lp)
        th, b = O.outer_nesterov(th, delta, b, 0.7, 0.9)
        torch.cuda.synchronize()
        assert np.array_equal(s_d.cpu().numpy(), th)
        assert np.array_equal(now_d.cpu().numpy(), th), "the next round starts from theta"
        assert np.array_equal(b_d.cpu().numpy(), b)
        assert np.array_equal(lp.float().cpu().numpy(), rne_bf16(th))


@pytest.mark.parametrize("n,n_peers", [(5, 0), (4097, 1), (300_001, 3), (1000, 16)])
def test_replica_mean_bit_exact(gpu_lib, n, n_peers):
    g = np.random.default_rng(n + n_peers)
    x = g.standard_normal(n).astype(np.float32)
    peers = [g.standard_normal(n).astype(np.float32) for _ in range(n_peers)]
    ref = O.replica_mean(x, peers)
    x_d = dev(x)
    out = torch.full_like(x_d, float("nan"))
    B.moe_replica_mean(x_d, [dev(p) for p in peers], n_peers, n, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy(), ref)
    B.moe_replica_mean(x_d, [dev(p) for p in peers], n_peers, n, x_d)  # in place
    torch.cuda.synchronize()
    assert np.array_equal(x_d.cpu().numpy(), ref)


def test_adamw_full_size_resident_experts(gpu_lib):
    """The fine-grained workload's 16 resident experts (3 H d parameters each)."""
    cfg = I.workload(2, 42)
    n = cfg["E_r"] * 3 * cfg["H"] * cfg["d"]
    say(f"[optim] adamw full size n={n}")
    dpar = I.make_delta_inputs(2, n)
    theta, grad = dpar["theta_start"], dpar["peers"][0] * np.float32(100)
    m0 = (dpar["peers"][1] * np.float32(10)).astype(np.float32)
    v0 = (dpar["peers"][2] * dpar["peers"][2] * np.float32(100)).astype(np.float32)
    del dpar
    th_d, m_d, v_d = dev(theta), dev(m0), dev(v0)
    B.moe_adamw_step(th_d, dev(grad), m_d, v_d, n, 7, 3e-4, 0.9, 0.95, 1e-8, 0.0, None)
    th, m, v = O.adamw_step(theta, grad, m0, v0, 7, 3e-4, 0.9, 0.95, 1e-8, 0.0)
    torch.cuda.synchronize()
    assert np.array_equal(th_d.cpu().numpy(), th)
    assert np.array_equal(m_d.cpu().numpy(), m) and np.array_equal(v_d.cpu().numpy(), v)


def test_copy_expert_rows_bit_exact(gpu_lib):
    """Migration copies: rows from a store by index (zeros for -1) into
    consecutive rows, and rows back into chosen rows of a store."""
    g = np.random.default_rng(51)
    row_len, n_store = 3 * 64 * 128 + 4, 12
    store = g.standard_normal((n_store, row_len)).astype(np.float32)
    idx = np.array([3, -1, 0, 11, -1, 7], np.int32)
    out = torch.empty(len(idx), row_len, device="cuda")
    B.moe_copy_expert_rows(dev(store), idx, out, len(idx), row_len)
    torch.cuda.synchronize()
    ref = np.where(idx[:, None] >= 0, store[np.maximum(idx, 0)], 0.0).astype(np.float32)
    assert np.array_equal(out.cpu().numpy(), ref)
    back = dev(store)
    rows = np.array([0, 2, 3, 5], np.int32)
    dst_rows = np.array([9, 1, 4, 6], np.int32)
    B.moe_copy_expert_rows(out, rows, back, len(rows), row_len, dst_row=dst_rows)
    torch.cuda.synchronize()
    ref_back = store.copy()
    ref_back[dst_rows] = ref[rows]
    assert np.array_equal(back.cpu().numpy(), ref_back)


def test_adamw_rows_with_own_steps_and_rates(gpu_lib):
    """Per-expert step counts and learning rates (restarted experts with a
    warm-up) give row by row the single-array AdamW of the oracle."""
    g = np.random.default_rng(52)
    n_rows, row_len = 6, 4100
    theta = (g.standard_normal((n_rows, row_len)) * 0.02).astype(np.float32)
    m0 = (g.standard_normal((n_rows, row_len)) * 1e-3).astype(np.float32)
    v0 = (g.standard_normal((n_rows, row_len)) ** 2 * 1e-6).astype(np.float32)
    grad = (g.standard_normal((n_rows, row_len)) * 0.1).astype(np.float32)
    steps = np.array([7, 7, 1, 1, 7, 3], np.int32)
    lr = np.array([1e-3, 1e-3, 1e-3 * O.warmup_scale(1, 4), 1e-3 * O.warmup_scale(1, 4), 1e-3,
                   1e-3 * O.warmup_scale(3, 4)], np.float32)
    th_d, m_d, v_d = dev(theta), dev(m0), dev(v0)
    lp = torch.full((n_rows, row_len), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.moe_adamw_step_rows(th_d, dev(grad), m_d, v_d, n_rows, row_len, steps, lr, theta_bf16=lp)
    torch.cuda.synchronize()
    for r in range(n_rows):
        th, m, v = O.adamw_step(theta[r], grad[r], m0[r], v0[r], int(steps[r]), float(lr[r]))
        assert np.array_equal(th_d[r].cpu().numpy(), th), r
        assert np.array_equal(m_d[r].cpu().numpy(), m) and np.array_equal(v_d[r].cpu().numpy(), v)
        assert np.array_equal(lp[r].float().cpu().numpy(), rne_bf16(th))
