"""A round boundary with random placement, end to end on the GPU through the C
ABI, against the oracle: the new placement and migration map, the migrated
weights (from the global store, with their bf16 working copy) and optimiser
state (kept for experts the worker already held, restarted otherwise), then a
local step of the layer on the new resident set and the per-expert AdamW
update with the warm-up of the reassigned experts."""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_19025_amd import binding as B
from paper_2606_19025_amd import inputs as I
from paper_2606_19025_amd.layer import ResidentMoELayer

from .parity_helpers import TOL, assert_close, dev, gpu_outputs, say

pytestmark = pytest.mark.gpu

N_E, O_E, M = 8, 2, 4
T, D, K, H = 512, 128, 2, 128
WARMUP = 4


def f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def test_random_placement_round_boundary(gpu_lib):
    g = np.random.default_rng(61)
    N_le = N_E * O_E // M
    gu_len, dn_len = 2 * H * D, D * H
    # the server's model of all experts (fp32), the worker's previous set and state
    store_gu = (g.standard_normal((N_E, gu_len)) * 0.02).astype(np.float32)
    store_dn = (g.standard_normal((N_E, dn_len)) * 0.02).astype(np.float32)
    prev = O.gen_placement(N_E, O_E, M)[0]
    m_old = (g.standard_normal((N_le, gu_len)) * 1e-3).astype(np.float32)
    v_old = (g.standard_normal((N_le, gu_len)) ** 2 * 1e-6).astype(np.float32)
    steps_old = np.array([9, 9, 9, 9])
    # new random placement: the worker's new set and what moves
    ep, wp = g.permutation(N_E), g.permutation(M)
    new = B.moe_gen_placement(N_E, O_E, M, ep, wp)[0]
    assert np.array_equal(new, O.gen_placement(N_E, O_E, M, ep, wp)[0])
    mig = B.moe_migration_map(prev, new)
    assert np.array_equal(mig, O.migration_map(prev, new))
    say(f"[placement] prev {prev.tolist()} new {new.tolist()} map {mig.tolist()}")

    # migration on the GPU: weights from the store (+ bf16 copy), state by the map
    theta_gu = torch.full((N_le, gu_len), float("nan"), device="cuda")
    theta_dn = torch.full((N_le, dn_len), float("nan"), device="cuda")
    w_gu = torch.full((N_le, 2 * H, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    w_dn = torch.full((N_le, D, H), float("nan"), dtype=torch.bfloat16, device="cuda")
    B.moe_copy_expert_rows(f32(store_gu), new, theta_gu, N_le, gu_len, dst_bf16=w_gu)
    B.moe_copy_expert_rows(f32(store_dn), new, theta_dn, N_le, dn_len, dst_bf16=w_dn)
    m_new = torch.full((N_le, gu_len), float("nan"), device="cuda")
    v_new = torch.full((N_le, gu_len), float("nan"), device="cuda")
    B.moe_copy_expert_rows(f32(m_old), mig, m_new, N_le, gu_len)
    B.moe_copy_expert_rows(f32(v_old), mig, v_new, N_le, gu_len)
    steps = np.where(mig >= 0, steps_old[np.maximum(mig, 0)], 0)
    torch.cuda.synchronize()
    assert np.array_equal(theta_gu.cpu().numpy(), store_gu[new])
    assert np.array_equal(theta_dn.cpu().numpy(), store_dn[new])
    assert np.array_equal(w_gu.float().cpu().numpy().reshape(N_le, -1),
                          torch.from_numpy(store_gu[new]).to(torch.bfloat16).float().numpy())
    keep = mig >= 0
    assert np.array_equal(m_new.cpu().numpy()[keep], m_old[mig[keep]])
    assert np.all(m_new.cpu().numpy()[~keep] == 0) and np.all(v_new.cpu().numpy()[~keep] == 0)

    # one local step of the layer on the new resident set
    res = np.zeros(N_E, np.uint8)
    res[new] = 1
    x = I.bf16_round(g.standard_normal((T, D)).astype(np.float32))
    dy = I.bf16_round(g.standard_normal((T, D)).astype(np.float32))
    w_router = I.bf16_round((g.standard_normal((N_E, D)) * 0.08).astype(np.float32))
    L = ResidentMoELayer(T, D, N_E, K, H, np.isin(np.arange(N_E), prev).astype(np.uint8),
                         dtype=torch.bfloat16)
    L.set_resident(res)
    xb, dyb, wrb = (dev(a, torch.bfloat16) for a in (x, dy, w_router))
    L.forward(xb, wrb, w_gu, w_dn)
    L.backward(dyb, xb, wrb, w_gu, w_dn)
    torch.cuda.synchronize()
    inp = dict(cfg=dict(T=T, d=D, E=N_E, k=K, H=H, E_r=N_le, resident=new.tolist(),
                        dtype="bf16"),
               x=x, dy=dy, w_router=w_router, resident=res, router_bias=None,
               w_gate_up=w_gu.float().cpu().numpy(), w_down=w_dn.float().cpu().numpy())
    out = gpu_outputs(L)
    fwd = O.layer_fwd(inp, logits=out["logits"])
    assert np.array_equal(out["local"], fwd["local"])
    assert_close("y", out["y"], fwd["y"], TOL["bf16"])
    bwd = O.layer_bwd(inp, fwd, dy)
    assert_close("dW_gate_up", out["dW_gate_up"], bwd["dW_gate_up"], TOL["bf16"])

    # per-expert AdamW: kept experts continue their count, new ones restart
    # with the warm-up
    steps = steps + 1
    lr = B.moe_warmup_lr(steps, 1e-3, WARMUP)
    assert np.array_equal(lr, np.array([1e-3 * O.warmup_scale(int(s), WARMUP) for s in steps],
                                       np.float32))
    # the kept experts are past their warm-up, the new ones start it
    assert np.all(lr[mig >= 0] == np.float32(1e-3)) and np.all(lr[mig < 0] < np.float32(1e-3))
    grad = L.dw_gate_up.reshape(N_le, gu_len)
    th_before, m_before, v_before = (t.cpu().numpy().copy() for t in (theta_gu, m_new, v_new))
    g_host = grad.cpu().numpy()
    B.moe_adamw_step_rows(theta_gu, grad, m_new, v_new, N_le, gu_len, steps, lr, theta_bf16=w_gu)
    torch.cuda.synchronize()
    for r in range(N_le):
        th, mm, vv = O.adamw_step(th_before[r], g_host[r], m_before[r], v_before[r],
                                  int(steps[r]), float(lr[r]))
        assert np.array_equal(theta_gu[r].cpu().numpy(), th), r
        assert np.array_equal(m_new[r].cpu().numpy(), mm) and np.array_equal(v_new[r].cpu().numpy(), vv)
