"""Each plausible mistake planted in the oracle must make at least one pin fail.

The mistakes are planted on the CPU, in the oracle module only, for the
duration of one test (pytest's monkeypatch restores the original).
"""
import numpy as np
import pytest

from oracle import moe_oracle as O
from tests import test_oracle_pins as P

FAST_PINS = [
    P.test_topk_matches_brute_force_sort, P.test_topk_tie_goes_to_lower_id,
    P.test_route_closed_form_golden, P.test_gate_special_cases_reduce_to_library_softmax_and_sigmoid,
    P.test_gate_invariants, P.test_routing_is_independent_of_residency,
    P.test_mask_is_set_membership_and_rank, P.test_dispatch_plan_is_a_stable_bijection,
    P.test_dispatch_empty_resident_set, P.test_single_expert_reduces_to_dense_swiglu_torch,
    P.test_swiglu_closed_form, P.test_full_replica_identity_no_renormalisation_over_survivors,
    P.test_fully_skipped_tokens_get_exact_zero, P.test_empty_resident_set_gives_zero_routed_output,
    lambda: P.test_backward_matches_central_differences("softmax_topk", "swiglu"),
    lambda: P.test_backward_matches_central_differences("softmax", "swiglu"),
    lambda: P.test_backward_matches_central_differences("sigmoid", "swiglu"),
    lambda: P.test_backward_matches_central_differences("sigmoid", "silu"),
    P.test_silu_expert_matches_torch_dense_and_autograd,
    P.test_silu_expert_single_resident_layer_is_dense_mlp,
    P.test_backward_matches_torch_autograd_dense_formulation, P.test_backward_is_linear_in_dy,
    P.test_expert_delta_closed_forms, P.test_expert_delta_within_fp32_bound_of_exact_mean,
    lambda: P.test_partitioned_router_brute_force(2, (1, 2, 4)),
    lambda: P.test_partitioned_router_brute_force(2, (3,)),
    P.test_partitioned_router_single_resident_expert_is_dense_swiglu,
    lambda: P.test_adamw_matches_torch_optim_adamw(0.0),
    lambda: P.test_adamw_matches_torch_optim_adamw(0.1),
    P.test_adamw_first_step_is_a_sign_step, P.test_outer_nesterov_matches_torch_sgd_nesterov,
    P.test_outer_nesterov_zero_delta_is_identity, P.test_replica_mean_closed_forms,
]

_orig = {name: getattr(O, name) for name in dir(O) if callable(getattr(O, name))}


def _topk_ties_high(z, k):
    z = np.asarray(z, np.float64)
    E = z.shape[1]
    return np.array([(E - 1 - np.argsort(-z[t, ::-1], kind="stable"))[:k] for t in range(z.shape[0])])


def _combine_renorm(Yp, w, inv_perm, y_add=None):
    w = np.array(w, np.float64)
    keep = inv_perm >= 0
    s = (w * keep).sum(1, keepdims=True)
    w = np.where(s > 0, w / np.where(s > 0, s, 1), w)
    return _orig["combine_fwd"](Yp, w, inv_perm, y_add)


def _bwd_variant(dY, X, G, U, Hh, w_gate_up, w_down, drop_u=False, gate_only=False):
    o = _orig["swiglu_bwd"](dY, X, G, U, Hh, w_gate_up, w_down)
    H = w_gate_up.shape[0] // 2
    G = np.asarray(G, np.float64); X = np.asarray(X, np.float64)
    if drop_u:
        sg = 1 / (1 + np.exp(-G))
        o["dG"] = o["dHh"] * (sg * (1 + G * (1 - sg)))
        o["dX"] = o["dG"] @ np.asarray(w_gate_up[:H], np.float64) + o["dU"] @ np.asarray(w_gate_up[H:], np.float64)
        o["dW_gate_up"] = np.concatenate([o["dG"].T @ X, o["dU"].T @ X])
    if gate_only:
        o["dX"] = o["dG"] @ np.asarray(w_gate_up[:H], np.float64)
    return o


def _gate_bwd_sign(z, idx, w, dw, gate="softmax_topk"):
    return -_orig["gate_bwd"](z, idx, w, dw, gate)


def _dispatch_tokens_desc(local, E_r):
    p = _orig["dispatch_plan"](local, E_r)
    local = np.asarray(local)
    k = local.shape[1]
    perm = []
    inv = np.full(local.shape, -1, np.int64)
    for r in range(E_r):
        for t in range(local.shape[0] - 1, -1, -1):
            for j in range(k):
                if local[t, j] == r:
                    inv[t, j] = len(perm)
                    perm.append(t * k + j)
    p.update(perm=np.array(perm, np.int64), inv_perm=inv)
    return p


def _swiglu_swap(X, w_gate_up, w_down):
    H = w_gate_up.shape[0] // 2
    return _orig["swiglu_fwd"](X, np.concatenate([w_gate_up[H:], w_gate_up[:H]]), w_down)


def _route_bwd_no_tau(x, w_router, idx, w, logits, dw, inv_tau=1.0, gate="softmax_topk"):
    return _orig["route_bwd"](x, w_router, idx, w, logits, dw, 1.0, gate)


def _delta_sign(theta_start, theta_now, peers):
    return _orig["expert_delta"](theta_now, theta_start, peers)


def _mask_global_ids(idx, resident):
    res = np.asarray(resident).astype(bool)
    return np.where(res[idx], idx, -1)


def _softmax_topk_full_denominator(z, idx, gate="softmax_topk"):
    if gate == "softmax_topk":
        gate = "softmax"
    return _orig["gate_weights"](z, idx, gate)


def _partition_keeps_all_router_rows(inp):
    out = _orig["partition_router"](inp)
    out["w_router"] = np.asarray(inp["w_router"])[:out["cfg"]["E"]]
    return out


def _adamw_weight_decay_sign(theta, grad, m, v, step, lr, beta1=0.9, beta2=0.95, eps=1e-8,
                             weight_decay=0.0):
    return _orig["adamw_step"](theta, grad, m, v, step, lr, beta1, beta2, eps, -weight_decay)


def _nesterov_old_buffer(theta_start, delta_avg, momentum, lr=0.7, mu=0.9):
    f32 = np.float32
    th, dl, b = (np.asarray(a, f32) for a in (theta_start, delta_avg, momentum))
    b1 = (f32(mu) * b + dl).astype(f32)
    return (th - f32(lr) * (dl + f32(mu) * b)).astype(f32), b1


def _replica_mean_over_peers_only(local, peers):
    f32 = np.float32
    acc = np.asarray(local, f32).copy()
    for p in peers:
        acc = (acc + np.asarray(p, f32)).astype(f32)
    return (acc * (f32(1.0) / f32(max(len(peers), 1)))).astype(f32)


def _silu_bwd_sigmoid_derivative(dY, X, A, Hh, w_up, w_down):
    o = _orig["silu_mlp_bwd"](dY, X, A, Hh, w_up, w_down)
    A = np.asarray(A, np.float64)
    o["dG"] = o["dHh"] / (1 + np.exp(-A))  # sigma(A) instead of silu'(A)
    o["dX"] = o["dG"] @ np.asarray(w_up, np.float64)
    o["dW_gate_up"] = o["dG"].T @ np.asarray(X, np.float64)
    return o


MUTANTS = {
    "SiLU expert backward uses sigma instead of silu'": ("silu_mlp_bwd", _silu_bwd_sigmoid_derivative),
    "partitioned router keeps the first rows, not the resident ones":
        ("partition_router", _partition_keeps_all_router_rows),
    "AdamW without bias correction": ("adamw_bias_corrections", lambda *a: (np.float32(1), np.float32(1))),
    "AdamW weight decay with the wrong sign": ("adamw_step", _adamw_weight_decay_sign),
    "Nesterov look-ahead uses the old momentum": ("outer_nesterov", _nesterov_old_buffer),
    "replica mean divides by the peer count": ("replica_mean", _replica_mean_over_peers_only),
    "topk ties to the higher id": ("topk_select", _topk_ties_high),
    "combine renormalises over surviving routes": ("combine_fwd", _combine_renorm),
    "dG drops the up factor": ("swiglu_bwd", lambda *a: _bwd_variant(*a, drop_u=True)),
    "dX drops the up-projection term": ("swiglu_bwd", lambda *a: _bwd_variant(*a, gate_only=True)),
    "gate backward sign flipped": ("gate_bwd", _gate_bwd_sign),
    "dispatch not stable in token order": ("dispatch_plan", _dispatch_tokens_desc),
    "gate and up projections swapped": ("swiglu_fwd", _swiglu_swap),
    "router backward ignores the temperature": ("route_bwd", _route_bwd_no_tau),
    "delta sign flipped": ("expert_delta", _delta_sign),
    "mask keeps global ids instead of ranks": ("mask_routes", _mask_global_ids),
    "top-k weights not renormalised": ("gate_weights", _softmax_topk_full_denominator),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(O, attr, fn)
    caught = 0
    for pin in FAST_PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught += 1
    assert caught >= 1, f"no pin caught: {name}"
