"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these compares the oracle with itself: each check uses brute force on
tiny inputs, a closed form, an invariant, a library routine in a special case
that reduces to it, or finite differences.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special as sps

from oracle import moe_oracle as O
from paper_2606_19025_amd import inputs as I

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_inputs(T=24, d=16, E=6, k=2, H=8, resident=(1, 2, 4), seed=0, shared=0, bias=False,
                expert="swiglu"):
    g = np.random.default_rng(seed)
    Er = len(resident)
    res = np.zeros(E, np.uint8)
    res[list(resident)] = 1
    r1 = 2 if expert == "swiglu" else 1  # rows of the first weight per hidden unit
    inp = dict(cfg=dict(T=T, d=d, E=E, k=k, H=H, E_r=Er, resident=sorted(resident), expert=expert),
               x=g.standard_normal((T, d)), w_router=g.standard_normal((E, d)) * 0.5,
               w_gate_up=g.standard_normal((Er, r1 * H, d)) * 0.3,
               w_down=g.standard_normal((Er, d, H)) * 0.3, resident=res,
               router_bias=g.standard_normal(E) * 0.3 if bias else None)
    if shared:
        inp["shared_gate_up"] = g.standard_normal((1, r1 * shared, d)) * 0.3
        inp["shared_down"] = g.standard_normal((1, d, shared)) * 0.3
    return inp


# ---------------------------------------------------------------- routing

def test_topk_matches_brute_force_sort():
    g = np.random.default_rng(1)
    for E, k in [(8, 2), (16, 6), (5, 5), (64, 8)]:
        z = g.standard_normal((50, E))
        # round to a coarse grid so that exact ties occur often
        z = np.round(z * 2) / 2
        idx = O.topk_select(z, k)
        for t in range(z.shape[0]):
            brute = sorted(range(E), key=lambda e: (-z[t, e], e))[:k]
            assert list(idx[t]) == brute


def test_topk_tie_goes_to_lower_id():
    z = np.array([[1.0, 3.0, 3.0, 0.5, 3.0]])
    assert list(O.topk_select(z, 3)[0]) == [1, 2, 4]
    assert list(O.topk_select(z, 2)[0]) == [1, 2]


def test_route_closed_form_golden():
    # logits ln(1..4): top-2 = experts 3, 2 with weights 4/7, 3/7 (hand-derived)
    with open(os.path.join(GOLDEN, "route_closed_form.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        z = np.log(np.array([case["exp_logits"]], dtype=np.float64))
        idx = O.topk_select(z, case["k"])
        w = O.gate_weights(z, idx, case["gate"])
        assert list(idx[0]) == case["idx"]
        np.testing.assert_allclose(w[0], [eval(s) for s in case["w"]], rtol=1e-14)


def test_gate_special_cases_reduce_to_library_softmax_and_sigmoid():
    g = np.random.default_rng(2)
    z = g.standard_normal((40, 7)) * 3
    # k = E: renormalised-over-top-k softmax is the full softmax (scipy)
    idx = O.topk_select(z, 7)
    w = O.gate_weights(z, idx, "softmax_topk")
    ref = sps.softmax(z, axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(ref, idx, 1), rtol=1e-13)
    # raw softmax mode: probabilities of the selected experts (scipy)
    idx3 = O.topk_select(z, 3)
    np.testing.assert_allclose(O.gate_weights(z, idx3, "softmax"),
                               np.take_along_axis(ref, idx3, 1), rtol=1e-13)
    # sigmoid gate (sigma-MoE, App. B.3.2): logistic function (scipy)
    np.testing.assert_allclose(O.gate_weights(z, idx3, "sigmoid"),
                               sps.expit(np.take_along_axis(z, idx3, 1)), rtol=1e-13)


def test_gate_invariants():
    g = np.random.default_rng(3)
    z = g.standard_normal((60, 16)) * 2
    for k in (1, 2, 6):
        idx = O.topk_select(z, k)
        w = O.gate_weights(z, idx, "softmax_topk")
        np.testing.assert_allclose(w.sum(1), 1.0, rtol=1e-14)  # renormalised value
        assert np.all(np.diff(w, axis=1) <= 0)  # ordered like the logits
        if k == 1:
            assert np.all(w == 1.0)
        # renormalised weights are the raw probabilities divided by their sum
        raw = O.gate_weights(z, idx, "softmax")
        np.testing.assert_allclose(w, raw / raw.sum(1, keepdims=True), rtol=1e-13)
        assert np.all(raw.sum(1) <= 1 + 1e-14)


def test_routing_is_independent_of_residency():
    inp = tiny_inputs()
    a = O.route(inp["x"], inp["w_router"], 2, inp["resident"])
    b = O.route(inp["x"], inp["w_router"], 2, np.ones(6, np.uint8))
    assert np.array_equal(a["idx"], b["idx"]) and np.array_equal(a["w"], b["w"])


def test_mask_is_set_membership_and_rank():
    g = np.random.default_rng(4)
    E = 12
    for _ in range(10):
        res = (g.random(E) < 0.5).astype(np.uint8)
        idx = np.array([g.permutation(E)[:4] for _ in range(9)])
        local = O.mask_routes(idx, res)
        resid = sorted(np.flatnonzero(res).tolist())
        for t in range(9):
            for j in range(4):
                e = idx[t, j]
                assert local[t, j] == (resid.index(e) if e in resid else -1)
    idx = np.array([[0, 1], [2, 3]])
    assert np.all(O.mask_routes(idx, np.ones(4, np.uint8)) >= 0)
    assert np.all(O.mask_routes(idx, np.zeros(4, np.uint8)) == -1)


# ---------------------------------------------------------------- dispatch

def test_dispatch_plan_is_a_stable_bijection():
    g = np.random.default_rng(5)
    T, k, Er = 40, 3, 5
    local = np.full((T, k), -1)
    for t in range(T):
        ch = g.permutation(Er + 3)[:k]  # ids >= Er stand for ghosts
        local[t] = np.where(ch < Er, ch, -1)
    p = O.dispatch_plan(local, Er)
    n = int((local >= 0).sum())
    assert p["counts"].sum() == n == p["offsets"][-1] == len(p["perm"])
    assert np.array_equal(p["offsets"], np.concatenate([[0], np.cumsum(p["counts"])]))
    # bijection between slots and resident routes
    assert len(set(p["perm"].tolist())) == n
    for q, rid in enumerate(p["perm"]):
        assert p["inv_perm"][rid // k, rid % k] == q
    assert np.all((p["inv_perm"] >= 0) == (local >= 0))
    # brute force: sort resident routes by (expert, token)
    brute = sorted((local[t, j], t, j) for t in range(T) for j in range(k) if local[t, j] >= 0)
    assert [t * k + j for (_, t, j) in brute] == p["perm"].tolist()


def test_dispatch_empty_resident_set():
    local = np.full((7, 2), -1)
    p = O.dispatch_plan(local, 3)
    assert p["offsets"].tolist() == [0, 0, 0, 0] and len(p["perm"]) == 0
    assert np.all(p["inv_perm"] == -1)


# ---------------------------------------------------------------- expert FFN

def test_single_expert_reduces_to_dense_swiglu_torch():
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    inp = tiny_inputs(E=1, k=1, resident=(0,), shared=0)
    fwd = O.layer_fwd(inp)
    x = torch.tensor(inp["x"], dtype=torch.float64)
    Wgu = torch.tensor(inp["w_gate_up"][0]); Wd = torch.tensor(inp["w_down"][0])
    H = Wgu.shape[0] // 2
    ref = F.linear(F.silu(F.linear(x, Wgu[:H])) * F.linear(x, Wgu[H:]), Wd)
    np.testing.assert_allclose(fwd["y"], ref.numpy(), rtol=1e-12, atol=1e-13)
    assert np.all(fwd["w"] == 1.0)


def test_swiglu_closed_form():
    # x = e_0, Wg row = ln(3) e_0, Wu row = 2 e_0, Wd = [[1]] -> y = ln3 * 3/4 * 2
    X = np.array([[1.0, 0.0]])
    Wgu = np.array([[math.log(3.0), 0.0], [2.0, 0.0]])
    Wd = np.array([[1.0], [0.5]])
    o = O.swiglu_fwd(X, Wgu, Wd)
    np.testing.assert_allclose(o["Y"], [[1.5 * math.log(3.0), 0.75 * math.log(3.0)]], rtol=1e-15)
    # silu'(g) = s(1 + g(1 - s)) at g = ln 3, s = 3/4
    b = O.swiglu_bwd(np.array([[1.0, 0.0]]), X, o["G"], o["U"], o["Hh"], Wgu, Wd)
    np.testing.assert_allclose(b["dG"], [[2.0 * 0.75 * (1 + math.log(3.0) * 0.25)]], rtol=1e-14)
    np.testing.assert_allclose(b["dU"], [[0.75 * math.log(3.0)]], rtol=1e-14)


# ---------------------------------------------------------------- skip token

def _full_replica_layer(inp, gi):
    """Same draw with every expert resident (ghost weights supplied by the test)."""
    cfg = dict(inp["cfg"])
    E, H, d = cfg["E"], cfg["H"], cfg["d"]
    wgu = np.zeros((E, 2 * H, d)); wd = np.zeros((E, d, H))
    for r, e in enumerate(cfg["resident"]):
        wgu[e], wd[e] = inp["w_gate_up"][r], inp["w_down"][r]
    for r, e in enumerate(gi["ids"]):
        wgu[e], wd[e] = gi["gate_up"][r], gi["down"][r]
    cfg.update(E_r=E, resident=list(range(E)))
    full = dict(inp, cfg=cfg, w_gate_up=wgu, w_down=wd, resident=np.ones(E, np.uint8))
    return full


def test_full_replica_identity_no_renormalisation_over_survivors():
    inp = tiny_inputs(T=30, E=6, k=3, resident=(0, 3, 4), shared=4)
    g = np.random.default_rng(9)
    ghosts = [1, 2, 5]
    gi = dict(ids=ghosts, gate_up=g.standard_normal((3, 16, 16)) * 0.3,
              down=g.standard_normal((3, 16, 8)) * 0.3)
    part = O.layer_fwd(inp)
    full = O.layer_fwd(_full_replica_layer(inp, gi))
    # y_full = y_resident + sum over ghost routes of w * FFN_ghost(x)
    extra = np.zeros_like(part["y"])
    for t in range(30):
        for j in range(3):
            e = part["idx"][t, j]
            if e in ghosts:
                r = ghosts.index(e)
                extra[t] += part["w"][t, j] * O.swiglu_fwd(inp["x"][t:t + 1], gi["gate_up"][r], gi["down"][r])["Y"][0]
    np.testing.assert_allclose(part["y"] + extra, full["y"], rtol=1e-12, atol=1e-12)


def test_fully_skipped_tokens_get_exact_zero():
    inp = tiny_inputs(T=60, E=8, k=2, resident=(0,), shared=0)
    fwd = O.layer_fwd(inp)
    dy = np.random.default_rng(7).standard_normal((60, 16))
    bwd = O.layer_bwd(inp, fwd, dy)
    skipped = np.all(fwd["local"] < 0, axis=1)
    assert skipped.sum() > 10
    assert np.all(fwd["y"][skipped] == 0.0)
    assert np.all(bwd["dz"][skipped] == 0.0)  # w * (0 - <w, 0>) = 0
    assert np.all(bwd["dx"][skipped] == 0.0)
    assert np.all(bwd["dw"][fwd["local"] < 0] == 0.0)


def test_empty_resident_set_gives_zero_routed_output():
    inp = tiny_inputs(T=20, E=4, k=2, resident=(), shared=0)
    inp["w_gate_up"] = np.zeros((0, 16, 16)); inp["w_down"] = np.zeros((0, 16, 8))
    fwd = O.layer_fwd(inp)
    assert fwd["offsets"][-1] == 0 and fwd["y"].shape == (20, 16) and np.all(fwd["y"] == 0.0)


def test_skip_fraction_matches_sigma_st():
    with open(os.path.join(GOLDEN, "skip_fraction.json")) as f:
        gold = json.load(f)
    for case in gold["cases"]:
        wl = I.workload(case["workload"])
        assert case["E_r"] == wl["E_r"] and case["E"] == wl["E"]
        inp = I.make_layer_inputs(case["workload"], T=case["T_sample"], with_experts=False)
        r = O.route(inp["x"], inp["w_router"], wl["k"], inp["resident"])
        frac = float((r["local"] >= 0).mean())
        assert abs(frac - case["sigma_st"]) < case["tol"], (case, frac)


def test_zipf_workload_skips_seventy_percent_of_top1():
    inp = I.make_layer_inputs(3, with_experts=False)
    r = O.route(inp["x"], inp["w_router"], 2, inp["resident"], bias=inp["router_bias"])
    frac = float((r["local"][:, 0] < 0).mean())
    assert abs(frac - 0.70) <= 0.01, frac


# ---------------------------------------------------------------- backward

def _loss(inp, dy, gate, inv_tau, idx_ref):
    f = O.layer_fwd(inp, inv_tau=inv_tau, gate=gate)
    assert np.array_equal(f["idx"], idx_ref), "finite-difference step flipped a top-k choice"
    return float((f["y"] * dy).sum())


@pytest.mark.parametrize("gate,expert", [("softmax_topk", "swiglu"), ("softmax", "swiglu"),
                                          ("sigmoid", "swiglu"), ("sigmoid", "silu")])
def test_backward_matches_central_differences(gate, expert):
    inp = tiny_inputs(T=10, d=6, E=5, k=2, H=4, resident=(0, 2, 3), shared=3, bias=True, seed=11,
                      expert=expert)
    inv_tau = 0.7
    g = np.random.default_rng(12)
    dy = g.standard_normal((10, 6))
    fwd = O.layer_fwd(inp, inv_tau=inv_tau, gate=gate)
    bwd = O.layer_bwd(inp, fwd, dy, inv_tau=inv_tau, gate=gate)
    # margin guard: skip if any token's k-th / (k+1)-th logits are close
    zs = np.sort(fwd["logits"], axis=1)[:, ::-1]
    assert np.min(zs[:, 1] - zs[:, 2]) > 1e-4
    checks = [("x", bwd["dx"]), ("w_router", bwd["dW_router"]), ("w_gate_up", bwd["dW_gate_up"]),
              ("w_down", bwd["dW_down"]), ("router_bias", bwd["d_bias"]),
              ("shared_gate_up", bwd["shared"]["dW_gate_up"][None]),
              ("shared_down", bwd["shared"]["dW_down"][None])]
    for name, grad in checks:
        base = inp[name]
        flat = base.reshape(-1)
        sel = g.choice(flat.size, size=min(25, flat.size), replace=False)
        for i in sel:
            h = 1e-6 * max(1.0, abs(flat[i]))
            old = flat[i]
            flat[i] = old + h
            lp = _loss(inp, dy, gate, inv_tau, fwd["idx"])
            flat[i] = old - h
            lm = _loss(inp, dy, gate, inv_tau, fwd["idx"])
            flat[i] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(fd)), (name, i, fd, grad.reshape(-1)[i])


def test_backward_matches_torch_autograd_dense_formulation():
    """Independent formulation: every expert on every token, masked by the
    (fixed) resident top-k gates, differentiated by torch.autograd in fp64."""
    torch = pytest.importorskip("torch")
    F = torch.nn.functional
    inp = tiny_inputs(T=16, d=8, E=6, k=3, H=5, resident=(1, 2, 5), shared=2, seed=21)
    fwd = O.layer_fwd(inp)
    dy = np.random.default_rng(22).standard_normal((16, 8))
    bwd = O.layer_bwd(inp, fwd, dy)
    t = lambda a: torch.tensor(np.asarray(a, np.float64), requires_grad=True)
    x, wr, wgu, wd = t(inp["x"]), t(inp["w_router"]), t(inp["w_gate_up"]), t(inp["w_down"])
    sgu, sd = t(inp["shared_gate_up"]), t(inp["shared_down"])
    z = x @ wr.T
    sel = torch.tensor(fwd["idx"])
    zk = torch.gather(z, 1, sel)
    wk = torch.softmax(zk, dim=1)
    H = 5
    y = torch.zeros(16, 8, dtype=torch.float64)
    for r, e in enumerate(inp["cfg"]["resident"]):
        gate = (wk * (sel == e)).sum(1, keepdim=True)
        he = F.silu(x @ wgu[r, :H].T) * (x @ wgu[r, H:].T)
        y = y + gate * (he @ wd[r].T)
    y = y + (F.silu(x @ sgu[0, :2].T) * (x @ sgu[0, 2:].T)) @ sd[0].T
    (y * torch.tensor(dy)).sum().backward()
    np.testing.assert_allclose(fwd["y"], y.detach().numpy(), rtol=1e-12, atol=1e-13)
    for a, b in [(bwd["dx"], x.grad), (bwd["dW_router"], wr.grad), (bwd["dW_gate_up"], wgu.grad),
                 (bwd["dW_down"], wd.grad), (bwd["shared"]["dW_gate_up"], sgu.grad[0]),
                 (bwd["shared"]["dW_down"], sd.grad[0])]:
        np.testing.assert_allclose(a, b.numpy(), rtol=1e-11, atol=1e-12)


def test_backward_is_linear_in_dy():
    inp = tiny_inputs(T=12, shared=2, seed=31)
    fwd = O.layer_fwd(inp)
    g = np.random.default_rng(32)
    a, b = g.standard_normal((12, 16)), g.standard_normal((12, 16))
    ga, gb, gab = (O.layer_bwd(inp, fwd, v) for v in (a, b, 2 * a - 3 * b))
    for key in ("dx", "dW_router", "dW_gate_up", "dW_down"):
        np.testing.assert_allclose(gab[key], 2 * ga[key] - 3 * gb[key], rtol=1e-10, atol=1e-12)


# ---------------------------------------------------------------- expert delta

def test_expert_delta_closed_forms():
    g = np.random.default_rng(41)
    a = g.standard_normal(1000).astype(np.float32)
    dl, avg = O.expert_delta(a, a, [np.zeros(1000, np.float32)] * 3)
    assert np.all(dl == 0) and np.all(avg == 0)
    # two copies of the same delta average to that delta exactly
    b = (a + g.standard_normal(1000).astype(np.float32) * 1e-3).astype(np.float32)
    dl, avg = O.expert_delta(a, b, [(a - b).astype(np.float32)])
    assert np.array_equal(avg, dl)
    # small integers: every fp32 operation is exact -> arithmetic mean
    ints = [g.integers(-50, 50, 1000).astype(np.float32) for _ in range(5)]
    dl, avg = O.expert_delta(ints[0], ints[1], ints[2:])
    exact = ((ints[0].astype(np.float64) - ints[1]) + ints[2] + ints[3] + ints[4]) / 4
    assert np.array_equal(avg.astype(np.float64), exact)


def test_expert_delta_within_fp32_bound_of_exact_mean():
    g = np.random.default_rng(42)
    n = 20000
    s = (g.standard_normal(n) * 0.02).astype(np.float32)
    now = (s + g.standard_normal(n) * 1e-3).astype(np.float32)
    peers = [(g.standard_normal(n) * 1e-3).astype(np.float32) for _ in range(3)]
    dl, avg = O.expert_delta(s, now, peers)
    exact = ((s.astype(np.float64) - now) + sum(p.astype(np.float64) for p in peers)) / 4
    mag = (np.abs(s.astype(np.float64) - now) + sum(np.abs(p.astype(np.float64)) for p in peers)) / 4
    assert np.all(np.abs(avg - exact) <= 6 * np.finfo(np.float32).eps * (mag + 1e-30))


# ---------------------------------------------------------------- partitioned router

@pytest.mark.parametrize("k,resident", [(2, (1, 2, 4)), (4, (0, 5)), (2, (3,))])
def test_partitioned_router_brute_force(k, resident):
    """Partitioned mode: a token's routes are the top-min(k, N_le) of its logits
    over the resident experts alone (per-token brute-force sort of plain dot
    products), all routes are local, every token executes exactly min(k, N_le)
    of them, and the gates are the softmax over the selected resident logits."""
    T, d = 20, 7
    inp = tiny_inputs(T=T, d=d, E=6, k=k, H=5, resident=resident, seed=21, bias=True)
    f = O.layer_fwd(O.partition_router(inp))
    res = sorted(resident)
    kk = min(k, len(res))
    for t in range(T):
        z = [sum(inp["x"][t, c] * inp["w_router"][e, c] for c in range(d)) + inp["router_bias"][e]
             for e in res]
        brute = sorted(range(len(res)), key=lambda i: (-z[i], i))[:kk]
        assert list(f["idx"][t]) == brute
        assert list(f["local"][t]) == brute
        zs = np.array([z[i] for i in brute])
        wref = np.exp(zs - zs.max())
        wref /= wref.sum()
        assert np.allclose(f["w"][t], wref, rtol=1e-12, atol=0)
    assert int(f["offsets"][-1]) == T * kk


def test_partitioned_router_with_every_expert_resident_is_skip_token():
    inp = tiny_inputs(T=16, d=6, E=5, k=2, H=4, resident=(0, 1, 2, 3, 4), seed=22, shared=3,
                      bias=True)
    a = O.layer_fwd(inp)
    b = O.layer_fwd(O.partition_router(inp))
    for key in ("idx", "w", "local", "perm", "inv_perm", "offsets"):
        assert np.array_equal(a[key], b[key]), key
    assert np.array_equal(a["y"], b["y"])


def test_partitioned_router_single_resident_expert_is_dense_swiglu():
    """N_le = 1 < k: every token takes its one local route with weight 1, so
    the routed output is the dense SwiGLU of that expert (checked against
    torch.nn.functional in fp64)."""
    torch = pytest.importorskip("torch")
    inp = tiny_inputs(T=12, d=6, E=4, k=2, H=5, resident=(2,), seed=23)
    f = O.layer_fwd(O.partition_router(inp))
    assert np.all(f["w"] == 1.0) and f["w"].shape == (12, 1)
    x = torch.from_numpy(inp["x"])
    wg = torch.from_numpy(inp["w_gate_up"][0, :5])
    wu = torch.from_numpy(inp["w_gate_up"][0, 5:])
    wd = torch.from_numpy(inp["w_down"][0])
    ref = (torch.nn.functional.silu(x @ wg.T) * (x @ wu.T)) @ wd.T
    assert np.allclose(f["y"], ref.numpy(), rtol=1e-12, atol=1e-14)


def test_partitioned_router_backward_matches_central_differences():
    inp = tiny_inputs(T=9, d=5, E=6, k=2, H=4, resident=(0, 3, 4, 5), seed=24, bias=True)
    part = O.partition_router(inp)
    g = np.random.default_rng(25)
    dy = g.standard_normal((9, 5))
    fwd = O.layer_fwd(part)
    bwd = O.layer_bwd(part, fwd, dy)
    zs = np.sort(fwd["logits"], axis=1)[:, ::-1]
    assert np.min(zs[:, 1] - zs[:, 2]) > 1e-4
    assert bwd["dW_router"].shape == (4, 5)
    for name, grad in [("x", bwd["dx"]), ("w_router", bwd["dW_router"]),
                       ("router_bias", bwd["d_bias"]), ("w_gate_up", bwd["dW_gate_up"])]:
        flat = part[name].reshape(-1)
        for i in g.choice(flat.size, size=min(20, flat.size), replace=False):
            h = 1e-6 * max(1.0, abs(flat[i]))
            old = flat[i]
            flat[i] = old + h
            lp = _loss(part, dy, "softmax_topk", 1.0, fwd["idx"])
            flat[i] = old - h
            lm = _loss(part, dy, "softmax_topk", 1.0, fwd["idx"])
            flat[i] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grad.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(fd)), (name, i)


# ---------------------------------------------------------------- optimisers

@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_adamw_matches_torch_optim_adamw(wd):
    """Three AdamW steps against torch.optim.AdamW on the CPU (fp32); the two
    order their fp32 operations differently, so they agree to a few ulps."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(31)
    n = 4096
    theta = (g.standard_normal(n) * 0.02).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(theta.copy()))
    opt = torch.optim.AdamW([p], lr=0.01, betas=(0.9, 0.95), eps=1e-8, weight_decay=wd)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    th = theta.copy()
    for t in range(1, 4):
        grad = (g.standard_normal(n) * 0.1).astype(np.float32)
        p.grad = torch.from_numpy(grad.copy())
        opt.step()
        th, m, v = O.adamw_step(th, grad, m, v, t, 0.01, 0.9, 0.95, 1e-8, wd)
        ref = p.detach().numpy()
        assert np.max(np.abs(th - ref)) <= 4e-7 * np.max(np.abs(ref)), t
        st = opt.state[p]
        # torch updates m by lerp, v by mul + addcmul: a few ulps apart
        # (normwise: single entries may cancel to near zero)
        for mine, theirs in ((m, st["exp_avg"].numpy()), (v, st["exp_avg_sq"].numpy())):
            assert np.max(np.abs(mine - theirs)) <= 1e-6 * np.max(np.abs(theirs))


def test_adamw_first_step_is_a_sign_step():
    """From zero moments, step 1 gives m/c1 = g and v/c2 = g^2 (up to
    rounding), so the update is lr * g / (|g| + eps), i.e. lr * sign(g)."""
    g = np.random.default_rng(32)
    theta = g.standard_normal(1000).astype(np.float32)
    grad = (g.standard_normal(1000) + np.sign(g.standard_normal(1000)) * 0.5).astype(np.float32)
    z = np.zeros(1000, np.float32)
    th, m, v = O.adamw_step(theta, grad, z, z, 1, 1e-3)
    # exact difference in fp64; theta' carries one rounding of |theta| ~ 1
    step = theta.astype(np.float64) - th.astype(np.float64)
    assert np.allclose(step, 1e-3 * np.sign(grad), rtol=1e-5, atol=2.5e-7)
    assert np.allclose(m, 0.1 * grad, rtol=1e-6) and np.allclose(v, 0.05 * grad * grad, rtol=1e-6)


def test_outer_nesterov_matches_torch_sgd_nesterov():
    """The outer step equals torch.optim.SGD(momentum=0.9, nesterov=True,
    lr=0.7) applied to the averaged pseudo-gradient, round after round."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(33)
    n = 2048
    theta = (g.standard_normal(n) * 0.02).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(theta.copy()))
    opt = torch.optim.SGD([p], lr=0.7, momentum=0.9, nesterov=True)
    b = np.zeros(n, np.float32)
    th = theta.copy()
    for _ in range(3):
        delta = (g.standard_normal(n) * 1e-3).astype(np.float32)
        p.grad = torch.from_numpy(delta.copy())
        opt.step()
        th, b = O.outer_nesterov(th, delta, b, 0.7, 0.9)
        ref = p.detach().numpy()
        assert np.max(np.abs(th - ref)) <= 2e-7 * np.max(np.abs(ref))
        assert np.allclose(b, opt.state[p]["momentum_buffer"].numpy(), rtol=1e-6, atol=1e-12)


def test_outer_nesterov_zero_delta_is_identity():
    th = np.random.default_rng(34).standard_normal(100).astype(np.float32)
    z = np.zeros(100, np.float32)
    th1, b1 = O.outer_nesterov(th, z, z)
    assert np.array_equal(th1, th) and np.array_equal(b1, z)


def test_replica_mean_closed_forms():
    g = np.random.default_rng(35)
    x = g.standard_normal(999).astype(np.float32)
    # identical copies over a power-of-two group: the mean is the copy, exactly
    assert np.array_equal(O.replica_mean(x, [x, x, x]), x)
    assert np.array_equal(O.replica_mean(x, [x]), x)
    # any copies: within the fp32 bound of the exact mean
    peers = [g.standard_normal(999).astype(np.float32) for _ in range(3)]
    exact = (x.astype(np.float64) + sum(p.astype(np.float64) for p in peers)) / 4
    got = O.replica_mean(x, peers)
    bound = 4 * 2.0 ** -24 * (np.abs(x) + sum(np.abs(p) for p in peers)).astype(np.float64)
    assert np.all(np.abs(got - exact) <= bound)


# ---------------------------------------------------------------- SiLU expert

def test_silu_expert_matches_torch_dense_and_autograd():
    """The paper's own expert (App. B.3.1) on every token of one dense expert:
    forward against torch.nn.functional.silu and backward against
    torch.autograd, in fp64 on the CPU."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(41)
    X, W1, W2 = g.standard_normal((13, 7)), g.standard_normal((5, 7)), g.standard_normal((7, 5))
    dY = g.standard_normal((13, 7))
    f = O.silu_mlp_fwd(X, W1, W2)
    b = O.silu_mlp_bwd(dY, X, f["G"], f["Hh"], W1, W2)
    tx, t1, t2 = (torch.tensor(a, requires_grad=True) for a in (X, W1, W2))
    y = torch.nn.functional.silu(tx @ t1.T) @ t2.T
    y.backward(torch.from_numpy(dY))
    assert np.allclose(f["Y"], y.detach().numpy(), rtol=1e-12, atol=1e-12)
    for mine, ref in ((b["dX"], tx.grad), (b["dW_gate_up"], t1.grad), (b["dW_down"], t2.grad)):
        assert np.allclose(mine, ref.numpy(), rtol=1e-11, atol=1e-11)


def test_silu_expert_single_resident_layer_is_dense_mlp():
    inp = tiny_inputs(T=12, d=6, E=4, k=1, H=5, resident=(0, 1, 2, 3), seed=42, expert="silu")
    f = O.layer_fwd(inp)
    x = inp["x"]
    for t in range(12):
        e = int(f["idx"][t, 0])
        a = x[t] @ inp["w_gate_up"][e].T
        ref = (a / (1 + np.exp(-a))) @ inp["w_down"][e].T
        assert np.allclose(f["y"][t], f["w"][t, 0] * ref, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- placement (Alg. 1)

@pytest.mark.parametrize("N_e,O_e,M", [(64, 4, 8), (16, 1, 4), (16, 4, 4), (12, 2, 8), (8, 3, 6)])
def test_placement_meets_the_constraints(N_e, O_e, M):
    """Every expert on exactly O_e workers, every worker N_le distinct experts,
    for the fixed map and for random relabelings."""
    g = np.random.default_rng(N_e * 100 + O_e * 10 + M)
    for draw in range(4):
        ep = None if draw == 0 else g.permutation(N_e)
        wp = None if draw == 0 else g.permutation(M)
        P = O.gen_placement(N_e, O_e, M, ep, wp)
        N_le = N_e * O_e // M
        assert P.shape == (M, N_le)
        for m in range(M):
            assert len(set(P[m])) == N_le and list(P[m]) == sorted(P[m])
        hosts = np.zeros(N_e, int)
        for m in range(M):
            hosts[P[m]] += 1
        assert np.all(hosts == O_e)


def test_placement_limits():
    # O_e = M: full replication; O_e = 1: a disjoint partition
    assert np.array_equal(O.gen_placement(8, 4, 4), np.tile(np.arange(8), (4, 1)))
    P = O.gen_placement(16, 1, 4)
    assert sorted(P.reshape(-1).tolist()) == list(range(16))
    with pytest.raises(ValueError):
        O.gen_placement(10, 3, 4)  # 4 does not divide 30


def test_migration_map_and_warmup():
    prev, new = np.array([1, 4, 6, 9]), np.array([0, 4, 9, 11])
    assert list(O.migration_map(prev, new)) == [-1, 1, 3, -1]
    assert list(O.migration_map(new, new)) == [0, 1, 2, 3]  # fixed placement keeps all state
    assert O.warmup_scale(0, 10) == 0.0 and O.warmup_scale(5, 10) == 0.5
    assert O.warmup_scale(25, 10) == 1.0 and O.warmup_scale(3, 0) == 1.0
