"""GPU parity at the full sizes of the two large workloads, through the same
ResidentMoELayer calls and launch shapes that bench.py times.

The oracle cannot run these layers whole in a test, so it is compared on what
it can compute piece by piece, and the rest is checked through properties that
hold at any size:

* routing, mask, counts, offsets and the permutation of ALL tokens, bit-exact,
  from the oracle's selection on the GPU's logits;
* logits, y, dx, dz and the gate gradients of 512 sampled tokens (each token's
  outputs depend only on its own row and the weights);
* dW_gate_up / dW_down of two sampled resident experts (they depend only on the
  routes to that expert), and the shared expert's dW over all tokens;
* dW_router = inv_tau * dz^T x and d_bias = inv_tau * sum_t dz over all tokens,
  recomputed in fp64 from the layer's own dz (which the samples pin);
* exact skip-token outputs of every fully skipped token;
* the round-boundary delta of the fine-grained workload at its full parameter
  count, bit-exact.
* run-to-run determinism of the mid-size and fine-grained layers (K parts,
  dynamically dealt tiles), bit-exact.
"""
import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_19025_amd import inputs as I
from paper_2606_19025_amd.layer import expert_delta

from .parity_helpers import (TOL, assert_close, gpu_outputs, host, make_layer, record_errors,
                             run_gpu_layer, say)

pytestmark = pytest.mark.gpu

N_SAMPLE = 512


def sub_problem(inp, tok, resident=None, expert=None):
    """The layer restricted to tokens `tok` (and optionally to one resident expert)."""
    cfg = dict(inp["cfg"])
    out = dict(inp)
    out["x"], out["dy"] = inp["x"][tok], inp["dy"][tok]
    cfg["T"] = len(tok)
    if resident is not None:
        out["resident"] = resident
        cfg["E_r"] = int(resident.sum())
        out["w_gate_up"] = inp["w_gate_up"][expert:expert + 1]
        out["w_down"] = inp["w_down"][expert:expert + 1]
        out["shared_gate_up"] = out["shared_down"] = None
    out["cfg"] = cfg
    return out


@pytest.mark.parametrize("wl", [2, 4])
def test_full_size_layer(gpu_lib, wl):
    say(f"[full] workload {wl}: inputs")
    inp = I.make_layer_inputs(wl)
    cfg = inp["cfg"]
    T, d, E, k, E_r = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["E_r"]
    tol = TOL[cfg["dtype"]]
    L = make_layer(inp)
    say(f"[full] workload {wl}: layer T={T} d={d} E={E} k={k} H={cfg['H']} E_r={E_r}")
    L, d_in = run_gpu_layer(inp, layer=L)

    # routing and dispatch of every token, bit-exact on the GPU's logits
    z = host(L.logits)
    idx = O.topk_select(z, k)
    local = O.mask_routes(idx, inp["resident"])
    plan = O.dispatch_plan(local, E_r)
    n = int(plan["offsets"][-1])
    assert np.array_equal(host(L.topk_idx), idx)
    assert np.array_equal(host(L.topk_local), local)
    assert np.array_equal(host(L.counts)[:E_r], plan["counts"])
    assert np.array_equal(host(L.offsets), plan["offsets"])
    assert np.array_equal(host(L.inv_perm), plan["inv_perm"])
    perm = host(L.perm)[:n]
    assert np.array_equal(perm, plan["perm"])
    rng = np.random.default_rng(7)
    rows = rng.choice(n, min(n, 2048), replace=False)
    xp = L.xp[torch.from_numpy(rows).cuda()].float().cpu().numpy()
    assert np.array_equal(xp, inp["x"][perm[rows] // k]), "gathered rows are not exact copies"
    say(f"[full] workload {wl}: routing, mask and permutation of {T} tokens exact (n={n})")

    # sampled tokens through the oracle
    tok = np.sort(rng.choice(T, N_SAMPLE, replace=False))
    tk = torch.from_numpy(tok).cuda()
    sub = sub_problem(inp, tok)
    z_own = O.router_logits(sub["x"], inp["w_router"], 1.0, inp.get("router_bias"))
    assert_close("logits", z[tok], z_own, 1e-5)
    fwd = O.layer_fwd(sub, logits=z[tok])
    bwd = O.layer_bwd(sub, fwd, sub["dy"])
    errs = {}
    errs["w"] = assert_close("topk_w", host(L.topk_w)[tok], fwd["w"], 1e-5)
    errs["y"] = assert_close("y", L.y[tk].float().cpu().numpy(), fwd["y"], tol)
    errs["dx"] = assert_close("dx", L.dx[tk].float().cpu().numpy(), bwd["dx"], tol)
    dz = host(L.dz)
    errs["dz"] = assert_close("dz", dz[tok], bwd["dz"], tol)
    errs["dtopk_w"] = assert_close("d_topk_w", host(L.dtopk_w)[tok], bwd["dw"], tol)
    record_errors(f"full_size_layer[{wl}] {N_SAMPLE} sampled tokens", errs)

    # weight gradients of two sampled resident experts
    res_ids = np.flatnonzero(inp["resident"])
    for r in sorted(rng.choice(E_r, 2, replace=False)):
        g = res_ids[r]
        t_e = np.flatnonzero((idx == g).any(axis=1))
        only = np.zeros(E, np.uint8)
        only[g] = 1
        se = sub_problem(inp, t_e, resident=only, expert=r)
        fe = O.layer_fwd(se, logits=z[t_e])
        be = O.layer_bwd(se, fe, se["dy"])
        e1 = assert_close(f"dW_gate_up[{r}]", L.dw_gate_up[r].cpu().numpy(), be["dW_gate_up"][0], tol)
        e2 = assert_close(f"dW_down[{r}]", L.dw_down[r].cpu().numpy(), be["dW_down"][0], tol)
        record_errors(f"full_size_layer[{wl}] expert {g} ({len(t_e)} tokens)",
                      {"dW_gate_up": e1, "dW_down": e2})

    # shared expert: all tokens, weight 1
    if L.Hs:
        x64, dy64 = inp["x"].astype(np.float64), inp["dy"].astype(np.float64)
        sf = O.swiglu_fwd(x64, inp["shared_gate_up"][0], inp["shared_down"][0])
        sb = O.swiglu_bwd(dy64, x64, sf["G"], sf["U"], sf["Hh"], inp["shared_gate_up"][0],
                          inp["shared_down"][0])
        e1 = assert_close("shared dW_gate_up", L.s_dw_gate_up[0].cpu().numpy(), sb["dW_gate_up"], tol)
        e2 = assert_close("shared dW_down", L.s_dw_down[0].cpu().numpy(), sb["dW_down"], tol)
        record_errors(f"full_size_layer[{wl}] shared expert", {"dW_gate_up": e1, "dW_down": e2})

    # router weight gradient over all tokens from the layer's own dz
    dzx = dz.T @ inp["x"].astype(np.float64)
    assert_close("dW_router vs dz^T x", host(L.dw_router), dzx, 1e-4)
    assert_close("d_bias vs sum dz", host(L.d_bias), dz.sum(axis=0), 1e-4)

    # skip-token: routed contribution exactly zero for fully skipped tokens
    skipped = np.flatnonzero(np.all(local < 0, axis=1))
    if len(skipped):
        sk = torch.from_numpy(skipped).cuda()
        y_sk = L.y[sk]
        if L.Hs:
            assert torch.equal(y_sk, L.s_y[sk]), "skipped tokens must get exactly the shared output"
        else:
            assert torch.count_nonzero(y_sk).item() == 0
        assert np.all(dz[skipped] == 0.0)
    assert np.all(host(L.dtopk_w)[local < 0] == 0.0)
    say(f"[full] workload {wl}: {len(skipped)} fully skipped tokens exact")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("wl", [2, 4])
def test_full_size_expert_delta(gpu_lib, wl):
    """Round-boundary delta over every resident-expert fp32 master parameter
    of the workload (16 x 3Hd = 138,412,032 for the fine-grained layer,
    32 x 3Hd = 805,306,368 for the large one), averaged with the site copies
    (S = 4 copies: this one and 3 peers, Alg. 2 round end), bit-exact."""
    cfg = I.workload(wl, 42)
    n = cfg["E_r"] * 3 * cfg["H"] * cfg["d"]
    say(f"[full] expert delta over {n} parameters, {cfg['n_peers']} peers: inputs")
    dpar = I.make_delta_inputs(wl, n)
    say("[full] expert delta: oracle")
    dl_ref, avg_ref = O.expert_delta(dpar["theta_start"], dpar["theta_now"], list(dpar["peers"]))
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    ts, tn = dev(dpar["theta_start"]), dev(dpar["theta_now"])
    peers = [dev(p) for p in dpar["peers"]]
    del dpar
    dl = torch.full_like(ts, float("nan"))
    say("[full] expert delta: kernel")
    avg = expert_delta(ts, tn, peers, delta_local=dl)
    torch.cuda.synchronize()
    del ts, tn, peers
    assert torch.equal(dl.cpu().view(torch.int32), torch.from_numpy(dl_ref).view(torch.int32))
    assert torch.equal(avg.cpu().view(torch.int32), torch.from_numpy(avg_ref).view(torch.int32))
    say(f"[full] expert delta over {n} parameters bit-exact")


@pytest.mark.parametrize("wl", [1, 2])
def test_full_size_layer_is_deterministic(gpu_lib, wl):
    """Three steps of the mid-size layer (its down projection and dX cut into K
    parts) and of the fine-grained one (shared expert, merged backward
    launches) give bit-identical outputs and gradients, whichever blocks the
    dynamically dealt tiles ran on."""
    say(f"[determinism] workload {wl}: inputs")
    inp = I.make_layer_inputs(wl)
    L, _ = run_gpu_layer(inp)
    first = gpu_outputs(L)
    for rep in (1, 2):
        say(f"[determinism] workload {wl}: repeat {rep}")
        run_gpu_layer(inp, layer=L)
        again = gpu_outputs(L)
        for key, v in first.items():
            assert np.array_equal(v, again[key]), f"{key} differs on repeat {rep}"
