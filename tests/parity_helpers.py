"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
binding, run the CPU oracle on the same seeded inputs, compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import moe_oracle as O
from paper_2606_19025_amd import inputs as I
from paper_2606_19025_amd.layer import ResidentMoELayer

TOL = {"f32": 1e-5, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def canary(*shape, dtype=torch.bfloat16):
    """A device output buffer filled with NaN: an element the kernels fail to
    write then fails every comparison (torch.empty would hold stale values)."""
    return torch.full(shape, float("nan"), dtype=dtype, device="cuda")


def record_errors(test, errs):
    """Print a test's per-tensor errors and, when MOE_PARITY_LOG names a file,
    append them to it as one JSON line (the record of a GPU parity run)."""
    import json
    import os

    vals = {k: float(v) for k, v in errs.items()}
    worst = max((v for k, v in vals.items() if k != "excluded_near_ties"), default=0.0)
    say(f"[errors] {test}: max {worst:.2e} " +
        " ".join(f"{k}={v:.1e}" for k, v in vals.items()))
    path = os.environ.get("MOE_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"test": test, "max": worst, "errors": vals}) + "\n")


def dev(a, dtype):
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(dtype)


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64) if t.is_floating_point() \
        else t.detach().cpu().numpy()


def rel_err(a, b):
    """normwise relative error max|a - b| / max|b|"""
    a = np.asarray(a, np.float64); b = np.asarray(b, np.float64)
    if a.size == 0:
        return 0.0
    den = np.max(np.abs(b))
    num = np.max(np.abs(a - b))
    return float(num / den) if den > 0 else float(num)


def assert_close(name, a, b, tol):
    e = rel_err(a, b)
    assert e <= tol, f"{name}: normwise relative error {e:.3e} > {tol:.1e}"
    return e


def torch_dtype(cfg):
    return torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32


def make_layer(inp, gate="softmax_topk", inv_tau=1.0):
    cfg = inp["cfg"]
    hs = cfg.get("n_shared", 0) * cfg.get("Hs", 0) if inp.get("shared_gate_up") is not None else 0
    return ResidentMoELayer(inp["x"].shape[0], cfg["d"], cfg["E"], cfg["k"], cfg["H"],
                            inp["resident"], dtype=torch_dtype(cfg), n_shared_hidden=hs,
                            gate=gate, inv_tau=inv_tau, expert=cfg.get("expert", "swiglu"),
                            canary=True)


def run_gpu_layer(inp, gate="softmax_topk", inv_tau=1.0, layer=None):
    """Forward + backward of the HIP path; returns the layer and the device inputs."""
    cfg = inp["cfg"]
    dt = torch_dtype(cfg)
    L = layer or make_layer(inp, gate, inv_tau)
    d_in = dict(x=dev(inp["x"], dt), dy=dev(inp["dy"], dt), w_router=dev(inp["w_router"], dt),
                w_gate_up=dev(inp["w_gate_up"], dt), w_down=dev(inp["w_down"], dt),
                router_bias=dev(inp.get("router_bias"), torch.float32),
                shared_gate_up=dev(inp.get("shared_gate_up"), dt),
                shared_down=dev(inp.get("shared_down"), dt))
    L.forward(d_in["x"], d_in["w_router"], d_in["w_gate_up"], d_in["w_down"], d_in["router_bias"],
              d_in["shared_gate_up"], d_in["shared_down"])
    L.backward(d_in["dy"], d_in["x"], d_in["w_router"], d_in["w_gate_up"], d_in["w_down"],
               d_in["shared_gate_up"], d_in["shared_down"])
    torch.cuda.synchronize()
    return L, d_in


def gpu_outputs(L):
    n = int(L.offsets[-1].item())
    out = dict(logits=host(L.logits), idx=host(L.topk_idx), w=host(L.topk_w),
               local=host(L.topk_local), counts=host(L.counts)[:L.E_r], offsets=host(L.offsets),
               perm=host(L.perm)[:n], inv_perm=host(L.inv_perm), n=n,
               xp=host(L.xp[:n]), gu=host(L.gu[:n]), h=host(L.h[:n]), yp=host(L.yp[:n]),
               y=host(L.y), dyp=host(L.dyp[:n]), dw=host(L.dtopk_w), dgu=host(L.dgu[:n]),
               dxp=host(L.dxp[:n]), dW_gate_up=host(L.dw_gate_up)[:L.E_r],
               dW_down=host(L.dw_down)[:L.E_r], dx=host(L.dx), dz=host(L.dz),
               dW_router=host(L.dw_router), d_bias=host(L.d_bias))
    if L.Hs:
        out.update(s_y=host(L.s_y), s_dW_gate_up=host(L.s_dw_gate_up)[0],
                   s_dW_down=host(L.s_dw_down)[0])
    return out


def check_layer_against_oracle(inp, g, gate="softmax_topk", inv_tau=1.0, check_own_routing=True):
    """Full-layer parity: the oracle runs on the GPU's logits (identical routing
    decisions); the logits themselves are checked against the oracle's own."""
    cfg = inp["cfg"]
    tol = TOL[cfg["dtype"]]
    errs = {}
    z_own = O.router_logits(inp["x"], inp["w_router"], inv_tau, inp.get("router_bias"))
    errs["logits"] = assert_close("logits", g["logits"], z_own, 1e-5)
    fwd = O.layer_fwd(inp, inv_tau=inv_tau, gate=gate, logits=g["logits"])
    # bit-exact routing decisions, mask and permutation on the same logits
    assert np.array_equal(g["idx"], fwd["idx"]), "topk_idx differs"
    assert np.array_equal(g["local"], fwd["local"]), "topk_local differs"
    assert np.array_equal(g["counts"], fwd["counts"]), "counts differ"
    assert np.array_equal(g["offsets"], fwd["offsets"]), "offsets differ"
    assert np.array_equal(g["perm"], fwd["perm"]), "perm differs"
    assert np.array_equal(g["inv_perm"], fwd["inv_perm"]), "inv_perm differs"
    assert np.array_equal(g["xp"], fwd["Xp"]), "gathered rows are not exact copies"
    errs["w"] = assert_close("topk_w", g["w"], fwd["w"], 1e-5)
    errs["y"] = assert_close("y", g["y"], fwd["y"], tol)
    if g["n"]:
        errs["yp"] = assert_close("yp", g["yp"], fwd["Yp"], tol)
    bwd = O.layer_bwd(inp, fwd, inp["dy"], inv_tau=inv_tau, gate=gate)
    errs["dw"] = assert_close("d_topk_w", g["dw"], bwd["dw"], tol)
    errs["dx"] = assert_close("dx", g["dx"], bwd["dx"], tol)
    errs["dz"] = assert_close("dz", g["dz"], bwd["dz"], tol)
    errs["dW_router"] = assert_close("dW_router", g["dW_router"], bwd["dW_router"], tol)
    errs["d_bias"] = assert_close("d_bias", g["d_bias"], bwd["d_bias"], tol)
    # expert weight gradients one expert at a time (each against its own
    # scale); an expert without routes gets exactly zero
    errs["dW_gate_up"] = errs["dW_down"] = 0.0
    for r in range(len(g["counts"])):
        for key in ("dW_gate_up", "dW_down"):
            if g["counts"][r] == 0:
                assert np.all(g[key][r] == 0.0), f"{key}[{r}] of an expert without routes"
            else:
                errs[key] = max(errs[key], assert_close(f"{key}[{r}]", g[key][r], bwd[key][r], tol))
    if bwd["shared"] is not None:
        errs["s_dW_gate_up"] = assert_close("shared dW_gate_up", g["s_dW_gate_up"],
                                            bwd["shared"]["dW_gate_up"], tol)
        errs["s_dW_down"] = assert_close("shared dW_down", g["s_dW_down"],
                                         bwd["shared"]["dW_down"], tol)
    # skip-token: tokens whose routes all hit ghost experts
    skipped = np.all(g["local"] < 0, axis=1)
    if skipped.any():
        if bwd["shared"] is None:
            assert np.all(g["y"][skipped] == 0.0), "fully skipped tokens must give exactly 0"
            assert np.all(g["dx"][skipped] == 0.0), "fully skipped tokens must get dx exactly 0"
        else:
            assert np.array_equal(g["y"][skipped], g["s_y"][skipped])
        assert np.all(g["dz"][skipped] == 0.0)
    assert np.all(g["dw"][g["local"] < 0] == 0.0), "ghost routes must get zero gate gradient"
    if check_own_routing:
        # the oracle's own selection agrees except where the k-th/(k+1)-th margin is tiny
        k = cfg["k"]
        own_idx = O.topk_select(z_own, k)
        zs = -np.sort(-z_own, axis=1)
        margin = zs[:, k - 1] - zs[:, k] if k < z_own.shape[1] else np.full(z_own.shape[0], np.inf)
        safe = margin > (1e-3 if cfg["dtype"] == "bf16" else 1e-5)
        assert np.array_equal(np.sort(own_idx[safe], 1), np.sort(g["idx"][safe], 1))
        errs["excluded_near_ties"] = int((~safe).sum())
    return errs
