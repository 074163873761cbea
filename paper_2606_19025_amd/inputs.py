"""Seeded synthetic inputs for the resident-expert MoE layer.

This module only describes workload shapes and draws seeded random tensors
(plus rounding of those draws to bfloat16).  It contains none of the layer's
arithmetic, so both the CPU oracle and the HIP path can be fed from it without
sharing any computation.

Workloads (shapes of the paper's fine-grained MoE layers, Sec. 3.2 and App. B;
the method's skip-token setting is Sec. 3.3 "Ghost Experts and Skip-Token"):

  0  tiny fp32:      T=256,  d=64,   E=8,  resident {0..3},        k=2, H=128
  1  mid bf16:       T=4096, d=1024, E=16, resident even ids,      k=2, H=2816
  2  fine-grained:   T=8192, d=2048, E=64, resident {16..31},      k=6, H=1408,
                     plus 2 always-active shared experts of hidden 1408 each
  3  skewed routing: shapes of 1, router logits biased by a Zipf(1.2) ranking
                     that puts the 8 non-resident experts first
  4  large:          T=16384, d=4096, E=64, 32 resident (seeded subset), k=8,
                     H=2048, plus the round-boundary expert delta over 4 site
                     copies of every resident expert

Distributions: activations and upstream gradients ~ N(0, 1); router and expert
weights ~ N(0, 0.02) (standard deviation); peer deltas ~ N(0, 1e-3).
Every tensor comes from its own substream ``default_rng([seed, workload,
stream])`` so that a tensor does not change when another one is resized.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "WORKLOADS",
    "ZIPF_S",
    "ZIPF_BETA_W3",
    "bf16_round",
    "workload",
    "make_layer_inputs",
    "make_delta_inputs",
    "rng_for",
]

# Zipf exponent of the skewed-routing workload and the logit scale beta that
# makes ~70% of top-1 routes land on non-resident experts for seed 42.  beta
# was found by bisection with tests/golden/calibrate_zipf_beta.py, which calls
# only the oracle; tests/test_oracle_pins.py re-checks the realised fraction.
ZIPF_S = 1.2
ZIPF_BETA_W3 = 0.18798828125

_STREAMS = {
    "x": 0, "dy": 1, "w_router": 2, "w_gate_up": 3, "w_down": 4,
    "shared_gate_up": 5, "shared_down": 6, "resident": 7,
    "theta_start": 8, "theta_now": 9, "peers": 10, "ghost_weights": 11,
}

WORKLOADS = {
    0: dict(name="tiny-fp32", T=256, d=64, E=8, resident=[0, 1, 2, 3], k=2,
            H=128, dtype="f32", n_shared=0, Hs=0, zipf=False, n_peers=0),
    1: dict(name="mid-bf16", T=4096, d=1024, E=16,
            resident=list(range(0, 16, 2)), k=2, H=2816, dtype="bf16",
            n_shared=0, Hs=0, zipf=False, n_peers=0),
    2: dict(name="fine-grained-shared-bf16", T=8192, d=2048, E=64,
            resident=list(range(16, 32)), k=6, H=1408, dtype="bf16",
            n_shared=2, Hs=1408, zipf=False, n_peers=3),
    3: dict(name="skewed-zipf-bf16", T=4096, d=1024, E=16,
            resident=list(range(0, 16, 2)), k=2, H=2816, dtype="bf16",
            n_shared=0, Hs=0, zipf=True, n_peers=0),
    4: dict(name="large-round-sync-bf16", T=16384, d=4096, E=64,
            resident=None, k=8, H=2048, dtype="bf16", n_shared=0, Hs=0,
            zipf=False, n_peers=3),
}


def rng_for(seed: int, wl: int, stream: str) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(wl), _STREAMS[stream]])


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    # finite inputs only: the 32-bit sum cannot wrap below the NaN range
    r = (u >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r &= np.uint32(0xFFFF0000)
    return r.view(np.float32)


def workload(wl: int, seed: int = 42, resident=None) -> dict:
    """Shape description of workload ``wl`` with its resident set resolved
    (``resident`` replaces the workload's own set, e.g. for a sweep over the
    number of ghost experts)."""
    cfg = dict(WORKLOADS[wl])
    cfg["id"] = wl
    if resident is not None:
        cfg["resident"] = sorted(int(e) for e in resident)
    if cfg["resident"] is None:
        r = rng_for(seed, wl, "resident")
        cfg["resident"] = sorted(int(e) for e in r.choice(cfg["E"], cfg["E"] // 2, replace=False))
    cfg["E_r"] = len(cfg["resident"])
    return cfg


def _normal(g: np.random.Generator, shape, std: float) -> np.ndarray:
    out = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        out *= np.float32(std)
    return out


def zipf_logit_bias(cfg: dict, beta: float) -> np.ndarray:
    """Per-expert router logit bias beta*log(p_e), p_e proportional to rank_e**-s.

    Non-resident experts take ranks 1..E-E_r in ascending id order, resident
    experts the remaining ranks, so the bias favours the ghost experts.
    """
    E = cfg["E"]
    res = set(cfg["resident"])
    order = [e for e in range(E) if e not in res] + [e for e in range(E) if e in res]
    rank = np.empty(E, dtype=np.float64)
    for r, e in enumerate(order):
        rank[e] = r + 1
    p = rank ** (-ZIPF_S)
    p /= p.sum()
    return (beta * np.log(p)).astype(np.float32)


def make_layer_inputs(wl: int, seed: int = 42, T: int | None = None,
                      zipf_beta: float | None = None, ghost_weights: bool = False,
                      with_experts: bool = True, resident=None) -> dict:
    """All inputs of one layer step as float32 numpy arrays (bf16-valued for bf16 workloads).

    Expert weights are held only for the resident experts, in the layouts the
    library uses: w_gate_up [E_r, 2H, d] (gate rows then up rows),
    w_down [E_r, d, H].  The shared experts are merged along the hidden
    dimension into one expert of hidden n_shared*Hs.  ``T`` truncates the
    token dimension (the first T tokens of the full draw); ``with_experts``
    False skips drawing the expert weights (routing-only uses); ``resident``
    replaces the workload's resident set.
    """
    cfg = workload(wl, seed, resident)
    Tf, d, E, H, Er = cfg["T"], cfg["d"], cfg["E"], cfg["H"], cfg["E_r"]
    T = Tf if T is None else int(T)
    rnd = bf16_round if cfg["dtype"] == "bf16" else (lambda a: np.ascontiguousarray(a, np.float32))
    x = rnd(_normal(rng_for(seed, wl, "x"), (Tf, d), 1.0)[:T])
    dy = rnd(_normal(rng_for(seed, wl, "dy"), (Tf, d), 1.0)[:T])
    w_router = rnd(_normal(rng_for(seed, wl, "w_router"), (E, d), 0.02))
    if with_experts:
        w_gate_up = rnd(_normal(rng_for(seed, wl, "w_gate_up"), (Er, 2 * H, d), 0.02))
        w_down = rnd(_normal(rng_for(seed, wl, "w_down"), (Er, d, H), 0.02))
    else:
        w_gate_up = w_down = None
    resident = np.zeros(E, dtype=np.uint8)
    resident[cfg["resident"]] = 1
    out = dict(cfg=cfg, x=x, dy=dy, w_router=w_router, w_gate_up=w_gate_up,
               w_down=w_down, resident=resident, router_bias=None)
    if cfg["n_shared"] and with_experts:
        Hs = cfg["n_shared"] * cfg["Hs"]
        out["shared_gate_up"] = rnd(_normal(rng_for(seed, wl, "shared_gate_up"), (1, 2 * Hs, d), 0.02))
        out["shared_down"] = rnd(_normal(rng_for(seed, wl, "shared_down"), (1, d, Hs), 0.02))
    if cfg["zipf"]:
        beta = ZIPF_BETA_W3 if zipf_beta is None else zipf_beta
        out["router_bias"] = zipf_logit_bias(cfg, beta)
    if ghost_weights and with_experts:
        # weights of the experts this worker does NOT hold (used only to build
        # the full-replica comparison layer in tests)
        ghosts = [e for e in range(E) if e not in set(cfg["resident"])]
        g = rng_for(seed, wl, "ghost_weights")
        out["ghost_ids"] = ghosts
        out["ghost_gate_up"] = rnd(_normal(g, (len(ghosts), 2 * H, d), 0.02))
        out["ghost_down"] = rnd(_normal(g, (len(ghosts), d, H), 0.02))
    return out


def make_delta_inputs(wl: int, n_params: int, seed: int = 42) -> dict:
    """fp32 master copies for the round-boundary delta.

    theta_start ~ N(0, 0.02); theta_now = theta_start + N(0, 1e-3) (the local
    steps' drift); n_peers site copies of the delta ~ N(0, 1e-3).
    """
    cfg = workload(wl, seed)
    n_peers = max(1, cfg["n_peers"])
    theta_start = _normal(rng_for(seed, wl, "theta_start"), (n_params,), 0.02)
    theta_now = theta_start + _normal(rng_for(seed, wl, "theta_now"), (n_params,), 1e-3)
    peers = _normal(rng_for(seed, wl, "peers"), (n_peers, n_params), 1e-3)
    return dict(theta_start=theta_start, theta_now=theta_now.astype(np.float32), peers=peers)
