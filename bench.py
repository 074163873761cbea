"""Benchmark of one worker's local training step through the resident-expert
MoE layer on one MI355X.

A step is one forward + backward of the whole layer (router, ghost-expert
mask, dispatch, grouped SwiGLU experts, shared experts, combine, and all of
their backward), and - at the round cadence (every ``--round-every`` steps,
32 = the smallest number of local steps between synchronisations in the
paper's sweep grid, App. F) - the round-boundary expert delta averaged over
the expert's replica group.  Inputs are seeded synthetic tensors already
resident in HBM; the timed region holds exactly ``--steps`` steps bracketed by
torch.cuda.synchronize().

Prints ONE JSON line.  Besides the contract fields it carries:
  step_spread   median, p10 and p90 of single steps, timed again one by one;
  roofline      the dominant kernel's achieved rate vs the MI355X peak, from
                algorithmic flops (or bytes) per launch and its average launch
                duration measured with HIP events in a second pass of the same
                steps (the library's moe_timing facility);
  kernels       the same for every kernel of the step (warm: inputs may sit in
                L2 or the Infinity Cache from the kernel that wrote them);
  kernels_cold  the HBM-bound kernels again with a 512 MiB read before every
                library call (``--cold-steps`` steps), so that each call's first
                kernel reads its inputs from HBM;
  cpu_baseline  the CPU oracle on a bounded token sample of the same workload;
  hbm_copy      a plain device copy of 1 GiB and, for each cold-timed kernel,
                a cold copy moving that kernel's bytes (frac_of_copy_at_size);
  blas_reference torch.matmul (hipBLASLt) on each GEMM launch's dense
                equivalent (reference for the MFMA fractions, not in the step).

    python bench.py [--gpus 1] [--steps 64] [--warmup 10] [--workload 2]

``--ghost-sweep`` instead measures the layer analogue of the paper's skip-token
throughput experiment (Sec. 6.4, "Measured Skip-Token Throughput"): the mid-size
layer (workload 1 shapes: T=4096, d=1024, E=16, top-2, H=2816, bf16) with 16,
12, 8 and 4 resident experts, each with the unpartitioned router and
skip-token and with the partitioned router, as one JSON line.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
FLUSH_BYTES = 512 << 20     # twice the 256 MB Infinity Cache
SWEEP_TRIALS = 3            # timed runs per configuration of --ghost-sweep


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=2)
    ap.add_argument("--round-every", type=int, default=32)
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--cpu-sample-tokens", type=int, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--cold-steps", type=int, default=8,
                    help="steps of the cold per-kernel pass (a 512 MiB read before every "
                         "library call evicts L2 and the Infinity Cache); 0 skips it")
    ap.add_argument("--optimizer", action="store_true",
                    help="time whole training steps: fwd + bwd + AdamW on the resident and shared "
                         "experts every step, and at the round cadence the delta average and the "
                         "outer Nesterov step")
    ap.add_argument("--placement", choices=["fixed", "random"], default="fixed",
                    help="with --optimizer: random placement (Alg. 1) redraws the worker's "
                         "resident set every --reshuffle-every rounds and migrates weights and "
                         "optimiser state")
    ap.add_argument("--reshuffle-every", type=int, default=1)
    ap.add_argument("--expert", choices=["swiglu", "silu"], default="swiglu",
                    help="expert form: SwiGLU (the workloads') or the paper's SiLU expert "
                         "(its first weight is the first H rows of the SwiGLU draw)")
    ap.add_argument("--ghost-sweep", action="store_true",
                    help="tokens/s vs number of ghost experts, skip-token and partitioned router")
    ap.add_argument("--traffic-calibration", action="store_true",
                    help="make one plain device-to-device copy of a known size before the "
                         "steps, the scale for rocprofv3 FETCH_SIZE / WRITE_SIZE counts")
    ap.add_argument("--no-blas-reference", dest="blas_reference", action="store_false",
                    help="skip timing torch.matmul (hipBLASLt) on the GEMMs' dense equivalents")
    ap.add_argument("--no-copy-baseline", dest="copy_baseline", action="store_false",
                    help="skip timing torch's device-to-device copy and read-only sum of 1 GiB "
                         "(the HBM rates a plain streaming kernel reaches on the box; on by "
                         "default)")
    return ap.parse_args()


def algorithmic_work(cfg, n, t_act, s, expert="swiglu"):
    """Per-step algorithmic flops / bytes of every kernel (summed over its launches).

    n: executed (resident) routes; t_act: tokens with at least one resident
    route; s: bytes per activation element; expert: "swiglu" or "silu" (one
    first projection of width H instead of two).
    """
    T, d, E, k, H = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["H"]
    Hs = cfg["n_shared"] * cfg["Hs"]
    rows = [(n, H)] + ([(T, Hs)] if Hs else [])
    w = {}
    # grouped GEMMs: flops (MFMA-bound)
    w["gemm_gu_fwd"] = ("flop", sum(2.0 * m * d * 2 * h for m, h in rows))
    w["gemm_down_fwd"] = ("flop", sum(2.0 * m * h * d for m, h in rows))
    w["gemm_dhh_bwd"] = ("flop", sum(2.0 * m * d * h for m, h in rows))
    w["gemm_dx_bwd"] = ("flop", sum(2.0 * m * 2 * h * d for m, h in rows))
    w["gemm_dwd"] = ("flop", sum(2.0 * m * d * h for m, h in rows))
    w["gemm_dwgu"] = ("flop", sum(2.0 * m * 2 * h * d for m, h in rows))
    if expert == "silu":
        w["gemm_up_fwd"] = ("flop", sum(2.0 * m * d * h for m, h in rows))
        w["gemm_dh_bwd"] = w.pop("gemm_dhh_bwd")
        w["gemm_dx_bwd"] = ("flop", sum(2.0 * m * h * d for m, h in rows))
        w["gemm_dwgu"] = ("flop", sum(2.0 * m * h * d for m, h in rows))
        del w["gemm_gu_fwd"]
    # bf16 layers run the backward GEMMs as two launches of two kinds each
    # (dHh with dW_d, dX with dW_gu)
    first = "gemm_dh_bwd" if expert == "silu" else "gemm_dhh_bwd"
    w["gemm_dh_dwd" if expert == "silu" else "gemm_dhh_dwd"] = (
        "flop", w[first][1] + w["gemm_dwd"][1])
    w["gemm_dx_dwgu"] = ("flop", w["gemm_dx_bwd"][1] + w["gemm_dwgu"][1])
    w["zero_counters"] = ("byte", 64)
    # routing / data movement: bytes (HBM-bound)
    w["route_fwd"] = ("byte", T * d * s + E * d * s + T * E * 4 + 3 * T * k * 4)
    w["dispatch_count"] = ("byte", T * k * 4)
    w["dispatch_scan"] = ("byte", 0)
    w["dispatch_scatter"] = ("byte", T * k * 4 + n * 4 + T * k * 4)
    w["dispatch_gather"] = ("byte", t_act * d * s + n * d * s + T * k * 4)
    # fused scan + slots + gather: every x row read, n rows written, the
    # local ids read and perm / inv_perm written
    w["dispatch_place"] = ("byte", T * d * s + n * d * s + T * k * 4 + n * 4 + T * k * 4)
    w["combine_fwd"] = ("byte", n * d * s + (T * d * s if Hs else 0) + T * d * s + T * k * 8)
    w["combine_bwd"] = ("byte", t_act * d * s + 2 * n * d * s + T * k * 12)
    w["unpermute"] = ("byte", n * d * s + (T * d * s if Hs else 0) + T * d * s + T * k * 4)
    w["route_dz"] = ("byte", T * k * 12 + T * E * 4)
    w["route_dw_partial"] = ("byte", T * E * 4 + T * d * s)
    w["route_dw_reduce"] = ("byte", (-(-T // 256) + 1) * E * d * 4)
    w["route_dx"] = ("byte", T * E * 4 + 2 * T * d * s + E * d * s)
    # fused bf16 router backward: x, dz and W_r in, dx read-modify-write,
    # one fp32 dW_r partial per 256-token chunk out
    w["route_bwd_mfma"] = ("byte", T * E * 4 + 3 * T * d * s + E * d * s
                           + -(-T // 256) * E * d * 4)
    return w


def survey_bytes(cfg, n, s):
    """Bytes per step of the routing, dispatch and combine kernels under the
    scope table's formulas (each kernel's compulsory row traffic as the method
    defines it; they count neither the shared experts' output that the combine
    adds, nor the dx that the un-permute accumulates into, nor the tokens
    without resident routes, which the kernels here skip or add)."""
    T, d, E, k = cfg["T"], cfg["d"], cfg["E"], cfg["k"]
    return {"route_fwd": T * d * s + E * d * s + 4 * T * E + 9 * T * k,
            "dispatch_place": 2 * n * d * s,
            "dispatch_gather": 2 * n * d * s,
            "combine_fwd": n * d * s + T * d * s,
            "combine_bwd": T * d * s + 2 * n * d * s + 8 * T * k,
            "unpermute": n * d * s + T * d * s}


def blas_reference(cfg, n, expert="swiglu", reps=10):
    """torch.matmul (hipBLASLt) time of each GEMM launch's work as dense bf16
    GEMMs: every set as one GEMM over all its rows (routed: M = n executed
    routes, as if no expert boundaries; shared: M = T), K-ragged kinds as one
    GEMM with K = those rows.  A reference for the MFMA fractions, not part
    of the step."""
    import torch
    T, d, H = cfg["T"], cfg["d"], cfg["H"]
    Hs = cfg["n_shared"] * cfg["Hs"]
    r1 = 1 if expert == "silu" else 2
    sets = [(n, H)] + ([(T, Hs)] if Hs else [])
    kinds = {  # launch -> [(M, N, K)]
        "gemm_gu_fwd": [(m, r1 * h, d) for m, h in sets],
        "gemm_down_fwd": [(m, d, h) for m, h in sets],
        "gemm_dhh_dwd": [(m, h, d) for m, h in sets] + [(d, h, m) for m, h in sets],
        "gemm_dx_dwgu": [(m, d, r1 * h) for m, h in sets] + [(r1 * h, d, m) for m, h in sets],
    }
    # and one large square GEMM: what the library reaches at its best shape
    kinds["dense_8192_cubed"] = [(8192, 8192, 8192)]
    out = {}
    for name, shapes in kinds.items():
        tot_ms, flops = 0.0, 0.0
        for M, N, K in shapes:
            if min(M, N, K) <= 0:
                continue
            a = torch.randn(M, K, device="cuda", dtype=torch.bfloat16)
            b = torch.randn(K, N, device="cuda", dtype=torch.bfloat16)
            c = a @ b
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                c = a @ b
            e1.record()
            e1.synchronize()
            tot_ms += e0.elapsed_time(e1) / reps
            flops += 2.0 * M * N * K
            del a, b, c
        if tot_ms > 0:
            tf = flops / (tot_ms * 1e-3) / 1e12
            out[name] = {"us": round(tot_ms * 1e3, 1), "tflops": round(tf, 1),
                         "frac": round(tf / PEAK_BF16_TFLOPS, 4)}
    return out


def optimizer_work(n_step_params, n_round_params, n_peers):
    """Per-step bytes of the optimiser kernels: AdamW reads theta, g, m, v and
    writes theta, m, v and the bf16 copy (30 B per parameter); the outer step
    reads start, delta, momentum and writes momentum, start, now and the bf16
    copy (26 B); the replica mean reads 1 + peers copies and writes one."""
    return {"adamw_step": ("byte", 30.0 * n_step_params),
            "outer_nesterov": ("byte", 26.0 * n_round_params),
            "replica_mean": ("byte", 4.0 * (n_peers + 2) * n_round_params)}


def ghost_sweep(args):
    """Step time of the mid-size layer at 16, 12, 8 and 4 resident experts of
    16: skip-token (unpartitioned router, ghost routes skipped) and the
    partitioned router (routes over the resident experts only, top-min(k, E_r),
    nothing skipped).  Resident sets are spread evenly over the expert ids."""
    import numpy as np
    import torch

    from paper_2606_19025_amd import inputs as I
    from paper_2606_19025_amd.layer import ResidentMoELayer

    wl = 1
    base = I.workload(wl, args.seed)
    E = base["E"]
    rows = []
    for Er in (16, 12, 8, 4):
        resident = sorted({i * E // Er for i in range(Er)})
        inp = I.make_layer_inputs(wl, seed=args.seed, resident=resident)
        cfg = inp["cfg"]
        T, d, k, H = cfg["T"], cfg["d"], cfg["k"], cfg["H"]
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda().to(torch.bfloat16)
        x, dy, wgu, wd = (dev(inp[n]) for n in ("x", "dy", "w_gate_up", "w_down"))
        for mode in ("skip-token", "partitioned"):
            part = mode == "partitioned"
            wr = dev(inp["w_router"][np.flatnonzero(inp["resident"])] if part else inp["w_router"])
            L = ResidentMoELayer(T, d, E, k, H, inp["resident"], dtype=torch.bfloat16,
                                 partitioned=part)

            def step():
                L.forward(x, wr, wgu, wd)
                L.backward(dy, x, wr, wgu, wd)

            for _ in range(args.warmup):
                step()
            torch.cuda.synchronize()
            # median of SWEEP_TRIALS timed runs: single runs of these short
            # steps showed occasional 1.5x outliers on an otherwise idle GPU
            trials = []
            for _ in range(SWEEP_TRIALS):
                ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                ev0.record()
                for _ in range(args.steps):
                    step()
                ev1.record()
                torch.cuda.synchronize()
                trials.append(ev0.elapsed_time(ev1) / args.steps)
            ms = sorted(trials)[len(trials) // 2]
            n = int(L.offsets[-1].item())
            rows.append(dict(E_resident=Er, ghost_experts=E - Er, mode=mode, ms_per_step=round(ms, 4),
                             tokens_per_s=round(T / (ms / 1e3), 1), executed_routes=n,
                             trials_ms=[round(t, 4) for t in trials]))
            log(f"[sweep] E_r={Er:2d} {mode:11s} {ms:.3f} ms/step n={n}")
            del L
    full = {r["mode"]: r["tokens_per_s"] for r in rows if r["ghost_experts"] == 0}
    for r in rows:
        r["speedup_vs_no_ghosts"] = round(r["tokens_per_s"] / full[r["mode"]], 3)
    out = {"metric": "MoE layer fwd+bwd tokens/s vs ghost experts (1 GPU)", "unit": "tokens/s",
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "bf16",
           "data": "synthetic (seeded, shapes of the workload)",
           "config": {"workload": base["name"], "T": base["T"], "d": base["d"], "E": E,
                      "k": base["k"], "H": base["H"]},
           "sweep": rows}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); this build has no "
              "multi-GPU path", file=sys.stderr)
        sys.exit(2)
    if args.ghost_sweep:
        from paper_2606_19025_amd import binding as B
        B.lib()
        ghost_sweep(args)
        return
    import numpy as np
    import torch

    from paper_2606_19025_amd import binding as B
    from paper_2606_19025_amd import inputs as I
    from paper_2606_19025_amd.layer import ResidentMoELayer, expert_delta

    B.lib()
    wl = args.workload
    log(f"[bench] workload {wl}: generating inputs")
    inp = I.make_layer_inputs(wl, seed=args.seed)
    cfg = inp["cfg"]
    T, d, E, k, H, Er = cfg["T"], cfg["d"], cfg["E"], cfg["k"], cfg["H"], cfg["E_r"]
    Hs = cfg["n_shared"] * cfg["Hs"]
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    s_bytes = 2 if dt == torch.bfloat16 else 4
    dev = lambda a, t=dt: None if a is None else torch.from_numpy(
        np.ascontiguousarray(a, np.float32)).cuda().to(t)
    silu = args.expert == "silu"
    if silu:  # the SiLU expert's W1 [H, d]: the first H rows of the drawn [2H, d]
        inp["w_gate_up"] = np.ascontiguousarray(inp["w_gate_up"][:, :H])
        if inp.get("shared_gate_up") is not None:
            inp["shared_gate_up"] = np.ascontiguousarray(inp["shared_gate_up"][:, :Hs])
    x, dy, wr, wgu, wd = (dev(inp[n]) for n in ("x", "dy", "w_router", "w_gate_up", "w_down"))
    bias = dev(inp.get("router_bias"), torch.float32)
    sgu, sd = dev(inp.get("shared_gate_up")), dev(inp.get("shared_down"))
    L = ResidentMoELayer(T, d, E, k, H, inp["resident"], dtype=dt, n_shared_hidden=Hs,
                         expert=args.expert)
    r1 = 1 if silu else 2  # rows of the first expert weight per hidden unit
    # round boundary: fp32 master copies of the resident experts
    n_params = Er * (r1 * H * d + d * H)
    log(f"[bench] round-boundary state: {n_params / 1e6:.1f} M fp32 params x {2 + max(1, cfg['n_peers'])}")
    dpar = I.make_delta_inputs(wl, n_params, seed=args.seed)
    th0, th1 = dev(dpar["theta_start"], torch.float32), dev(dpar["theta_now"], torch.float32)
    peers = [dev(p, torch.float32) for p in dpar["peers"]]
    avg = torch.empty_like(th0)
    del dpar
    opt = None
    if args.optimizer:
        # the resident experts' fp32 masters (theta_now) in the weights'
        # layout: w_gate_up then w_down, each expert contiguous; the bf16
        # weights the GEMMs read are views of one buffer of the same layout
        n_gu = Er * r1 * H * d
        w_lp = torch.empty(n_params, dtype=dt, device="cuda")
        w_lp[:n_gu].copy_(wgu.reshape(-1))
        w_lp[n_gu:].copy_(wd.reshape(-1))
        wgu, wd = w_lp[:n_gu].view(Er, r1 * H, d), w_lp[n_gu:].view(Er, d, H)
        th1.copy_(w_lp.float())
        th0.copy_(th1)
        opt = dict(m=torch.zeros_like(th1), v=torch.zeros_like(th1), mom=torch.zeros_like(th1),
                   t=0, gu=th1[:n_gu], down=th1[n_gu:])
        if Hs:
            n_s = (r1 + 1) * Hs * d
            s_lp = torch.empty(n_s, dtype=dt, device="cuda")
            s_lp[:r1 * Hs * d].copy_(sgu.reshape(-1))
            s_lp[r1 * Hs * d:].copy_(sd.reshape(-1))
            sgu, sd = s_lp[:r1 * Hs * d].view(1, r1 * Hs, d), s_lp[r1 * Hs * d:].view(1, d, Hs)
            opt.update(s_master=s_lp.float(), s_m=torch.zeros(n_s, device="cuda"),
                       s_v=torch.zeros(n_s, device="cuda"), s_lp=s_lp)
        opt["lp"] = w_lp
        opt["rows"] = [(0, n_gu, r1 * H * d), (n_gu, n_params, d * H)]  # (begin, end, row_len)
        opt["steps"] = np.zeros(Er, np.int64)
        if args.placement == "random":
            # the server's store of every expert (weights and outer momentum),
            # a placement with replica groups of n_peers + 1 workers, and
            # spare state buffers for the migration copies
            O_e = len(peers) + 1
            M_w = E * O_e // Er
            gs = np.random.default_rng([args.seed, 99])
            store = [torch.from_numpy(gs.standard_normal((E, row), dtype=np.float32)
                                      * np.float32(0.02)).cuda() for _, _, row in opt["rows"]]
            opt.update(O_e=O_e, M=M_w, rng=gs, store_th=store,
                       store_mom=[torch.zeros_like(t) for t in store], m2=torch.empty_like(th1),
                       v2=torch.empty_like(th1), set=np.array(inp["cfg"]["resident"]),
                       copy_bytes=0.0)
            log(f"[bench] random placement: {E} experts on {M_w} workers, O_e = {O_e}, "
                f"reshuffle every {args.reshuffle_every} round(s)")
        log(f"[bench] optimiser state: AdamW m, v and outer momentum of {n_params / 1e6:.1f} M "
            f"expert params" + (f" (+{(r1 + 1) * Hs * d / 1e6:.1f} M shared)" if Hs else ""))

    def part_view(t, p):
        b, e, row = opt["rows"][p]
        return t[b:e].view(Er, row)

    def copy_rows(src, src_row, dst, dst_row=None, bf16=None):
        """Expert-row copy (Alg. 1 migration); counts its algorithmic bytes."""
        rl = src.shape[1] if src is not None else dst.shape[1]
        n_src = int(np.sum(np.asarray(src_row) >= 0))
        opt["copy_bytes"] += rl * (4 * n_src + 4 * len(src_row) + (2 * len(src_row) if bf16 is not None else 0))
        B.moe_copy_expert_rows(src, src_row, dst, len(src_row), rl, dst_row=dst_row, dst_bf16=bf16)

    def reshuffle():
        """Round boundary of random placement for this worker: resident rows
        back to the store, a new placement, migration of weights, outer
        momentum and AdamW state, restart of the new experts' step counts."""
        o = opt
        local = np.arange(Er)
        for p in range(2):
            copy_rows(part_view(th1, p), local, o["store_th"][p], o["set"])
            copy_rows(part_view(o["mom"], p), local, o["store_mom"][p], o["set"])
        ep, wp = o["rng"].permutation(E), o["rng"].permutation(o["M"])
        new = B.moe_gen_placement(E, o["O_e"], o["M"], ep, wp)[0]
        mig = B.moe_migration_map(o["set"], new)
        for p in range(2):
            b, e, _ = o["rows"][p]
            copy_rows(o["store_th"][p], new, part_view(th1, p), bf16=o["lp"][b:e])
            copy_rows(o["store_th"][p], new, part_view(th0, p))
            copy_rows(o["store_mom"][p], new, part_view(o["mom"], p))
            copy_rows(part_view(o["m"], p), mig, part_view(o["m2"], p))
            copy_rows(part_view(o["v"], p), mig, part_view(o["v2"], p))
        o["m"], o["m2"], o["v"], o["v2"] = o["m2"], o["m"], o["v2"], o["v"]
        o["steps"] = np.where(mig >= 0, o["steps"][np.maximum(mig, 0)], 0)
        mask = np.zeros(E, np.uint8)
        mask[new] = 1
        L.set_resident(mask)
        o["set"] = new

    def optimizer_step(i):
        o = opt
        o["t"] += 1
        lr = 3e-4
        # local AdamW on the resident experts (gradients of the layer's last
        # backward), writing the bf16 weights in the same pass
        n_gu = o["gu"].numel()
        if args.placement == "fixed":
            B.moe_adamw_step(o["gu"], L.dw_gate_up, o["m"][:n_gu], o["v"][:n_gu], n_gu, o["t"],
                             lr, theta_bf16=o["lp"][:n_gu])
            n_dn = o["down"].numel()
            B.moe_adamw_step(o["down"], L.dw_down, o["m"][n_gu:], o["v"][n_gu:], n_dn, o["t"],
                             lr, theta_bf16=o["lp"][n_gu:])
        else:
            # every expert at its own step count; restarted experts warm up
            # over one round
            o["steps"] = o["steps"] + 1
            lrs = B.moe_warmup_lr(o["steps"], lr, args.round_every)
            for p, grad in ((0, L.dw_gate_up), (1, L.dw_down)):
                b, e, row = o["rows"][p]
                B.moe_adamw_step_rows(th1[b:e], grad, o["m"][b:e], o["v"][b:e], Er, row,
                                      o["steps"], lrs, theta_bf16=o["lp"][b:e])
        if Hs:
            n_sg = r1 * Hs * d
            B.moe_adamw_step(o["s_master"][:n_sg], L.s_dw_gate_up, o["s_m"][:n_sg],
                             o["s_v"][:n_sg], n_sg, o["t"], lr, theta_bf16=o["s_lp"][:n_sg])
            B.moe_adamw_step(o["s_master"][n_sg:], L.s_dw_down, o["s_m"][n_sg:], o["s_v"][n_sg:],
                             Hs * d, o["t"], lr, theta_bf16=o["s_lp"][n_sg:])
        if (i + 1) % args.round_every == 0:
            # round boundary: replica-group average of the pseudo-gradient,
            # outer Nesterov step, every replica restarts from its result
            expert_delta(th0, th1, peers, delta_avg=avg)
            B.moe_outer_nesterov(th0, th1, avg, o["mom"], n_params, 0.7, 0.9, theta_bf16=o["lp"])
            if args.placement == "random" and ((i + 1) // args.round_every) % args.reshuffle_every == 0:
                reshuffle()

    def step(i):
        L.forward(x, wr, wgu, wd, bias, sgu, sd)
        L.backward(dy, x, wr, wgu, wd, sgu, sd)
        if opt is not None:
            optimizer_step(i)
        elif (i + 1) % args.round_every == 0:
            expert_delta(th0, th1, peers, delta_avg=avg)

    if args.traffic_calibration:
        from paper_2606_19025_amd.profiling import CALIBRATION_BYTES
        src = torch.ones(CALIBRATION_BYTES, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"[bench] calibration copy of {CALIBRATION_BYTES} B done")

    log(f"[bench] warmup {args.warmup}")
    for i in range(args.warmup):
        step(i)
    expert_delta(th0, th1, peers, delta_avg=avg)
    torch.cuda.synchronize()

    log(f"[bench] timing {args.steps} steps")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for i in range(args.steps):
        step(i)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = ev0.elapsed_time(ev1)
    ms_per_step = ms_total / args.steps
    value = T / (ms_per_step / 1e3)
    n = int(L.offsets[-1].item())
    local = L.topk_local.cpu().numpy()
    t_act = int((local >= 0).any(axis=1).sum())
    log(f"[bench] {ms_per_step:.3f} ms/step ({wall:.2f} s wall), n={n}, tokens/s={value:.4g}")

    # the spread of single steps: the same steps again, an event pair around
    # each (a round-boundary step includes the expert delta)
    import numpy as np
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for i in range(args.steps):
        evs[i][0].record()
        step(i)
        evs[i][1].record()
    torch.cuda.synchronize()
    per = np.array([a.elapsed_time(b) for a, b in evs])
    step_spread = {"median_ms": round(float(np.median(per)), 4),
                   "p10_ms": round(float(np.percentile(per, 10)), 4),
                   "p90_ms": round(float(np.percentile(per, 90)), 4)}

    kernels = {}
    roofline = None
    if not args.no_kernel_timing:
        B.moe_timing_enable(256 * (args.steps + 2))
        torch.cuda.synchronize()
        if opt is not None and args.placement == "random":
            opt["copy_bytes"] = 0.0
        for i in range(args.steps):
            step(i)
        if opt is not None and args.placement == "random":
            opt["copy_bytes_timed"] = opt["copy_bytes"]
        torch.cuda.synchronize()
        stats = B.moe_timing_collect()
        B.moe_timing_enable(0)
        work = algorithmic_work(cfg, n, t_act, s_bytes, args.expert)
        n_delta = args.steps // args.round_every
        work["expert_delta"] = ("byte", 4.0 * n_params * (3 + len(peers)))
        if opt is not None:
            work.update(optimizer_work(n_params + (r1 + 1) * Hs * d, n_params, len(peers)))
            if args.placement == "random":
                # bytes of the timed pass's migration copies, spread per step
                work["copy_expert_rows"] = ("byte", opt["copy_bytes_timed"] / args.steps)
        per_round = ("expert_delta", "outer_nesterov", "replica_mean")
        for name, (launches, tot, mn, mx) in stats.items():
            kind, per_step = work.get(name, ("byte", 0.0))
            steps_with = n_delta if name in per_round else args.steps
            amount = per_step * steps_with
            rate = amount / (tot / 1e3) if tot > 0 else 0.0
            if kind == "flop":
                ent = dict(unit="TFLOP/s", achieved=rate / 1e12,
                           peak=PEAK_BF16_TFLOPS if s_bytes == 2 else PEAK_F32_TFLOPS)
            else:
                ent = dict(unit="GB/s", achieved=rate / 1e9, peak=PEAK_HBM_GBS)
            ent["frac"] = ent["achieved"] / ent["peak"]
            ent.update(launches=launches, avg_us=1e3 * tot / max(launches, 1),
                       ms_per_step=tot / args.steps,
                       per_launch=amount / max(launches, 1))
            kernels[name] = {k2: (round(v, 5) if isinstance(v, float) else v) for k2, v in ent.items()}
        dom = max((nm for nm in kernels if nm not in per_round + ("copy_expert_rows",)),
                  key=lambda nm: kernels[nm]["ms_per_step"])
        kd = kernels[dom]
        kind, per_step = work[dom]
        # HBM bytes per launch from the committed rocprofv3 counter summary of
        # this workload, only while the kernel's source is the one measured
        from paper_2606_19025_amd.profiling import load_traffic, source_digest
        tr = load_traffic(os.path.join(ROOT, "profiles", f"hbm_traffic_{cfg['name']}.txt"))
        traffic = None
        if dom in tr and tr[dom][1] == source_digest(dom):
            traffic = tr[dom][0]
        roofline = dict(kernel=dom, bound="mfma" if kind == "flop" else "hbm",
                        achieved=kd["achieved"], peak=kd["peak"], unit=kd["unit"],
                        frac=kd["frac"], avg_us=kd["avg_us"],
                        per_launch=per_step / max(1, kd["launches"] // args.steps),
                        traffic=traffic)

    kernels_cold = {}
    if not args.no_kernel_timing and args.cold_steps > 0:
        # cold per-kernel samples: before every library call a read of a
        # 512 MiB scratch buffer evicts L2 and the 256 MB Infinity Cache, so
        # each call's first kernel reads its inputs from HBM (later kernels of
        # the same call read what the earlier ones just wrote).  A read, not a
        # write, so that the caches hold clean lines and the timed kernel
        # does not also pay for the write-back of the scratch data.
        flush = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")

        def evict():
            flush.sum()

        log(f"[bench] cold pass: {args.cold_steps} steps, cache flush before every call")
        B.moe_timing_enable(256 * (args.cold_steps + 2))
        torch.cuda.synchronize()
        for i in range(args.cold_steps):
            L.forward(x, wr, wgu, wd, bias, sgu, sd, hook=evict)
            L.backward(dy, x, wr, wgu, wd, sgu, sd, hook=evict)
            evict()
            expert_delta(th0, th1, peers, delta_avg=avg)
        torch.cuda.synchronize()
        stats = B.moe_timing_collect()
        B.moe_timing_enable(0)
        del flush
        work = algorithmic_work(cfg, n, t_act, s_bytes, args.expert)
        work["expert_delta"] = ("byte", 4.0 * n_params * (3 + len(peers)))
        for name, (launches, tot, mn, mx) in stats.items():
            kind, per_step = work.get(name, ("byte", 0.0))
            if kind != "byte" or per_step <= 0:
                continue
            amount = per_step * args.cold_steps
            ach = amount / (tot / 1e3) / 1e9 if tot > 0 else 0.0
            kernels_cold[name] = dict(unit="GB/s", achieved=round(ach, 3), peak=PEAK_HBM_GBS,
                                      frac=round(ach / PEAK_HBM_GBS, 5), launches=launches,
                                      avg_us=round(1e3 * tot / max(launches, 1), 3))
            sb = survey_bytes(cfg, n, s_bytes).get(name)
            if sb is not None and tot > 0:
                # the same duration under the scope table's byte formula
                ach_s = sb * args.cold_steps / (tot / 1e3) / 1e9
                kernels_cold[name].update(achieved_survey=round(ach_s, 3),
                                          frac_survey=round(ach_s / PEAK_HBM_GBS, 5))

    hbm_copy = None
    if args.copy_baseline:
        # context for the HBM-bound kernels: a plain streaming copy (2 GiB
        # moved) and a read-only sum of 1 GiB, event-timed, best of 5 after
        # one untimed call
        nb = 1 << 30
        src = torch.ones(nb // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)

        def best_ms(fn):
            ts = []
            for _ in range(6):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                fn()
                e1.record()
                e1.synchronize()
                ts.append(e0.elapsed_time(e1))
            return min(ts[1:])

        t_copy = best_ms(lambda: dst.copy_(src))
        t_read = best_ms(lambda: src.sum())
        hbm_copy = {"bytes": nb, "copy_GBps": round(2 * nb / t_copy / 1e6, 1),
                    "read_GBps": round(nb / t_read / 1e6, 1), "peak": PEAK_HBM_GBS}
        # the same copy at each cold-timed kernel's own size (half its bytes
        # read, half written), the caches flushed before every timed call as
        # in the cold pass: what a streaming kernel of that size reaches
        if kernels_cold:
            flush = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
            at_size = {}
            for name, ent in kernels_cold.items():
                moved = ent["achieved"] * 1e9 * ent["avg_us"] * 1e-6  # algorithmic bytes
                # fp32 elements of each half, at most the 1 GiB buffers
                half = min(max(int(moved / 8) // 4 * 4, 4), src.numel())
                a_, b_ = src[:half], dst[:half]
                ts = []
                for _ in range(6):
                    flush.sum()
                    e0 = torch.cuda.Event(enable_timing=True)
                    e1 = torch.cuda.Event(enable_timing=True)
                    e0.record()
                    b_.copy_(a_)
                    e1.record()
                    e1.synchronize()
                    ts.append(e0.elapsed_time(e1))
                rate = 2 * 4 * half / min(ts[1:]) / 1e6
                at_size[name] = {"bytes": 8 * half, "copy_GBps": round(rate, 1)}
                ent["frac_of_copy_at_size"] = round(ent["achieved"] / rate, 4)
            hbm_copy["cold_copy_at_kernel_size"] = at_size
            del flush
        del src, dst
        log(f"[bench] copy baseline {hbm_copy}")

    blas = None
    if args.blas_reference and s_bytes == 2:
        blas = blas_reference(cfg, n, args.expert)
        log(f"[bench] hipBLASLt dense reference {blas}")

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import moe_oracle as O
        ts = args.cpu_sample_tokens or T
        sample = inp if ts == T else I.make_layer_inputs(wl, seed=args.seed, T=ts)
        try:
            from threadpoolctl import threadpool_info
            blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        except Exception:  # pragma: no cover
            blas_threads = None
        cores = len(os.sched_getaffinity(0))
        log(f"[bench] cpu oracle on {ts} tokens ({cores} cores)")
        reps, csec = 0, 0.0
        while reps < 5 and (reps == 0 or csec < 10.0):  # about 10 s of CPU work
            c0 = time.perf_counter()
            f = O.layer_fwd(sample)
            O.layer_bwd(sample, f, sample["dy"])
            csec += time.perf_counter() - c0
            reps += 1
            log(f"[bench] cpu oracle pass {reps}: {csec:.1f} s")
        cpu = dict(value=round(reps * ts / csec, 3), unit="tokens/s", cores=blas_threads or cores,
                   kind="oracle", seconds=round(csec, 2),
                   sample=f"{reps} pass(es) of fwd+bwd over {ts} of {T} tokens of the same "
                          f"workload, fp64 NumPy oracle (round-boundary delta not included); "
                          f"{cores} cores in the affinity mask, BLAS threads {blas_threads}")

    out = {
        "metric": ("MoE layer training step (fwd+bwd+AdamW) tokens/s (1 GPU)" if opt is not None
                   else "MoE layer fwd+bwd tokens/s (1 GPU)"),
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "step_spread": step_spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if s_bytes == 2 else "f32",
        "data": "synthetic (seeded, shapes of the workload)",
        "config": {"workload": cfg["name"], "T": T, "d": d, "E": E, "E_resident": Er, "k": k,
                   "H": H, "shared_hidden": Hs, "round_every": args.round_every,
                   "executed_routes": n, "skip_fraction": round(1 - n / (T * k), 4),
                   "optimizer": "adamw+outer-nesterov" if opt is not None else None,
                   "placement": args.placement if opt is not None else None,
                   "expert": args.expert},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "kernels_cold": kernels_cold,
        "hbm_copy": hbm_copy,
        "blas_reference": blas,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
