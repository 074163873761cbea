"""Plain CPU oracle of the resident-expert MoE layer (fp64 NumPy).

TEST INFRASTRUCTURE.  Only tests/, the package's smoke() entry and bench.py's
cpu_baseline leg may import this module.  It shares no code with the HIP path
and imports nothing from it.  It is written to be read against the paper, not
to be fast: no blocking, no fusion, no reordering beyond what the definitions
state.

What it computes (arxiv 2606.19025):

* The layer output is the gate-weighted sum of the selected experts' outputs,
  y = sum_{i in T(x)} s_i(x) E_i(x), with T(x) the top-k of the router scores
  (App. A, "MoE architectures and scaling", the two displayed equations;
  App. B.3 "Sigmoid Routing").
* Skip-token (Sec. 3.3 "Ghost Experts and Skip-Token"; Fig. "skipped-token"):
  the router is NOT partitioned, so T(x) is chosen over all E experts; a route
  whose expert is not resident on this worker (a "ghost expert") is dropped
  from the local computation graph.  It contributes nothing to y and receives
  no gradient through an expert path.  The gate weights of the surviving
  routes are NOT renormalised over the surviving routes (App. B.3: the
  unavailability of an expert must not skew the distribution over the
  remaining ones).
* Partitioned router (the paper's default mode; Sec. 3.3 opening paragraph,
  App. D "Router Efficiency"): partition_router() restates a step as the same
  layer over the resident experts alone, with top-min(k, N_le) routing.
* The worker holds a resident subset S_m of the experts (Sec. 3.3.1/3.3.2 and
  Alg. 1); routing is strictly local (Sec. 3.3.2 "System context and routing
  logic"), so the dispatch groups routes only by resident expert.
* Expert FFN: SwiGLU without biases, hidden H (the workloads' choice), or,
  with cfg["expert"] = "silu", the paper's own expert (App. B.3.1): a
  projection to H followed by SiLU and the projection back.
  Shared experts are dense, always active, weight 1 (Sec. 3.2).
* Round boundary (Alg. 2 "Simplified View"; Sec. 3.4): the expert-wise
  pseudo-gradient delta theta_start - theta_now of each resident expert,
  averaged over the expert's replica group.

Readings where the paper is silent (each is a convention of this build):
  gate "softmax_topk" = softmax over all E experts renormalised over the global
  top-k (before masking), so the k weights sum to 1; "softmax" = raw softmax
  probabilities of the selected experts; "sigmoid" = the paper's sigma-MoE gate.
  Selection is on the logits; ties go to the lower expert id.  Router
  temperature enters as z = (x W_r^T + b) * inv_tau.  Dispatch order: groups in
  ascending resident id, tokens ascending inside a group.  Dropless (no
  capacity factor).  Delta average order: (((d0 + d1) + d2) + ...) * fp32(1/S).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def _f64(a):
    return np.asarray(a, dtype=F64)


# --------------------------------------------------------------------------
# Routing: logits, top-k selection, gate weights, residency mask
# --------------------------------------------------------------------------

def router_logits(x, w_router, inv_tau=1.0, bias=None):
    """z_t = (x_t . W_r^T + b) * inv_tau over ALL E experts.

    Skip-token keeps the router unpartitioned (Sec. 3.3 "Ghost Experts and
    Skip-Token"), so every worker scores every expert; the router is the
    gating projection of App. B.3.2.
    """
    z = _f64(x) @ _f64(w_router).T
    if bias is not None:
        z = z + _f64(bias)[None, :]
    return z * F64(inv_tau)


def topk_select(z, k):
    """T(x): the k experts with the largest logits, ties to the lower id.

    App. A (TopK of the router scores).  The score map (sigmoid or softmax) is
    monotone, so selecting on logits selects the same set.
    """
    z = _f64(z)
    Tn, E = z.shape
    idx = np.empty((Tn, k), dtype=np.int64)
    for t in range(Tn):
        # stable sort of -z keeps equal logits in ascending expert id
        order = np.argsort(-z[t], kind="stable")
        idx[t] = order[:k]
    return idx


def gate_weights(z, idx, gate="softmax_topk"):
    """s_i(x) for the selected experts (App. A; App. B.3.2 for sigmoid)."""
    z = _f64(z)
    Tn, k = idx.shape
    w = np.empty((Tn, k), dtype=F64)
    for t in range(Tn):
        zs = z[t, idx[t]]
        if gate == "sigmoid":
            w[t] = 1.0 / (1.0 + np.exp(-zs))
        elif gate == "softmax":
            m = z[t].max()
            e = np.exp(z[t] - m)
            w[t] = e[idx[t]] / e.sum()
        elif gate == "softmax_topk":
            m = zs.max()
            e = np.exp(zs - m)
            w[t] = e / e.sum()
        else:
            raise ValueError(gate)
    return w


def resident_local_ids(resident):
    """local id of every expert: its rank in the sorted resident set, -1 if ghost."""
    resident = np.asarray(resident).astype(bool)
    local = np.full(resident.shape[0], -1, dtype=np.int64)
    r = 0
    for e in range(resident.shape[0]):
        if resident[e]:
            local[e] = r
            r += 1
    return local


def mask_routes(idx, resident):
    """Ghost-expert mask (Sec. 3.3): local expert id per route, -1 for a ghost."""
    lid = resident_local_ids(resident)
    return lid[idx]


def route(x, w_router, k, resident, inv_tau=1.0, gate="softmax_topk", bias=None):
    z = router_logits(x, w_router, inv_tau, bias)
    idx = topk_select(z, k)
    w = gate_weights(z, idx, gate)
    local = mask_routes(idx, resident)
    return dict(logits=z, idx=idx, w=w, local=local)


# --------------------------------------------------------------------------
# Dispatch: stable grouping of the resident routes by local expert
# --------------------------------------------------------------------------

def dispatch_plan(local, E_r):
    """counts, exclusive-scan offsets, perm (route id t*k+j per slot) and inv_perm.

    Tokens go only to experts hosted on this worker (Sec. 3.3.2 "System
    context and routing logic"); ghost routes get no slot (inv_perm = -1).
    """
    local = np.asarray(local)
    Tn, k = local.shape
    counts = np.zeros(E_r, dtype=np.int64)
    for t in range(Tn):
        for j in range(k):
            if local[t, j] >= 0:
                counts[local[t, j]] += 1
    offsets = np.zeros(E_r + 1, dtype=np.int64)
    for r in range(E_r):
        offsets[r + 1] = offsets[r] + counts[r]
    perm = []
    inv_perm = np.full((Tn, k), -1, dtype=np.int64)
    for r in range(E_r):
        for t in range(Tn):
            for j in range(k):
                if local[t, j] == r:
                    inv_perm[t, j] = len(perm)
                    perm.append(t * k + j)
    return dict(counts=counts, offsets=offsets, perm=np.array(perm, dtype=np.int64),
                inv_perm=inv_perm)


def gather_rows(x, perm, k):
    """Xp[p] = x[perm[p] // k]."""
    x = _f64(x)
    return x[np.asarray(perm, dtype=np.int64) // k] if len(perm) else np.zeros((0, x.shape[1]))


# --------------------------------------------------------------------------
# Expert FFN (SwiGLU, no biases)
# --------------------------------------------------------------------------

def silu(a):
    return a / (1.0 + np.exp(-a))


def swiglu_fwd(X, w_gate_up, w_down):
    """One expert: G = X Wg^T, U = X Wu^T, Hh = silu(G)*U, Y = Hh Wd^T.

    w_gate_up [2H, d] holds the gate rows then the up rows; w_down [d, H].
    """
    X = _f64(X)
    H = w_gate_up.shape[0] // 2
    Wg = _f64(w_gate_up[:H])
    Wu = _f64(w_gate_up[H:])
    G = X @ Wg.T
    U = X @ Wu.T
    Hh = silu(G) * U
    Y = Hh @ _f64(w_down).T
    return dict(G=G, U=U, Hh=Hh, Y=Y)


def swiglu_bwd(dY, X, G, U, Hh, w_gate_up, w_down):
    """Chain rule of swiglu_fwd for one expert.

    dHh = dY Wd; dWd = dY^T Hh; dG = dHh*U*silu'(G); dU = dHh*silu(G);
    dX = dG Wg + dU Wu; dWg = dG^T X; dWu = dU^T X.
    """
    dY, X, G, U, Hh = map(_f64, (dY, X, G, U, Hh))
    H = w_gate_up.shape[0] // 2
    Wg = _f64(w_gate_up[:H])
    Wu = _f64(w_gate_up[H:])
    Wd = _f64(w_down)
    dHh = dY @ Wd
    dWd = dY.T @ Hh
    sg = 1.0 / (1.0 + np.exp(-G))
    dG = dHh * U * (sg * (1.0 + G * (1.0 - sg)))
    dU = dHh * (G * sg)
    dX = dG @ Wg + dU @ Wu
    dWgu = np.concatenate([dG.T @ X, dU.T @ X], axis=0)
    return dict(dHh=dHh, dG=dG, dU=dU, dX=dX, dW_gate_up=dWgu, dW_down=dWd)


def silu_mlp_fwd(X, w_up, w_down):
    """The paper's own expert (App. B.3.1): a projection to the expert's hidden
    size followed by SiLU, then the projection back (no biases):
    A = X W1^T, Hh = silu(A), Y = Hh W2^T; w_up [H, d], w_down [d, H].
    Returned in the SwiGLU layout with G = A and no U."""
    X = _f64(X)
    A = X @ _f64(w_up).T
    Hh = silu(A)
    return dict(G=A, U=None, Hh=Hh, Y=Hh @ _f64(w_down).T)


def silu_mlp_bwd(dY, X, A, Hh, w_up, w_down):
    """Chain rule of silu_mlp_fwd: dHh = dY W2; dW2 = dY^T Hh;
    dA = dHh silu'(A); dX = dA W1; dW1 = dA^T X."""
    dY, X, A, Hh = map(_f64, (dY, X, A, Hh))
    dHh = dY @ _f64(w_down)
    sg = 1.0 / (1.0 + np.exp(-A))
    dA = dHh * (sg * (1.0 + A * (1.0 - sg)))
    return dict(dHh=dHh, dG=dA, dU=None, dX=dA @ _f64(w_up), dW_gate_up=dA.T @ X,
                dW_down=dY.T @ Hh)


EXPERTS = ("swiglu", "silu")


def expert_hidden(w_gate_up, expert):
    """Hidden size H of one expert's first weight: [2H, d] (SwiGLU) or [H, d]."""
    return w_gate_up.shape[-2] // (2 if expert == "swiglu" else 1)


def grouped_ffn_fwd(Xp, offsets, w_gate_up, w_down, expert="swiglu"):
    """Per resident group r: rows [offsets[r], offsets[r+1]) of Xp through expert r."""
    Xp = _f64(Xp)
    n = int(offsets[-1])
    H = expert_hidden(w_gate_up, expert)
    d = w_down.shape[1]
    G = np.zeros((n, H)); Hh = np.zeros((n, H)); Y = np.zeros((n, d))
    U = np.zeros((n, H)) if expert == "swiglu" else None
    for r in range(len(offsets) - 1):
        a, b = int(offsets[r]), int(offsets[r + 1])
        if b > a:
            if expert == "swiglu":
                o = swiglu_fwd(Xp[a:b], w_gate_up[r], w_down[r])
                U[a:b] = o["U"]
            else:
                o = silu_mlp_fwd(Xp[a:b], w_gate_up[r], w_down[r])
            G[a:b], Hh[a:b], Y[a:b] = o["G"], o["Hh"], o["Y"]
    return dict(G=G, U=U, Hh=Hh, Y=Y)


def grouped_ffn_bwd(dYp, Xp, G, U, Hh, offsets, w_gate_up, w_down, expert="swiglu"):
    n = int(offsets[-1])
    Er = len(offsets) - 1
    H = expert_hidden(w_gate_up, expert)
    d = w_down.shape[1]
    rows_w1 = 2 * H if expert == "swiglu" else H
    dXp = np.zeros((n, d)); dG = np.zeros((n, H))
    dU = np.zeros((n, H)) if expert == "swiglu" else None
    dWgu = np.zeros((Er, rows_w1, d)); dWd = np.zeros((Er, d, H))
    for r in range(Er):
        a, b = int(offsets[r]), int(offsets[r + 1])
        if b > a:
            if expert == "swiglu":
                o = swiglu_bwd(dYp[a:b], Xp[a:b], G[a:b], U[a:b], Hh[a:b], w_gate_up[r], w_down[r])
                dU[a:b] = o["dU"]
            else:
                o = silu_mlp_bwd(dYp[a:b], Xp[a:b], G[a:b], Hh[a:b], w_gate_up[r], w_down[r])
            dXp[a:b], dG[a:b] = o["dX"], o["dG"]
            dWgu[r], dWd[r] = o["dW_gate_up"], o["dW_down"]
    return dict(dXp=dXp, dG=dG, dU=dU, dW_gate_up=dWgu, dW_down=dWd)


# --------------------------------------------------------------------------
# Combine (weighted sum over resident routes) and its backward
# --------------------------------------------------------------------------

def combine_fwd(Yp, w, inv_perm, y_add=None):
    """y_t = sum_{j: route resident} w_tj * Yp[inv_perm[t,j]]  (+ y_add_t).

    A route to a ghost expert contributes nothing (Sec. 3.3); a token whose
    k routes are all ghosts gets exactly y_add_t (0 without shared experts).
    """
    Yp = _f64(Yp)
    Tn, k = inv_perm.shape
    y = np.zeros((Tn, Yp.shape[1]))
    for t in range(Tn):
        for j in range(k):
            p = inv_perm[t, j]
            if p >= 0:
                y[t] += F64(w[t, j]) * Yp[p]
    if y_add is not None:
        y = y + _f64(y_add)
    return y


def combine_bwd(dy, Yp, w, inv_perm):
    """dYp[p] = w_tj * dy_t ; dw_tj = <dy_t, Yp[p]>  (0 for a ghost route)."""
    dy = _f64(dy); Yp = _f64(Yp)
    Tn, k = inv_perm.shape
    dYp = np.zeros_like(Yp)
    dw = np.zeros((Tn, k))
    for t in range(Tn):
        for j in range(k):
            p = inv_perm[t, j]
            if p >= 0:
                dYp[p] = F64(w[t, j]) * dy[t]
                dw[t, j] = dy[t] @ Yp[p]
    return dict(dYp=dYp, dw=dw)


def dispatch_bwd(dXp, inv_perm, d, dx_add=None):
    """dx_t = sum_{j: resident} dXp[inv_perm[t,j]]  (+ dx_add_t)."""
    dXp = _f64(dXp)
    Tn, k = inv_perm.shape
    dx = np.zeros((Tn, d))
    for t in range(Tn):
        for j in range(k):
            p = inv_perm[t, j]
            if p >= 0:
                dx[t] += dXp[p]
    if dx_add is not None:
        dx = dx + _f64(dx_add)
    return dx


# --------------------------------------------------------------------------
# Router backward
# --------------------------------------------------------------------------

def gate_bwd(z, idx, w, dw, gate="softmax_topk"):
    """dL/dz [T, E] from dL/dw [T, k], with the top-k set held fixed.

    softmax_topk: w = softmax over the selected logits -> dz_Kj = w_j (dw_j - <w, dw>)
    softmax:      w_j = p_Kj, p = softmax(z) over all E -> dz_e = p_e (g_e - <w, dw>),
                  g_e = dw_j where e = K_j, else 0
    sigmoid:      dz_Kj = dw_j w_j (1 - w_j)
    """
    z = _f64(z); w = _f64(w); dw = _f64(dw)
    Tn, E = z.shape
    k = idx.shape[1]
    dz = np.zeros((Tn, E))
    for t in range(Tn):
        if gate == "softmax_topk":
            s = float(w[t] @ dw[t])
            for j in range(k):
                dz[t, idx[t, j]] = w[t, j] * (dw[t, j] - s)
        elif gate == "softmax":
            p = np.exp(z[t] - z[t].max()); p /= p.sum()
            g = np.zeros(E)
            for j in range(k):
                g[idx[t, j]] = dw[t, j]
            dz[t] = p * (g - float(w[t] @ dw[t]))
        elif gate == "sigmoid":
            for j in range(k):
                dz[t, idx[t, j]] = dw[t, j] * w[t, j] * (1.0 - w[t, j])
        else:
            raise ValueError(gate)
    return dz


def route_bwd(x, w_router, idx, w, logits, dw, inv_tau=1.0, gate="softmax_topk"):
    """Backward of z = (x W_r^T + b) * inv_tau through the gate weights.

    ds = dz * inv_tau;  dW_r = ds^T x;  db = sum_t ds_t;  dx_router = ds W_r.
    """
    dz = gate_bwd(logits, idx, w, dw, gate)
    ds = dz * F64(inv_tau)
    x = _f64(x)
    return dict(dz=dz, dW_router=ds.T @ x, d_bias=ds.sum(axis=0), dx=ds @ _f64(w_router))


# --------------------------------------------------------------------------
# Whole layer (composition of the steps)
# --------------------------------------------------------------------------

def layer_fwd(inp, inv_tau=1.0, gate="softmax_topk", logits=None):
    """Forward of the resident-expert layer.

    ``logits`` (optional) replaces the router projection, so the selection can
    be checked on exactly the logits another implementation produced.
    """
    cfg = inp["cfg"]
    k, E_r = cfg["k"], cfg["E_r"]
    x = _f64(inp["x"])
    if logits is None:
        z = router_logits(x, inp["w_router"], inv_tau, inp.get("router_bias"))
    else:
        z = _f64(logits)
    idx = topk_select(z, k)
    w = gate_weights(z, idx, gate)
    local = mask_routes(idx, inp["resident"])
    plan = dispatch_plan(local, E_r)
    Xp = gather_rows(x, plan["perm"], k)
    expert = cfg.get("expert", "swiglu")
    f = grouped_ffn_fwd(Xp, plan["offsets"], inp["w_gate_up"], inp["w_down"], expert)
    ys = None
    shared = None
    if inp.get("shared_gate_up") is not None:
        one = swiglu_fwd if expert == "swiglu" else silu_mlp_fwd
        shared = one(x, inp["shared_gate_up"][0], inp["shared_down"][0])
        ys = shared["Y"]
    y = combine_fwd(f["Y"], w, plan["inv_perm"], ys)
    return dict(logits=z, idx=idx, w=w, local=local, **plan, Xp=Xp, G=f["G"], U=f["U"],
                Hh=f["Hh"], Yp=f["Y"], shared=shared, y=y)


def layer_bwd(inp, fwd, dy, inv_tau=1.0, gate="softmax_topk"):
    """Backward of the resident-expert layer for upstream gradient dy."""
    cfg = inp["cfg"]
    d = cfg["d"]
    x = _f64(inp["x"])
    cb = combine_bwd(dy, fwd["Yp"], fwd["w"], fwd["inv_perm"])
    expert = cfg.get("expert", "swiglu")
    gb = grouped_ffn_bwd(cb["dYp"], fwd["Xp"], fwd["G"], fwd["U"], fwd["Hh"], fwd["offsets"],
                         inp["w_gate_up"], inp["w_down"], expert)
    dx_shared = None
    sb = None
    if fwd["shared"] is not None:
        s = fwd["shared"]
        if expert == "swiglu":
            sb = swiglu_bwd(dy, x, s["G"], s["U"], s["Hh"], inp["shared_gate_up"][0],
                            inp["shared_down"][0])
        else:
            sb = silu_mlp_bwd(dy, x, s["G"], s["Hh"], inp["shared_gate_up"][0],
                              inp["shared_down"][0])
        dx_shared = sb["dX"]
    dx = dispatch_bwd(gb["dXp"], fwd["inv_perm"], d, dx_shared)
    rb = route_bwd(x, inp["w_router"], fwd["idx"], fwd["w"], fwd["logits"], cb["dw"], inv_tau, gate)
    dx = dx + rb["dx"]
    return dict(dYp=cb["dYp"], dw=cb["dw"], dXp=gb["dXp"], dG=gb["dG"], dU=gb["dU"],
                dW_gate_up=gb["dW_gate_up"], dW_down=gb["dW_down"], shared=sb,
                dz=rb["dz"], dW_router=rb["dW_router"], d_bias=rb["d_bias"], dx=dx)


# --------------------------------------------------------------------------
# Partitioned router (the paper's default mode, compared with skip-token)
# --------------------------------------------------------------------------

def partition_router(inp):
    """The same local step with the router partitioned along with the experts.

    Sec. 3.3 ("Ghost Experts and Skip-Token", opening paragraph): in most of
    the paper's runs the router is partitioned with the experts, so a token is
    never routed to an expert the worker does not hold; App. D ("Router
    Efficiency"): the router then projects onto the N_le resident experts only;
    Sec. 3.3.1: each token takes min(k, N_le) local routes.  The partitioned
    step is therefore this layer over the resident experts alone: router rows
    W_r[S_m] (and bias entries b[S_m]), every expert resident, top-min(k, N_le).
    Expert ids in its results are local ids (rank in S_m).
    """
    res = np.flatnonzero(np.asarray(inp["resident"]))
    if len(res) == 0:
        raise ValueError("a partitioned router needs at least one resident expert")
    cfg = dict(inp["cfg"])
    out = dict(inp)
    out["w_router"] = np.asarray(inp["w_router"])[res]
    if inp.get("router_bias") is not None:
        out["router_bias"] = np.asarray(inp["router_bias"])[res]
    out["resident"] = np.ones(len(res), dtype=np.uint8)
    cfg.update(E=len(res), E_r=len(res), k=min(cfg["k"], len(res)), resident=list(range(len(res))))
    out["cfg"] = cfg
    return out


# --------------------------------------------------------------------------
# Round boundary: expert-wise pseudo-gradient delta
# --------------------------------------------------------------------------

def expert_delta(theta_start, theta_now, peers):
    """Delta of this site and its average over the replica group, in fp32.

    Alg. 2 (round end): sparse parameters are aggregated within each expert's
    replica group.  Delta_local = theta_start - theta_now; the group average is
    (((Delta_local + D_1) + D_2) + ...) * fp32(1 / (n_peers + 1)), evaluated
    in exactly that order in fp32, so the result is reproducible bit for bit.
    """
    f32 = np.float32
    a = np.asarray(theta_start, dtype=f32)
    b = np.asarray(theta_now, dtype=f32)
    dl = (a - b).astype(f32)
    acc = dl.copy()
    for p in peers:
        acc = (acc + np.asarray(p, dtype=f32)).astype(f32)
    scale = f32(1.0) / f32(len(peers) + 1)
    return dl, (acc * scale).astype(f32)


# --------------------------------------------------------------------------
# Optimisers of the resident experts (local steps and round boundary)
# --------------------------------------------------------------------------
#
# Sec. 3.4 ("Outer optimization"): workers run AdamW locally on their own
# parameters and keep the optimiser state across rounds, only for their own
# experts; the aggregated model is updated by a momentum outer optimiser.
# App. F (reproducibility details): AdamW with weight decay 0, betas (0.9, 0.95),
# eps 1e-8; the DiLoCo/Nesterov outer step uses learning rate 0.7 and
# momentum 0.9; LocalAdamW also averages the first and second moments.
# All of it is fp32 elementwise arithmetic, written here one rounding at a
# time in a fixed order, so that an fp32 implementation performing the same
# operations (correctly rounded division and square root, no fused
# multiply-add) reproduces it bit for bit.

def adamw_bias_corrections(step, beta1, beta2):
    """fp32 (1 - beta1^t, 1 - beta2^t) for step t >= 1: the betas are fp32
    hyper-parameters like every other operand here, the power is evaluated
    in fp64 from their fp32 values and the result rounded to fp32."""
    f32 = np.float32
    b1, b2 = float(f32(beta1)), float(f32(beta2))
    return f32(1.0 - b1 ** int(step)), f32(1.0 - b2 ** int(step))


def adamw_step(theta, grad, m, v, step, lr, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0):
    """One AdamW step (decoupled weight decay, Loshchilov & Hutter) in fp32.

      m' = b1 m + (1 - b1) g;  v' = b2 v + (1 - b2) g^2
      theta' = theta - lr ((m' / c1) / (sqrt(v' / c2) + eps) + wd theta)
    with c1, c2 the bias corrections of step t.  Returns (theta', m', v').
    """
    f32 = np.float32
    th, g = np.asarray(theta, f32), np.asarray(grad, f32)
    m0, v0 = np.asarray(m, f32), np.asarray(v, f32)
    b1, b2, ep, wd, lr_ = f32(beta1), f32(beta2), f32(eps), f32(weight_decay), f32(lr)
    c1, c2 = adamw_bias_corrections(step, beta1, beta2)
    m1 = (b1 * m0).astype(f32) + ((f32(1) - b1) * g).astype(f32)
    v1 = (b2 * v0).astype(f32) + ((f32(1) - b2) * (g * g).astype(f32)).astype(f32)
    mh = (m1 / c1).astype(f32)
    vh = (v1 / c2).astype(f32)
    den = (np.sqrt(vh).astype(f32) + ep).astype(f32)
    upd = ((mh / den).astype(f32) + (wd * th).astype(f32)).astype(f32)
    th1 = (th - (lr_ * upd).astype(f32)).astype(f32)
    return th1, m1.astype(f32), v1.astype(f32)


def outer_nesterov(theta_start, delta_avg, momentum, lr=0.7, mu=0.9):
    """Outer step on the replica-group average of the pseudo-gradient (Alg. 2,
    OuterOpt; DiLoCo's Nesterov momentum), in fp32:

      b' = mu b + delta;  theta' = theta_start - lr (delta + mu b')
    Returns (theta', b').  theta' is where every worker starts the next round.
    """
    f32 = np.float32
    th, dl, b = (np.asarray(a, f32) for a in (theta_start, delta_avg, momentum))
    mu_, lr_ = f32(mu), f32(lr)
    b1 = ((mu_ * b).astype(f32) + dl).astype(f32)
    upd = (dl + (mu_ * b1).astype(f32)).astype(f32)
    return (th - (lr_ * upd).astype(f32)).astype(f32), b1


def replica_mean(local, peers):
    """Average of a tensor over the expert's replica group (LocalAdamW moment
    sync): (((x + p_1) + p_2) + ...) * fp32(1 / (n_peers + 1)) in fp32."""
    f32 = np.float32
    acc = np.asarray(local, f32).copy()
    for p in peers:
        acc = (acc + np.asarray(p, f32)).astype(f32)
    return (acc * (f32(1.0) / f32(len(peers) + 1))).astype(f32)


# --------------------------------------------------------------------------
# Expert placement and migration (Alg. 1)
# --------------------------------------------------------------------------
#
# Sec. 3.3 ("Expert placement modes", Alg. 1): every expert of a layer lives on
# exactly O_e of the M workers and every worker holds N_le = O_e N_e / M
# distinct experts.  Fixed placement maps experts to workers once; random
# placement redraws the map every T rounds.  After a redraw a worker fetches
# the experts new to it (Delta_in = S^t \ S^(t-1)), keeps the optimiser state
# of the experts it already held, and restarts the state of the new ones with a
# learning-rate warm-up applied only to them (Sec. 3.4, "Outer optimization").
#
# Reading (the paper gives the constraints, not a construction): the
# placement lays the N_e O_e (expert, replica) slots out in expert order and
# deals them to the workers in turn, so expert e sits on workers
# (e O_e + j) mod M, j < O_e; random placement relabels the experts and the
# workers by two uniformly drawn permutations (passed in, so that both
# implementations see the same draw).

def gen_placement(N_e, O_e, M, expert_perm=None, worker_perm=None):
    """[M, N_le] int array: row m = the sorted expert ids worker m holds."""
    if not (1 <= O_e <= M) or (N_e * O_e) % M:
        raise ValueError("need 1 <= O_e <= M and M | N_e O_e")
    N_le = N_e * O_e // M
    ep = np.arange(N_e) if expert_perm is None else np.asarray(expert_perm)
    wp = np.arange(M) if worker_perm is None else np.asarray(worker_perm)
    sets = [[] for _ in range(M)]
    for e in range(N_e):
        for j in range(O_e):
            sets[int(wp[(e * O_e + j) % M])].append(int(ep[e]))
    out = np.array([sorted(s) for s in sets], dtype=np.int64).reshape(M, N_le)
    return out


def migration_map(prev_set, new_set):
    """For each slot of the new resident set (ascending expert id): the slot
    the expert had in the previous set (its state is kept), or -1 if the
    expert is new to the worker (Delta_in: fetched, state restarted)."""
    prev = {int(e): i for i, e in enumerate(prev_set)}
    return np.array([prev.get(int(e), -1) for e in new_set], dtype=np.int64)


def warmup_scale(steps_since_reset, warmup_steps):
    """Learning-rate factor of a reassigned expert: linear warm-up over
    warmup_steps local steps (reading: the paper does not give the shape)."""
    if warmup_steps <= 0:
        return 1.0
    return min(1.0, float(steps_since_reset) / float(warmup_steps))
