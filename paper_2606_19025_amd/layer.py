"""One worker's local step through the resident-expert MoE layer.

``ResidentMoELayer`` owns the device buffers of one layer shape and issues the
C entry points in order; it computes nothing itself.

Forward:  moe_route_mask -> moe_dispatch -> moe_grouped_ffn_fwd_sets (resident
          experts [+ shared experts on x, identity dispatch]) -> moe_combine_fwd
Backward: moe_combine_bwd -> moe_grouped_ffn_bwd_sets (resident [+ shared,
          writing dx]) -> moe_dispatch_bwd -> moe_route_bwd (adds the router's dx)
Round boundary: moe_expert_delta over the fp32 master copies.

With ``partitioned=True`` the router is partitioned along with the experts
(the paper's default mode, Sec. 3.3; App. D "Router Efficiency"): it holds
only the resident experts' rows ``w_router[E_r, d]``, every token takes
min(k, E_r) routes, all local, and expert ids are local ids.  The same entry
points run with E := E_r and every expert resident.
"""
from __future__ import annotations

import torch

from . import binding as B


class ResidentMoELayer:
    def __init__(self, T, d, E, k, H, resident, dtype=torch.bfloat16, n_shared_hidden=0,
                 gate="softmax_topk", inv_tau=1.0, device="cuda", partitioned=False,
                 expert="swiglu", canary=False):
        """canary: fill every output and workspace buffer with NaN (integers:
        -7, workspaces: 0xFF bytes) instead of leaving it uninitialised, so
        that tests see any element the kernels fail to write."""
        self.T, self.d, self.E, self.k, self.H = int(T), int(d), int(E), int(k), int(H)
        res = torch.as_tensor(resident, dtype=torch.uint8).reshape(-1)
        assert res.numel() == self.E
        self.E_r = int(res.sum().item())
        self.E_full = self.E
        self.partitioned = bool(partitioned)
        # expert form: SwiGLU ([Wg; Wu] and [G | U], 2H wide) or the paper's
        # SiLU expert (W1 and A, H wide)
        self.act = B.ACTIVATIONS[expert]
        r1 = 2 if self.act == B.MOE_ACT_SWIGLU else 1
        if self.partitioned:
            if self.E_r == 0:
                raise ValueError("a partitioned router needs at least one resident expert")
            # route over the resident experts only: E := E_r, all resident
            self.E = self.E_r
            self.k = min(self.k, self.E_r)
            res = torch.ones(self.E_r, dtype=torch.uint8)
        self.cap = self.T * min(self.k, self.E_r)
        self.dtype = dtype
        self.dt = B.MOE_BF16 if dtype == torch.bfloat16 else B.MOE_F32
        self.gate = B.GATES[gate] if isinstance(gate, str) else int(gate)
        self.inv_tau = float(inv_tau)
        self.Hs = int(n_shared_hidden)
        self.device = device
        dev = torch.device(device)
        T, d, E, k, H, cap = self.T, self.d, self.E, self.k, self.H, self.cap
        f32, i32, act = torch.float32, torch.int32, dtype
        def e(*s, dt=act):
            if not canary:
                return torch.empty(*s, dtype=dt, device=dev)
            fill = 0xFF if dt == torch.uint8 else -7 if dt == torch.int32 else float("nan")
            return torch.full(s, fill, dtype=dt, device=dev)
        self._alloc = e
        self.resident = res.to(dev)
        # routing
        self.logits = e(T, E, dt=f32)
        self.topk_idx = e(T, k, dt=i32)
        self.topk_w = e(T, k, dt=f32)
        self.topk_local = e(T, k, dt=i32)
        # dispatch
        self.counts = e(max(self.E_r, 1), dt=i32)
        self.offsets = e(self.E_r + 1, dt=i32)
        self.perm = e(max(cap, 1), dt=i32)
        self.inv_perm = e(T, k, dt=i32)
        self.ws_dispatch_bytes = B.moe_dispatch_workspace_size(T, k, self.E_r)
        self.ws_dispatch = e(self.ws_dispatch_bytes, dt=torch.uint8)
        # experts
        rows = max(cap, 1)
        self.xp = e(rows, d)
        self.gu = e(rows, r1 * H)
        self.h = e(rows, H)
        self.yp = e(rows, d)
        self.y = e(T, d)
        # backward
        self.dyp = e(rows, d)
        self.dtopk_w = e(T, k, dt=f32)
        self.dgu = e(rows, r1 * H)
        self.dxp = e(rows, d)
        self.dw_gate_up = e(max(self.E_r, 1), r1 * H, d, dt=f32)
        self.dw_down = e(max(self.E_r, 1), d, H, dt=f32)
        self.dx = e(T, d)
        self.dz = e(T, E, dt=f32)
        self.dw_router = e(E, d, dt=f32)
        self.d_bias = e(E, dt=f32)
        self.ws_route_bytes = B.moe_route_bwd_workspace_size(T, d, E)
        self.ws_route = e(self.ws_route_bytes, dt=torch.uint8)
        self.ws_ffn, self.ws_ffn_bytes = None, 0  # sized on the first backward
        self.ws_fwd, self.ws_fwd_bytes = None, 0  # sized on the first forward
        if self.Hs:
            Hs = self.Hs
            self.s_offsets = torch.tensor([0, T], dtype=i32, device=dev)
            self.s_gu = e(T, r1 * Hs)
            self.s_h = e(T, Hs)
            self.s_y = e(T, d)
            self.s_dgu = e(T, r1 * Hs)
            self.s_dw_gate_up = e(1, r1 * Hs, d, dt=f32)
            self.s_dw_down = e(1, d, Hs, dt=f32)

    def set_resident(self, resident):
        """Switch to another resident set of the same size (a new placement,
        Alg. 1).  The caller migrates the expert weights and optimiser state;
        with a partitioned router it also passes the new router rows."""
        res = torch.as_tensor(resident, dtype=torch.uint8).reshape(-1)
        if res.numel() != self.E_full or int(res.sum().item()) != self.E_r:
            raise ValueError("a new resident set must hold the same number of experts")
        if not self.partitioned:
            self.resident.copy_(res.to(self.resident.device))

    # ------------------------------------------------------------ validation
    def _check(self, name, t, shape, dtype=None):
        """Raise ValueError unless t is a contiguous tensor on this layer's
        device with the given shape and dtype (the layer's own by default)."""
        dtype = self.dtype if dtype is None else dtype
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name} must be a tensor, got {type(t).__name__}")
        if t.device != self.resident.device:
            raise ValueError(f"{name} is on {t.device}, the layer on {self.resident.device}")
        if t.dtype != dtype:
            raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")

    def _check_weights(self, x, w_router, w_gate_up, w_down, shared_gate_up, shared_down):
        r1 = 2 if self.act == B.MOE_ACT_SWIGLU else 1
        self._check("x", x, (self.T, self.d))
        self._check("w_router", w_router, (self.E, self.d))
        self._check("w_gate_up", w_gate_up, (self.E_r, r1 * self.H, self.d))
        self._check("w_down", w_down, (self.E_r, self.d, self.H))
        if self.Hs:
            self._check("shared_gate_up", shared_gate_up, (1, r1 * self.Hs, self.d))
            self._check("shared_down", shared_down, (1, self.d, self.Hs))
        elif shared_gate_up is not None or shared_down is not None:
            raise ValueError("shared expert weights given to a layer built without them")

    # ------------------------------------------------------------------ forward
    def forward(self, x, w_router, w_gate_up, w_down, router_bias=None, shared_gate_up=None,
                shared_down=None, stream=None, hook=None):
        """hook: called before each library call (e.g. a cache flush between
        kernels for cold per-kernel timing); None in normal use."""
        T, d, E, k, H, cap, dt = self.T, self.d, self.E, self.k, self.H, self.cap, self.dt
        self._check_weights(x, w_router, w_gate_up, w_down, shared_gate_up, shared_down)
        if router_bias is not None:
            self._check("router_bias", router_bias, (E,), torch.float32)
        hook = hook or (lambda: None)
        hook()
        B.moe_route_mask(x, w_router, router_bias, dt, T, d, E, k, self.inv_tau, self.gate,
                         self.resident, self.logits, self.topk_idx, self.topk_w, self.topk_local,
                         stream)
        hook()
        B.moe_dispatch(x, dt, T, d, k, self.E_r, self.topk_local, self.counts, self.offsets,
                       self.perm, self.inv_perm, self.xp, self.ws_dispatch, self.ws_dispatch_bytes,
                       stream)
        sets = [B.ffn_set(self.xp, w_gate_up, w_down, self.offsets, cap, H, self.E_r, self.gu,
                          self.h, yp=self.yp, activation=self.act)]
        y_add = None
        if self.Hs:
            # the shared experts see every token: their "dispatched rows" are x
            sets.append(B.ffn_set(x, shared_gate_up, shared_down, self.s_offsets, T, self.Hs, 1,
                                  self.s_gu, self.s_h, yp=self.s_y, activation=self.act))
            y_add = self.s_y
        if self.ws_fwd is None:
            self.ws_fwd_bytes = B.moe_grouped_ffn_fwd_workspace_size(sets, dt, d)
            self.ws_fwd = self._alloc(max(self.ws_fwd_bytes, 1), dt=torch.uint8)
        hook()
        B.moe_grouped_ffn_fwd_sets(sets, dt, d, self.ws_fwd if self.ws_fwd_bytes else None,
                                   self.ws_fwd_bytes, stream)
        hook()
        B.moe_combine_fwd(self.yp, dt, T, d, k, cap, self.topk_w, self.inv_perm, y_add, self.y,
                          stream)
        return self.y

    # ----------------------------------------------------------------- backward
    def backward(self, dy, x, w_router, w_gate_up, w_down, shared_gate_up=None, shared_down=None,
                 accumulate_dw=0, stream=None, hook=None):
        T, d, E, k, H, cap, dt = self.T, self.d, self.E, self.k, self.H, self.cap, self.dt
        self._check_weights(x, w_router, w_gate_up, w_down, shared_gate_up, shared_down)
        self._check("dy", dy, (T, d))
        hook = hook or (lambda: None)
        hook()
        B.moe_combine_bwd(dy, self.yp, dt, T, d, k, cap, self.topk_w, self.inv_perm, self.dyp,
                          self.dtopk_w, stream)
        sets = [B.ffn_set(self.xp, w_gate_up, w_down, self.offsets, cap, H, self.E_r, self.gu,
                          self.h, dyp=self.dyp, dgu=self.dgu, dxp=self.dxp,
                          dw_gate_up=self.dw_gate_up, dw_down=self.dw_down, activation=self.act)]
        if self.Hs:
            # the shared experts see every token with weight 1: their dxp is dx
            sets.append(B.ffn_set(x, shared_gate_up, shared_down, self.s_offsets, T, self.Hs, 1,
                                  self.s_gu, self.s_h, dyp=dy, dgu=self.s_dgu, dxp=self.dx,
                                  dw_gate_up=self.s_dw_gate_up, dw_down=self.s_dw_down,
                                  activation=self.act))
        if self.ws_ffn is None:
            self.ws_ffn_bytes = B.moe_grouped_ffn_bwd_workspace_size(sets, dt, d)
            self.ws_ffn = self._alloc(self.ws_ffn_bytes, dt=torch.uint8)
        hook()
        B.moe_grouped_ffn_bwd_sets(sets, dt, d, accumulate_dw, self.ws_ffn, self.ws_ffn_bytes,
                                   stream)
        hook()
        B.moe_dispatch_bwd(self.dxp, dt, T, d, k, cap, self.inv_perm, self.dx, 1 if self.Hs else 0,
                           stream)
        hook()
        B.moe_route_bwd(x, w_router, dt, T, d, E, k, self.inv_tau, self.gate, self.topk_idx,
                        self.topk_w, self.logits, self.dtopk_w, self.dz, self.dw_router,
                        self.d_bias, self.dx, 1, self.ws_route, self.ws_route_bytes, stream)
        return self.dx


def expert_delta(theta_start, theta_now, peers, delta_local=None, delta_avg=None, stream=None):
    """Round-boundary pseudo-gradient of the resident experts and its replica-group average."""
    n = theta_start.numel()
    if delta_avg is None:
        delta_avg = torch.empty_like(theta_start)
    B.moe_expert_delta(theta_start, theta_now, list(peers), len(peers), n, delta_local, delta_avg,
                       stream)
    return delta_avg
