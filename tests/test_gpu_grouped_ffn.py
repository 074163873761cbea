"""Grouped expert FFN (forward and backward) through the C ABI against the
oracle, with the group sizes chosen around the GEMM tile edges.

The layer tests reach only the group sizes that routing happens to give.
Here they are set directly: empty groups (also first and last), one row, and
one below, at and above 128 rows (a wave pair's share of a tile) and the
256-row tile height; hidden and model widths that leave a partial 256-wide column tile;
K extents (d, H, 2H) of one to several k-steps of 32 and 64 and ragged token
counts for the weight-gradient kinds; the backward both without a workspace
(static tile dealing, no split) and with one (dynamic dealing, split-K of a
single large group, summed by splitk_reduce); with workspaces, launches with
far fewer tiles than CUs, whose down projection and dX cut their reduction
into parts (summed by splitk_rows_reduce).  Both expert forms.

Every output is compared with the oracle (Sec. 3.2 expert FFN per resident
expert, App. B.3.1 for the SiLU form) at the bf16 tolerance, normwise.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import moe_oracle as O
from paper_2606_19025_amd import binding as B
from paper_2606_19025_amd import inputs as I

from .parity_helpers import TOL, assert_close, canary, host, record_errors, say

pytestmark = pytest.mark.gpu

EDGES = [0, 1, 127, 128, 129, 0, 255, 256, 257, 383, 511, 513, 0]

# name: (group sizes, d, H, expert, workspace, accumulate_dw)
CASES = {
    "edges-swiglu": (EDGES, 128, 192, "swiglu", False, 0),
    "edges-swiglu-ws": (EDGES, 128, 192, "swiglu", True, 0),
    "edges-silu-ws": ([3, 128, 0, 130, 256, 300], 256, 320, "silu", True, 0),
    "accumulate-ws": ([64, 200, 0, 129], 192, 128, "swiglu", True, 1),
    "one-large-group-splitk": ([4100], 256, 256, "swiglu", True, 0),
    "one-large-group-splitk-acc": ([4100], 256, 256, "swiglu", True, 1),
    "wide-d": ([200, 700, 1], 1024, 128, "swiglu", True, 0),
    # one to four k-steps per tile for every kind (d = H = 64: one 64-deep
    # k-step for the forward GEMMs; 1-4 k-steps of 32 rows for the weight
    # gradients), so the load ring is never full
    "short-k": ([33, 64, 65, 96, 97, 0, 1, 31, 32], 64, 64, "swiglu", True, 0),
    "short-k-silu": ([33, 64, 65, 96, 97, 0, 1, 31, 32], 64, 64, "silu", False, 0),
    # far fewer output tiles than CUs with long reductions: the down
    # projection and dX cut K into parts (fp32 partial rows, then summed)
    "few-tiles-long-k": ([300, 0, 257, 511], 256, 2048, "swiglu", True, 0),
    "few-tiles-long-k-silu": ([129, 640], 512, 1536, "silu", True, 1),
}


def _bf16(g, shape, std):
    return I.bf16_round(g.standard_normal(shape, dtype=np.float32) * np.float32(std))


def _dev(a, dtype=torch.bfloat16):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda().to(dtype)


@pytest.mark.parametrize("name", sorted(CASES))
def test_grouped_ffn_tile_edges(gpu_lib, name):
    sizes, d, H, expert, use_ws, acc = CASES[name]
    say(f"[grouped-ffn] {name}")
    g = np.random.default_rng([17, len(sizes), d, H])
    G = len(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    n = int(offsets[-1])
    cap = n + 64  # rows n..cap-1 are outside every group (never converted: unset)
    r1 = 2 if expert == "swiglu" else 1
    xp = _bf16(g, (cap, d), 1.0)
    dyp = _bf16(g, (cap, d), 1.0)
    w_gu = _bf16(g, (G, r1 * H, d), d ** -0.5)
    w_d = _bf16(g, (G, d, H), H ** -0.5)
    # accumulated-into gradients small beside the step's own, so that the
    # comparison still sees the step's contribution
    dw_gu0 = (g.standard_normal((G, r1 * H, d)) * 0.01).astype(np.float32) if acc else None
    dw_d0 = (g.standard_normal((G, d, H)) * 0.01).astype(np.float32) if acc else None

    act = B.MOE_ACT_SWIGLU if expert == "swiglu" else B.MOE_ACT_SILU
    t_xp, t_dyp, t_wgu, t_wd = _dev(xp), _dev(dyp), _dev(w_gu), _dev(w_d)
    t_off = torch.from_numpy(offsets).cuda()
    # outputs start as NaN so that a row or gradient the kernels leave
    # unwritten fails the comparison
    gu = canary(cap, r1 * H)
    h = canary(cap, H)
    yp = canary(cap, d)
    dgu = canary(cap, r1 * H)
    dxp = canary(cap, d)
    t_dwgu = (torch.from_numpy(dw_gu0).cuda() if acc else canary(G, r1 * H, d, dtype=torch.float32))
    t_dwd = (torch.from_numpy(dw_d0).cuda() if acc else canary(G, d, H, dtype=torch.float32))
    fset = B.ffn_set(t_xp, t_wgu, t_wd, t_off, cap, H, G, gu, h, yp=yp, activation=act)
    fws, fws_bytes = None, 0
    if use_ws:
        fws_bytes = B.moe_grouped_ffn_fwd_workspace_size([fset], B.MOE_BF16, d)
        fws = torch.full((max(fws_bytes, 1),), 0xFF, dtype=torch.uint8, device="cuda")
    B.moe_grouped_ffn_fwd_sets([fset], B.MOE_BF16, d, fws, fws_bytes)
    bset = B.ffn_set(t_xp, t_wgu, t_wd, t_off, cap, H, G, gu, h, dyp=t_dyp, dgu=dgu, dxp=dxp,
                     dw_gate_up=t_dwgu, dw_down=t_dwd, activation=act)
    ws, ws_bytes = None, 0
    if use_ws:
        ws_bytes = B.moe_grouped_ffn_bwd_workspace_size([bset], B.MOE_BF16, d)
        ws = torch.full((ws_bytes,), 0xFF, dtype=torch.uint8, device="cuda")
    B.moe_grouped_ffn_bwd_sets([bset], B.MOE_BF16, d, acc, ws, ws_bytes)
    torch.cuda.synchronize()

    tol = TOL["bf16"]
    f = O.grouped_ffn_fwd(xp[:n], offsets, w_gu, w_d, expert)
    b = O.grouped_ffn_bwd(dyp[:n], xp[:n], f["G"], f["U"], f["Hh"], offsets, w_gu, w_d, expert)
    g_gu = host(gu[:n])
    errs = {}
    errs["G"] = assert_close("G", g_gu[:, :H], f["G"], tol)
    if expert == "swiglu":
        errs["U"] = assert_close("U", g_gu[:, H:], f["U"], tol)
    errs["h"] = assert_close("h", host(h[:n]), f["Hh"], tol)
    errs["yp"] = assert_close("yp", host(yp[:n]), f["Y"], tol)
    g_dgu = host(dgu[:n])
    errs["dG"] = assert_close("dG", g_dgu[:, :H], b["dG"], tol)
    if expert == "swiglu":
        errs["dU"] = assert_close("dU", g_dgu[:, H:], b["dU"], tol)
    errs["dxp"] = assert_close("dxp", host(dxp[:n]), b["dXp"], tol)
    want_gu = b["dW_gate_up"] + (dw_gu0 if acc else 0.0)
    want_d = b["dW_down"] + (dw_d0 if acc else 0.0)
    got_gu, got_d = host(t_dwgu), host(t_dwd)
    for r, sz in enumerate(sizes):
        # per expert: an empty group's gradient is exactly 0 (or the
        # accumulated value unchanged)
        if sz == 0:
            assert np.array_equal(got_gu[r], want_gu[r]), f"dW_gate_up of empty group {r}"
            assert np.array_equal(got_d[r], want_d[r]), f"dW_down of empty group {r}"
        else:
            errs[f"dWgu{r}"] = assert_close(f"dW_gate_up[{r}]", got_gu[r], want_gu[r], tol)
            errs[f"dWd{r}"] = assert_close(f"dW_down[{r}]", got_d[r], want_d[r], tol)
    record_errors(f"grouped_ffn[{name}]", errs)


@pytest.mark.parametrize("acc", [0, 1])
def test_grouped_ffn_single_set_entry_points(gpu_lib, acc):
    """moe_grouped_ffn_fwd / moe_grouped_ffn_bwd (one expert set, no
    workspace) against the oracle, and bit-exact against the same set passed
    through the _sets entry points without a workspace."""
    sizes, d, H = [0, 5, 128, 300, 0, 257, 64], 192, 128
    say(f"[grouped-ffn] single-set entry points accumulate={acc}")
    g = np.random.default_rng([23, acc])
    G = len(sizes)
    offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    n = int(offsets[-1])
    cap = n + 40
    xp, dyp = _bf16(g, (cap, d), 1.0), _bf16(g, (cap, d), 1.0)
    w_gu, w_d = _bf16(g, (G, 2 * H, d), d ** -0.5), _bf16(g, (G, d, H), H ** -0.5)
    dw_gu0 = (g.standard_normal((G, 2 * H, d)) * 0.01).astype(np.float32)
    dw_d0 = (g.standard_normal((G, d, H)) * 0.01).astype(np.float32)
    t_xp, t_dyp, t_wgu, t_wd = _dev(xp), _dev(dyp), _dev(w_gu), _dev(w_d)
    t_off = torch.from_numpy(offsets).cuda()

    def outputs():
        o = dict(gu=canary(cap, 2 * H), h=canary(cap, H), yp=canary(cap, d),
                 dgu=canary(cap, 2 * H), dxp=canary(cap, d))
        if acc:
            o["dwgu"], o["dwd"] = torch.from_numpy(dw_gu0).cuda(), torch.from_numpy(dw_d0).cuda()
        else:
            o["dwgu"] = canary(G, 2 * H, d, dtype=torch.float32)
            o["dwd"] = canary(G, d, H, dtype=torch.float32)
        return o

    one = outputs()
    B.moe_grouped_ffn_fwd(t_xp, t_wgu, t_wd, B.MOE_BF16, cap, d, H, G, t_off, one["gu"],
                          one["h"], one["yp"])
    B.moe_grouped_ffn_bwd(t_dyp, t_xp, one["gu"], one["h"], t_wgu, t_wd, B.MOE_BF16, cap, d, H,
                          G, t_off, one["dgu"], one["dxp"], one["dwgu"], one["dwd"], acc)
    sets = outputs()
    fset = B.ffn_set(t_xp, t_wgu, t_wd, t_off, cap, H, G, sets["gu"], sets["h"], yp=sets["yp"])
    B.moe_grouped_ffn_fwd_sets([fset], B.MOE_BF16, d)
    bset = B.ffn_set(t_xp, t_wgu, t_wd, t_off, cap, H, G, sets["gu"], sets["h"], dyp=t_dyp,
                     dgu=sets["dgu"], dxp=sets["dxp"], dw_gate_up=sets["dwgu"],
                     dw_down=sets["dwd"])
    B.moe_grouped_ffn_bwd_sets([bset], B.MOE_BF16, d, acc)
    torch.cuda.synchronize()

    rows = {"gu": n, "h": n, "yp": n, "dgu": n, "dxp": n, "dwgu": G, "dwd": G}
    for key, r in rows.items():
        a, b = one[key][:r].cpu(), sets[key][:r].cpu()
        assert torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else a.view(torch.int32),
                           b.view(torch.int16) if b.dtype == torch.bfloat16 else b.view(torch.int32)), \
            f"{key}: single-set and _sets entry points differ"

    tol = TOL["bf16"]
    f = O.grouped_ffn_fwd(xp[:n], offsets, w_gu, w_d, "swiglu")
    b = O.grouped_ffn_bwd(dyp[:n], xp[:n], f["G"], f["U"], f["Hh"], offsets, w_gu, w_d, "swiglu")
    errs = {}
    g_gu = host(one["gu"][:n])
    errs["G"] = assert_close("G", g_gu[:, :H], f["G"], tol)
    errs["U"] = assert_close("U", g_gu[:, H:], f["U"], tol)
    errs["h"] = assert_close("h", host(one["h"][:n]), f["Hh"], tol)
    errs["yp"] = assert_close("yp", host(one["yp"][:n]), f["Y"], tol)
    g_dgu = host(one["dgu"][:n])
    errs["dG"] = assert_close("dG", g_dgu[:, :H], b["dG"], tol)
    errs["dU"] = assert_close("dU", g_dgu[:, H:], b["dU"], tol)
    errs["dxp"] = assert_close("dxp", host(one["dxp"][:n]), b["dXp"], tol)
    want_gu = b["dW_gate_up"] + (dw_gu0 if acc else 0.0)
    want_d = b["dW_down"] + (dw_d0 if acc else 0.0)
    got_gu, got_d = host(one["dwgu"]), host(one["dwd"])
    for r, sz in enumerate(sizes):
        if sz == 0:
            assert np.array_equal(got_gu[r], want_gu[r]), f"dW_gate_up of empty group {r}"
            assert np.array_equal(got_d[r], want_d[r]), f"dW_down of empty group {r}"
        else:
            errs[f"dWgu{r}"] = assert_close(f"dW_gate_up[{r}]", got_gu[r], want_gu[r], tol)
            errs[f"dWd{r}"] = assert_close(f"dW_down[{r}]", got_d[r], want_d[r], tol)
    record_errors(f"grouped_ffn_single_set[acc={acc}]", errs)
