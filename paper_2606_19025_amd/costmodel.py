"""Analytic cost model of federated MoE training with partial expert replication.

The paper's compute, memory, communication and wall-clock model (Sec. 4 and
App. D), as plain functions of the partitioning (M workers, overlap O_e,
N_le = O_e N_e / M local experts), the synchronisation interval K, the batch
and the hardware.  Nothing here runs on the GPU; the layer's own measured
step time can be put in for t_comp.

Compute (Sec. 4.1): per-token flops, eq. flops_per_token (partitioned router)
and eq. flops_per_token_st (skip-token, with sigma_st = N_le / N_e, eq.
skip_token_scaling); memory: about 18 bytes per parameter for mixed-precision
AdamW, the expert share scaled by O_e / M.
Communication (Sec. 4.2): dense ring all-reduce 2 (M - 1) / M S_dense
(eq. dense_bytes_cost); experts: ring factor R = 2 (O_e - 1) / O_e (eq.
experts_ring_factor) plus the migration factor P = gamma (1 - O_e / M) (eq.
experts_broadcast) times the local expert bytes (eq. sparse_bytes_cost);
LocalAdamW multiplies the expert payload by 3; bytes per token
BPT = M B_site / (K B_g).
Time (Sec. 4.3): t_comp = F_token (B_g / M) / (MFU Phi_peak);
t_comm = rho (B_dense + B_sparse) / B_eff; the total over N_tok tokens,
T_tot = N_tok / (M B_l K) [K t_comp + (1 - alpha) t_comm] (eq. master_equation).
"""
from __future__ import annotations

import argparse
from dataclasses import dataclass

BYTES_PER_PARAM = 2 + 4 + 8 + 4  # fp16 weights, fp32 master, two moments, gradients
LOCALADAMW_FACTOR = 3.0         # parameters plus both moments


def local_experts(N_e: int, O_e: int, M: int) -> float:
    """N_le = O_e N_e / M."""
    return O_e * N_e / M


def skip_token_scale(N_le: float, N_e: int) -> float:
    """sigma_st = N_le / N_e: the executed fraction of routes under balanced
    routing with ghost experts skipped."""
    return N_le / N_e


@dataclass
class MoELayerCost:
    """Per-token flops of one MoE layer: F_ffn of the unpartitioned expert
    FFNs (all k routes), F_gate of the full router."""
    F_ffn: float
    F_gate: float
    N_e: int
    k: int


def flops_per_token(F_dense: float, layers: list[MoELayerCost], O_e: int, M: int,
                    skip_token: bool = False) -> float:
    """F_token = F_dense + sum_l (s min(k, N_le)/k F_ffn + N_le/N_e F_gate),
    s = sigma_st with skip-token, else 1 (the equations as printed)."""
    total = F_dense
    for c in layers:
        n_le = local_experts(c.N_e, O_e, M)
        s = skip_token_scale(n_le, c.N_e) if skip_token else 1.0
        total += s * min(c.k, n_le) / c.k * c.F_ffn + n_le / c.N_e * c.F_gate
    return total


def steady_state_memory(expert_params: float, dense_params: float, O_e: int, M: int,
                        bytes_per_param: float = BYTES_PER_PARAM) -> float:
    """Bytes per site: (O_e / M expert_params + dense_params) bytes_per_param,
    with the parameter counts of all experts and of the dense part."""
    return (O_e / M * expert_params + dense_params) * bytes_per_param


def dense_bytes(M: int, S_dense: float) -> float:
    """Ring all-reduce of the replicated parameters: 2 (M - 1) / M S_dense."""
    return 2.0 * (M - 1) / M * S_dense


def ring_factor(O_e: int) -> float:
    """R(O_e) = 2 (O_e - 1) / O_e (0 for disjoint experts)."""
    return 2.0 * (O_e - 1) / O_e


def p_hit(O_e: int, M: int) -> float:
    return O_e / M


def p_miss(O_e: int, M: int) -> float:
    return 1.0 - O_e / M


def migration_factor(O_e: int, M: int, gamma: float) -> float:
    """P(O_e, M, gamma) = gamma (1 - O_e / M); gamma = 0 fixed, 1 random placement."""
    return gamma * p_miss(O_e, M)


def sparse_bytes(O_e: int, M: int, gamma: float, local_expert_bytes: float,
                 localadamw: bool = False) -> float:
    """(R + P) sum_l N_le s_expert; local_expert_bytes = sum_l N_le s_expert."""
    b = (ring_factor(O_e) + migration_factor(O_e, M, gamma)) * local_expert_bytes
    return b * (LOCALADAMW_FACTOR if localadamw else 1.0)


def bytes_per_token(B_site: float, K: int, B_g: float, M: int) -> float:
    """BPT = B_site / (K B_l) = M B_site / (K B_g)."""
    return M * B_site / (K * B_g)


def t_comp(F_token: float, B_g: float, M: int, mfu: float, peak_flops: float) -> float:
    """Seconds per local step: F_token (B_g / M) / (MFU Phi_peak)."""
    return F_token * (B_g / M) / (mfu * peak_flops)


def t_comm(B_dense: float, B_sparse: float, B_eff: float, rho: float = 1.0) -> float:
    """Seconds per synchronisation: rho (B_dense + B_sparse) / B_eff (bytes/s)."""
    return rho * (B_dense + B_sparse) / B_eff


def t_total(N_tok: float, M: int, B_l: float, K: int, tc: float, tm: float,
            alpha: float = 0.0) -> float:
    """T_tot = N_tok / (M B_l K) [K t_comp + (1 - alpha) t_comm]."""
    return N_tok / (M * B_l * K) * (K * tc + (1.0 - alpha) * tm)


def main() -> None:
    """Per-site payload and bytes per token for a layer shaped like the
    fine-grained workload, over the overlap factor."""
    ap = argparse.ArgumentParser()
    ap.add_argument("--M", type=int, default=8)
    ap.add_argument("--N-e", type=int, default=64)
    ap.add_argument("--d", type=int, default=2048)
    ap.add_argument("--H", type=int, default=1408)
    ap.add_argument("--K", type=int, default=32)
    ap.add_argument("--B-g", type=float, default=8 * 8192, help="global batch in tokens")
    ap.add_argument("--gamma", type=float, default=0.0)
    a = ap.parse_args()
    s_expert = 3 * a.H * a.d * 2  # bf16 SwiGLU expert bytes
    print("O_e  N_le  R      P      sparse_MB  BPT")
    O_e = 1
    while O_e <= a.M:
        if (a.N_e * O_e) % a.M == 0:
            n_le = local_experts(a.N_e, O_e, a.M)
            b = sparse_bytes(O_e, a.M, a.gamma, n_le * s_expert)
            print(f"{O_e:<4d} {n_le:<5g} {ring_factor(O_e):<6.3f} "
                  f"{migration_factor(O_e, a.M, a.gamma):<6.3f} {b / 1e6:<10.1f} "
                  f"{bytes_per_token(b, a.K, a.B_g, a.M):.1f}")
        O_e *= 2


if __name__ == "__main__":
    main()
