"""ctypes binding of libmoe_resident.so (see include/moe_resident.h).

Argument marshalling only: every function here has the name of the C entry
point it calls, takes torch tensors (or None for NULL, or raw integer device
addresses), passes their device pointers and sizes through unchanged and
raises MoeError with the library's message when the status is not MOE_OK.
No arithmetic of the layer happens in Python.  There is no fallback: if the
native library is missing, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os

from .build import LIB_PATH

MOE_F32, MOE_BF16 = 0, 1
MOE_GATE_SOFTMAX_TOPK, MOE_GATE_SOFTMAX, MOE_GATE_SIGMOID = 0, 1, 2
GATES = {"softmax_topk": MOE_GATE_SOFTMAX_TOPK, "softmax": MOE_GATE_SOFTMAX,
         "sigmoid": MOE_GATE_SIGMOID}

EXPORTS = [
    "moe_last_error", "moe_abi_version", "moe_route_mask", "moe_route_bwd_workspace_size",
    "moe_route_bwd", "moe_dispatch_workspace_size", "moe_dispatch", "moe_dispatch_noalloc", "moe_dispatch_bwd",
    "moe_grouped_ffn_fwd", "moe_grouped_ffn_bwd", "moe_grouped_ffn_fwd_workspace_size",
    "moe_grouped_ffn_fwd_sets",
    "moe_grouped_ffn_bwd_workspace_size", "moe_grouped_ffn_bwd_sets", "moe_combine_fwd",
    "moe_combine_bwd",
    "moe_expert_delta", "moe_adamw_step", "moe_outer_nesterov", "moe_replica_mean",
    "moe_gen_placement", "moe_migration_map", "moe_copy_expert_rows", "moe_warmup_lr",
    "moe_adamw_step_rows", "moe_timing_enable", "moe_timing_collect",
]


class MoeError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn} returned {status}: {msg}")
        self.status = status


_lib = None

_P = C.c_void_p
_I = C.c_int
_F = C.c_float
_Z = C.c_size_t

_SIGS = {
    "moe_last_error": (C.c_char_p, []),
    "moe_abi_version": (_I, []),
    "moe_route_mask": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _F, _I, _P, _P, _P, _P, _P, _P]),
    "moe_route_bwd_workspace_size": (_Z, [_I, _I, _I]),
    "moe_route_bwd": (_I, [_P, _P, _I, _I, _I, _I, _I, _F, _I, _P, _P, _P, _P, _P, _P, _P, _P,
                           _I, _P, _Z, _P]),
    "moe_dispatch_workspace_size": (_Z, [_I, _I, _I]),
    "moe_dispatch": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P, _Z, _P]),
    "moe_dispatch_noalloc": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _P]),
    "moe_dispatch_bwd": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _I, _P]),
    "moe_grouped_ffn_fwd": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "moe_grouped_ffn_bwd": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P,
                                 _I, _P]),
    "moe_grouped_ffn_fwd_workspace_size": (_Z, [_P, _I, _I, _I]),
    "moe_grouped_ffn_fwd_sets": (_I, [_P, _I, _I, _I, _P, _Z, _P]),
    "moe_grouped_ffn_bwd_workspace_size": (_Z, [_P, _I, _I, _I]),
    "moe_grouped_ffn_bwd_sets": (_I, [_P, _I, _I, _I, _I, _P, _Z, _P]),
    "moe_combine_fwd": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "moe_combine_bwd": (_I, [_P, _P, _I, _I, _I, _I, _I, _P, _P, _P, _P, _P]),
    "moe_expert_delta": (_I, [_P, _P, C.POINTER(C.c_void_p), _I, _Z, _P, _P, _P]),
    "moe_adamw_step": (_I, [_P, _P, _P, _P, _Z, _I, _F, _F, _F, _F, _F, _P, _P]),
    "moe_outer_nesterov": (_I, [_P, _P, _P, _P, _Z, _F, _F, _P, _P]),
    "moe_replica_mean": (_I, [_P, C.POINTER(C.c_void_p), _I, _Z, _P, _P]),
    "moe_gen_placement": (_I, [_I, _I, _I, _P, _P, _P]),
    "moe_migration_map": (_I, [_P, _I, _P, _I, _P]),
    "moe_copy_expert_rows": (_I, [_P, _P, _P, _P, _I, _Z, _P, _P]),
    "moe_warmup_lr": (_I, [_P, _I, C.c_double, _I, _P]),
    "moe_adamw_step_rows": (_I, [_P, _P, _P, _P, _I, _Z, _P, _P, _F, _F, _F, _F, _P, _P]),
    "moe_timing_enable": (_I, [_I]),
    "moe_timing_collect": (_I, [_P, _I, C.POINTER(C.c_int)]),
}


class moe_kernel_time(C.Structure):
    _fields_ = [("name", C.c_char_p), ("launches", C.c_int), ("total_ms", C.c_float),
                ("min_ms", C.c_float), ("max_ms", C.c_float)]


class moe_ffn_set(C.Structure):
    """One expert set (struct moe_ffn_set of include/moe_resident.h)."""
    _fields_ = [("xp", _P), ("w_gate_up", _P), ("w_down", _P), ("offsets", _P),
                ("cap", _I), ("H", _I), ("n_groups", _I),
                ("gu", _P), ("h", _P), ("yp", _P), ("dyp", _P), ("dgu", _P), ("dxp", _P),
                ("dw_gate_up", _P), ("dw_down", _P), ("activation", _I)]


MOE_ACT_SWIGLU, MOE_ACT_SILU = 0, 1
ACTIVATIONS = {"swiglu": MOE_ACT_SWIGLU, "silu": MOE_ACT_SILU}


def ffn_set(xp, w_gate_up, w_down, offsets, cap, H, n_groups, gu, h, yp=None, dyp=None,
            dgu=None, dxp=None, dw_gate_up=None, dw_down=None, activation=MOE_ACT_SWIGLU):
    """A moe_ffn_set from tensors (or raw addresses / None)."""
    return moe_ffn_set(_ptr(xp), _ptr(w_gate_up), _ptr(w_down), _ptr(offsets), cap, H, n_groups,
                       _ptr(gu), _ptr(h), _ptr(yp), _ptr(dyp), _ptr(dgu), _ptr(dxp),
                       _ptr(dw_gate_up), _ptr(dw_down), activation)


def lib(path: str | None = None):
    """Load the native library once (raises if it has not been built)."""
    global _lib
    if _lib is None:
        p = path or LIB_PATH
        if not os.path.exists(p):
            raise RuntimeError(f"{p} is missing: build it with __graft_entry__.build() "
                               "or python -m paper_2606_19025_amd.build")
        # torch first: the library must bind to the HIP runtime torch already
        # initialised (one runtime per process)
        import torch  # noqa: F401
        handle = C.CDLL(p)
        for name, (res, args) in _SIGS.items():
            f = getattr(handle, name)
            f.restype = res
            f.argtypes = args
        _lib = handle
    return _lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(fn: str, status: int):
    if status != 0:
        raise MoeError(fn, status, lib().moe_last_error().decode())
    return status


def dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return MOE_BF16
    if t.dtype == torch.float32:
        return MOE_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def moe_last_error() -> str:
    return lib().moe_last_error().decode()


def moe_abi_version() -> int:
    return lib().moe_abi_version()


def moe_route_mask(x, w_router, router_bias, dtype, T, d, E, k, inv_tau, gate, resident, logits,
                   topk_idx, topk_w, topk_local, stream=None):
    return _check("moe_route_mask", lib().moe_route_mask(
        _ptr(x), _ptr(w_router), _ptr(router_bias), dtype, T, d, E, k, inv_tau, gate,
        _ptr(resident), _ptr(logits), _ptr(topk_idx), _ptr(topk_w), _ptr(topk_local),
        _stream(stream)))


def moe_route_bwd_workspace_size(T, d, E) -> int:
    return lib().moe_route_bwd_workspace_size(T, d, E)


def moe_route_bwd(x, w_router, dtype, T, d, E, k, inv_tau, gate, topk_idx, topk_w, logits,
                  d_topk_w, dz, dw_router, d_bias, dx, accumulate_dx, ws, ws_bytes, stream=None):
    return _check("moe_route_bwd", lib().moe_route_bwd(
        _ptr(x), _ptr(w_router), dtype, T, d, E, k, inv_tau, gate, _ptr(topk_idx), _ptr(topk_w),
        _ptr(logits), _ptr(d_topk_w), _ptr(dz), _ptr(dw_router), _ptr(d_bias), _ptr(dx),
        accumulate_dx, _ptr(ws), ws_bytes, _stream(stream)))


def moe_dispatch_workspace_size(T, k, E_r) -> int:
    return lib().moe_dispatch_workspace_size(T, k, E_r)


def moe_dispatch(x, dtype, T, d, k, E_r, topk_local, counts, offsets, perm, inv_perm, xp, ws,
                 ws_bytes, stream=None):
    return _check("moe_dispatch", lib().moe_dispatch(
        _ptr(x), dtype, T, d, k, E_r, _ptr(topk_local), _ptr(counts), _ptr(offsets), _ptr(perm),
        _ptr(inv_perm), _ptr(xp), _ptr(ws), ws_bytes, _stream(stream)))


def moe_dispatch_noalloc(x, dtype, T, d, k, E_r, topk_local, counts, offsets, perm, inv_perm, xp,
                         stream=None):
    return _check("moe_dispatch_noalloc", lib().moe_dispatch_noalloc(
        _ptr(x), dtype, T, d, k, E_r, _ptr(topk_local), _ptr(counts), _ptr(offsets), _ptr(perm),
        _ptr(inv_perm), _ptr(xp), _stream(stream)))


def moe_dispatch_bwd(dxp, dtype, T, d, k, cap, inv_perm, dx, accumulate, stream=None):
    return _check("moe_dispatch_bwd", lib().moe_dispatch_bwd(
        _ptr(dxp), dtype, T, d, k, cap, _ptr(inv_perm), _ptr(dx), accumulate, _stream(stream)))


def moe_grouped_ffn_fwd(xp, w_gate_up, w_down, dtype, cap, d, H, n_groups, offsets, gu, h, yp,
                        stream=None):
    return _check("moe_grouped_ffn_fwd", lib().moe_grouped_ffn_fwd(
        _ptr(xp), _ptr(w_gate_up), _ptr(w_down), dtype, cap, d, H, n_groups, _ptr(offsets),
        _ptr(gu), _ptr(h), _ptr(yp), _stream(stream)))


def moe_grouped_ffn_bwd(dyp, xp, gu, h, w_gate_up, w_down, dtype, cap, d, H, n_groups, offsets,
                        dgu, dxp, dw_gate_up, dw_down, accumulate_dw, stream=None):
    return _check("moe_grouped_ffn_bwd", lib().moe_grouped_ffn_bwd(
        _ptr(dyp), _ptr(xp), _ptr(gu), _ptr(h), _ptr(w_gate_up), _ptr(w_down), dtype, cap, d, H,
        n_groups, _ptr(offsets), _ptr(dgu), _ptr(dxp), _ptr(dw_gate_up), _ptr(dw_down),
        accumulate_dw, _stream(stream)))


def moe_grouped_ffn_fwd_workspace_size(sets, dtype, d):
    arr = (moe_ffn_set * len(sets))(*sets)
    return lib().moe_grouped_ffn_fwd_workspace_size(C.cast(arr, C.c_void_p), len(sets), dtype, d)


def moe_grouped_ffn_fwd_sets(sets, dtype, d, ws=None, ws_bytes=0, stream=None):
    arr = (moe_ffn_set * len(sets))(*sets)
    return _check("moe_grouped_ffn_fwd_sets", lib().moe_grouped_ffn_fwd_sets(
        C.cast(arr, C.c_void_p), len(sets), dtype, d, _ptr(ws), ws_bytes, _stream(stream)))


def moe_grouped_ffn_bwd_workspace_size(sets, dtype, d):
    arr = (moe_ffn_set * len(sets))(*sets)
    return lib().moe_grouped_ffn_bwd_workspace_size(C.cast(arr, C.c_void_p), len(sets), dtype, d)


def moe_grouped_ffn_bwd_sets(sets, dtype, d, accumulate_dw, ws=None, ws_bytes=0, stream=None):
    arr = (moe_ffn_set * len(sets))(*sets)
    return _check("moe_grouped_ffn_bwd_sets", lib().moe_grouped_ffn_bwd_sets(
        C.cast(arr, C.c_void_p), len(sets), dtype, d, accumulate_dw, _ptr(ws), ws_bytes,
        _stream(stream)))


def moe_combine_fwd(yp, dtype, T, d, k, cap, topk_w, inv_perm, y_add, y, stream=None):
    return _check("moe_combine_fwd", lib().moe_combine_fwd(
        _ptr(yp), dtype, T, d, k, cap, _ptr(topk_w), _ptr(inv_perm), _ptr(y_add), _ptr(y),
        _stream(stream)))


def moe_combine_bwd(dy, yp, dtype, T, d, k, cap, topk_w, inv_perm, dyp, d_topk_w, stream=None):
    return _check("moe_combine_bwd", lib().moe_combine_bwd(
        _ptr(dy), _ptr(yp), dtype, T, d, k, cap, _ptr(topk_w), _ptr(inv_perm), _ptr(dyp),
        _ptr(d_topk_w), _stream(stream)))


def moe_expert_delta(theta_start, theta_now, peers, n_peers, n_params, delta_local, delta_avg,
                     stream=None):
    arr = (C.c_void_p * max(1, n_peers))(*[_ptr(p) for p in (peers or [])][:n_peers]) \
        if n_peers else None
    return _check("moe_expert_delta", lib().moe_expert_delta(
        _ptr(theta_start), _ptr(theta_now), arr, n_peers, n_params, _ptr(delta_local),
        _ptr(delta_avg), _stream(stream)))


def moe_adamw_step(theta, grad, m, v, n, step, lr, beta1=0.9, beta2=0.95, eps=1e-8,
                   weight_decay=0.0, theta_bf16=None, stream=None):
    return _check("moe_adamw_step", lib().moe_adamw_step(
        _ptr(theta), _ptr(grad), _ptr(m), _ptr(v), n, step, lr, beta1, beta2, eps, weight_decay,
        _ptr(theta_bf16), _stream(stream)))


def moe_outer_nesterov(theta_start, theta_now, delta_avg, momentum, n, lr=0.7, mu=0.9,
                       theta_bf16=None, stream=None):
    return _check("moe_outer_nesterov", lib().moe_outer_nesterov(
        _ptr(theta_start), _ptr(theta_now), _ptr(delta_avg), _ptr(momentum), n, lr, mu,
        _ptr(theta_bf16), _stream(stream)))


def moe_replica_mean(local, peers, n_peers, n, out, stream=None):
    arr = (C.c_void_p * max(1, n_peers))(*[_ptr(p) for p in (peers or [])][:n_peers]) \
        if n_peers else None
    return _check("moe_replica_mean", lib().moe_replica_mean(
        _ptr(local), arr, n_peers, n, _ptr(out), _stream(stream)))


def _host_i32(a):
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(a), dtype=np.int32)
    return arr, arr.ctypes.data_as(C.c_void_p)


def moe_gen_placement(N_e, O_e, M, expert_perm=None, worker_perm=None):
    """[M, N_le] numpy int32 array of each worker's sorted expert ids."""
    import numpy as np
    N_le = N_e * O_e // M if M else 0
    out = np.zeros((max(M, 1), max(N_le, 1)), np.int32)
    ep = _host_i32(expert_perm) if expert_perm is not None else (None, None)
    wp = _host_i32(worker_perm) if worker_perm is not None else (None, None)
    _check("moe_gen_placement", lib().moe_gen_placement(
        N_e, O_e, M, ep[1], wp[1], out.ctypes.data_as(C.c_void_p)))
    return out[:M, :N_le]


def moe_migration_map(prev_set, new_set):
    import numpy as np
    prev, pp = _host_i32(prev_set)
    new, npp = _host_i32(new_set)
    out = np.zeros(max(len(new), 1), np.int32)
    _check("moe_migration_map", lib().moe_migration_map(
        pp, len(prev), npp, len(new), out.ctypes.data_as(C.c_void_p)))
    return out[:len(new)]


def moe_warmup_lr(steps, lr, warmup_steps):
    """fp32 learning rate per expert row from its steps since its state (re)started."""
    import numpy as np
    st, sp = _host_i32(steps)
    out = np.zeros(max(len(st), 1), np.float32)
    _check("moe_warmup_lr", lib().moe_warmup_lr(sp, len(st), float(lr), int(warmup_steps),
                                                out.ctypes.data_as(C.c_void_p)))
    return out[:len(st)]


def moe_copy_expert_rows(src, src_row, dst, n_rows, row_len, dst_row=None, dst_bf16=None,
                         stream=None):
    rows, rp = _host_i32(src_row)
    drows, dp = _host_i32(dst_row) if dst_row is not None else (None, None)
    return _check("moe_copy_expert_rows", lib().moe_copy_expert_rows(
        _ptr(src), rp, _ptr(dst), dp, n_rows, row_len, _ptr(dst_bf16), _stream(stream)))


def moe_adamw_step_rows(theta, grad, m, v, n_rows, row_len, steps, lr, beta1=0.9, beta2=0.95,
                        eps=1e-8, weight_decay=0.0, theta_bf16=None, stream=None):
    import numpy as np
    st, sp = _host_i32(steps)
    lr_arr = np.ascontiguousarray(np.asarray(lr, np.float32))
    return _check("moe_adamw_step_rows", lib().moe_adamw_step_rows(
        _ptr(theta), _ptr(grad), _ptr(m), _ptr(v), n_rows, row_len, sp,
        lr_arr.ctypes.data_as(C.c_void_p), beta1, beta2, eps, weight_decay, _ptr(theta_bf16),
        _stream(stream)))


def moe_timing_enable(capacity):
    return _check("moe_timing_enable", lib().moe_timing_enable(capacity))


def moe_timing_collect(max_out=64):
    """{kernel name: (launches, total_ms, min_ms, max_ms)} of the recorded launches."""
    arr = (moe_kernel_time * max_out)()
    n = C.c_int(0)
    _check("moe_timing_collect", lib().moe_timing_collect(C.cast(arr, C.c_void_p), max_out,
                                                          C.byref(n)))
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms, arr[i].min_ms, arr[i].max_ms)
            for i in range(n.value)}
