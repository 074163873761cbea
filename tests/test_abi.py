"""The C ABI on the CPU: the library loads, exports what include/*.h declares,
and rejects invalid arguments on the host without launching anything."""
import ctypes as C
import glob
import os
import re

import pytest

from paper_2606_19025_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

ERR_ARG, ERR_UNSUPPORTED = -1, -2


def declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(moe_\w+)\s*\(", src))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    return B.lib()


def test_library_exports_every_declared_symbol(lib):
    decl = declared_functions()
    assert len(decl) >= 13
    for name in decl:
        assert hasattr(lib, name), name
    assert set(decl) == set(B.EXPORTS)


def test_abi_version(lib):
    assert B.moe_abi_version() == 3


def test_workspace_sizes_are_host_only(lib):
    assert B.moe_dispatch_workspace_size(8192, 6, 16) >= 2 * 32 * 16 * 4
    assert B.moe_route_bwd_workspace_size(8192, 2048, 64) >= 16 * 64 * 2048 * 4
    assert B.moe_dispatch_workspace_size(-1, 2, 4) == 0


def _gpu_visible():
    # device_count() does not initialise the GPU runtime
    import torch
    return torch.cuda.device_count() > 0


def call_status(fn, *args):
    """Call the raw C entry point with stream 0 and return its status.

    The rejection tests pass fake device addresses that must never reach a
    kernel: where a GPU is visible they are skipped, so that an argument check
    that wrongly passed could not launch on those addresses."""
    if _gpu_visible():
        pytest.skip("host-only rejection test: runs where no GPU is visible")
    return fn(*args, None)


def test_route_mask_rejects_bad_arguments(lib):
    f = lib.moe_route_mask
    p = 256  # a fake, never dereferenced, 16-byte aligned address
    base = [p, p, None, B.MOE_BF16, 16, 64, 8, 2, 1.0, 0, p, None, p, p, p]
    assert call_status(f, *base[:3], 7, *base[4:]) == ERR_UNSUPPORTED       # dtype
    bad_k = list(base); bad_k[7] = 9
    assert call_status(f, *bad_k) == ERR_ARG                                # k > E
    bad_e = list(base); bad_e[6] = 257; bad_e[7] = 2
    assert call_status(f, *bad_e) == ERR_ARG                                # E > 256
    null_w = list(base); null_w[1] = None
    assert call_status(f, *null_w) == ERR_ARG
    bad_tau = list(base); bad_tau[8] = float("nan")
    assert call_status(f, *bad_tau) == ERR_ARG
    bad_gate = list(base); bad_gate[9] = 5
    assert call_status(f, *bad_gate) == ERR_ARG
    bad_d = list(base); bad_d[5] = 60
    assert call_status(f, *bad_d) == ERR_UNSUPPORTED                        # bf16 needs d % 8
    misaligned = list(base); misaligned[0] = p + 2
    assert call_status(f, *misaligned) == ERR_UNSUPPORTED
    assert "aligned" in B.moe_last_error()


def test_dispatch_rejects_small_workspace_and_bad_er(lib):
    f = lib.moe_dispatch
    p = 256
    ws = B.moe_dispatch_workspace_size(100, 2, 4)
    args = [p, B.MOE_BF16, 100, 64, 2, 4, p, p, p, p, p, p, p, ws - 1]
    assert call_status(f, *args) == ERR_ARG
    assert "workspace" in B.moe_last_error()
    args[5] = 300
    args[13] = ws
    assert call_status(f, *args) == ERR_ARG


def test_grouped_ffn_rejects_unsupported_shapes(lib):
    f = lib.moe_grouped_ffn_fwd
    p = 256
    assert call_status(f, p, p, p, B.MOE_BF16, 64, 96, 128, 2, p, p, p, p) == ERR_UNSUPPORTED  # d % 64
    assert call_status(f, p, p, p, B.MOE_BF16, 64, 128, 100, 2, p, p, p, p) == ERR_UNSUPPORTED  # H % 64
    assert call_status(f, p, p, p, B.MOE_BF16, 64, 128, 128, 2, None, p, p, p) == ERR_ARG  # offsets
    g = lib.moe_grouped_ffn_bwd
    assert call_status(g, p, p, p, p, p, p, B.MOE_BF16, 64, 128, 128, -1, p, p, p, p, p, 0) == ERR_ARG
    # bf16 operands of 4 GiB or more (32-bit DMA offsets): rows (cap x 2H)
    # and weights (groups x 2H x d)
    assert call_status(f, p, p, p, B.MOE_BF16, 1 << 20, 2048, 1024, 1, p, p, p, p) == ERR_UNSUPPORTED
    assert call_status(f, p, p, p, B.MOE_BF16, 64, 4096, 4096, 64, p, p, p, p) == ERR_UNSUPPORTED
    assert call_status(g, p, p, p, p, p, p, B.MOE_BF16, 1 << 20, 2048, 1024, 1, p, p, p, p, p,
                       0) == ERR_UNSUPPORTED


def test_combine_and_unpermute_reject_bad_arguments(lib):
    p = 256
    assert call_status(lib.moe_combine_fwd, p, B.MOE_BF16, 10, 12, 2, 20, p, p, None, p) == ERR_UNSUPPORTED
    assert call_status(lib.moe_combine_bwd, p, p, B.MOE_F32, 10, 64, 0, 20, p, p, p, p) == ERR_ARG
    assert call_status(lib.moe_combine_fwd, p, B.MOE_BF16, 10, 64, 2, -1, p, p, None, p) == ERR_ARG
    assert call_status(lib.moe_dispatch_bwd, p, B.MOE_F32, 10, 64, 2, 20, None, p, 0) == ERR_ARG


def test_route_bwd_requires_logits_for_raw_softmax(lib):
    p = 256
    ws = B.moe_route_bwd_workspace_size(10, 64, 8)
    st = call_status(lib.moe_route_bwd, p, p, B.MOE_BF16, 10, 64, 8, 2, 1.0, B.MOE_GATE_SOFTMAX,
                     p, p, None, p, p, p, None, p, 1, p, ws)
    assert st == ERR_ARG and "logits" in B.moe_last_error()


def test_expert_delta_rejects_too_many_peers(lib):
    p = 256
    arr = (C.c_void_p * 17)(*([p] * 17))
    assert call_status(lib.moe_expert_delta, p, p, arr, 17, 1024, None, p) == ERR_ARG
    arr2 = (C.c_void_p * 1)(p + 4)
    assert call_status(lib.moe_expert_delta, p, p, arr2, 1, 1024, None, p) == ERR_UNSUPPORTED


def test_ffn_sets_reject_bad_arguments(lib):
    p = 256
    ok = B.ffn_set(p, p, p, p, 64, 128, 2, p, p, yp=p)
    assert B.lib().moe_grouped_ffn_fwd_sets(None, 1, B.MOE_BF16, 128, None, 0, None) == ERR_ARG
    arr = (B.moe_ffn_set * 3)(ok, ok, ok)
    assert B.lib().moe_grouped_ffn_fwd_sets(C.cast(arr, C.c_void_p), 3, B.MOE_BF16, 128, None, 0,
                                            None) == ERR_ARG
    bad_h = B.ffn_set(p, p, p, p, 64, 100, 2, p, p, yp=p)
    arr = (B.moe_ffn_set * 2)(ok, bad_h)
    assert B.lib().moe_grouped_ffn_fwd_sets(C.cast(arr, C.c_void_p), 2, B.MOE_BF16, 128, None, 0,
                                            None) == ERR_UNSUPPORTED
    no_grad = B.ffn_set(p, p, p, p, 64, 128, 2, p, p, dyp=p, dgu=p, dxp=p)  # dW pointers NULL
    arr = (B.moe_ffn_set * 1)(no_grad)
    assert B.lib().moe_grouped_ffn_bwd_sets(C.cast(arr, C.c_void_p), 1, B.MOE_BF16, 128, 0,
                                            None, 0, None) == ERR_ARG
    assert "gradients" in B.moe_last_error()
    good = B.ffn_set(p, p, p, p, 8192, 1408, 1, p, p, dyp=p, dgu=p, dxp=p, dw_gate_up=p,
                     dw_down=p)
    need = B.moe_grouped_ffn_bwd_workspace_size([good], B.MOE_BF16, 2048)
    assert need >= 64  # the tile counters at least
    arr = (B.moe_ffn_set * 1)(good)
    assert B.lib().moe_grouped_ffn_bwd_sets(C.cast(arr, C.c_void_p), 1, B.MOE_BF16, 2048, 0,
                                            4096, need - 1, None) == ERR_ARG
    assert "workspace" in B.moe_last_error()
    assert B.lib().moe_grouped_ffn_bwd_sets(C.cast(arr, C.c_void_p), 1, B.MOE_BF16, 2048, 0,
                                            4096 + 16, need, None) == ERR_UNSUPPORTED


def test_optimiser_entry_points_reject_bad_arguments(lib):
    p = 256
    # AdamW: NULL arrays, step 0, betas out of range, misalignment
    assert call_status(lib.moe_adamw_step, None, p, p, p, 10, 1, 0.01, 0.9, 0.95, 1e-8, 0.0,
                       None) == ERR_ARG
    assert call_status(lib.moe_adamw_step, p, p, p, p, 10, 0, 0.01, 0.9, 0.95, 1e-8, 0.0,
                       None) == ERR_ARG
    assert call_status(lib.moe_adamw_step, p, p, p, p, 10, 1, 0.01, 1.0, 0.95, 1e-8, 0.0,
                       None) == ERR_ARG
    assert call_status(lib.moe_adamw_step, p, p, p, p + 4, 10, 1, 0.01, 0.9, 0.95, 1e-8, 0.0,
                       None) == ERR_UNSUPPORTED
    # outer step: NULL momentum, misaligned bf16 copy
    assert call_status(lib.moe_outer_nesterov, p, p, p, None, 10, 0.7, 0.9, None) == ERR_ARG
    assert call_status(lib.moe_outer_nesterov, p, p, p, p, 10, 0.7, 0.9, p + 2) == ERR_UNSUPPORTED
    # replica mean: too many peers, NULL peer
    arr = (C.c_void_p * 17)(*([p] * 17))
    assert call_status(lib.moe_replica_mean, p, arr, 17, 10, p) == ERR_ARG
    arr1 = (C.c_void_p * 1)(None)
    assert call_status(lib.moe_replica_mean, p, arr1, 1, 10, p) == ERR_ARG


def test_ffn_forward_workspace_holds_the_down_projection_parts(lib):
    """The forward workspace reserves up to 8 fp32 partials of [cap, d] per
    set within 256 MiB (none when two do not fit, or in fp32), and a call with
    a smaller workspace is rejected on the host."""
    p = 256
    d = 1024
    small = B.ffn_set(p, p, p, p, 8192, 2816, 8, p, p, yp=p)     # 32 MiB per part: 8 parts
    big = B.ffn_set(p, p, p, p, 49152, 1408, 16, p, p, yp=p)     # 192 MiB per part: none
    one = B.moe_grouped_ffn_fwd_workspace_size([small], B.MOE_BF16, d)
    assert one >= 8 * 8192 * d * 4
    assert B.moe_grouped_ffn_fwd_workspace_size([big], B.MOE_BF16, d) == 0
    assert B.moe_grouped_ffn_fwd_workspace_size([small], B.MOE_F32, d) == 0
    assert B.moe_grouped_ffn_fwd_workspace_size([small, big], B.MOE_BF16, d) == one
    arr = (B.moe_ffn_set * 1)(small)
    assert call_status(lib.moe_grouped_ffn_fwd_sets, C.cast(arr, C.c_void_p), 1, B.MOE_BF16, d,
                       p * 1024, one - 256) == ERR_ARG
    assert "workspace" in B.moe_last_error()
    # the backward's workspace holds dX's parts besides its counters
    bwd = B.ffn_set(p, p, p, p, 8192, 2816, 8, p, p, dyp=p, dgu=p, dxp=p, dw_gate_up=p, dw_down=p)
    assert B.moe_grouped_ffn_bwd_workspace_size([bwd], B.MOE_BF16, d) >= one
