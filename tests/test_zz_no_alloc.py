"""moe_dispatch_noalloc (the dispatch with its workspace in a library-owned
device array, for callers that cannot allocate) against moe_dispatch with a
caller workspace: bit-exact counts, offsets, perm, inv_perm and gathered rows,
on two calls in a row, the second with a smaller input."""
import numpy as np
import pytest

from paper_2606_19025_amd import binding as B

pytestmark = pytest.mark.gpu


def routes(T, k, E_r, seed):
    """Seeded local expert ids [T, k]: distinct per token, about a third ghosts (-1)."""
    g = np.random.default_rng([seed, T, k, E_r])
    E = max(E_r * 3 // 2, k)
    ids = np.argsort(g.random((T, E)), axis=1)[:, :k]
    return np.where(ids < E_r, ids, -1).astype(np.int32)


def run_both(T, d, k, E_r, seed, dtype):
    import torch
    tdt = torch.bfloat16 if dtype == B.MOE_BF16 else torch.float32
    dev = torch.device("cuda")
    g = torch.Generator().manual_seed(seed)
    x = torch.randn(T, d, generator=g).to(tdt).to(dev)
    local = torch.from_numpy(routes(T, k, E_r, seed)).to(dev)
    cap = T * min(k, E_r)
    outs = []
    for noalloc in (False, True):
        counts = torch.full((max(E_r, 1),), -7, dtype=torch.int32, device=dev)
        offsets = torch.full((E_r + 1,), -7, dtype=torch.int32, device=dev)
        perm = torch.full((max(cap, 1),), -7, dtype=torch.int32, device=dev)
        inv = torch.full((T, k), -7, dtype=torch.int32, device=dev)
        xp = torch.full((max(cap, 1), d), float("nan"), dtype=tdt, device=dev)
        if noalloc:
            B.moe_dispatch_noalloc(x, dtype, T, d, k, E_r, local, counts, offsets, perm, inv, xp)
        else:
            ws_bytes = B.moe_dispatch_workspace_size(T, k, E_r)
            ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
            B.moe_dispatch(x, dtype, T, d, k, E_r, local, counts, offsets, perm, inv, xp, ws,
                           ws_bytes)
        torch.cuda.synchronize()
        n = int(offsets[-1].item())
        outs.append(dict(counts=counts[:E_r].cpu(), offsets=offsets.cpu(), perm=perm[:n].cpu(),
                         inv=inv.cpu(), xp=xp[:n].view(torch.int16 if tdt == torch.bfloat16
                                                        else torch.int32).cpu(), n=n))
    return outs


@pytest.mark.parametrize("dtype", [B.MOE_BF16, B.MOE_F32])
def test_noalloc_dispatch_matches_workspace_dispatch(gpu_lib, dtype):
    # the second call is smaller, so stale contents of the library's array
    # from the first call must not leak into its result
    for T, d, k, E_r, seed in ((8192, 2048, 6, 16, 1), (1000, 256, 2, 5, 2)):
        print(f"[noalloc] T={T} d={d} k={k} E_r={E_r} dtype={dtype}", flush=True)
        ref, got = run_both(T, d, k, E_r, seed, dtype)
        assert ref["n"] == got["n"] > 0
        for key in ("counts", "offsets", "perm", "inv", "xp"):
            assert np.array_equal(ref[key].numpy(), got[key].numpy()), (T, key)


def test_noalloc_dispatch_rejects_sizes_beyond_its_array(gpu_lib):
    import torch
    T, d, k, E_r = 130816 + 256, 64, 8, 256
    assert B.moe_dispatch_workspace_size(T, k, E_r) > (1 << 20)
    t = torch.empty(16, dtype=torch.int32, device="cuda")
    with pytest.raises(B.MoeError) as e:
        # rejected on the host before any launch (sizes are checked first)
        B.moe_dispatch_noalloc(t, B.MOE_BF16, T, d, k, E_r, t, t, t, t, t, t)
    assert e.value.status == -2 and "workspace" in str(e.value)
    # the largest accepted size for E_r = 256
    assert B.moe_dispatch_workspace_size(130816, k, E_r) <= (1 << 20)
