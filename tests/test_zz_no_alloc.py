"""The allocation-free permutation (moe_permute_noalloc) against the
workspace one (moe_permute), through the C ABI (needs an MI355X).

Both are called on the same routing; every output must be identical.  Two
calls in a row, the second on a smaller input, check that the static
scratch the first call left behind does not leak into the second; every
path that uses the scratch is covered (256- and 1024-pair chunks, the
combined scan-and-scatter launch for at most 64 local experts and the
separate scan above that), and the one-workgroup path, which uses none.
"""
import ctypes

import numpy as np
import pytest
import torch

import moe_inputs as mi
import paper_2606_26607_amd as moe

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    moe.lib()


def _outputs(T, k, El, H):
    cap = T * min(k, El)
    return dict(counts=torch.full((El,), -5, dtype=torch.int32, device="cuda"),
                offsets=torch.full((El + 1,), -5, dtype=torch.int32, device="cuda"),
                r2p=torch.full((max(cap, 1),), -5, dtype=torch.int32, device="cuda"),
                p2r=torch.full((max(T * k, 1),), -5, dtype=torch.int32, device="cuda"),
                xp=torch.zeros((max(cap, 1), H), dtype=torch.bfloat16, device="cuda"))


def _p(t):
    return ctypes.c_void_p(t.data_ptr())


def run_pair(T, E, k, e0, El, seed, H=64):
    ids = torch.from_numpy(mi.random_topk_ids(T, E, k, seed=seed)).cuda()
    x = torch.from_numpy(mi.random_bf16((T, H), seed=seed).view(np.int16)).view(torch.bfloat16).cuda()
    L = moe.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    ref, got = _outputs(T, k, El, H), _outputs(T, k, El, H)
    ws = torch.empty(max(moe.permute_workspace_size(T, k, El), 256), dtype=torch.uint8, device="cuda")
    st = L.moe_permute(_p(ids), T, k, E, e0, El, _p(ref["counts"]), _p(ref["offsets"]), _p(ref["r2p"]),
                       _p(ref["p2r"]), _p(x), H, _p(ref["xp"]), _p(ws), ws.numel(), stream)
    assert st == 0, L.moe_last_error()
    st = L.moe_permute_noalloc(_p(ids), T, k, E, e0, El, _p(got["counts"]), _p(got["offsets"]), _p(got["r2p"]),
                               _p(got["p2r"]), _p(x), H, _p(got["xp"]), stream)
    assert st == 0, L.moe_last_error()
    torch.cuda.synchronize()
    n = int(ref["offsets"][-1].item())
    for name in ("counts", "offsets"):
        assert torch.equal(got[name], ref[name]), name
    assert torch.equal(got["r2p"][:n], ref["r2p"][:n]), "row_to_pair"
    assert torch.equal(got["p2r"][:T * k], ref["p2r"][:T * k]), "pair_to_row"
    assert torch.equal(got["xp"][:n].view(torch.int16), ref["xp"][:n].view(torch.int16)), "x_perm"
    return n


@pytest.mark.parametrize("big,small", [
    # 256-pair chunks, scan and scatter in one launch (<= 64 local experts)
    ((8192, 128, 8, 0, 16), (3000, 128, 8, 16, 16)),
    # separate scan (more than 64 local experts)
    ((4096, 256, 8, 0, 256), (1500, 256, 8, 0, 128)),
    # 1024-pair chunks (pairs x local experts above 2^24), then 256-pair chunks
    ((65536, 64, 8, 0, 64), (9000, 64, 8, 0, 32)),
    # then the one-workgroup path (no scratch), then the chunked one again
    ((40000, 8, 2, 0, 8), (64, 8, 2, 0, 8)),
])
def test_noalloc_matches_workspace_path(big, small):
    n1 = run_pair(*big, seed=big[0])
    n2 = run_pair(*small, seed=small[0] + 1)
    assert n1 > 0 and n2 > 0
    # and the large input once more after the small one
    run_pair(*big, seed=big[0] + 2)
