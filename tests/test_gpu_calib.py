"""The matrix-core reference loop (moe_calib_mfma), a measurement aid the
bench uses for the device's sustained bf16 MFMA rate (needs an MI355X).

Its output is checked against numpy: each wave multiplies fixed hashed
operands iters times, so every thread's result is iters times a sum of
entries of 32x32x16 block products, which the test rebuilds from the same
hash, bf16 rounding and MFMA lane layout.
"""
import numpy as np
import pytest
import torch

import paper_2606_26607_amd as moe

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    moe.lib()


def mix32(x):
    x = x ^ (x >> np.uint32(16))
    x = x * np.uint32(0x7feb352d)
    x = x ^ (x >> np.uint32(15))
    x = x * np.uint32(0x846ca68b)
    return x ^ (x >> np.uint32(16))


def to_bf16(v):
    u = np.asarray(v, dtype=np.float32).view(np.uint32)
    u = (u + np.uint32(0x7fff) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xffff0000)
    return u.view(np.float32).astype(np.float64)


def expected(grid, iters):
    with np.errstate(over="ignore"):
        gid = np.arange(grid * 512, dtype=np.uint32)
        h = gid * np.uint32(0x9e3779b9) + np.uint32(1)
        vals = []
        for _ in range(6 * 8):
            h = mix32(h)
            vals.append(((h & np.uint32(0xffff)).astype(np.float64) - 32768.0) / 32768.0)
    vals = np.stack(vals, axis=1).astype(np.float32)  # [threads, 48]
    a = to_bf16(vals[:, :16]).reshape(-1, 2, 8)
    b = to_bf16(vals[:, 16:] * np.float32(0.02)).reshape(-1, 4, 8)
    out = np.zeros(grid * 512)
    waves = grid * 8
    a = a.reshape(waves, 64, 2, 8)
    b = b.reshape(waves, 64, 4, 8)
    lane = np.arange(64)
    for w in range(waves):
        for i in range(2):
            # operand matrices of the 32x32x16 MFMA: lane l holds row (l % 32),
            # k = 8 * (l // 32) + 0..7, of A and of B (B's row is an output column)
            A = np.zeros((32, 16))
            B = np.zeros((32, 16))
            for l in range(64):
                A[l % 32, 8 * (l // 32):8 * (l // 32) + 8] = a[w, l, i]
            for j in range(4):
                for l in range(64):
                    B[l % 32, 8 * (l // 32):8 * (l // 32) + 8] = b[w, l, j]
                P = A @ B.T  # [row, col]
                # lane l holds column l % 32, rows 8*(q//4) + 4*(l//32) + q%4
                for l in range(64):
                    rows = [8 * (q // 4) + 4 * (l // 32) + q % 4 for q in range(16)]
                    out[w * 64 + l] += iters * P[rows, l % 32].sum()
        del A, B
    return out


def test_calib_zero_operands_give_zero():
    out = torch.full((2 * 512,), 7.0, dtype=torch.float32, device="cuda")
    flops = moe.calib_mfma(out, 5, zero_operands=True)
    torch.cuda.synchronize()
    assert flops == 2 * 8 * 5 * 8 * 32768
    assert torch.count_nonzero(out).item() == 0


def test_calib_random_operands_match_numpy():
    grid, iters = 2, 3
    out = torch.zeros(grid * 512, dtype=torch.float32, device="cuda")
    moe.calib_mfma(out, iters)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = expected(grid, iters)
    scale = np.abs(ref).max()
    assert scale > 0
    assert np.abs(got - ref).max() <= 1e-5 * scale * 64, np.abs(got - ref).max() / scale


def test_calib_rejects():
    L = moe.lib()
    out = torch.zeros(512, dtype=torch.float32, device="cuda")
    assert L.moe_calib_mfma(0, 1, 0, out.data_ptr(), None) == 1
    assert L.moe_calib_mfma(1, 0, 0, out.data_ptr(), None) == 1
    assert L.moe_calib_mfma(1, 1, 0, None, None) == 1
