"""The register-only MFMA loop behind bench.py's measured matrix-core rate does the arithmetic
its flop count claims: the sum of one wave's outputs is fixed by the inputs the kernel forms
(bf16 of 0.5 + 1e-3 * thread + i and of 0.5 - i for k-slot i) whatever the MFMA's lane layout."""
import numpy as np
import pytest
import torch

from paper_2609_16450_amd import eb_probe_mfma_bf16

pytestmark = pytest.mark.gpu


def _bf16(x):
    return torch.tensor(x, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()


def expected_wave_sums(iters):
    """Per wave w of a workgroup: 8 chains x iters x sum over the 32x32 tile of A @ B, where
    A[m][k] comes from lane m + 32 (k // 8), slot k % 8, and B[k][n] = bf16(0.5 - k % 8)."""
    b = _bf16([0.5 - i for i in range(8)])
    out = []
    for w in range(4):
        total = 0.0
        for m in range(32):
            for kb in range(2):
                t = 64 * w + m + 32 * kb
                a = _bf16([np.float32(0.5) + np.float32(1e-3) * np.float32(t) + np.float32(i)
                           for i in range(8)])
                total += float(a @ b)
        out.append(8 * iters * 32 * total)
    return np.array(out)


@pytest.mark.parametrize("groups,iters", [(1, 1), (3, 7), (300, 64)])
def test_mfma_probe_flops_are_real(groups, iters):
    out = torch.full((groups * 256,), float("nan"), dtype=torch.float32, device="cuda:0")
    flops = eb_probe_mfma_bf16(out, groups, iters)
    torch.cuda.synchronize()
    assert flops == groups * iters * 8 * 4 * 2 * 32 * 32 * 16
    got = out.cpu().double().numpy().reshape(groups, 4, 64).sum(axis=2)
    want = expected_wave_sums(iters)
    np.testing.assert_allclose(got, np.broadcast_to(want, got.shape), rtol=1e-5)
