"""The measurement probes (promoe_peak_hbm_read, promoe_peak_mfma_bf16) through
the C ABI: the MFMA loop's output against its closed form, the read probe's
XOR fold of a uniform buffer, and the size checks."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2410_22134_amd import _abi  # noqa: E402
from paper_2410_22134_amd._abi import PromoeError  # noqa: E402


def _bf16(x):
    """fp32 -> bf16 (round to nearest even) -> fp32, for finite values."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def test_mfma_probe_closed_form():
    blocks, iters = 2, 3
    sink = torch.full((blocks * 512,), -1.0, dtype=torch.float32, device="cuda")
    _abi.peak_mfma_bf16(sink, blocks, iters)
    torch.cuda.synchronize()
    # lane l holds a[j] = bf16((l % 64) / 1024 + j), b[j] = bf16(j / 2); in a
    # 16x16x32 MFMA, A[m][k] comes from lane m + 16 (k // 8), element k % 8, and
    # B[n][k] from lane n + 16 (k // 8) -- b does not depend on the lane.
    k = np.arange(32)
    A = np.array([[_bf16(np.float32((m + 16 * (kk // 8)) / 1024.0 + kk % 8)) for kk in k] for m in range(16)])
    B = np.array([_bf16(np.float32((kk % 8) * 0.5)) for kk in k])
    C = iters * (A @ B)  # [16], the same for every column n
    lanes = np.arange(512) % 64
    want = np.array([32 * sum(C[4 * (l // 16) + r] for r in range(4)) for l in lanes])
    got = sink.cpu().numpy().reshape(blocks, 512)
    for b in range(blocks):
        np.testing.assert_allclose(got[b], want, rtol=1e-5)  # fp32 fold of 128 terms


def test_hbm_read_probe_uniform_buffer():
    n = 1 << 20
    buf = torch.ones(n, dtype=torch.uint8, device="cuda")
    sink = torch.full((64,), -1.0, dtype=torch.float32, device="cuda")
    _abi.peak_hbm_read(buf, n, sink, 64)
    torch.cuda.synchronize()
    # every thread folds an even number of identical 32-bit words
    assert torch.all(sink == 0.0)


def test_probe_argument_checks():
    buf = torch.ones(64, dtype=torch.uint8, device="cuda")
    sink = torch.empty(512, dtype=torch.float32, device="cuda")
    for args in ((buf, 60, sink, 1), (buf, 0, sink, 1), (buf, 64, sink, 0)):
        with pytest.raises(PromoeError):
            _abi.peak_hbm_read(*args)
    with pytest.raises(PromoeError):
        _abi.peak_mfma_bf16(sink, 1, 0)
