"""The measurement probes against plain definitions (needs an MI355X).

The HBM read probe's checksum is the sum of the buffer's 32-bit words modulo
2^32; the MFMA probe's output is, per wave, the sum over its 8 chains of
iters x (A_j B_j^T) in the documented lane layout of the 32x32x16 bf16
operation.  Both are exact or near-exact definitions computed with numpy.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nbytes,wgs", [(16, 1), (1 << 20, 3), ((1 << 20) + 48, 2048)])
def test_hbm_read_probe_checksum(nbytes, wgs):
    import torch
    from paper_2608_02438_amd.xpress import probe_hbm_read
    print(f"case: read probe bytes={nbytes} workgroups={wgs}", flush=True)
    rng = np.random.default_rng(nbytes + wgs)
    words = rng.integers(0, 2**32, size=nbytes // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(words.view(np.int32)).cuda()
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    probe_hbm_read(buf, out, wgs)
    torch.cuda.synchronize()
    got = int(out.cpu().numpy().view(np.uint32)[0])
    assert got == int(words.astype(np.uint64).sum() % (1 << 32))


def _bf16_bits(x):
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def test_mfma_probe_matches_the_32x32x16_definition():
    import torch
    from paper_2608_02438_amd.xpress import probe_mfma_bf16
    print("case: mfma probe workgroups=2 iters=3", flush=True)
    rng = np.random.default_rng(7)
    bits = _bf16_bits(rng.standard_normal((8, 64, 2, 8)).astype(np.float32))
    vals = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    ops = torch.from_numpy(bits.view(np.int16)).cuda()
    wgs, iters = 2, 3
    out = torch.zeros(wgs * 4 * 64 * 16, dtype=torch.float32, device="cuda")
    probe_mfma_bf16(ops, wgs, iters, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(wgs * 4, 64, 16)
    # A_j[m][k]: lane l = m + 32 (k // 8) holds element k % 8; B_j[n][k] likewise
    D = np.zeros((32, 32))
    for j in range(8):
        A = np.zeros((32, 16))
        Bm = np.zeros((32, 16))
        for l in range(64):
            A[l % 32, 8 * (l // 32):8 * (l // 32) + 8] = vals[j, l, 0]
            Bm[l % 32, 8 * (l // 32):8 * (l // 32) + 8] = vals[j, l, 1]
        D += iters * (A @ Bm.T)
    want = np.zeros((64, 16))
    for l in range(64):
        for i in range(16):
            want[l, i] = D[8 * (i // 4) + 4 * (l // 32) + i % 4, l % 32]
    tol = 1e-5 * (np.abs(D).max() + 1.0)
    for w in range(wgs * 4):
        assert np.abs(got[w] - want).max() <= tol, w
