"""GPU checks of the measurement probes (through the C ABI): the read probe
folds exactly the words each thread streamed (bit-exact against a host XOR
over the same grid-stride assignment), and the MFMA probe's sums equal the
closed form of its products (its pseudo-random bf16 operands regenerated on
the host; the 32x32 C layout puts row 8(v/4) + 4(l/32) + v%4, column l%32 in
element v of lane l)."""
import numpy as np
import pytest
import torch

import paper_2609_38767_amd as dt

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("n16,wgs", [(4096, 4), (4096 * 7 + 13, 3), (5, 2)])
def test_read_probe_folds_every_word(n16, wgs):
    print(f"[probe] read n16={n16} workgroups={wgs}", flush=True)
    g = torch.Generator(device="cpu").manual_seed(n16)
    words = torch.randint(-(1 << 31), (1 << 31) - 1, (n16 * 4,), generator=g, dtype=torch.int64).to(torch.int32)
    buf = words.to(DEV)
    sink = torch.zeros(wgs * 256, dtype=torch.int32, device=DEV)
    dt.dattri_probe_read(buf, n16 * 16, sink, wgs)
    torch.cuda.synchronize()
    w = words.numpy().reshape(n16, 4)
    per16 = w[:, 0] ^ w[:, 1] ^ w[:, 2] ^ w[:, 3]
    step = wgs * 256
    want = np.zeros(step, dtype=np.int32)
    for t in range(step):
        want[t] = np.bitwise_xor.reduce(per16[t::step]) if t < n16 else 0
    assert np.array_equal(sink.cpu().numpy(), want)


def _operand(lane, e, c, side):
    """bf16 value of the probe's operand hash (sign, exponent -2..1, 7-bit mantissa)."""
    M = 0xFFFFFFFF
    h = (lane * 0x9E3779B1 + e * 0x85EBCA77 + c * 0xC2B2AE3D + side * 0x27D4EB2F + 0x165667B1) & M
    h ^= h >> 15
    h = (h * 0x2C1B3C6D) & M
    h ^= h >> 12
    sign, expo, mant = (h >> 31) & 1, 125 + ((h >> 8) & 3), h & 0x7F
    return (-1.0) ** sign * 2.0 ** (expo - 127) * (1 + mant / 128.0)


def test_mfma_probe_closed_form():
    wgs, iters = 3, 4
    sink = torch.zeros(wgs * 256, dtype=torch.float32, device=DEV)
    flops = dt.dattri_probe_mfma(sink, wgs, iters)
    torch.cuda.synchronize()
    assert flops == wgs * 4 * iters * 8 * 2 * 32 * 32 * 16
    want, scale = np.zeros(64), np.zeros(64)
    for c in range(8):
        A = np.array([[_operand(m + 32 * (k // 8), k % 8, c, 0) for k in range(16)] for m in range(32)])
        B = np.array([[_operand(n + 32 * (k // 8), k % 8, c, 1) for n in range(32)] for k in range(16)])
        C = A @ B
        Cabs = np.abs(A) @ np.abs(B)
        for lane in range(64):
            rows = [8 * (v // 4) + 4 * (lane // 32) + v % 4 for v in range(16)]
            want[lane] += iters * sum(C[r, lane % 32] for r in rows)
            scale[lane] += iters * sum(Cabs[r, lane % 32] for r in rows)
    got = sink.cpu().numpy().reshape(-1, 64).astype(np.float64)
    assert np.all(np.abs(got - want[None, :]) <= 1e-5 * scale[None, :])
