"""The device probes through the C ABI. Matrix-core probe: with small-integer
operands every product and sum is exact in fp32, so each thread's sink value
must equal, bit for bit, the same sum taken in numpy from the operand layout
of a 32x32x16 matrix multiply-accumulate (A element (m, k) in lane m + 32 (k/8),
B element (k, n) in lane n + 32 (k/8), accumulator r of lane l = element
(8 (r/4) + 4 (l/32) + r%4, l%32)); all-ones operands give the closed form
8192 per round. HBM read probe: the XOR of its sink equals the XOR of every
32-bit word of the buffer (numpy over the same bytes), on sizes with ragged
tails."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

rf = pytest.importorskip("paper_2606_06309_amd.binding")


def _lane_sums(ops, rounds):
    """ops: float array [12][64][8]; the probe's per-lane sink value."""
    A = np.zeros((6, 32, 16))
    B = np.zeros((6, 16, 32))
    for k in range(16):
        A[:, :, k] = ops[:6, 32 * (k // 8):32 * (k // 8) + 32, k % 8]
        B[:, k, :] = ops[6:, 32 * (k // 8):32 * (k // 8) + 32, k % 8]
    sums = np.zeros(64)
    for j in range(4):
        C = rounds * sum(A[(u + 2 * j) % 6] @ B[(3 * u + j) % 6] for u in range(8))
        for lane in range(64):
            for r in range(16):
                sums[lane] += C[8 * (r // 4) + 4 * (lane // 32) + r % 4, lane % 32]
    return sums


@pytest.mark.parametrize("wg,rounds,seed", [(1, 1, 0), (3, 2, 1), (5, 7, 2), (2, 40, 3)])
def test_mfma_probe_integer_operands(wg, rounds, seed):
    print(f"[case] mfma probe wg={wg} rounds={rounds} seed={seed}", flush=True)
    g = torch.Generator(device="cpu").manual_seed(seed)
    ops = torch.randint(-3, 4, (12, 64, 8), generator=g).to(torch.bfloat16)
    sink = rf.rf_probe_mfma_bf16(ops.cuda(), wg, rounds)
    torch.cuda.synchronize()
    want = np.tile(_lane_sums(ops.float().numpy().astype(np.float64), rounds), wg * 4)
    assert np.abs(want).max() < 2 ** 24
    got = sink.cpu().numpy().astype(np.float64)
    assert np.array_equal(got, want), np.abs(got - want).max()


def test_mfma_probe_all_ones():
    ops = torch.ones((12, 64, 8), dtype=torch.bfloat16, device="cuda")
    sink = rf.rf_probe_mfma_bf16(ops, 4, 100)
    torch.cuda.synchronize()
    assert bool((sink == 8192.0 * 100).all())


def test_mfma_probe_random_operands_close():
    """Random normal operands (the benchmark's): the sink matches the numpy
    sum to fp32 accumulation accuracy."""
    g = torch.Generator(device="cpu").manual_seed(7)
    ops = torch.randn((12, 64, 8), generator=g).to(torch.bfloat16)
    sink = rf.rf_probe_mfma_bf16(ops.cuda(), 2, 3)
    torch.cuda.synchronize()
    want = np.tile(_lane_sums(ops.float().numpy().astype(np.float64), 3), 8)
    got = sink.cpu().numpy().astype(np.float64)
    assert np.allclose(got, want, rtol=1e-4, atol=1e-2)


@pytest.mark.parametrize("nbytes,wg", [(16, 1), (48, 3), (4096 * 16 + 48, 7), ((8 << 20) + 16 * 5, 64),
                                       (64 << 20, 1024)])
def test_hbm_read_probe_xor(nbytes, wg):
    print(f"[case] hbm read probe bytes={nbytes} wg={wg}", flush=True)
    g = torch.Generator(device="cpu").manual_seed(nbytes)
    host = torch.randint(-2 ** 31, 2 ** 31, (nbytes // 4,), dtype=torch.int64, generator=g).to(torch.int32)
    src = host.cuda()
    sink = rf.rf_probe_hbm_read(src, wg)
    torch.cuda.synchronize()
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    want = np.bitwise_xor.reduce(host.numpy().view(np.uint32))
    assert got == want
