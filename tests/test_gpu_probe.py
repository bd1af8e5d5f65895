"""The device probes through the C ABI. Matrix-core probe: with small-integer
operands every product and sum is exact in fp32, so each thread's sink value
must equal, bit for bit, the same sum taken in numpy from the operand layout
of a 32x32x16 matrix multiply-accumulate (A element (m, k) in lane m + 32 (k/8),
B element (k, n) in lane n + 32 (k/8), accumulator r of lane l = element
(8 (r/4) + 4 (l/32) + r%4, l%32)); all-ones operands give the closed form
8192 per round. HBM read probe: the XOR of its sink equals the XOR of every
32-bit word of the buffer (numpy over the same bytes), on sizes with ragged
tails. LDS read probe: with 16-byte reads each thread's sum equals the numpy
sum of the words its lane's columns hold over the rounds; with transposing
8-byte reads (which redistribute 16-bit elements within 16-lane groups) the
XOR over each group of 16 lanes, folded to 16 bits, equals the numpy XOR of
the 16-bit elements those lanes addressed, in the V-tile layout of the
attention kernel (odd round counts: over an even count a group's XOR
cancels)."""
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


@pytest.mark.parametrize("nbytes,wg", [(16, 1), (48, 3), (48, 5), (4096 * 16 + 48, 7), ((8 << 20) + 16 * 5, 64),
                                       (64 << 20, 1024), (64 << 20, 4096)])
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


LDS_WORDS = (np.arange(16384, dtype=np.uint64) * 2654435761) % (1 << 32)   # the probe's array


def _lds_thread_sums_16(rounds):
    """Per-lane sums of the 16-byte form: lane l reads, in round r, column
    (l + r) % 64 (16 bytes = 4 words) of each of the 64 rows of 1 KB."""
    col = LDS_WORDS.reshape(64, 64, 4).sum(axis=(0, 2))   # [column]
    return np.array([sum(int(col[(l + r) % 64]) for r in range(rounds)) % (1 << 32) for l in range(64)],
                    dtype=np.uint64)


def _lds_group_xors_8(rounds):
    """Per 16-lane group of the transposing 8-byte form: the XOR of the 16-bit
    elements at the bytes the group's lanes address (the addressing the header
    states), over all reads of all rounds."""
    halves = LDS_WORDS.astype(np.uint32).view(np.uint16)   # 16-bit elements in address order
    out = np.zeros(4, dtype=np.uint64)
    for lane in range(64):
        h, q, e = lane >> 4, (lane >> 2) & 3, lane & 3
        for r in range(rounds):
            for t in range(128):
                byte = (8 * (t // 4) + 4 * (h // 2) + q) * 256 + ((2 * ((t + r) % 4) + h % 2) ^ (2 * q)) * 32 + 8 * e
                out[h] ^= int(np.bitwise_xor.reduce(halves[byte // 2:byte // 2 + 4]))
    return out


@pytest.mark.parametrize("wg,rounds", [(1, 1), (3, 5), (512, 3)])
def test_lds_read_probe_16_byte_sums(wg, rounds):
    print(f"[case] lds read probe width 16 wg={wg} rounds={rounds}", flush=True)
    sink, ticks = rf.rf_probe_lds_read(wg, rounds, 16)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32).astype(np.uint64).reshape(wg, 4, 64)
    want = _lds_thread_sums_16(rounds)
    assert (got == want[None, None, :]).all()
    assert bool((ticks.cpu() > 0).all())


@pytest.mark.parametrize("wg,rounds", [(1, 1), (2, 5), (512, 3)])
def test_lds_read_probe_transposing_group_xors(wg, rounds):
    print(f"[case] lds read probe width 8 wg={wg} rounds={rounds}", flush=True)
    sink, ticks = rf.rf_probe_lds_read(wg, rounds, 8)
    torch.cuda.synchronize()
    words = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32).reshape(wg, 4, 4, 16), axis=3)
    got = ((words & 0xffff) ^ (words >> 16)).astype(np.uint64)
    want = _lds_group_xors_8(rounds)
    assert (got == want[None, None, :]).all()
    assert bool((ticks.cpu() > 0).all())
