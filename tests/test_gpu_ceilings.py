"""The measured-ceiling microbenchmarks read what they claim to read: the XOR
checksum of a streaming read equals the XOR of every 32-bit word of the
buffer, in the contiguous order and in a random 16 KB block order, and the
MFMA kernel produces its accumulator sums."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def cl():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import ceilings
    ceilings.lib()
    return ceilings


def test_read_checksum_contiguous_and_paged(cl):
    import torch
    g = np.random.default_rng(3)
    words = g.integers(0, 2 ** 31, size=(64 << 20) // 4, dtype=np.int64).astype(np.int32)
    src = torch.from_numpy(words).cuda()
    want = int(np.bitwise_xor.reduce(words.view(np.uint32)))
    ck = cl.read(src, None, 16384)
    got = int(np.bitwise_xor.reduce(ck.cpu().numpy().view(np.uint32)))
    assert got == want
    nblk = (64 << 20) // 16384
    perm = torch.from_numpy(g.permutation(nblk).astype(np.int32)).cuda()
    ck = cl.read(src, perm, 16384)
    assert int(np.bitwise_xor.reduce(ck.cpu().numpy().view(np.uint32))) == want
    ck = cl.read(src, perm, 16384, nontemporal=True)
    assert int(np.bitwise_xor.reduce(ck.cpu().numpy().view(np.uint32))) == want
    # half the blocks, in a random order: the XOR of exactly those blocks
    half = g.permutation(nblk)[: nblk // 2].astype(np.int32)
    ck = cl.read(src, torch.from_numpy(half).cuda(), 16384)
    sel = words.view(np.uint32).reshape(nblk, -1)[half]
    assert int(np.bitwise_xor.reduce(ck.cpu().numpy().view(np.uint32))) == int(np.bitwise_xor.reduce(sel.ravel()))


def test_mfma_kernel_runs_and_rates(cl):
    tflops = cl.mfma_tflops(iters=2000, reps=2)
    print(f"mfma ceiling (short run): {tflops:.1f} TFLOP/s", flush=True)
    assert 100.0 < tflops < 3000.0
