"""GPU log-prob gather: oracle parity, batch invariance, ratio exactly one."""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
gu = pytest.importorskip("gpu_util")

# fp32 reduction of up to ~1.5e5 terms in a fixed tree; logp ~ -14 +/- 4 for
# N(0,4) logits over 151,936 entries: a few fp32 ulps of |logp| plus the
# relative error of the sum.
ATOL = 2e-5


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


@pytest.mark.parametrize("rows,vocab,sigma,it", [(64, 151936, 2.0, 1.0), (33, 1000, 1.0, 0.7), (5, 13, 3.0, 1.0),
                                                (7, 4099, 2.0, 1.3)])
def test_logprob_matches_oracle(ua, rows, vocab, sigma, it):
    lg = inputs.logits_bf16(rows, vocab, sigma, tag=vocab)
    tg = inputs.targets(rows, vocab, tag=vocab)
    # rows live in a buffer whose stride is a multiple of 8 elements (16 bytes)
    stride = (vocab + 7) // 8 * 8
    buf = np.zeros((rows, stride), dtype=np.uint16)
    buf[:, :vocab] = lg
    got = ua.logprob(gu.dev(buf)[:, :vocab], gu.dev_i32(tg), inv_temperature=it).cpu().numpy().astype(np.float64)
    ref = oracle.logprob_fp64(lg, tg, inv_temperature=it)
    err = np.abs(got - ref)
    print("logprob max err", err.max(), flush=True)
    assert err.max() < ATOL


def test_logprob_strided_rows(ua):
    import torch
    lg = inputs.logits_bf16(9, 1024, 2.0, tag=5)
    tg = inputs.targets(9, 1000, tag=5)
    big = gu.dev(lg)
    got = ua.logprob(big[:, :1000], gu.dev_i32(tg)).cpu().numpy()
    ref = oracle.logprob_fp64(lg[:, :1000], tg)
    assert np.max(np.abs(got - ref)) < ATOL
    dense = ua.logprob(big[:, :1000].contiguous(), gu.dev_i32(tg)).cpu().numpy()
    assert np.array_equal(got.view(np.uint32), dense.view(np.uint32))


def test_logprob_batch_invariance_and_unit_ratio(ua):
    """A row alone, in a batch of 8192, reversed: the same bits, so
    exp(logp_upd - logp_roll) is exactly 1.0 (Section 3.1)."""
    import torch
    V = 151936
    lg = gu.dev(inputs.logits_bf16(512, V, 2.0, tag=9))
    tg = gu.dev_i32(inputs.targets(512, V, tag=9))
    big = lg.repeat(16, 1)          # 8192 rows
    bigt = tg.repeat(16)
    full = ua.logprob(big, bigt)
    first = full[:512]
    for rep in range(1, 16):
        assert torch.equal(full[rep * 512:(rep + 1) * 512].view(torch.int32), first.view(torch.int32))
    rev = ua.logprob(lg.flip(0).contiguous(), tg.flip(0).contiguous()).flip(0)
    assert torch.equal(rev.view(torch.int32), first.view(torch.int32))
    for r in [0, 100, 511]:
        single = ua.logprob(lg[r:r + 1].contiguous(), tg[r:r + 1].contiguous())
        assert torch.equal(single.view(torch.int32), first[r:r + 1].view(torch.int32))
    ratio = torch.exp(full[:512].double() - rev.double())
    assert bool((ratio == 1.0).all())


def test_logprob_constant_row(ua):
    import torch
    V = 4096
    lg = torch.full((3, V), 1.5, dtype=torch.bfloat16, device="cuda")
    tg = gu.dev_i32([0, 5, V - 1])
    got = ua.logprob(lg, tg).cpu().numpy()
    assert np.max(np.abs(got + np.log(V))) < 2e-6
