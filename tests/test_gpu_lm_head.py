"""GPU LM head: oracle parity, and the same logits bits for a row however
the batch is formed -- which, fed to the log-prob, gives a reuse ratio of
exactly one end to end (Section 3.1)."""
import numpy as np
import pytest

import oracle
from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu
gu = pytest.importorskip("gpu_util")


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


@pytest.mark.parametrize("T,V,H", [(300, 1000, 512), (129, 257, 64), (1, 4099, 1024), (256, 512, 4096)])
def test_matches_oracle(ua, T, V, H):
    h = inputs.normal_bf16((T, H), 1.0, 94, T, V)
    w = inputs.normal_bf16((V, H), float(2.0 / np.sqrt(H)), 95, T, V)
    got = gu.host_bits(ua.lm_head(gu.dev(h), gu.dev(w)))
    ref = oracle.logits_fp64(h, w)
    err = np.abs(oracle.bf16_to_f64(got) - ref)
    # bf16 output rounding plus fp32 accumulation over H terms
    bound = 2.0 ** -8 * np.abs(ref) + H * 2.0 ** -24 * oracle.abs_dot(h, w)
    exact = np.mean(got == oracle.logits_bf16(h, w))
    print(f"T={T} V={V} H={H}: {exact:.4f} equal to the rounded fp64 logits, max err {err.max():.3g}", flush=True)
    assert np.all(err <= bound) and exact > 0.95


def test_rows_are_batch_invariant_and_ratio_is_one(ua):
    import torch
    T, V, H = 640, 1500, 1024
    h = gu.dev(inputs.normal_bf16((T, H), 1.0, 96))
    w = gu.dev(inputs.normal_bf16((V, H), 0.0625, 97))
    full = ua.lm_head(h, w)
    tg = gu.dev_i32(inputs.targets(T, V, tag=98))
    lp_full = ua.logprob(full, tg)
    g = inputs.rng(99)
    for n in (1, 2, 7, 128, 129, 300):
        idx = torch.from_numpy(g.permutation(T)[:n]).cuda()
        part = ua.lm_head(h[idx].contiguous(), w)
        assert torch.equal(part.view(torch.int16), full[idx].view(torch.int16)), n
        lp = ua.logprob(part, tg[idx].contiguous())
        assert torch.equal(lp.view(torch.int32), lp_full[idx].view(torch.int32)), n
        assert bool((torch.exp(lp.double() - lp_full[idx].double()) == 1.0).all())
    # a row alone
    one = ua.lm_head(h[5:6], w)
    assert torch.equal(one.view(torch.int16), full[5:6].view(torch.int16))


@pytest.mark.parametrize("T,V,H,it", [(300, 1000, 512, 1.0), (129, 257, 64, 1.0), (1, 4099, 1024, 0.7),
                                       (256, 512, 4096, 1.0), (70, 20000, 256, 1.3)])
def test_fused_logprob_matches_oracle(ua, T, V, H, it):
    import torch
    h = inputs.normal_bf16((T, H), 1.0, 94, T, V)
    w = inputs.normal_bf16((V, H), float(2.0 / np.sqrt(H)), 95, T, V)
    tg = inputs.targets(T, V, tag=T)
    hd, wd, td = gu.dev(h), gu.dev(w), gu.dev_i32(tg)
    lp = ua.lm_head_logprob(hd, wd, td, inv_temperature=it).cpu().numpy().astype(np.float64)
    ref, bound = oracle.lm_head_logprob_fp64(h, w, tg, it)
    err = np.abs(lp - ref)
    print(f"T={T} V={V} H={H} it={it}: max err {err.max():.3g}, max err/bound {np.max(err / bound):.3f}, "
          f"median bound {np.median(bound):.3g}", flush=True)
    assert np.all(err <= bound)
    # the same logits through the two-call path: both fp32 log-softmaxes of identical logits
    logits = torch.empty((T, (V + 7) // 8 * 8), dtype=torch.bfloat16, device="cuda")[:, :V]
    lp2 = ua.lm_head_logprob(hd, wd, td, inv_temperature=it, logits=logits)
    assert torch.equal(logits.view(torch.int16), ua.lm_head(hd, wd).view(torch.int16))
    two = ua.logprob(logits, td, inv_temperature=it)
    assert float((lp2.double() - two.double()).abs().max()) < 2e-5


def test_fused_logprob_rows_are_batch_invariant(ua):
    import torch
    T, V, H = 640, 1500, 1024
    h = gu.dev(inputs.normal_bf16((T, H), 1.0, 96))
    w = gu.dev(inputs.normal_bf16((V, H), 0.0625, 97))
    tg = gu.dev_i32(inputs.targets(T, V, tag=98))
    full = ua.lm_head_logprob(h, w, tg)
    g = inputs.rng(99, 1)
    for n in (1, 2, 7, 128, 129, 257, 300):
        idx = torch.from_numpy(g.permutation(T)[:n]).cuda()
        part = ua.lm_head_logprob(h[idx].contiguous(), w, tg[idx].contiguous())
        assert torch.equal(part.view(torch.int32), full[idx].view(torch.int32)), n
        assert bool((torch.exp(part.double() - full[idx].double()) == 1.0).all())
    # repeated calls, and a target outside the vocabulary
    again = ua.lm_head_logprob(h, w, tg)
    assert torch.equal(again.view(torch.int32), full.view(torch.int32))
    bad = tg.clone()
    bad[3] = V
    bad[5] = -1
    out = ua.lm_head_logprob(h, w, bad)
    assert bool(torch.isnan(out[3])) and bool(torch.isnan(out[5]))
    keep = torch.ones(T, dtype=torch.bool, device="cuda")
    keep[3] = keep[5] = False
    assert torch.equal(out[keep].view(torch.int32), full[keep].view(torch.int32))
