"""The fp64 attention oracle against brute force, a library routine, closed
forms and invariants; planted mistakes must be caught by those checks."""
import numpy as np
import pytest

import oracle
import oracle.attention as oa
import oracle_checks as oc


@pytest.mark.parametrize("chk", oc.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pinned(chk):
    chk(oracle.causal_attention_fp64)


# ---------------------------------------------------------------- mutants
def _mut_head(kind):
    def f(qh, kh, vh, scale):
        L = qh.shape[0]
        if kind == "transposed_scores":
            s = (kh @ qh.T) * scale
        elif kind == "no_scale":
            s = qh @ kh.T
        elif kind == "scale_squared":
            s = (qh @ kh.T) * scale * scale
        else:
            s = (qh @ kh.T) * scale
        diag = {"mask_includes_next": 2, "mask_excludes_self": 0}.get(kind, 1)
        s = s.copy()
        s[np.triu(np.ones((L, L), dtype=bool), k=diag)] = -np.inf
        m = s.max(axis=1, keepdims=True)
        e = np.exp(m - s) if kind == "sign_flip" else np.exp(s - m)
        if kind == "normalize_wrong_axis":
            z = e.sum(axis=0, keepdims=True)
        else:
            z = e.sum(axis=1, keepdims=True)
        p = e / z
        o = p @ vh
        if kind == "drop_last_key":
            p2 = e[:, :-1] / z
            o = p2 @ vh[:-1]
        lse = (np.log(z) if kind == "lse_without_max" else m + np.log(z))[:, 0] if kind != "normalize_wrong_axis" \
            else (m + np.log(e.sum(axis=1, keepdims=True)))[:, 0]
        return o, lse
    return f


HEAD_MUTANTS = ["transposed_scores", "no_scale", "scale_squared", "mask_includes_next", "mask_excludes_self",
                "sign_flip", "normalize_wrong_axis", "drop_last_key", "lse_without_max"]


@pytest.mark.parametrize("kind", HEAD_MUTANTS)
def test_planted_mistake_is_caught(kind, monkeypatch):
    monkeypatch.setattr(oa, "_one_head_causal", _mut_head(kind))
    with np.errstate(all="ignore"):
        failures = oc.run_all(oa.causal_attention_fp64)
    assert failures, f"planted mistake {kind!r} passed every pin"


def test_planted_gqa_map_is_caught():
    def wrong_map(q, k, v, cu, scale=None):
        hq, hkv = q.shape[1], k.shape[1]
        o = np.zeros(q.shape); lse = np.zeros(q.shape[:2])
        for b in range(len(cu) - 1):
            lo, hi = int(cu[b]), int(cu[b + 1])
            for h in range(hq):
                oh, lh = oa._one_head_causal(q[lo:hi, h], k[lo:hi, h % hkv], v[lo:hi, h % hkv], scale)
                o[lo:hi, h], lse[lo:hi, h] = oh, lh
        return o, lse
    assert oc.run_all(wrong_map), "h % Hkv map passed every pin"


def test_bf16_decode_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0001, 0x7F7F, 0x4049], dtype=np.uint16)
    vals = oracle.bf16_to_f64(bits)
    assert vals[0] == 1.0 and vals[1] == -1.0
    assert vals[2] == 2.0 ** -133        # smallest bf16 subnormal
    assert vals[3] == (2 - 2 ** -7) * 2.0 ** 127
    assert vals[4] == 3.140625


def test_round_to_bf16_ties_to_even():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20, -1.0 - 2 ** -8], dtype=np.float32)
    r = oracle.round_to_bf16(x)
    assert list(r) == [1.0, 1.0 + 2 ** -6, 1.0 + 2 ** -7, -1.0]


def test_rows_match_full():
    from paper_2609_35140_amd import inputs
    w = inputs.custom(4, 2, 32, [70, 33], sigma=1.0)
    t = inputs.packed_qkv(w)
    o, lse = oracle.causal_attention_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"])
    rows = [(0, 0), (69, 3), (70, 1), (102, 2), (85, 0)]
    orows, lrows = oracle.attention_rows_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"], rows)
    for r, (tok, h) in enumerate(rows):
        assert np.max(np.abs(orows[r] - o[tok, h])) < 1e-12
        assert abs(lrows[r] - lse[tok, h]) < 1e-12
