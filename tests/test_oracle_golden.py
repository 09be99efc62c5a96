"""Oracle regression snapshots (written by tests/golden/make_golden.py from the oracle)."""
import json
import os

import numpy as np

import oracle
from paper_2609_35140_amd import inputs

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_tiny_rows_snapshot():
    g = json.load(open(os.path.join(GOLD, "tiny_seed42_rows.json")))
    t = inputs.packed_qkv(inputs.tiny(), seed=g["seed"])
    rows = [tuple(r) for r in g["rows"]]
    o, lse = oracle.attention_rows_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"], rows, scale=g["scale"])
    assert np.allclose(o, np.array([[float(x) for x in r] for r in g["o"]]), rtol=0, atol=1e-13)
    assert np.allclose(lse, np.array([float(x) for x in g["lse"]]), rtol=0, atol=1e-13)


def test_logprob_snapshot():
    g = json.load(open(os.path.join(GOLD, "logprob_seed42_rows.json")))
    lg = inputs.logits_bf16(g["rows"], g["vocab"], g["sigma"], seed=g["seed"])
    tg = inputs.targets(g["rows"], g["vocab"], seed=g["seed"])
    assert list(tg) == g["targets"]
    lp = oracle.logprob_fp64(lg, tg)
    assert np.allclose(lp, np.array([float(x) for x in g["logp"]]), rtol=0, atol=1e-13)
