"""Write the oracle regression snapshots in this folder (calls only oracle/)."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2609_35140_amd import inputs  # noqa: E402

TINY_ROWS = [(0, 0), (0, 1), (1, 0), (31, 1), (63, 0), (64, 1), (65, 0), (100, 1), (126, 0), (127, 0), (127, 1), (96, 0)]


def main():
    w = inputs.tiny()
    t = inputs.packed_qkv(w, seed=42)
    o, lse = oracle.attention_rows_fp64(t["q"], t["k"], t["v"], t["cu_seqlens"], TINY_ROWS)
    with open(os.path.join(HERE, "tiny_seed42_rows.json"), "w") as f:
        json.dump({"workload": "tiny", "seed": 42, "scale": oracle.default_scale(64), "rows": TINY_ROWS,
                   "o": [[repr(float(x)) for x in r] for r in o], "lse": [repr(float(x)) for x in lse]}, f, indent=0)
    lg = inputs.logits_bf16(8, 4096, 2.0, seed=42)
    tg = inputs.targets(8, 4096, seed=42)
    lp = oracle.logprob_fp64(lg, tg)
    with open(os.path.join(HERE, "logprob_seed42_rows.json"), "w") as f:
        json.dump({"rows": 8, "vocab": 4096, "sigma": 2.0, "seed": 42, "targets": [int(x) for x in tg],
                   "logp": [repr(float(x)) for x in lp]}, f, indent=0)


if __name__ == "__main__":
    main()
