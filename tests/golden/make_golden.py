"""Write tests/golden/oracle_small.json: oracle outputs for a small seeded batch.

Regression fixture for the fp64 oracle (any later change to its arithmetic shows
up as a mismatch) and a fixed reference for the GPU path. Inputs are not
stored: they are regenerated from the recorded seed and shapes by the input
generator. Expected values come from ``oracle/`` only.

    python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2411_01142_amd import workloads as W  # noqa: E402

SPEC = dict(seq_lens=[1, 5, 16, 17, 40], num_q_heads=4, num_kv_heads=2, head_dim=128,
            block_size=16, seed=20241102)


def build():
    return W.build_case(SPEC["seq_lens"], SPEC["num_q_heads"], SPEC["num_kv_heads"],
                        SPEC["head_dim"], SPEC["block_size"], seed=SPEC["seed"])


def main():
    case = build()
    out, out64 = oracle.decode_attention(case, want_f64=True)
    rec = {
        "what": "fp64 oracle output (rounded to float32) for the seeded batch in 'spec'",
        "spec": SPEC,
        "out_f32_hex": [[[float(x).hex() for x in row] for row in head] for head in out.astype(np.float64)],
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "oracle_small.json")
    with open(path, "w") as f:
        json.dump(rec, f, separators=(",", ":"))
    print(f"wrote {path}")


if __name__ == "__main__":
    main()
