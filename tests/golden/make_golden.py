"""Write tests/golden/tiny_layer_oracle.json: a regression lock on the oracle.

The stored outputs are the oracle's own (this script calls only oracle/ and
the seeded input generator), for a tiny float32 layer: L_d = 24, L_q = 4,
7 important tokens, 4 query heads / 2 KV heads, head_dim 8. Re-run only when
a change to the oracle's arithmetic is justified by the paper, and say which
passage in the commit message.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import daf_inputs as di  # noqa: E402
import oracle  # noqa: E402

SHAPE = di.Shape("golden_tiny", L_d=24, L_q=4, n=7, hq=4, hkv=2, d=8, dtype=di.F32,
                 qkv_std=1.0, cache_std=1.0, seed=77)


def compute():
    b = di.make_batch(SHAPE)
    r = b.request(0)
    out = oracle.get().layer(r["idx"], r["q_imp"], r["k_imp"], r["v_imp"], r["q_q"], r["k_q"],
                             r["v_q"], r["k_cache"], r["v_cache"], r["hidden"],
                             scale=oracle.default_scale(SHAPE.d), L_d=SHAPE.L_d)
    return r, out


def main():
    r, out = compute()
    doc = {
        "what": "oracle outputs for a tiny seeded float32 DAF layer (regression lock)",
        "shape": {k: getattr(SHAPE, k) for k in ("L_d", "L_q", "n", "hq", "hkv", "d", "seed")},
        "idx": r["idx"].tolist(),
        "o_imp": [float(x) for x in out["o_imp"].ravel()],
        "lse_imp": [float(x) for x in out["lse_imp"].ravel()],
        "o_q": [float(x) for x in out["o_q"].ravel()],
        "lse_q": [float(x) for x in out["lse_q"].ravel()],
    }
    with open(os.path.join(HERE, "tiny_layer_oracle.json"), "w") as f:
        json.dump(doc, f, indent=0)


if __name__ == "__main__":
    main()
