"""Writes tests/golden/oracle_small.json: a regression record of the fp64 oracle.

Calls only ``oracle/`` and the seeded input generator; no value here comes from
the GPU path.  Re-run only when the oracle's arithmetic is deliberately changed
(and say which passage of the paper justifies the change).
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import gdn_inputs  # noqa: E402
import oracle  # noqa: E402

SHAPE = dict(B=2, T=9, H=2, Dk=4, Dv=3)
SEED = 424242


def main():
    inp = gdn_inputs.make_inputs(0, seed=SEED, state="normal0.02", **SHAPE)
    out, st = oracle.gdn_forward(inp["q"], inp["k"], inp["v"], inp["alpha"],
                                 inp["beta"], inp["state_in"], nthreads=1)
    rec = dict(note="fp64 oracle on gdn_inputs.make_inputs(0, seed=%d, state='normal0.02', %s)"
               % (SEED, ", ".join(f"{k}={v}" for k, v in SHAPE.items())),
               seed=SEED, shape=SHAPE,
               out=[float(x).hex() for x in out.ravel()],
               state=[float(x).hex() for x in st.ravel()])
    with open(os.path.join(HERE, "oracle_small.json"), "w") as f:
        json.dump(rec, f, indent=0)
        f.write("\n")


if __name__ == "__main__":
    main()
