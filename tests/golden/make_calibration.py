"""Writes tests/golden/calibration.json: the output scale of every int8 op.

Calls only the CPU oracle (oracle/) and the seeded input generators
(workloads/). Each int8 op's scale is so = max|g| / 127 over its fp32
pre-requant output g on the full seed-0 batch, computed in the chain order
(an op fed by another uses that op's calibrated scale as its activation scale).

    python tests/golden/make_calibration.py            # all workloads
    python tests/golden/make_calibration.py c1 c2      # a subset (merged in)
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle.chain as chain  # noqa: E402
import workloads as wk  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "calibration.json")


def main(names):
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data = json.load(f)
    wls = wk.workloads()
    for name in names or list(wls):
        t = time.time()
        _, scales, _ = chain.run(wls[name], keep_outputs=False)
        data[name] = {k: float(v) for k, v in scales.items()}
        print(f"{name}: {len(scales)} scales in {time.time() - t:.1f} s", flush=True)
        with open(OUT, "w") as f:
            json.dump({"generator": "tests/golden/make_calibration.py (CPU oracle, seed 0)",
                       **{k: v for k, v in data.items() if k != "generator"}}, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:])
