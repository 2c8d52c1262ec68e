"""Write tests/golden/*.json: oracle outputs on seeded workloads.

Calls only ``oracle`` and ``workloads``.  The paper prints no numeric example
for the RNN loop (its Table 1 reports throughput only), so these files are a
regression record of the pinned oracle on the generator's inputs, not values
taken from the paper.  Run from the repository root:
    python tests/golden/make_golden.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle      # noqa: E402
import workloads   # noqa: E402


def main():
    for name in ["tiny_f32"]:
        inp = workloads.workload_inputs(name)
        h, c = oracle.forward_inputs(inp)
        rec = {
            "workload": name,
            "source": "fp64 oracle (oracle/lstm_oracle.c) on workloads.workload_inputs; "
                      "definition: AutoGraph Section 9 'RNN cells' and Appendix A",
            "lengths": inp.lengths.tolist(),
            "h": [[float.hex(float(v)) for v in row] for row in h],
            "c": [[float.hex(float(v)) for v in row] for row in c],
        }
        with open(os.path.join(HERE, f"{name}.json"), "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")


if __name__ == "__main__":
    main()
