"""Write input_sha256.json: SHA-256 of each seeded workload's fp32 bytes.

Calls only ``workloads.generate``; freezes the draw order so that the GPU
tests, the bench and the oracle all see the same inputs.  Run from the repo
root:  python tests/golden/make_input_hashes.py
"""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(
    os.path.abspath(__file__)))))

import workloads  # noqa: E402


def main():
    out = {}
    for key, w in workloads.WORKLOADS.items():
        x = workloads.generate(key)
        out[key] = {"rows": w.rows, "cols": w.cols, "seed": w.seed,
                    "sha256": workloads.sha256_f32(x)}
    path = os.path.join(os.path.dirname(__file__), "input_sha256.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
