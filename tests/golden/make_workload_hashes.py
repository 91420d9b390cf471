"""Writes workload_hashes.json: SHA-256 of the seeded generators' tensors.

    python tests/golden/make_workload_hashes.py

The hashes pin the generators' determinism only (no expected result of the
method is stored here)."""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

import torch  # noqa: E402
from test_workloads import _hash_specs  # noqa: E402
import workloads as wl  # noqa: E402


def main():
    out = {}
    for key, spec in _hash_specs().items():
        t = wl.draw(spec)
        out[key] = {n: hashlib.sha256(t[n].contiguous().view(torch.uint8).numpy().tobytes()).hexdigest()
                    for n in ("x", "w", "dy")}
    with open(os.path.join(HERE, "workload_hashes.json"), "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
