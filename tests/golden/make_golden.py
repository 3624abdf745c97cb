"""Writes tests/golden/host_rules_oracle.json from the oracle alone.

The stored values are the oracle's seeded candidate sample on fixed family
sizes and its CU masks for every share and slot; the test that reads them
holds the oracle to what it computed when they were written. Run from the
repository root: python tests/golden/make_golden.py
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle.host_rules as HR  # noqa: E402

SAMPLES = [
    # (families, sizes, n, seed, config_id, layer_id)
    ([1, 4], [7000, 13000], 256, 0, 2, 3),
    ([1, 2, 3, 4], [50, 0, 10, 3000], 96, 7, 5, 11),
    ([4], [20], 64, 1, 1, 0),
]
SHARES = [(0.125, 8), (0.25, 4), (0.5, 2), (0.75, 1), (1.0, 1)]


def main() -> None:
    out = {"about": "written by tests/golden/make_golden.py from oracle.host_rules only",
           "samples": [{"families": f, "sizes": s, "n": n, "seed": seed, "config_id": c, "layer_id": l,
                        "positions": HR.sample_positions(f, s, n, seed, c, l)}
                       for f, s, n, seed, c, l in SAMPLES],
           "cu_masks": [{"fraction": fr, "slot": k, "words": HR.cu_mask(256, fr, k)}
                        for fr, slots in SHARES for k in range(slots)]}
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "host_rules_oracle.json")
    with open(path, "w") as fh:
        json.dump(out, fh)
        fh.write("\n")


if __name__ == "__main__":
    main()
