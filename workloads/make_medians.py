"""Stores the median pairwise distance of every workload in medians.json.

The values are median_pairwise_distance(make_data(w)[0]) exactly (as float
hex strings); make_inputs uses them instead of recomputing (the
n = 40000 workload's 800 million pairs take minutes).

Usage (from the repository root): python -m workloads.make_medians [NAME ...]
"""
import json
import sys

from . import MEDIANS_PATH, WORKLOADS, make_data, median_pairwise_distance


def main(names):
    try:
        with open(MEDIANS_PATH) as fh:
            out = json.load(fh)
    except OSError:
        out = {}
    for name in names or sorted(WORKLOADS):
        X, _ = make_data(WORKLOADS[name])
        out[name] = float(median_pairwise_distance(X)).hex()
        print(name, float.fromhex(out[name]), flush=True)
        with open(MEDIANS_PATH, "w") as fh:
            json.dump(out, fh, indent=1, sort_keys=True)
            fh.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:])
