"""Writes format_v1_fingerprint.json: the sha256 of the oracle's format-v1 map
(reading R19) over the class radices and the points of a fixed index list
(first and last index of every class, then 256 indices from numpy PCG64 seed
2609).  Calls only oracle/.

    python tests/golden/make_format_v1_fingerprint.py
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

from oracle import index as I  # noqa: E402


def indices():
    offs = I.class_offsets()
    idx = []
    for c in range(len(offs) - 1):
        idx += [offs[c], offs[c + 1] - 1]
    rng = np.random.default_rng(2609)
    idx += [int(v) for v in rng.integers(0, offs[-1], 256, dtype=np.int64)]
    return idx


if __name__ == "__main__":
    idx = indices()
    out = {"what": "sha256 over (class id, radices in composition order) of every class, then "
                   "(index, point) for each index of the list",
           "n_indices": len(idx), "sha256": I.fingerprint(idx)}
    with open(os.path.join(HERE, "format_v1_fingerprint.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(out)
