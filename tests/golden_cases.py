"""Loader for the hand-worked fixtures under tests/golden/."""
import json
import os

import numpy as np

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(HERE, name)) as f:
        d = json.load(f)
    gj = d["graph"]
    g = dict(num_states=gj["num_states"], start_state=gj["start_state"],
             row_ptr=np.array(gj["row_ptr"], np.uint32), dst=np.array(gj["dst"], np.uint32),
             ilabel=np.array(gj["ilabel"], np.int32), olabel=np.array(gj["olabel"], np.int32),
             weight=np.array(gj["weight"], np.float32),
             final_weight=None if gj.get("final_weight") is None
             else np.array(gj["final_weight"], np.float32))
    L = np.array(d["loglikes"], np.float32)
    return d, g, L
