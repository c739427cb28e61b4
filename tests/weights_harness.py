"""Test harness for the weight-shard rebuild: model specs and stores in the
shapes the oracle and the C-ABI take (no slicing arithmetic here)."""
from __future__ import annotations

import json
import os

import numpy as np

import synthkv
from synthkv.models import FIRST_STAGE, LAST_STAGE, REPLICATED, SPLIT_COLS, SPLIT_ROWS

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SPLITS = {"replicated": REPLICATED, "rows": SPLIT_ROWS, "cols": SPLIT_COLS}
LAYERS = {"first": FIRST_STAGE, "last": LAST_STAGE}


def oracle_tensors(spec, store, layers=None):
    """[(layer, [(full part array, split, units), ...])] per GPU tensor."""
    return [(t.layer, [(synthkv.models.part_array(spec, store, p), p.split, p.units) for p in t.parts])
            for t in spec.tensors(layers)]


def abi_tensors(spec, store, layers=None):
    """[(layer, [(host address, rows, cols, split, units), ...])] per GPU tensor."""
    return [(t.layer, [(store[p.name].data_ptr(), p.rows, p.cols, p.split, p.units) for p in t.parts])
            for t in spec.tensors(layers)]


def load_golden(name):
    """(golden dict, tensor names, oracle-form tensors, host part arrays by name)."""
    with open(os.path.join(GOLDEN, name)) as f:
        g = json.load(f)
    arrays = {}
    for pname, p in g["parts"].items():
        r = np.arange(p["rows"]).reshape(-1, 1)
        c = np.arange(p["cols"]).reshape(1, -1)
        arrays[pname] = np.ascontiguousarray((100 * p["id"] + 10 * r + c).astype(np.uint16))
    tensors, names = [], []
    for t in g["tensors"]:
        layer = LAYERS.get(t["layer"], t["layer"])
        tensors.append((layer, [(arrays[n], SPLITS[g["parts"][n]["split"]], g["parts"][n]["units"])
                                for n in t["parts"]]))
        names.append(t["name"])
    return g, names, tensors, arrays
