"""Parser for the hand-typed fixtures under tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _lines(path):
    with open(path) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if line:
                yield line


def load_lookup(name):
    it = _lines(os.path.join(GOLDEN, name))
    case = {"tables": [], "dims": [], "pooling": [], "ids": {}, "offsets": {}}
    for line in it:
        tok = line.split()
        if tok[0] == "tables":
            case["T"] = int(tok[1])
        elif tok[0] == "table":
            dtype = np.float16 if tok[2] == "f16" else np.float32
            dim = int(tok[4])
            pool = 1 if tok[6] == "mean" else 0
            rows = []
            for row in it:
                if row == "end":
                    break
                rows.append([float(x) for x in row.split()])
            arr = np.array(rows, dtype=np.float64)
            assert arr.shape[1] == dim
            assert np.array_equal(arr.astype(dtype).astype(np.float64), arr), "fixture value not exact"
            case["tables"].append(arr.astype(dtype))
            case["dims"].append(dim)
            case["pooling"].append(pool)
        elif tok[0] == "batch":
            case["B"] = int(tok[1])
        elif tok[0] == "offsets":
            if tok[1] == "none":
                case["offsets"] = None
            else:
                case["offsets"][int(tok[1])] = [int(x) for x in tok[3:]]
        elif tok[0] == "ids":
            case["ids"][int(tok[1])] = [int(x) for x in tok[3:]]
        elif tok[0] == "expected":
            rows = []
            for row in it:
                if row == "end":
                    break
                rows.append([float(x) for x in row.split()])
            case["expected"] = np.array(rows, dtype=np.float64)
    T = case["T"]
    case["ids"] = np.concatenate([np.array(case["ids"][t], dtype=np.int32) for t in range(T)])
    if case["offsets"] is not None:
        case["offsets"] = np.array([case["offsets"][t] for t in range(T)], dtype=np.int32)
    return case


def load_plan(name):
    case = {"offsets": {}}
    for line in _lines(os.path.join(GOLDEN, name)):
        tok = line.split()
        key, vals = tok[0], tok[1:]
        if key == "offsets":
            case["offsets"][int(vals[0])] = [int(x) for x in vals[2:]]
        elif key == "dtypes":
            case["dtypes"] = [1 if v == "f16" else 0 for v in vals]
        elif key == "out":
            case["out_dtype"] = 1 if vals[0] == "f16" else 0
        elif len(vals) == 1 and key in ("batch", "chunk_rows", "item_cost", "waves", "flags", "total_ids"):
            case[key] = int(vals[0])
        else:
            case[key] = np.array([int(v) for v in vals], dtype=np.int64)
    T = len(case["dims"])
    case["offsets"] = np.array([case["offsets"][t] for t in range(T)], dtype=np.int32)
    return case
