"""Parity records of the GPU tests: when DERF_PARITY_RECORD names a file,
each check appends one JSON line to it (test label, sample and ray counts,
near-bisector counts, largest differences, tolerance), so that a run leaves a
written summary of what it asserted."""
import json
import os


def record(**fields):
    path = os.environ.get("DERF_PARITY_RECORD")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps(fields, default=_plain) + "\n")


def _plain(v):
    """numpy scalars and arrays as plain Python values."""
    return v.item() if hasattr(v, "item") and getattr(v, "size", 1) == 1 else v.tolist()
