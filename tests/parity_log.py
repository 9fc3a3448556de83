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


# columns of the summary, per record kind: (heading, field)
_COLUMNS = {
    "cells": [("samples", "samples"), ("near bisector", "near_bisector"),
              ("mismatches", "mismatches")],
    "cells at the emitted depths": [("samples", "samples"), ("mismatches", "mismatches")],
    "pixels": [("rays", "rays"), ("max abs rgb", "max_abs_rgb"),
               ("max abs depth", "max_abs_depth"), ("max abs opacity", "max_abs_opacity"),
               ("tol", "tol")],
    "pixels at the emitted depths": [("rays", "rays"), ("max abs rgb", "max_abs_rgb"),
                                     ("max abs depth", "max_abs_depth"),
                                     ("max abs opacity", "max_abs_opacity"), ("tol", "tol")],
    "fine depths and merged composite": [("rays", "rays"), ("max abs t", "max_abs_t"),
                                         ("tol t", "tol_t"),
                                         ("max abs composite", "max_abs_composite"),
                                         ("tol", "tol_composite")],
    "end to end": [("rays", "rays"), ("well conditioned", "well_conditioned"),
                   ("flipped", "flipped"), ("max abs (well)", "max_abs_well"),
                   ("tol (well)", "tol_well"), ("max abs (other)", "max_abs_other"),
                   ("tol (other)", "tol_other")],
    "gated cells and pixels": [("rays", "rays"), ("near-tie samples", "near_tie_samples"),
                               ("clean rays", "clean_rays"), ("runs per ray", "runs_per_ray"),
                               ("max abs", "max_abs"), ("tol", "tol")],
}


def _cell(v):
    if isinstance(v, float):
        return "%.3g" % v
    return "{:,}".format(v) if isinstance(v, int) else str(v)


def summarize(path):
    """Markdown tables of a parity record file, one per kind of check, one
    row per record in the order the tests wrote them."""
    recs = [json.loads(line) for line in open(path) if line.strip()]
    kinds = []
    for r in recs:
        if r.get("kind") not in kinds:
            kinds.append(r.get("kind"))
    out = []
    for kind in kinds:
        cols = _COLUMNS.get(kind)
        rows = [r for r in recs if r.get("kind") == kind]
        if cols is None:
            cols = [(k, k) for k in rows[0] if k not in ("test", "kind")]
        out.append("### %s\n" % kind)
        out.append("| test | " + " | ".join(h for h, _ in cols) + " |")
        out.append("|---|" + "---|" * len(cols))
        for r in rows:
            out.append("| %s | " % r.get("test", "") +
                       " | ".join(_cell(r.get(f, "")) for _, f in cols) + " |")
        out.append("")
    return "\n".join(out)


if __name__ == "__main__":
    import sys
    print(summarize(sys.argv[1]))
