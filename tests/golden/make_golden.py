"""Write the stored oracle values of tests/golden/ (calls only the oracle and
the seeded input generator).

The paper prints no worked numeric example (no intermediate or output value
of a render), so the fixtures here are regression values of the oracle on
the 32x32 tiny scene: they catch any later, unintended change to the
oracle's arithmetic.  Re-running this script is a deliberate act that a
commit message must justify.
"""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
from paper_2011_12490_amd import scenes  # noqa: E402

RAYS = [0, 1, 31, 500, 517, 1023]


def main():
    oracle.build(force=False)
    cfg = scenes.CONFIGS["tiny"]
    sc = scenes.make_scene(cfg)
    ids = np.array(RAYS)
    r = oracle.render(sc.sites, cfg.arch, sc.weights, sc.rays_o[ids], sc.rays_d[ids], cfg.near,
                      cfg.far, cfg.n_coarse, 0, seed=scenes.SEED_RENDER, ray_ids=ids,
                      per_sample=True)
    out = {
        "what": "oracle render of the 32x32 tiny scene (4 uniform sites, 4x64 heads, "
                "32 jittered samples on [2, 6]); regression fixture, not a paper value",
        "seed": scenes.SEED_RENDER,
        "rays": RAYS,
        "rgb": r.rgb.tolist(),
        "depth": r.depth.tolist(),
        "opacity": r.opacity.tolist(),
        "cells": r.cell.tolist(),
        "t": [[float(v) for v in row] for row in r.t],
    }
    with open(os.path.join(HERE, "tiny_oracle.json"), "w") as f:
        json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
