"""Write tests/golden/calib/<workload>.npz: static step sizes and the mean-correction term of
each named workload, calibrated by the CPU oracle on the calibration draw (stream s = 2) of the
seeded generator.  Only the oracle computes these values.

    python tests/golden/make_calibration.py [workload ...]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import calibrate  # noqa: E402
from paper_2608_21952_amd import synth  # noqa: E402


def main(names):
    os.makedirs(os.path.join(HERE, "calib"), exist_ok=True)
    for name in names:
        cfg = synth.CONFIGS[name]
        t = time.time()
        d = synth.draw(cfg, 2)
        sc = calibrate.calibrate(d["x"], d["dt_raw"], d["A"], d["B"], d["C"], d["D"],
                                 chunk=cfg.chunk, xs_per_head=cfg.xs_per_head)
        np.savez(os.path.join(HERE, "calib", name + ".npz"), **sc)
        print(f"{name}: {time.time() - t:.1f} s", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:] or synth.CONFIG_ORDER)
