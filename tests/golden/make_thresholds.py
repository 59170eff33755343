"""Write tests/golden/thresholds.json: CATS thresholds (Eq. 3) of the five workloads.

Calls only the oracle (oracle.calibrate) on inputs from the seeded generators
(workloads.synth).  For each workload the calibration tokens run through the
dense stack and layer l's threshold is the k_l-percentile of the pooled
|SiLU(h_l W_gate_l)| values (Section 2, Eq. 3).

Usage:  python tests/golden/make_thresholds.py [config-name-prefix ...]
With no argument every workload is computed (the 32/36-layer stacks take a
few minutes each: 1024 tokens x 3 projections x L layers in float64).
Existing entries for other workloads are kept.
"""
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import calibrate  # noqa: E402
from workloads import CONFIGS, synth  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "thresholds.json")


class _Layers:
    """Sequence view of one weight matrix across layers, generated on demand."""

    def __init__(self, cfg, which, cache):
        self.cfg, self.which, self.cache = cfg, which, cache

    def __len__(self):
        return self.cfg.n_layers

    def __getitem__(self, l):
        if self.cache.get("layer") != l:
            c = self.cfg
            self.cache["layer"] = l
            self.cache["w"] = synth.layer_weights(c.seed, l, c.d, c.d_ff, c.dtype)
        return self.cache["w"][self.which]


def weights_digest(cfg) -> str:
    wg, wu, wd = synth.layer_weights(cfg.seed, 0, cfg.d, cfg.d_ff, cfg.dtype)
    h = hashlib.sha256()
    for w in (wg, wu, wd):
        h.update(np.ascontiguousarray(w).tobytes())
    return h.hexdigest()


def run(cfg):
    t0 = time.time()
    cache = {}
    lay = [_Layers(cfg, i, cache) for i in range(3)]
    ks = synth.k_levels(cfg)
    xcal = synth.calibration_x(cfg)
    ts, vals = calibrate.calibrate_stack(xcal, lay[0], lay[1], lay[2], ks, cfg.dtype,
                                         return_values=True)
    realized = [float(np.mean(v < np.float64(t))) for v, t in zip(vals, ts)]
    print(f"{cfg.name}: {time.time() - t0:.1f}s  t[0]={ts[0]:.6g}  "
          f"cal sparsity[0]={realized[0]:.4f}", flush=True)
    return dict(thresholds=[float(t) for t in ts], k=[float(k) for k in ks],
                n_cal=cfg.n_cal, cal_sparsity=realized, weights_sha256_layer0=weights_digest(cfg),
                source="oracle.calibrate.calibrate_stack (CATS percentile, Eq. 3)")


def main(argv):
    data = {}
    if os.path.exists(OUT):
        with open(OUT) as f:
            data = json.load(f)
    todo = [c for c in CONFIGS if not argv or any(c.name.startswith(a) for a in argv)]
    for cfg in todo:
        data[cfg.name] = run(cfg)
        with open(OUT, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)
            f.write("\n")


if __name__ == "__main__":
    main(sys.argv[1:])
