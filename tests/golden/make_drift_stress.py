"""Write the oracle's drift-stress reference for sequence 0 (test infrastructure).

Calls only the CPU oracle (oracle/) and the seeded input generators; nothing here comes
from the GPU path.  The GPU drift-stress test loads the result instead of recomputing it
(about ten minutes of float64 CPU work at the large-v3 shape).

Workload: the drift-stress decode loop (batch 32, k 8, 1500 frames, large-v3 shape);
sequence 0 from the start token at position 0.  Stored:
  y        the oracle's greedy tokens at positions 1 .. N + k + 2 (autoregressive)
  margins  their top-1 minus top-2 margins (float32-rounded logits)
  accepts  per speculative round, the accepted length with drafts planted by
           synth.plant_drift on y (misaligned by +-1 after each anchor)
  tokens   the tokens those rounds emit (the first N)

Run: python tests/golden/make_drift_stress.py   (writes drift_stress_seq0.json beside it)
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import decoder as od  # noqa: E402
from paper_2608_12703_amd import synth  # noqa: E402
from paper_2608_12703_amd.configs import CONFIGS, MAX_POS, SOT_TOKEN  # noqa: E402

N_TOKENS = 128
SEQ = 0


def main():
    cfg = CONFIGS["drift_stress"]
    t0 = time.time()
    model = od.Model(cfg, synth.make_params(cfg))
    cross = od.cross_kv(model, synth.make_encoder(cfg, SEQ, cfg.frames))
    print(f"encoder K/V {time.time() - t0:.0f} s", flush=True)
    n_ar = N_TOKENS + cfg.k + 2
    y, margins, st = [], [], od.new_state(model, cross, SOT_TOKEN)
    for i in range(n_ar):
        r = od.ar_step(model, st)
        y.append(int(r.emitted[0]))
        margins.append(float(r.margins[0]))
        st = r.state
        if i % 16 == 0:
            print(f"autoregressive {i}/{n_ar} ({time.time() - t0:.0f} s)", flush=True)
    ys = np.array([SOT_TOKEN] + y, np.int64)
    plan = synth.make_drift_plan(cfg, SEQ)
    st, n, accepts, tokens = od.new_state(model, cross, SOT_TOKEN), 0, [], []
    while len(tokens) < N_TOKENS:
        k = min(cfg.k, MAX_POS - 1 - n)
        r = od.verify(model, st, synth.plant_drift(ys, n, k, plan))
        accepts.append(int(r.accepted))
        tokens += [int(t) for t in r.emitted]
        n += r.accepted + 1
        st = r.state
    print(f"{len(accepts)} rounds, accepts {accepts} ({time.time() - t0:.0f} s)", flush=True)
    out = {"workload": "drift_stress", "sequence": SEQ, "n_tokens": N_TOKENS,
           "y": y, "margins": margins, "accepts": accepts, "tokens": tokens[:N_TOKENS]}
    with open(os.path.join(HERE, "drift_stress_seq0.json"), "w") as fh:
        json.dump(out, fh)
        fh.write("\n")


if __name__ == "__main__":
    main()
