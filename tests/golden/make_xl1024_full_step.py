"""Write the oracle's full-depth DiT-XL/2 1024px full-image step on sampled
token rows (tests/golden/xl1024_full_step_rows.npz).

The unpartitioned step (every token row in the band, nothing stale) at the
first step after a 10-step warm-up of the 50-step grid (t 780 -> 760), with
the seeded weights, latent and labels (seed 0).  Only the oracle and the
seeded input generators run here; a full-depth oracle step over 4096 tokens
takes minutes on the host, so the GPU test reads the stored rows instead of
recomputing them.

    python tests/golden/make_xl1024_full_step.py
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import blob as oblob  # noqa: E402
from oracle import dit  # noqa: E402
from seeded_inputs import configs, generate  # noqa: E402

OUT = os.path.join(HERE, "xl1024_full_step_rows.npz")
# token rows: both ends of the grid, the rows on either side of its middle,
# and a few in between (128-query tiles hold two token rows each)
ROWS = [0, 1, 17, 31, 32, 47, 62, 63]


def main():
    cfg = configs.get("dit_xl2_1024")
    t, tp = configs.headline_timestep_pair(cfg)
    hdr, params = oblob.read_blob(generate.make_weight_blob(cfg, 0), np.float32)
    x = generate.make_latent(cfg, 0)
    labels = generate.make_labels(cfg, 0)
    t0 = time.time()
    r = dit.full_step(hdr, params, x, t, tp, labels, cfg.cfg_scale, dtype=np.float32,
                      out_rows=ROWS)
    np.savez_compressed(OUT, rows=np.array(ROWS, dtype=np.int32),
                        eps=r["eps"].astype(np.float32), x_out=r["x_out"].astype(np.float32),
                        t=np.int32(t), t_prev=np.int32(tp), labels=np.asarray(labels, np.int32),
                        seed=np.int32(0), n_blocks=np.int32(cfg.n_blocks))
    print(f"wrote {OUT} ({time.time() - t0:.0f} s of oracle)")


if __name__ == "__main__":
    main()
