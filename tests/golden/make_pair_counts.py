"""Writes pair_counts.json: visible (query, key) pairs per head for every workload.

Counts come from the CPU oracle's explicit visibility mask (built in row blocks), so
they follow the visibility rule of Avatar V §1 (contributions), §2.1 and §4.3, with one
reference latent frame per self-attention group (and, for varlen_window, the temporal window
of §2.4; for varlen_tokens, the reference token masks of that workload). Run from the repository root:
    python tests/golden/make_pair_counts.py
"""
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from sra_inputs import SWEEP_POINTS, workload  # noqa: E402

names = ["tiny", "480p"] + [f"sweep_{n}" for n in SWEEP_POINTS] + ["720p", "varlen", "varlen_window", "varlen_tokens"]
out = {"_source": "oracle.pair_counts over the explicit mask; per head, summed over samples"}
for name in names:
    w = workload(name)
    t0 = time.time()
    gp, rp = oracle.pair_counts(w.samples, block_rows=4096)
    out[name] = {"gen_pairs": gp, "ref_pairs": rp, "heads": w.heads, "head_dim": w.head_dim}
    print(name, gp, rp, f"{time.time() - t0:.1f}s", flush=True)
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "pair_counts.json"), "w") as f:
    json.dump(out, f, indent=1)
