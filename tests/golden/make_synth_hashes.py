"""Writes synth_sha256.json: SHA-256 of the first 4096 fp32 draws of each workload's
Q/K/V streams. A regression pin of the input generator (it calls only ``synth``)."""
import hashlib
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from synth import WORKLOADS, normal, stream_key  # noqa: E402

out = {}
for name, spec in WORKLOADS.items():
    for t in range(3):
        out[f"{name}/{t}"] = hashlib.sha256(normal(stream_key(spec.config_id, t), 4096).numpy().tobytes()).hexdigest()
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "synth_sha256.json"), "w") as f:
    json.dump(out, f, indent=1, sort_keys=True)
