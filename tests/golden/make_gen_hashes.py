"""Writes gen_hashes.json: SHA-256 of the generator's traces (regression pins
of the seeded input module; no simulator is involved).

    python tests/golden/make_gen_hashes.py
"""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

from test_gen import _sha, golden_traces  # noqa: E402

out = {}
for name, t, m in golden_traces():
    out[name] = {"sha256": _sha(t, m), "n": int(len(t))}
with open(os.path.join(HERE, "gen_hashes.json"), "w") as f:
    json.dump(out, f, indent=1, sort_keys=True)
print(json.dumps(out, indent=1))
