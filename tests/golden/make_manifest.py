"""Rewrite tiny_manifest.json from the seeded generator."""
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from paper_2509_17863_amd import synth  # noqa: E402

with open(os.path.join(os.path.dirname(__file__), "tiny_manifest.json"), "w") as f:
    json.dump(synth.manifest(synth.make_workload("tiny")), f, indent=1)
