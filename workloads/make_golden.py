"""Write workloads/golden.json: SHA-256 of every array of every workload.

These checksums pin the input generator only (same seed -> same bytes on any
machine); they say nothing about search results."""
import hashlib
import json
import os

from workloads import configs


def digests() -> dict:
    out = {}
    for cfg in configs.CONFIGS:
        d = configs.make(cfg)
        out[cfg.name] = {k: hashlib.sha256(v.tobytes()).hexdigest() for k, v in d.items() if hasattr(v, "tobytes")}
    return out


if __name__ == "__main__":
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden.json")
    with open(path, "w") as f:
        json.dump(digests(), f, indent=1, sort_keys=True)
    print("wrote", path)
