import json
import os

_HERE = os.path.dirname(os.path.abspath(__file__))


def load(name: str) -> dict:
    """Parse a `key = <json>` fixture file (lines starting with # are comments)."""
    out = {}
    with open(os.path.join(_HERE, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split("=", 1)
            out[k.strip()] = json.loads(v.strip())
    return out
