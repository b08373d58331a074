"""Per-block cutoff thresholds as a file (thresholds.json).

The cutoff t of each gated-MLP block is fixed once, from calibration data,
before the model is used (Section 4.1: the thresholds are set on the base
model and kept through fine-tuning), so it is an artefact to store with the
weights rather than something to recompute per run.  Each entry records the
block (layer index), the target sparsity k, t itself in hexadecimal (the
exact fp32 value the kernels compare against) and in decimal (for reading),
the number of calibration vectors, the seed they were drawn with and the
configuration name.  Loading parses the hexadecimal form, so a reloaded t is
bit-identical to the calibrated one.
"""
from __future__ import annotations

import json
import os
import struct
from typing import Iterable, Optional

FORMAT = "cats-thresholds/1"


def _f32(t: float) -> float:
    """t rounded to the fp32 value the library uses."""
    return struct.unpack("<f", struct.pack("<f", float(t)))[0]


def entry(layer: int, k: float, t: float, n_calib: int, seed: int, config: str) -> dict:
    t32 = _f32(t)
    if not (t32 >= 0.0):
        raise ValueError(f"threshold must be >= 0, got {t!r}")
    return {"layer": int(layer), "k": float(k), "t_hex": float.hex(t32), "t": repr(t32),
            "n_calib": int(n_calib), "seed": int(seed), "config": str(config)}


def save(path: str, entries: Iterable[dict]) -> None:
    """Write entries (from entry()) as thresholds.json (atomic replace)."""
    rows = list(entries)
    keys = set()
    for e in rows:
        key = (e["config"], e["layer"], e["k"])
        if key in keys:
            raise ValueError(f"duplicate threshold entry {key}")
        keys.add(key)
        if float.fromhex(e["t_hex"]) != _f32(float.fromhex(e["t_hex"])):
            raise ValueError(f"t_hex of {key} is not an fp32 value")
    doc = {"format": FORMAT, "thresholds": rows}
    tmp = path + ".tmp"
    with open(tmp, "w") as f:
        json.dump(doc, f, indent=1)
        f.write("\n")
    os.replace(tmp, path)


def load(path: str, config: Optional[str] = None) -> dict:
    """{(layer, k): t} from a thresholds file, t parsed from its hexadecimal
    form; entries of other configurations are skipped when config is given.
    Raises ValueError on a malformed file or a t that disagrees with its
    decimal form."""
    with open(path) as f:
        doc = json.load(f)
    if doc.get("format") != FORMAT:
        raise ValueError(f"{path}: not a {FORMAT} file")
    out = {}
    for e in doc["thresholds"]:
        if config is not None and e["config"] != config:
            continue
        t = float.fromhex(e["t_hex"])
        if t != _f32(t) or not (t >= 0.0):
            raise ValueError(f"{path}: t_hex {e['t_hex']} is not a non-negative fp32 value")
        if float(e["t"]) != t:
            raise ValueError(f"{path}: t {e['t']} disagrees with t_hex {e['t_hex']}")
        key = (int(e["layer"]), float(e["k"]))
        if key in out:
            raise ValueError(f"{path}: duplicate entry {key}")
        out[key] = t
    return out
