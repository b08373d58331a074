"""thresholds.json: per-block cutoffs saved with their exact fp32 bits and
reloaded bit for bit (host logic only)."""
import json
import struct

import pytest

from paper_2404_08763_amd import thresholds as T


def _bits(t):
    return struct.pack("<f", t)


def test_round_trip_is_bit_exact(tmp_path):
    ts = [0.2718903422355652, 1.2155812978744507, 3.569502830505371, 0.0, 1e-30, float("inf")]
    rows = [T.entry(0, k, t, 2048, 7, "C2") for k, t in zip((0.5, 0.7, 0.9, 0.0, 0.1, 1.0), ts)]
    rows.append(T.entry(3, 0.5, 0.31, 1024, 7, "C4"))
    p = tmp_path / "thresholds.json"
    T.save(str(p), rows)
    back = T.load(str(p), config="C2")
    assert len(back) == 6
    for k, t in zip((0.5, 0.7, 0.9, 0.0, 0.1, 1.0), ts):
        assert _bits(back[(0, k)]) == _bits(t)
    assert set(T.load(str(p))) == set(back) | {(3, 0.5)}
    doc = json.loads(p.read_text())
    assert doc["format"] == T.FORMAT
    assert doc["thresholds"][0]["t_hex"] == float.hex(struct.unpack("<f", _bits(ts[0]))[0])
    assert doc["thresholds"][0]["n_calib"] == 2048 and doc["thresholds"][0]["seed"] == 7


def test_t_is_rounded_to_fp32():
    e = T.entry(0, 0.5, 0.1, 8, 7, "C1")
    assert float.fromhex(e["t_hex"]) == struct.unpack("<f", struct.pack("<f", 0.1))[0]


def test_rejects_bad_files(tmp_path):
    p = tmp_path / "t.json"
    with pytest.raises(ValueError):
        T.entry(0, 0.5, -1.0, 8, 7, "C1")
    with pytest.raises(ValueError):
        T.save(str(p), [T.entry(0, 0.5, 0.1, 8, 7, "C1"), T.entry(0, 0.5, 0.2, 8, 7, "C1")])
    p.write_text(json.dumps({"format": "other", "thresholds": []}))
    with pytest.raises(ValueError):
        T.load(str(p))
    good = T.entry(0, 0.5, 0.25, 8, 7, "C1")
    bad = dict(good, t="0.5")
    p.write_text(json.dumps({"format": T.FORMAT, "thresholds": [bad]}))
    with pytest.raises(ValueError):
        T.load(str(p))
    bad = dict(good, t_hex=float.hex(0.1))  # not an fp32 value
    p.write_text(json.dumps({"format": T.FORMAT, "thresholds": [bad]}))
    with pytest.raises(ValueError):
        T.load(str(p))
