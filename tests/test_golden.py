"""Generator and oracle drift: the realised per-head statistics of small seeded layers
(written by tests/golden/make_manifests.py, which calls only the oracle and the
generator) must come out the same when recomputed.  Routes, PE cutoffs, VS block
lists, selection sizes and pair counts are compared exactly; the float64 masses,
block scores and output statistics to 1e-9 relative (BLAS summation order may differ
between machines).  A VS direction whose residual is below float32 resolution (E3) or
whose blocks sit within the floor band (E1/E2) may select differently under another
summation order: there the lists are compared outside those blocks, and the sizes and
pair counts that follow from them are not compared."""
import importlib.util
import json
import os

import pytest

from tests import parity as PR

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")


def _maker():
    spec = importlib.util.spec_from_file_location("make_manifests", os.path.join(GOLDEN, "make_manifests.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _close(a, b):
    return a == pytest.approx(b, rel=1e-9, abs=1e-12)


def test_manifests_are_reproduced():
    with open(os.path.join(GOLDEN, "manifests.json")) as f:
        stored = json.load(f)
    fresh = _maker().build()
    assert sorted(stored) == sorted(fresh)
    for name, rec in stored.items():
        new = fresh[name]
        for key in ("generator", "layer", "seq_len", "block", "alpha"):
            assert rec[key] == new[key], (name, key)
        assert sorted(rec["heads"]) == sorted(new["heads"]), name
        k_min = -(-1024 // rec["block"])
        for h, st in rec["heads"].items():
            nw = new["heads"][h]
            assert sorted(st) == sorted(nw), (name, h)
            exact_lists = True
            for d in ("v", "s") if st["route"] == "VS" else ():
                degenerate, ex = PR.vs_direction_exempt(st["p_" + d], rec["alpha"], k_min)
                diff = set(st["S_" + d]) ^ set(nw["S_" + d])
                assert degenerate or not (diff - ex), (name, h, d, sorted(diff - ex))
                exact_lists &= not diff
            for key, val in st.items():
                if key in ("S_v", "S_s") or (not exact_lists and key in ("k_v", "k_s", "pairs", "density")):
                    continue
                if isinstance(val, list):
                    assert len(nw[key]) == len(val) and all(_close(a, b) for a, b in zip(nw[key], val)), (name, h, key)
                elif isinstance(val, float):
                    assert _close(nw[key], val), (name, h, key, nw[key], val)
                else:
                    assert nw[key] == val, (name, h, key, nw[key], val)


def test_manifests_show_the_planted_structure():
    """What the generator promises, read off the stored file: concentrated heads route VS
    with most of their proxy mass on the sink tag, i.i.d. diffuse heads route PE with a
    near-uniform proxy (C_struct about (w_sink + w_local) / n plus the proxy's own block)
    and select about 90% of the causal pairs, and the three adversarial heads behave as
    designed (under sink collapse the vertical residual lies below float32 resolution, a
    degenerate direction; the flat head selects like a diffuse one; the head at the floor
    routes VS with about half of its mass in the sinks and keeps k_min vertical blocks)."""
    with open(os.path.join(GOLDEN, "manifests.json")) as f:
        m = json.load(f)
    tiny = m["tiny-4k"]["heads"]
    assert tiny["0"]["route"] == "VS" and tiny["0"]["sink_mass"] > 0.95
    assert tiny["1"]["route"] == "PE" and tiny["1"]["c_struct"] < 0.1 and 0.85 < tiny["1"]["density"] < 0.95
    llama = m["llama3-8b-32k-heads0-3"]["heads"]
    for h, r in llama.items():
        if r["route"] == "VS":
            assert r["c_struct"] >= 0.25 and r["density"] < 0.2, h
        else:
            assert r["c_struct"] <= 0.15 and 0.85 < r["density"] < 0.95, h
    adv = m["stress-64k-a1-b128-adversarial"]["heads"]
    assert adv["0"]["route"] == "VS" and adv["0"]["sink_mass"] > 1 - 1e-9 and adv["0"]["residual_v"] < 2 ** -20
    assert adv["1"]["route"] == "PE" and 0.85 < adv["1"]["density"] < 0.95
    assert adv["2"]["route"] == "VS" and 0.45 < adv["2"]["sink_mass"] < 0.55
