"""Writes tests/golden/manifests.json: the realised per-head statistics of small seeded
layers, computed by the oracle alone (this script imports only oracle/ and workloads/).

Each record names the generator version and the layer, and per head gives the quantities
that decide the path: C_struct (the structural mass of Sec. 3.2), the proxy's sink mass
(keys 0..3, the planted sink tag), the route (Alg. 2), the VS selections' sizes k_v and
k_s and, for VS heads, the block scores p_v, p_s and the selected blocks S_v, S_s of
each direction (Alg. 3 with the noise floor of Sec. 4.3), the PE cutoff K* (Alg. 4), the
executed block pairs and their density over the causal pairs, and, where the attention
is run, the mean and the largest magnitude of the head's output (Eq. 1 over the
selected blocks).  Inputs are drawn by the
generator on the CPU (the generator's stream depends on the device), only the listed
heads being filled.  A later change of the generator or of the oracle's arithmetic shows
up as a difference against this file.

Run from the repository root:  python tests/golden/make_manifests.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import crisp_oracle as O  # noqa: E402
from workloads import CONFIGS, GEN_VERSION, make_layer, stress_config  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "manifests.json")

# (name, layer, heads, run the attention)
LAYERS = [
    ("tiny-4k", CONFIGS[0], [0, 1], True),
    ("llama3-8b-32k-heads0-3", CONFIGS[1], [0, 1, 2, 3], False),
    ("stress-64k-a1-b128-adversarial", stress_config(1.0, 128), [0, 1, 2], False),
]


def head_record(q, k, v, block, params, attend):
    n = q.shape[0]
    nb = O.n_blocks(n, block)
    r = O.crisp_head(q, k, v, block, params, attend=attend)
    ahat = O.proxy_attention(q, k, block, params.scale(q.shape[1]))
    pairs = sum(len(s) for s in r.sets)
    rec = {
        "c_struct": float(r.c_struct),
        "sink_mass": float(ahat[:, :4].sum() / ahat.shape[0]),
        "route": "VS" if r.route == O.ROUTE_VS else "PE",
        "k_v": len(r.S_v),
        "k_s": len(r.S_s),
        "pe_k_star": None if r.pe_info is None else int(r.pe_info["kstar"]),
        # VS residual r_d = 1 - p_d[0] - p_d[N_b - 1] per direction (Alg. 3); below float32
        # resolution next to 1 the floor, and with it the VS selection, is degenerate
        "residual_v": float(max(1.0 - r.p_v[0] - r.p_v[nb - 1], 0.0)),
        "residual_s": float(max(1.0 - r.p_s[0] - r.p_s[nb - 1], 0.0)),
        "pairs": int(pairs),
        "density": pairs / (nb * (nb + 1) / 2),
    }
    if r.route == O.ROUTE_VS:
        rec["p_v"] = [float(x) for x in r.p_v]
        rec["p_s"] = [float(x) for x in r.p_s]
        rec["S_v"] = [int(J) for J in r.S_v]
        rec["S_s"] = [int(J) for J in r.S_s]
    if attend:
        rec["out_mean"] = float(r.out.mean())
        rec["out_max_abs"] = float(np.abs(r.out).max())
    return rec


def manifest(name, cfg, heads, attend):
    q, k, v, _ = make_layer(cfg, heads=heads)
    params = O.Params(alpha=cfg.alpha)
    out = {}
    for h in heads:
        g = h // cfg.group
        out[str(h)] = head_record(q[h].double().numpy(), k[g].double().numpy(),
                                  v[g].double().numpy() if attend else None, cfg.block, params, attend)
    return {"generator": GEN_VERSION, "layer": cfg.name, "seq_len": cfg.seq_len, "block": cfg.block,
            "alpha": cfg.alpha, "heads": out}


def build():
    return {name: manifest(name, cfg, heads, attend) for name, cfg, heads, attend in LAYERS}


if __name__ == "__main__":
    with open(OUT, "w") as f:
        json.dump(build(), f, indent=1, sort_keys=True)
        f.write("\n")
    print("wrote", OUT)
