"""CPU checks of the synthetic workloads (they stand in for the paper's model activations).

Determinism and the calibration the generators promise, measured with the oracle
on a few heads of small layers: concentrated heads route VS with their mass in
the planted structure, i.i.d. diffuse heads route PE, and the structured PE heads
of the paper-like workload route PE with their top-50 blocks holding a fraction of
the mass (App. B reports 15% to 80% for real diffuse heads) and a PE selection
clearly below the ~90% of i.i.d. heads.
"""
import numpy as np
import torch

from oracle import crisp_oracle as O
from workloads import CONFIGS, GEN_VERSION, custom_config, head_specs, make_layer, structured_pe_config


def test_generator_is_deterministic_and_versioned():
    assert GEN_VERSION == "gen-v1"
    cfg = custom_config(2048, 4, 2, config_id=190)
    a = make_layer(cfg)
    b = make_layer(cfg, heads=[3])
    assert torch.equal(a[0][3], b[0][3]) and torch.equal(a[1][1], b[1][1]) and torch.equal(a[2][1], b[2][1])
    assert not b[0][0].any()


def test_structured_pe_heads_calibration():
    cfg = structured_pe_config(65536)
    specs = head_specs(cfg)
    kinds = [s.kind for s in specs]
    assert kinds.count("structured") == 13 and kinds.count("concentrated") == 19
    struct = [h for h in range(32) if kinds[h] == "structured"][:4]
    conc = [h for h in range(32) if kinds[h] == "concentrated"][:2]
    q, k, _, _ = make_layer(cfg, heads=struct + conc)
    op = O.Params()
    nb = cfg.seq_len // cfg.block
    for h in struct + conc:
        r = O.crisp_head(q[h].double().numpy(), k[h // cfg.group].double().numpy(), None, cfg.block, op,
                         attend=False)
        top50 = float(np.sort(r.p_v)[::-1][:50].sum())
        density = sum(len(s) for s in r.sets) / (nb * (nb + 1) / 2)
        if kinds[h] == "structured":
            assert r.route == O.ROUTE_PE and r.c_struct < 0.1, (h, r.c_struct)
            assert 0.15 <= top50 <= 0.8, (h, top50)
            assert density < 0.88, (h, density)
        else:
            assert r.route == O.ROUTE_VS and r.c_struct >= 0.25, (h, r.c_struct)


def test_existing_configs_keep_iid_diffuse_heads():
    for cid in (1, 2, 3):
        kinds = {s.kind for s in head_specs(CONFIGS[cid])}
        assert kinds == {"concentrated", "diffuse"}
