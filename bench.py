"""CRISP prefill attention benchmark on one MI355X.

One step = one full CRISP pass over one attention layer (estimate, route and
select, block-sparse attention) on seeded synthetic bf16 inputs already resident
in HBM.  The FlexPrefill comparator of App. A (JSD pattern search, gamma VS
selection) and the two ablation mixes run on the same kernels and layers and
are reported under "comparators".  The headline workload is the Llama-3-8B GQA layer at 128k tokens
(32 query heads, 8 KV heads, d = 128, B = 128); the 512k Qwen2-7B-like layer is
reported alongside.  The dense causal baseline is the same attention kernel with
every causal block listed.

Prints one JSON line (see the `record` dict below).  Timing uses HIP events on
the stream the kernels run on (torch's current stream).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import statistics
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (published)
HBM_PEAK_GBS = 8000.0            # MI355X HBM3E (published)
# VALU issue: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane slots per second (the published
# 157.3 TFLOP/s fp32 vector rate counts an FMA as two FLOPs and packs two lanes' worth per slot)
VALU_LANE_SLOTS_PER_S = 256 * 4 * 16 * 2.4e9
# per proxy score: exp2, which issues at half the full rate on this chip (measured_peaks:
# 9.0 SIMD cycles per wave-wide v_exp_f32 against 3.75 for v_fma_f32), so 2 slots, + fma + add
VALU_SLOTS_PER_PROXY_SCORE = 4.0
METRIC = "CRISP prefill attention ms/layer at 128k & 512k; speedup vs dense HIP attention"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--skip-512k", action="store_true")
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--steps-512k", type=int, default=7)
    ap.add_argument("--skip-sweep", action="store_true",
                    help="skip the length sweep 2k..512k on the paper-like structured-PE workload "
                         "(CRISP, dense and FlexPrefill; locates the crossover with dense)")
    ap.add_argument("--skip-configs", action="store_true",
                    help="skip the per-config records of the 4k tiny layer, the 32k Llama layer and the six "
                         "alpha x B cells of the 64k selection-stress layer")
    ap.add_argument("--skip-peaks", action="store_true", help="skip the MFMA and copy peak microbenchmarks")
    ap.add_argument("--skip-comparators", action="store_true",
                    help="skip the FlexPrefill comparator, ablation and noise-floor variant timings")
    ap.add_argument("--config", type=int, default=2, help="headline config id (2 = 128k Llama GQA layer)")
    ap.add_argument("--structured", type=int, default=0, metavar="N",
                    help="headline layer: the structured-PE layer of N tokens (Llama-3-8B shape) instead of "
                         "--config (for profiling the length sweep's layers)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy, the reference for rocprofv3 byte counters")
    ap.add_argument("--summarize", metavar="ROCPROF_DIR",
                    help="summarize rocprofv3 output under ROCPROF_DIR (one sub-folder per rocprofv3 run) "
                         "into profiles/ and exit (no GPU)")
    ap.add_argument("--label", default="crisp_kernels_llama3_8b_128k", help="file stem for --summarize")
    ap.add_argument("--command", action="append", default=[],
                    help="a profiling command, recorded by --summarize (repeatable)")
    ap.add_argument("--clock-power", action="store_true",
                    help="sample socket power and GFX clock (amd-smi) under several loads on the 128k layer, "
                         "print one JSON line and exit")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def src_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def time_events(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t0 = time.perf_counter()
    for a, b in evs:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    ms = sorted(a.elapsed_time(b) for a, b in evs)
    pct = lambda f: ms[min(len(ms) - 1, int(round(f * (len(ms) - 1))))]
    return {"median": ms[len(ms) // 2], "mean": sum(ms) / len(ms), "min": ms[0], "max": ms[-1],
            "p10": pct(0.1), "p90": pct(0.9), "wall_per_step": wall}


def layer_measure(cfg, steps, warmup, label):
    """Times CRISP (whole path and per stage) and the dense baseline on one layer."""
    import torch
    from paper_2609_01925_amd import crisp as C
    from workloads import make_layer

    dev = "cuda:0"
    t = time.perf_counter()
    q, k, v, specs = make_layer(cfg, device=dev)
    torch.cuda.synchronize()
    log(f"{label}: generated {cfg.name} in {time.perf_counter() - t:.1f}s")
    block = cfg.block
    params = C.make_params(alpha=cfg.alpha)
    sh = C.shape_of(q, k, block)
    ws = C.workspace(sh, dev, prefill=True)
    o = torch.empty_like(q)

    # one checked pass to get the routes and block lists (outside the timed region)
    o_, route, rp, ci = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
    torch.cuda.synchronize()
    nb = C.n_blocks(cfg.seq_len, block)
    pairs_per_head = rp[:, nb].double().cpu()
    executed_pairs = float(pairs_per_head.sum())
    dense_pairs = cfg.n_q_heads * nb * (nb + 1) / 2
    route_c = route.cpu()
    n_vs = int((route_c == 0).sum())
    del o_

    crisp = time_events(lambda: C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o), steps, warmup)
    log(f"{label}: CRISP {crisp['wall_per_step']:.3f} ms/layer")

    # per-stage timing (same stream, same buffers)
    cs, pv, ps = C.crisp_estimate(q, k, params, block)
    wss = C.workspace(sh, dev)
    est = time_events(lambda: C.crisp_estimate(q, k, params, block, ws=wss), steps, warmup)
    sel = time_events(lambda: C.crisp_route_select(q, k, cs, pv, ps, params, block, want_mask=False, ws=wss),
                      steps, warmup)
    att = time_events(lambda: C.crisp_sparse_attn(q, k, v, rp, ci, block, out=o), steps, warmup)
    dense = time_events(lambda: C.crisp_dense_attn(q, k, v, block, out=o), steps, warmup)
    log(f"{label}: stages est {est['mean']:.3f} sel {sel['mean']:.3f} attn {att['mean']:.3f}; "
        f"dense {dense['wall_per_step']:.3f} ms")

    d = 128
    # algorithmic HBM bytes: the estimator reads each KV head's K once (one pass); the
    # selection pools Q of the PE heads and K of their groups, writes the pooled scores
    # A~ once, then reads/writes them in the softmax, reads them in the three radix passes
    # and the two CSR passes (32 bytes per causal pair per PE head), and writes the lists
    est_gbs = cfg.n_kv_heads * cfg.seq_len * d * 2.0 / (est["mean"] * 1e-3) / 1e9
    pe_heads = [h for h in range(cfg.n_q_heads) if int(route_c[h]) == 1]
    pe_groups = len({h // cfg.group for h in pe_heads})
    sel_bytes = ((len(pe_heads) + pe_groups) * cfg.seq_len * d * 2.0 + 32.0 * nb * (nb + 1) / 2 * len(pe_heads)
                 + 4.0 * executed_pairs)
    sel_gbs = sel_bytes / (sel["mean"] * 1e-3) / 1e9
    pair_flop = 4.0 * block * block * d
    attn_flop = executed_pairs * pair_flop
    dense_flop_exec = dense_pairs * pair_flop
    dense_useful = 2.0 * cfg.n_q_heads * cfg.seq_len * cfg.seq_len * d   # causal half: 4 n^2 d / 2
    est_scores = cfg.n_q_heads * min(block, cfg.seq_len) * cfg.seq_len
    est_valu_ms = est_scores * VALU_SLOTS_PER_PROXY_SCORE / VALU_LANE_SLOTS_PER_S * 1e3
    res = {
        "workload": cfg.name, "seq_len": cfg.seq_len, "n_q_heads": cfg.n_q_heads, "n_kv_heads": cfg.n_kv_heads,
        "block": block, "alpha": cfg.alpha,
        # exactly `steps` prefills between two synchronisations, per step; the per-step
        # event times give the median and spread
        "ms_per_layer": crisp["wall_per_step"], "ms_median": crisp["median"], "ms_p10": crisp["p10"],
        "ms_p90": crisp["p90"], "ms_p_min": crisp["min"], "ms_p_max": crisp["max"],
        "dense_ms_per_layer": dense["wall_per_step"], "dense_ms_median": dense["median"],
        "speedup_vs_dense": dense["wall_per_step"] / crisp["wall_per_step"],
        "stage_ms": {"estimate": est["mean"], "route_select": sel["mean"], "sparse_attn": att["mean"]},
        "routes": {"vs": n_vs, "pe": cfg.n_q_heads - n_vs},
        "executed_pairs": executed_pairs, "density": executed_pairs / dense_pairs,
        "density_by_route": {name: float(pairs_per_head[route_c == rt].sum()) / max(1, int((route_c == rt).sum()))
                             / (nb * (nb + 1) / 2) for name, rt in (("vs", 0), ("pe", 1))},
        "sparse_attn_tflops_executed": attn_flop / (att["mean"] * 1e-3) / 1e12,
        "sparse_attn_mfma_frac": attn_flop / (att["mean"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
        "dense_tflops_executed": dense_flop_exec / (dense["mean"] * 1e-3) / 1e12,
        "dense_mfma_frac": dense_flop_exec / (dense["mean"] * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS,
        "effective_tflops_dense_equiv": dense_useful / (crisp["wall_per_step"] * 1e-3) / 1e12,
        "estimate_hbm_gbs": est_gbs, "estimate_hbm_frac": est_gbs / HBM_PEAK_GBS,
        # the estimator's proxy scores on MFMA: 2 b n d FLOP per query head (b = block)
        "estimate_tflops": 2.0 * cfg.n_q_heads * block * cfg.seq_len * d / (est["mean"] * 1e-3) / 1e12,
        "estimate_mfma_frac": 2.0 * cfg.n_q_heads * block * cfg.seq_len * d / (est["mean"] * 1e-3) / 1e12
        / MFMA_BF16_PEAK_TFLOPS,
        "select_hbm_gbs": sel_gbs, "select_hbm_frac": sel_gbs / HBM_PEAK_GBS,
        # the estimator's VALU floor: per proxy score one exp2 (half the full VALU rate, so 2
        # lane slots) and two full-rate ops (scale-and-subtract, sum)
        "estimate_valu_bound_ms": est_valu_ms,
        "estimate_valu_frac": est_valu_ms / est["mean"],
    }
    res["_attn_launch_ms"] = att["mean"]
    res["_attn_flop"] = attn_flop
    res["_tensors"] = (q, k, v, specs, route_c, rp.cpu(), ci.cpu(), pairs_per_head)
    return res


def add_measured_fracs(res, peaks):
    """Adds each roofline fraction against the rates measured on this GPU beside the one
    against the published peak."""
    if not peaks:
        return
    m, c = peaks["mfma_bf16_tflops"], peaks["copy_gbs"]
    res["sparse_attn_frac_of_measured_mfma"] = res["sparse_attn_tflops_executed"] / m
    res["dense_frac_of_measured_mfma"] = res["dense_tflops_executed"] / m
    res["estimate_frac_of_measured_mfma"] = res["estimate_tflops"] / m
    res["estimate_frac_of_measured_copy"] = res["estimate_hbm_gbs"] / c
    res["select_frac_of_measured_copy"] = res["select_hbm_gbs"] / c
    # the same VALU floor from this GPU's measured issue costs: per 64 scores one exp2 and
    # two FMA-class instructions on one SIMD, 1024 SIMDs at 2.4 GHz
    v = peaks.get("valu_cycles_per_wave_instruction")
    if v and res.get("estimate_valu_bound_ms"):
        per64 = v["exp2_f32"] + 2.0 * v["fma_f32"]
        scores = res["estimate_valu_bound_ms"] * 1e-3 * VALU_LANE_SLOTS_PER_S / VALU_SLOTS_PER_PROXY_SCORE
        ms = scores / 64.0 * per64 / (1024 * 2.4e9) * 1e3
        res["estimate_valu_bound_ms_measured_issue"] = ms
        res["estimate_valu_frac_measured_issue"] = ms / res["stage_ms"]["estimate"]


def comparator_measure(cfg, res, steps, warmup, label, mixes=True):
    """The FlexPrefill comparator of App. A on the same kernels (JSD pattern search and gamma
    VS selection), and the two ablation mixes, timed end to end like CRISP on the same layer."""
    import torch
    from paper_2609_01925_amd import crisp as C

    q, k, v = res["_tensors"][:3]
    block = cfg.block
    route_cs = res["_tensors"][4]
    nb = C.n_blocks(cfg.seq_len, block)
    dense_pairs = cfg.n_q_heads * nb * (nb + 1) / 2
    sh = C.shape_of(q, k, block)
    ws = C.workspace(sh, q.device, prefill=True)
    o = torch.empty_like(q)
    modes = [("flexprefill", C.flexprefill_params(alpha=cfg.alpha))]
    if mixes:
        modes += [("cstruct_route_gamma_vs", C.make_params(alpha=cfg.alpha, vs_mode=C.VS_GAMMA)),
                  ("jsd_route_floor_vs", C.make_params(alpha=cfg.alpha, route_mode=C.ROUTE_BY_JSD))]
    out = {}
    for name, params in modes:
        _, route, rp, _ = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
        torch.cuda.synchronize()
        pairs = float(rp[:, nb].double().sum())
        t = time_events(lambda: C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o), steps, warmup)
        rc = route.cpu()
        n_vs = int((rc == 0).sum())
        rec = {"ms_per_layer": t["wall_per_step"], "speedup_vs_dense": res["dense_ms_per_layer"] / t["wall_per_step"],
               "crisp_speedup_vs_this": t["wall_per_step"] / res["ms_per_layer"],
               "routes": {"vs": n_vs, "pe": cfg.n_q_heads - n_vs}, "executed_pairs": pairs,
               "density": pairs / dense_pairs,
               "route_agreement_with_cstruct": float((rc == route_cs).double().mean())}
        if params.route_mode == C.ROUTE_BY_JSD:
            cs, pv, ps = C.crisp_estimate(q, k, params, block)
            wsj = C.workspace(sh, q.device)
            rec["pattern_search_ms"] = time_events(lambda: C.crisp_jsd(q, k, pv, params, block, ws=wsj),
                                                   steps, warmup)["mean"]
        out[name] = rec
        log(f"{label}: {name} {t['wall_per_step']:.3f} ms/layer, density {rec['density']:.3f}, "
            f"routes VS {n_vs}, agreement {rec['route_agreement_with_cstruct']:.2f}")
    return out


def floor_variants_measure(cfg, res, steps, warmup, label):
    """The noise-floor variants (App. H and the alpha sweep): the median floor and alpha in
    {0.75, 1.25, 1.5}, each timed end to end on the same layer with its executed density."""
    import torch
    from paper_2609_01925_amd import crisp as C

    q, k, v = res["_tensors"][:3]
    block = cfg.block
    nb = C.n_blocks(cfg.seq_len, block)
    dense_pairs = cfg.n_q_heads * nb * (nb + 1) / 2
    ws = C.workspace(C.shape_of(q, k, block), q.device, prefill=True)
    o = torch.empty_like(q)
    out = {}
    for name, params in (("median_alpha1.0", C.make_params(floor_mode=C.FLOOR_MEDIAN)),
                         ("mean_alpha0.75", C.make_params(alpha=0.75)),
                         ("mean_alpha1.25", C.make_params(alpha=1.25)),
                         ("mean_alpha1.5", C.make_params(alpha=1.5))):
        _, _, rp, _ = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
        torch.cuda.synchronize()
        pairs = float(rp[:, nb].double().sum())
        t = time_events(lambda: C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o), steps, warmup)
        out[name] = {"ms_per_layer": t["wall_per_step"], "density": pairs / dense_pairs, "executed_pairs": pairs}
        log(f"{label}: floor {name} {t['wall_per_step']:.3f} ms/layer, density {pairs / dense_pairs:.4f}")
    return out


def pe_sweep_measure(peaks=None):
    """Length sweep on the structured-PE workload (the regime of the paper's latency table):
    CRISP, the dense baseline and the FlexPrefill comparator at each length, and the shortest
    length at which CRISP beats dense (the context-length gate's threshold)."""
    import torch
    from workloads import PE_SWEEP_LENGTHS, structured_pe_config

    rows = []
    for n in sorted(PE_SWEEP_LENGTHS):
        cfg = structured_pe_config(n)
        steps, warmup = (10, 3) if n <= 131072 else (3, 1)
        res = layer_measure(cfg, steps, warmup, f"sweep {n // 1024}k")
        fp = comparator_measure(cfg, res, steps, warmup, f"sweep {n // 1024}k", mixes=False)["flexprefill"]
        rows.append({"seq_len": n, "workload": cfg.name, "crisp_ms": res["ms_per_layer"],
                     "dense_ms": res["dense_ms_per_layer"], "speedup_vs_dense": res["speedup_vs_dense"],
                     "crisp_ms_event_median": res["ms_median"], "dense_ms_event_median": res["dense_ms_median"],
                     "density": res["density"], "routes": res["routes"], "stage_ms": res["stage_ms"],
                     "flexprefill_ms": fp["ms_per_layer"], "flexprefill_density": fp["density"],
                     "crisp_speedup_vs_flexprefill": fp["crisp_speedup_vs_this"],
                     "sparse_attn_mfma_frac": res["sparse_attn_mfma_frac"],
                     "sparse_attn_frac_of_measured_mfma": (res["sparse_attn_tflops_executed"] / peaks["mfma_bf16_tflops"]
                                                           if peaks else None)})
        del res
        torch.cuda.empty_cache()
    faster = [r["seq_len"] for r in rows if r["crisp_ms"] < r["dense_ms"]]
    faster_ev = [r["seq_len"] for r in rows if r["crisp_ms_event_median"] < r["dense_ms_event_median"]]
    return {"rows": rows, "crisp_beats_dense_from": min(faster) if faster else None,
            "crisp_beats_dense_from_event_median": min(faster_ev) if faster_ev else None}


def cpu_baseline(cfg, res, budget_s=25.0, full=False):
    """The oracle, as it stands, on the host cores: estimate + route/select for every head
    (or as many as fit 60% of the budget, scaled to all heads), attention on a sample of
    (head, query block) units, extrapolated to ms per layer by the oracle's own executed
    block pairs.  full=True runs and times the oracle on every head and query block (no
    extrapolation; for layers the oracle finishes in seconds)."""
    import numpy as np
    import torch
    from oracle import crisp_oracle as O

    from threadpoolctl import threadpool_info
    torch.set_num_threads(len(os.sched_getaffinity(0)))
    blas = [p["num_threads"] for p in threadpool_info() if p.get("user_api") == "blas"]
    cores = max(blas) if blas else 1
    q, k, v, specs, route, rp, ci, _ = res["_tensors"]
    G = cfg.group
    block = cfg.block
    op = O.Params(alpha=cfg.alpha)
    nb = O.n_blocks(cfg.seq_len, block)
    t0 = time.perf_counter()
    heads_done, sel_time, pairs_total, sets = 0, 0.0, 0, {}
    Kc, Vc = {}, {}
    order = sorted(range(cfg.n_q_heads), key=lambda h: (h % 2, h))
    for h in order:
        g = h // G
        if g not in Kc:
            Kc[g] = k[g].float().cpu().numpy().astype(np.float64)
            Vc[g] = v[g].float().cpu().numpy().astype(np.float64)
        Qh = q[h].float().cpu().numpy().astype(np.float64)
        t = time.perf_counter()
        r = O.crisp_head(Qh, Kc[g], None, block, op, attend=False)
        sel_time += time.perf_counter() - t
        sets[h] = (Qh, r.sets)
        pairs_total_h = sum(len(s) for s in r.sets)
        pairs_total += pairs_total_h
        heads_done += 1
        if not full and time.perf_counter() - t0 > budget_s * 0.6 and heads_done >= 2:
            break
    # extrapolate selection to all heads by the measured mean
    sel_ms_layer = sel_time / heads_done * cfg.n_q_heads * 1e3
    pairs_layer = pairs_total / heads_done * cfg.n_q_heads
    # attention sample: spread query blocks over the selected heads
    att_time, att_pairs, units = 0.0, 0, 0
    rng = np.random.default_rng(0)
    hs = list(sets.keys())
    if full:
        for h in hs:
            Qh, s = sets[h]
            t = time.perf_counter()
            O.sparse_attention(Qh, Kc[h // G], Vc[h // G], s, block, op.scale(128))
            att_time += time.perf_counter() - t
            att_pairs += sum(len(x) for x in s)
            units += nb
        total = (sel_time + att_time) * 1e3
        return {"value": total, "unit": "ms/layer", "cores": cores, "kind": "oracle",
                "sample": (f"{cfg.name}: the whole oracle (estimate, route, select and attention) on every head "
                           f"and query block ({cfg.n_q_heads} heads, {units} units, {att_pairs} block pairs); "
                           f"float64 numpy, {cores} BLAS threads of {len(os.sched_getaffinity(0))} host cores"),
                "measured_s": time.perf_counter() - t0}
    while time.perf_counter() - t0 < budget_s and units < 512:
        h = hs[units % len(hs)]
        Qh, s = sets[h]
        qb = int(rng.integers(0, nb))
        t = time.perf_counter()
        O.sparse_attention(Qh, Kc[h // G], Vc[h // G], s, block, op.scale(128), qbs=[qb])
        att_time += time.perf_counter() - t
        att_pairs += len(s[qb])
        units += 1
    attn_ms_layer = att_time / max(att_pairs, 1) * pairs_layer * 1e3
    total = sel_ms_layer + attn_ms_layer
    return {
        "value": total, "unit": "ms/layer", "cores": cores, "kind": "oracle",
        "sample": (f"{cfg.name}: oracle estimate+route+select on {heads_done} of {cfg.n_q_heads} heads "
                   f"({sel_time:.1f}s, scaled to all heads), attention on {units} (head, query-block) units "
                   f"({att_pairs} block pairs, {att_time:.1f}s) scaled by the oracle's own executed block pairs; "
                   f"float64 numpy, {cores} BLAS threads of {len(os.sched_getaffinity(0))} host cores"),
        "measured_s": time.perf_counter() - t0,
    }


def manifest_id():
    """Generator version and sha256[:16] of tests/golden/manifests.json (the seeded workloads'
    realised per-head statistics: C_struct, sink mass, route, k_v, k_s, density)."""
    from workloads import GEN_VERSION
    path = os.path.join(ROOT, "tests", "golden", "manifests.json")
    return {"gen_version": GEN_VERSION, "manifests_sha": src_hash(path) if os.path.exists(path) else None}


def measured_peaks():
    """The rates this GPU sustains, beside the published peaks: bf16 MFMA from a register-only
    loop of independent v_mfma_f32_32x32x16_bf16 (2048 workgroups, the chip's clock under
    MFMA load) and HBM bandwidth from a plain 1 GiB device copy (16-byte loads and stores;
    read plus written bytes).  Both kernels are in libcrisp_peaks.so."""
    import ctypes
    import torch
    path = os.path.join(ROOT, "paper_2609_01925_amd", "libcrisp_peaks.so")
    lib = ctypes.CDLL(path)
    lib.crisp_peak_mfma_flop.restype = ctypes.c_double
    lib.crisp_peak_mfma_flop.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.crisp_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.crisp_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    dev = "cuda:0"
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    wg, iters = 2048, 20000
    out = torch.empty(wg * 256, dtype=torch.float32, device=dev)

    def mfma():
        assert lib.crisp_peak_mfma_bf16(wg, iters, ctypes.c_void_p(out.data_ptr()), stream) == 0

    t_mfma = time_events(mfma, 10, 3)
    mfma_tflops = lib.crisp_peak_mfma_flop(wg, iters) / (t_mfma["median"] * 1e-3) / 1e12
    # the same MFMAs on operands that change every instruction (random normal bf16 values),
    # each launch about as long as the 128k attention launch, so the clock settles where
    # it does under that kernel
    lib.crisp_peak_mfma_bf16_toggling.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p]
    g = torch.Generator(device="cpu").manual_seed(20261202)
    ops = torch.randn(64 * 16 * 8, generator=g).to(torch.bfloat16).to(dev)
    iters_t = 80000

    def mfma_t():
        assert lib.crisp_peak_mfma_bf16_toggling(wg, iters_t, ctypes.c_void_p(ops.data_ptr()),
                                                 ctypes.c_void_p(out.data_ptr()), stream) == 0

    t_tog = time_events(mfma_t, 10, 3)
    tog_tflops = lib.crisp_peak_mfma_flop(wg, iters_t) / (t_tog["median"] * 1e-3) / 1e12
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)

    def copy():
        assert lib.crisp_peak_copy(ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()), nbytes,
                                   8192, stream) == 0

    t_copy = time_events(copy, 10, 3)
    torch.cuda.synchronize()
    assert bool(torch.equal(src, dst))
    copy_gbs = 2.0 * nbytes / (t_copy["median"] * 1e-3) / 1e9
    del src, dst, out, ops
    torch.cuda.empty_cache()
    log(f"peaks: bf16 MFMA {mfma_tflops:.0f} TFLOP/s (constant operands), {tog_tflops:.0f} TFLOP/s "
        f"(toggling operands), copy {copy_gbs:.0f} GB/s")
    # LDS read rates in the attention kernel's operand patterns and the VALU issue cost of
    # exp2 against a full-rate FMA, clocked by the waves themselves (s_memtime, core cycles)
    lib.crisp_peak_lds_bytes_per_wave.restype = ctypes.c_double
    lib.crisp_peak_lds_bytes_per_wave.argtypes = [ctypes.c_int, ctypes.c_int]
    lib.crisp_peak_lds_read.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p]
    lib.crisp_peak_valu.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p]
    wg_c, it_c = 512, 20000  # two workgroups (eight waves) per CU, two waves per SIMD
    cyc = torch.empty(wg_c * 4, dtype=torch.int64, device=dev)
    sink = torch.empty(wg_c * 256, dtype=torch.int32, device=dev)

    def median_cycles(launch):
        for _ in range(2):
            assert launch() == 0
        torch.cuda.synchronize()
        v = sorted(cyc.cpu().tolist())
        return v[len(v) // 2]

    lds = {}
    for kind, name in ((0, "b128_k_operand"), (1, "b64_tr_b16_v_operand"), (2, "b64")):
        c = median_cycles(lambda: lib.crisp_peak_lds_read(kind, wg_c, it_c, ctypes.c_void_p(cyc.data_ptr()),
                                                          ctypes.c_void_p(sink.data_ptr()), stream))
        lds[name] = 8 * lib.crisp_peak_lds_bytes_per_wave(kind, it_c) / c  # bytes per clock per CU (8 waves)
    valu = {}
    for kind, name in ((0, "exp2_f32"), (1, "fma_f32"), (2, "exp2_f16")):
        c = median_cycles(lambda: lib.crisp_peak_valu(kind, wg_c, it_c, ctypes.c_void_p(cyc.data_ptr()),
                                                      ctypes.c_void_p(sink.data_ptr()), stream))
        valu[name] = c / (2 * it_c * 8)  # SIMD cycles per wave-wide instruction (two waves per SIMD)
    log(f"peaks: LDS read B/clk/CU {', '.join(f'{k} {v:.0f}' for k, v in lds.items())}; VALU cycles per "
        f"wave instruction {', '.join(f'{k} {v:.2f}' for k, v in valu.items())}")
    return {"mfma_bf16_tflops": tog_tflops, "mfma_bf16_constant_operand_tflops": mfma_tflops,
            "lds_read_bytes_per_clk_per_cu": lds, "valu_cycles_per_wave_instruction": valu,
            "mfma_bf16_published_tflops": MFMA_BF16_PEAK_TFLOPS,
            "copy_gbs": copy_gbs, "hbm_published_gbs": HBM_PEAK_GBS,
            "method": ("MFMA: 2048 workgroups x 4 waves, 4 independent v_mfma_f32_32x32x16_bf16 chains per wave, "
                       f"median of 10 launches; mfma_bf16_tflops: operands cycling through 16 random normal "
                       f"bf16 registers per lane ({iters_t} rounds, launches about as long as the 128k attention's); "
                       f"constant_operand: the same registers every MFMA ({iters} rounds); copy: 1 GiB device to "
                       "device, 16-byte loads and stores, read + written bytes, median of 10 launches; LDS: "
                       "512 workgroups (8 waves per CU) x 20000 rounds of 8 reads in the attention kernel's K and "
                       "V operand patterns, bytes per core clock per CU from each wave's s_memtime cycles "
                       "(median wave); VALU: 8 independent chains of v_exp_f32, v_fma_f32 or v_exp_f16 per wave, two waves "
                       "per SIMD, SIMD cycles per wave-wide instruction")}


def config_records(steps, warmup, skip_cpu, peaks):
    """Per-config records of the smaller layers: the 4k tiny layer, the 32k Llama-3-8B layer and
    the six alpha x B cells of the 64k selection-stress layer, each timed like the headline
    (CRISP end to end, stages, dense), with the oracle beside it: the whole oracle on the 4k
    and 32k layers, a bounded sample (about 4 s) on each 64k cell."""
    import torch
    from workloads import CONFIGS, STRESS_ALPHAS, STRESS_BLOCKS, stress_config
    layers = [("c0", CONFIGS[0], 0.0, True), ("c1", CONFIGS[1], 0.0, True)]
    layers += [(f"c4_a{a:g}_b{b}", stress_config(a, b), 4.0, False) for a in STRESS_ALPHAS for b in STRESS_BLOCKS]
    out = {}
    for key, cfg, budget, full in layers:
        r = layer_measure(cfg, steps, warmup, key)
        rec = {k_: v_ for k_, v_ in r.items() if not k_.startswith("_")}
        if peaks:
            rec["sparse_attn_frac_of_measured_mfma"] = (r["_attn_flop"] / (r["_attn_launch_ms"] * 1e-3) / 1e12
                                                        / peaks["mfma_bf16_tflops"])
        if not skip_cpu:
            rec["cpu_baseline"] = cpu_baseline(cfg, r, budget_s=budget, full=full)
            log(f"{key}: oracle {rec['cpu_baseline']['value']:.0f} ms/layer "
                f"({rec['cpu_baseline']['measured_s']:.1f}s)")
        out[key] = rec
        del r
        torch.cuda.empty_cache()
    return out


def profile_path(workload):
    return os.path.join(ROOT, "profiles", f"crisp_kernels_{workload}.md")


def attn_traffic(kernel_src_hash, workload):
    """HBM bytes (fetch + write) per launch of the sparse attention kernel on `workload`, from the
    committed rocprofv3 counter summary, if it was taken on the current attention kernel source;
    else None."""
    path = profile_path(workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    if f"attn.hip sha256[:16]: {kernel_src_hash}" not in text:
        return None
    for line in text.splitlines():
        if "PMC_RECORD " in line:
            rec = json.loads(line.split("PMC_RECORD ", 1)[1].rstrip("`"))
            k = rec.get("kernels", {}).get("attn_kernel<128, false>", {})
            if k.get("FETCH_bytes") is not None and k.get("WRITE_bytes") is not None:
                return k["FETCH_bytes"] + k["WRITE_bytes"]
    return None


COPY_BYTES = 1 << 30
SIMDS = 256 * 4  # MI355X: 256 CUs x 4 SIMDs


def copy_calibration():
    """A plain device copy of COPY_BYTES (libcrisp_peaks.so's peak_copy): its FETCH_SIZE /
    WRITE_SIZE give the scale from counter units to bytes."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_01925_amd", "libcrisp_peaks.so"))
    lib.crisp_peak_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    x = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    assert lib.crisp_peak_copy(ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), COPY_BYTES, 8192,
                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)) == 0
    torch.cuda.synchronize()
    del x, y


def _short_kernel(name):
    """'void crisp::(anonymous namespace)::attn_kernel<128, false>(crisp::...)' -> 'attn_kernel<128, false>'."""
    import re
    for pre in ("void ", "crisp::(anonymous namespace)::", "(anonymous namespace)::", "crisp::"):
        name = name.replace(pre, "")
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            name = name[:i]
            break
    return re.sub(r"\s+", " ", name).strip()


def summarize(args):
    """Turns rocprofv3 csv output into a short markdown summary under profiles/: the kernel
    trace statistics, and per kernel the median per dispatch of every counter collected
    (one rocprofv3 run per counter set), with the derived figures: HBM bytes read and
    written (FETCH_SIZE / WRITE_SIZE scaled by what they read for a plain copy of known
    size), bf16 and fp32 MFMA work (MOPS x 512 FLOP), MFMA and LDS utilisation
    (rocprofv3's MfmaUtil, LdsUtil), the L2 hit rate, the counter-run dispatch duration and
    the clock (GRBM_GUI_ACTIVE per XCD over that duration)."""
    import csv
    import glob
    import statistics
    root = args.summarize
    out = [f"# {args.label}\n\n"]
    out.append("Commands (rocprofv3 runs of committed files; `<out>` is the output folder):\n\n")
    for c in args.command:
        out.append(f"* `{c}`\n")
    out.append("\nSource hashes:\n\n")
    csrc = os.path.join(ROOT, "paper_2609_01925_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith(".hip"):
            out.append(f"* {f} sha256[:16]: {src_hash(os.path.join(csrc, f))}\n")
    stats = sorted(glob.glob(os.path.join(root, "**", "*kernel_stats.csv"), recursive=True))
    if stats:
        out.append("\n## Kernel time (rocprofv3 --kernel-trace --stats)\n\n")
        out.append("| kernel | calls | avg us | min us | max us | total ms |\n|---|---|---|---|---|---|\n")
        for r in csv.DictReader(open(stats[0])):
            if "crisp" not in r["Name"]:
                continue
            out.append(f"| {_short_kernel(r['Name'])} | {r['Calls']} | {float(r['AverageNs'])/1e3:.1f} | "
                       f"{float(r['MinNs'])/1e3:.1f} | {float(r['MaxNs'])/1e3:.1f} | "
                       f"{float(r['TotalDurationNs'])/1e6:.2f} |\n")
    per, dur = {}, {}
    for path in sorted(glob.glob(os.path.join(root, "**", "*counter_collection.csv"), recursive=True)):
        for r in csv.DictReader(open(path)):
            name = r["Kernel_Name"]
            if "crisp" in name:
                key = _short_kernel(name)
            elif "peak_copy" in name:
                key = "copy (1 GiB calibration)"
            else:
                continue
            per.setdefault((key, r["Counter_Name"]), []).append(float(r["Counter_Value"]))
            d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
            dur.setdefault((key, r["Counter_Name"]), []).append(d)
    rec = {"kernels": {}}
    if per:
        med = {k: statistics.median(v) for k, v in per.items()}
        kernels = sorted({k for k, _ in per})
        counters = sorted({c for _, c in per})
        scale = {}
        for c, known in (("FETCH_SIZE", COPY_BYTES), ("WRITE_SIZE", COPY_BYTES)):
            cal = med.get(("copy (1 GiB calibration)", c))
            if cal:
                scale[c] = known / cal
                rec[c + "_bytes_per_unit"] = scale[c]
        out.append("\n## Counters per dispatch (rocprofv3 --pmc), median over dispatches\n\n")
        out.append("| kernel | " + " | ".join(counters) + " | dispatches |\n")
        out.append("|---" * (len(counters) + 2) + "|\n")
        for k in kernels:
            n_disp = max(len(per.get((k, c), [])) for c in counters)
            cells = [f"{med[(k, c)]:.6g}" if (k, c) in med else "" for c in counters]
            out.append(f"| {k} | " + " | ".join(cells) + f" | {n_disp} |\n")
        out.append("\n## Derived per dispatch\n\n")
        out.append("| kernel | counter-run ms | HBM read GB | HBM written GB | bf16 MFMA TFLOP | fp32 MFMA TFLOP "
                   "| MfmaUtil % | LdsUtil % | L2 hit % | clock GHz |\n|---|---|---|---|---|---|---|---|---|---|\n")
        for k in kernels:
            d = {}
            dms = [statistics.median(v) for (kk, c), v in dur.items() if kk == k]
            if dms:
                d["counter_run_ms"] = statistics.median(dms) * 1e3
            if ("FETCH_SIZE" in scale) and (k, "FETCH_SIZE") in med:
                d["FETCH_bytes"] = med[(k, "FETCH_SIZE")] * scale["FETCH_SIZE"]
            if ("WRITE_SIZE" in scale) and (k, "WRITE_SIZE") in med:
                d["WRITE_bytes"] = med[(k, "WRITE_SIZE")] * scale["WRITE_SIZE"]
            for c, key in (("SQ_INSTS_VALU_MFMA_MOPS_BF16", "bf16_mfma_flop"), ("SQ_INSTS_VALU_MFMA_MOPS_F32",
                                                                                  "f32_mfma_flop")):
                if (k, c) in med:
                    d[key] = med[(k, c)] * 512.0
            for c in ("MfmaUtil", "LdsUtil"):
                if (k, c) in med:
                    d[c] = med[(k, c)]
            if (k, "TCC_HIT_sum") in med and (k, "TCC_MISS_sum") in med:
                tot = med[(k, "TCC_HIT_sum")] + med[(k, "TCC_MISS_sum")]
                d["L2_hit"] = med[(k, "TCC_HIT_sum")] / tot if tot else None
            if (k, "GRBM_GUI_ACTIVE") in med and (k, "GRBM_GUI_ACTIVE") in dur:
                d["clock_ghz"] = med[(k, "GRBM_GUI_ACTIVE")] / 8.0 / statistics.median(dur[(k, "GRBM_GUI_ACTIVE")]) / 1e9
            # Issue and overlap of the SIMDs, in SIMD-cycles over GRBM_GUI_ACTIVE / 8 XCDs x 1024
            # SIMDs: SQ_VALU_MFMA_BUSY_CYCLES and SQ_VALU_MFMA_COEXEC_CYCLES count SIMD-cycles,
            # SQ_ACTIVE_INST_VALU quad-cycles (x 4; it includes the issue of MFMAs, 4 cycles each,
            # taken out below), SQ_WAIT_INST_ANY and SQ_WAVE_CYCLES wave quad-cycles.
            if (k, "GRBM_GUI_ACTIVE") in med:
                simd_cycles = med[(k, "GRBM_GUI_ACTIVE")] / 8.0 * SIMDS
                if (k, "SQ_VALU_MFMA_BUSY_CYCLES") in med:
                    d["mfma_busy"] = med[(k, "SQ_VALU_MFMA_BUSY_CYCLES")] / simd_cycles
                if (k, "SQ_VALU_MFMA_COEXEC_CYCLES") in med:
                    d["coexec"] = med[(k, "SQ_VALU_MFMA_COEXEC_CYCLES")] / simd_cycles
                if (k, "SQ_ACTIVE_INST_VALU") in med and (k, "SQ_INSTS_MFMA") in med:
                    d["valu_busy"] = (4.0 * med[(k, "SQ_ACTIVE_INST_VALU")] - 4.0 * med[(k, "SQ_INSTS_MFMA")]) / simd_cycles
                if "mfma_busy" in d and "coexec" in d and "valu_busy" in d:
                    d["valu_only"] = d["valu_busy"] - d["coexec"]
                    d["neither"] = 1.0 - d["mfma_busy"] - d["valu_only"]
            if (k, "SQ_WAIT_INST_ANY") in med and (k, "SQ_WAVE_CYCLES") in med:
                d["wait_inst_frac"] = med[(k, "SQ_WAIT_INST_ANY")] / med[(k, "SQ_WAVE_CYCLES")]
            rec["kernels"][k] = d
            f = lambda key, sc=1.0, fmt="{:.3g}": fmt.format(d[key] / sc) if d.get(key) is not None else ""
            out.append(f"| {k} | {f('counter_run_ms')} | {f('FETCH_bytes', 1e9)} | {f('WRITE_bytes', 1e9)} | "
                       f"{f('bf16_mfma_flop', 1e12)} | {f('f32_mfma_flop', 1e12)} | {f('MfmaUtil')} | {f('LdsUtil')} | "
                       f"{f('L2_hit', 0.01)} | {f('clock_ghz')} |\n")
        if any("mfma_busy" in d or "valu_busy" in d for d in rec["kernels"].values()):
            out.append("\n## SIMD issue and overlap per dispatch\n\n")
            out.append("| kernel | MFMA busy % | VALU busy % (no MFMA issue) | MFMA and VALU together % "
                       "| VALU with MFMA idle % | neither % | waves waiting on an instruction % |\n"
                       "|---|---|---|---|---|---|---|\n")
            for k in kernels:
                d = rec["kernels"][k]
                if not any(x in d for x in ("mfma_busy", "valu_busy", "coexec")):
                    continue
                g = lambda key: f"{100 * d[key]:.1f}" if d.get(key) is not None else ""
                out.append(f"| {k} | {g('mfma_busy')} | {g('valu_busy')} | {g('coexec')} | {g('valu_only')} | "
                           f"{g('neither')} | {g('wait_inst_frac')} |\n")
            out.append("\nFractions of SIMD-cycles (GRBM_GUI_ACTIVE / 8 XCDs x 1024 SIMDs): MFMA busy = "
                       "SQ_VALU_MFMA_BUSY_CYCLES; VALU busy = 4 x SQ_ACTIVE_INST_VALU (quad-cycles) less 4 cycles "
                       "per MFMA issued (SQ_INSTS_MFMA); together = SQ_VALU_MFMA_COEXEC_CYCLES; VALU with MFMA "
                       "idle = VALU busy - together; neither = the rest (waits on LDS, memory, barriers, "
                       "dependences).  The last column is SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES.\n")
        out.append("\nMfmaUtil = 100 * (sum of SQ_VALU_MFMA_BUSY_CYCLES) / (GRBM_GUI_ACTIVE * SIMD count), "
                   "rocprofv3's own derived metric; clock = GRBM_GUI_ACTIVE / 8 XCDs / dispatch duration "
                   "in the counter run (counter runs serialise dispatches, so their durations are close to, "
                   "not equal to, the trace's).\n")
    out.append("\nMachine-readable: `PMC_RECORD " + json.dumps(rec) + "`\n")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    dst = os.path.join(ROOT, "profiles", args.label + ".md")
    with open(dst, "w") as f:
        f.write("".join(out))
    print(dst)


def clock_power(seconds=8.0):
    """Socket power and GFX clock while each of several loads runs for `seconds`: idle, the
    sparse attention (on the layer's own CRISP lists) and the dense attention of the 128k
    Llama layer, the MFMA loop of measured_peaks on toggling and on constant operands, and the
    estimator.  amd-smi is sampled in a child process about every 0.3 s; the first second of
    each load is left out.  The published power cap is read from rocm-smi."""
    import ctypes
    import re
    import shutil
    import subprocess
    import threading
    import torch
    from paper_2609_01925_amd import crisp as C
    from workloads import CONFIGS, make_layer
    smi = shutil.which("amd-smi") or "/opt/rocm/bin/amd-smi"
    samples, stop = [], threading.Event()

    def sampler():
        while not stop.is_set():
            try:
                r = subprocess.run([smi, "metric", "-p", "-c"], capture_output=True, text=True, timeout=10)
            except (OSError, subprocess.SubprocessError):
                return
            pw = re.search(r"SOCKET_POWER:\s*(\d+)\s*W", r.stdout)
            ck = [int(x) for x in re.findall(r"GFX_\d+:\s*\n\s*CLK:\s*(\d+)\s*MHz", r.stdout)]
            if pw and ck:
                samples.append((time.time(), int(pw.group(1)), sum(ck) / len(ck)))
            stop.wait(0.2)

    dev = "cuda:0"
    cfg = CONFIGS[2]
    q, k, v, _ = make_layer(cfg, device=dev)
    p = C.make_params(alpha=cfg.alpha)
    o, _, rp, ci = C.crisp_prefill_attn(q, k, v, p, cfg.block, return_lists=True)
    ws = torch.empty(C.crisp_sparse_workspace_size(C.shape_of(q, k, cfg.block)), dtype=torch.uint8, device=dev)
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_01925_amd", "libcrisp_peaks.so"))
    lib.crisp_peak_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.crisp_peak_mfma_bf16_toggling.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                                  ctypes.c_void_p]
    stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    out = torch.empty(2048 * 256, dtype=torch.float32, device=dev)
    g = torch.Generator(device="cpu").manual_seed(20261202)
    ops = torch.randn(64 * 16 * 8, generator=g).to(torch.bfloat16).to(dev)
    phases = [
        ("idle", None),
        ("sparse_attn_128k", lambda: C.crisp_sparse_attn(q, k, v, rp, ci, cfg.block, out=o, ws=ws)),
        ("dense_attn_128k", lambda: C.crisp_dense_attn(q, k, v, cfg.block, out=o)),
        ("mfma_loop_toggling_operands", lambda: lib.crisp_peak_mfma_bf16_toggling(
            2048, 80000, ctypes.c_void_p(ops.data_ptr()), ctypes.c_void_p(out.data_ptr()), stream)),
        ("mfma_loop_constant_operands", lambda: lib.crisp_peak_mfma_bf16(
            2048, 20000, ctypes.c_void_p(out.data_ptr()), stream)),
        ("estimate_128k", lambda: C.crisp_estimate(q, k, p, cfg.block)),
    ]
    cap = None
    try:
        r = subprocess.run([shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi", "--showmaxpower"],
                           capture_output=True, text=True, timeout=30)
        m = re.search(r"Max Graphics Package Power \(W\):\s*([0-9.]+)", r.stdout)
        cap = float(m.group(1)) if m else None
    except (OSError, subprocess.SubprocessError):
        pass
    torch.cuda.synchronize()
    th = threading.Thread(target=sampler, daemon=True)
    th.start()
    rows = []
    for name, fn in phases:
        t0 = time.time()
        while time.time() - t0 < seconds:
            if fn is None:
                time.sleep(0.25)
            else:
                for _ in range(4):
                    fn()
                torch.cuda.synchronize()
        t1 = time.time()
        sel = [s for s in samples if t0 + 1.0 <= s[0] <= t1]
        row = {"load": name, "samples": len(sel),
               "socket_power_w_median": statistics.median([s[1] for s in sel]) if sel else None,
               "socket_power_w_max": max(s[1] for s in sel) if sel else None,
               "gfx_clock_mhz_median": statistics.median([s[2] for s in sel]) if sel else None}
        rows.append(row)
        log(f"clock/power {row}")
    stop.set()
    th.join(timeout=15)
    return {"power_cap_w": cap, "loads": rows, "seconds_per_load": seconds}


def main():
    args = parse()
    if args.summarize:
        summarize(args)
        return
    if args.clock_power:
        print(json.dumps({"clock_power": clock_power()}), flush=True)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this implementation runs on one GPU only; --gpus must be 1",
                          "n_gpus_requested": args.gpus}))
        sys.exit(2)
    import torch
    from workloads import CONFIGS

    assert torch.cuda.is_available(), "no GPU visible"
    if args.structured:
        from workloads import structured_pe_config
        cfg = structured_pe_config(args.structured)
    else:
        cfg = CONFIGS[args.config]
    if args.copy_calibration:
        copy_calibration()
    peaks = None if args.skip_peaks else measured_peaks()
    res = layer_measure(cfg, args.steps, args.warmup, "headline")
    if not args.skip_comparators:
        res["comparators"] = comparator_measure(cfg, res, args.steps, args.warmup, "headline")
        res["floor_variants"] = floor_variants_measure(cfg, res, args.steps, args.warmup, "headline")
    attn_src = src_hash(os.path.join(ROOT, "paper_2609_01925_amd", "csrc", "attn.hip"))
    achieved = res["_attn_flop"] / (res["_attn_launch_ms"] * 1e-3) / 1e12
    roofline = {
        "bound": "mfma", "achieved": achieved, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
        "frac": achieved / MFMA_BF16_PEAK_TFLOPS,
        "traffic": attn_traffic(attn_src, cfg.name) if cfg.config_id in (2, 3) else None,
        "kernel": "attn_kernel<128,false> (crisp_sparse_attn)",
        "flop_per_launch": res["_attn_flop"], "launch_ms": res["_attn_launch_ms"],
    }
    if peaks:
        roofline["measured_peak"] = peaks["mfma_bf16_tflops"]
        roofline["frac_of_measured_peak"] = achieved / peaks["mfma_bf16_tflops"]
    for r_ in (res,):
        add_measured_fracs(r_, peaks)
    extra = {}
    if not args.skip_512k and args.config != 3 and not args.structured:
        try:
            r3 = layer_measure(CONFIGS[3], args.steps_512k, 1, "512k")
            if not args.skip_comparators:
                r3["comparators"] = comparator_measure(CONFIGS[3], r3, args.steps_512k, 1, "512k", mixes=False)
            add_measured_fracs(r3, peaks)
            extra = {k_: v_ for k_, v_ in r3.items() if not k_.startswith("_")}
            extra["sparse_attn_traffic_bytes"] = attn_traffic(attn_src, CONFIGS[3].name)
            del r3
            torch.cuda.empty_cache()
        except Exception as e:  # noqa: BLE001 -- the headline line must still be printed
            extra = {"error": repr(e)}
    configs = None
    if not args.skip_configs:
        try:
            configs = config_records(args.steps, args.warmup, args.skip_cpu, peaks)
        except Exception as e:  # noqa: BLE001
            configs = {"error": repr(e)}
    sweep = None
    if not args.skip_sweep:
        try:
            sweep = pe_sweep_measure(peaks)
        except Exception as e:  # noqa: BLE001
            sweep = {"error": repr(e)}
    cpu = None
    if not args.skip_cpu:
        cpu = cpu_baseline(cfg, res)
    headline = {k_: v_ for k_, v_ in res.items() if not k_.startswith("_")}
    record = {
        "metric": METRIC,
        "value": res["ms_per_layer"],
        "unit": "ms/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_layer"],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded generator, gen-v1)",
        "config": {"workload": cfg.name, "seq_len": cfg.seq_len, "n_q_heads": cfg.n_q_heads,
                   "n_kv_heads": cfg.n_kv_heads, "head_dim": 128, "block": cfg.block, "alpha": cfg.alpha,
                   "tau_proxy": 0.2, "gamma": 0.95, "parallelism": "single GPU"},
        "speedup_vs_dense": res["speedup_vs_dense"],
        "dense_ms_per_layer": res["dense_ms_per_layer"],
        "roofline": roofline,
        "cpu_baseline": cpu,
        "measured_peaks": peaks,
        "headline_detail": headline,
        "at_512k": extra,
        "per_config": configs,
        "src_sha": {f: src_hash(os.path.join(ROOT, "paper_2609_01925_amd", "csrc", f))
                    for f in sorted(os.listdir(os.path.join(ROOT, "paper_2609_01925_amd", "csrc")))
                    if f.endswith((".hip", ".cpp", ".h"))},
        "attn_src_sha": attn_src,
        # the workload generator's version and the hash of the committed workload manifests
        # (per-head statistics the generator realises), so that drift in the inputs is visible
        "workload_manifest": manifest_id(),
    }
    if sweep is not None:
        record["pe_sweep"] = sweep
    print(json.dumps(record))


if __name__ == "__main__":
    main()
