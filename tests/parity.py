"""GPU-vs-oracle parity rules for CRISP.

Integer results (routes, block sets, CSR lists) must match exactly, except for
decisions whose deciding value lies within 1e-4 (relative) of the threshold in
the oracle's own arithmetic, where a different rounding order may legitimately
flip them:
  E1  VS floor band:   |p_d[J] - alpha mu_d| <= 1e-4 alpha mu_d
  E2  VS top-up band:  when fewer than k_min blocks pass the floor, blocks with
                       |p_d[J] - t| <= 1e-4 t, t = the k_min-th largest p_d
  E3  degenerate residual: r_d < 2^-20 (below float32 resolution next to 1):
                       only the forced blocks and the invariants are checked
  E4  PE cutoff band:  pairs with |A~ - t*| <= 1e-4 t*, t* = A~ of the last pair
                       taken; if the cumulative mass before or at the cutoff is
                       within 1e-4 gamma of gamma, the pairs at K* and K*+1 too
  E5  JSD route band:  |D_JS - tau_jsd| <= JSD_BAND (the oracle's D_JS)
  E6  VS gamma band:   blocks with |p_d[J] - t| <= 1e-4 t, t = p_d of the last block
                       taken; if the cumulative mass before or at the cutoff is within
                       1e-4 gamma of gamma, the blocks at positions k and k+1 too
Floating-point outputs: attention max-abs <= 2e-2 and mean-abs <= 2e-3 (bf16 against
the float64 oracle); C_struct abs 1e-5; p_v, p_s rtol 1e-4 with atol 1e-7; D_JS abs
JSD_ABS (the pooled estimate in fp32 from bf16 inputs; a p_v error of 1e-6 relative
moves D_JS by far less).
"""
from __future__ import annotations

import numpy as np

from oracle import crisp_oracle as O

BAND = 1e-4
ATTN_MAX_ABS = 2e-2
ATTN_MEAN_ABS = 2e-3
CS_ABS = 1e-5
P_RTOL, P_ATOL = 1e-4, 1e-7
JSD_ABS = 1e-4
JSD_BAND = 1e-3


def csr_to_sets(row_ptr: np.ndarray, col_idx: np.ndarray, h: int, nb: int):
    rp = row_ptr[h]
    return [col_idx[h, rp[qb]:rp[qb + 1]].tolist() for qb in range(nb)]


def check_structure(sets, nb, where=""):
    assert len(sets) == nb, where
    for qb, s in enumerate(sets):
        assert s == sorted(set(s)), f"{where} row {qb} not sorted/unique: {s[:20]}"
        assert s and s[0] == 0 and s[-1] == qb, f"{where} row {qb} misses forced blocks: {s[:10]}..{s[-3:]}"


def vs_direction_exempt(p: np.ndarray, alpha: float, k_min: int, floor: str = "mean"):
    """Returns (degenerate, exempt block set) for one VS direction, from oracle values."""
    nb = len(p)
    r64 = max(1.0 - p[0] - p[nb - 1], 0.0)
    if r64 < 2.0 ** -20:
        return True, set(range(nb))
    _, _, thr = O.vs_floor(p, alpha, floor)
    thr = float(thr)
    ex = {J for J in range(nb) if abs(p[J] - thr) <= BAND * thr}
    c = int(np.count_nonzero(np.asarray(p, np.float32) > np.float32(thr)))
    if c < k_min:
        t = float(np.sort(p)[::-1][min(k_min, nb) - 1])
        ex |= {J for J in range(nb) if abs(p[J] - t) <= BAND * t}
    return False, ex


def compare_vs(gpu_mask: np.ndarray, ores: O.HeadResult, alpha: float, k_min: int, where="", floor: str = "mean"):
    """gpu_mask: uint8 [2, N_b] (S_v, S_s membership)."""
    nb = gpu_mask.shape[1]
    for dir_, (p, S) in enumerate(((ores.p_v, ores.S_v), (ores.p_s, ores.S_s))):
        gsel = set(np.nonzero(gpu_mask[dir_])[0].tolist())
        if nb <= 2:
            assert not gsel, where
            continue
        degenerate, ex = vs_direction_exempt(p, alpha, k_min, floor)
        if degenerate:
            continue
        diff = gsel ^ set(S)
        bad = diff - ex
        assert not bad, f"{where} dir {'vs'[dir_]}: blocks {sorted(bad)[:20]} differ (gpu {sorted(gsel)[:30]}, oracle {S[:30]})"
        assert len(gsel) >= min(k_min, nb), f"{where} dir {'vs'[dir_]}: only {len(gsel)} blocks"


def gamma_direction_info(p: np.ndarray, gamma: float, k_min: int):
    """(order, k, c, t, csum_before, csum_at) of the oracle's gamma selection of one direction."""
    nb = len(p)
    p32 = np.asarray(p, dtype=np.float32)
    order = sorted(range(nb), key=lambda J: (-float(p32[J]), J))
    csum = np.cumsum(p32[order].astype(np.float64))
    hit = np.nonzero(csum >= np.float64(np.float32(gamma)))[0]
    c = int(hit[0]) + 1 if len(hit) else nb
    kd = min(max(c, k_min), nb)
    return order, kd, c, float(p32[order[kd - 1]]), float(csum[kd - 2]) if kd >= 2 else 0.0, float(csum[kd - 1])


def compare_vs_gamma(gpu_mask: np.ndarray, ores: O.HeadResult, gamma: float, k_min: int, where=""):
    """gpu_mask: uint8 [2, N_b] of a VS head selected by gamma coverage; E6 exemptions."""
    nb = gpu_mask.shape[1]
    g = float(np.float32(gamma))
    for dir_, (p, S) in enumerate(((ores.p_v, ores.S_v), (ores.p_s, ores.S_s))):
        gsel = set(np.nonzero(gpu_mask[dir_])[0].tolist())
        if nb <= 2:
            assert not gsel, where
            continue
        order, kd, c, t, cb, ca = gamma_direction_info(p, gamma, k_min)
        ex = {J for J in range(nb) if abs(p[J] - t) <= BAND * t}
        if abs(cb - g) <= BAND * g or abs(ca - g) <= BAND * g:
            ex |= {order[i] for i in (kd - 1, kd) if 0 <= i < nb}
        bad = (gsel ^ set(S)) - ex
        assert not bad, f"{where} dir {'vs'[dir_]}: blocks {sorted(bad)[:20]} differ (gpu {len(gsel)}, oracle {len(S)})"
        assert len(gsel) >= min(k_min, nb), f"{where} dir {'vs'[dir_]}: only {len(gsel)} blocks"


def compare_pe(gpu_sets, ores: O.HeadResult, gamma: float, where=""):
    """Row-by-row comparison of a PE head's block sets with the oracle's, E4 exemptions applied."""
    At = ores.A_tilde
    nb = At.shape[0]
    info = ores.pe_info
    vals = At.astype(np.float32)
    tstar = np.float32(info["t_star"])
    g = float(np.float32(gamma))
    exempt_val = lambda v: abs(float(v) - float(tstar)) <= BAND * float(tstar)
    near_cut = abs(info["csum_before"] - g) <= BAND * g or abs(info["csum_at"] - g) <= BAND * g
    extra = set()
    if near_cut:
        qb, kb = np.tril_indices(nb)
        flat = qb.astype(np.int64) * nb + kb
        order = np.lexsort((flat, -vals[qb, kb].astype(np.float64)))
        K = info["kstar"]
        for pos in (K - 1, K):
            if 0 <= pos < len(order):
                extra.add((int(qb[order[pos]]), int(kb[order[pos]])))
    n_bad = 0
    first = None
    for qb_ in range(nb):
        a, b = set(gpu_sets[qb_]), set(ores.sets[qb_])
        for kb_ in a ^ b:
            if exempt_val(vals[qb_, kb_]) or (qb_, kb_) in extra:
                continue
            n_bad += 1
            if first is None:
                first = (qb_, kb_, float(vals[qb_, kb_]), kb_ in a)
    assert n_bad == 0, f"{where}: {n_bad} PE pairs differ outside the E4 band, first {first}, t*={float(tstar)}"


def check_pe_threshold(row_ptr_h: np.ndarray, col_idx_h: np.ndarray, At: np.ndarray, gamma: float, where=""):
    """PE parity for layers too large for the oracle's full pair sort (Alg. 4).  P_sel is
    the prefix of the A_tilde-descending order whose mass first reaches gamma, so with t*
    the value of its last pair: every causal pair above t* is selected and every pair below
    it is not, except the forced {0, qb} blocks (R18).  The E4 band is exempt: values within
    BAND of t*, and, when the mass sum is within BAND of gamma at the cut, of the next
    value too.  Ties at t* are ordered by flat index in the oracle; they lie in the band.
    row_ptr_h, col_idx_h: one head's CSR; At: the oracle's [N_b, N_b] A_tilde."""
    nb = At.shape[0]
    causal = np.tri(nb, dtype=bool)
    vals = At.astype(np.float32)
    desc = np.sort(vals[causal])[::-1]
    csum = np.cumsum(desc.astype(np.float64))
    g = float(np.float32(gamma))
    hit = np.nonzero(csum >= g)[0]
    kstar = int(hit[0]) + 1 if len(hit) else len(desc)
    tstar = float(desc[kstar - 1])
    lo, hi = tstar * (1 - BAND), tstar * (1 + BAND)
    near_cut = (kstar >= 2 and abs(csum[kstar - 2] - g) <= BAND * g) or abs(csum[kstar - 1] - g) <= BAND * g
    if near_cut and kstar < len(desc):
        lo = min(lo, float(desc[kstar]) * (1 - BAND))
    mask = np.zeros((nb, nb), dtype=bool)
    mask[np.repeat(np.arange(nb), np.diff(row_ptr_h)), col_idx_h[:row_ptr_h[-1]]] = True
    assert not (mask & ~causal).any(), f"{where}: pair above the diagonal"
    forced = np.zeros((nb, nb), dtype=bool)
    forced[:, 0] = True
    forced[np.arange(nb), np.arange(nb)] = True
    assert mask[forced].all(), f"{where}: forced block missing"
    missing = causal & (vals > hi) & ~mask
    extra = causal & ~forced & (vals < lo) & mask
    assert not missing.any(), f"{where}: {int(missing.sum())} pairs above t*={tstar:.4g} not selected"
    assert not extra.any(), f"{where}: {int(extra.sum())} pairs below t*={tstar:.4g} selected"
    return kstar, tstar


def compare_attention(o_gpu: np.ndarray, o_ref: np.ndarray, rows=None, where=""):
    if rows is not None:
        o_gpu, o_ref = o_gpu[rows], o_ref[rows]
    err = np.abs(o_gpu.astype(np.float64) - o_ref)
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    assert mx <= ATTN_MAX_ABS and mean <= ATTN_MEAN_ABS, f"{where}: attention max-abs {mx:.3e} mean-abs {mean:.3e}"
    return mx, mean


def compare_scores(cs_gpu, pv_gpu, ps_gpu, ores: O.HeadResult, where=""):
    assert abs(float(cs_gpu) - ores.c_struct) <= CS_ABS, f"{where}: C_struct {float(cs_gpu)} vs {ores.c_struct}"
    for name, g, o in (("p_v", pv_gpu, ores.p_v), ("p_s", ps_gpu, ores.p_s)):
        err = np.abs(np.asarray(g, np.float64) - o)
        tol = P_ATOL + P_RTOL * np.abs(o)
        bad = np.nonzero(err > tol)[0]
        assert not len(bad), f"{where}: {name} blocks {bad[:10].tolist()} off: gpu {np.asarray(g)[bad[:5]]} oracle {o[bad[:5]]}"


def qb_rows(qbs, block, n):
    rows = []
    for qb in qbs:
        rows.extend(range(qb * block, min((qb + 1) * block, n)))
    return np.asarray(rows, dtype=np.int64)
