"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, a library routine (torch softmax / scaled_dot_product_attention in
float64), an invariant implied by the definitions, or brute force over explicit
index sets.  They are chosen so that a dropped term, a wrong sign or index, or a
transposed operand in any oracle stage fails at least one of them.

Stage -> pins:
  proxy attention (Alg. 2)        P3 causal rows, P3 n == b equals dense softmax, P4 flat closed form, P5
  C_struct (Sec. 3.2)             P3 brute force over the anchor set, P3 limits, P4 closed form
  route (Alg. 2)                  P4 flat head routes PE; sink head routes VS; tie rule
  a_v / a_s / p (Alg. 3)          P5 closed form for p_v, brute-force diagonal walk for a_s, P8 identities
  floor and top-k (Alg. 3, Sec. 4.3)  P5 exact set, P6 exact sets at alpha 0.5 / 2, P7 metamorphic
  PE scores and cutoff (Alg. 4)   P4 closed-form A_tilde and K*, P12 loop-by-loop pooled scores,
                                  brute-force cutoff, P7 gamma monotone
  block sets                      P9 structure, slash geometry walk
  sparse attention (Eq. 1)        P1 all blocks == dense SDPA, P2 explicit-mask softmax
  JSD pattern search (App. A)     P10 closed forms and scipy for D_JS, closed-form pooled estimate
                                  (flat and sink heads), loop-by-loop pooled estimate, routes by
                                  visible-key counting
  gamma VS selection (App. A)     P10 explicit cases, brute-force minimal subsets, mass-cliff count
  median noise floor (App. H)     P11 odd/even closed forms, clumpy-noise case, brute-force median
"""
import math

import numpy as np
import pytest
import torch

from oracle import crisp_oracle as O
from tests import parity as PR
from tests.helpers import bf16_round, random_head, sink_head

S128 = 1.0 / math.sqrt(128)


# ---------------------------------------------------------------- P1, P2 (Eq. 1)

def _sdpa_causal(q, k, v, scale):
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None], torch.from_numpy(v)[None, None],
        is_causal=True, scale=scale)
    return out[0, 0].numpy()


@pytest.mark.parametrize("n,block", [(512, 128), (300, 64), (1000, 128), (96, 128)])
@pytest.mark.parametrize("kind", ["vs", "pe"])
def test_p1_all_blocks_is_dense(n, block, kind):
    """k_min = N_b (VS) or gamma = 1 (PE) selects every causal pair, so Eq. 1 is dense causal attention."""
    if kind == "vs":
        q, k, v = sink_head(n, beta=6.0, seed=1)
        q = q + bf16_round(np.random.default_rng(2).standard_normal(q.shape) * 0.3)
    else:
        q, k, v = random_head(n, seed=3, scale=0.05)
    nb = O.n_blocks(n, block)
    # tau = 0 forces VS, tau > 1 forces PE (C_struct lies in [0, 1])
    p = O.Params(k_min_blocks=nb, gamma=1.0, tau_proxy=0.0 if kind == "vs" else 1.5)
    r = O.crisp_head(q, k, v, block, p)
    assert r.route == (O.ROUTE_VS if kind == "vs" else O.ROUTE_PE)
    assert r.sets == O.dense_causal_sets(nb)
    ref = _sdpa_causal(q, k, v, S128)
    assert np.max(np.abs(r.out - ref)) < 1e-12


def test_layer_gqa_mapping_matches_sdpa():
    """crisp_layer over a GQA layer (6 query heads on 3 KV heads, so h // G and h % H_kv
    differ for heads 1, 3 and 4): with every block selected, each head's output is torch's
    grouped-query causal SDPA (enable_gqa, whose grouping is its own), and with the default
    parameters each head's result is the same as the single-head path run on the KV head of
    that grouping."""
    n, block, hq, hkv = 384, 128, 6, 3
    rng = np.random.default_rng(7)
    Q = bf16_round(rng.standard_normal((hq, n, 128)) * 0.3)
    K = bf16_round(rng.standard_normal((hkv, n, 128)))
    V = bf16_round(rng.standard_normal((hkv, n, 128)))
    Q[1, :, 0] += 3.0                 # heads differ in structure so a wrong grouping shows
    K[:, :4, 0] = 8.0
    nb = O.n_blocks(n, block)
    dense = O.crisp_layer(Q, K, V, block, O.Params(k_min_blocks=nb, gamma=1.0))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q)[None], torch.from_numpy(K)[None], torch.from_numpy(V)[None],
        is_causal=True, scale=S128, enable_gqa=True)[0].numpy()
    assert sorted(dense) == list(range(hq))
    for h in range(hq):
        assert np.max(np.abs(dense[h].out - ref[h])) < 1e-12, h
    sparse = O.crisp_layer(Q, K, V, block, O.Params(), heads=[1, 4], qbs={4: [0, 2]})
    assert sorted(sparse) == [1, 4]
    for h in (1, 4):
        g = torch.arange(hq).reshape(hkv, hq // hkv).tolist()
        g = next(i for i, hs in enumerate(g) if h in hs)
        one = O.crisp_head(Q[h], K[g], V[g], block, O.Params(), qbs=[0, 2] if h == 4 else None)
        assert sparse[h].sets == one.sets and np.array_equal(sparse[h].out, one.out)


def test_p2_masked_softmax_identity():
    """Eq. 1 with the explicit n x n mask M_S (0 on selected, -inf elsewhere) equals the oracle's
    blockwise attention on the same sets."""
    n, block = 256, 32
    q, k, v = random_head(n, seed=5, scale=0.3)
    nb = O.n_blocks(n, block)
    rng = np.random.default_rng(6)
    sets = []
    for qb in range(nb):
        s = {0, qb} | {int(x) for x in rng.choice(qb + 1, size=min(qb + 1, 3), replace=False)}
        sets.append(sorted(s))
    out = O.sparse_attention(q, k, v, sets, block, S128)
    M = np.full((n, n), -np.inf)
    for i in range(n):
        for j in range(i + 1):
            if (j // block) in sets[i // block]:
                M[i, j] = 0.0
    logits = torch.from_numpy(q @ k.T * S128 + M)
    ref = (torch.softmax(logits, dim=-1) @ torch.from_numpy(v)).numpy()
    assert np.max(np.abs(out - ref)) < 1e-12


def test_p2_sampled_query_blocks_match_full():
    n, block = 640, 128
    q, k, v = random_head(n, seed=7)
    sets = O.dense_causal_sets(O.n_blocks(n, block))
    full = O.sparse_attention(q, k, v, sets, block, S128)
    part = O.sparse_attention(q, k, v, sets, block, S128, qbs=[1, 4])
    assert np.array_equal(part[128:256], full[128:256]) and np.array_equal(part[512:], full[512:])
    assert not part[:128].any()


# ---------------------------------------------------------------- P3 (Alg. 2, C_struct)

@pytest.mark.parametrize("n,block", [(700, 128), (4096, 128), (50, 64)])
def test_p3_proxy_rows(n, block):
    q, k, _ = random_head(n, seed=11)
    A = O.proxy_attention(q, k, block, S128)
    b = min(block, n)
    assert A.shape == (b, n)
    assert np.allclose(A.sum(axis=1), 1.0, atol=1e-13)
    for r in range(b):
        assert not A[r, n - b + r + 1:].any()
        assert (A[r, : n - b + r + 1] > 0).all()


def test_p3_proxy_equals_dense_softmax_when_n_equals_b():
    n = 128
    q, k, _ = random_head(n, seed=12)
    A = O.proxy_attention(q, k, 128, S128)
    z = torch.from_numpy(q @ k.T * S128)
    z = z.masked_fill(torch.triu(torch.ones(n, n, dtype=torch.bool), 1), float("-inf"))
    assert np.max(np.abs(A - torch.softmax(z, -1).numpy())) < 1e-14


def test_p3_c_struct_brute_force_and_limits():
    n, block = 200, 64
    q, k, _ = random_head(n, seed=13, scale=0.5)
    A = O.proxy_attention(q, k, block, S128)
    for ws, wl in [(16, 16), (64, 64), (0, 10), (10, 0), (150, 100), (0, 0), (200, 0), (0, 200)]:
        anchors = set(range(min(ws, n))) | set(range(max(0, n - wl), n))
        brute = 0.0
        for r in range(A.shape[0]):
            for j in anchors:
                brute += A[r, j]
        brute /= A.shape[0]
        cs = O.c_struct(A, n, ws, wl)
        assert abs(cs - brute) < 1e-13
        assert -1e-15 <= cs <= 1 + 1e-12
        if ws + wl >= n or ws >= n or wl >= n:
            assert abs(cs - 1.0) < 1e-12
        if ws == 0 and wl == 0:
            assert cs == 0.0


def test_route_tie_and_sides():
    assert O.route(0.2, 0.2) == O.ROUTE_VS          # ">=" in Alg. 2
    assert O.route(np.nextafter(np.float32(0.2), np.float32(0)), 0.2) == O.ROUTE_PE
    q, k, _ = sink_head(1024, beta=20.0)
    assert O.crisp_head(q, k, None, 128, O.Params(), attend=False).route == O.ROUTE_VS


# ---------------------------------------------------------------- P4 (flat head, closed forms)

def test_p4_flat_head_proxy_and_c_struct():
    n, block = 4096, 128
    q = np.zeros((n, 128))
    k = bf16_round(np.random.default_rng(20).standard_normal((n, 128)))
    A = O.proxy_attention(q, k, block, S128)
    b = block
    for r in (0, 57, 127):
        i = n - b + r
        assert np.allclose(A[r, : i + 1], 1.0 / (i + 1), rtol=0, atol=1e-16)
    closed = sum((128 + r + 1) / (n - b + r + 1) for r in range(b)) / b
    assert abs(closed - 0.047657) < 5e-7
    assert abs(O.c_struct(A, n, 128, 128) - closed) < 1e-14
    assert O.route(closed, 0.2) == O.ROUTE_PE


def _flat_kstar(nb, gamma):
    """Closed form for a flat head: A_tilde[qb, kb] = 1 / (N_b (qb + 1)); whole rows are taken in
    order until the remainder fits into part of the next row (Alg. 4 with descending order)."""
    g = float(np.float32(gamma))
    m = 0
    while (m + 1) / nb < g:
        m += 1
    rest = g - m / nb
    part = math.ceil(rest * nb * (m + 1) - 1e-9)
    return m, part, m * (m + 1) // 2 + part


@pytest.mark.parametrize("nb,expected", [(512, 118536), (1024, 473657), (32, None), (7, None)])
def test_p4_flat_head_pe_closed_form(nb, expected):
    block = 128
    n = nb * block
    q = np.zeros((n, 128))
    k = bf16_round(np.random.default_rng(21).standard_normal((n, 128)))
    At = O.pe_scores(q, k, block, S128)
    qb, kb = np.tril_indices(nb)
    assert np.allclose(At[qb, kb], 1.0 / (nb * (qb + 1)), rtol=1e-14, atol=0)
    assert not At[np.triu_indices(nb, 1)].any()
    pairs, kstar, _ = O.pe_select(At, 0.95)
    m, part, ks = _flat_kstar(nb, 0.95)
    if expected is not None:
        assert ks == expected
    assert kstar == ks
    want = {(a, c) for a in range(m) for c in range(a + 1)} | {(m, c) for c in range(part)}
    assert set(pairs) == want


def test_pe_cutoff_brute_force():
    """K* = min{k : sum of the k largest >= gamma} by exhaustive prefix search on a tiny matrix."""
    rng = np.random.default_rng(22)
    for trial in range(20):
        nb = int(rng.integers(1, 9))
        L = rng.standard_normal((nb, nb)) * rng.uniform(0.1, 4)
        L[np.triu_indices(nb, 1)] = -np.inf
        E = np.exp(L - L.max(1, keepdims=True))
        A = E / E.sum(1, keepdims=True)
        At = A / A.sum()
        gamma = float(rng.uniform(0.3, 1.0))
        items = [(float(np.float32(At[a, c])), a * nb + c, (a, c)) for a in range(nb) for c in range(a + 1)]
        items.sort(key=lambda t: (-t[0], t[1]))
        total, want = 0.0, []
        for val, _, pair in items:
            if total >= float(np.float32(gamma)):
                break
            total += val
            want.append(pair)
        pairs, kstar, _ = O.pe_select(At, gamma)
        assert pairs == want and kstar == len(want)


def test_pe_gamma_one_takes_everything():
    rng = np.random.default_rng(23)
    nb = 12
    L = rng.standard_normal((nb, nb))
    L[np.triu_indices(nb, 1)] = -np.inf
    E = np.exp(L - L.max(1, keepdims=True))
    At = (E / E.sum(1, keepdims=True)) / nb
    _, kstar, _ = O.pe_select(At, 1.0)
    assert kstar == nb * (nb + 1) // 2


# ---------------------------------------------------------------- P5 (mass cliff, App. C)

def _cliff_inputs(n, a_sink, a_col, cols, d=128):
    q = np.zeros((n, d))
    k = np.zeros((n, d))
    k[:4, 0] = 8.0
    for c in cols:
        k[c, 1] = 8.0
    q[:, 0] = a_sink
    q[:, 1] = a_col
    return q, k


def test_p5_app_c_background_mass():
    """Last proxy row with k signal keys at logit Delta above n - k background keys:
    each background key carries eps = e^-Delta / (k + (n - k) e^-Delta) (App. C)."""
    n = 2048
    q, k = _cliff_inputs(n, 14.0, 0.0, [])
    A = O.proxy_attention(q, k, 128, S128)
    delta = 8 * 14.0 * S128
    eps = math.exp(-delta) / (4 + (n - 4) * math.exp(-delta))
    assert abs(A[-1, 100] - eps) < 1e-18 and abs(A[-1, 2000] - eps) < 1e-18
    assert abs(A[-1, 0] - (1 - (n - 4) * eps) / 4) < 1e-15


def test_p5_cliff_closed_form_scores_and_selection():
    n, block = 2048, 128
    cols = [5 * 128 + 17, 11 * 128 + 90]
    q, k = _cliff_inputs(n, 14.0, 6.0, cols)
    ds, dc = 8 * 14.0 * S128, 8 * 6.0 * S128
    b, nb = block, n // block
    # closed form of p_v per block
    p_v = np.zeros(nb)
    for r in range(b):
        i = n - b + r
        Z = 4 * math.exp(ds) + 2 * math.exp(dc) + (i + 1 - 6)
        for J in range(nb):
            lo, hi = J * block, min((J + 1) * block, i + 1)
            if hi <= lo:
                continue
            w = hi - lo
            if J == 0:
                w += 4 * (math.exp(ds) - 1)
            w += sum(math.exp(dc) - 1 for c in cols if lo <= c < hi)
            p_v[J] += w / Z / b
    r_ = O.crisp_head(q, k, None, block, O.Params(k_min_blocks=1), attend=False)
    assert np.allclose(r_.p_v, p_v, rtol=1e-12, atol=1e-18)
    assert r_.route == O.ROUTE_VS
    assert r_.S_v == [0, 5, 11]
    # with a very large alpha only the top k_min blocks survive
    assert O.vs_select(r_.p_v, 1e6, 3) == [0, 5, 11]
    assert O.vs_select(r_.p_v, 1e6, 1) == [0]


def test_diagonal_scores_by_brute_force_walk():
    """a_s[j] is the mass on the diagonal through (last proxy row, key j): walk every proxy
    entry (r, key), take its query-key offset o = i_r - key and the diagonal's key on the last
    row n - 1 - o, and accumulate -- independent of the oracle's shifted-row sum."""
    for n, block in [(300, 64), (256, 128), (77, 32)]:
        q, k, _ = random_head(n, seed=31, scale=0.7)
        A = O.proxy_attention(q, k, block, S128)
        b = A.shape[0]
        a_s = np.zeros(n)
        a_v = np.zeros(n)
        for r in range(b):
            i = n - b + r
            for key in range(i + 1):
                o = i - key
                a_s[n - 1 - o] += A[r, key] / b
                a_v[key] += A[r, key] / b
        av, as_, pv, ps = O.vs_scores(A, n, block)
        assert np.allclose(as_, a_s, rtol=1e-12, atol=1e-17)
        assert np.allclose(av, a_v, rtol=1e-12, atol=1e-17)
        for J in range(O.n_blocks(n, block)):
            assert abs(ps[J] - a_s[J * block:(J + 1) * block].sum()) < 1e-14


# ---------------------------------------------------------------- P6 (noise exactly at the floor)

def test_p6_noise_at_floor():
    n, block = 4096, 128
    q, k, _ = sink_head(n, beta=math.log(n / 4))
    r = O.crisp_head(q, k, None, block, O.Params(), attend=False)
    assert r.route == O.ROUTE_VS
    nb = n // block
    mids = r.p_v[1:nb - 1]
    assert np.all(mids == mids[0])                        # exactly tied middle blocks
    # alpha = 0.5: every middle block is above half the mean, and so is the last block, whose
    # rows see on average (B + 1) / 2 of its B keys: mass (B + 1) / (2B) of a middle block
    assert O.vs_select(r.p_v, 0.5, 8) == list(range(nb))
    # alpha = 2: only the sink block passes; k_min tops up with the lowest-index ties
    assert O.vs_select(r.p_v, 2.0, 8) == list(range(8))
    # alpha = 1: every middle block sits within 1e-4 of the floor (the exemption band)
    _, _, thr = O.vs_floor(r.p_v, 1.0)
    assert np.all(np.abs(mids - thr) <= 1e-4 * thr)


def test_degenerate_residual_sink_collapse():
    """Sink collapse (E3): logits beta on keys 0..3 and exactly 0 elsewhere, so proxy row r
    (query i) has Z = 4 e^beta + (i + 1 - 4) and every inner block the same mass
    (1/b) sum_r B / Z -- about 1.4e-16, far below float32 resolution next to 1.  The
    block scores match that closed form; the residual, evaluated as printed in float64
    ((1 - p_0) - p_last), equals the inner-block mass up to the cancellation's rounding
    (a few dozen ulps of 1; reading R20) and lies below 2^-20, so the direction is
    degenerate and its floor decisions are rounding noise.  Whatever the floor, the
    k_min top-up takes the sink block and then the tied inner blocks in index order."""
    n, block = 8192, 128
    nb, b = n // block, block
    q, k, _ = sink_head(n, beta=40.0)
    r = O.crisp_head(q, k, None, block, O.Params(), attend=False)
    assert r.route == O.ROUTE_VS
    beta = q[0, 0] * k[0, 0] / math.sqrt(128)           # the exact logit of the bf16 tag values
    rows = np.arange(n - b, n)
    Z = 4.0 * np.exp(beta) + (rows + 1 - 4)
    p_inner = np.mean(block / Z)
    p_last = np.mean((rows - (nb - 1) * block + 1) / Z)
    assert np.allclose(r.p_v[1:nb - 1], p_inner, rtol=1e-12, atol=0)
    assert abs(r.p_v[nb - 1] - p_last) <= 1e-12 * p_last
    rr, mu, thr = O.vs_floor(r.p_v, 1.0)
    assert abs(rr - (nb - 2) * p_inner) <= 1e-14 and rr < 2 ** -20
    assert mu == rr / (nb - 2) and thr == mu
    degenerate, _ = PR.vs_direction_exempt(r.p_v, 1.0, 8)
    assert degenerate
    for alpha in (0.5, 1.0, 2.0, 4.0):
        assert O.vs_select(r.p_v, alpha, 8)[:8] == list(range(8))


# ---------------------------------------------------------------- P7 (metamorphic)

def _structured(n, seed):
    rng = np.random.default_rng(seed)
    q, k, v = sink_head(n, beta=float(rng.uniform(5, 9)), seed=seed)
    cols = rng.choice(np.arange(8, n - 256), size=4, replace=False)
    for i, c in enumerate(cols):
        k[c, 1 + i] = 8.0
        q[:, 1 + i] = bf16_round(np.array([rng.uniform(0.5, 1.2) * math.log(n) * math.sqrt(128) / 8]))[0]
    q = q + bf16_round(rng.standard_normal(q.shape) * 0.4)
    return q, k, v


@pytest.mark.parametrize("seed", [40, 41, 42])
def test_p7_alpha_monotone_and_budget(seed):
    n, block = 4096, 128
    q, k, _ = _structured(n, seed)
    A = O.proxy_attention(q, k, block, S128)
    _, _, pv, ps = O.vs_scores(A, n, block)
    for p in (pv, ps):
        prev = None
        for alpha in (0.25, 0.5, 1.0, 1.5, 2.0, 4.0):
            for km in (1, 8, 40):
                S = O.vs_select(p, alpha, km)
                assert len(S) >= min(km, len(p))
                _, _, thr = O.vs_floor(p, alpha)
                above = {J for J in range(len(p)) if np.float32(p[J]) > thr}
                assert above <= set(S)
            S1 = set(O.vs_select(p, alpha, 1))
            if prev is not None:
                assert S1 <= prev
            prev = S1


def test_p7_gamma_monotone():
    rng = np.random.default_rng(43)
    nb = 40
    L = rng.standard_normal((nb, nb)) * 2
    L[np.triu_indices(nb, 1)] = -np.inf
    E = np.exp(L - L.max(1, keepdims=True))
    At = (E / E.sum(1, keepdims=True)) / nb
    prev = set()
    for g in (0.1, 0.5, 0.8, 0.9, 0.95, 0.99, 1.0):
        cur = set(O.pe_select(At, g)[0])
        assert prev <= cur
        prev = cur


# ---------------------------------------------------------------- P8 (mass identities)

@pytest.mark.parametrize("n,block", [(4096, 128), (1000, 64), (333, 128)])
def test_p8_mass_identities(n, block):
    q, k, _ = _structured(max(n, 600), 44)
    q, k = q[:n], k[:n]
    A = O.proxy_attention(q, k, block, S128)
    av, as_, pv, ps = O.vs_scores(A, n, block)
    assert abs(av.sum() - 1) < 1e-12 and abs(as_.sum() - 1) < 1e-12
    assert abs(pv.sum() - 1) < 1e-12 and abs(ps.sum() - 1) < 1e-12
    assert (pv >= 0).all() and (ps >= 0).all()
    nb = len(pv)
    for p in (pv, ps):
        assert abs(max(1 - p[0] - p[nb - 1], 0) - p[1:nb - 1].sum()) < 1e-12


# ---------------------------------------------------------------- P9 (block sets)

def _check_structure(sets, nb):
    assert len(sets) == nb
    for qb, s in enumerate(sets):
        assert s == sorted(set(s)) and s[0] == 0 and s[-1] == qb
        assert all(0 <= kb <= qb for kb in s)


def test_p9_structure_vs_and_pe():
    n, block = 4096, 128
    nb = n // block
    q, k, v = _structured(n, 45)
    r = O.crisp_head(q, k, None, block, O.Params(), attend=False)
    assert r.route == O.ROUTE_VS
    _check_structure(r.sets, nb)
    q2, k2, _ = random_head(n, seed=46, scale=0.05)
    r2 = O.crisp_head(q2, k2, None, block, O.Params(), attend=False)
    assert r2.route == O.ROUTE_PE
    _check_structure(r2.sets, nb)
    assert sum(len(s) for s in r2.sets) >= r2.pe_info["kstar"]


def test_p9_slash_geometry_walk():
    """A selected slash block J holds the diagonals with last-row key j in block J.  Walked from
    the last row of each query block qb, each such diagonal must land in a key block of S(qb)."""
    nb, block = 24, 64
    n = nb * block
    rng = np.random.default_rng(47)
    S_s = sorted(int(x) for x in rng.choice(nb, size=6, replace=False))
    S_v = sorted(int(x) for x in rng.choice(nb, size=4, replace=False))
    sets = O.vs_block_sets(S_v, S_s, nb)
    for qb in range(nb):
        i = (qb + 1) * block - 1
        for J in S_s:
            for j in range(J * block, (J + 1) * block):
                o = n - 1 - j
                key = i - o
                if key >= 0:
                    assert key // block in sets[qb]
        for J in S_v:
            if J <= qb:
                assert J in sets[qb]
        extra = set(sets[qb]) - {0, qb} - {J for J in S_v if J <= qb} - {qb - (nb - 1 - J) for J in S_s}
        assert not extra


def test_p9_mass_accounting_brute_force():
    """For each query row, the dense softmax mass inside its selected blocks, counted key by key,
    equals one minus the mass outside, counted block by block."""
    n, block = 512, 64
    q, k, _ = _structured(n, 48)
    r = O.crisp_head(q, k, None, block, O.Params(k_min_blocks=2), attend=False)
    z = q @ k.T * S128
    for i in range(0, n, 37):
        row = np.exp(z[i, : i + 1] - z[i, : i + 1].max())
        row /= row.sum()
        inside = sum(row[j] for j in range(i + 1) if (j // block) in r.sets[i // block])
        outside = sum(row[J * block: min((J + 1) * block, i + 1)].sum()
                      for J in range(i // block + 1) if J not in r.sets[i // block])
        assert abs(inside + outside - 1) < 1e-12


# ---------------------------------------------------------------- P10 (FlexPrefill comparator, App. A)

def test_p10_js_distance_closed_forms_and_library():
    """D_JS: 0 on equal inputs, sqrt(ln 2) on disjoint supports, a closed form for a
    one-hot against uniform, symmetric, bounded, and equal to scipy's independent
    jensenshannon (natural logarithm)."""
    from scipy.spatial.distance import jensenshannon
    p = np.array([0.2, 0.3, 0.5])
    assert O.js_distance(p, p) == 0.0
    assert abs(O.js_distance([1.0, 0.0], [0.0, 1.0]) - math.sqrt(math.log(2))) < 1e-15
    assert abs(O.js_distance([1.0, 0.0], [0.5, 0.5]) - math.sqrt(0.75 * math.log(4 / 3))) < 1e-15
    rng = np.random.default_rng(30)
    for _ in range(50):
        m = int(rng.integers(1, 40))
        a = rng.dirichlet(np.full(m, rng.uniform(0.05, 3)))
        b = rng.dirichlet(np.full(m, rng.uniform(0.05, 3)))
        if rng.random() < 0.3:
            a[rng.integers(0, m)] = 0.0
            a /= a.sum()
        d = O.js_distance(a, b)
        assert abs(d - O.js_distance(b, a)) < 1e-15
        assert 0.0 <= d <= math.sqrt(math.log(2)) + 1e-15
        assert abs(d - jensenshannon(a, b)) < 1e-12


def test_p10_pooled_estimate_flat_and_sink_closed_forms():
    """Q = 0: the pooled estimate is uniform over the N_b key blocks whatever K is.  A sink
    head (query carries only the sink tag): pool(K) block 0 = (8 * 4 / 128) e_0, so
    the pooled logit of block 0 is beta / 32 and every other block's is 0."""
    n, block = 4096, 128
    nb = n // block
    k = bf16_round(np.random.default_rng(31).standard_normal((n, 128)))
    ab = O.pooled_estimate(np.zeros((n, 128)), k, block, S128)
    assert np.allclose(ab, 1.0 / nb, rtol=0, atol=1e-16)
    beta = 40.0
    q, ks, _ = sink_head(n, beta=beta)
    ab = O.pooled_estimate(q, ks, block, S128)
    logit0 = q[0, 0] * (8.0 * 4 / 128) * S128          # q carries bf16(beta sqrt(d) / 8) on dim 0
    assert abs(logit0 - beta / 32) < 0.01
    z = math.exp(logit0) + (nb - 1)
    assert abs(ab[0] - math.exp(logit0) / z) < 1e-14
    assert np.allclose(ab[1:], 1.0 / z, rtol=1e-14, atol=0)


def test_p10_jsd_routes_flat_pe_and_sink_vs():
    """The flat head's per-block proxy mass follows from counting visible keys; its
    distance to the uniform pooled estimate is small (routes PE at tau 0.1), while a
    sink head puts all proxy mass in block 0 (routes VS)."""
    n, block = 4096, 128
    nb, b = n // block, block
    p_flat = np.zeros(nb)
    for r in range(b):
        i = n - b + r                      # proxy row r sees keys 0..i
        for J in range(nb):
            p_flat[J] += max(0, min((J + 1) * block, i + 1) - J * block) / (i + 1)
    p_flat /= b
    k = bf16_round(np.random.default_rng(32).standard_normal((n, 128)))
    q0 = np.zeros((n, 128))
    A = O.proxy_attention(q0, k, block, S128)
    _, _, p_v, _ = O.vs_scores(A, n, block)
    assert np.allclose(p_v, p_flat, rtol=0, atol=1e-14)
    d_flat = O.jsd_score(q0, k, p_v, block, S128)
    assert abs(d_flat - O.js_distance(p_flat, np.full(nb, 1.0 / nb))) < 1e-12
    assert d_flat < 0.05 and O.route_jsd(d_flat, 0.1) == O.ROUTE_PE
    q, ks, v = sink_head(n, beta=40.0)
    res = O.crisp_head(q, ks, v, block, O.Params(route_mode="jsd"), attend=False)
    assert res.p_v[0] > 1 - 1e-9 and res.jsd > 0.5 and res.route == O.ROUTE_VS
    assert abs(res.jsd - O.js_distance(res.p_v, O.pooled_estimate(q, ks, block, S128))) < 1e-15


def test_p10_gamma_selection_cases():
    p = np.array([0.5, 0.1, 0.3, 0.1], dtype=np.float32)
    assert O.vs_select_gamma(p, 0.8, 1) == [0, 2]
    assert O.vs_select_gamma(p, 0.85, 1) == [0, 1, 2]           # tie at 0.1: lower block first
    assert O.vs_select_gamma(p, 0.5, 3) == [0, 1, 2]            # k_min raises the budget
    assert O.vs_select_gamma(p, 1.0, 1) == [0, 1, 2, 3]
    short = np.array([0.4, 0.3, 0.2, 0.0], dtype=np.float32)    # sums to 0.9 < gamma
    assert O.vs_select_gamma(short, 0.95, 1) == [0, 1, 2, 3]
    assert O.vs_select_gamma(np.array([0.6, 0.4]), 0.5, 1) == []  # N_b <= 2: forced blocks cover all


def test_p10_gamma_selection_brute_force():
    """|S| is the smallest number of blocks whose mass can reach gamma (exhaustive search
    over subsets), and S is a prefix of the (value desc, block asc) order."""
    import itertools
    rng = np.random.default_rng(33)
    for _ in range(60):
        nb = int(rng.integers(3, 10))
        p = rng.dirichlet(np.full(nb, rng.uniform(0.2, 2))).astype(np.float32)
        if rng.random() < 0.3:
            p[rng.integers(0, nb)] = p[rng.integers(0, nb)]       # plant a tie
        gamma = float(np.float32(rng.uniform(0.2, 0.99)))
        vals = p.astype(np.float64)
        best = nb
        for size in range(1, nb + 1):
            if any(sum(vals[list(c)]) >= gamma for c in itertools.combinations(range(nb), size)):
                best = size
                break
        S = O.vs_select_gamma(p, gamma, 1)
        assert len(S) == max(best, 1)
        rest = [J for J in range(nb) if J not in S]
        for J in S:
            for K in rest:
                assert p[J] > p[K] or (p[J] == p[K] and J < K)


def test_p10_gamma_pulls_in_the_noise_floor_does_not():
    """App. C's mass cliff in one direction: 3 signal blocks holding 0.8 of the mass and
    0.2 spread evenly over the other blocks.  gamma = 0.95 has to add
    ceil(0.15 / noise share) noise blocks; the sink-aware floor keeps the signal."""
    nb = 100
    signal = {0: 0.5, 40: 0.2, 70: 0.1}
    p = np.full(nb, 0.2 / (nb - 3))
    for J, m in signal.items():
        p[J] = m
    p = p.astype(np.float32)
    noise = float(np.float32(0.2 / (nb - 3)))
    S = O.vs_select_gamma(p, 0.95, 1)
    csum_signal = float(sum(np.float64(p[J]) for J in signal))
    need = math.ceil((float(np.float32(0.95)) - csum_signal) / noise - 1e-9)
    assert len(S) == 3 + need and set(signal) <= set(S)
    assert O.vs_select(p, 1.0, 1) == sorted(signal)


# ---------------------------------------------------------------- P11 (median noise floor, App. H)

def test_p11_median_floor_closed_forms():
    """The median of the N_b - 2 non-anchor scores (odd and even counts), and App. H's
    clumpy-noise case: one dominant non-anchor block lifts the mean above a genuine
    weaker block, which the median floor keeps."""
    p = np.array([0.3, 0.05, 0.2, 0.01, 0.02, 0.03, 0.39], dtype=np.float32)   # middle: 5 values
    _, mu, thr = O.vs_floor(p, 1.0, "median")
    assert mu == np.float32(0.03) and thr == np.float32(0.03)
    q = np.array([0.3, 0.05, 0.2, 0.01, 0.02, 0.42], dtype=np.float32)         # middle: 4 values
    _, mu, _ = O.vs_floor(q, 2.0, "median")
    assert mu == (np.float32(0.02) + np.float32(0.05)) * np.float32(0.5)
    nb = 40
    clump = np.full(nb, 0.004, dtype=np.float64)
    clump[0], clump[nb - 1] = 0.2, 0.1
    clump[10] = 0.45                      # dominant non-anchor block
    clump[20] = 0.015                     # weaker genuine signal, below the mean of the residual
    clump[1:nb - 1][clump[1:nb - 1] == 0.004] = (1 - 0.2 - 0.1 - 0.45 - 0.015) / (nb - 4)
    p32 = clump.astype(np.float32)
    mean_sel = O.vs_select(p32, 1.0, 1, "mean")
    med_sel = O.vs_select(p32, 1.0, 1, "median")
    _, mu_mean, _ = O.vs_floor(p32, 1.0, "mean")
    _, mu_med, _ = O.vs_floor(p32, 1.0, "median")
    assert abs(float(mu_mean) - 0.7 / 38) < 1e-7 and mu_med == p32[1]   # the noise level
    assert mean_sel == [0, 10, nb - 1]
    assert med_sel == [0, 10, 20, nb - 1]


def test_p11_median_floor_brute_force():
    """Median by brute force (the value with as many scores above as below) on random vectors."""
    rng = np.random.default_rng(34)
    for _ in range(40):
        nb = int(rng.integers(3, 30))
        p = rng.dirichlet(np.full(nb, rng.uniform(0.2, 3))).astype(np.float32)
        mid = [float(x) for x in p[1:nb - 1]]
        m = len(mid)
        cands = [x for x in mid if sum(y < x for y in mid) <= (m - 1) // 2 and sum(y > x for y in mid) <= m // 2]
        _, mu, _ = O.vs_floor(p, 1.0, "median")
        if m % 2:
            assert float(mu) in cands
        else:
            lo = sorted(mid)[m // 2 - 1]
            hi = sorted(mid)[m // 2]
            assert float(mu) == float((np.float32(lo) + np.float32(hi)) * np.float32(0.5))
        S = O.vs_select(p, 1.0, 0, "median")
        assert S == sorted(J for J in range(nb) if p[J] > mu) or len(S) == 0 and not (p > mu).any()


def _pooled_scores_brute(q, k, block, scale):
    """Alg. 4 written out with loops: block means (a partial last block averaged over the rows
    it has), dot products, a row softmax over kb <= qb, then division by the total."""
    n, d = len(q), len(q[0])
    nb = -(-n // block)
    def mean_rows(x, J):
        rows = range(J * block, min((J + 1) * block, n))
        return [sum(x[i][c] for i in rows) / len(rows) for c in range(d)]
    qbar = [mean_rows(q, J) for J in range(nb)]
    kbar = [mean_rows(k, J) for J in range(nb)]
    abar = [[0.0] * nb for _ in range(nb)]
    for a in range(nb):
        logits = [scale * sum(qbar[a][c] * kbar[b][c] for c in range(d)) for b in range(a + 1)]
        m = max(logits)
        e = [math.exp(x - m) for x in logits]
        z = sum(e)
        for b in range(a + 1):
            abar[a][b] = e[b] / z
    total = sum(sum(r) for r in abar)
    return [[x / total for x in r] for r in abar]


@pytest.mark.parametrize("n,block,d,seed", [(18, 4, 6, 41), (32, 8, 5, 42), (9, 3, 7, 43)])
def test_p12_pooled_scores_brute_force(n, block, d, seed):
    """P12: pooled PE scores (Alg. 4) against the loop-by-loop statement, on random Q != K (so a
    swapped or transposed product, a wrong scale, sum pooling or a column softmax all fail)."""
    rng = np.random.default_rng(seed)
    q = bf16_round(rng.standard_normal((n, d)) * 2.0)
    k = bf16_round(rng.standard_normal((n, d)) * 2.0 + 0.5)
    scale = 0.7
    At = O.pe_scores(q, k, block, scale)
    want = np.array(_pooled_scores_brute(q.tolist(), k.tolist(), block, scale))
    assert np.allclose(At, want, rtol=1e-12, atol=1e-15)
    # the mistakes above do change the result on these inputs
    assert not np.allclose(O.pe_scores(k, q, block, scale), want, rtol=1e-6, atol=1e-9)
    assert not np.allclose(O.pe_scores(q, k, block, 2 * scale), want, rtol=1e-6, atol=1e-9)


@pytest.mark.parametrize("n,block,d,seed", [(18, 4, 6, 44), (30, 8, 5, 45), (5, 8, 4, 46)])
def test_p10_pooled_estimate_brute_force(n, block, d, seed):
    """The pattern search's pooled estimate (App. A) against the loop-by-loop statement on
    random Q != K: the mean of the last b = min(B, n) query rows against each key block's mean
    (a partial last block over its own rows), scaled, softmax over the blocks."""
    rng = np.random.default_rng(seed)
    q = bf16_round(rng.standard_normal((n, d)) * 2.0)
    k = bf16_round(rng.standard_normal((n, d)) * 2.0 - 0.3)
    scale = 0.6
    b = min(block, n)
    qp = [sum(q[i][c] for i in range(n - b, n)) / b for c in range(d)]
    nb = -(-n // block)
    z = []
    for J in range(nb):
        rows = range(J * block, min((J + 1) * block, n))
        kb = [sum(k[i][c] for i in rows) / len(rows) for c in range(d)]
        z.append(scale * sum(qp[c] * kb[c] for c in range(d)))
    e = [math.exp(x - max(z)) for x in z]
    want = np.array([x / sum(e) for x in e])
    got = O.pooled_estimate(q, k, block, scale)
    assert np.allclose(got, want, rtol=1e-12, atol=1e-15)
    if n > b:   # pooling the first b rows instead of the last would differ
        qf = [sum(q[i][c] for i in range(b)) / b for c in range(d)]
        assert not np.allclose(qf, qp)
