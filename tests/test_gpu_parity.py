"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every case prints its name before touching the GPU so that a failing run names
its case.  Inputs come from the seeded generators in workloads/ (generated on
the GPU, copied to the host for the oracle) or from small hand-built tensors.
"""
import math
import sys

import numpy as np
import pytest
import torch

from oracle import crisp_oracle as O
from tests import parity as PR
from tests.helpers import to_f64
from workloads import CONFIGS, custom_config, make_layer, stress_config
from workloads.synth import structured_pe_config

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _crisp():
    from paper_2609_01925_amd import crisp
    return crisp


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def _rand(h, n, d=128, seed=0, scale=1.0):
    g = torch.Generator(device="cpu").manual_seed(seed)
    return (torch.randn(h, n, d, generator=g) * scale).to(torch.bfloat16)


def _oracle_params(p, block):
    return O.Params(alpha=p.alpha, tau_proxy=p.tau_proxy, gamma=p.gamma, w_sink=p.w_sink, w_local=p.w_local,
                    k_min_blocks=p.k_min_blocks, softmax_scale=p.softmax_scale,
                    route_mode="jsd" if p.route_mode == 1 else "cstruct",
                    vs_mode="gamma" if p.vs_mode == 1 else "floor", tau_jsd=p.tau_jsd,
                    floor_mode="median" if p.floor_mode == 1 else "mean")


# ------------------------------------------------------------------ attention kernel

@pytest.mark.parametrize("n,block,hq,hkv", [(4096, 128, 2, 1), (1000, 128, 4, 2), (200, 64, 2, 2), (64, 128, 1, 1),
                                            (1, 128, 1, 1), (4160, 64, 8, 8), (2048, 128, 16, 4),
                                            (1500, 128, 6, 3), (1000, 64, 12, 12)])
def test_dense_attention_matches_oracle(n, block, hq, hkv):
    """Every workgroup-to-unit mapping of the fixed grid: KV-group counts dividing 8, multiples
    of 8, and neither (3, 12)."""
    C = _crisp()
    _say(f"dense n={n} B={block} hq={hq} hkv={hkv}")
    q, k, v = _rand(hq, n, seed=1), _rand(hkv, n, seed=2), _rand(hkv, n, seed=3)
    o = C.crisp_dense_attn(q.to(DEV), k.to(DEV), v.to(DEV), block)
    torch.cuda.synchronize()
    og = to_f64(o)
    Q, K, V = to_f64(q), to_f64(k), to_f64(v)
    G = hq // hkv
    nb = O.n_blocks(n, block)
    for h in range(hq):
        ref = O.sparse_attention(Q[h], K[h // G], V[h // G], O.dense_causal_sets(nb), block, 1 / math.sqrt(128))
        PR.compare_attention(og[h], ref, where=f"dense h{h}")


def _random_lists(hq, nb, seed, density=0.3, junk=False):
    rng = np.random.default_rng(seed)
    cap = nb * (nb + 1) // 2
    rp = np.zeros((hq, nb + 1), np.int32)
    ci = np.zeros((hq, cap + (8 if junk else 0)), np.int32)
    sets = []
    for h in range(hq):
        hs, off = [], 0
        for qb in range(nb):
            s = {0, qb} | {int(x) for x in np.nonzero(rng.random(qb + 1) < density)[0]}
            s = sorted(s)
            hs.append(s)
            row = list(s)
            if junk and qb % 3 == 1:
                row = row + [qb + 1, -5, nb + 7]  # invalid entries the kernel must ignore
            ci[h, off:off + len(row)] = row
            rp[h, qb] = off
            off += len(row)
        rp[h, nb] = off
        sets.append(hs)
    return rp, ci, sets


@pytest.mark.parametrize("n,block,junk", [(2048, 128, False), (1100, 64, False), (1500, 128, True)])
def test_sparse_attention_on_given_lists(n, block, junk):
    C = _crisp()
    _say(f"sparse lists n={n} B={block} junk={junk}")
    hq, hkv = 4, 2
    nb = O.n_blocks(n, block)
    q, k, v = _rand(hq, n, seed=4), _rand(hkv, n, seed=5), _rand(hkv, n, seed=6)
    rp, ci, sets = _random_lists(hq, nb, seed=7, junk=junk)
    o = C.crisp_sparse_attn(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(rp).to(DEV),
                            torch.from_numpy(ci).to(DEV), block)
    o_again = C.crisp_sparse_attn(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(rp).to(DEV),
                                  torch.from_numpy(ci).to(DEV), block)
    o_fixed = C.crisp_sparse_attn(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(rp).to(DEV),
                                  torch.from_numpy(ci).to(DEV), block, balance=False)
    torch.cuda.synchronize()
    assert torch.equal(o, o_again)   # which workgroup runs an item never changes a result
    Q, K, V = to_f64(q), to_f64(k), to_f64(v)
    for name, out in (("work list", o), ("fixed order", o_fixed)):
        og = to_f64(out)
        for h in range(hq):
            ref = O.sparse_attention(Q[h], K[h // 2], V[h // 2], sets[h], block, 1 / math.sqrt(128))
            PR.compare_attention(og[h], ref, where=f"sparse {name} h{h}")


@pytest.mark.parametrize("block", [128, 64])
def test_full_lists_equal_dense_bitwise(block):
    """Full causal lists through the sparse kernel give the dense kernel's bits at 128-row
    blocks (same tiles, same order).  Dense 64-row layers run as 128-row ones, so their
    output equals the 128-row output bit for bit; the 64-row sparse kernel (32-key tiles)
    matches the oracle."""
    C = _crisp()
    _say(f"full lists == dense, B={block}")
    n, hq, hkv = 3000, 4, 1
    nb = O.n_blocks(n, block)
    q, k, v = (_rand(hq, n, seed=8).to(DEV), _rand(hkv, n, seed=9).to(DEV), _rand(hkv, n, seed=10).to(DEV))
    sets = O.dense_causal_sets(nb)
    rp = np.zeros((hq, nb + 1), np.int32)
    ci = np.zeros((hq, nb * (nb + 1) // 2), np.int32)
    for h in range(hq):
        off = 0
        for qb in range(nb):
            ci[h, off:off + qb + 1] = sets[qb]
            rp[h, qb] = off
            off += qb + 1
        rp[h, nb] = off
    o_s = C.crisp_sparse_attn(q, k, v, torch.from_numpy(rp).to(DEV), torch.from_numpy(ci).to(DEV), block,
                              balance=False)
    o_d = C.crisp_dense_attn(q, k, v, block)
    torch.cuda.synchronize()
    if block == 128:
        assert torch.equal(o_s, o_d)
        return
    assert torch.equal(o_d, C.crisp_dense_attn(q, k, v, 128))
    Q, K, V = to_f64(q), to_f64(k), to_f64(v)
    og = to_f64(o_s)
    for h in range(hq):
        ref = O.sparse_attention(Q[h], K[0], V[0], sets, block, 1 / math.sqrt(128))
        PR.compare_attention(og[h], ref, where=f"full lists B=64 h{h}")


def _csr_from_rows(rows, nb):
    rp = np.zeros((1, nb + 1), np.int32)
    flat = [x for r in rows for x in r]
    ci = np.zeros((1, max(nb * (nb + 1) // 2, len(flat))), np.int32)
    ci[0, :len(flat)] = flat
    rp[0, 1:] = np.cumsum([len(r) for r in rows])
    return rp, ci


@pytest.mark.parametrize("case", ["full-b128", "full-b128-8k", "full-b64-ragged", "junk-first-chunk"])
def test_split_rows(case):
    """Rows far longer than the layer's work per workgroup are split into chunks whose
    partial results are merged (online-softmax merge of (O, m, l) in chunk order).  Few heads
    with full causal lists force it (on the persistent grid); the merged rows match the
    oracle, runs are bitwise repeatable, and the split rows round differently
    from the unsplit fixed-order launch (which shows the split path ran).  junk-first-chunk:
    a row's first chunk holds only invalid entries (m = -inf, weighing nothing in the
    merge)."""
    C = _crisp()
    _say(f"split rows {case}")
    if case == "junk-first-chunk":
        # rows from N_b / 2 on: even ones [-5] * 60 + [0, qb] (first chunk all invalid, then
        # merged with weight exactly 1), odd ones ten valid blocks at each end around 40
        # invalid entries (both chunks count; 32 entries per chunk)
        n, block, hq = 16384, 128, 1
        nb = n // block
        rows, sets = [], []
        for qb in range(nb):
            if qb < nb // 2:
                r = sorted({0, qb})
            elif qb % 2 == 0:
                r = [-5] * 60 + [0, qb]
            else:
                r = list(range(10)) + [-5] * 40 + list(range(qb - 9, qb + 1))
            rows.append(r)
            sets.append(sorted({x for x in r if 0 <= x <= qb}))
        rp, ci = _csr_from_rows(rows, nb)
        long_rows = [qb for qb in range(nb // 2, nb) if qb % 2]
    else:
        # 8k: a short layer (units from one list in a fixed stride) with too few units for
        # one workgroup each
        n, block, hq = {"full-b128": (16384, 128, 1), "full-b128-8k": (8192, 128, 1),
                        "full-b64-ragged": (16000, 64, 2)}[case]
        nb = O.n_blocks(n, block)
        sets = O.dense_causal_sets(nb)
        rp = np.zeros((hq, nb + 1), np.int32)
        ci = np.zeros((hq, nb * (nb + 1) // 2), np.int32)
        for h in range(hq):
            ci[h] = np.concatenate([np.asarray(s_, np.int32) for s_ in sets])
            rp[h, 1:] = np.cumsum([len(s_) for s_ in sets])
        long_rows = list(range(nb - nb // 4, nb))
    q, k, v = _rand(hq, n, seed=21), _rand(1, n, seed=22), _rand(1, n, seed=23)
    args = (q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(rp).to(DEV), torch.from_numpy(ci).to(DEV), block)
    o1 = C.crisp_sparse_attn(*args)
    o2 = C.crisp_sparse_attn(*args)
    o_fixed = C.crisp_sparse_attn(*args, balance=False)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)
    rows_idx = torch.from_numpy(PR.qb_rows(long_rows, block, n)).to(DEV)
    assert not torch.equal(o1[:, rows_idx], o_fixed[:, rows_idx]), "no row was split"
    Q, K, V = to_f64(q), to_f64(k)[0], to_f64(v)[0]
    qbs = sorted({0, 1, nb // 2, long_rows[0], nb - 2, nb - 1})
    rows = PR.qb_rows(qbs, block, n)
    for h in range(hq):
        ref = O.sparse_attention(Q[h], K, V, sets, block, 1 / math.sqrt(128), qbs=qbs)
        PR.compare_attention(to_f64(o1[h]), ref, rows=rows, where=f"{case} h{h}")
        PR.compare_attention(to_f64(o1[h]), to_f64(o_fixed[h]), rows=rows, where=f"{case} h{h} vs fixed")


def test_more_than_2p21_units():
    """A layer with more (head, query block) units than a split work item can name
    (2^21): 65 query heads over one KV head at the longest length with B = 64 (2,129,920
    units, one unit per workgroup), each row listing only its diagonal block.  Sampled
    rows of the first and the last head (whose units all lie past 2^21) against float64
    attention over the visible keys of the diagonal block."""
    C = _crisp()
    _say("2^21+ units: 65 heads x 2^21 tokens, B = 64, diagonal lists")
    n, block, hq = 1 << 21, 64, 65
    nb = n // block
    g = torch.Generator(device=DEV).manual_seed(5)
    q = torch.randn(hq, n, 128, generator=g, device=DEV, dtype=torch.bfloat16)
    k = torch.randn(1, n, 128, generator=g, device=DEV, dtype=torch.bfloat16)
    v = torch.randn(1, n, 128, generator=g, device=DEV, dtype=torch.bfloat16)
    rp = torch.arange(nb + 1, dtype=torch.int32, device=DEV).repeat(hq, 1)
    ci = torch.arange(nb, dtype=torch.int32, device=DEV).repeat(hq, 1)
    o = C.crisp_sparse_attn(q, k, v, rp, ci, block)
    torch.cuda.synchronize()
    rng = np.random.default_rng(11)
    rows = [(h, int(i)) for h in (0, 64) for i in rng.integers(0, n, 40)] + [(64, n - 1), (64, 0), (0, n - 1)]
    K, V = k[0], v[0]
    for h, i in rows:
        lo = (i // block) * block
        qi = to_f64(q[h, i:i + 1])[0]
        kk = to_f64(K[lo:i + 1])
        vv = to_f64(V[lo:i + 1])
        sc = kk @ qi / math.sqrt(128)
        w = np.exp(sc - sc.max())
        ref = w @ vv / w.sum()
        got = to_f64(o[h, i:i + 1])[0]
        assert np.abs(got - ref).max() <= PR.ATTN_MAX_ABS, f"head {h} row {i}: {np.abs(got - ref).max():.3e}"
    del q, k, v, o
    torch.cuda.empty_cache()


def test_caller_lists_unordered_and_repeated_entries():
    """crisp_sparse_attn reads rows as given: a row in another order gives the same output
    up to rounding, and an entry listed twice counts its block twice (its keys' softmax
    weights doubled), checked against a float64 statement of exactly that."""
    C = _crisp()
    _say("caller lists: unordered and repeated entries")
    n, block, nb = 1024, 128, 8
    q, k, v = _rand(1, n, seed=31), _rand(1, n, seed=32), _rand(1, n, seed=33)
    rows = [sorted({0, qb, qb // 2, max(qb - 3, 0)}) for qb in range(nb)]
    cap = nb * (nb + 1) // 2
    def csr(rs):
        rp = np.zeros((1, nb + 1), np.int32)
        ci = np.zeros((1, cap), np.int32)
        for qb, r in enumerate(rs):
            rp[0, qb + 1] = rp[0, qb] + len(r)
            ci[0, rp[0, qb]:rp[0, qb + 1]] = r
        return torch.from_numpy(rp).to(DEV), torch.from_numpy(ci).to(DEV)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    o_sorted = to_f64(C.crisp_sparse_attn(qd, kd, vd, *csr(rows), block))[0]
    rng = np.random.default_rng(7)
    shuffled = [list(rng.permutation(r)) for r in rows]
    o_shuf = to_f64(C.crisp_sparse_attn(qd, kd, vd, *csr(shuffled), block))[0]
    assert np.abs(o_shuf - o_sorted).max() <= 1e-2 and np.abs(o_shuf - o_sorted).mean() <= 1e-3
    doubled = [r + [r[0]] for r in rows]  # block 0 listed twice in every row
    o_dup = to_f64(C.crisp_sparse_attn(qd, kd, vd, *csr(doubled), block))[0]
    torch.cuda.synchronize()
    Q, K, V = to_f64(q)[0], to_f64(k)[0], to_f64(v)[0]
    ref = np.zeros((n, 128))
    for i in range(n):
        qb = i // block
        mult = np.zeros(n)
        for kb in doubled[qb]:
            mult[kb * block:(kb + 1) * block] += 1.0
        mult[i + 1:] = 0.0
        sc = (K @ Q[i]) / math.sqrt(128)
        w = mult * np.exp(sc - sc[mult > 0].max())
        ref[i] = w @ V / w.sum()
    PR.compare_attention(o_dup, ref, rows=np.arange(n), where="repeated entries")


def test_attention_custom_scale_and_empty_rows():
    C = _crisp()
    _say("custom scale, empty rows")
    n, block = 512, 128
    nb = O.n_blocks(n, block)
    q, k, v = _rand(1, n, seed=11), _rand(1, n, seed=12), _rand(1, n, seed=13)
    rp = np.array([[0, 1, 1, 3, 3]], np.int32)        # row 1 and row 3 have no entries
    ci = np.zeros((1, nb * (nb + 1) // 2), np.int32)
    ci[0, :3] = [0, 0, 2]
    o = C.crisp_sparse_attn(q.to(DEV), k.to(DEV), v.to(DEV), torch.from_numpy(rp).to(DEV),
                            torch.from_numpy(ci).to(DEV), block, softmax_scale=0.05)
    torch.cuda.synchronize()
    og = to_f64(o)[0]
    assert not og[128:256].any() and not og[384:].any()
    ref = O.sparse_attention(to_f64(q)[0], to_f64(k)[0], to_f64(v)[0], [[0], [], [0, 2], []], block, 0.05,
                             qbs=[0, 2])
    PR.compare_attention(og, ref, rows=PR.qb_rows([0, 2], block, n), where="scale 0.05")


# ------------------------------------------------------------------ estimate / route / select

def _run_stages(C, q, k, v, params, block, want_jsd=False):
    cs, pv, ps = C.crisp_estimate(q, k, params, block)
    jsd = C.crisp_jsd(q, k, pv, params, block) if (params.route_mode == 1 or want_jsd) else None
    score = jsd if params.route_mode == 1 else cs
    route, rp, ci, dm = C.crisp_route_select(q, k, score, pv, ps, params, block)
    torch.cuda.synchronize()
    out = (cs.cpu().numpy(), pv.cpu().numpy(), ps.cpu().numpy(), route.cpu().numpy(), rp.cpu().numpy(),
           ci.cpu().numpy(), dm.cpu().numpy())
    return out + ((jsd.cpu().numpy(),) if want_jsd else ())


def _check_layer(C, cfg, params, heads=None, qbs_per_head=None, attn=True, where=""):
    """Runs estimate + route/select (+ prefill) for the layer on the GPU and checks the given heads."""
    block = cfg.block
    q, k, v, specs = make_layer(cfg, device=DEV)
    cs, pv, ps, route, rp, ci, dm, jsd = _run_stages(C, q, k, v, params, block, want_jsd=True)
    nb = O.n_blocks(cfg.seq_len, block)
    op = _oracle_params(params, block)
    k_min = op.k_min(block)
    heads = list(range(cfg.n_q_heads)) if heads is None else heads
    o = C.crisp_prefill_attn(q, k, v, params, block) if attn else None
    torch.cuda.synchronize()
    Q = to_f64(q[heads]) if heads else None
    G = cfg.group
    groups = sorted(set(h // G for h in heads))
    Kg = {g: to_f64(k[g]) for g in groups}
    Vg = {g: to_f64(v[g]) for g in groups}
    og = {h: to_f64(o[h]) for h in heads} if attn else {}
    for i, h in enumerate(heads):
        w = f"{where} h{h} ({specs[h].kind})"
        res = O.crisp_head(Q[i], Kg[h // G], None, block, op, attend=False)
        PR.compare_scores(cs[h], pv[h], ps[h], res, where=w)
        d_or = O.jsd_score(Q[i], Kg[h // G], res.p_v, block, op.scale(128))
        assert abs(float(jsd[h]) - d_or) <= PR.JSD_ABS, f"{w}: D_JS gpu {float(jsd[h]):.6f} oracle {d_or:.6f}"
        if op.route_mode == "jsd" and abs(d_or - op.tau_jsd) <= PR.JSD_BAND:
            continue  # E5: the route itself may flip; the rest follows the GPU's route
        assert route[h] == res.route, (f"{w}: route gpu {route[h]} oracle {res.route} "
                                       f"(C_struct {res.c_struct:.5f}, D_JS {d_or:.5f})")
        gsets = PR.csr_to_sets(rp, ci, h, nb)
        PR.check_structure(gsets, nb, where=w)
        if res.route == O.ROUTE_VS and op.vs_mode == "gamma":
            PR.compare_vs_gamma(dm[h], res, op.gamma, k_min, where=w)
            for dir_, p_gpu in enumerate((pv[h], ps[h])):  # the selection itself, on the GPU's own scores
                want = O.vs_select_gamma(p_gpu, op.gamma, k_min)
                assert np.nonzero(dm[h, dir_])[0].tolist() == want, f"{w} dir {dir_}: gamma selection on gpu p"
            S_v = np.nonzero(dm[h, 0])[0].tolist()
            S_s = np.nonzero(dm[h, 1])[0].tolist()
            assert gsets == O.vs_block_sets(S_v, S_s, nb), f"{w}: CSR differs from the expansion of its own masks"
        elif res.route == O.ROUTE_VS:
            PR.compare_vs(dm[h], res, op.alpha, k_min, where=w, floor=op.floor_mode)
            S_v = np.nonzero(dm[h, 0])[0].tolist()
            S_s = np.nonzero(dm[h, 1])[0].tolist()
            assert gsets == O.vs_block_sets(S_v, S_s, nb), f"{w}: CSR differs from the expansion of its own masks"
        else:
            assert not dm[h].any()
            PR.compare_pe(gsets, res, op.gamma, where=w)
        if attn:
            qbs = list(range(nb)) if qbs_per_head is None else qbs_per_head(h, nb)
            ref = O.sparse_attention(Q[i], Kg[h // G], Vg[h // G], gsets, block, op.scale(128), qbs=qbs)
            PR.compare_attention(og[h], ref, rows=PR.qb_rows(qbs, block, cfg.seq_len), where=w + " attn(gpu lists)")
            if gsets == res.sets:
                pass  # identical sets: the comparison above is also the end-to-end one
    return route


def test_config0_full_path():
    C = _crisp()
    _say("config 0 (4k tiny) full path")
    params = C.make_params(alpha=CONFIGS[0].alpha)
    route = _check_layer(C, CONFIGS[0], params, where="c0")
    assert route.tolist() == [0, 1]


@pytest.mark.parametrize("n,block,hq,hkv", [(1000, 128, 2, 1), (777, 64, 4, 2), (130, 64, 2, 1), (100, 128, 2, 2),
                                            (4096, 64, 4, 1), (1, 128, 1, 1), (200, 128, 2, 1), (256, 128, 2, 2),
                                            (65, 64, 2, 2), (529, 128, 2, 1), (1553, 128, 2, 2)])
def test_ragged_and_small_layers(n, block, hq, hkv):
    """Ragged tails, one block (n < B, b = n), one token, and exactly two blocks (N_b <= 2:
    every causal pair is selected) through the whole path against the oracle.  The
    estimator takes ranges of at least four blocks, so at n = 529 (N_b = 5) and n = 1553
    (N_b = 13) the last range is the ragged last block alone, which most proxy rows
    cannot see (their running max stays -inf there)."""
    C = _crisp()
    _say(f"ragged layer n={n} B={block} hq={hq} hkv={hkv}")
    cfg = custom_config(n, hq, hkv, block=block, config_id=100 + n % 97)
    _check_layer(C, cfg, C.make_params(), where=f"n{n}")


def _random_cases(count=24, seed=20260901):
    """Seeded random small layers and parameter sets (the same list every run)."""
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        block = int(rng.choice([64, 128]))
        hq, hkv = [(2, 1), (4, 2), (6, 3), (8, 2), (4, 4), (5, 1)][int(rng.integers(6))]
        n = int(rng.integers(65, 3001))
        route_mode, vs_mode = [(0, 0), (1, 1), (0, 1), (1, 0)][int(rng.integers(4))]
        cases.append(dict(
            n=n, block=block, hq=hq, hkv=hkv, config_id=200 + i,
            diffuse_frac=float(rng.choice([0.25, 0.5, 0.75])), structured_pe=bool(n >= 1024 and rng.random() < 0.5),
            params=dict(alpha=float(rng.choice([0.5, 0.75, 1.0, 1.5, 2.0])),
                        gamma=float(rng.choice([0.8, 0.9, 0.95, 1.0])),
                        tau_proxy=float(rng.choice([0.1, 0.2, 0.3])),
                        w_sink=int(rng.choice([0, 64, 128, 300])), w_local=int(rng.choice([0, 128, 500])),
                        k_min_blocks=int(rng.choice([0, 1, 3, 8])),
                        softmax_scale=float(rng.choice([0.0, 0.05, 0.1])),
                        route_mode=route_mode, vs_mode=vs_mode,
                        floor_mode=int(rng.integers(2)) if vs_mode == 0 else 0)))
    return cases


@pytest.mark.parametrize("case", _random_cases(), ids=lambda c: f"n{c['n']}-b{c['block']}-{c['hq']}x{c['hkv']}")
def test_random_layers_and_parameters(case):
    """Seeded random small layers (length, block, GQA grouping, head mixture) under random
    parameters (alpha, gamma, tau, anchor windows, k_min, scale, route and VS modes, floor)
    through the whole path against the oracle, every head and query block."""
    C = _crisp()
    _say(f"random layer {case}")
    cfg = custom_config(case["n"], case["hq"], case["hkv"], block=case["block"], config_id=case["config_id"],
                        diffuse_frac=case["diffuse_frac"], structured_pe=case["structured_pe"])
    _check_layer(C, cfg, C.make_params(**case["params"]), where=f"random{case['config_id']}")


@pytest.mark.parametrize("n,hq,hkv,block", [(4000, 12, 3, 128), (3000, 10, 5, 64), (2500, 32, 16, 128)])
def test_unusual_gqa_groupings(n, hq, hkv, block):
    """KV-group counts that do not divide 8 (the sparse kernel's queues then leave some XCDs
    without a home queue; they take work from the others) and more groups than XCDs (several
    groups per queue), through the whole path against the oracle."""
    C = _crisp()
    _say(f"GQA grouping n={n} hq={hq} hkv={hkv} B={block}")
    cfg = custom_config(n, hq, hkv, block=block, config_id=150 + hkv)
    _check_layer(C, cfg, C.make_params(), qbs_per_head=lambda h, nb: [0, nb // 2, nb - 1], where=f"gqa{hq}x{hkv}")


@pytest.mark.parametrize("tau", [0.0, 1.5])
def test_forced_routes_and_params(tau):
    C = _crisp()
    _say(f"forced route tau={tau}")
    cfg = custom_config(3000, 4, 2, block=128, config_id=131)
    params = C.make_params(tau_proxy=tau, alpha=1.25, gamma=0.9, w_sink=64, w_local=200, k_min_blocks=3)
    route = _check_layer(C, cfg, params, where=f"tau{tau}")
    assert (route == (0 if tau == 0.0 else 1)).all()


def test_config1_every_head():
    """The 32k Llama-3-8B layer: every head's scores, route and block sets against the
    oracle, and the attention rows of six query blocks per head."""
    C = _crisp()
    _say("config 1 (32k Llama shape), every head, sampled query blocks")
    cfg = CONFIGS[1]
    qsel = lambda h, nb: sorted({0, 1, nb // 3, nb // 2, nb - 2, nb - 1})
    _check_layer(C, cfg, C.make_params(), qbs_per_head=qsel, where="c1")


def _check_head_lists(res, gsets, nb, op, block, where):
    """One head's block lists against the oracle's: VS rows exact outside the E1/E2 bands,
    PE pairs exact outside the E4 band."""
    PR.check_structure(gsets, nb, where=where)
    if res.route == O.ROUTE_VS:
        assert gsets == [sorted(set(s_)) for s_ in gsets]
        diff = [qb for qb in range(nb) if set(gsets[qb]) != set(res.sets[qb])]
        if diff:   # the direction sets may differ only inside the E1/E2 bands
            ex_v = PR.vs_direction_exempt(res.p_v, op.alpha, op.k_min(block))[1]
            ex_s = PR.vs_direction_exempt(res.p_s, op.alpha, op.k_min(block))[1]
            for qb in diff:
                for kb in set(gsets[qb]) ^ set(res.sets[qb]):
                    assert kb in ex_v or (nb - 1 - (qb - kb)) in ex_s, f"{where}: row {qb} block {kb}"
    else:
        PR.compare_pe(gsets, res, op.gamma, where=where)


@pytest.mark.parametrize("cid", [2, 3])
def test_full_size_layer_in_bench_launch(cid):
    """The headline layers at full size (128k Llama, 512k Qwen-like), run as bench.py runs them
    (crisp_prefill_attn over the whole layer with the prefill workspace): every head's scores,
    route and block lists against the oracle (list invariants checked on the device too), the
    attention rows of sampled query blocks of a VS and a PE head, the PE head's longest row
    among them, and the dense baseline's first and last query blocks (the last attends to
    every key of the layer) on the first and last head."""
    C = _crisp()
    cfg = CONFIGS[cid]
    block, G = cfg.block, cfg.group
    nb = O.n_blocks(cfg.seq_len, block)
    _say(f"full size {cfg.name}: generate and run the layer")
    q, k, v, specs = make_layer(cfg, device=DEV)
    params = C.make_params(alpha=cfg.alpha)
    ws = C.workspace(C.shape_of(q, k, block), DEV, prefill=True)
    o = torch.empty_like(q)
    C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o)
    o2, route_d, rp_d, ci_d = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
    cs, pv, ps = C.crisp_estimate(q, k, params, block)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)
    for h in range(cfg.n_q_heads):
        _check_rows_on_gpu(rp_d[h], ci_d[h], nb, f"{cfg.name} h{h}")
    route, rp = route_d.cpu().numpy(), rp_d.cpu().numpy()
    cs, pv, ps = cs.cpu().numpy(), pv.cpu().numpy(), ps.cpu().numpy()
    op = _oracle_params(params, block)
    hv = next(h for h in range(cfg.n_q_heads) if specs[h].kind == "concentrated")
    hp = next(h for h in range(cfg.n_q_heads) if specs[h].kind == "diffuse")
    full_lists = range(cfg.n_q_heads)
    Kc, Vc = {}, {}
    for h in range(cfg.n_q_heads):
        g = h // G
        if g not in Kc:
            Kc = {g: to_f64(k[g])}
            Vc = {g: to_f64(v[g])}
        w = f"{cfg.name} h{h} ({specs[h].kind})"
        Qh = to_f64(q[h])
        if h in full_lists:
            _say(f"  oracle for {w}")
            res = O.crisp_head(Qh, Kc[g], None, block, op, attend=False)
        else:
            ahat = O.proxy_attention(Qh, Kc[g], block, op.scale(128))
            res = O.HeadResult(route=0, c_struct=O.c_struct(ahat, cfg.seq_len, op.w_sink, op.w_local),
                               p_v=None, p_s=None)
            _, _, res.p_v, res.p_s = O.vs_scores(ahat, cfg.seq_len, block)
            res.route = O.route(res.c_struct, op.tau_proxy)
            del ahat
        PR.compare_scores(cs[h], pv[h], ps[h], res, where=w)
        assert route[h] == res.route, f"{w}: route gpu {route[h]} oracle {res.route}"
        if h in full_lists:
            cih = ci_d[h, :int(rp[h, nb])].cpu().numpy()
            gsets = [cih[rp[h, qb]:rp[h, qb + 1]].tolist() for qb in range(nb)]
            _check_head_lists(res, gsets, nb, op, block, w)
            if h in (hv, hp):
                # the PE head also at its longest row (the lazy rescale and the float32
                # running sums over the most tiles any unit of the layer takes)
                longest = int(np.argmax(np.diff(rp[h])))
                qbs = [0, nb // 2, nb - 1] if h == hv else sorted({1, nb // 8, longest})
                _say(f"  attention rows for {w} (query blocks {qbs}; longest row {longest}: "
                     f"{int(rp[h, longest + 1] - rp[h, longest])} blocks)")
                ref = O.sparse_attention(Qh, Kc[g], Vc[g], gsets, block, op.scale(128), qbs=qbs)
                PR.compare_attention(to_f64(o[h]), ref, rows=PR.qb_rows(qbs, block, cfg.seq_len), where=w + " attn")
                del ref
            del gsets
        del Qh, res
    # the dense baseline's last query block (every key of the layer) and its first
    _say(f"  dense baseline rows of {cfg.name}")
    od = C.crisp_dense_attn(q, k, v, block)
    torch.cuda.synchronize()
    for h in (0, cfg.n_q_heads - 1):
        g = h // G
        Kh, Vh, Qh = to_f64(k[g]), to_f64(v[g]), to_f64(q[h])
        sets = [[] for _ in range(nb)]
        sets[0], sets[nb - 1] = [0], list(range(nb))
        ref = O.sparse_attention(Qh, Kh, Vh, sets, block, op.scale(128), qbs=[0, nb - 1])
        PR.compare_attention(to_f64(od[h]), ref, rows=PR.qb_rows([0, nb - 1], block, cfg.seq_len),
                             where=f"{cfg.name} h{h} dense")
        del Kh, Vh, Qh, ref


@pytest.mark.parametrize("block", [64, 128])
def test_long_layer_one_unit_per_workgroup(block):
    """From 512k tokens on the sparse kernel runs one unit per workgroup from a single
    longest-first list; below that, a persistent grid.  At a ragged length past 512k, with
    a few heads of one KV group, the result equals the fixed-order launch bit for bit (every
    unit is computed the same way whichever workgroup takes it), and sampled rows of the
    longest query blocks match the oracle."""
    C = _crisp()
    n = (1 << 19) + 77
    cfg = custom_config(n, 3, 1, block=block, config_id=180 + block // 64)
    _say(f"one unit per workgroup: {cfg.name}")
    q, k, v, _ = make_layer(cfg, device=DEV)
    o, route, rp, ci = C.crisp_prefill_attn(q, k, v, C.make_params(), block, return_lists=True)
    fixed = C.crisp_sparse_attn(q, k, v, rp, ci, block, balance=False)
    torch.cuda.synchronize()
    assert torch.equal(o, fixed)
    nb = O.n_blocks(n, block)
    rpn, cin = rp.cpu().numpy(), ci.cpu().numpy()
    for h in range(cfg.n_q_heads):
        gsets = PR.csr_to_sets(rpn, cin, h, nb)
        PR.check_structure(gsets, nb, where=f"{cfg.name} h{h}")
        qbs = [nb - 1] if h else [0, nb - 2, nb - 1]
        Qh, Kh, Vh = to_f64(q[h]), to_f64(k[0]), to_f64(v[0])
        ref = O.sparse_attention(Qh, Kh, Vh, gsets, block, 1.0 / math.sqrt(128), qbs=qbs)
        PR.compare_attention(to_f64(o[h]), ref, rows=PR.qb_rows(qbs, block, n), where=f"{cfg.name} h{h}")
        del Qh, Kh, Vh


def _check_rows_on_gpu(rp, ci, nb, where):
    """Structural invariants of one head's CSR, on the device: rows non-empty, ascending and
    unique, within [0, qb], first entry 0 and last entry qb."""
    r = rp.long()
    tot = int(r[-1])
    c = ci[:tot].long()
    starts, ends = r[:-1], r[1:]
    assert bool((ends > starts).all()), f"{where}: empty row"
    qbs = torch.arange(nb, device=c.device)
    assert bool((c[starts] == 0).all()) and bool((c[ends - 1] == qbs).all()), f"{where}: forced blocks"
    rowid = torch.repeat_interleave(qbs, ends - starts)
    assert bool((c >= 0).all()) and bool((c <= rowid).all()), f"{where}: block outside [0, qb]"
    same_row = rowid[1:] == rowid[:-1]
    assert bool((c[1:][same_row] > c[:-1][same_row]).all()), f"{where}: row not ascending"


def test_max_length_layer():
    """The longest supported layer: 2^21 tokens (N_b = 16384 at B = 128), 17 query heads on
    one KV head.  Head 16's CSR region starts past 2^31 entries, so every offset on the path
    must be 64-bit.  Every head: structural invariants.  Head 16 and the last head of the
    other route: scores and route against the oracle, a VS head's sets exactly (E1/E2), a
    PE head's pairs against the oracle's A_tilde threshold (E4; the full pair sort is too
    large here), and sampled attention rows."""
    C = _crisp()
    n, block, hq = 1 << 21, 128, 17
    nb = n // block
    cfg = custom_config(n, hq, 1, block=block, config_id=190)
    _say(f"max length: {cfg.name}: generate and run the layer")
    q, k, v, specs = make_layer(cfg, device=DEV)
    params = C.make_params()
    o, route, rp, ci = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
    cs, pv, ps = C.crisp_estimate(q, k, params, block)
    torch.cuda.synchronize()
    assert ci.shape[1] * (hq - 1) > 2 ** 31 - 1
    for h in range(hq):
        _check_rows_on_gpu(rp[h], ci[h], nb, f"max length h{h}")
    route = route.cpu().numpy()
    cs, pv, ps = cs.cpu().numpy(), pv.cpu().numpy(), ps.cpu().numpy()
    op = _oracle_params(params, block)
    s = op.scale(128)
    last = hq - 1
    other = max(h for h in range(hq) if specs[h].kind != specs[last].kind)
    Kh, Vh = to_f64(k[0]), to_f64(v[0])
    for h in (last, other):
        w = f"max length h{h} ({specs[h].kind})"
        _say(f"  oracle for {w}")
        Qh = to_f64(q[h])
        ahat = O.proxy_attention(Qh, Kh, block, s)
        res = O.HeadResult(route=0, c_struct=O.c_struct(ahat, n, op.w_sink, op.w_local), p_v=None, p_s=None)
        _, _, res.p_v, res.p_s = O.vs_scores(ahat, n, block)
        del ahat
        res.route = O.route(res.c_struct, op.tau_proxy)
        PR.compare_scores(cs[h], pv[h], ps[h], res, where=w)
        assert route[h] == res.route, f"{w}: route gpu {route[h]} oracle {res.route}"
        rph = rp[h].cpu().numpy().astype(np.int64)
        cih = ci[h, :int(rph[-1])].cpu().numpy()
        if res.route == O.ROUTE_VS:
            km = op.k_min(block)
            sets = O.vs_block_sets(O.vs_select(res.p_v, op.alpha, km), O.vs_select(res.p_s, op.alpha, km), nb)
            gsets = [cih[rph[qb]:rph[qb + 1]].tolist() for qb in range(nb)]
            ex_v = PR.vs_direction_exempt(res.p_v, op.alpha, km)[1]
            ex_s = PR.vs_direction_exempt(res.p_s, op.alpha, km)[1]
            for qb in range(nb):
                for kb in set(gsets[qb]) ^ set(sets[qb]):
                    assert kb in ex_v or (nb - 1 - (qb - kb)) in ex_s, f"{w}: row {qb} block {kb}"
            qbs = [0, nb // 2, nb - 1]
        else:
            At = O.pe_scores(Qh, Kh, block, s)
            PR.check_pe_threshold(rph, cih, At, op.gamma, where=w)
            del At
            qbs = [1, nb // 64]
            gsets = [[] for _ in range(nb)]
            for qb in qbs:
                gsets[qb] = cih[rph[qb]:rph[qb + 1]].tolist()
        _say(f"  attention rows for {w}")
        ref = O.sparse_attention(Qh, Kh, Vh, gsets, block, s, qbs=qbs)
        rows = PR.qb_rows(qbs, block, n)
        PR.compare_attention(to_f64(o[h][torch.from_numpy(rows).to(DEV)]), ref[rows], where=w + " attn")
        del Qh, ref


@pytest.mark.parametrize("alpha,block", [(a, b) for a in (0.5, 1.0, 2.0) for b in (64, 128)])
def test_stress_config4(alpha, block):
    """The 64k selection-stress layer in every cell of alpha x B (Alg. 3 with the noise
    floor of Sec. 4.3): every head's scores, route and block sets against the oracle (the
    three adversarial heads included), and the attention rows of three query blocks per
    head."""
    C = _crisp()
    _say(f"config 4 stress alpha={alpha} B={block}")
    cfg = stress_config(alpha, block)
    qsel = lambda h, nb: sorted({0, nb // 2, nb - 1})
    _check_layer(C, cfg, C.make_params(alpha=alpha), qbs_per_head=qsel, where=cfg.name)


# ------------------------------------------------------------------ FlexPrefill comparator (App. A)

def test_flexprefill_config0_full_path():
    C = _crisp()
    _say("FlexPrefill mode, config 0 full path")
    route = _check_layer(C, CONFIGS[0], C.flexprefill_params(), where="fp c0")
    assert route.tolist() == [0, 1]


@pytest.mark.parametrize("n,block,hq,hkv,gamma", [(1000, 128, 2, 1, 0.95), (777, 64, 4, 2, 0.9),
                                                  (4096, 64, 4, 1, 0.95), (3000, 128, 4, 2, 1.0)])
def test_flexprefill_ragged_and_gamma(n, block, hq, hkv, gamma):
    C = _crisp()
    _say(f"FlexPrefill mode n={n} B={block} hq={hq} hkv={hkv} gamma={gamma}")
    cfg = custom_config(n, hq, hkv, block=block, config_id=150 + n % 89)
    _check_layer(C, cfg, C.flexprefill_params(gamma=gamma), where=f"fp n{n}")


@pytest.mark.parametrize("seq_len", [65536])
def test_structured_pe_workload(seq_len):
    """The paper-like workload of the length sweep (structured PE heads whose pooled scores
    concentrate, Llama GQA shape): every head's scores, route and lists against the oracle,
    and the attention rows of two query blocks per head."""
    C = _crisp()
    cfg = structured_pe_config(seq_len)
    _say(f"structured-PE workload {cfg.name}, every head")
    _check_layer(C, cfg, C.make_params(), qbs_per_head=lambda h, nb: [nb // 3, nb - 1], where=cfg.name)


def test_flexprefill_full_size_128k():
    """The comparator (App. A) at the headline 128k layer: every head's D_JS, route (E5),
    gamma VS masks (E6, and bit-exact on the GPU's own scores) or PE pairs (E4), and the
    attention rows of each head's last query block."""
    C = _crisp()
    _say("FlexPrefill comparator at 128k, every head")
    cfg = CONFIGS[2]
    _check_layer(C, cfg, C.flexprefill_params(alpha=cfg.alpha), qbs_per_head=lambda h, nb: [nb - 1],
                 where="fp128k")


def test_flexprefill_config1_sampled():
    C = _crisp()
    _say("FlexPrefill mode, config 1 (32k), 8 heads, sampled query blocks")
    heads = [0, 1, 3, 8, 11, 17, 21, 31]
    qsel = lambda h, nb: sorted({0, 1, nb // 2, nb - 1})
    _check_layer(C, CONFIGS[1], C.flexprefill_params(), heads=heads, qbs_per_head=qsel, where="fp c1")


@pytest.mark.parametrize("route_mode,vs_mode,tau_jsd", [(0, 1, 0.1), (1, 0, 0.1), (1, 1, 0.0), (1, 1, 2.0)])
def test_comparator_mixes_and_forced_routes(route_mode, vs_mode, tau_jsd):
    """The two ablation mixes (C_struct + gamma, JSD + sink-aware floor) and forced JSD routes."""
    C = _crisp()
    _say(f"comparator mix route_mode={route_mode} vs_mode={vs_mode} tau_jsd={tau_jsd}")
    cfg = custom_config(6000, 4, 2, block=128, config_id=161)
    params = C.make_params(route_mode=route_mode, vs_mode=vs_mode, tau_jsd=tau_jsd, k_min_blocks=2)
    route = _check_layer(C, cfg, params, where=f"mix{route_mode}{vs_mode}")
    if route_mode == 1 and tau_jsd == 0.0:
        assert (route == 0).all()
    if route_mode == 1 and tau_jsd == 2.0:
        assert (route == 1).all()


@pytest.mark.parametrize("alpha,block,n", [(1.0, 128, 6000), (0.75, 64, 3001), (1.5, 128, 300)])
def test_median_floor(alpha, block, n):
    """App. H's median noise floor against the oracle (odd and even non-anchor counts)."""
    C = _crisp()
    _say(f"median floor alpha={alpha} B={block} n={n}")
    cfg = custom_config(n, 4, 2, block=block, config_id=170 + n % 53)
    _check_layer(C, cfg, C.make_params(alpha=alpha, floor_mode=C.FLOOR_MEDIAN, k_min_blocks=1), where=f"med{n}")


def test_median_floor_stress_config4():
    C = _crisp()
    _say("median floor on the config 4 stress layer")
    cfg = stress_config(1.0, 128)
    qsel = lambda h, nb: sorted({0, nb // 2, nb - 1})
    _check_layer(C, cfg, C.make_params(floor_mode=C.FLOOR_MEDIAN), heads=[0, 1, 2, 5, 13], qbs_per_head=qsel,
                 where="med stress")


@pytest.mark.parametrize("n,hq,hkv,block", [(8192, 16, 4, 64), (6000, 24, 8, 128)])
def test_short_layer_one_workgroup_per_unit(n, hq, hkv, block):
    """Short layers with at least as many (head, query block) units as the persistent grid
    holds run one workgroup per unit from one longest-first list (B = 64: 2048 units; B =
    128: 1128 units, ragged tail): every head's selection and sampled attention rows
    against the oracle, and the balanced launch equal to the fixed-order one bit for bit
    (no row is split)."""
    C = _crisp()
    _say(f"short layer, one workgroup per unit: n={n} {hq}/{hkv} B={block}")
    cfg = custom_config(n, hq, hkv, block=block, config_id=157 + block)
    qsel = lambda h, nb: sorted({0, 1, nb // 2, nb - 2, nb - 1})
    _check_layer(C, cfg, C.make_params(), qbs_per_head=qsel, where=f"one-per-unit n{n} B{block}")
    q, k, v, _ = make_layer(cfg, device=DEV)
    o, _, rp, ci = C.crisp_prefill_attn(q, k, v, C.make_params(), block, return_lists=True)
    o_fixed = C.crisp_sparse_attn(q, k, v, rp, ci, block, balance=False)
    torch.cuda.synchronize()
    assert torch.equal(o, o_fixed)


@pytest.mark.parametrize("n,block", [(4000, 128), (777, 64)])
def test_context_length_gate_is_dense(n, block):
    """Below the gate, prefill equals the dense kernel bit for bit and reports dense routes and
    full causal lists; at the gate length it runs the sparse path again."""
    C = _crisp()
    _say(f"context-length gate n={n} B={block}")
    cfg = custom_config(n, 4, 2, block=block, config_id=180 + n % 31)
    q, k, v, _ = make_layer(cfg, device=DEV)
    gated = C.make_params(dense_below_len=n + 1)
    o1, route, rp, ci = C.crisp_prefill_attn(q, k, v, gated, block, return_lists=True)
    o2 = C.crisp_dense_attn(q, k, v, block)
    o3 = C.crisp_prefill_attn(q, k, v, gated, block)
    o4, route4, _, _ = C.crisp_prefill_attn(q, k, v, C.make_params(dense_below_len=n), block, return_lists=True)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(o3, o2)
    assert (route.cpu() == 2).all() and (route4.cpu() != 2).all()
    nb = O.n_blocks(n, block)
    for h in range(4):
        assert PR.csr_to_sets(rp.cpu().numpy(), ci.cpu().numpy(), h, nb) == O.dense_causal_sets(nb)


def test_flexprefill_prefill_matches_stagewise():
    """crisp_prefill_attn in the comparator mode (pattern search inside, pooled K reused) gives the
    lists and output of the stage-by-stage calls."""
    C = _crisp()
    _say("FlexPrefill prefill lists == stages")
    cfg = custom_config(5000, 4, 1, block=128, config_id=141)
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.flexprefill_params()
    _, _, _, route, rp, ci, _ = _run_stages(C, q, k, v, params, 128)
    o1, r2, rp2, ci2 = C.crisp_prefill_attn(q, k, v, params, 128, return_lists=True)
    o2 = C.crisp_sparse_attn(q, k, v, torch.from_numpy(rp).to(DEV), torch.from_numpy(ci).to(DEV), 128)
    torch.cuda.synchronize()
    assert np.array_equal(r2.cpu().numpy(), route) and np.array_equal(rp2.cpu().numpy(), rp)
    nb = O.n_blocks(cfg.seq_len, 128)
    for h in range(4):
        assert PR.csr_to_sets(rp2.cpu().numpy(), ci2.cpu().numpy(), h, nb) == PR.csr_to_sets(rp, ci, h, nb)
    assert torch.equal(o1, o2)


def _stagewise_cases():
    # (name, layer, parameters); up to 64 blocks prefill's selection forms p_v and p_s from
    # the estimator's sums itself, past that it reads the estimator's own p_v and p_s
    return [("5000 4/1", lambda: custom_config(5000, 4, 1, block=128, config_id=140), {}),
            ("pe8k 32/8 nb64", lambda: structured_pe_config(8192), {}),
            ("4000 8/2 B64 median kmin3", lambda: custom_config(4000, 8, 2, block=64, config_id=142),
             dict(floor_mode=1, k_min_blocks=3)),
            ("3000 6/3 gamma VS", lambda: custom_config(3000, 6, 3, block=128, config_id=143), dict(vs_mode=1)),
            ("8320 4/2 nb65", lambda: custom_config(8320, 4, 2, block=128, config_id=144), {})]


@pytest.mark.parametrize("name,make_cfg,kw", _stagewise_cases(), ids=[c[0] for c in _stagewise_cases()])
def test_prefill_lists_match_stagewise(name, make_cfg, kw):
    """crisp_prefill_attn with caller lists reproduces the stage-by-stage calls exactly, on
    either side of the short-layer selection's 64 blocks."""
    C = _crisp()
    _say(f"prefill lists == stages: {name}")
    cfg = make_cfg()
    block = cfg.block
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.make_params(**kw)
    cs, pv, ps, route, rp, ci, _ = _run_stages(C, q, k, v, params, block)
    o1, r2, rp2, ci2 = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
    o2 = C.crisp_sparse_attn(q, k, v, torch.from_numpy(rp).to(DEV), torch.from_numpy(ci).to(DEV), block)
    o3 = C.crisp_prefill_attn(q, k, v, params, block)
    torch.cuda.synchronize()
    assert np.array_equal(r2.cpu().numpy(), route) and np.array_equal(rp2.cpu().numpy(), rp)
    nb = O.n_blocks(cfg.seq_len, block)
    for h in range(cfg.n_q_heads):
        assert PR.csr_to_sets(rp2.cpu().numpy(), ci2.cpu().numpy(), h, nb) == PR.csr_to_sets(rp, ci, h, nb)
    assert torch.equal(o1, o2) and torch.equal(o1, o3)


def test_run_to_run_determinism():
    C = _crisp()
    _say("determinism")
    cfg = custom_config(6000, 8, 2, block=128, config_id=141)
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.make_params()
    a = _run_stages(C, q, k, v, params, 128)
    b = _run_stages(C, q, k, v, params, 128)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_concurrent_streams():
    """The library keeps no state between calls: two layers (different shapes, block sizes
    and parameters) run at the same time on two streams with their own workspaces give
    exactly their results run one after the other."""
    C = _crisp()
    _say("two layers on two streams")
    cfg_a = custom_config(6000, 8, 2, block=128, config_id=151)
    cfg_b = custom_config(5000, 6, 3, block=64, config_id=152)
    pa, pb = C.make_params(), C.make_params(alpha=1.5, gamma=0.9)
    qa, ka, va, _ = make_layer(cfg_a, device=DEV)
    qb, kb, vb, _ = make_layer(cfg_b, device=DEV)
    wa = C.workspace(C.shape_of(qa, ka, 128), DEV, prefill=True)
    wb = C.workspace(C.shape_of(qb, kb, 64), DEV, prefill=True)
    ref_a = C.crisp_prefill_attn(qa, ka, va, pa, 128, ws=wa).clone()
    ref_b = C.crisp_prefill_attn(qb, kb, vb, pb, 64, ws=wb).clone()
    oa, ob = torch.empty_like(qa), torch.empty_like(qb)
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for _ in range(3):
        with torch.cuda.stream(s1):
            C.crisp_prefill_attn(qa, ka, va, pa, 128, ws=wa, out=oa)
        with torch.cuda.stream(s2):
            C.crisp_prefill_attn(qb, kb, vb, pb, 64, ws=wb, out=ob)
        torch.cuda.synchronize()
        assert torch.equal(oa, ref_a) and torch.equal(ob, ref_b)


def test_empty_layer_is_noop():
    C = _crisp()
    _say("empty layer")
    q = torch.zeros(0, 16, 128, dtype=torch.bfloat16, device=DEV)
    k = torch.zeros(1, 16, 128, dtype=torch.bfloat16, device=DEV)
    o = C.crisp_dense_attn(q, k, k, 128)
    assert o.shape == q.shape
    q = torch.zeros(2, 0, 128, dtype=torch.bfloat16, device=DEV)
    k = torch.zeros(1, 0, 128, dtype=torch.bfloat16, device=DEV)
    C.crisp_prefill_attn(q, k, k, C.make_params(), 128)
    torch.cuda.synchronize()


def test_binding_rejects_mismatched_tensors():
    """The C ABI sees only pointers, so the binding checks every tensor's dtype, shape and
    device before a call: a mismatch raises ValueError and nothing is launched."""
    C = _crisp()
    _say("binding validation")
    n, block = 1024, 128
    q, k, v = _rand(4, n).to(DEV), _rand(2, n).to(DEV), _rand(2, n).to(DEV)
    nb = O.n_blocks(n, block)
    rp = torch.zeros(4, nb + 1, dtype=torch.int32, device=DEV)
    ci = torch.zeros(4, nb * (nb + 1) // 2, dtype=torch.int32, device=DEV)
    bad = [
        lambda: C.crisp_dense_attn(q, k, v[:, : n // 2].contiguous()),                       # v shorter than k
        lambda: C.crisp_dense_attn(q, k, _rand(1, n).to(DEV)),                                # v heads != k heads
        lambda: C.crisp_dense_attn(q, _rand(2, n // 2).to(DEV), _rand(2, n // 2).to(DEV)),   # k shorter than q
        lambda: C.crisp_dense_attn(q, k, v, out=torch.empty(4, n, 64, dtype=torch.bfloat16, device=DEV)),
        lambda: C.crisp_sparse_attn(q, k, v, rp[:, :-1].contiguous(), ci),                  # row_ptr one short
        lambda: C.crisp_sparse_attn(q, k, v, rp.long(), ci),                                 # wrong dtype
        lambda: C.crisp_sparse_attn(q, k, v, rp[:2].contiguous(), ci[:2].contiguous()),     # too few heads
        lambda: C.crisp_sparse_attn(q, k, v, rp, ci, ws=torch.empty(64, dtype=torch.float32, device=DEV)),
        lambda: C.crisp_prefill_attn(q, k, v, C.make_params(), block, out=q.float()),
        lambda: C.crisp_jsd(q, k, torch.zeros(4, nb + 1, device=DEV), C.make_params(), block),
        lambda: C.crisp_route_select(q, k, torch.zeros(3, device=DEV), torch.zeros(4, nb, device=DEV),
                                     torch.zeros(4, nb, device=DEV), C.make_params(), block),
    ]
    for i, call in enumerate(bad):
        with pytest.raises(ValueError):
            call()
    torch.cuda.synchronize()


@pytest.mark.parametrize("n,block", [(6000, 128), (4100, 64)])
def test_prefill_in_a_hip_graph(n, block):
    """The whole prefill (estimate, route/select, work lists, attention, merge of split rows)
    enqueues only kernels on the caller's stream -- no allocation, copy, memset or host
    synchronisation -- so it can be captured in a HIP graph.  Each replay, with eager work
    and synchronisations between replays, gives the eager result bit for bit."""
    C = _crisp()
    _say(f"prefill in a HIP graph n={n} B={block}")
    cfg = custom_config(n, 4, 2, block=block, config_id=195 + block // 64)
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.make_params()
    ws = C.workspace(C.shape_of(q, k, block), DEV, prefill=True)
    o_eager = C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=torch.empty_like(q))
    torch.cuda.synchronize()
    o = torch.zeros_like(q)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        C.crisp_prefill_attn(q, k, v, params, block, ws=ws, out=o)
    torch.cuda.synchronize()
    for rep in range(3):
        o.zero_()
        C.crisp_dense_attn(q, k, v, block, out=torch.empty_like(q))  # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, o_eager), f"replay {rep} differs from the eager result"


# ------------------------------------------------------------------ stored values

def test_golden_manifests_on_gpu():
    """The GPU path against values stored in tests/golden/manifests.json (written by the
    oracle-only script beside it): routes exact, C_struct to the stage tolerance; on VS
    heads the block scores p_v, p_s to the stage tolerances and each direction's selected
    blocks against the stored S_v, S_s, exactly outside the E1/E2 bands of the stored
    scores (a direction whose stored residual is below float32 resolution, E3, is checked
    for its forced blocks and k_min only), and the lists against the expansion of the GPU's
    own direction sets; a PE head's pair count to 0.1% of the causal pairs (ties at the
    gamma cutoff may fall either way); and for the layer whose attention is stored, the
    output's mean and largest magnitude to the attention tolerances.  The stored values come from inputs
    drawn by the generator on the CPU (its stream differs by device), so the same heads are
    drawn on the CPU here and copied to the GPU; the other heads of each layer stay zero."""
    import json
    import os
    from workloads import GEN_VERSION
    C = _crisp()
    with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "manifests.json")) as f:
        golden = json.load(f)
    layers = {"tiny-4k": CONFIGS[0], "llama3-8b-32k-heads0-3": CONFIGS[1],
              "stress-64k-a1-b128-adversarial": stress_config(1.0, 128)}
    assert sorted(layers) == sorted(golden)
    for name, cfg in layers.items():
        rec = golden[name]
        assert rec["generator"] == GEN_VERSION and rec["layer"] == cfg.name and rec["seq_len"] == cfg.seq_len
        _say(f"golden manifest {name}")
        heads = [int(h) for h in rec["heads"]]
        q, k, v, _ = (t.to(DEV) if torch.is_tensor(t) else t for t in make_layer(cfg, heads=heads))
        params = C.make_params(alpha=cfg.alpha)
        cs, pv, ps, route, rp, ci, dm = _run_stages(C, q, k, v, params, cfg.block)
        nb = O.n_blocks(cfg.seq_len, cfg.block)
        attend = any("out_mean" in r for r in rec["heads"].values())
        o = C.crisp_prefill_attn(q, k, v, params, cfg.block) if attend else None
        torch.cuda.synchronize()
        for hs, st in rec["heads"].items():
            h = int(hs)
            w = f"{name} h{h}"
            assert (route[h] == O.ROUTE_VS) == (st["route"] == "VS"), f"{w}: route {route[h]} vs {st['route']}"
            assert abs(float(cs[h]) - st["c_struct"]) <= PR.CS_ABS, f"{w}: C_struct {float(cs[h])} vs {st['c_struct']}"
            gsets = PR.csr_to_sets(rp, ci, h, nb)
            pairs = sum(len(s) for s in gsets)
            if st["route"] == "PE":
                assert abs(pairs - st["pairs"]) <= 1e-3 * nb * (nb + 1) / 2, f"{w}: pairs {pairs} vs {st['pairs']}"
                assert not dm[h].any()
            else:
                k_min = -(-1024 // cfg.block)
                stored = O.HeadResult(route=O.ROUTE_VS, c_struct=st["c_struct"], p_v=np.asarray(st["p_v"]),
                                      p_s=np.asarray(st["p_s"]), S_v=st["S_v"], S_s=st["S_s"])
                PR.compare_scores(cs[h], pv[h], ps[h], stored, where=w)
                PR.compare_vs(dm[h], stored, cfg.alpha, k_min, where=w)
                for d in (0, 1):   # also for a degenerate direction (E3)
                    assert int(dm[h, d].sum()) >= min(k_min, nb), f"{w}: direction {d} below k_min"
                PR.check_structure(gsets, nb, where=w)
                S_v, S_s = (np.nonzero(dm[h, d])[0].tolist() for d in (0, 1))
                assert gsets == O.vs_block_sets(S_v, S_s, nb), f"{w}: lists differ from the direction sets"
                if st["S_v"] == S_v and st["S_s"] == S_s:
                    assert pairs == st["pairs"], f"{w}: pairs {pairs} vs {st['pairs']}"
            if attend:
                og = to_f64(o[h])
                assert abs(og.mean() - st["out_mean"]) <= 2e-3, f"{w}: output mean {og.mean()} vs {st['out_mean']}"
                assert abs(np.abs(og).max() - st["out_max_abs"]) <= 2e-2, f"{w}: max |O| {np.abs(og).max()}"
        del q, k, v, o


@pytest.mark.parametrize("layer", ["config0", "ragged-b64", "pe-8k", "16k-split-rows", "one-shot-512k"])
def test_debug_build_race_check(layer):
    """The debug build's attention runs the same arithmetic with its tile pipeline
    serialised (each tile load waited for, a barrier after every LDS phase): its outputs
    equal the pipelined kernel's bit for bit, so the overlapped loads and reads of the
    LDS rings never race.  Layers: the 4k tiny layer, a ragged B = 64 layer, the 8k
    structured layer (one unit per workgroup from one list), a 16k two-head layer whose
    long PE rows are split (persistent grid, partial results merged: checked against the
    unsplit fixed-order launch), and a 512k layer (one unit per workgroup)."""
    C = _crisp()
    _say(f"debug race check {layer}")
    cfg, block = {"config0": (CONFIGS[0], 128), "ragged-b64": (custom_config(3001, 4, 2, block=64, config_id=154), 64),
                  "pe-8k": (structured_pe_config(8192), 128),
                  "16k-split-rows": (custom_config(16384, 2, 1, block=128, config_id=156, tiny=True), 128),
                  "one-shot-512k": (custom_config(1 << 19, 2, 1, block=128, config_id=155), 128)}[layer]
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.make_params(alpha=cfg.alpha)
    release = C.lib
    o_rel, _, rp, ci = C.crisp_prefill_attn(q, k, v, params, block, return_lists=True)
    d_rel = C.crisp_dense_attn(q, k, v, block)
    if layer == "16k-split-rows":
        o_fixed = C.crisp_sparse_attn(q, k, v, rp, ci, block, balance=False)
        torch.cuda.synchronize()
        assert not torch.equal(o_rel, o_fixed), "no row was split"
    torch.cuda.synchronize()
    try:
        C.lib = C._load(C.DEBUG_LIB_PATH)
        o_dbg = C.crisp_prefill_attn(q, k, v, params, block)
        d_dbg = C.crisp_dense_attn(q, k, v, block)
        torch.cuda.synchronize()
    finally:
        C.lib = release
    assert torch.equal(o_dbg, o_rel) and torch.equal(d_dbg, d_rel)


def test_debug_build_checks_inputs():
    """libcrisp_debug.so: on valid inputs the same results as the release library, bit for
    bit; infinite or NaN values in Q, K or V, and caller lists with an entry outside
    [0, qb], entries out of order or a decreasing row_ptr, are CRISP_EINVAL with a
    message naming them, before any of the call's kernels run."""
    C = _crisp()
    _say("debug build input checks")
    release = C.lib
    cfg = custom_config(1000, 2, 1, block=128, config_id=153)
    q, k, v, _ = make_layer(cfg, device=DEV)
    params = C.make_params()
    o_rel, _, rp, ci = C.crisp_prefill_attn(q, k, v, params, 128, return_lists=True)
    s_rel = C.crisp_sparse_attn(q, k, v, rp, ci, 128)
    d_rel = C.crisp_dense_attn(q, k, v, 128)
    torch.cuda.synchronize()
    try:
        C.lib = C._load(C.DEBUG_LIB_PATH)
        assert torch.equal(C.crisp_prefill_attn(q, k, v, params, 128), o_rel)
        assert torch.equal(C.crisp_sparse_attn(q, k, v, rp, ci, 128), s_rel)
        assert torch.equal(C.crisp_dense_attn(q, k, v, 128), d_rel)

        def rejects(fn, text):
            with pytest.raises(C.CrispError) as err:
                fn()
            assert err.value.status == C.CRISP_EINVAL and text in str(err.value), str(err.value)

        kn = k.clone()
        kn[0, 517, 33] = float("nan")
        rejects(lambda: C.crisp_prefill_attn(q, kn, v, params, 128), "k holds")
        rejects(lambda: C.crisp_estimate(q, kn, params, 128), "k holds")
        qi = q.clone()
        qi[1, 999, 127] = float("inf")
        rejects(lambda: C.crisp_dense_attn(qi, k, v, 128), "q holds")
        vi = v.clone()
        vi[0, 0, 0] = float("-inf")
        rejects(lambda: C.crisp_sparse_attn(q, k, vi, rp, ci, 128), "v holds")
        nb = O.n_blocks(1000, 128)
        cap = ci.shape[1]
        # head 0, last row: one entry past the diagonal
        bad = ci.clone()
        last = int(rp[0, nb - 1])
        bad[0, last] = nb
        rejects(lambda: C.crisp_sparse_attn(q, k, v, rp, bad, 128), "outside [0, qb]")
        # head 1, row 3 holds {0, 3} and more: swap two entries
        bad = ci.clone()
        b3 = int(rp[1, 3])
        bad[1, b3], bad[1, b3 + 1] = ci[1, b3 + 1], ci[1, b3]
        rejects(lambda: C.crisp_sparse_attn(q, k, v, rp, bad, 128), "strictly increasing")
        badp = rp.clone()
        badp[0, 2] = badp[0, 1] - 1
        rejects(lambda: C.crisp_sparse_attn(q, k, v, badp, ci, 128), "row_ptr")
        badp = rp.clone()
        badp[1, nb] = cap + 1
        rejects(lambda: C.crisp_sparse_attn(q, k, v, badp, ci, 128), "row_ptr")
        torch.cuda.synchronize()
    finally:
        C.lib = release
