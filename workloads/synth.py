"""Seeded synthetic layer inputs with the mass structure CRISP is built around.

The paper measures real Llama-3.1-8B / Qwen2.5-7B prefill activations on
InfiniteBench-style inputs (Sec. 5, Setup).  Neither weights nor datasets are
available here, so these generators stand in for them: they produce bf16
Q [H_q, n, d], K and V [H_kv, n, d] with the paper's layer shapes (d = 128,
GQA) and plant the structures the paper names -- attention sinks on the first
tokens, vertical columns, slash diagonals, a local window (Sec. 4.1, App. F) --
on "concentrated" heads, while "diffuse" heads are i.i.d. noise.

Every tensor is drawn from its own torch generator seeded by
(BASE_SEED, config id, variant, role, index), so one head or one KV group can be
regenerated alone, on CPU or GPU.  The same device and seed always give the same
bits.  Values are built in fp32 (fp64 for the running sums of the local code) and
rounded once to bf16 (round-to-nearest-even); the bf16 tensors are what every
consumer sees.

Strengths are in nats: a planted logit of ln(n / m) + s on m keys gives those
keys a mass that does not change with n, so only the count of background keys
grows with n -- the regime of the paper's mass-cliff analysis (App. C).  The
local window is a fixed boost of about LOCAL_PEAK nats instead.

Key layout per KV group (d = 128):
  dims   0..47   local code: box-filtered white noise (window 128), rows scaled to
                 norm sqrt(48); q_i . k_j is large when |i - j| < 128
  dims  48..111  slash code: i.i.d. rows scaled to norm 8; a query that carries
                 k_{i-o}'s code attends to the diagonal at offset o
  dim  112       sink tag: TAG on keys 0..3, else 0
  dims 113..127  vertical tags: TAG on one planted column each (15 per group)
Configs with `structured_pe` (the paper-like PE workload) give dims 96..111 to a
smooth position code instead (the slash code keeps dims 48..95, rows still of
norm 8): SMOOTH_SCALE * (cos, sin)(2 pi m j / n) for m = 1..8.  Their PE heads
("structured") carry a few of these frequencies, so every query prefers keys by
a gently varying log-weight sum_m A_m cos(2 pi m j / n - phi_m) of 1.5-5 nats:
block masses that decay smoothly with no floor to cut, whose top-50 blocks hold
a fraction of the mass rather than almost all of it (App. B's diffuse heads).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

import numpy as np
import torch

GEN_VERSION = "gen-v1"
BASE_SEED = 260901925
HEAD_DIM = 128
TAG = 8.0                  # value of a tag coordinate on a planted key
N_SINKS = 4                # keys 0..3 carry the sink tag
N_GROUP_COLUMNS = 15       # planted vertical columns per KV group
LOCAL_DIMS = (0, 48)
SLASH_DIMS = (48, 112)
SINK_DIM = 112
VERT_DIM0 = 113
LOCAL_WINDOW = 128         # box filter width of the local code
BG_SIGMA = 0.5             # std of the per-query background direction (concentrated heads)
SMOOTH_DIMS = (96, 112)    # smooth position code of structured-PE configs (8 frequencies x cos, sin)
SMOOTH_SCALE = 4.0
LOCAL_PEAK = 2.5           # local-window logit boost at |i - j| = 0, in nats (not length-scaled:
                           # neighbouring queries share the local code, so its cross-talk on far
                           # keys does not average out over the proxy rows and must stay small)

ROLE_Q, ROLE_K, ROLE_V, ROLE_STRUCT = 0, 1, 2, 3


@dataclass(frozen=True)
class LayerConfig:
    """One attention layer's shape plus its head mixture."""
    name: str
    config_id: int
    seq_len: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int = HEAD_DIM
    block: int = 128
    alpha: float = 1.0
    diffuse_frac: float = 0.4
    vertical_range: str = "tail"   # "tail": columns in [4, n - 2B); "half": [4, n / 2)
    tiny: bool = False             # head 0 concentrated, head 1 diffuse with i.i.d. K
    adversarial: bool = False      # heads 0..2 replaced by the three stress heads
    variant: int = 0
    structured_pe: bool = False    # PE heads carry a smooth key preference (see module notes)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads


@dataclass(frozen=True)
class HeadSpec:
    """Structure planted on one query head (strengths in nats, see module doc)."""
    kind: str                                   # concentrated | diffuse | sink_collapse | flat | floor
    s_sink: float = 0.0
    verticals: Tuple[int, ...] = ()             # indices into the group's planted columns
    s_vert: Tuple[float, ...] = ()
    slash_offsets: Tuple[int, ...] = ()
    s_slash: Tuple[float, ...] = ()
    s_loc: float = 0.0
    smooth: Tuple[Tuple[int, float, float], ...] = ()   # structured PE: (cycles m, amplitude A, phase phi)


CONFIGS = {
    0: LayerConfig("tiny-4k", 0, 4096, 2, 2, tiny=True),
    1: LayerConfig("llama3-8b-32k", 1, 32768, 32, 8),
    2: LayerConfig("llama3-8b-128k", 2, 131072, 32, 8),
    3: LayerConfig("qwen2-7b-512k", 3, 524288, 28, 4, diffuse_frac=0.5, vertical_range="half"),
}

STRESS_ALPHAS = (0.5, 1.0, 2.0)
STRESS_BLOCKS = (64, 128)


PE_SWEEP_LENGTHS = (8192, 65536, 131072, 262144, 524288, 16384, 32768, 2048, 4096)   # variant = position here


def structured_pe_config(seq_len: int = 131072) -> LayerConfig:
    """The paper-like PE workload: the Llama-3-8B GQA mix (60% concentrated heads) whose other
    heads are structured PE heads instead of i.i.d. noise; one config per length of the sweep."""
    return LayerConfig(f"llama3-8b-pe-{seq_len // 1024}k", 5, seq_len, 32, 8, structured_pe=True,
                       variant=PE_SWEEP_LENGTHS.index(seq_len) if seq_len in PE_SWEEP_LENGTHS else 99)


def stress_config(alpha: float, block: int) -> LayerConfig:
    """Selection-stress layer at 64k (Llama GQA shape) with the three adversarial heads."""
    variant = STRESS_ALPHAS.index(alpha) * len(STRESS_BLOCKS) + STRESS_BLOCKS.index(block)
    return LayerConfig(f"stress-64k-a{alpha:g}-b{block}", 4, 65536, 32, 8, block=block,
                       alpha=alpha, adversarial=True, variant=variant)


def _seed(cfg: LayerConfig, role: int, index: int) -> int:
    ss = np.random.SeedSequence([BASE_SEED, cfg.config_id, cfg.variant, role, index])
    return int(ss.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1))


def _torch_gen(cfg: LayerConfig, role: int, index: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(cfg, role, index))
    return g


def _np_rng(cfg: LayerConfig, role: int, index: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([BASE_SEED, cfg.config_id, cfg.variant, role, index]))


def kv_group_columns(cfg: LayerConfig, g: int) -> Tuple[int, ...]:
    """The 15 planted vertical key positions of KV group g (sorted, distinct)."""
    n, blk = cfg.seq_len, cfg.block
    hi = n // 2 if cfg.vertical_range == "half" else n - 2 * blk
    lo = N_SINKS
    if hi - lo < N_GROUP_COLUMNS:
        return ()
    rng = _np_rng(cfg, ROLE_STRUCT, 1000 + g)
    cols = rng.choice(np.arange(lo, hi), size=N_GROUP_COLUMNS, replace=False)
    return tuple(int(c) for c in np.sort(cols))


def _offset_range(n: int, blk: int) -> np.ndarray:
    """Slash offsets are drawn from [B, n/2); short sequences fall back to [1, n)."""
    if n // 2 - blk >= 8:
        return np.arange(blk, n // 2)
    return np.arange(1, max(n, 9))


def head_specs(cfg: LayerConfig) -> List[HeadSpec]:
    """Per query head structure, drawn from the config's structure stream."""
    n, blk, H = cfg.seq_len, cfg.block, cfg.n_q_heads
    rng = _np_rng(cfg, ROLE_STRUCT, 0)
    if cfg.tiny:
        cols = rng.choice(N_GROUP_COLUMNS, size=3, replace=False)
        offs = rng.choice(_offset_range(n, blk), size=2, replace=False)
        conc = HeadSpec("concentrated", s_sink=6.0, verticals=tuple(int(c) for c in cols),
                        s_vert=(0.0, 0.0, 0.0), slash_offsets=tuple(int(o) for o in offs),
                        s_slash=(0.5, 0.5))
        return [conc, HeadSpec("diffuse")]
    n_diffuse = int(round(cfg.diffuse_frac * H))
    perm = rng.permutation(H)
    diffuse = set(int(h) for h in perm[:n_diffuse])
    specs = []
    for h in range(H):
        if h in diffuse and cfg.structured_pe:
            n_f = int(rng.integers(1, 4))
            ms = rng.choice(np.arange(1, 9), size=n_f, replace=False)
            total = float(rng.uniform(1.5, 5.0))
            w = rng.dirichlet(np.ones(n_f))
            ph = rng.uniform(0.0, 2 * math.pi, size=n_f)
            specs.append(HeadSpec("structured", smooth=tuple((int(m), float(total * wi), float(p))
                                                             for m, wi, p in zip(ms, w, ph))))
            continue
        if h in diffuse:
            specs.append(HeadSpec("diffuse"))
            continue
        n_vert = int(rng.integers(1, 9))
        n_slash = int(rng.integers(1, 5))
        verts = rng.choice(N_GROUP_COLUMNS, size=n_vert, replace=False)
        offs = rng.choice(_offset_range(n, blk), size=n_slash, replace=False)
        specs.append(HeadSpec(
            "concentrated",
            s_sink=float(rng.uniform(2.0, 8.0)),
            verticals=tuple(int(v) for v in verts),
            s_vert=tuple(float(x) for x in rng.uniform(-1.5, 0.0, size=n_vert)),
            slash_offsets=tuple(int(o) for o in offs),
            s_slash=tuple(float(x) for x in rng.uniform(0.0, 1.0, size=n_slash)),
            s_loc=float(rng.uniform(-0.5, 0.5)),
        ))
    if cfg.adversarial:
        specs[0] = HeadSpec("sink_collapse")
        specs[1] = HeadSpec("flat")
        specs[2] = HeadSpec("floor")
    return specs


def _key_parts(cfg: LayerConfig, g: int, device) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Local code [n, 48], slash code [n, 64], tags [n, 16] of KV group g, fp32."""
    n = cfg.seq_len
    gen = _torch_gen(cfg, ROLE_K, g, device)
    nl = LOCAL_DIMS[1] - LOCAL_DIMS[0]
    ns = SLASH_DIMS[1] - SLASH_DIMS[0]
    white = torch.randn(n + LOCAL_WINDOW - 1, nl, generator=gen, device=device, dtype=torch.float32)
    c = torch.cumsum(white.double(), dim=0)
    c = torch.cat([torch.zeros(1, nl, device=device, dtype=torch.float64), c], dim=0)
    loc = (c[LOCAL_WINDOW:] - c[:n]).float()           # sum of LOCAL_WINDOW consecutive white rows
    loc = loc * (math.sqrt(nl) / loc.norm(dim=1, keepdim=True).clamp_min(1e-20))
    sl = torch.randn(n, ns, generator=gen, device=device, dtype=torch.float32)
    if cfg.structured_pe:
        nsm = SMOOTH_DIMS[1] - SMOOTH_DIMS[0]
        sl = sl[:, : ns - nsm]
        sl = sl * (8.0 / sl.norm(dim=1, keepdim=True).clamp_min(1e-20))
        j = torch.arange(n, device=device, dtype=torch.float64)
        cols = []
        for m in range(1, nsm // 2 + 1):
            ang = (2 * math.pi * m / n) * j
            cols += [torch.cos(ang), torch.sin(ang)]
        sl = torch.cat([sl, (SMOOTH_SCALE * torch.stack(cols, dim=1)).float()], dim=1)
    else:
        sl = sl * (8.0 / sl.norm(dim=1, keepdim=True).clamp_min(1e-20))
    tags = torch.zeros(n, HEAD_DIM - SINK_DIM, device=device, dtype=torch.float32)
    tags[: min(N_SINKS, n), 0] = TAG
    for c_i, col in enumerate(kv_group_columns(cfg, g)):
        tags[col, 1 + c_i] = TAG
    return loc, sl, tags


def _query_head(cfg: LayerConfig, h: int, spec: HeadSpec, parts, device) -> torch.Tensor:
    n, d = cfg.seq_len, cfg.head_dim
    gen = _torch_gen(cfg, ROLE_Q, h, device)
    rt = math.sqrt(d)
    if spec.kind == "diffuse":
        return torch.randn(n, d, generator=gen, device=device, dtype=torch.float32) / rt
    if spec.kind == "structured":
        q = torch.randn(n, d, generator=gen, device=device, dtype=torch.float32) / rt
        for m, amp, ph in spec.smooth:   # s * q . k = amp * cos(2 pi m j / n - ph) on the smooth code
            c = SMOOTH_DIMS[0] + 2 * (m - 1)
            q[:, c] += amp * rt / SMOOTH_SCALE * math.cos(ph)
            q[:, c + 1] += amp * rt / SMOOTH_SCALE * math.sin(ph)
        return q
    q = torch.zeros(n, d, device=device, dtype=torch.float32)
    if spec.kind == "flat":
        return q
    if spec.kind in ("sink_collapse", "floor"):
        beta = 40.0 if spec.kind == "sink_collapse" else math.log(n / N_SINKS)
        q[:, SINK_DIM] = beta * rt / TAG
        return q
    loc, sl, _ = parts
    q += BG_SIGMA * torch.randn(n, d, generator=gen, device=device, dtype=torch.float32)
    nl = LOCAL_DIMS[1] - LOCAL_DIMS[0]
    a_loc = (LOCAL_PEAK + spec.s_loc) * rt / nl
    q[:, LOCAL_DIMS[0]:LOCAL_DIMS[1]] += a_loc * loc
    # slash code width (structured-PE configs keep the smooth code out of the slash boost)
    ns = SLASH_DIMS[1] - SLASH_DIMS[0] - ((SMOOTH_DIMS[1] - SMOOTH_DIMS[0]) if cfg.structured_pe else 0)
    for o, s in zip(spec.slash_offsets, spec.s_slash):
        if o >= n:
            continue
        b = (math.log(n / 64.0) + s) * rt / 64.0
        q[o:, SLASH_DIMS[0]:SLASH_DIMS[0] + ns] += b * sl[: n - o, :ns]
    q[:, SINK_DIM] += (math.log(n / N_SINKS) + spec.s_sink) * rt / TAG
    for v, s in zip(spec.verticals, spec.s_vert):
        q[:, VERT_DIM0 + v] += (math.log(n) + s) * rt / TAG
    return q


def make_layer(cfg: LayerConfig, device="cpu", heads: Optional[List[int]] = None):
    """Build (q, k, v) bf16 tensors [H_q|H_kv, n, d] on `device`.

    If `heads` is given, only those query heads are filled (others are zero) and
    only their KV groups are built; this lets a CPU check regenerate a few heads
    of a large layer.  Returns (q, k, v, specs).
    """
    n, d, Hq, Hkv, G = cfg.seq_len, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads, cfg.group
    specs = head_specs(cfg)
    want = list(range(Hq)) if heads is None else sorted(set(heads))
    groups = sorted(set(h // G for h in want))
    q = torch.zeros(Hq, n, d, device=device, dtype=torch.bfloat16)
    k = torch.zeros(Hkv, n, d, device=device, dtype=torch.bfloat16)
    v = torch.zeros(Hkv, n, d, device=device, dtype=torch.bfloat16)
    for g in groups:
        gen_v = _torch_gen(cfg, ROLE_V, g, device)
        v[g] = torch.randn(n, d, generator=gen_v, device=device, dtype=torch.float32).to(torch.bfloat16)
        if cfg.tiny and g == 1:
            gen_k = _torch_gen(cfg, ROLE_K, g, device)
            k[g] = (torch.randn(n, d, generator=gen_k, device=device, dtype=torch.float32)
                    / math.sqrt(d)).to(torch.bfloat16)
            parts = None
        else:
            parts = _key_parts(cfg, g, device)
            k[g] = torch.cat(parts, dim=1).to(torch.bfloat16)
        for h in want:
            if h // G != g:
                continue
            q[h] = _query_head(cfg, h, specs[h], parts, device).to(torch.bfloat16)
        del parts
    return q, k, v, specs


def custom_config(seq_len: int, n_q_heads: int = 2, n_kv_heads: int = 1, block: int = 128,
                  config_id: int = 100, **kw) -> LayerConfig:
    """A small layer with the default mixture, for tests (config ids >= 100)."""
    return LayerConfig(f"custom-{seq_len}-{n_q_heads}x{n_kv_heads}-b{block}", config_id, seq_len,
                       n_q_heads, n_kv_heads, block=block, **kw)
