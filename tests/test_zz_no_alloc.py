"""crisp_sparse_attn_noalloc (the sparse attention entry point that allocates nothing: its
work list lives in the library's static schedule area) against crisp_sparse_attn with a
caller workspace, through the C ABI: on two calls in a row, the second on a smaller layer
(so the area still holds the first call's larger schedule), outputs agree to the attention
tolerances (max-abs 2e-2, mean-abs 2e-3; rows the area splits differently differ by
rounding only), and bit for bit where neither call splits a row; a layer past the area's
size is CRISP_EINVAL."""
import sys

import numpy as np
import pytest
import torch

from tests import parity as PR
from tests.helpers import to_f64
from workloads import custom_config, make_layer
from workloads.synth import structured_pe_config

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def _layer(C, cfg):
    q, k, v, _ = make_layer(cfg, device=DEV)
    _, _, rp, ci = C.crisp_prefill_attn(q, k, v, C.make_params(alpha=cfg.alpha), cfg.block, return_lists=True)
    return q, k, v, rp, ci


def _agree(a, b, where):
    torch.cuda.synchronize()
    PR.compare_attention(to_f64(a).reshape(-1, 128), to_f64(b).reshape(-1, 128).astype(np.float64), where=where)


def test_no_alloc_matches_workspace_entry_point_twice():
    from paper_2609_01925_amd import crisp as C
    # first call: a 16k two-head layer whose long PE rows the workspace entry point splits
    # (persistent grid, partial slots; the area's fewer slots split fewer rows)
    big = custom_config(16384, 2, 1, block=128, config_id=156, tiny=True)
    _say(f"no-alloc sparse attention, first call: {big.name}")
    q, k, v, rp, ci = _layer(C, big)
    o_ws = C.crisp_sparse_attn(q, k, v, rp, ci, big.block)
    o_na = C.crisp_sparse_attn_noalloc(q, k, v, rp, ci, big.block)
    _agree(o_na, o_ws, "16k layer")
    del q, k, v, rp, ci
    # the 8k structured layer: one unit per workgroup from one list in both, bit for bit
    mid = structured_pe_config(8192)
    _say(f"no-alloc sparse attention, second call: {mid.name}")
    q, k, v, rp, ci = _layer(C, mid)
    o_ws = C.crisp_sparse_attn(q, k, v, rp, ci, mid.block)
    o_na = C.crisp_sparse_attn_noalloc(q, k, v, rp, ci, mid.block)
    torch.cuda.synchronize()
    assert torch.equal(o_na, o_ws)
    del q, k, v, rp, ci
    # third call, smaller: ragged B = 64 layer
    small = custom_config(3001, 4, 2, block=64, config_id=154)
    _say(f"no-alloc sparse attention, third call: {small.name}")
    q, k, v, rp, ci = _layer(C, small)
    o_ws = C.crisp_sparse_attn(q, k, v, rp, ci, small.block)
    o_na = C.crisp_sparse_attn_noalloc(q, k, v, rp, ci, small.block)
    _agree(o_na, o_ws, "3001-token B=64 layer")


def test_no_alloc_one_unit_per_workgroup_is_bitwise():
    """From 2^19 tokens on rows are never split, so both entry points compute every unit
    the same way: the outputs are equal bit for bit (and so on a repeated call)."""
    from paper_2609_01925_amd import crisp as C
    cfg = custom_config(1 << 19, 2, 1, block=128, config_id=155)
    _say(f"no-alloc sparse attention, one unit per workgroup: {cfg.name}")
    q, k, v, rp, ci = _layer(C, cfg)
    o_ws = C.crisp_sparse_attn(q, k, v, rp, ci, cfg.block)
    o_na = C.crisp_sparse_attn_noalloc(q, k, v, rp, ci, cfg.block)
    o_na2 = C.crisp_sparse_attn_noalloc(q, k, v, rp, ci, cfg.block)
    torch.cuda.synchronize()
    assert torch.equal(o_na, o_ws) and torch.equal(o_na2, o_ws)


def test_no_alloc_rejects_a_layer_past_the_area():
    from paper_2609_01925_amd import crisp as C
    _say("no-alloc sparse attention: layer past the static area")
    # 128 heads x 32768 blocks of 64 tokens: the work list is one int past 16 MiB; nothing
    # is launched, so small stand-in tensors of the declared shape are never read
    sh = C.CrispShape(128, 1, 1 << 21, 128, 64)
    t = torch.zeros(16, dtype=torch.int32, device=DEV)
    st = C.lib.crisp_sparse_attn_noalloc(C.ctypes.byref(sh), 0.0, C._ptr(t), C._ptr(t), C._ptr(t), C._ptr(t),
                                         C._ptr(t), 1 << 40, C._ptr(t), C._stream(t.device))
    assert st == C.CRISP_EINVAL and b"static area" in C.lib.crisp_last_error()
