"""GPU parity on seeded random shapes: group sizes, lengths (fixed and
varlen, with ragged tails and empty sequences), batch sizes and launch
plans drawn from a fixed-seed generator -- the planner's own plan and a
forced one (split count, packing, tile width, V slices, merge, fetch path
and cache hint where the plan check allows them) -- each against the fp64
oracle, and the forced plan's two merges with the same bits."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, fit_waves, say

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def draw_case(i: int):
    rng = np.random.default_rng(20_000 + i)
    H_KV = int(rng.choice([1, 2, 4, 8, 16]))
    g = int(rng.choice([1, 2, 3, 5, 8, 12, 16, 24, 32, 48, 64]))
    while H_KV * g > 256:
        g //= 2
    B = int(rng.integers(1, 7))
    L = int(rng.choice([1, 2, 31, 33, 64, 100, 511, 513, 1000, 2049, 4097]))
    varlen = bool(rng.integers(0, 2))
    lengths = None
    if varlen:
        lengths = [int(x) for x in rng.integers(0, L + 1, size=B)]
        lengths[int(rng.integers(0, B))] = L
    s = int(rng.choice([1, 2, 3, 5, 8, 13, 16, 33, 64]))
    pack = int(rng.choice([0, 1, 2]))
    return dict(B=B, H_Q=H_KV * g, H_KV=H_KV, L=L, varlen=varlen, lengths=lengths, s=s, pack=pack,
                vs=int(rng.choice([1, 2, 4])), hint=int(rng.integers(0, 2)), fetch=int(rng.choice([0, 1, 2])),
                seed=int(rng.integers(0, 1 << 30)))


CASES = [draw_case(i) for i in range(160)]


def run(q, k, v, cu, L, plan):
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device="cuda")
    out = da.da_decode_attn_planned(q, k, v, plan, cu, lse_out=lse, L_K_max=L if cu is not None else None)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c['B']}-H{c['H_Q']}-KV{c['H_KV']}-L{c['L']}"
                                                      f"{'v' if c['varlen'] else ''}-s{c['s']}-p{c['pack']}")
def test_random_shape_parity(case):
    c = case
    sh = custom_shape(c["B"], c["H_Q"], c["H_KV"], c["L"], varlen=c["varlen"])
    inp = make_inputs(sh, seed=c["seed"], lengths=c["lengths"])
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    L = c["L"]
    fin = np.isfinite(lse)
    plans = {"planned": da.da_choose_splits(c["B"], c["H_Q"], c["H_KV"], L)}
    forced = da.da_make_plan(c["B"], c["H_Q"], c["H_KV"], L, num_splits=c["s"], pack_gqa=c["pack"])
    g = c["H_Q"] // c["H_KV"]
    # edits the plan check allows: V slices only straight into LDS with a packed group (not the paper's
    # packing) or a group of one; the cache hint anywhere; fetch path anywhere without slices
    if c["vs"] > 1 and (forced.pack_gqa == 1 or (forced.pack_gqa == 0 and g == 1)):
        forced.v_slices, forced.kv_fetch = c["vs"], 2
        chunks = forced.tiles * forced.num_splits
        forced.grid = c["vs"] * 8 * -(-chunks // 8)
    else:
        forced.v_slices, forced.kv_fetch = 1, c["fetch"]
        forced.grid = forced.tiles * forced.num_splits
    forced.kv_nontemporal = c["hint"]
    fit_waves(forced)       # two waves only with K/V through registers and one V slice
    plans["forced"] = forced
    results = {}
    for name, plan in plans.items():
        say(f"random shape {c} {name} {plan.as_dict()}")
        out, lse_t = run(q, k, v, cu, L, plan)
        assert_parity(out, O, f"{name} {plan.as_dict()}")
        lg = lse_t.cpu().numpy().astype(np.float64)
        assert np.array_equal(np.isfinite(lg), fin)
        assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL
        results[name] = (out, lse_t)
    if forced.num_splits > 1 and forced.group_waves == 4:     # two-wave plans merge by a second launch only
        other = da.DaPlan.from_buffer_copy(forced)
        other.combine = 1 - forced.combine
        if other.combine == 0 or forced.tiles <= 4096:
            say(f"random shape {c} other merge")
            out, lse_t = run(q, k, v, cu, L, other)
            assert torch.equal(out.view(torch.int16), results["forced"][0].view(torch.int16))
            assert torch.equal(lse_t, results["forced"][1])


def draw_paged_case(i: int):
    c = draw_case(1000 + i)
    rng = np.random.default_rng(30_000 + i)
    c["page"] = int(rng.choice([32, 64, 96, 256]))
    c["varlen"] = True
    if c["lengths"] is None:
        c["lengths"] = [int(x) for x in rng.integers(0, c["L"] + 1, size=c["B"])]
        c["lengths"][0] = c["L"]
    c["chunk"] = int(rng.choice([0, 0, 1, 2, 5, 40]))
    return c


PAGED_CASES = [draw_paged_case(i) for i in range(60)]


@pytest.mark.parametrize("case", PAGED_CASES, ids=lambda c: f"B{c['B']}-H{c['H_Q']}-KV{c['H_KV']}-L{c['L']}"
                                                            f"-page{c['page']}-s{c['s']}-c{c['chunk']}")
def test_random_paged_and_scheduled_parity(case):
    """The same draws over a paged cache: the planned paged entry point with
    the planner's plan and a forced split count, and the per-sequence
    schedule (modelled or forced chunk length) with both merges, against the
    oracle on the contiguous keys; the schedule's two merges give the same
    bits."""
    from workloads import paged_layout
    from tests.gpu_helpers import to_dev
    c = case
    sh = custom_shape(c["B"], c["H_Q"], c["H_KV"], c["L"], varlen=True)
    inp = make_inputs(sh, seed=c["seed"], lengths=c["lengths"])
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    pg = paged_layout(inp, c["page"], seed=c["seed"] % 1000 + 1)
    q = to_dev(inp.q)
    kc, vc = to_dev(pg.k_cache), to_dev(pg.v_cache)
    bt, sl = torch.from_numpy(pg.block_table).cuda(), torch.from_numpy(pg.seq_lens).cuda()
    L = c["L"]
    fin = np.isfinite(lse)

    def check(out, lse_t, what):
        assert_parity(out, O, what)
        lg = lse_t.cpu().numpy().astype(np.float64)
        assert np.array_equal(np.isfinite(lg), fin)
        assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL

    plans = {"planned": da.da_choose_splits(c["B"], c["H_Q"], c["H_KV"], L),
             "forced": da.da_make_plan(c["B"], c["H_Q"], c["H_KV"], L, num_splits=c["s"], pack_gqa=c["pack"])}
    for name, plan in plans.items():
        say(f"random paged {c} {name} {plan.as_dict()}")
        lse_t = torch.empty(c["B"], c["H_Q"], dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_paged_planned(q, kc, vc, bt, sl, L, plan, lse_out=lse_t)
        torch.cuda.synchronize()
        check(out, lse_t, f"paged {name} {plan.as_dict()}")
    sched, meta = da.da_make_schedule(c["lengths"], c["H_Q"], c["H_KV"], L, pack_gqa=c["pack"], chunk_tiles=c["chunk"])
    meta_dev = meta.cuda()
    combs = (sched.combine, 1 - sched.combine) if sched.state_rows > 0 and sched.tiles <= 4096 else (sched.combine,)
    first = None
    for comb in combs:
        sched.combine = comb
        say(f"random scheduled {c} {sched.as_dict()}")
        lse_t = torch.empty(c["B"], c["H_Q"], dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_scheduled(q, kc, vc, sched, meta_dev, block_table=bt, seq_lens=sl, lse_out=lse_t)
        torch.cuda.synchronize()
        check(out, lse_t, f"scheduled {sched.as_dict()}")
        if first is None:
            first = (out, lse_t)
        else:
            assert torch.equal(out.view(torch.int16), first[0].view(torch.int16))
            assert torch.equal(lse_t, first[1])
