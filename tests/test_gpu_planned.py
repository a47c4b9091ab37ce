"""GPU parity of the planned entry point (a plan made beforehand, run as it
is) against the fp64 oracle, and its bits against the planning entry point:
the plan decides how the work is spread and cached, never the result."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import config_shapes, custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, say

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def planned(q, k, v, cu, L, plan):
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device="cuda")
    out = da.da_decode_attn_planned(q, k, v, plan, cu, lse_out=lse, L_K_max=L)
    torch.cuda.synchronize()
    return out, lse


def same_bits(a, b):
    return torch.equal(a[0].view(torch.int16), b[0].view(torch.int16)) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("B,H_Q,H_KV,L,varlen", [
    (1, 64, 8, 512, False),     # Llama-70B shape
    (1, 8, 1, 128, False),      # MQA
    (3, 32, 1, 777, False),     # a group of 32: two tile widths
    (2, 128, 2, 300, False),    # a group of 64
    (4, 32, 4, 200, True),      # varlen GQA
    (5, 8, 1, 2049, False),     # ragged tail
    (2, 16, 2, 45, False),      # chunks shorter than a tile per wave (two waves: the second may have none)
])
def test_plans_of_every_kind(B, H_Q, H_KV, L, varlen):
    """Plans from each policy, with and without a CU margin and with every
    K/V fetch path, V slice count and cache hint edited in: oracle parity,
    and the same bits for the same split count and head tiles."""
    sh = custom_shape(B, H_Q, H_KV, L, varlen=varlen)
    inp = make_inputs(sh, seed=B * 31 + L)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    plans = [da.da_choose_splits(B, H_Q, H_KV, L, policy=pol)
             for pol in (da.POLICY_MI355X, da.POLICY_STREAMED, da.POLICY_PAPER, da.POLICY_EVOLVED)]
    plans.append(da.da_choose_splits(B, H_Q, H_KV, L, cu_margin=200))
    plans += [da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=pk) for s in (1, 3) for pk in (0, 1, 2)]
    first = {}
    g = H_Q // H_KV
    for plan in plans:
        # V slices only with K/V straight into LDS, packed (not the paper's packing) or one head per group
        vss = (1, 2, 4) if plan.pack_gqa == 1 or (plan.pack_gqa == 0 and g == 1) else (1,)
        # packed groups of more than 16 heads: both tile widths
        widths = {plan.heads_per_tile} | ({16, 32} if plan.pack_gqa == 1 and g > 16 else set())
        # four waves with every fetch path; two (K/V through registers, one V slice) with the merge
        # in a second launch
        combos = [(f, v, 4) for f, v in [(0, 1), (1, 1)] + [(2, v) for v in vss]] + [(0, 1, 2), (1, 1, 2)]
        for w, fetch, vs, waves in [(w, f, v, n) for w in sorted(widths) for f, v, n in combos]:
            for hint in (0, 1):
                p = da.DaPlan.from_buffer_copy(plan)
                p.heads_per_tile, p.tiles = w, B * H_Q // w
                p.kv_fetch, p.kv_nontemporal, p.v_slices, p.group_waves = fetch, hint, vs, waves
                if waves == 2:
                    p.combine = 0
                chunks = p.tiles * p.num_splits
                p.grid = chunks if vs == 1 else vs * 8 * -(-chunks // 8)
                say(f"planned B{B}-H{H_Q}-KV{H_KV}-L{L} {p.as_dict()}")
                got = planned(q, k, v, cu, L, p)
                assert_parity(got[0], O, f"planned {p.as_dict()}")
                lg = got[1].cpu().numpy().astype(np.float64)
                fin = np.isfinite(lse)
                assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL
                key = (p.num_splits, p.heads_per_tile, p.group_waves)
                if key in first:
                    assert same_bits(got, first[key]), (key, p.as_dict())
                else:
                    first[key] = got
                if hint == 0:
                    # one workgroup per CU at a time: where workgroups run, not what they compute
                    p.wg_per_cu = 1
                    say(f"planned, one workgroup per CU {p.as_dict()}")
                    assert same_bits(planned(q, k, v, cu, L, p), got), p.as_dict()
                    p.wg_per_cu = 0
                if p.num_splits > 1 and p.group_waves == 4:
                    # the other merge (a second launch, or inside the split launch): the same bits
                    p.combine = 1 - p.combine
                    say(f"planned, other merge {p.as_dict()}")
                    assert same_bits(planned(q, k, v, cu, L, p), got), p.as_dict()


@pytest.mark.parametrize("shape", config_shapes(2) + config_shapes(1), ids=lambda s: s.name)
def test_planned_equals_planning_entry(shape):
    """The plan da_decode_attn makes for itself, passed explicitly, gives the
    same bits."""
    inp = make_inputs(shape)
    q, k, v, cu = dev_inputs(inp)
    for s, pack in ((0, -1), (1, 1), (4, 1), (2, 0)):
        plan = da.da_make_plan(shape.B, shape.H_Q, shape.H_KV, shape.L_K, num_splits=s, pack_gqa=pack)
        say(f"planned vs planning {shape.name} s={s} pack={pack}")
        lse = torch.empty(shape.B, shape.H_Q, dtype=torch.float32, device="cuda")
        a = da.da_decode_attn(q, k, v, lse_out=lse, num_splits=s, pack_gqa=pack)
        torch.cuda.synchronize()
        assert same_bits((a, lse), planned(q, k, v, cu, shape.L_K, plan))


@pytest.mark.parametrize("B,H_Q,H_KV,L", [
    (1, 64, 8, 384),     # streamed table: 4 splits, 4 V slices, merged in the launch
    (1, 64, 8, 512),
    (1, 8, 1, 640),      # 6 splits, 4 V slices
    (1, 32, 1, 768),     # a group of 32 in 16-head tiles
    (16, 32, 4, 512),    # streamed table: 4 splits, nontemporal
    (4, 256, 32, 256),
])
def test_table_policy_plans(B, H_Q, H_KV, L):
    """Plans of the configuration-specific split tables on shapes they hold:
    oracle parity, and the same bits as the same split count and tile width
    launched one workgroup per chunk with K/V through registers."""
    sh = custom_shape(B, H_Q, H_KV, L)
    inp = make_inputs(sh, seed=B * 37 + L)
    O, _ = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    for pol in (da.POLICY_TABLE, da.POLICY_TABLE_STREAMED):
        plan = da.da_choose_splits(B, H_Q, H_KV, L, policy=pol)
        say(f"table policy {pol} B{B}-H{H_Q}-KV{H_KV}-L{L} {plan.as_dict()}")
        got = planned(q, k, v, cu, L, plan)
        assert_parity(got[0], O, f"table policy {pol} {plan.as_dict()}")
        p = da.DaPlan.from_buffer_copy(plan)
        p.v_slices, p.kv_fetch, p.kv_nontemporal = 1, 1, 0
        p.grid = p.tiles * p.num_splits
        say(f"same split, registers {p.as_dict()}")
        assert same_bits(planned(q, k, v, cu, L, p), got), (plan.as_dict(), p.as_dict())
