"""GPU parity over the launch plans of the paper's regression matrix
(Section 5.3: Batch x L_K x H_KV with H_Q = 8 H_KV), including the H_KV = 32
family (H_Q = 256: 8 KiB K/V rows) and the L_K = 640 boundary, where the
paper reports the standard behaviour again (Section 4.1): the heuristic's
plan, one split as the paper launches it, one split as the planner makes
it, and fixed split counts, each against the fp64 oracle (sampled
sequences at 8192 keys)."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, say

pytestmark = pytest.mark.gpu

CASES = [(B, H_KV, L) for H_KV in (32,) for B in (1, 8) for L in (128, 512, 640, 8192)] + \
        [(B, H_KV, 640) for H_KV in (1, 2, 4, 8) for B in (1, 4)] + [(2, 4, 576), (4, 8, 768)]


@pytest.mark.parametrize("B,H_KV,L", CASES, ids=lambda x: str(x))
def test_regression_family_plans(B, H_KV, L):
    H_Q = 8 * H_KV
    sh = custom_shape(B, H_Q, H_KV, L)
    inp = make_inputs(sh, seed=7000 + 97 * B + 13 * H_KV + L)
    picks = list(range(B)) if B * L <= 8192 else [0, B - 1]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    q, k, v, cu = dev_inputs(inp)
    plans = {"heuristic": da.da_choose_splits(B, H_Q, H_KV, L),
             "paper policy": da.da_choose_splits(B, H_Q, H_KV, L, policy=da.POLICY_PAPER),
             "streamed policy": da.da_choose_splits(B, H_Q, H_KV, L, policy=da.POLICY_STREAMED),
             "s1 paper launch": da.da_make_plan(B, H_Q, H_KV, L, num_splits=1, pack_gqa=2),
             "s1 same plan": da.da_make_plan(B, H_Q, H_KV, L, num_splits=1, pack_gqa=-1)}
    for s in (2, 3, 4, 16):
        plans[f"s{s}"] = da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=1)
    for name, plan in plans.items():
        say(f"regression family B={B} H_KV={H_KV} L={L} {name} {plan.as_dict()}")
        lse_t = torch.empty(B, H_Q, dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_planned(q, k, v, plan, lse_out=lse_t)
        torch.cuda.synchronize()
        assert_parity(out[picks], O, f"B={B} H_KV={H_KV} L={L} {name}")
        assert np.max(np.abs(lse_t.cpu().numpy()[picks] - lse)) <= 1e-3
        assert torch.isfinite(out.float()).all()
