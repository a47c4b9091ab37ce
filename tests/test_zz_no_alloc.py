"""The no-allocation entry point (da_decode_attn_noalloc) on the GPU: its
output, through the C-ABI, against the entry point that takes a workspace
(the same plan, so the same bits) and against the fp64 oracle, on two calls
in a row with the second smaller, and with no torch allocation during the
calls."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import config_shapes, custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, say

pytestmark = pytest.mark.gpu


def both(inp, s, pack):
    """(noalloc output, lse), (workspace output, lse) for one problem."""
    q, k, v, cu = dev_inputs(inp)
    L = inp.shape.L_K
    B, H_Q = inp.shape.B, inp.shape.H_Q
    out_n = torch.empty(B, H_Q, 128, dtype=torch.bfloat16, device="cuda")
    lse_n = torch.empty(B, H_Q, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    before = torch.cuda.memory_allocated()
    da.da_decode_attn_noalloc(q, k, v, cu, out=out_n, lse_out=lse_n, L_K_max=L, num_splits=s, pack_gqa=pack)
    torch.cuda.synchronize()
    assert torch.cuda.memory_allocated() == before       # nothing allocated through torch
    lse_w = torch.empty_like(lse_n)
    out_w = da.da_decode_attn(q, k, v, cu, lse_out=lse_w, L_K_max=L, num_splits=s, pack_gqa=pack)
    torch.cuda.synchronize()
    return (out_n, lse_n), (out_w, lse_w)


@pytest.mark.parametrize("s,pack", [(0, -1), (1, 1), (4, 1), (16, 1), (3, 0), (6, 2)])
def test_noalloc_matches_workspace_entry_on_two_calls(s, pack):
    big = config_shapes(2)[3]                                # B=1, H_Q=64, H_KV=8, L_K=512
    small = custom_shape(1, 8, 1, 200)                       # then a smaller problem
    for sh, seed in ((big, None), (small, 5)):
        inp = make_inputs(sh) if seed is None else make_inputs(sh, seed=seed)
        O, lse = decode_attention(inp.q, inp.k, inp.v)
        say(f"noalloc {sh.name} s={s} pack={pack}")
        (on, ln), (ow, lw) = both(inp, s, pack)
        assert_parity(on, O, f"noalloc {sh.name} s={s}")
        assert np.max(np.abs(ln.cpu().numpy() - lse)) <= 1e-3
        assert torch.equal(on.view(torch.int16), ow.view(torch.int16)), f"bits {sh.name} s={s} pack={pack}"
        assert torch.equal(ln, lw)


def test_noalloc_varlen_and_highload_sampled():
    """A varlen batch, then the full high-load shape at a split count whose
    chunk states fit the scratch (s = 4: 4.3 MB); the oracle computes three
    sampled sequences of the large call."""
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    O, _ = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    say("noalloc varlen")
    (on, _), (ow, _) = both(inp, 4, 1)
    assert_parity(on, O, "noalloc varlen")
    assert torch.equal(on.view(torch.int16), ow.view(torch.int16))
    sh = config_shapes(5)[0]
    inp = make_inputs(sh)
    picks = [0, 17, 31]
    O, _ = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    say("noalloc highload s=4")
    (on, _), (ow, _) = both(inp, 4, 1)
    assert_parity(on[picks], O, "noalloc highload")
    assert torch.equal(on.view(torch.int16), ow.view(torch.int16))


def test_noalloc_refuses_a_split_beyond_its_scratch():
    sh = config_shapes(5)[0]
    q = torch.zeros(sh.B, sh.H_Q, 128, dtype=torch.bfloat16, device="cuda")
    k = torch.zeros(sh.B, 64, sh.H_KV, 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(da.DecodeAttnError) as e:
        da.da_decode_attn_noalloc(q, k, k, num_splits=64, pack_gqa=1)
    assert e.value.code == da._binding.DA_ERR_WORKSPACE
