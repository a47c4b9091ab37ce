"""GPU parity of the single-launch merge (da_plan.combine = 1): the last
workgroup of each tile to finish merges the tile's chunk states inside the
split launch, in place of the second combine launch (the paper's final
reduction, Sections 3.1 and 5.3).  Checked against the fp64 oracle, bit for
bit against the two-launch merge of the same plan, and for the arrival
counters it leaves behind (zero after every call)."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import config_shapes, custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, fit_waves, say

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def edited(plan, combine=None, vs=None, fetch=None, hpt=None, B=None, H_Q=None):
    """A copy of `plan` with fields edited in (grid kept consistent)."""
    p = da.DaPlan.from_buffer_copy(plan)
    if hpt is not None:
        p.heads_per_tile, p.tiles = hpt, B * H_Q // hpt
    if fetch is not None:
        p.kv_fetch = fetch
    if vs is not None:
        p.v_slices = vs
    if combine is not None:
        p.combine = combine
    chunks = p.tiles * p.num_splits
    p.grid = chunks if p.v_slices == 1 else p.v_slices * 8 * -(-chunks // 8)
    return fit_waves(p)


ARRIVAL_BYTES = 1 << 20


def arrivals_region(ws):
    """The arrival counters: the last 1 MiB of the workspace buffer (its
    size here is a multiple of 256 bytes)."""
    assert ws.numel() % 256 == 0
    return ws[ws.numel() - ARRIVAL_BYTES:].view(torch.int32)


def run_plan(q, k, v, cu, L, plan, ws=None):
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device="cuda")
    out = da.da_decode_attn_planned(q, k, v, plan, cu, lse_out=lse, L_K_max=L, workspace=ws)
    torch.cuda.synchronize()
    return out, lse


def check(out, lse_t, O, lse, what):
    assert_parity(out, O, what)
    lg = lse_t.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse)
    assert np.array_equal(np.isfinite(lg), fin), what
    assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL, what


def same_bits(a, b):
    return torch.equal(a[0].view(torch.int16), b[0].view(torch.int16)) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("shape", [s for c in (1, 2, 3, 4) for s in config_shapes(c)], ids=lambda s: s.name)
def test_fused_matches_oracle_and_two_launch(shape):
    inp = make_inputs(shape)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    B, H_Q, H_KV, L = shape.B, shape.H_Q, shape.H_KV, shape.L_K
    for s, pack in [(2, 1), (3, 1), (4, 1), (8, 1), (16, 1), (64, 1), (3, 0), (4, 2), (6, 2)]:
        base = da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=pack)
        say(f"fused {shape.name} s={s} pack={pack} {base.as_dict()}")
        # both merges on the launch the in-launch merge runs on (four waves)
        fused = edited(base, combine=1)
        two = run_plan(q, k, v, cu, L, edited(fused, combine=0))
        one = run_plan(q, k, v, cu, L, fused)
        check(*one, O, lse, f"fused {shape.name} s={s} pack={pack}")
        assert same_bits(one, two), f"fused vs two-launch {shape.name} s={s} pack={pack}"


@pytest.mark.parametrize("B,H_Q,H_KV,L", [(1, 64, 8, 512), (1, 32, 1, 700), (2, 8, 1, 300), (3, 128, 2, 257)])
def test_fused_every_fetch_path_slices_and_tile_width(B, H_Q, H_KV, L):
    """Each K/V fetch path, V slice count and packed tile width, with the
    merge inside the launch: oracle parity and the two-launch bits."""
    sh = custom_shape(B, H_Q, H_KV, L)
    inp = make_inputs(sh, seed=7 * B + L)
    O, lse = decode_attention(inp.q, inp.k, inp.v)
    q, k, v, cu = dev_inputs(inp)
    g = H_Q // H_KV
    for s in (2, 5, 16):
        base = da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=1)
        widths = sorted({base.heads_per_tile} | ({16, 32} if g > 16 else set()))
        for w in widths:
            ref = None
            for fetch, vs in [(0, 1), (1, 1), (2, 1), (2, 2), (2, 4)]:
                p1 = edited(base, combine=1, vs=vs, fetch=fetch, hpt=w, B=B, H_Q=H_Q)
                say(f"fused B{B}-H{H_Q}-KV{H_KV}-L{L} {p1.as_dict()}")
                got = run_plan(q, k, v, cu, L, p1)
                check(*got, O, lse, f"fused {p1.as_dict()}")
                two = run_plan(q, k, v, cu, L, edited(p1, combine=0))
                assert same_bits(got, two), p1.as_dict()
                if ref is None:
                    ref = got
                else:
                    assert same_bits(got, ref), p1.as_dict()     # same split count and tile width


def test_fused_counters_return_to_zero_and_workspace_is_shared():
    """Calls of different shapes, split counts and slice counts share one
    workspace; after each, the arrival counters are all zero again."""
    ws = torch.zeros(da.da_workspace_bytes(4, 64, 128, 64), dtype=torch.uint8, device="cuda")
    cases = [(1, 64, 8, 512, 4, 1), (4, 64, 8, 1000, 64, 1), (1, 32, 1, 333, 7, 4), (2, 8, 1, 129, 2, 2),
             (1, 64, 8, 512, 4, 1)]
    for B, H_Q, H_KV, L, s, vs in cases:
        sh = custom_shape(B, H_Q, H_KV, L)
        inp = make_inputs(sh, seed=B + L + s)
        O, lse = decode_attention(inp.q, inp.k, inp.v)
        q, k, v, cu = dev_inputs(inp)
        p = edited(da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=1), combine=1,
                   vs=vs, fetch=2 if vs > 1 else None)
        say(f"shared fused workspace {p.as_dict()}")
        got = run_plan(q, k, v, cu, L, p, ws=ws)
        check(*got, O, lse, f"shared workspace {p.as_dict()}")
        region = arrivals_region(ws)
        assert int(region.abs().sum()) == 0, "arrival counters not reset"


@pytest.mark.parametrize("s", [3, 16])
def test_fused_repeats_and_graph_replay(s):
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    plan = edited(da.da_make_plan(sh.B, sh.H_Q, sh.H_KV, sh.L_K, num_splits=s, pack_gqa=1), combine=1)
    say(f"fused repeats s={s}")
    first = run_plan(q, k, v, cu, sh.L_K, plan)
    for _ in range(10):
        assert same_bits(run_plan(q, k, v, cu, sh.L_K, plan), first)
    say(f"fused graph replay s={s}")
    stream = torch.cuda.Stream()
    ws = torch.zeros(da.da_workspace_bytes(sh.B, sh.H_Q, 128, s), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(first[0])
    lse = torch.empty_like(first[1])
    stream.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for _ in range(3):
            da.da_decode_attn_planned(q, k, v, plan, out=out, lse_out=lse, workspace=ws)
    for r in range(4):
        out.zero_()
        lse.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert same_bits((out, lse), first), f"replay {r}"
        assert int(arrivals_region(ws).abs().sum()) == 0
        assert same_bits(run_plan(q, k, v, cu, sh.L_K, plan), first)     # eager work between replays


def test_fused_empty_and_short_sequences():
    """Sequences shorter than the split count (empty chunks) and empty
    sequences (O = 0, lse = -inf) through the single-launch merge."""
    sh = custom_shape(6, 16, 2, 80, varlen=True)
    inp = make_inputs(sh, seed=77, lengths=[0, 1, 3, 80, 17, 0])
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    for s in (2, 8, 64):
        base = da.da_make_plan(sh.B, sh.H_Q, sh.H_KV, sh.L_K, num_splits=s, pack_gqa=1)
        say(f"fused short/empty s={s}")
        fused = edited(base, combine=1)
        got = run_plan(q, k, v, cu, sh.L_K, fused)
        check(*got, O, lse, f"fused short/empty s={s}")
        assert same_bits(got, run_plan(q, k, v, cu, sh.L_K, edited(fused, combine=0)))
        assert torch.all(got[0][0] == 0) and torch.all(got[0][5] == 0)
        assert torch.all(torch.isneginf(got[1][0])) and torch.all(torch.isneginf(got[1][5]))


def test_fused_highload_sampled_sequences():
    """The full 1 GiB high-load workload (B=32, H_Q=64, H_KV=8, L_K=8192)
    with the merge inside the launch; the oracle computes three sampled
    sequences."""
    sh = config_shapes(5)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    picks = [0, 13, 31]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    for s in (2, 4, 16):
        base = da.da_make_plan(sh.B, sh.H_Q, sh.H_KV, sh.L_K, num_splits=s, pack_gqa=1)
        say(f"fused highload s={s} {base.as_dict()}")
        fused = edited(base, combine=1)
        one = run_plan(q, k, v, cu, sh.L_K, fused)
        assert_parity(one[0][picks], O, f"fused highload s={s}")
        assert np.max(np.abs(one[1].cpu().numpy()[picks] - lse)) <= LSE_TOL
        assert torch.isfinite(one[0].float()).all()
        two = run_plan(q, k, v, cu, sh.L_K, edited(fused, combine=0))
        assert same_bits(one, two)
        if base.group_waves == 2:
            # the planner's own launch (two waves, at two splits held to one workgroup per CU)
            say(f"highload planned s={s} {base.as_dict()}")
            own = run_plan(q, k, v, cu, sh.L_K, base)
            assert_parity(own[0][picks], O, f"highload planned s={s}")
            assert np.max(np.abs(own[1].cpu().numpy()[picks] - lse)) <= LSE_TOL
