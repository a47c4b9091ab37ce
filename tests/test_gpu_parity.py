"""GPU parity: the HIP path through the C-ABI against the fp64 oracle.

Bar (bf16 inputs and outputs): max-abs <= 2e-2 and mean-abs <= 2e-3 on O;
lse within 1e-3; bit-identical outputs across repeats at a fixed
(num_splits, pack_gqa); special cases exact where the arithmetic is exact."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import bf16_bits_to_f64, combine_partials, decode_attention, even_bounds, split_partials
from workloads import config_shapes, custom_shape, make_inputs
from tests.gpu_helpers import assert_parity, dev_inputs, errors, say, to_dev, to_f64

pytestmark = pytest.mark.gpu

VARIANTS = [(0, -1), (1, 1), (1, 0), (2, 1), (3, 1), (4, 1), (8, 1), (16, 1), (64, 1), (4, 0), (64, 0), (1, 2), (6, 2)]
LSE_TOL = 1e-3


def run(q, k, v, cu, L, s, pack, lse=True, scale=0.0):
    lse_t = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device) if lse else None
    out = da.da_decode_attn(q, k, v, cu, lse_out=lse_t, L_K_max=L, num_splits=s, pack_gqa=pack,
                            softmax_scale=scale)
    torch.cuda.synchronize()
    return out, lse_t


def check_case(inp, variants, what):
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    L = inp.shape.L_K
    for s, pack in variants:
        say(f"{what} s={s} pack={pack}")
        out, lse_t = run(q, k, v, cu, L, s, pack)
        assert_parity(out, O, f"{what} s={s} pack={pack}")
        lg = lse_t.cpu().numpy().astype(np.float64)
        fin = np.isfinite(lse)
        assert np.array_equal(np.isfinite(lg), fin)
        assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL


@pytest.mark.parametrize("shape", [s for c in (1, 2, 3, 4) for s in config_shapes(c)], ids=lambda s: s.name)
def test_workload_parity(shape):
    check_case(make_inputs(shape), VARIANTS, shape.name)


def test_highload_parity_sampled_sequences():
    """Full-size high-load workload in the launch configurations the
    benchmark times; the oracle computes three sampled sequences."""
    sh = config_shapes(5)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    picks = [0, 13, 31]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    plan = da.da_choose_splits(sh.B, sh.H_Q, sh.H_KV, sh.L_K)
    assert plan.kv_nontemporal == 1          # 1 GiB of K/V: streaming loads
    for s, pack in [(0, -1), (1, 1), (plan.num_splits, 1), (4, 1), (16, 1), (64, 1), (8, 0)]:
        say(f"highload s={s} pack={pack}")
        out, lse_t = run(q, k, v, cu, sh.L_K, s, pack)
        assert_parity(out[picks], O, f"highload s={s}")
        assert np.max(np.abs(lse_t.cpu().numpy()[picks] - lse)) <= LSE_TOL
        # every sequence is finite, not only the sampled ones
        assert torch.isfinite(out.float()).all()


def test_two_wave_launches_at_full_load_sampled_sequences():
    """1 GiB of pure-MQA K/V (B=256, H_Q=8, H_KV=1, L_K=8192), which the
    planner launches with two waves per workgroup and K straight into the
    operand layout: oracle parity on sampled sequences through both register
    fetch paths, the same bits for both, and the same bits on a repeat."""
    sh = custom_shape(256, 8, 1, 8192)
    inp = make_inputs(sh, seed=43)
    q, k, v, _ = dev_inputs(inp)
    picks = [0, 101, 255]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    plan = da.da_choose_splits(sh.B, sh.H_Q, sh.H_KV, sh.L_K)
    assert (plan.group_waves, plan.kv_fetch, plan.num_splits) == (2, 0, 1), plan.as_dict()
    first = None
    for fetch in (0, 1, 0):
        p = da.DaPlan.from_buffer_copy(plan)
        p.kv_fetch = fetch
        say(f"two-wave full load fetch={fetch} {p.as_dict()}")
        lse_t = torch.empty(sh.B, sh.H_Q, dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_planned(q, k, v, p, None, lse_out=lse_t)
        torch.cuda.synchronize()
        assert_parity(out[picks], O, f"two-wave full load fetch={fetch}")
        assert np.max(np.abs(lse_t.cpu().numpy()[picks] - lse)) <= LSE_TOL
        assert torch.isfinite(out.float()).all()
        if first is None:
            first = out
        else:
            assert torch.equal(out.view(torch.int16), first.view(torch.int16)), fetch


def test_device_lengths_launch_four_waves():
    """Where the planner gives a fixed-length batch two waves (B=32, H_Q=64,
    H_KV=8, L_K=1024: 256 workgroups of 1024 keys), the same batch passed
    with cu_seqlens_k (lengths read on the device) runs the four-wave
    launch: its bits are those of the four-wave plan on the fixed layout,
    and both match the oracle on sampled sequences."""
    sh = custom_shape(32, 64, 8, 1024)
    inp = make_inputs(sh, seed=47)
    q, k, v, _ = dev_inputs(inp)
    picks = [0, 31]
    O, _ = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    two = da.da_choose_splits(32, 64, 8, 1024)
    assert (two.group_waves, two.num_splits) == (2, 1), two.as_dict()
    four = da.DaPlan.from_buffer_copy(two)
    four.group_waves, four.kv_fetch = 4, 2
    cu = torch.arange(0, 33 * 1024, 1024, dtype=torch.int32, device="cuda")
    say("device lengths: four waves")
    a = da.da_decode_attn_planned(q, k, v, two, None)
    b = da.da_decode_attn_planned(q, k, v, four, None)
    c = da.da_decode_attn(q, k.view(-1, 8, 128), v.view(-1, 8, 128), cu, L_K_max=1024)
    torch.cuda.synchronize()
    for out, what in ((a, "two waves"), (b, "four waves"), (c, "varlen")):
        assert_parity(out[picks], O, what)
    assert torch.equal(c.view(torch.int16), b.view(torch.int16))
    d = da.da_decode_attn(q, k, v)                       # the fixed layout plans two waves
    torch.cuda.synchronize()
    assert torch.equal(d.view(torch.int16), a.view(torch.int16))


def test_streaming_wide_group_sampled_sequences():
    """537 MB of K/V (streaming loads) with groups of 32 heads in one
    workgroup (two 16-column tiles), through each K/V fetch path; the oracle
    computes three sampled sequences."""
    sh = custom_shape(64, 32, 1, 16384)
    inp = make_inputs(sh, seed=41)
    q, k, v, cu = dev_inputs(inp)
    picks = [0, 37, 63]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    for s in (1, 8, 64):
        p = da.da_make_plan(sh.B, sh.H_Q, sh.H_KV, sh.L_K, num_splits=s, pack_gqa=2)
        assert p.kv_nontemporal == 1 and p.heads_per_tile == 32
        say(f"streaming wide s={s} fetch={p.kv_fetch}")
        out, lse_t = run(q, k, v, cu, sh.L_K, s, 2)
        assert_parity(out[picks], O, f"streaming wide s={s}")
        assert np.max(np.abs(lse_t.cpu().numpy()[picks] - lse)) <= LSE_TOL


@pytest.mark.parametrize("s,pack", [(1, 1), (2, 1), (64, 1), (1, 0), (7, 0)])
def test_single_key_returns_v_bitwise(s, pack):
    sh = custom_shape(2, 16, 2, 1)
    inp = make_inputs(sh, seed=21)
    q, k, v, cu = dev_inputs(inp)
    say(f"single key s={s} pack={pack}")
    out, lse_t = run(q, k, v, cu, 1, s, pack)
    vv = v[:, 0].repeat_interleave(8, dim=1)            # [B, H_Q, D]: query head h reads KV head h // 8
    assert torch.equal(out.view(torch.int16), vv.view(torch.int16))


def test_identical_keys_and_zero_query_give_mean_v():
    rng = np.random.default_rng(22)
    sh = custom_shape(1, 8, 1, 300)
    inp = make_inputs(sh, seed=22)
    inp.k[:] = inp.k[:, :1]
    mean = bf16_bits_to_f64(inp.v)[0, :, 0, :].mean(axis=0)
    q, k, v, cu = dev_inputs(inp)
    for s in (1, 5):
        say(f"identical keys s={s}")
        out, _ = run(q, k, v, cu, 300, s, 1)
        g = to_f64(out)[0]
        assert np.max(np.abs(g - mean)) <= 4e-3
    q0 = torch.zeros_like(q)
    inp2 = make_inputs(sh, seed=23)
    _, k2, v2, _ = dev_inputs(inp2)
    mean2 = bf16_bits_to_f64(inp2.v)[0, :, 0, :].mean(axis=0)
    say("zero query")
    out, lse_t = run(q0, k2, v2, None, 300, 3, 1)
    assert np.max(np.abs(to_f64(out)[0] - mean2)) <= 4e-3
    assert np.allclose(lse_t.cpu().numpy(), np.log(300), atol=1e-5)


def test_empty_and_short_sequences():
    sh = custom_shape(2, 8, 2, 0)
    inp = make_inputs(sh, seed=24)
    q = to_dev(inp.q)
    kz = torch.zeros(2, 0, 2, 128, dtype=torch.bfloat16, device="cuda")
    for s in (1, 4):
        say(f"empty fixed s={s}")
        out, lse_t = run(q, kz, kz, None, 0, s, 1)
        assert torch.all(out.float() == 0) and torch.all(torch.isneginf(lse_t))
    # varlen: an empty sequence, sequences shorter than the split count
    shv = custom_shape(4, 8, 2, 40, varlen=True)
    inpv = make_inputs(shv, seed=25, lengths=[0, 3, 40, 1])
    check_case(inpv, [(1, 1), (5, 1), (64, 1), (8, 0), (0, -1)], "varlen-short")


@pytest.mark.parametrize("B,H_Q,H_KV,L", [
    (3, 4, 4, 97),       # MHA, nothing to pack
    (2, 12, 4, 33),      # group of 3
    (1, 16, 1, 1000),    # group of 16
    (2, 64, 2, 129),     # group of 32: two head tiles
    (1, 128, 2, 70),     # group of 64: two tiles per KV head
    (5, 8, 1, 2049),     # ragged long tail
    (2, 34, 2, 300),     # group of 17: one 17-column tile (two 16-column MFMA tiles)
    (1, 48, 2, 200),     # group of 24
    (1, 66, 2, 130),     # group of 33: three tiles of 11 heads
    (1, 96, 2, 257),     # group of 48: two tiles of 24 heads
    (3, 40, 1, 77),      # group of 40: two tiles of 20 heads
])
def test_group_and_ragged_shapes(B, H_Q, H_KV, L):
    sh = custom_shape(B, H_Q, H_KV, L)
    check_case(make_inputs(sh, seed=B * 1000 + L), [(1, 1), (3, 1), (17, 1), (2, 0), (0, -1), (1, 2), (5, 2)],
               f"B{B}-H{H_Q}-KV{H_KV}-L{L}")


@pytest.mark.parametrize("B,H_Q,H_KV,L", [(1, 32, 1, 512), (2, 64, 2, 129), (1, 128, 2, 70), (1, 48, 2, 200)])
def test_tile_width_does_not_change_results(B, H_Q, H_KV, L):
    """A packed group served by one wide workgroup (pack_gqa=2) or by
    16-head workgroups (what pack_gqa=1 picks at these sizes) computes every
    head column with the same operations in the same order."""
    sh = custom_shape(B, H_Q, H_KV, L)
    inp = make_inputs(sh, seed=29 + L)
    q, k, v, cu = dev_inputs(inp)
    for s in (1, 3):
        assert da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=1).heads_per_tile <= 16
        say(f"width B{B}-H{H_Q}-KV{H_KV}-L{L} s={s}")
        a, la = run(q, k, v, cu, L, s, 1)
        b, lb = run(q, k, v, cu, L, s, 2)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
        assert torch.equal(la, lb)


def test_softmax_scale_argument():
    sh = custom_shape(1, 8, 1, 200)
    inp = make_inputs(sh, seed=26)
    O, _ = decode_attention(inp.q, inp.k, inp.v, scale=0.3)
    q, k, v, cu = dev_inputs(inp)
    say("scale 0.3")
    out, _ = run(q, k, v, cu, 200, 3, 1, scale=0.3)
    assert_parity(out, O, "scale 0.3")


@pytest.mark.parametrize("s,pack", [(1, 1), (3, 1), (16, 1), (4, 0), (0, -1)])
def test_bit_identical_repeats(s, pack):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    say(f"repeats s={s} pack={pack}")
    first, lse0 = run(q, k, v, cu, sh.L_K, s, pack)
    for _ in range(10):
        out, lse_t = run(q, k, v, cu, sh.L_K, s, pack)
        assert torch.equal(out.view(torch.int16), first.view(torch.int16))
        assert torch.equal(lse_t, lse0)


def test_varlen_with_equal_lengths_matches_fixed_layout_bitwise():
    sh = custom_shape(3, 32, 4, 150)
    inp = make_inputs(sh, seed=27)
    q, k, v, _ = dev_inputs(inp)
    cu = torch.tensor([0, 150, 300, 450], dtype=torch.int32, device="cuda")
    for s in (1, 4):
        say(f"varlen==fixed s={s}")
        a, _ = run(q, k, v, None, 150, s, 1)
        b, _ = run(q, k.view(450, 4, 128), v.view(450, 4, 128), cu, 150, s, 1)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("s,pack", [(1, 1), (3, 1), (8, 0), (64, 1)])
def test_split_partials_match_oracle_chunks(s, pack):
    sh = custom_shape(2, 16, 2, 200)
    inp = make_inputs(sh, seed=28)
    q, k, v, cu = dev_inputs(inp)
    say(f"partials s={s} pack={pack}")
    op, mp, lp = da.da_split_partials(q, k, v, num_splits=s, pack_gqa=pack)
    torch.cuda.synchronize()
    bounds = [da.da_split_bounds(200, s)] * 2
    assert bounds[0] == even_bounds(200, s)
    rop, rmp, rlp = split_partials(inp.q, inp.k, inp.v, bounds)
    gop, gmp, glp = (t.cpu().numpy().astype(np.float64) for t in (op, mp, lp))
    empty = rlp == 0
    assert np.array_equal(glp == 0, empty)
    assert np.all(np.isneginf(gmp[empty]))
    ne = ~empty
    assert np.max(np.abs(gmp[ne] - rmp[ne])) <= 1e-4
    assert np.max(np.abs(glp[ne] / rlp[ne] - 1)) <= 1e-4
    # normalised chunk outputs, at the output tolerance
    go = gop[ne] / glp[ne][:, None]
    ro = rop[ne] / rlp[ne][:, None]
    mx, mean = errors(go, ro)
    assert mx <= 2e-2 and mean <= 2e-3


def test_combine_of_oracle_partials():
    sh = custom_shape(2, 8, 1, 300)
    inp = make_inputs(sh, seed=29)
    rng = np.random.default_rng(30)
    bounds = []
    for _ in range(2):
        cuts = np.sort(rng.integers(0, 301, 5))
        bounds.append([0] + cuts.tolist() + [300])
    rop, rmp, rlp = split_partials(inp.q, inp.k, inp.v, bounds)
    Oref, lseref = combine_partials(rop, rmp, rlp)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    lse_t = torch.empty(2, 8, dtype=torch.float32, device="cuda")
    say("combine of oracle partials")
    out = da.da_combine_splits(t(rop), t(rmp), t(rlp), lse_out=lse_t)
    torch.cuda.synchronize()
    g = to_f64(out)
    # only the final bf16 rounding separates the two
    assert np.all(np.abs(g - Oref) <= 2.0 ** -8 * np.abs(Oref) + 1e-6)
    assert np.max(np.abs(lse_t.cpu().numpy() - lseref)) <= 1e-5


@pytest.mark.parametrize("s,pack", [(2, 1), (5, 1), (64, 1), (3, 0)])
def test_decode_attn_equals_split_then_combine(s, pack):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    say(f"fused vs two-launch s={s} pack={pack}")
    fused, lse_f = run(q, k, v, cu, sh.L_K, s, pack)
    op, mp, lp = da.da_split_partials(q, k, v, cu, num_splits=s, pack_gqa=pack, L_K_max=sh.L_K)
    lse_c = torch.empty_like(lse_f)
    two = da.da_combine_splits(op, mp, lp, lse_out=lse_c)
    torch.cuda.synchronize()
    assert torch.equal(fused.view(torch.int16), two.view(torch.int16))
    assert torch.equal(lse_f, lse_c)


@pytest.mark.parametrize("s", [1, 6])
def test_graph_replay_matches_eager(s):
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    say(f"graph replay s={s}")
    eager, _ = run(q, k, v, cu, sh.L_K, s, 1)
    out = torch.empty_like(eager)
    da.da_decode_attn(q, k, v, out=out, num_splits=s, pack_gqa=1)   # warm the workspace cache
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        da.da_decode_attn(q, k, v, out=out, num_splits=s, pack_gqa=1)   # workspace for this stream
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        for _ in range(3):
            da.da_decode_attn(q, k, v, out=out, num_splits=s, pack_gqa=1)
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {r}"
        # eager work between replays
        again, _ = run(q, k, v, cu, sh.L_K, s, 1)
        assert torch.equal(again.view(torch.int16), eager.view(torch.int16))


def test_workspace_reused_across_split_counts():
    """One workspace serves calls with different split counts back to back."""
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    O, _ = decode_attention(inp.q, inp.k, inp.v)
    q, k, v, cu = dev_inputs(inp)
    ws = torch.full((da.da_workspace_bytes(sh.B, sh.H_Q, 128, 64),), 255, dtype=torch.uint8, device="cuda")
    outs = {}
    for s in (64, 8, 2, 5, 8, 64, 3):
        say(f"shared workspace s={s}")
        ws[:-(1 << 20)].fill_(255)      # chunk states need no initialisation
        ws[-(1 << 20):].zero_()         # arrival counters of a single-launch merge start at zero
        out = da.da_decode_attn(q, k, v, num_splits=s, pack_gqa=1, workspace=ws)
        torch.cuda.synchronize()
        assert_parity(out, O, f"shared workspace s={s}")
        if s in outs:
            assert torch.equal(out.view(torch.int16), outs[s].view(torch.int16))
        outs[s] = out


def test_graph_keeps_its_workspace_after_the_cache_grows():
    """A graph captured at s=2 holds the cached workspace's address; an eager
    call at s=64 on the same stream makes the cache grow.  The replaced
    buffer must stay allocated, so later replays still give the captured
    call's bits."""
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    O, _ = decode_attention(inp.q, inp.k, inp.v)
    q, k, v, cu = dev_inputs(inp)
    say("graph workspace after cache growth: capture s=2, eager s=64")
    ref2, _ = run(q, k, v, cu, sh.L_K, 2, 1)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    out = torch.empty_like(ref2)
    with torch.cuda.stream(stream):
        da.da_decode_attn(q, k, v, out=out, num_splits=2, pack_gqa=1)    # cache a workspace for this stream
    stream.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        da.da_decode_attn(q, k, v, out=out, num_splits=2, pack_gqa=1)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        big = da.da_decode_attn(q, k, v, num_splits=64, pack_gqa=1)       # grows the cache
        junk = torch.full((1 << 22,), 7, dtype=torch.uint8, device="cuda")  # new allocations on the stream
    stream.synchronize()
    assert_parity(big, O, "eager s=64 after capture")
    for r in range(3):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref2.view(torch.int16)), f"replay {r}"
    del junk
