"""GPU parity of the paged-KV entry point against the fp64 oracle.

The oracle runs on the contiguous keys; the HIP path reads the same keys
scattered into a pool of pages in a seeded random order, with noise in every
row, page and table entry that no sequence owns.  Same bar as the contiguous
path: max-abs <= 2e-2 and mean-abs <= 2e-3 on O, lse within 1e-3."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import config_shapes, custom_shape, make_inputs, paged_layout
from tests.gpu_helpers import assert_parity, dev_inputs, say, to_dev

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def dev_paged(pg):
    return (to_dev(pg.k_cache), to_dev(pg.v_cache), torch.from_numpy(pg.block_table).cuda(),
            torch.from_numpy(pg.seq_lens).cuda())


def run_paged(q, kc, vc, bt, sl, L, s, pack, scale=0.0):
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device=q.device)
    out = da.da_decode_attn_paged(q, kc, vc, bt, sl, L, lse_out=lse, num_splits=s, pack_gqa=pack,
                                  softmax_scale=scale)
    torch.cuda.synchronize()
    return out, lse


def check_lse(lse_t, lse):
    lg = lse_t.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL


def check_paged(inp, page, variants, what, seed=0, max_pages=None):
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    pg = paged_layout(inp, page, seed=seed, max_pages=max_pages)
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    L = int(max(inp.lengths.max(initial=0), 0))
    for s, pack in variants:
        say(f"paged {what} page={page} s={s} pack={pack}")
        out, lse_t = run_paged(q, kc, vc, bt, sl, L, s, pack)
        assert_parity(out, O, f"paged {what} page={page} s={s} pack={pack}")
        check_lse(lse_t, lse)


VARIANTS = [(0, -1), (1, 1), (3, 1), (16, 1), (64, 1), (1, 0), (5, 0), (2, 2)]


@pytest.mark.parametrize("page", [32, 64, 96, 256])
def test_varlen_gqa_paged(page):
    sh = config_shapes(4)[0]
    check_paged(make_inputs(sh), page, VARIANTS, sh.name, seed=page)


@pytest.mark.parametrize("shape", config_shapes(2) + config_shapes(1), ids=lambda s: s.name)
def test_workload_shapes_paged(shape):
    check_paged(make_inputs(shape), 64, VARIANTS, shape.name, seed=7)


@pytest.mark.parametrize("B,H_Q,H_KV,lengths,page", [
    (3, 8, 1, [0, 1, 1000], 32),          # empty and single-key sequences
    (2, 64, 2, [129, 70], 64),            # group of 32, partial last pages
    (2, 128, 2, [33, 64], 32),            # group of 64: two tiles per KV head
    (4, 12, 4, [31, 32, 33, 95], 96),     # group of 3, lengths around a tile
    (1, 8, 1, [9000], 32),                # 282 pages: a wave crosses 64 page ids
])
def test_ragged_paged(B, H_Q, H_KV, lengths, page):
    sh = custom_shape(B, H_Q, H_KV, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=B * 100 + page, lengths=lengths)
    check_paged(inp, page, [(1, 1), (2, 1), (7, 1), (64, 1), (3, 0), (0, -1), (1, 2), (4, 2)],
                f"B{B}-H{H_Q}-KV{H_KV}-{lengths}", seed=page + 1)


def test_wide_block_table():
    """max_pages larger than any sequence needs: the extra columns hold
    valid ids of other pages and must not be read."""
    sh = custom_shape(4, 32, 4, 300, varlen=True)
    inp = make_inputs(sh, seed=31, lengths=[300, 5, 129, 256])
    check_paged(inp, 64, [(1, 1), (4, 1), (0, -1)], "wide-table", seed=32, max_pages=40)


def test_invalid_page_ids_read_zero_keys():
    sh = custom_shape(2, 16, 2, 256, varlen=True)
    inp = make_inputs(sh, seed=41, lengths=[256, 200])
    pg = paged_layout(inp, 64, seed=42)
    pg.block_table[0, 1] = -1
    pg.block_table[1, 2] = pg.num_pages + 7
    # the oracle sees zero keys and values in those pages
    ref = make_inputs(sh, seed=41, lengths=[256, 200])
    cu = ref.cu_seqlens_k
    ref.k[cu[0] + 64:cu[0] + 128] = 0
    ref.v[cu[0] + 64:cu[0] + 128] = 0
    ref.k[cu[1] + 128:cu[1] + 192] = 0
    ref.v[cu[1] + 128:cu[1] + 192] = 0
    O, lse = decode_attention(ref.q, ref.k, ref.v, ref.lengths, ref.cu_seqlens_k)
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    for s in (1, 3, 0):
        say(f"invalid page ids s={s}")
        out, lse_t = run_paged(q, kc, vc, bt, sl, 256, s, 1 if s else -1)
        assert_parity(out, O, f"invalid page s={s}")
        check_lse(lse_t, lse)


def test_seq_lens_clamped_to_max():
    """A length above L_K_max is read as L_K_max; a negative one as 0."""
    sh = custom_shape(3, 8, 1, 128, varlen=True)
    inp = make_inputs(sh, seed=51, lengths=[128, 128, 0])
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    pg = paged_layout(inp, 32, seed=52, max_pages=8)
    pg.seq_lens[1] = 250
    pg.seq_lens[2] = -5
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    say("clamped seq_lens")
    out, lse_t = run_paged(q, kc, vc, bt, sl, 128, 2, 1)
    assert_parity(out, O, "clamped seq_lens")
    check_lse(lse_t, lse)


@pytest.mark.parametrize("s,pack", [(1, 1), (2, 1), (4, 1), (4, 0)])
def test_paged_equals_contiguous_when_cuts_coincide(s, pack):
    """With L a multiple of 32 keys x 4 waves x s chunks the key-granular
    and tile-aligned cuts are the same ranges, so the two layouts give the
    same bits."""
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    q, k, v, _ = dev_inputs(inp)
    pg = paged_layout(inp, 128, seed=61)
    kc, vc, bt, sl = dev_paged(pg)
    say(f"paged vs contiguous s={s} pack={pack}")
    a = da.da_decode_attn(q, k, v, L_K_max=sh.L_K, num_splits=s, pack_gqa=pack)
    bb, _ = run_paged(q, kc, vc, bt, sl, sh.L_K, s, pack)
    assert torch.equal(a.view(torch.int16), bb.view(torch.int16))


@pytest.mark.parametrize("s,pack", [(1, 1), (5, 1), (3, 0), (0, -1)])
def test_paged_bit_identical_repeats(s, pack):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    pg = paged_layout(inp, 64, seed=71)
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    say(f"paged repeats s={s} pack={pack}")
    first, lse0 = run_paged(q, kc, vc, bt, sl, sh.L_K, s, pack)
    for _ in range(3):
        again, lse1 = run_paged(q, kc, vc, bt, sl, sh.L_K, s, pack)
        assert torch.equal(first.view(torch.int16), again.view(torch.int16))
        assert torch.equal(lse0, lse1)


@pytest.mark.parametrize("s", [1, 6])
def test_paged_graph_replay_matches_eager(s):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    pg = paged_layout(inp, 64, seed=81)
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    say(f"paged graph replay s={s}")
    eager, _ = run_paged(q, kc, vc, bt, sl, sh.L_K, s, 1)
    out = torch.empty_like(eager)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        da.da_decode_attn_paged(q, kc, vc, bt, sl, sh.L_K, out=out, num_splits=s, pack_gqa=1)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        da.da_decode_attn_paged(q, kc, vc, bt, sl, sh.L_K, out=out, num_splits=s, pack_gqa=1)
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {r}"
        again, _ = run_paged(q, kc, vc, bt, sl, sh.L_K, s, 1)
        assert torch.equal(again.view(torch.int16), eager.view(torch.int16))


def test_highload_paged_full_size():
    """The full high-load workload (32 x 8192 keys, 1 GiB of KV) in 256-key
    pages scattered over the pool on the device: three sequences against the
    oracle, and the same bits as the contiguous layout at split counts that
    divide 8192 / 128."""
    sh = config_shapes(5)[0]
    inp = make_inputs(sh)
    q, k, v, _ = dev_inputs(inp)
    P = 256
    npg = sh.L_K // P
    n_pages = sh.B * npg + 5
    g = torch.Generator().manual_seed(91)
    perm = torch.randperm(n_pages, generator=g)[: sh.B * npg]
    kc = torch.zeros(n_pages, P, sh.H_KV, 128, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    kc[perm.cuda()] = k.reshape(sh.B * npg, P, sh.H_KV, 128)
    vc[perm.cuda()] = v.reshape(sh.B * npg, P, sh.H_KV, 128)
    bt = perm.to(torch.int32).reshape(sh.B, npg).cuda()
    sl = torch.full((sh.B,), sh.L_K, dtype=torch.int32, device="cuda")
    picks = [0, 17, 31]
    O, lse = decode_attention(inp.q[picks], inp.k[picks], inp.v[picks])
    plan = da.da_choose_splits(sh.B, sh.H_Q, sh.H_KV, sh.L_K)
    for s, pack in [(0, -1), (plan.num_splits, 1), (4, 1), (16, 1)]:
        say(f"highload paged s={s} pack={pack}")
        out, lse_t = run_paged(q, kc, vc, bt, sl, sh.L_K, s, pack)
        assert_parity(out[picks], O, f"highload paged s={s}")
        assert np.max(np.abs(lse_t.cpu().numpy()[picks] - lse)) <= LSE_TOL
        assert torch.isfinite(out.float()).all()
    for s in (1, 4):
        # the planned launch (two waves at one split here) and its four-wave form, on both layouts;
        # the paged entry point, which reads the lengths on the device, launches the four-wave form
        plan = da.da_make_plan(sh.B, sh.H_Q, sh.H_KV, sh.L_K, num_splits=s, pack_gqa=1)
        four = da.DaPlan.from_buffer_copy(plan)
        if four.group_waves == 2:
            # K/V straight into LDS with one workgroup per CU, through registers where CUs hold more
            four.group_waves, four.kv_fetch, four.wg_per_cu = 4, 2 if four.grid <= four.num_cus else 1, 0
        for p in (plan, four):
            say(f"highload paged vs contiguous s={s} {p.as_dict()}")
            a = da.da_decode_attn_planned(q, k, v, p, None, L_K_max=sh.L_K)
            b = da.da_decode_attn_paged_planned(q, kc, vc, bt, sl, sh.L_K, p)
            torch.cuda.synchronize()
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), p.as_dict()
        b, _ = run_paged(q, kc, vc, bt, sl, sh.L_K, s, 1)
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("B,H_Q,H_KV,lengths,page", [
    (1, 64, 8, [512], 64),                # Llama-70B shape, one sequence
    (3, 32, 1, [777, 40, 300], 32),       # a group of 32: two tile widths
    (4, 12, 4, [31, 32, 33, 95], 96),     # group of 3, lengths around a tile
])
def test_paged_planned_plans_of_every_kind(B, H_Q, H_KV, lengths, page):
    """Plans made beforehand (each policy, a CU margin, forced splits and
    packings, every fetch path, V slice count and cache hint edited in) run
    on a paged cache: oracle parity, and the bits of the planning paged entry
    point for the same split count and packing."""
    sh = custom_shape(B, H_Q, H_KV, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=B * 7 + page, lengths=lengths)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    pg = paged_layout(inp, page, seed=page + 3)
    q = to_dev(inp.q)
    kc, vc, bt, sl = dev_paged(pg)
    L = max(lengths)
    plans = [da.da_choose_splits(B, H_Q, H_KV, L, policy=pol)
             for pol in (da.POLICY_MI355X, da.POLICY_STREAMED, da.POLICY_PAPER)]
    plans.append(da.da_choose_splits(B, H_Q, H_KV, L, cu_margin=200))
    plans += [da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=pk) for s in (1, 4) for pk in (0, 1, 2)]
    g = H_Q // H_KV
    for plan in plans:
        # the entry point's own plan for this split count and packing, and its bits per wave count
        ref_plan = da.da_make_plan(B, H_Q, H_KV, L, num_splits=plan.num_splits, pack_gqa=plan.pack_gqa)
        by_waves = {ref_plan.group_waves: run_paged(q, kc, vc, bt, sl, L, plan.num_splits, plan.pack_gqa)}
        vss = (1, 2, 4) if plan.pack_gqa == 1 or (plan.pack_gqa == 0 and g == 1) else (1,)
        for fetch, vs, waves in [(0, 1, 4), (1, 1, 4), (0, 1, 2), (1, 1, 2)] + [(2, v, 4) for v in vss]:
            for hint in (0, 1):
                p = da.DaPlan.from_buffer_copy(plan)
                p.kv_fetch, p.kv_nontemporal, p.v_slices, p.group_waves = fetch, hint, vs, waves
                if waves == 2:
                    p.combine = 0    # two-wave launches merge by a second launch
                chunks = p.tiles * p.num_splits
                p.grid = chunks if vs == 1 else vs * 8 * -(-chunks // 8)
                say(f"paged planned B{B}-H{H_Q}-KV{H_KV}-{lengths} page={page} {p.as_dict()}")
                lse_t = torch.empty(B, H_Q, dtype=torch.float32, device="cuda")
                out = da.da_decode_attn_paged_planned(q, kc, vc, bt, sl, L, p, lse_out=lse_t)
                torch.cuda.synchronize()
                assert_parity(out, O, f"paged planned {p.as_dict()}")
                check_lse(lse_t, lse)
                # neither the tile width, the fetch path, V slices nor the hint change the bits; the wave
                # count cuts the chunk differently, so two-wave launches are compared among themselves
                ref = by_waves.setdefault(p.group_waves, (out, lse_t))
                assert torch.equal(out.view(torch.int16), ref[0].view(torch.int16)), p.as_dict()
                assert torch.equal(lse_t, ref[1]), p.as_dict()
