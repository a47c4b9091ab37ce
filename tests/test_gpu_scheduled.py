"""GPU parity of the per-sequence scheduled entry point against the fp64
oracle, for contiguous (fixed and varlen) and paged K/V.  Same bar as the
other paths: max-abs <= 2e-2 and mean-abs <= 2e-3 on O, lse within 1e-3;
bit-identical repeats; the same bits as the uniform launch where the chunk
cuts coincide."""

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from oracle import decode_attention
from workloads import config_shapes, custom_shape, make_inputs, paged_layout
from tests.gpu_helpers import assert_parity, dev_inputs, say, to_dev

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def check_lse(lse_t, lse):
    lg = lse_t.cpu().numpy().astype(np.float64)
    fin = np.isfinite(lse)
    assert np.array_equal(np.isfinite(lg), fin)
    assert np.max(np.abs(lg[fin] - lse[fin]), initial=0.0) <= LSE_TOL


def run_sched(q, k, v, lens, H_KV, L_K_max, cu=None, paged=None, chunk_tiles=0, cu_margin=0, pack=-1):
    sched, meta = da.da_make_schedule(lens, q.shape[1], H_KV, L_K_max, pack_gqa=pack, chunk_tiles=chunk_tiles,
                                      cu_margin=cu_margin)
    meta_dev = meta.cuda()
    lse = torch.empty(q.shape[0], q.shape[1], dtype=torch.float32, device="cuda")
    if paged is None:
        out = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu, lse_out=lse)
    else:
        bt, sl = paged
        out = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, block_table=bt, seq_lens=sl, lse_out=lse)
    torch.cuda.synchronize()
    return out, lse, sched


CHUNKS = [0, 1, 2, 5, 40]   # 0: chosen by the cost model


def check_inputs(inp, what, chunks=CHUNKS, page=None, packs=(-1,)):
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    lens = [int(x) for x in inp.lengths]
    L = max(lens + [0]) if inp.cu_seqlens_k is not None else inp.shape.L_K
    H_KV = inp.shape.H_KV
    if page is None:
        q, k, v, cu = dev_inputs(inp)
        paged = None
    else:
        pg = paged_layout(inp, page, seed=page + 3)
        q = to_dev(inp.q)
        k, v = to_dev(pg.k_cache), to_dev(pg.v_cache)
        paged = (torch.from_numpy(pg.block_table).cuda(), torch.from_numpy(pg.seq_lens).cuda())
        cu = None
    for pack in packs:
        for c in chunks:
            say(f"scheduled {what} page={page} chunk={c} pack={pack}")
            out, lse_t, sched = run_sched(q, k, v, lens, H_KV, L, cu=cu, paged=paged, chunk_tiles=c, pack=pack)
            assert_parity(out, O, f"scheduled {what} chunk={c} pack={pack} ({sched.as_dict()})")
            check_lse(lse_t, lse)


@pytest.mark.parametrize("page", [None, 64])
def test_varlen_gqa_scheduled(page):
    sh = config_shapes(4)[0]
    check_inputs(make_inputs(sh), sh.name, page=page, packs=(-1, 0))


@pytest.mark.parametrize("shape", config_shapes(2) + config_shapes(1), ids=lambda s: s.name)
def test_fixed_layout_scheduled(shape):
    check_inputs(make_inputs(shape), shape.name)


@pytest.mark.parametrize("B,H_Q,H_KV,lengths", [
    (4, 8, 1, [0, 1, 1000, 33]),             # empty and single-key sequences
    (4, 8, 1, [5000, 40, 40, 0]),             # one long sequence among short ones
    (3, 128, 2, [700, 2100, 3]),              # two head tiles per KV head
    (2, 12, 4, [300, 95]),                    # group of 3
    (1, 8, 1, [9000]),                        # a single long sequence: up to 64 chunks
    (2, 66, 2, [130, 700]),                   # group of 33: three head tiles of 11 per KV head
    (3, 32, 1, [300, 40, 511]),               # group of 32: 16-head tiles, or one tile with pack_gqa=2
])
@pytest.mark.parametrize("page", [None, 32])
def test_ragged_scheduled(B, H_Q, H_KV, lengths, page):
    sh = custom_shape(B, H_Q, H_KV, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=B * 10 + H_Q, lengths=lengths)
    check_inputs(inp, f"B{B}-H{H_Q}-KV{H_KV}-{lengths}", page=page, packs=(-1, 2) if H_Q // H_KV > 16 else (-1,))


def test_cu_margin_schedule():
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    lens = [int(x) for x in inp.lengths]
    for margin in (0, 64, 200, 255):
        say(f"scheduled cu_margin={margin}")
        out, lse_t, sched = run_sched(q, k, v, lens, sh.H_KV, sh.L_K, cu=cu, cu_margin=margin)
        assert sched.num_cus == da.da_device_info()[0] - margin
        assert_parity(out, O, f"cu_margin={margin}")
        check_lse(lse_t, lse)


@pytest.mark.parametrize("s,pack", [(1, 1), (2, 1), (4, 1), (4, 0)])
def test_scheduled_equals_uniform_when_cuts_coincide(s, pack):
    """Equal lengths of 512 keys cut into s chunks of 512/s keys (whole
    tiles, whole tiles per wave): the scheduled launch computes the same
    chunk states as the uniform one and merges them in the same order."""
    sh = config_shapes(2)[3]
    inp = make_inputs(sh)
    q, k, v, _ = dev_inputs(inp)
    say(f"scheduled vs uniform s={s} pack={pack}")
    a = da.da_decode_attn(q, k, v, num_splits=s, pack_gqa=pack)
    sched, meta = da.da_make_schedule([512], 64, 8, pack_gqa=pack, chunk_tiles=16 // s)
    assert sched.max_splits == s
    b = da.da_decode_attn_scheduled(q, k, v, sched, meta.cuda())
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("page", [None, 32])
@pytest.mark.parametrize("B,H_Q,H_KV,lengths,c", [
    (4, 8, 1, [0, 1, 1000, 33], 0),
    (3, 128, 2, [700, 2100, 3], 2),
    (2, 12, 4, [300, 95], 40),
    (3, 32, 1, [300, 40, 511], 1),
])
def test_scheduled_streaming_hint_same_bits(B, H_Q, H_KV, lengths, c, page):
    """The nontemporal K/V hint (set by the scheduler only past the cache's
    capacity, forced on here) changes how lines are cached, never a
    result: the same bits as without it, on every K/V fetch path the
    schedule picks."""
    sh = custom_shape(B, H_Q, H_KV, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=B * 7 + H_Q, lengths=lengths)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    kw = dict(cu_seqlens_k=cu)
    if page is not None:
        pg = paged_layout(inp, page, seed=page)
        k, v = to_dev(pg.k_cache), to_dev(pg.v_cache)
        kw = dict(block_table=torch.from_numpy(pg.block_table).cuda(), seq_lens=torch.from_numpy(pg.seq_lens).cuda())
    sched, meta = da.da_make_schedule(lengths, H_Q, H_KV, max(lengths), chunk_tiles=c)
    assert sched.kv_nontemporal == 0
    meta_dev = meta.cuda()
    outs = []
    for hint in (0, 1):
        sched.kv_nontemporal = hint
        say(f"scheduled hint={hint} B{B}-H{H_Q}-KV{H_KV} chunk={c} page={page} fetch={sched.kv_fetch}")
        lse_t = torch.empty(B, H_Q, dtype=torch.float32, device="cuda")
        outs.append((da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, lse_out=lse_t, **kw), lse_t))
        torch.cuda.synchronize()
    assert_parity(outs[1][0], O, "streaming hint")
    check_lse(outs[1][1], lse)
    assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
    assert torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("c", [0, 3])
def test_scheduled_bit_identical_repeats(c):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    lens = [int(x) for x in inp.lengths]
    say(f"scheduled repeats chunk={c}")
    first, lse0, _ = run_sched(q, k, v, lens, sh.H_KV, sh.L_K, cu=cu, chunk_tiles=c)
    for _ in range(3):
        again, lse1, _ = run_sched(q, k, v, lens, sh.H_KV, sh.L_K, cu=cu, chunk_tiles=c)
        assert torch.equal(first.view(torch.int16), again.view(torch.int16))
        assert torch.equal(lse0, lse1)


@pytest.mark.parametrize("c", [0, 2])
def test_scheduled_graph_replay_matches_eager(c):
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    q, k, v, cu = dev_inputs(inp)
    lens = [int(x) for x in inp.lengths]
    sched, meta = da.da_make_schedule(lens, sh.H_Q, sh.H_KV, sh.L_K, chunk_tiles=c)
    meta_dev = meta.cuda()
    say(f"scheduled graph replay chunk={c}")
    eager = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu)
    torch.cuda.synchronize()
    out = torch.empty_like(eager)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu, out=out)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu, out=out)
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {r}"
        again = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu)
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int16), eager.view(torch.int16))


def test_ragged_highload_scheduled_sampled():
    """A ragged high-load batch at full size (32 sequences of 1024..16384
    keys, H_Q 64, H_KV 8; about 1.1 GB of K/V): three sequences against the
    oracle, every output finite."""
    rng = np.random.default_rng(2024)
    lengths = [int(x) for x in rng.integers(1024, 16385, 32)]
    sh = custom_shape(32, 64, 8, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=2025, lengths=lengths)
    q, k, v, cu = dev_inputs(inp)
    picks = [int(np.argmax(lengths)), int(np.argmin(lengths)), 7]
    cuh = inp.cu_seqlens_k
    for c in (0, 64):
        say(f"ragged highload scheduled chunk={c}")
        out, lse_t, sched = run_sched(q, k, v, lengths, 8, max(lengths), cu=cu, chunk_tiles=c)
        for b in picks:
            O, lse = decode_attention(inp.q[b:b + 1], inp.k[cuh[b]:cuh[b + 1]][None], inp.v[cuh[b]:cuh[b + 1]][None])
            assert_parity(out[b:b + 1], O, f"ragged highload b={b} chunk={c}")
            assert np.max(np.abs(lse_t[b].cpu().numpy() - lse[0])) <= LSE_TOL
        assert torch.isfinite(out.float()).all()


def test_concurrent_kernel_on_reserved_cus():
    """cu_margin with a concurrent kernel: a GEMM runs on a quarter of the
    CUs (a masked stream) while the decode runs on the rest, planned with
    that margin and without.  Every decode output is bit-identical to the
    same schedule run alone on the whole chip, and matches the oracle."""
    from paper_2604_00028_amd.streams import cu_mask_stream, destroy_stream, split_masks
    cus = da.da_device_info()[0]
    if cus % 32:
        pytest.skip("CU count not a multiple of 32")
    sh = config_shapes(4)[0]
    inp = make_inputs(sh)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    lens = [int(x) for x in inp.lengths]
    reserve_w, decode_w = split_masks(cus, 8)
    say("creating CU-masked streams")
    gs, n_res = cu_mask_stream(reserve_w)
    ds, n_dec = cu_mask_stream(decode_w)
    try:
        assert n_res == cus // 4 and n_dec == cus - cus // 4
        g = torch.Generator(device="cuda").manual_seed(5)
        A = torch.randn(4096, 4096, device="cuda", generator=g).to(torch.bfloat16)
        Bm = torch.randn(4096, 4096, device="cuda", generator=g).to(torch.bfloat16)
        for margin in (0, n_res):
            sched, meta = da.da_make_schedule(lens, sh.H_Q, sh.H_KV, sh.L_K, cu_margin=margin)
            md = meta.cuda()
            say(f"concurrent decode cu_margin={margin} ({sched.num_items} workgroups)")
            alone = da.da_decode_attn_scheduled(q, k, v, sched, md, cu_seqlens_k=cu)
            torch.cuda.synchronize()
            assert_parity(alone, O, f"alone cu_margin={margin}")
            outs = [torch.empty_like(alone) for _ in range(5)]
            with torch.cuda.stream(gs):
                for _ in range(4):
                    torch.matmul(A, Bm)
            for o in outs:
                da.da_decode_attn_scheduled(q, k, v, sched, md, cu_seqlens_k=cu, out=o, stream=ds)
            torch.cuda.synchronize()
            for o in outs:
                assert torch.equal(o.view(torch.int16), alone.view(torch.int16))
    finally:
        destroy_stream(gs)
        destroy_stream(ds)


@pytest.mark.parametrize("page", [None, 64])
def test_device_lengths_differ_from_scheduled(page):
    """The schedule is made for one set of lengths, the device holds others
    (longer and shorter, up to L_K_max): every key is still read once, so the
    result is the oracle's for the device lengths."""
    dev_lens = [700, 1, 333, 1500, 0, 64]
    host_lens = [300, 40, 333, 1500, 90, 1]
    sh = custom_shape(len(dev_lens), 16, 2, 1500, varlen=True)
    inp = make_inputs(sh, seed=61, lengths=dev_lens)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    if page is None:
        q, k, v, cu = dev_inputs(inp)
        extra = dict(cu_seqlens_k=cu)
    else:
        pg = paged_layout(inp, page, seed=62)
        q = to_dev(inp.q)
        k, v = to_dev(pg.k_cache), to_dev(pg.v_cache)
        extra = dict(block_table=torch.from_numpy(pg.block_table).cuda(),
                     seq_lens=torch.from_numpy(pg.seq_lens).cuda())
    for c in (0, 2, 7):
        sched, meta = da.da_make_schedule(host_lens, sh.H_Q, sh.H_KV, 1500, chunk_tiles=c)
        say(f"scheduled lengths differ page={page} chunk={c}")
        lse_t = torch.empty(sh.B, sh.H_Q, dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_scheduled(q, k, v, sched, meta.cuda(), lse_out=lse_t, **extra)
        torch.cuda.synchronize()
        assert_parity(out, O, f"lengths differ page={page} chunk={c}")
        check_lse(lse_t, lse)


@pytest.mark.parametrize("page", [None, 32])
@pytest.mark.parametrize("B,H_Q,H_KV,lengths,c", [
    (4, 8, 1, [0, 1, 1000, 33], 1),        # 32 chunks: batches of 8 through LDS
    (3, 128, 2, [700, 2100, 3], 2),        # 32-head tiles or 16-head ones, 17 chunks
    (2, 12, 4, [300, 95], 4),              # 3 chunks: one batch in registers
    (3, 32, 1, [300, 40, 511], 1),         # 16 chunks
    (2, 8, 1, [4096, 32], 2),              # 64 chunks, the most a sequence takes
    (5, 64, 8, [2000, 17, 0, 900, 4100], 0),
])
def test_scheduled_merge_in_launch(B, H_Q, H_KV, lengths, c, page):
    """The chunk states of split sequences merged by the last workgroup of
    each head tile inside the split launch, or by the combine launch: both
    against the oracle, with the same bits (the merge takes the same
    operations in the same order either way), twice in a row (the arrival
    counters return to zero)."""
    sh = custom_shape(B, H_Q, H_KV, max(lengths), varlen=True)
    inp = make_inputs(sh, seed=B * 13 + H_Q + c, lengths=lengths)
    O, lse = decode_attention(inp.q, inp.k, inp.v, inp.lengths, inp.cu_seqlens_k)
    q, k, v, cu = dev_inputs(inp)
    kw = dict(cu_seqlens_k=cu)
    if page is not None:
        pg = paged_layout(inp, page, seed=page + 1)
        k, v = to_dev(pg.k_cache), to_dev(pg.v_cache)
        kw = dict(block_table=torch.from_numpy(pg.block_table).cuda(), seq_lens=torch.from_numpy(pg.seq_lens).cuda())
    sched, meta = da.da_make_schedule(lengths, H_Q, H_KV, max(lengths), chunk_tiles=c)
    assert sched.state_rows > 0
    meta_dev = meta.cuda()
    got = {}
    for comb in (sched.combine, 1 - sched.combine, sched.combine, 1):
        sched.combine = comb
        say(f"scheduled merge combine={comb} B{B}-H{H_Q}-KV{H_KV} chunk={c} page={page} {sched.as_dict()}")
        lse_t = torch.empty(B, H_Q, dtype=torch.float32, device="cuda")
        out = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, lse_out=lse_t, **kw)
        torch.cuda.synchronize()
        assert_parity(out, O, f"scheduled merge combine={comb} ({sched.as_dict()})")
        check_lse(lse_t, lse)
        if got:
            first = next(iter(got.values()))
            assert torch.equal(out.view(torch.int16), first[0].view(torch.int16)), comb
            assert torch.equal(lse_t, first[1]), comb
        got[len(got)] = (out, lse_t)


@pytest.mark.parametrize("comb", [0, 1])
def test_scheduled_merge_graph_replay(comb):
    """A captured scheduled launch with either merge, replayed with eager
    calls in between: every replay gives the eager bits (the in-launch
    merge's counters are reset by the kernel itself, no memset node)."""
    lens = [2000, 17, 0, 900, 4100, 333]
    sh = custom_shape(len(lens), 64, 8, max(lens), varlen=True)
    inp = make_inputs(sh, seed=99, lengths=lens)
    q, k, v, cu = dev_inputs(inp)
    sched, meta = da.da_make_schedule(lens, 64, 8, max(lens), chunk_tiles=3)
    assert sched.state_rows > 0
    sched.combine = comb
    meta_dev = meta.cuda()
    say(f"scheduled merge graph replay combine={comb}")
    eager = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu)
    torch.cuda.synchronize()
    out = torch.empty_like(eager)
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(stream):
        da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu, out=out)
    torch.cuda.current_stream().wait_stream(stream)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu, out=out)
    for r in range(4):
        out.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {r}"
        again = da.da_decode_attn_scheduled(q, k, v, sched, meta_dev, cu_seqlens_k=cu)
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int16), eager.view(torch.int16))
