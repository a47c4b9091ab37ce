"""Host checks of the per-sequence schedule (da_make_schedule): every
sequence's keys are covered exactly once per head tile, state rows are laid
out as the combine reads them, and the planner's choices follow its model.
No device access: num_cus is given."""

import ctypes

import numpy as np
import pytest
import torch

import paper_2604_00028_amd as da
from paper_2604_00028_amd import _binding as bnd

CUS = 256
FAKE = 1 << 20


def unpack(sched, meta):
    items = meta[: sched.num_items * 16].view(torch.int32).view(-1, 4).numpy()
    seqs = meta[sched.seq_offset: sched.seq_offset + 8 * sched.B].view(torch.int32).view(-1, 2).numpy()
    return items, seqs


def check_schedule(lens, H_Q, H_KV, **kw):
    sched, meta = da.da_make_schedule(lens, H_Q, H_KV, num_cus=kw.pop("num_cus", CUS), **kw)
    items, seqs = unpack(sched, meta)
    B = len(lens)
    hpt = sched.heads_per_tile
    tps = H_Q // hpt
    assert sched.tiles == B * tps and len(items) == sched.num_items
    assert sched.meta_bytes == sched.num_items * 16 + 8 * B
    # per (sequence, head tile): the tile ranges partition [0, T_b)
    cover = {}
    for tile, t0, t1, row in items:
        assert 0 <= tile < sched.tiles and 0 <= t0 <= t1
        cover.setdefault(int(tile), []).append((int(t0), int(t1), int(row)))
    assert sorted(cover) == list(range(sched.tiles))
    rows_seen = set()
    for b, L in enumerate(lens):
        T = -(-L // 32)
        r0, s = (int(x) for x in seqs[b])
        assert 1 <= s <= 64 and s <= max(T, 1)
        for ht in range(tps):
            ranges = sorted(cover[b * tps + ht])
            assert len(ranges) == s
            # the last chunk runs to the sequence end (INT32_MAX), the others are exact
            assert ranges[0][0] == 0 and ranges[-1][1] == 2**31 - 1 and (s == 1 or ranges[-2][1] <= T)
            assert all(a[1] == c[0] for a, c in zip(ranges, ranges[1:]))
            if s == 1:
                assert r0 == -1 and ranges[0][2] == -1
            else:
                # chunk i of sequence b writes state row r0 + i, for every head tile
                assert [r for _, _, r in ranges] == list(range(r0, r0 + s))
        if s > 1:
            rows_seen.update(range(r0, r0 + s))
    assert rows_seen == set(range(sched.state_rows))
    assert sched.max_splits == max(int(s) for s in seqs[:, 1])
    return sched, items, seqs


RAGGED = [
    ([512], 64, 8),
    ([128], 8, 1),
    ([0, 1, 5, 31, 32, 33], 8, 1),
    (list(np.random.default_rng(1).integers(32, 513, 16)), 32, 4),
    (list(np.random.default_rng(2).integers(1024, 16385, 32)), 64, 8),
    ([32768] + [256] * 7, 8, 1),
    ([700, 9000, 3], 128, 2),      # two head tiles per KV head
    ([300, 40], 12, 4),            # unpacked-size group of 3
]


@pytest.mark.parametrize("lens,H_Q,H_KV", RAGGED)
def test_schedule_covers_every_key_once(lens, H_Q, H_KV):
    check_schedule([int(x) for x in lens], H_Q, H_KV)


@pytest.mark.parametrize("c", [1, 3, 16, 1000])
def test_forced_chunk_length(c):
    lens = [0, 1, 100, 2049, 5000]
    sched, items, seqs = check_schedule(lens, 16, 2, chunk_tiles=c)
    assert sched.chunk_tiles == c
    for b, L in enumerate(lens):
        T = -(-L // 32)
        assert seqs[b][1] == (min(64, -(-T // c)) if T else 1)


def test_longest_chunks_first():
    lens = [int(x) for x in np.random.default_rng(3).integers(1, 9000, 24)]
    sched, items, seqs = check_schedule(lens, 32, 4)
    tps = 32 // sched.heads_per_tile
    T = np.array([-(-L // 32) for L in lens])
    end = np.where(items[:, 2] == 2**31 - 1, T[items[:, 0] // tps], items[:, 2])
    n = end - items[:, 1]
    assert np.all(n[:-1] >= n[1:])


@pytest.mark.parametrize("lens,H_Q,H_KV", [([4096, 4096, 2000, 64], 128, 2), ([700, 33, 5000], 64, 1),
                                           ([300, 301], 16, 16), ([130, 700, 9000], 66, 2)])
def test_shared_kv_heads_grouped_on_one_xcd(lens, H_Q, H_KV):
    """Where G head tiles read one KV head, the G workgroups of one
    (sequence, KV head, chunk) start on one XCD (workgroup i on XCD i % 8),
    except in a last partial block of 8G workgroups."""
    sched, items, _ = check_schedule(lens, H_Q, H_KV)
    G = (H_Q // H_KV) // sched.heads_per_tile
    tps = H_Q // sched.heads_per_tile
    groups = {}
    for bid, (tile, t0, t1, row) in enumerate(items):
        b, t = divmod(int(tile), tps)
        groups.setdefault((b, t // G, int(t0)), []).append(bid)
    assert all(len(v) == G for v in groups.values())
    tail = sched.num_items - sched.num_items % (8 * G)
    for bids in groups.values():
        if max(bids) < tail:
            assert len({x % 8 for x in bids}) == 1
            assert max(bids) - min(bids) == 8 * (G - 1)


def test_equal_lengths_match_the_uniform_plan():
    """Where every sequence has the same length the schedule is the uniform
    launch: the same split count as the MI355X plan for L a multiple of 128
    (its key-granular waves then hold whole tiles).  Schedules do not share
    chunks among V slices, so the comparison is with the plan without them
    (the whole group in one tile gives it where a group is one tile; for
    wider groups only the uniform shape of the schedule is checked)."""
    for B, H_Q, H_KV in ((1, 64, 8), (1, 8, 1), (4, 32, 1), (32, 64, 8), (8, 16, 2)):
        for L in (128, 512, 2048, 8192):
            plan = da.da_choose_splits(B, H_Q, H_KV, L, num_cus=CUS)
            sched, _, seqs = check_schedule([L] * B, H_Q, H_KV)
            if plan.v_slices > 1 and H_Q // H_KV > 16:
                assert len(set(seqs[:, 1])) == 1 and sched.num_items == sched.tiles * seqs[0, 1]
                continue
            if plan.v_slices > 1:
                plan = da.da_make_plan(B, H_Q, H_KV, L, num_splits=0, pack_gqa=2, num_cus=CUS)
            assert set(seqs[:, 1]) == {plan.num_splits}, (B, H_Q, H_KV, L)
            # schedules keep four waves per workgroup; where the plan takes two (about a chip of long
            # chunks), the four-wave launch fetches straight into LDS with one workgroup per CU and
            # through registers where some CUs hold two
            fetch = plan.kv_fetch if plan.group_waves == 4 else (2 if plan.grid <= CUS else 1)
            assert sched.num_items == plan.grid and sched.kv_fetch == fetch, (B, H_Q, H_KV, L)


def test_split_counts_follow_length():
    lens = [32768] + [256] * 7
    _, _, seqs = check_schedule(lens, 8, 1)
    assert seqs[0][1] > 1 and all(s == 1 for s in seqs[1:, 1])


def test_cu_margin_plans_for_fewer_cus():
    lens = [int(x) for x in np.random.default_rng(4).integers(1024, 16385, 32)]
    a, _, _ = check_schedule(lens, 64, 8)
    b, _, _ = check_schedule(lens, 64, 8, cu_margin=128)
    assert a.num_cus == CUS and b.num_cus == CUS - 128
    # a single long sequence: fewer CUs, fewer useful chunks
    c, _, sc = check_schedule([16384], 8, 1)
    d, _, sd = check_schedule([16384], 8, 1, cu_margin=224)
    assert sd[0][1] <= sc[0][1]


def test_schedule_is_deterministic():
    lens = [int(x) for x in np.random.default_rng(5).integers(0, 5000, 40)]
    s1, m1 = da.da_make_schedule(lens, 32, 4, num_cus=CUS)
    s2, m2 = da.da_make_schedule(lens, 32, 4, num_cus=CUS)
    assert s1.as_dict() == s2.as_dict() and torch.equal(m1, m2)


def test_schedule_errors():
    lib = da.load()
    out = bnd.DaSchedule()
    lens = (ctypes.c_int32 * 3)(10, 20, 30)
    buf = (ctypes.c_uint8 * 4096)()
    call = lambda *a: lib.da_make_schedule(*a, ctypes.byref(out))  # noqa: E731
    assert call(None, 3, 8, 1, 30, 128, -1, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_NULL
    assert call(lens, 3, 8, 1, 29, 128, -1, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_SHAPE   # a length > L_K_max
    assert call(lens, 3, 8, 3, 30, 128, -1, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_SHAPE   # H_Q % H_KV
    assert call(lens, 3, 8, 1, 30, 64, -1, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_UNSUPPORTED
    assert call(lens, 3, 8, 1, 30, 128, 3, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_ARG
    assert call(lens, 3, 8, 1, 30, 128, -1, CUS, CUS, 0, buf, 4096) == bnd.DA_ERR_ARG   # cu_margin
    assert call(lens, 3, 8, 1, 30, 128, -1, CUS, 0, 0, buf, 8) == bnd.DA_ERR_WORKSPACE
    assert out.meta_bytes == 3 * 16 + 3 * 8          # the size needed is reported
    assert call(lens, 3, 8, 1, 30, 128, -1, CUS, 0, 0, buf, out.meta_bytes) == bnd.DA_OK
    neg = (ctypes.c_int32 * 1)(-1)
    assert call(neg, 1, 8, 1, 30, 128, -1, CUS, 0, 0, buf, 4096) == bnd.DA_ERR_SHAPE


def test_schedule_head_tile_width_checked():
    # g = 32 at short lengths: 16-head tiles; the launch accepts them (it gets
    # past the schedule check to the NULL output) and rejects widths the
    # packing mode cannot produce
    lib = da.load()
    s, _ = da.da_make_schedule([300, 40, 511], 32, 1, num_cus=CUS)
    assert (s.pack_gqa, s.heads_per_tile, s.tiles) == (1, 16, 6)
    need = da.da_schedule_workspace_bytes(s)
    assert scheduled(lib, s, out=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_NULL
    for pack, hpt in ((1, 8), (2, 16), (0, 16)):
        bad = bnd.DaSchedule.from_buffer_copy(s)
        bad.pack_gqa, bad.heads_per_tile = pack, hpt
        assert scheduled(lib, bad, out=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_ARG, (pack, hpt)
    # pack_gqa = 2 keeps the whole group in one tile
    w, _ = da.da_make_schedule([300, 40, 511], 32, 1, num_cus=CUS, pack_gqa=2)
    assert (w.pack_gqa, w.heads_per_tile, w.tiles) == (2, 32, 3)
    assert scheduled(lib, w, out=None, ws=FAKE, ws_bytes=da.da_schedule_workspace_bytes(w)) == bnd.DA_ERR_NULL


def test_schedule_workspace_bytes():
    s, _ = da.da_make_schedule([8192, 100], 16, 2, num_cus=CUS, chunk_tiles=16)
    assert s.state_rows == 16
    # Otilde [16 rows, 16 heads, 128] | m [16, 16] | l [16, 16], 256-byte aligned, then the
    # arrival counter region the merge inside the split launch counts in
    assert da.da_schedule_workspace_bytes(s) == 16 * 16 * 128 * 4 + 2 * 1024 + (1 << 20)
    one, _ = da.da_make_schedule([100, 100], 16, 2, num_cus=CUS)
    assert one.state_rows == 0 and da.da_schedule_workspace_bytes(one) == 0 and one.combine == 0


def test_schedule_merge_choice():
    """A schedule merges its split sequences inside the split launch when
    the MI355X model prices that below a second launch for its longest
    split count: the same choice as a uniform plan of that split count."""
    for lens, H_Q, H_KV, c in (([8192, 100], 16, 2, 16), ([4096, 64, 900], 64, 8, 4), ([32768] + [256] * 7, 8, 1, 0),
                               ([20000, 10], 8, 1, 4)):
        s, _ = da.da_make_schedule(lens, H_Q, H_KV, num_cus=CUS, chunk_tiles=c)
        assert s.state_rows > 0
        plan = da.da_make_plan(len(lens), H_Q, H_KV, max(lens), num_splits=s.max_splits, pack_gqa=s.pack_gqa,
                               num_cus=CUS)
        want = 1 if plan.heads_per_tile == s.heads_per_tile and plan.combine == 1 else None
        if want is not None:
            assert s.combine == want, (lens, s.as_dict())
        assert s.combine in (0, 1)
    # 4096-key sequence in 32-key tiles of 1: 64 chunks, beyond the register batch -- priced, still a choice
    s, _ = da.da_make_schedule([4096, 32], 8, 1, num_cus=CUS, chunk_tiles=2)
    assert s.max_splits == 64 and s.combine in (0, 1)


def scheduled(lib, sched, meta=FAKE, q=FAKE, k=FAKE, v=FAKE, cu=None, bt=None, sl=None, page=64, mp=4, npg=4,
              out=FAKE, ws=None, ws_bytes=0, d=128):
    return lib.da_decode_attn_scheduled(q, k, v, cu, bt, sl, page, mp, npg, out, None, d, 0.0, ctypes.byref(sched),
                                        meta, ws, ws_bytes, None)


def test_scheduled_argument_errors():
    lib = da.load()
    s, _ = da.da_make_schedule([200, 3000], 16, 2, num_cus=CUS, chunk_tiles=8)
    assert s.state_rows > 0
    need = da.da_schedule_workspace_bytes(s)
    assert scheduled(lib, s, ws=None) == bnd.DA_ERR_WORKSPACE
    assert scheduled(lib, s, ws=FAKE, ws_bytes=need - 1) == bnd.DA_ERR_WORKSPACE
    assert scheduled(lib, s, meta=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_NULL
    assert scheduled(lib, s, meta=FAKE + 4, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_ALIGN
    assert scheduled(lib, s, out=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_NULL
    assert scheduled(lib, s, q=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_NULL
    assert scheduled(lib, s, d=64, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_UNSUPPORTED
    # paged layout checks
    assert scheduled(lib, s, bt=FAKE, sl=None, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_NULL
    assert scheduled(lib, s, bt=FAKE, sl=FAKE, page=48, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_UNSUPPORTED
    assert scheduled(lib, s, bt=FAKE, sl=FAKE, page=64, mp=2, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_SHAPE
    # a schedule that does not describe this launch
    for field, val in (("tiles", 3), ("heads_per_tile", 4), ("max_splits", 65), ("num_items", 1),
                       ("seq_offset", 0), ("state_rows", 0), ("kv_fetch", 3), ("pack_gqa", 5),
                       ("kv_nontemporal", 2), ("kv_nontemporal", -1), ("combine", 2), ("combine", -1)):
        bad = bnd.DaSchedule.from_buffer_copy(s)
        setattr(bad, field, val)
        assert scheduled(lib, bad, ws=FAKE, ws_bytes=need) == bnd.DA_ERR_ARG, field
    assert lib.da_decode_attn_scheduled(FAKE, FAKE, FAKE, None, None, None, 0, 0, 0, FAKE, None, 128, 0.0, None,
                                        FAKE, None, 0, None) == bnd.DA_ERR_NULL
