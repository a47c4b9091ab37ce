"""Randomised checks of the planner and the scheduler on the CPU: whatever
shape, policy, forced split count, packing or CU margin a caller asks for,
the plan (or schedule) that comes back describes a launch the library's own
entry points accept, with consistent fields, workspace sizes and modelled
time.  No kernel runs: a plan that passes every check reaches the device
query, which fails here with DA_ERR_HIP."""

import ctypes

from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import paper_2604_00028_amd as da
from paper_2604_00028_amd import _binding as bnd
from paper_2604_00028_amd import calibrate as cal

FAKE = 1 << 20
P = ctypes.c_void_p
POLICIES = [da.POLICY_MI355X, da.POLICY_STREAMED, da.POLICY_PAPER, da.POLICY_EVOLVED, da.POLICY_TABLE,
            da.POLICY_TABLE_STREAMED]
# the shapes the split tables hold, so that the TABLE policies' own plans are drawn too
TABLE_SHAPES = sorted({e[:4] for t in ("warm", "streamed") for e in cal.tables_all()[t]})


def launch_grid(chunks, vs):
    return chunks if vs == 1 else vs * 8 * -(-chunks // 8)


@st.composite
def shapes(draw):
    H_KV = draw(st.sampled_from([1, 2, 4, 8, 32]))
    g = draw(st.sampled_from([1, 2, 3, 8, 16, 24, 32, 48, 64]))
    B = draw(st.integers(1, 64))
    L = draw(st.integers(0, 20000))
    return B, H_KV * g, H_KV, L


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.one_of(shapes(), st.sampled_from(TABLE_SHAPES)), st.sampled_from(POLICIES),
       st.one_of(st.just(0), st.integers(0, 64)), st.sampled_from([-1, -1, 0, 1, 2]), st.sampled_from([0, 0, 17, 200]))
def test_every_plan_is_a_launch_the_library_accepts(shape, policy, s, pack, margin):
    B, H_Q, H_KV, L = shape
    cus = 256
    state_bytes = lambda n: n * B * H_Q * 128 * 4
    try:
        plan = da.da_make_plan(B, H_Q, H_KV, L, num_splits=s, pack_gqa=pack, num_cus=cus, cu_margin=margin,
                               policy=policy)
    except bnd.DecodeAttnError as e:
        # a forced split whose chunk states would pass 2 GiB is refused
        assert e.code == bnd.DA_ERR_SHAPE and s > 1 and state_bytes(s) >= 1 << 31, (shape, s)
        return
    assert plan.num_splits == 1 or state_bytes(plan.num_splits) < 1 << 31
    g = H_Q // H_KV
    # fields
    assert 1 <= plan.num_splits <= 64 and (s == 0 or plan.num_splits == s)
    assert plan.pack_gqa in (0, 1, 2) and (pack < 0 or plan.pack_gqa == pack)
    assert H_Q % plan.heads_per_tile == 0 and plan.tiles == B * H_Q // plan.heads_per_tile
    assert plan.heads_per_tile <= 32 and (plan.pack_gqa > 0 or plan.heads_per_tile == 1)
    assert plan.v_slices in (1, 2, 4) and plan.grid == launch_grid(plan.tiles * plan.num_splits, plan.v_slices)
    assert plan.v_slices == 1 or (plan.kv_fetch == 2 and plan.grid <= cus - margin)
    assert plan.combine in (0, 1) and (plan.combine == 0 or (plan.num_splits > 1 and plan.tiles <= 4096))
    assert plan.num_cus == cus - margin and plan.kv_fetch in (0, 1, 2) and plan.kv_nontemporal in (0, 1)
    # two waves only for a launch of 3/4 to 5/4 as many workgroups as CUs, long chunks, keys read once
    assert plan.group_waves in (2, 4)
    C, chunk = cus - margin, -(-L // plan.num_splits)
    assert plan.wg_per_cu in (0, 1) and (plan.wg_per_cu == 0 or plan.group_waves == 2)
    if plan.group_waves == 2 and plan.wg_per_cu == 1:
        # two waves held to one workgroup per CU: 2-4 nearly full rounds of long chunks, 2+ KV heads
        rounds = -(-plan.grid // C)
        assert 4 * plan.grid > 5 * C and 2 <= rounds <= 4 and 8 * (rounds * C - plan.grid) <= C and H_KV >= 2
        assert chunk >= (4096 if rounds == 4 else 2048) and plan.kv_fetch == 1
        assert plan.v_slices == 1 and plan.combine == 0 and plan.heads_per_tile == g
    elif plan.group_waves == 2:
        assert plan.kv_fetch in (0, 1) and plan.v_slices == 1 and plan.combine == 0
        top = (4 * C if chunk >= 2048 else 3 * C if chunk >= 1024 else 5 * C // 4) if H_KV == 1 else 5 * C // 4
        assert 4 * plan.grid >= 3 * C and plan.grid <= top
        assert plan.kv_fetch == (0 if H_KV == 1 and plan.grid <= cus - margin else 1)
        assert -(-L // plan.num_splits) >= 512 and plan.heads_per_tile == g
    if g > 1 and plan.pack_gqa == 1:
        assert plan.heads_per_tile in {min(g, 32) if g <= 32 else max(h for h in range(1, 33) if g % h == 0),
                                       min(g, 16) if g <= 16 else max(h for h in range(1, 17) if g % h == 0)}
    # workspace and modelled time
    ws = da.da_workspace_bytes(B, H_Q, 128, plan.num_splits)
    assert (ws == 0) == (plan.num_splits == 1)
    assert da.da_model_time(policy, B, H_Q, H_KV, L, plan.heads_per_tile, plan.num_splits, plan.v_slices,
                            plan.combine, cus - margin) > 0
    # the planned entry point accepts it (and refuses it without its workspace)
    call = lambda w, wb: da.load().da_decode_attn_planned(P(FAKE), P(FAKE), P(FAKE), None, P(FAKE), None, B, H_Q,
                                                          H_KV, L, 128, 0.0, ctypes.byref(plan), w, wb, None)
    assert call(P(FAKE), max(ws, 256)) == bnd.DA_ERR_HIP
    if ws:
        assert call(P(FAKE), ws - 1) == bnd.DA_ERR_WORKSPACE


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.lists(st.integers(0, 40000), min_size=1, max_size=96), st.sampled_from([(8, 1), (64, 8), (32, 4), (32, 1),
                                                                              (128, 2), (24, 8)]),
       st.sampled_from([0, 0, 1, 3, 40]), st.sampled_from([-1, 0, 1, 2]), st.sampled_from([0, 64]))
def test_every_schedule_is_a_launch_the_library_accepts(lens, heads, chunk, pack, margin):
    H_Q, H_KV = heads
    L = max(lens)
    sched, meta = da.da_make_schedule(lens, H_Q, H_KV, L, pack_gqa=pack, chunk_tiles=chunk, num_cus=256,
                                      cu_margin=margin)
    assert sched.B == len(lens) and sched.tiles == len(lens) * (H_Q // sched.heads_per_tile)
    assert 1 <= sched.max_splits <= 64 and (sched.state_rows > 0) == (sched.max_splits > 1)
    assert sched.combine in (0, 1) and (sched.combine == 0 or (sched.state_rows > 0 and sched.tiles <= 4096))
    assert sched.num_cus == 256 - margin and meta.numel() >= sched.meta_bytes
    # per-sequence table: split counts, first state rows, one item per (sequence chunk, head tile)
    raw = bytes(meta.numpy()[:sched.meta_bytes])
    seq = memoryview(raw)[sched.seq_offset:sched.seq_offset + 8 * sched.B].cast("i")
    tps = H_Q // sched.heads_per_tile
    assert sum(seq[2 * b + 1] for b in range(sched.B)) * tps == sched.num_items
    rows = 0
    for b in range(sched.B):
        first, count = seq[2 * b], seq[2 * b + 1]
        assert 1 <= count <= 64
        assert (first == -1) == (count == 1) and (first == -1 or first == rows)
        rows += count if count > 1 else 0
    assert rows == sched.state_rows
    ws = da.da_schedule_workspace_bytes(sched)
    assert (ws == 0) == (sched.state_rows == 0)
    call = lambda w, wb: da.load().da_decode_attn_scheduled(P(FAKE), P(FAKE), P(FAKE), None, None, None, 0, 0, 0,
                                                            P(FAKE), None, 128, 0.0, ctypes.byref(sched), P(FAKE),
                                                            w, wb, None)
    assert call(P(FAKE), max(ws, 256)) == bnd.DA_ERR_HIP
    if ws:
        assert call(P(FAKE), ws - 1) == bnd.DA_ERR_WORKSPACE
