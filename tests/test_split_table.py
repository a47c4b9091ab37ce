"""The configuration-specific split table (policies TABLE and TABLE_STREAMED;
the paper leaves learning split counts per configuration to future work,
Sections 3.3, 4.1 and 4.2): the generated table holds, for every shape of the
committed calibration sweeps, the launch measured fastest there, and the
library plans those shapes with it and every other shape as the cost model
does.  CPU only: the sweeps are read from profiles/, the plans from the
library's host planner."""

import json
import os

import pytest

import paper_2604_00028_amd as da
from paper_2604_00028_amd import calibrate as cal

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SWEEPS = {"warm": os.path.join(ROOT, "profiles", "calibration_warm.json"),
          "streamed": os.path.join(ROOT, "profiles", "calibration_streamed.json")}
POLICY = {"warm": (da.POLICY_TABLE, da.POLICY_MI355X), "streamed": (da.POLICY_TABLE_STREAMED, da.POLICY_STREAMED)}
FIELDS = ("num_splits", "pack_gqa", "heads_per_tile", "tiles", "grid", "num_cus", "group_waves", "kv_fetch",
          "kv_nontemporal", "v_slices", "combine", "wg_per_cu")


def fastest(shape):
    """The launch the table must hold for one sweep shape, read straight from
    the sweep: among the launches the planner may choose (V slices only up to
    16 MiB of K/V), the fewest chunks within 1% of the fastest, then the
    fastest of those."""
    kv = shape["B"] * shape["L"] * shape["H_KV"] * 512
    runs = [r for r in shape["launches"] if r[2] == 1 or kv <= 16 << 20]
    best = min(r[4] for r in runs)
    near = sorted((r[1], r[4], tuple(r[:4])) for r in runs if r[4] <= 1.01 * best)
    return near[0][2]


def fields(p):
    return {f: getattr(p, f) for f in FIELDS}


def test_header_is_generated_from_the_committed_sweeps():
    got = cal.parse_table(open(cal.TABLE_SPLIT).read())
    want = cal.tables_all()
    assert got["warm"] == want["warm"] and got["streamed"] == want["streamed"]
    for which, path in SWEEPS.items():
        assert got["cus"] == json.load(open(path))["device_cus"]


@pytest.mark.parametrize("which", ["warm", "streamed"])
def test_table_holds_the_fastest_launch_of_every_swept_shape(which):
    sweep = json.load(open(SWEEPS[which]))
    table = {e[:4]: e[4:] for e in cal.parse_table(open(cal.TABLE_SPLIT).read())[which]}
    assert len(table) == len(sweep["shapes"])
    for sh in sweep["shapes"]:
        assert table[(sh["B"], sh["H_Q"], sh["H_KV"], sh["L"])] == fastest(sh), sh


@pytest.mark.parametrize("which", ["warm", "streamed"])
def test_swept_shapes_are_planned_from_the_table(which):
    policy, model = POLICY[which]
    sweep = json.load(open(SWEEPS[which]))
    for sh in sweep["shapes"]:
        B, H_Q, H_KV, L = sh["B"], sh["H_Q"], sh["H_KV"], sh["L"]
        hpt, s, vs, comb = fastest(sh)
        p = da.da_choose_splits(B, H_Q, H_KV, L, num_cus=256, policy=policy)
        assert (p.heads_per_tile, p.num_splits, p.v_slices, p.combine) == (hpt, s, vs, comb), sh
        # the rest of the launch as the sweep ran it: the planner's fetch path and cache hint
        assert p.pack_gqa == 1 and p.tiles == B * H_Q // hpt and p.num_cus == 256
        assert p.grid == (p.tiles * s if vs == 1 else vs * 8 * -(-(p.tiles * s) // 8))
        chunk = -(-L // s)
        tpw = -(-(-(-chunk // 4)) // 32)
        readers = (H_Q // H_KV // hpt) * vs
        # two waves where the launch has 3/4 to 5/4 as many workgroups as CUs (3 times as many for pure
        # MQA over chunks of >= 1024 keys), one workgroup reads each key, chunks hold >= 512 keys and no
        # merge runs in the launch; the sweep timed four waves
        top = (1024 if chunk >= 2048 else 768 if chunk >= 1024 else 320) if H_KV == 1 else 320
        two = vs == 1 and readers == 1 and comb == 0 and 192 <= p.grid <= top and chunk >= 512
        # or two waves held to one workgroup per CU over 2-4 nearly full rounds of long chunks
        rounds = -(-p.grid // 256)
        held = (not two and vs == 1 and readers == 1 and comb == 0 and H_KV >= 2 and p.grid > 320 and
                2 <= rounds <= 4 and 8 * (rounds * 256 - p.grid) <= 256 and chunk >= (4096 if rounds == 4 else 2048))
        two = two or held
        assert p.group_waves == (2 if two else 4) and p.wg_per_cu == int(held), sh
        fetch = (0 if H_KV == 1 and p.grid <= 256 else 1) if two else (2 if p.grid <= 256 else (1 if tpw >= 2 else 0))
        assert p.kv_fetch == fetch, sh
        nt = readers == 1 if which == "streamed" else (readers == 1 and B * L * H_KV * 512 > 288 << 20)
        assert p.kv_nontemporal == int(nt), sh


@pytest.mark.parametrize("which", ["warm", "streamed"])
def test_other_requests_fall_back_to_the_cost_model(which):
    policy, model = POLICY[which]
    def same(shape, **kw):
        return fields(da.da_make_plan(*shape, 128, policy=policy, **kw)) == \
            fields(da.da_make_plan(*shape, 128, policy=model, **kw))
    sweep = json.load(open(SWEEPS[which]))
    timed = {(sh["B"], sh["H_Q"], sh["H_KV"], sh["L"]) for sh in sweep["shapes"]}
    # shapes the sweep did not time: a neighbouring length, batch or head count
    others = [(1, 64, 8, 500), (2, 64, 8, 512), (3, 16, 2, 1000), (1, 24, 8, 512), (7, 32, 1, 8191), (1, 8, 1, 0),
              (64, 64, 8, 4096), (1, 64, 8, 100000)]
    for sh in others:
        assert sh not in timed
        assert same(sh, num_splits=0, pack_gqa=-1, num_cus=256), sh
    for sh in sorted(timed)[::7]:
        # a forced split count or packing, another CU count or a CU margin: the model plans it
        assert same(sh, num_splits=2, pack_gqa=-1, num_cus=256), sh
        assert same(sh, num_splits=0, pack_gqa=2, num_cus=256), sh
        assert same(sh, num_splits=0, pack_gqa=0, num_cus=256), sh
        assert same(sh, num_splits=0, pack_gqa=-1, num_cus=304), sh
        assert same(sh, num_splits=0, pack_gqa=-1, num_cus=256, cu_margin=16), sh
        # an explicit pack_gqa = 1 is the default packing: the table still applies
        t = da.da_make_plan(*sh, 128, num_splits=0, pack_gqa=1, num_cus=256, policy=policy)
        assert fields(t) == fields(da.da_choose_splits(*sh, num_cus=256, policy=policy)), sh


def test_table_policies_price_launches_with_their_models():
    for table, model in POLICY.values():
        for args in ((1, 64, 8, 512, 8, 4, 4, 1, 256), (32, 64, 8, 8192, 8, 1, 1, 0, 256)):
            assert da.da_model_time(table, *args) == da.da_model_time(model, *args)


def test_nearest_shape_lookup_does_worse_than_the_model_on_held_out_shapes():
    """Why the table is looked up by exact shape only: each swept shape planned
    from its nearest swept neighbour (that shape left out) lands further from
    the fastest launch than the cost model does, on both sweeps."""
    fields = ["base0", "base1", "tt0", "tt1", "ts0", "ts1", "merge0", "merge1_0", "merge1_1", "fused0", "fused1_0",
              "fused1_1", "fused2", "hbm_rate", "hbm0", "pnorm", "contig", "vs1", "vs2", "vs4"]
    consts = cal.parse_header(open(cal.HEADER).read())
    for which in SWEEPS:
        c = dict(zip(fields, consts[which]))
        r = cal.table_holdout(json.load(open(SWEEPS[which])), c)
        assert r["nearest"]["mean_vs_best"] > r["model"]["mean_vs_best"], (which, r)
        assert r["nearest"]["within_5pct"] < r["model"]["within_5pct"], (which, r)
