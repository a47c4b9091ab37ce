"""Calibration of the planner's cost models from measured sweeps.

    python -m paper_2604_00028_amd.calibrate            # fit and print
    python -m paper_2604_00028_amd.calibrate --write    # also regenerate csrc/cost_model.inc and split_table.inc

The split policy (paper Section 4) replaces the paper's H100 rule with a cost
model over num_splits in [1, 64]; its constants are measured on MI355X.  The
measurements are committed sweep summaries under profiles/ (written by
`bench.py --calibrate OUT.json --calibrate-set warm|streamed`): for each shape
(B, H_Q, H_KV, L_K), the microseconds per call of every launch the planner can
choose -- split count, packed tile width, V slices, and the merge of the chunk
states (a second launch, or inside the split launch).  This module fits the
constants to them and writes them to csrc/cost_model.inc, which plan.cpp
includes.  A CPU test refits the committed sweeps and checks that they give
the committed constants.

The model (the same arithmetic as model_time in csrc/plan.cpp, for a launch
of `wgs` workgroups of four waves over chunks of ceil(L_K / s) keys):

    compute = base + ceil(wgs / CUs) * (32-key tiles per wave) * t_tile * contig^[H_KV = 1] * vs_tile
    stream  = hbm0 + (K/V bytes + chunk-state bytes) / hbm_rate
    T = (compute^p + stream^p)^(1/p) + [s > 1] merge
    merge = merge0 + merge1 s                                  (second launch)
          | fused0 + fused1 s hpt / 8 + fused2 (ceil(s / n) - 1)  (in the split launch)

t_tile is t_tile_staged when every workgroup has a CU to itself.  Each term
has a 16-column and a 32-column (more than 16 heads per workgroup) value.
The merge inside the split launch is done by one workgroup per tile, which
loads the s x hpt chunk states in batches of n = 8 chunks (16-column tiles)
or 4 (32-column): its cost grows with the state bytes and with the batches.

Fit: least squares of log(model) - log(measured) over every launch within
1.6x of its shape's fastest (the launches a planner might pick), in the logs
of the parameters, from fixed starting values: deterministic for a given
sweep.  Policy MI355X (K/V resident, as in graph replays of one call) fits
every constant but contig (1) and hbm0 (0); policy STREAMED (every call
reads its cache from HBM) holds p at 4 and fits contig.  Both tie the 32-column tile time of
launches with several workgroups per CU to the 16-column one (TIED).
"""

from __future__ import annotations

import argparse
import json
import math
import os
from typing import Dict, List

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
HEADER = os.path.join(HERE, "csrc", "cost_model.inc")
SWEEPS = {"warm": os.path.join(ROOT, "profiles", "calibration_warm.json"),
          "streamed": os.path.join(ROOT, "profiles", "calibration_streamed.json")}
SCHEDULE_SWEEP = os.path.join(ROOT, "profiles", "calibration_schedule.json")

CUS = 256
HEAD_DIM = 128
ROW_BYTES = 2.0 * HEAD_DIM * 2.0          # K and V row of one KV head per key
STATE_BYTES = (HEAD_DIM + 2) * 4.0        # Otilde, m, l of one head and chunk
WINDOW = 1.6
SLICE_KV_BYTES = 16 << 20   # K/V bytes up to which the planner considers V slices (half the L2)

# name, 16-column / 32-column pair index (None: one value)
NAMES = ["base0", "base1", "tt0", "tt1", "ts0", "ts1", "merge0", "merge1_0", "merge1_1", "fused0", "fused1_0",
         "fused1_1", "fused2", "hbm_rate", "hbm0", "pnorm", "contig", "vs2", "vs4"]
HELD = {"warm": {"contig": 1.0, "hbm0": 0.0}, "streamed": {"pnorm": 4.0}}
# 32-column tiles with several workgroups per CU are rare among the fastest
# launches, so their tile time is tied to the 16-column one by the ratio the
# two widths show with K/V straight into LDS: tt1 = tt0 * ts1 / ts0.
TIED = ("tt1",)
START = {   # starting values of the fit
    "warm": dict(base0=2.841, base1=4.042, tt0=0.809, tt1=1.130, ts0=0.671, ts1=0.854, merge0=2.458, merge1_0=0.218,
                 merge1_1=0.253, fused0=1.5, fused1_0=0.1, fused1_1=0.12, fused2=0.5, hbm_rate=6.319e6, hbm0=0.05, pnorm=2.389,
                 contig=1.0, vs2=0.812, vs4=0.714),
    "streamed": dict(base0=2.095, base1=3.679, tt0=1.576, tt1=2.2, ts0=1.609, ts1=1.643, merge0=2.308,
                     merge1_0=0.235, merge1_1=0.254, fused0=1.5, fused1_0=0.1, fused1_1=0.12, fused2=0.5, hbm_rate=6.498e6,
                     hbm0=3.366, pnorm=4.0, contig=0.744, vs2=0.943, vs4=0.856),
}


def launch_grid(chunks, vs):
    return np.where(vs == 1, chunks, vs * 8 * ((chunks + 7) // 8))


def kv_fetch(grid, tiles_per_wave, cus=CUS):
    """2: K/V straight into LDS (one workgroup per CU); 1: through registers
    (several per CU, at least two tiles per wave); 0: K into the operand
    layout (one tile per wave)."""
    return np.where(grid <= cus, 2, np.where(tiles_per_wave >= 2, 1, 0))


def fused_batch(hpt):
    """Chunk states the merging workgroup loads at once (merge_tile's batch)."""
    return np.where(np.asarray(hpt) > 16, 4, 8)


def merge_cost(c: Dict[str, float], hpt, s, fused):
    """Microseconds the merge of s > 1 chunk states adds: a second launch
    (fused 0) or the last-arriving workgroup of each tile (fused 1)."""
    hpt, s, fused = (np.asarray(x, dtype=np.int64) for x in (hpt, s, fused))
    wide = hpt > 16
    n = fused_batch(hpt)
    f = c["fused0"] + np.where(wide, c["fused1_1"], c["fused1_0"]) * s * hpt / 8.0 + \
        c["fused2"] * ((s + n - 1) // n - 1)
    m = c["merge0"] + np.where(wide, c["merge1_1"], c["merge1_0"]) * s
    return np.where(s > 1, np.where(fused == 1, f, m), 0.0)


def model_time(c: Dict[str, float], B, H_Q, H_KV, L, hpt, s, vs, fused, cus=CUS):
    """Modelled microseconds per call (arrays broadcast)."""
    B, H_Q, H_KV, L, hpt, s, vs, fused = (np.asarray(x, dtype=np.int64) for x in (B, H_Q, H_KV, L, hpt, s, vs, fused))
    wide = hpt > 16
    tiles = B * H_Q // hpt
    wgs = launch_grid(tiles * s, vs)
    chunk = (L + s - 1) // s
    per_wave = (chunk + 3) // 4
    tpw = (per_wave + 31) // 32
    per_cu = (wgs + cus - 1) // cus
    staged = kv_fetch(wgs, tpw, cus) == 2
    tt = np.where(staged, np.where(wide, c["ts1"], c["ts0"]), np.where(wide, c["tt1"], c["tt0"]))
    tt = tt * np.where(H_KV == 1, c["contig"], 1.0) * np.where(vs == 4, c["vs4"], np.where(vs == 2, c["vs2"], 1.0))
    compute = np.where(wide, c["base1"], c["base0"]) + per_cu * tpw * tt
    nbytes = B * L * H_KV * ROW_BYTES + np.where(s > 1, 2.0 * s * B * H_Q * STATE_BYTES, 0.0)
    stream = c["hbm0"] + nbytes / c["hbm_rate"]
    p = c["pnorm"]
    t = (compute ** p + stream ** p) ** (1.0 / p)
    return t + merge_cost(c, hpt, s, fused)


def choosable(sh: dict) -> list:
    """A shape's timed launches that the planner can choose: V slices only
    up to SLICE_KV_BYTES of K/V."""
    kv = sh["B"] * sh["L"] * sh["H_KV"] * ROW_BYTES
    return [t for t in sh["launches"] if t[2] == 1 or kv <= SLICE_KV_BYTES]


def launches(sweep: dict) -> Dict[str, np.ndarray]:
    """The sweep's choosable launches as arrays, with each shape's fastest time."""
    cols = {k: [] for k in ("B", "H_Q", "H_KV", "L", "hpt", "s", "vs", "fused", "us", "best", "shape")}
    for i, sh in enumerate(sweep["shapes"]):
        best = min(t[4] for t in choosable(sh))
        for hpt, s, vs, fused, us in choosable(sh):
            for k, v in (("B", sh["B"]), ("H_Q", sh["H_Q"]), ("H_KV", sh["H_KV"]), ("L", sh["L"]), ("hpt", hpt),
                         ("s", s), ("vs", vs), ("fused", fused), ("us", us), ("best", best), ("shape", i)):
                cols[k].append(v)
    return {k: np.asarray(v, dtype=np.float64 if k in ("us", "best") else np.int64) for k, v in cols.items()}


def fit(sweep: dict, which: str) -> Dict[str, float]:
    """Constants of policy `which` ("warm" or "streamed") fitted to a sweep."""
    from scipy.optimize import least_squares
    d = launches(sweep)
    keep = d["us"] <= WINDOW * d["best"]
    d = {k: v[keep] for k, v in d.items()}
    free = [n for n in NAMES if n not in HELD[which] and n not in TIED]
    start = START[which]
    x0 = np.log([start[n] for n in free])

    def consts(x):
        c = dict(HELD[which])
        c.update({n: float(math.exp(v)) for n, v in zip(free, x)})
        c["tt1"] = c["tt0"] * c["ts1"] / c["ts0"]
        return c

    def resid(x):
        t = model_time(consts(x), d["B"], d["H_Q"], d["H_KV"], d["L"], d["hpt"], d["s"], d["vs"], d["fused"])
        return np.log(t) - np.log(d["us"])

    res = least_squares(resid, x0, method="trf", x_scale=1.0, xtol=1e-12, ftol=1e-12, gtol=1e-12, max_nfev=4000)
    return {n: float(f"{v:.6g}") for n, v in consts(res.x).items()}


def fit_error(sweep: dict, c: Dict[str, float]) -> Dict[str, float]:
    """RMS and worst relative error of the model over the fitted window."""
    d = launches(sweep)
    keep = d["us"] <= WINDOW * d["best"]
    t = model_time(c, *(d[k][keep] for k in ("B", "H_Q", "H_KV", "L", "hpt", "s", "vs", "fused")))
    r = np.log(t) - np.log(d["us"][keep])
    return {"launches": int(keep.sum()), "rms_log_error": float(np.sqrt(np.mean(r * r))),
            "worst_ratio": float(np.exp(np.max(np.abs(r))))}


def heads_per_tile(H_Q: int, H_KV: int, cap: int) -> int:
    g = H_Q // H_KV
    return g if g <= cap else max(h for h in range(1, cap + 1) if g % h == 0)


def plan_mi355x(c: Dict[str, float], B: int, H_Q: int, H_KV: int, L: int, cus: int = CUS, gain: float = 0.99,
                l2_bytes: float = SLICE_KV_BYTES, max_arrival_tiles: int = 4096, split_gain: float = None,
                split_counts=None):
    """The choice the planner makes with constants `c` for num_splits and
    pack_gqa left to it (the steps of plan() in csrc/plan.cpp): per packed
    tile width the split count with its best V slices, a split, V slices or
    the narrow width only when modelled `gain` faster.  `split_counts`: the
    counts above one to consider (default 2..64).  (hpt, s, vs, combine)."""
    g = H_Q // H_KV
    kv_bytes = B * L * H_KV * ROW_BYTES

    def fused(h, s):
        return s > 1 and B * H_Q // h <= max_arrival_tiles and merge_cost(c, h, s, 1) < merge_cost(c, h, s, 0)

    def t(h, s, vs):
        return float(model_time(c, B, H_Q, H_KV, L, h, s, vs, 1 if fused(h, s) else 0, cus))

    def best_vs(h, s, slices):
        one = t(h, s, 1)
        bv, bt = 1, one
        tiles = B * H_Q // h
        slices = slices and kv_bytes <= l2_bytes
        vs = 2
        while slices and vs <= 4 and (tiles * s if vs == 1 else vs * 8 * -(-(tiles * s) // 8)) <= cus:
            tv = t(h, s, vs)
            if tv < bt and tv < gain * one:
                bv, bt = vs, tv
            vs *= 2
        return bv, bt

    def splits(h, slices):
        if L <= 0:
            return 1
        _, one = best_vs(h, 1, slices)
        bs, bt = 1, one
        for s in (range(2, 65) if split_counts is None else split_counts):
            _, ts = best_vs(h, s, slices)
            if ts < bt:
                bs, bt = s, ts
        return bs if bt < (gain if split_gain is None else split_gain) * one else 1

    pack = 1 if g > 1 else 0
    wide = heads_per_tile(H_Q, H_KV, 32) if pack else 1
    narrow = heads_per_tile(H_Q, H_KV, 16) if pack else 1
    slices = lambda h: pack == 1 or h == g
    s_w = splits(wide, slices(wide))
    _, t_w = best_vs(wide, s_w, slices(wide))
    hpt, s = wide, s_w
    if narrow != wide:
        s_n = splits(narrow, slices(narrow))
        _, t_n = best_vs(narrow, s_n, slices(narrow))
        if t_n < gain * t_w:
            hpt, s = narrow, s_n
    vs, _ = best_vs(hpt, s, slices(hpt))
    return hpt, s, vs, 1 if fused(hpt, s) else 0


def regret(sweep: dict, plan) -> Dict[str, object]:
    """How the launch the planner picks fares on a sweep: plan(B, H_Q, H_KV,
    L_K) gives (heads per tile, s, V slices, combine); its measured time (a
    split count the sweep did not time takes the nearest timed one below)
    over the shape's fastest, and over one split as the paper launches it
    (the whole group in one workgroup, no V slices)."""
    rows = []
    for sh in sweep["shapes"]:
        t = {(h, s, v, c): us for h, s, v, c, us in choosable(sh)}
        hpt, s, vs, comb = plan(sh["B"], sh["H_Q"], sh["H_KV"], sh["L"])
        timed = [k for k in t if k[0] == hpt and k[2] == vs and k[3] == comb and k[1] <= s]
        key = max(timed, key=lambda k: k[1]) if timed else min(t, key=t.get)
        wide = max(k[0] for k in t)
        rows.append({"B": sh["B"], "H_Q": sh["H_Q"], "H_KV": sh["H_KV"], "L": sh["L"], "plan": [hpt, s, vs, comb],
                     "us": t[key], "timed": key[1] == s, "best": min(t.values()),
                     "best_launch": list(min(t, key=t.get)), "s1_paper": t[(wide, 1, 1, 0)]})
    r = [x["us"] / x["best"] for x in rows]
    p = [x["s1_paper"] / x["us"] for x in rows]
    return {"shapes": len(rows), "mean_vs_best": float(np.mean(r)), "worst_vs_best": float(np.max(r)),
            "within_5pct": int(sum(x <= 1.05 for x in r)), "worst_speedup_vs_s1_paper": float(np.min(p)),
            "untimed": int(sum(not x["timed"] for x in rows)), "rows": rows}


def timed_split_counts(sweep: dict) -> List[int]:
    """The split counts above one that a sweep timed."""
    return sorted({t[1] for sh in sweep["shapes"] for t in sh["launches"] if t[1] > 1})


def planner_regret(sweep: dict, c: Dict[str, float]) -> Dict[str, Dict[str, object]]:
    """regret() of the planner with constants c: over the split counts the
    sweep timed (every choice measured), and over 1..64 as the library plans."""
    counts = timed_split_counts(sweep)
    return {"timed": regret(sweep, lambda B, H, K, L: plan_mi355x(c, B, H, K, L, split_counts=counts)),
            "all": regret(sweep, lambda B, H, K, L: plan_mi355x(c, B, H, K, L))}


# ---------------------------------------------------------------- per-sequence schedule model
#
# The chunk length of a per-sequence schedule (da_make_schedule) comes from
# its own model (schedule_time in csrc/plan.cpp): sequences cut into
# ceil(T_b / c) chunks of 32-key tiles, workgroups dealt longest first to the
# CUs, and a wave step costing tau(A) = (t_tile^p + (A x 64 KiB / R)^p)^(1/p)
# while A CUs are still busy, plus the merge of the split sequences: a second
# launch, merge0 + merge1 max_s, or inside the split launch, fused0 + fused1
# max_s hpt / 8 + fused2 (batches - 1), as in the uniform model.  The
# scheduler takes the chunk length and merge the model puts fastest.  Its
# 16-column constants are fitted to a sweep of timed schedules, every chunk
# length with either merge (bench.py --schedule-sweep); the 32-column ones
# carry the warm uniform model's ratios between the two tile widths.

SCHED_NAMES = ["base", "t_tile", "t_staged", "hbm_rate", "pnorm", "tail", "merge0", "merge1", "fused0", "fused1",
               "fused2"]
# tail scales the summed steps, which t_tile and hbm_rate already scale: it
# is held at 1 (a free tail leaves the fit one degree of freedom with no
# information, along which it drifts).
SCHED_HELD = {"tail": 1.0}
SCHED_START = dict(base=3.19, t_tile=0.9375, t_staged=0.8113, hbm_rate=11.144e6, pnorm=1.194, tail=1.289,
                   merge0=2.703, merge1=0.2368, fused0=1.5, fused1=0.1, fused2=0.5)
MAX_SPLITS = 64


def seq_splits(T: int, c: int) -> int:
    return 1 if T <= 0 else min(MAX_SPLITS, -(-T // c))


def schedule_time(sc: Dict[str, float], warm: Dict[str, float], tiles_of, H_Q: int, hpt: int, c: int,
                  combine: int = 0, cus: int = CUS) -> float:
    """Modelled microseconds of a schedule with target chunk c tiles (the
    arithmetic of schedule_time in csrc/plan.cpp)."""
    wide = hpt > 16
    ratio = lambda k0, k1: warm[k1] / warm[k0] if wide else 1.0
    base = sc["base"] * ratio("base0", "base1")
    t_tile = sc["t_tile"] * ratio("tt0", "tt1")
    t_staged = sc["t_staged"] * ratio("ts0", "ts1")
    merge1 = sc["merge1"] * ratio("merge1_0", "merge1_1")
    fused1 = sc["fused1"] * ratio("fused1_0", "fused1_1")
    tps = H_Q // hpt
    t_max = max(tiles_of) if len(tiles_of) else 0
    q_max = max(c, -(-t_max // MAX_SPLITS))
    count = [0] * ((q_max + 1 + 3) // 4 + 1)
    items = state_rows = 0
    max_s = 1
    for T in tiles_of:
        s = seq_splits(T, c)
        q, big = T // s, T % s
        count[(q + 1 + 3) // 4] += big * tps
        count[(q + 3) // 4] += (s - big) * tps
        items += s * tps
        if s > 1:
            state_rows += s
            max_s = max(max_s, s)
    share = [0] * (cus + 1)
    every = nxt = 0
    for w in range(len(count) - 1, 0, -1):
        n = count[w]
        if not n:
            continue
        rem = n % cus
        every += (n // cus) * w
        if rem:
            share[nxt] += w
            if nxt + rem <= cus:
                share[nxt + rem] -= w
            else:
                share[cus] -= w
                share[0] += w
                share[nxt + rem - cus] -= w
        nxt = (nxt + n) % cus
    run = every
    for j in range(cus):
        run += share[j]
        share[j] = run
    max_w = next((w for w in range(len(count) - 1, 0, -1) if count[w]), 0)
    staged = items <= cus
    t1 = t_staged if staged else t_tile
    p = sc["pnorm"]
    step_bytes = 4.0 * 32 * 2 * HEAD_DIM * 2
    steps = 0.0
    prev = 0
    for k in range(cus):
        sh = share[cus - 1 - k]
        if sh <= prev:
            continue
        a = cus - k
        tau = (t1 ** p + (a * step_bytes / sc["hbm_rate"]) ** p) ** (1.0 / p)
        steps += (sh - prev) * tau
        prev = sh
    t = base + sc["tail"] * steps + 2.0 * state_rows * H_Q * STATE_BYTES / sc["hbm_rate"]
    if state_rows > 0:
        if combine:
            n = 4 if wide else 8
            t += sc["fused0"] + fused1 * max_s * hpt / 8.0 + sc["fused2"] * ((max_s + n - 1) // n - 1)
        else:
            t += sc["merge0"] + merge1 * max_s
    return t


def schedule_batches_by_name():
    """(set, name) -> (lengths, H_Q, H_KV) of the batches the schedule sweep times."""
    import sys
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    from workloads import schedule_batches
    return {(kind, name): (lens, H_Q, H_KV) for kind in ("fit", "check")
            for name, lens, H_Q, H_KV in schedule_batches(kind)}


def chunk_times(row: dict) -> Dict[tuple, float]:
    """(chunk, merge) -> microseconds of a sweep row: every timed chunk
    length with each merge it was timed with."""
    return {(int(c), int(k)): float(us) for c, by in row["chunk_us_by_combine"].items() for k, us in by.items()}


def schedule_points(sweep: dict, kinds=("fit",)):
    """(tiles_of, H_Q, hpt, c, combine, us, batch best) for every timed
    chunk length and merge of the sweep's batches of the given sets."""
    batches = schedule_batches_by_name()
    pts = []
    for r in sweep["rows"]:
        if r["set"] not in kinds:
            continue
        lens, H_Q, _ = batches[(r["set"], r["batch"])]
        tiles_of = [-(-L // 32) for L in lens]
        ct = chunk_times(r)
        best = min(ct.values())
        for (c, k), us in ct.items():
            pts.append((tiles_of, H_Q, int(r["chunk_hpt"][str(c)]), c, k, us, best))
    return pts


def fit_schedule(sweep: dict, warm: Dict[str, float]) -> Dict[str, float]:
    """Schedule-model constants fitted to the sweep's "fit" batches (log-error
    least squares over the launches within 1.6x of each batch's fastest)."""
    from scipy.optimize import least_squares
    pts = [p for p in schedule_points(sweep) if p[5] <= WINDOW * p[6]]
    free = [n for n in SCHED_NAMES if n not in SCHED_HELD]

    def consts(x):
        sc = dict(SCHED_HELD)
        sc.update({n: float(math.exp(v)) for n, v in zip(free, x)})
        return sc

    def resid(x):
        sc = consts(x)
        return np.array([math.log(schedule_time(sc, warm, t, H_Q, hpt, c, k)) - math.log(us)
                         for t, H_Q, hpt, c, k, us, _ in pts])

    x0 = np.log([SCHED_START[n] for n in free])
    res = least_squares(resid, x0, method="trf", xtol=1e-10, ftol=1e-10, gtol=1e-10, max_nfev=2000)
    return {n: float(f"{v:.6g}") for n, v in consts(res.x).items()}


def choose_chunk(sc: Dict[str, float], warm: Dict[str, float], lens, H_Q: int, hpt: int, cus: int = CUS,
                 max_arrival_tiles: int = 4096):
    """The chunk length and merge da_make_schedule picks for unequal lengths
    at head tile width hpt: the fastest modelled of the longest sequence cut
    into 1..64 pieces, each with either merge (inside the split launch only
    while the tiles have arrival counters); on a tie the longer chunk and the
    second launch.  (chunk, combine)."""
    tiles_of = [-(-L // 32) for L in lens]
    t_max = max(tiles_of)
    combs = (0, 1) if len(lens) * (H_Q // hpt) <= max_arrival_tiles else (0,)

    def best_of(cand):
        ts = [(schedule_time(sc, warm, tiles_of, H_Q, hpt, cand, k, cus), k) for k in combs]
        t, k = ts[0]
        for tk, kk in ts[1:]:
            if tk < t:
                t, k = tk, kk
        return t, k

    best, comb = best_of(t_max)
    c, prev = t_max, t_max
    for s in range(2, MAX_SPLITS + 1):
        cand = -(-t_max // s)
        if cand == prev:
            continue
        prev = cand
        t, k = best_of(cand)
        if t < best:
            best, c, comb = t, cand, k
    return c, comb


def schedule_regret(sweep: dict, sc: Dict[str, float], warm: Dict[str, float]) -> Dict[str, object]:
    """The modelled chunk and merge against the fastest timed launch, per
    batch (both sets), at the tile width the sweep timed.  A chunk the sweep
    did not time is read at the next longer timed one (with the same merge
    where that was timed)."""
    batches = schedule_batches_by_name()
    out = {}
    for kind in ("fit", "check"):
        r_all = []
        for r in sweep["rows"]:
            if r["set"] != kind:
                continue
            lens, H_Q, _ = batches[(kind, r["batch"])]
            ct = chunk_times(r)
            hpt = int(r["auto_hpt"])
            c, k = choose_chunk(sc, warm, lens, H_Q, hpt)
            timed = sorted({x for x, _ in ct if x >= c})
            cc = timed[0] if timed else max(x for x, _ in ct)
            got = ct.get((cc, k), ct.get((cc, 0)))
            r_all.append(got / min(ct.values()))
        out[kind] = {"batches": len(r_all), "mean": float(np.mean(r_all)), "worst": float(np.max(r_all))}
    return out


# ---------------------------------------------------------------- configuration-specific split table
#
# The configurations the sweeps timed are planned from what was measured on
# them rather than from the model: for each shape (B, H_Q, H_KV, L_K) the
# launch the planner may choose (choosable) that ran fastest, except that a
# launch with fewer chunks within TABLE_GAIN of it is preferred, as the model
# takes a split only when it pays at least 1%.  Policies TABLE and
# TABLE_STREAMED look a shape up by exact match and plan every other shape
# with the model.  A nearest-configuration lookup for shapes between the
# timed ones was measured on the sweeps themselves, each shape planned from
# its neighbours with that shape left out (table_holdout): it did worse than
# the model, so the table is used only where it was measured.

TABLE_GAIN = 1.01
TABLE_SPLIT = os.path.join(HERE, "csrc", "split_table.inc")


def table_pick(sh: dict):
    """The launch the table keeps for one timed shape: (hpt, s, vs, combine)."""
    t = {(h, s, v, c): us for h, s, v, c, us in choosable(sh)}
    best = min(t.values())
    near = [k for k, us in t.items() if us <= TABLE_GAIN * best]
    return min(near, key=lambda k: (k[1], t[k]))


def split_table(sweep: dict) -> List[tuple]:
    """(B, H_Q, H_KV, L_K, hpt, s, vs, combine) for every shape of a sweep,
    sorted by shape."""
    return sorted((sh["B"], sh["H_Q"], sh["H_KV"], sh["L"]) + tuple(table_pick(sh)) for sh in sweep["shapes"])


def table_holdout(sweep: dict, c: Dict[str, float]) -> Dict[str, object]:
    """Each timed shape planned from the nearest other timed shape with the
    same group size H_Q / H_KV (distance |log2 of the ratio of B x H_KV| +
    |log2 of the ratio of L_K|, each at most 1; else the model), against the
    model's own plan; times read from the shape's own launches as regret()
    reads them."""
    shapes = sweep["shapes"]
    picks = [table_pick(sh) for sh in shapes]
    model = {(r["B"], r["H_Q"], r["H_KV"], r["L"]): r for r in regret(sweep, lambda B, H, K, L: plan_mi355x(c, B, H, K, L))["rows"]}
    out_t, out_m, fallback = [], [], 0
    for i, sh in enumerate(shapes):
        t = {(h, s, v, cc): us for h, s, v, cc, us in choosable(sh)}
        best = min(t.values())
        g = sh["H_Q"] // sh["H_KV"]
        near = None
        for j, o in enumerate(shapes):
            if j == i or o["H_Q"] // o["H_KV"] != g:
                continue
            db = abs(math.log2(sh["B"] * sh["H_KV"] / (o["B"] * o["H_KV"])))
            dl = abs(math.log2(sh["L"] / o["L"]))
            if db <= 1 and dl <= 1 and (near is None or (db + dl, db) < near[0]):
                near = ((db + dl, db), picks[j])
        m = model[(sh["B"], sh["H_Q"], sh["H_KV"], sh["L"])]["us"] / best
        out_m.append(m)
        got = None
        if near is not None:
            h, s, v, cc = near[1]
            same = [k for k in t if k[0] == h and k[2] == v and k[3] == cc and k[1] <= s]
            if same:
                got = t[max(same, key=lambda k: k[1])] / best
        if got is None:
            fallback += 1
            got = m
        out_t.append(got)
    st = lambda r: {"mean_vs_best": float(np.mean(r)), "worst_vs_best": float(np.max(r)),
                    "within_5pct": int(sum(x <= 1.05 for x in r))}
    return {"shapes": len(shapes), "nearest": st(out_t), "model": st(out_m), "fallback": fallback}


def table_summary_line(sweep: dict, c: Dict[str, float], which: str) -> str:
    h = table_holdout(sweep, c)
    n, t, m = h["shapes"], h["nearest"], h["model"]
    differ = sum(tuple(e[4:]) != tuple(r["plan"]) for e, r in
                 zip(split_table(sweep), sorted(regret(sweep, lambda B, H, K, L: plan_mi355x(c, B, H, K, L))["rows"],
                                                key=lambda r: (r["B"], r["H_Q"], r["H_KV"], r["L"]))))
    return (f"* Split table (policy {'TABLE' if which == 'warm' else 'TABLE_STREAMED'}): one entry per shape, the "
            f"fastest launch measured there (fewer chunks preferred within {TABLE_GAIN - 1:.0%}); it differs from the "
            f"model's choice on {differ} of {n} shapes. Planned from the nearest other swept shape instead (each shape "
            f"left out in turn), a shape lands {t['mean_vs_best']:.4f}x its fastest on average, {t['worst_vs_best']:.3f}x "
            f"at worst, within 5% on {t['within_5pct']}, against {m['mean_vs_best']:.4f}x, {m['worst_vs_best']:.3f}x and "
            f"{m['within_5pct']} for the model: so the library looks the table up by exact shape only.")


def table_literal(rows: List[tuple]) -> str:
    return ", ".join("{" + ", ".join(str(int(x)) for x in r) + "}" for r in rows)


def table_text(tables: Dict[str, List[tuple]], cus: int) -> str:
    lines = ["// Configuration-specific split table: for every shape the calibration",
             "// sweeps timed, the launch that ran fastest there (a launch with fewer",
             "// chunks within 1% of it preferred), as {B, H_Q, H_KV, L_K, heads per tile,",
             "// num_splits, v_slices, combine}, sorted by shape; measured with",
             "// DA_SPLIT_TABLE_CUS compute units.  Generated by",
             "// `python -m paper_2604_00028_amd.calibrate --write` from the sweeps",
             "// profiles/calibration_{warm,streamed}.json; do not edit by hand.",
             f"#define DA_SPLIT_TABLE_CUS {cus}",
             f"#define DA_SPLIT_TABLE_WARM {{{table_literal(tables['warm'])}}}",
             f"#define DA_SPLIT_TABLE_STREAMED {{{table_literal(tables['streamed'])}}}"]
    return "\n".join(lines + [""])


def parse_table(text: str) -> Dict[str, List[tuple]]:
    """The entries of each table in a generated split_table.inc."""
    import re
    out = {}
    for which, macro in (("warm", "DA_SPLIT_TABLE_WARM"), ("streamed", "DA_SPLIT_TABLE_STREAMED")):
        m = re.search(rf"#define {macro} (.*)", text)
        out[which] = [tuple(int(x) for x in e.split(",")) for e in re.findall(r"\{([-0-9, ]+)\}", m.group(1))]
    m = re.search(r"#define DA_SPLIT_TABLE_CUS (\d+)", text)
    out["cus"] = int(m.group(1))
    return out


def tables_all() -> Dict[str, List[tuple]]:
    return {which: split_table(json.load(open(path))) for which, path in SWEEPS.items()}


def model_literal(c: Dict[str, float]) -> str:
    f = lambda n: repr(float(c[n]))
    return ("{{{b0}, {b1}}}, {{{tt0}, {tt1}}}, {{{ts0}, {ts1}}}, {m0}, {{{m10}, {m11}}}, {f0}, {{{f10}, {f11}}}, "
            "{f2}, {rate}, {hbm0}, {p}, {contig}, {{1.0, {vs2}, {vs4}}}").format(
        b0=f("base0"), b1=f("base1"), tt0=f("tt0"), tt1=f("tt1"), ts0=f("ts0"), ts1=f("ts1"), m0=f("merge0"),
        m10=f("merge1_0"), m11=f("merge1_1"), f0=f("fused0"), f10=f("fused1_0"), f11=f("fused1_1"), f2=f("fused2"),
        rate=f("hbm_rate"), hbm0=f("hbm0"), p=f("pnorm"), contig=f("contig"), vs2=f("vs2"), vs4=f("vs4"))


def schedule_literal(sc: Dict[str, float], warm: Dict[str, float]) -> str:
    r = lambda k0, k1: warm[k1] / warm[k0]
    f = lambda x: repr(float(f"{x:.6g}"))
    return ("{{{b0}, {b1}}}, {{{t0}, {t1}}}, {{{s0}, {s1}}}, {rate}, {p}, {tail}, {m0}, {{{m10}, {m11}}}, {f0}, "
            "{{{f10}, {f11}}}, {f2}").format(
        b0=f(sc["base"]), b1=f(sc["base"] * r("base0", "base1")), t0=f(sc["t_tile"]),
        t1=f(sc["t_tile"] * r("tt0", "tt1")), s0=f(sc["t_staged"]), s1=f(sc["t_staged"] * r("ts0", "ts1")),
        rate=f(sc["hbm_rate"]), p=f(sc["pnorm"]), tail=f(sc["tail"]), m0=f(sc["merge0"]), m10=f(sc["merge1"]),
        m11=f(sc["merge1"] * r("merge1_0", "merge1_1")), f0=f(sc["fused0"]), f10=f(sc["fused1"]),
        f11=f(sc["fused1"] * r("fused1_0", "fused1_1")), f2=f(sc["fused2"]))


def header_text(models: Dict[str, Dict[str, float]], schedule: Dict[str, float] = None) -> str:
    lines = ["// Cost-model constants of the split policies, in the order of the CostModel",
             "// fields: base, t_tile, t_tile_staged, merge0, merge1, fused0, fused1, fused2, hbm_rate,",
             "// hbm0, pnorm, contig_tile, vs_tile; and of the per-sequence schedule, in the",
             "// order of the ScheduleModel fields.  Generated by",
             "// `python -m paper_2604_00028_amd.calibrate --write` from the sweeps",
             "// profiles/calibration_{warm,streamed,schedule}.json; do not edit by hand.",
             f"#define DA_COST_MODEL_WARM {{{model_literal(models['warm'])}}}",
             f"#define DA_COST_MODEL_STREAMED {{{model_literal(models['streamed'])}}}"]
    if schedule is not None:
        lines.append(f"#define DA_SCHEDULE_MODEL {{{schedule_literal(schedule, models['warm'])}}}")
    return "\n".join(lines + [""])


def parse_header(text: str) -> Dict[str, List[float]]:
    """The numbers of each model in a generated header, in field order."""
    import re
    out = {}
    for which, macro in (("warm", "DA_COST_MODEL_WARM"), ("streamed", "DA_COST_MODEL_STREAMED"),
                         ("schedule", "DA_SCHEDULE_MODEL")):
        m = re.search(rf"#define {macro} (.*)", text)
        if m:
            out[which] = [float(x) for x in re.findall(r"[-+0-9.e]+", m.group(1))]
    return out


def fit_all() -> Dict[str, Dict[str, float]]:
    return {which: fit(json.load(open(path)), which) for which, path in SWEEPS.items()}


def fit_schedule_all(models: Dict[str, Dict[str, float]]) -> Dict[str, float]:
    return fit_schedule(json.load(open(SCHEDULE_SWEEP)), models["warm"])


SUMMARY = os.path.join(ROOT, "profiles", "calibration_summary.md")


def write_summary(models, sched) -> None:
    """profiles/calibration_summary.md: the fitted constants, how well the model
    fits each sweep, and how the planner's choice fares on it."""
    lines = ["# Cost-model calibration on MI355X", "",
             "Made by `python -m paper_2604_00028_amd.calibrate --write --summary` from the committed sweeps",
             "(`python3 bench.py --calibrate profiles/calibration_{warm,streamed}.json --calibrate-set "
             "{warm,streamed} --rounds 5`,",
             "`python3 bench.py --schedule-sweep profiles/calibration_schedule.json`), each launch checked against "
             "the oracle before it was timed.", ""]
    for which, c in models.items():
        sweep = json.load(open(SWEEPS[which]))
        err = fit_error(sweep, c)
        both = planner_regret(sweep, c)
        r, a = both["timed"], both["all"]
        lines += [f"## Policy {'MI355X (K/V resident between calls)' if which == 'warm' else 'STREAMED (K/V read from HBM on every call)'}", "",
                  f"* Sweep: {len(sweep['shapes'])} shapes, {sweep['validated']} launches timed and validated, "
                  f"{len(sweep['invalid'])} invalid.",
                  f"* Fit: {err['launches']} launches within {WINDOW}x of their shape's fastest; RMS log error "
                  f"{err['rms_log_error']:.3f}, worst {err['worst_ratio']:.3f}x.",
                  f"* The planner's choice among the split counts the sweep timed ({', '.join(map(str, timed_split_counts(sweep)))}; "
                  f"every choice measured): {r['mean_vs_best']:.4f}x the fastest timed launch on average, "
                  f"{r['worst_vs_best']:.3f}x at worst, within 5% on {r['within_5pct']} of {r['shapes']} shapes; "
                  f"against one split as the paper launches it, never below "
                  f"{r['worst_speedup_vs_s1_paper']:.3f}x its speed.",
                  f"* The planner over 1..64 as the library plans: {a['untimed']} of {a['shapes']} choices are split "
                  f"counts the sweep did not time (read at the nearest timed count below, which overstates them); "
                  f"{a['mean_vs_best']:.4f}x on average, {a['worst_vs_best']:.3f}x at worst, within 5% on "
                  f"{a['within_5pct']}. The regression matrix times the library's own choices.",
                  table_summary_line(sweep, c, which),
                  "", "| constant | value |", "|---|---|"]
        lines += [f"| {n} | {v:.6g} |" for n, v in sorted(c.items())]
        lines.append("")
    sw = json.load(open(SCHEDULE_SWEEP))
    reg = schedule_regret(sw, sched, models["warm"])
    lines += ["## Per-sequence schedule", "",
              f"* Sweep: {len(sw['rows'])} mixed-length batches, {sw.get('validated', 0)} launches validated, "
              f"{len(sw.get('invalid', []))} invalid.",
              f"* The modelled chunk and merge against the fastest of 12 timed chunk lengths, each timed with either "
              f"merge (a chunk the sweep did not time is read at the next longer timed one): fitted batches {reg['fit']['mean']:.4f}x on average, "
              f"{reg['fit']['worst']:.3f}x at worst; batches never fitted {reg['check']['mean']:.4f}x, "
              f"{reg['check']['worst']:.3f}x at worst.", "", "| constant | value |", "|---|---|"]
    lines += [f"| {n} | {v:.6g} |" for n, v in sorted(sched.items())]
    with open(SUMMARY, "w") as f:
        f.write("\n".join(lines) + "\n")
    print(f"wrote {SUMMARY}")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--write", action="store_true", help="regenerate csrc/cost_model.inc and csrc/split_table.inc")
    ap.add_argument("--summary", action="store_true", help="write profiles/calibration_summary.md")
    args = ap.parse_args()
    models = fit_all()
    for which, c in models.items():
        sweep = json.load(open(SWEEPS[which]))
        err = fit_error(sweep, c)
        both = planner_regret(sweep, c)
        print(which, json.dumps(c), json.dumps(err),
              json.dumps({k: {n: v for n, v in r.items() if n != "rows"} for k, r in both.items()}))
    sched = fit_schedule_all(models)
    print("schedule", json.dumps(sched),
          json.dumps(schedule_regret(json.load(open(SCHEDULE_SWEEP)), sched, models["warm"])))
    for which, c in models.items():
        print(which, "table held out", json.dumps(table_holdout(json.load(open(SWEEPS[which])), c)))
    if args.write:
        with open(HEADER, "w") as f:
            f.write(header_text(models, sched))
        print(f"wrote {HEADER}")
        cus = {json.load(open(path))["device_cus"] for path in SWEEPS.values()}
        assert len(cus) == 1, "sweeps taken with different CU counts"
        with open(TABLE_SPLIT, "w") as f:
            f.write(table_text(tables_all(), cus.pop()))
        print(f"wrote {TABLE_SPLIT}")
    if args.summary:
        write_summary(models, sched)


if __name__ == "__main__":
    main()
