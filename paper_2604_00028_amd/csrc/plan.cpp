// Host-side planning: split policy (paper Section 4 and the MI355X cost
// model), the sequence partition, workspace sizing and error reporting.
#include "plan.h"

#include <limits.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <vector>

namespace da {

namespace {
thread_local char g_last_error[512] = "";
}

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

void clear_error() { g_last_error[0] = '\0'; }

int heads_per_tile(int H_Q, int H_KV, int pack_gqa, int cap) {
  if (!pack_gqa) return 1;
  const int g = H_Q / H_KV;
  if (g <= cap) return g;
  for (int h = cap; h > 1; --h)
    if (g % h == 0) return h;
  return 1;
}

bool heads_per_tile_valid(int H_Q, int H_KV, int pack, int hpt) {
  if (pack < 0 || pack > 2) return false;
  const int wide = heads_per_tile(H_Q, H_KV, pack);
  return hpt == wide || (pack == 1 && hpt == heads_per_tile(H_Q, H_KV, pack, kNarrowHeadsPerTile));
}

// The constants of both policies are fitted by paper_2604_00028_amd/calibrate.py
// (log-error least squares over the launches within 1.6x of each shape's
// fastest) to measured sweeps of every launch the planner can choose, and
// generated into cost_model.inc.
#include "cost_model.inc"

// Policy MI355X: K/V resident between calls, as in graph replays of one call.
const CostModel& mi355x_model() {
  static const CostModel m = DA_COST_MODEL_WARM;
  return m;
}

// Time of one call with s chunks per sequence, each shared by vs workgroups
// (V slices):
//   compute = base + (workgroups per CU) x (32-key tiles per wave) x t_tile x vs_tile[vs]
//   stream  = hbm0 + (K/V bytes + chunk-state traffic) / hbm_rate
//   T = (compute^p + stream^p)^(1/p) + merge_time
// Every workgroup has four waves, one per SIMD, and walks a quarter of its
// chunk each; workgroups that share a CU share its SIMDs.  The soft maximum
// reflects that a CU's tile loop slows as the chip nears its HBM rate.  The
// two-wave launch (group_waves) is a measured rule applied after the model
// has chosen; the model prices the four-wave launch.
double model_time(const CostModel& m, int B, int H_Q, int H_KV, int L_K, int hpt, int s, int cus, int vs,
                  bool fused) {
  const int wide = hpt > 16 ? 1 : 0;
  const double row_bytes = 2.0 * kHeadDim * 2.0;  // K and V row of one KV head
  const int64_t tiles = (int64_t)B * H_Q / hpt;
  const int64_t wgs = launch_grid(tiles * s, vs);
  const int64_t chunk = ((int64_t)L_K + s - 1) / s;
  const int64_t per_wave = (chunk + 3) / 4;
  const int64_t tiles_per_wave = (per_wave + 31) / 32;
  const int64_t per_cu = (wgs + cus - 1) / cus;
  const double tt = (kv_fetch(wgs, cus, tiles_per_wave) == kLoneFetch ? m.t_tile_staged[wide] : m.t_tile[wide]) *
                    (H_KV == 1 ? m.contig_tile : 1.0) * m.vs_tile[vs == 4 ? 2 : vs - 1];
  const double compute = m.base[wide] + (double)per_cu * (double)tiles_per_wave * tt;
  double bytes = (double)B * L_K * H_KV * row_bytes;
  if (s > 1) bytes += 2.0 * s * (double)B * H_Q * (kHeadDim + 2) * 4.0;
  const double stream = m.hbm0 + bytes / m.hbm_rate;
  double t = pow(pow(compute, m.pnorm) + pow(stream, m.pnorm), 1.0 / m.pnorm);
  return t + merge_time(m, hpt, s, fused);
}

// The merge of s > 1 chunk states: a second launch, merge0 + merge1 s; or
// inside the split launch, where one workgroup per tile loads the s x hpt
// chunk states in batches of kFusedBatch chunks: fused0 + fused1 s hpt / 8 +
// fused2 (batches - 1).
double merge_time(const CostModel& m, int hpt, int s, bool fused) {
  if (s <= 1) return 0.0;
  const int wide = hpt > 16 ? 1 : 0;
  if (!fused) return m.merge0 + m.merge1[wide] * s;
  const int n = kFusedBatch[wide];
  return m.fused0 + m.fused1[wide] * s * (hpt / 8.0) + m.fused2 * ((s + n - 1) / n - 1);
}

// The same model with K/V streamed from HBM on every call (each call reads
// its own copy of the cache, as a decode step that runs every layer evicts
// each layer's cache before it is read again), fitted to launches that read
// their own copy of the cache on every call (at least 1 GiB per timed
// replay).  Streaming from HBM, a tile of one KV head costs less when key
// rows hold just that head (H_KV = 1: contiguous rows) than when they
// interleave several heads and every workgroup reads a 256-byte slice of
// each row: contig_tile.
const CostModel& mi355x_streamed_model() {
  static const CostModel m = DA_COST_MODEL_STREAMED;
  return m;
}

// The configuration-specific split tables (generated beside the model
// constants from the same sweeps), sorted by shape.
#include "split_table.inc"

namespace {
const TableEntry kTableWarm[] = DA_SPLIT_TABLE_WARM;
const TableEntry kTableStreamed[] = DA_SPLIT_TABLE_STREAMED;

bool shape_less(const TableEntry& a, const TableEntry& b) {
  if (a.B != b.B) return a.B < b.B;
  if (a.H_Q != b.H_Q) return a.H_Q < b.H_Q;
  if (a.H_KV != b.H_KV) return a.H_KV < b.H_KV;
  return a.L_K < b.L_K;
}
}  // namespace

const TableEntry* table_entry(bool streamed, int B, int H_Q, int H_KV, int L_K) {
  const TableEntry* first = streamed ? kTableStreamed : kTableWarm;
  const TableEntry* last =
      first + (streamed ? sizeof(kTableStreamed) / sizeof(kTableStreamed[0]) : sizeof(kTableWarm) / sizeof(kTableWarm[0]));
  const TableEntry key = {B, H_Q, H_KV, L_K, 0, 0, 0, 0};
  const TableEntry* e = std::lower_bound(first, last, key, shape_less);
  return e != last && !shape_less(key, *e) ? e : nullptr;
}

// Whether s > 1 chunk states are merged inside the split launch by the last
// workgroup of each tile (da_plan.combine 1) rather than by a second launch:
// whichever merge the model prices lower.
bool fused_merge(const CostModel& m, int hpt, int s, int64_t tiles) {
  return s > 1 && tiles <= kMaxArrivalTiles && merge_time(m, hpt, s, true) < merge_time(m, hpt, s, false);
}

// V slices for s chunks per sequence when `slices` allows them: 2 or 4
// where the launch keeps one workgroup per CU, the call's K/V fit in L2 (so
// that the slices' repeated K reads stay there; the slice factors were
// measured on such calls) and the model puts them at least 1% ahead of one
// slice; *t gets the modelled time.
static int best_vslices(const CostModel& m, int B, int H_Q, int H_KV, int L_K, int hpt, int s, int cus, bool slices,
                        double* t) {
  const int64_t tiles = (int64_t)B * H_Q / hpt;
  const bool fused = fused_merge(m, hpt, s, tiles);
  const double one = model_time(m, B, H_Q, H_KV, L_K, hpt, s, cus, 1, fused);
  int best_vs = 1;
  double best = one;
  slices = slices && (double)B * L_K * H_KV * (2.0 * kHeadDim * 2.0) <= (double)kSliceKvBytes;
  for (int vs = 2; slices && vs <= 4 && launch_grid(tiles * s, vs) <= cus; vs *= 2) {
    const double tv = model_time(m, B, H_Q, H_KV, L_K, hpt, s, cus, vs, fused);
    if (tv < best && tv < kSplitGain * one) {
      best = tv;
      best_vs = vs;
    }
  }
  *t = best;
  return best_vs;
}

static int mi355x_splits(const CostModel& m, int B, int H_Q, int H_KV, int L_K, int hpt, int cus,
                         bool slices = false) {
  if (L_K <= 0) return 1;
  // Fastest modelled split count (each with its best V slices); the
  // smallest one on an exact tie.  A split must be modelled at least 1%
  // faster than one launch: closer than that the model cannot tell them
  // apart, and a second launch that brings nothing is the one outcome the
  // policy must avoid (never slower than one split).
  double one = 0.0;
  best_vslices(m, B, H_Q, H_KV, L_K, hpt, 1, cus, slices, &one);
  int best_s = 1;
  double best = one;
  for (int s = 2; s <= kMaxSplits; ++s) {
    double ts = 0.0;
    best_vslices(m, B, H_Q, H_KV, L_K, hpt, s, cus, slices, &ts);
    if (ts < best) {
      best = ts;
      best_s = s;
    }
  }
  return best < kSplitGain * one ? best_s : 1;
}

// The paper's rule (Section 4): 128-key blocks, Batch * H_KV tiles.
static int paper_splits(int B, int H_KV, int L_K, int H_Q, int hpt, int cus) {
  const int blocks = (L_K + 127) / 128;
  const int64_t tiles = (int64_t)B * H_KV;
  if (blocks <= 3) return 1;                 // short contexts stay unsplit
  if (blocks == 4) return tiles >= 4 ? 1 : 3;  // saturated vs low-tile boundary bucket
  // Longer contexts: the paper defers to the stack's own long-context path,
  // which here is the MI355X cost model.
  return mi355x_splits(mi355x_model(), B, H_Q, H_KV, L_K, hpt, cus);
}

int group_waves(int64_t grid, int cus, int64_t chunk, int H_KV, int readers, int vs, int combine) {
  // Four wave64s, one per SIMD, by default.  Where the launch puts one
  // workgroup on at least three quarters of the CUs and two on at most a
  // quarter of them, every key row is read by one workgroup and the chunks
  // hold at least 512 keys, two waves, each walking half the chunk (every
  // other 32-key tile of it where key rows hold at most 4 KV heads) with one
  // tile in flight through registers, read HBM faster than four waves with
  // two direct-to-LDS stages each: the chip then keeps about a quarter of
  // the loads in flight (8 instead of 32 MiB), and HBM serves the smaller
  // set of streams closer to its peak.  Measured on MI355X in one process
  // per comparison: 1 GiB of K/V at one split 1.8-6.2% faster (B=32,
  // H_Q=64, H_KV=8, L_K=8192: 157.9 -> 151.7 us), 1.9-8.3% at 128-512 MiB,
  // 4.2% and 7.4% with 192 and 224 of 256 CUs busy, 2.5-8.4% at 2-4 splits
  // merged by a second launch; neutral at 512 keys per chunk; slower below
  // that (0.84-0.91x at 128-256 keys), with 160 or 128 of 256 CUs busy
  // (0.98x, 0.95x) and where two workgroups share each key (16-head tiles
  // of a 32-head group: 0.91x).  Past one workgroup per CU (against four
  // waves fetching through LDS): 264-320 workgroups on 256 CUs 0.5-3%
  // faster with 8 KV heads and 3-9% with one, 384-512 within 1% with 8 KV
  // heads (0.97-1.0x with one), 576 slower (1.02-1.03x).  Pure MQA (key
  // rows of one head, whose two waves take alternate tiles) keeps the gain
  // further: at 384-768 workgroups with chunks of 1024-8192 keys 0.94-1.0x
  // (2.6% on average over 21 shapes), at 800-1024 with chunks of 2048-8192
  // keys 0.92-1.04x (2.2% on average over 31 shapes), while at 512-key
  // chunks (0.997-1.026x) and past four workgroups per CU (1.0-1.09x at
  // 1152-1536) it is no longer steady.  The
  // in-launch merge is sized for four waves, so two-wave plans merge by a
  // second launch.  Eight waves (two per SIMD, with K staged) measured
  // slower at chunks of a few hundred keys.
  const int64_t top = H_KV == 1 && chunk >= 2048   ? 4 * (int64_t)cus
                      : H_KV == 1 && chunk >= 1024 ? 3 * (int64_t)cus
                                                   : 5 * (int64_t)cus / 4;
  return vs == 1 && readers == 1 && combine == 0 && grid <= top && 4 * grid >= 3 * (int64_t)cus && chunk >= 512
             ? 2
             : 4;
}

bool round_waves(int64_t grid, int cus, int64_t chunk, int H_KV, int readers, int vs, int combine) {
  // Past the two-wave range of group_waves a four-wave launch keeps two or
  // more workgroups on each CU, 16-32 MiB of loads in flight.  Two-wave
  // workgroups held to one per CU keep 8 MiB in flight and run the grid in
  // rounds; each round start costs a ramp, so the rounds must be few, full
  // and long.  Measured on MI355X against the four-wave launch, in one
  // process per comparison (2 KV heads and more): 480-512 workgroups
  // (two rounds) 0.966-1.0x, 768 (three) 0.966-0.99x, 1024 (four) over
  // chunks of 4096-8192 keys 0.967-0.987x but 1.009-1.014x over 2048, and
  // 1.02-1.04x at 576 (a quarter-full third round).  Pure MQA keeps its own
  // two-wave range (group_waves), which shares CUs.
  if (vs != 1 || readers != 1 || combine != 0 || H_KV < 2 || 4 * grid <= 5 * (int64_t)cus) return false;
  const int64_t rounds = (grid + cus - 1) / cus;
  return rounds >= 2 && rounds <= 4 && 8 * (rounds * cus - grid) <= cus && chunk >= (rounds == 4 ? 4096 : 2048);
}

int kv_fetch(int64_t grid, int cus, int64_t tiles_per_wave) {
  // A workgroup with a CU to itself streams fastest with K and V loaded
  // straight into LDS, two tiles in flight per wave (144 KB of LDS).  When
  // CUs hold several workgroups, two of them per CU hide each other's
  // latency: K and V go row-contiguous through registers into LDS (72 KB).
  // On uniform and mixed-length launches of 128 to 2048 workgroups with at
  // least two tiles per wave that was 1-5% faster than K fetched straight
  // into the operand layout.  With a single tile per wave the per-workgroup
  // overheads dominate and the smaller footprint of the operand-layout fetch
  // (36 KB, three workgroups per CU) wins by up to 30%.
  if (grid <= cus) return kLoneFetch;
  return tiles_per_wave >= 2 ? 1 : 0;
}

void four_waves(da_plan* pl, int L_K_max) {
  if (pl->group_waves != 2) return;
  const int64_t chunk = ((int64_t)L_K_max + pl->num_splits - 1) / pl->num_splits;
  pl->group_waves = 4;
  pl->wg_per_cu = 0;
  pl->kv_fetch = kv_fetch(pl->grid, pl->num_cus, ((chunk + 3) / 4 + 31) / 32);
  // and the merge a four-wave plan takes (these entry points plan with policy MI355X)
  if (pl->num_splits > 1)
    pl->combine = fused_merge(mi355x_model(), pl->heads_per_tile, pl->num_splits, pl->tiles) ? 1 : 0;
}

bool v_slices_valid(int H_Q, int H_KV, const da_plan& pl) {
  if (pl.v_slices == 1) return true;
  // direct-to-LDS launches only; not the paper's packing, and unpacked only
  // where one head is the whole group
  return (pl.v_slices == 2 || pl.v_slices == 4) && pl.kv_fetch == kLoneFetch &&
         (pl.pack_gqa == 1 || (pl.pack_gqa == 0 && H_Q == H_KV));
}

int kv_nontemporal(double key_rows, int readers) {
  // Measured on MI355X (1 GiB of K/V at high load: 185 -> 160 us with the
  // hint; 537 MB: 103 -> 88 us).  Below the MALL's capacity the hint costs
  // what residency between calls saves (268 MB: 46 -> 48 us; 134 MB with 64
  // workgroups: 26.2 -> 26.8 us; 16-64 MB: up to 40%), so it is off there.
  // When several workgroups read the same keys (head tiles narrower than
  // the group), the later ones find them in L2 only without the hint.
  return readers == 1 && key_rows * (2.0 * kHeadDim * 2.0) > (double)DA_RESIDENT_BYTES ? 1 : 0;
}

int check_shape(int B, int H_Q, int H_KV, int L_K_max, int d) {
  if (d != kHeadDim) return fail(DA_ERR_UNSUPPORTED, "head dim %d unsupported (only %d)", d, kHeadDim);
  if (B <= 0 || H_Q <= 0 || H_KV <= 0)
    return fail(DA_ERR_SHAPE, "B=%d H_Q=%d H_KV=%d must be positive", B, H_Q, H_KV);
  if (H_Q % H_KV != 0) return fail(DA_ERR_SHAPE, "H_Q=%d is not a multiple of H_KV=%d", H_Q, H_KV);
  if (L_K_max < 0) return fail(DA_ERR_SHAPE, "L_K_max=%d is negative", L_K_max);
  // Per-sequence K/V byte offsets must fit the 32-bit buffer offsets the
  // kernels use; B*H_Q rows must fit a 32-bit grid.
  const int64_t seq_bytes = (int64_t)L_K_max * H_KV * kHeadDim * 2;
  if (seq_bytes >= ((int64_t)1 << 31))
    return fail(DA_ERR_SHAPE, "one sequence spans %lld bytes of K (limit 2 GiB)", (long long)seq_bytes);
  if ((int64_t)B * H_Q > (1 << 24)) return fail(DA_ERR_SHAPE, "B*H_Q=%lld too large", (long long)B * H_Q);
  return DA_OK;
}

int plan(int B, int H_Q, int H_KV, int L_K_max, int d, int num_splits, int pack_gqa, int num_cus,
         int cu_margin, int policy, da_plan* out) {
  if (!out) return fail(DA_ERR_NULL, "plan output is NULL");
  int rc = check_shape(B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  if (num_splits > kMaxSplits) return fail(DA_ERR_SPLITS, "num_splits=%d exceeds %d", num_splits, kMaxSplits);
  if (pack_gqa < -1 || pack_gqa > 2) return fail(DA_ERR_ARG, "pack_gqa=%d not in {-1,0,1,2}", pack_gqa);
  if (policy < DA_POLICY_MI355X || policy > DA_POLICY_TABLE_STREAMED)
    return fail(DA_ERR_ARG, "unknown policy %d", policy);
  if (num_cus <= 0) return fail(DA_ERR_ARG, "num_cus=%d must be positive here", num_cus);
  if (cu_margin < 0 || cu_margin >= num_cus)
    return fail(DA_ERR_ARG, "cu_margin=%d must be in [0, %d)", cu_margin, num_cus);
  const int cus = num_cus - cu_margin;
  const int g = H_Q / H_KV;
  const int pack = pack_gqa >= 0 ? pack_gqa : (g > 1 ? 1 : 0);
  int hpt = heads_per_tile(H_Q, H_KV, pack);
  // Chunk states are addressed with 32-bit byte offsets: a split launch
  // keeps them below 2 GiB.  A forced split count beyond that is refused; a
  // chosen one is capped (where it could bind, the chip is full anyway).
  const int64_t split_bytes = (int64_t)B * H_Q * kHeadDim * 4;
  const int max_s = (int)std::min<int64_t>(kMaxSplits, std::max<int64_t>(1, (((int64_t)1 << 31) - 1) / split_bytes));
  if (num_splits > 1 && num_splits > max_s)
    return fail(DA_ERR_SHAPE, "num_splits=%d: %lld bytes of chunk state exceed 2 GiB", num_splits,
                (long long)num_splits * split_bytes);
  const bool streamed = policy == DA_POLICY_STREAMED || policy == DA_POLICY_TABLE_STREAMED;
  int s = num_splits;
  int vs = 1, comb = 0;
  bool from_table = false;
  if (policy == DA_POLICY_TABLE || policy == DA_POLICY_TABLE_STREAMED) {
    // A shape the calibration sweep timed, on as many CUs as it had, with
    // the split count and tile width left to the policy, takes the launch
    // measured fastest there; any other goes to the cost model.
    const TableEntry* e = num_splits <= 0 && pack == (g > 1 ? 1 : 0) && cus == DA_SPLIT_TABLE_CUS
                              ? table_entry(streamed, B, H_Q, H_KV, L_K_max)
                              : nullptr;
    if (e) {
      const int64_t tiles = (int64_t)B * H_Q / e->hpt;
      da_plan t = {};
      t.pack_gqa = pack;
      t.v_slices = e->vs;
      t.kv_fetch = launch_grid(tiles * e->s, e->vs) <= cus ? kLoneFetch : 0;
      const bool ok = heads_per_tile_valid(H_Q, H_KV, pack, e->hpt) && e->s >= 1 && e->s <= max_s &&
                      (e->vs == 1 || e->vs == 2 || e->vs == 4) && v_slices_valid(H_Q, H_KV, t) &&
                      (e->combine == 0 || (e->combine == 1 && e->s > 1 && tiles <= kMaxArrivalTiles));
      if (!ok) e = nullptr;
    }
    if (e) {
      hpt = e->hpt;
      s = e->s;
      vs = e->vs;
      comb = e->combine;
      from_table = true;
    }
    policy = streamed ? DA_POLICY_STREAMED : DA_POLICY_MI355X;
  }
  if (from_table) {
    // planned above
  } else if (policy == DA_POLICY_PAPER || policy == DA_POLICY_EVOLVED) {
    if (s <= 0 && policy == DA_POLICY_PAPER)
      s = paper_splits(B, H_KV, L_K_max, H_Q, hpt, cus);
    else if (s <= 0 && B == 1)
      s = L_K_max < 256 ? 16 : 12;  // Fig. 1: the evolved single-batch setting
    else if (s <= 0)
      s = mi355x_splits(mi355x_model(), B, H_Q, H_KV, L_K_max, hpt, cus);
  } else {
    // With pack_gqa = 1 the model also picks the width of a packed tile when
    // the group is wider than one 16-column MFMA tile: all of it (up to 32
    // heads) in one workgroup, or 16-head tiles whose workgroups read the
    // same keys.  The narrow tile is cheaper per workgroup and doubles the
    // workgroups, which pays while CUs are idle; the wide one reads each key
    // once per group.  Narrow is taken only when modelled at least 1% faster.
    // V slices (the output dims of a chunk split over 2 or 4 workgroups that
    // share its scores) are considered for packed tiles of either width, not
    // with the paper's packing (pack_gqa 2), and unpacked only where one head
    // is the group.
    const CostModel& m = policy == DA_POLICY_STREAMED ? mi355x_streamed_model() : mi355x_model();
    auto best = [&](int h, double* t) {
      const bool slices = pack == 1 || (pack == 0 && h == g);
      const int sh = s > 0 ? s : mi355x_splits(m, B, H_Q, H_KV, L_K_max, h, cus, slices);
      best_vslices(m, B, H_Q, H_KV, L_K_max, h, sh, cus, slices, t);
      return sh;
    };
    double t_wide = 0.0, t_narrow = 0.0;
    const int s_wide = best(hpt, &t_wide);
    const int narrow = pack == 1 ? heads_per_tile(H_Q, H_KV, pack, kNarrowHeadsPerTile) : hpt;
    const int s_narrow = narrow != hpt ? best(narrow, &t_narrow) : s_wide;
    if (narrow != hpt && t_narrow < kSplitGain * t_wide) {
      hpt = narrow;
      s = s_narrow;
    } else {
      s = s_wide;
    }
  }
  if (!from_table) {
    s = std::min(s, max_s);
    const CostModel& m = streamed ? mi355x_streamed_model() : mi355x_model();
    if (policy == DA_POLICY_MI355X || policy == DA_POLICY_STREAMED) {
      double t = 0.0;
      vs = best_vslices(m, B, H_Q, H_KV, L_K_max, hpt, s, cus, pack == 1 || (pack == 0 && hpt == g), &t);
    }
    comb = fused_merge(m, hpt, s, (int64_t)B * H_Q / hpt) ? 1 : 0;
  }
  out->num_splits = s;
  out->combine = comb;
  out->pack_gqa = pack;
  out->heads_per_tile = hpt;
  out->tiles = (int32_t)((int64_t)B * H_Q / hpt);
  out->v_slices = vs;
  out->grid = (int32_t)launch_grid((int64_t)out->tiles * s, vs);
  out->num_cus = cus;
  // STREAMED plans for K/V that are not resident whatever their size.  The
  // V slices of a chunk all read its keys, as the head tiles of a group do.
  const int readers = (g / hpt) * vs;
  {
    const int64_t chunk = ((int64_t)L_K_max + s - 1) / s;
    int waves = group_waves(out->grid, cus, chunk, H_KV, readers, vs, comb);
    bool rounds = waves == 4 && round_waves(out->grid, cus, chunk, H_KV, readers, vs, comb);
    const bool two_c0 = group_waves(out->grid, cus, chunk, H_KV, readers, vs, 0) == 2;
    const bool rounds_c0 = !two_c0 && round_waves(out->grid, cus, chunk, H_KV, readers, vs, 0);
    if (waves == 4 && !rounds && comb == 1 && !from_table && (two_c0 || rounds_c0)) {
      // Two waves (sharing CUs, or held to one workgroup per CU in rounds)
      // merge by a second launch.  They take it where the share of
      // the split launch they save (kTwoWaveGain) is modelled to outweigh
      // what the second launch adds over the merge inside the launch:
      // measured at 1 GiB, 2 splits 84.3 -> 83.3 us and at 256 MiB, 4 splits
      // 43.7 -> 43.1 us, while 4 splits at 128 MiB stayed faster merged in
      // the launch (22.8 against 23.6 us).  Table plans keep the merge
      // their sweep measured.
      const CostModel& m = streamed ? mi355x_streamed_model() : mi355x_model();
      const double t_in = model_time(m, B, H_Q, H_KV, L_K_max, hpt, s, cus, vs, true);
      const double t_two = model_time(m, B, H_Q, H_KV, L_K_max, hpt, s, cus, vs, false);
      if (kTwoWaveGain * t_two < t_in) {
        comb = 0;
        out->combine = 0;
        waves = 2;
        rounds = rounds_c0;
      }
    }
    if (rounds) waves = 2;
    out->group_waves = waves;
    out->wg_per_cu = rounds ? 1 : 0;
    // two waves: K through registers, straight into the operand layout
    // where key rows hold one KV head and each CU holds one workgroup
    // (contiguous 256-byte rows, measured 1-3% faster there) and through LDS
    // otherwise (with one KV head on 300 workgroups: 5% faster)
    out->kv_fetch = out->group_waves == 2 ? (H_KV == 1 && out->grid <= cus ? 0 : 1)
                                          : kv_fetch(out->grid, cus, ((chunk + 3) / 4 + 31) / 32);
  }
  out->kv_nontemporal = streamed ? (readers == 1 ? 1 : 0) : kv_nontemporal((double)B * L_K_max * H_KV, readers);
  return DA_OK;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Constants fitted by paper_2604_00028_amd/calibrate.py (log-error least
// squares over chunk lengths within 1.6x of each batch's fastest) to timed
// schedules of mixed-length batches (bench.py --schedule-sweep: 18 batches of
// 2 to 128 sequences of 32 to 65536 keys at 12 chunk lengths each), and
// generated into cost_model.inc.  tail is held at 1 (t_tile and hbm_rate
// already scale the summed steps).  The 32-column values carry the uniform
// model's ratios between the two tile widths.
const ScheduleModel& mi355x_schedule_model() {
  static const ScheduleModel m = DA_SCHEDULE_MODEL;
  return m;
}

StepCost::StepCost(const ScheduleModel& m, int wide, int cus) : direct((size_t)cus + 1), staged((size_t)cus + 1) {
  const double step_bytes = 4.0 * 32 * 2 * kHeadDim * 2;
  for (int a = 1; a <= cus; ++a) {
    const double stream = pow((double)a * step_bytes / m.hbm_rate, m.pnorm);
    direct[a] = pow(pow(m.t_tile[wide], m.pnorm) + stream, 1.0 / m.pnorm);
    staged[a] = pow(pow(m.t_tile_staged[wide], m.pnorm) + stream, 1.0 / m.pnorm);
  }
}

// Sequence b becomes s_b chunks of q or q + 1 tiles, each walked by four
// waves (ceil(tiles / 4) steps) in every head tile.  Workgroups are issued
// longest first and dealt to the CUs in turn; a CU's share is the sum of
// its workgroups' steps.  Shares run out in increasing order, and while A
// CUs are busy a step costs tau(A) = (t^p + (A x 64 KiB / rate)^p)^(1/p).
double schedule_time(const ScheduleModel& m, const StepCost& step, const int64_t* tiles_of, int B, int H_Q,
                     int hpt, int64_t c, int cus, int combine) {
  const int wide = hpt > 16 ? 1 : 0;
  const int64_t tps = H_Q / hpt;
  // Workgroups per step count: sequence b gives `big` chunks of q + 1 tiles
  // and s_b - big of q, each walked in ceil(tiles / 4) steps.
  int64_t t_max = 0;
  for (int b = 0; b < B; ++b) t_max = tiles_of[b] > t_max ? tiles_of[b] : t_max;
  const int64_t q_max = c > (t_max + kMaxSplits - 1) / kMaxSplits ? c : (t_max + kMaxSplits - 1) / kMaxSplits;
  std::vector<int64_t> count((size_t)((q_max + 1 + 3) / 4 + 1), 0);
  int64_t items = 0, state_rows = 0;
  int max_s = 1;
  for (int b = 0; b < B; ++b) {
    const int64_t T = tiles_of[b];
    const int s = seq_splits(T, c);
    const int64_t q = T / s, big = T % s;
    count[(q + 1 + 3) / 4] += big * tps;
    count[(q + 3) / 4] += (s - big) * tps;
    items += s * tps;
    if (s > 1) {
      state_rows += s;
      if (s > max_s) max_s = s;
    }
  }
  // Dealt longest first, in turn: CU j takes workgroups j, j + cus, ... of
  // the sorted list, so shares never grow with j.  A group of n workgroups
  // of w steps adds (n / cus) * w to every CU and w to the next n % cus
  // (a circular window, kept as a difference array).
  std::vector<int64_t> share((size_t)cus + 1, 0);
  int64_t every = 0, next = 0;
  for (int64_t w = (int64_t)count.size() - 1; w >= 1; --w) {
    const int64_t n = count[w];
    if (!n) continue;
    const int64_t rem = n % cus;
    every += (n / cus) * w;
    if (rem) {
      share[next] += w;
      if (next + rem <= cus) {
        share[next + rem] -= w;
      } else {
        share[cus] -= w;
        share[0] += w;
        share[next + rem - cus] -= w;
      }
    }
    next = (next + n) % cus;
  }
  int64_t run = every;
  for (int j = 0; j < cus; ++j) {
    run += share[j];
    share[j] = run;
  }
  // Shares run out from the smallest (CU cus-1) up; while `busy` CUs still
  // stream, a step costs tau[busy].
  int64_t max_w = 0;
  for (int64_t w = (int64_t)count.size() - 1; w >= 1 && !max_w; --w)
    if (count[w]) max_w = w;
  const std::vector<double>& tau = kv_fetch(items, cus, max_w) == kLoneFetch ? step.staged : step.direct;
  double steps = 0.0;
  int64_t prev = 0;
  for (int k = 0; k < cus; ++k) {
    const int64_t sh = share[cus - 1 - k];
    if (sh <= prev) continue;
    steps += (double)(sh - prev) * tau[cus - k];
    prev = sh;
  }
  double t = m.base[wide] + m.tail * steps + 2.0 * (double)state_rows * H_Q * (kHeadDim + 2) * 4.0 / m.hbm_rate;
  if (state_rows > 0) t += schedule_merge_time(m, hpt, max_s, combine);
  return t;
}

double schedule_merge_time(const ScheduleModel& m, int hpt, int max_s, int combine) {
  const int wide = hpt > 16 ? 1 : 0;
  if (!combine) return m.merge0 + m.merge1[wide] * max_s;
  const int n = kFusedBatch[wide];
  return m.fused0 + m.fused1[wide] * max_s * (hpt / 8.0) + m.fused2 * ((max_s + n - 1) / n - 1);
}

namespace {
struct Item {
  int32_t tile, t0, t1, row;
};
}  // namespace

int make_schedule(const int32_t* seq_lens, int B, int H_Q, int H_KV, int L_K_max, int d, int pack_gqa,
                  int num_cus, int cu_margin, int chunk_tiles, void* meta, size_t meta_bytes, da_schedule* out) {
  if (!out) return fail(DA_ERR_NULL, "schedule output is NULL");
  if (!seq_lens) return fail(DA_ERR_NULL, "seq_lens is NULL");
  int rc = check_shape(B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  if (pack_gqa < -1 || pack_gqa > 2) return fail(DA_ERR_ARG, "pack_gqa=%d not in {-1,0,1,2}", pack_gqa);
  if (num_cus <= 0) return fail(DA_ERR_ARG, "num_cus=%d must be positive here", num_cus);
  if (cu_margin < 0 || cu_margin >= num_cus)
    return fail(DA_ERR_ARG, "cu_margin=%d must be in [0, %d)", cu_margin, num_cus);
  for (int b = 0; b < B; ++b)
    if (seq_lens[b] < 0 || seq_lens[b] > L_K_max)
      return fail(DA_ERR_SHAPE, "seq_lens[%d]=%d outside [0, L_K_max=%d]", b, seq_lens[b], L_K_max);
  const int cus = num_cus - cu_margin;
  const int g = H_Q / H_KV;
  const int pack = pack_gqa >= 0 ? pack_gqa : (g > 1 ? 1 : 0);

  std::vector<int64_t> T(B);
  int64_t t_max = 0;
  for (int b = 0; b < B; ++b) {
    T[b] = (seq_lens[b] + 31) / 32;
    if (T[b] > t_max) t_max = T[b];
  }
  bool equal = true;
  for (int b = 1; b < B; ++b) equal = equal && seq_lens[b] == seq_lens[0];
  // Chunk length (in tiles) for head tiles of h heads, the merge of the
  // split sequences (*comb), and the modelled time.  Equal lengths take the
  // uniform plan's split count and merge.  Otherwise the candidates are the
  // longest sequence cut into 1..64 pieces, each with either merge (inside
  // the split launch only while the tiles have arrival counters); the
  // fastest modelled one wins, on a tie the longer chunk and the second
  // launch.
  auto choose_chunk = [&](int h, double* t, int* comb) -> int64_t {
    const ScheduleModel& m = mi355x_schedule_model();
    const StepCost step(m, h > 16 ? 1 : 0, cus);
    const int max_comb = (int64_t)B * (H_Q / h) <= kMaxArrivalTiles ? 1 : 0;
    auto best_of = [&](int64_t cand, int* cb) {
      double bt = schedule_time(m, step, T.data(), B, H_Q, h, cand, cus, 0);
      *cb = 0;
      for (int k = 1; k <= max_comb; ++k) {
        const double tk = schedule_time(m, step, T.data(), B, H_Q, h, cand, cus, k);
        if (tk < bt) {
          bt = tk;
          *cb = k;
        }
      }
      return bt;
    };
    if (chunk_tiles > 0) {
      *t = best_of(chunk_tiles, comb);
      return chunk_tiles;
    }
    if (equal) {
      const CostModel& u = mi355x_model();
      const int s = t_max > 0 ? mi355x_splits(u, B, H_Q, H_KV, seq_lens[0], h, cus) : 1;
      *comb = fused_merge(u, h, s, (int64_t)B * (H_Q / h)) ? 1 : 0;
      *t = model_time(u, B, H_Q, H_KV, seq_lens[0], h, s, cus, 1, *comb == 1);
      return t_max > 0 ? (t_max + s - 1) / s : 1;
    }
    int64_t c = t_max;
    double best = best_of(c, comb);
    int64_t prev = c;
    for (int s = 2; s <= kMaxSplits; ++s) {
      const int64_t cand = (t_max + s - 1) / s;
      if (cand == prev) continue;
      prev = cand;
      int cb = 0;
      const double ts = best_of(cand, &cb);
      if (ts < best) {
        best = ts;
        c = cand;
        *comb = cb;
      }
    }
    *t = best;
    return c;
  };
  // Packed groups wider than 16 heads: one wide tile or 16-head tiles, as in
  // the uniform plan (narrow only when modelled at least 1% faster).
  int hpt = heads_per_tile(H_Q, H_KV, pack);
  double t_wide = 0.0, t_narrow = 0.0;
  int comb = 0, comb_narrow = 0;
  int64_t c = choose_chunk(hpt, &t_wide, &comb);
  const int narrow = pack == 1 ? heads_per_tile(H_Q, H_KV, pack, kNarrowHeadsPerTile) : hpt;
  if (narrow != hpt) {
    const int64_t c_narrow = choose_chunk(narrow, &t_narrow, &comb_narrow);
    if (t_narrow < kSplitGain * t_wide) {
      hpt = narrow;
      c = c_narrow;
      comb = comb_narrow;
    }
  }
  const int tps = H_Q / hpt;

  // Items and per-sequence rows.
  std::vector<int32_t> split(B), row0(B);
  int64_t n_items = 0, rows = 0;
  int max_s = 1;
  for (int b = 0; b < B; ++b) {
    split[b] = seq_splits(T[b], c);
    row0[b] = split[b] > 1 ? (int32_t)rows : -1;
    if (split[b] > 1) rows += split[b];
    if (split[b] > max_s) max_s = split[b];
    n_items += (int64_t)split[b] * tps;
  }
  const size_t seq_off = (size_t)n_items * 16;
  const size_t need = seq_off + (size_t)B * 8;
  if ((int64_t)rows * H_Q * kHeadDim * 4 >= ((int64_t)1 << 31) || need >= ((size_t)1 << 31))
    return fail(DA_ERR_SHAPE, "schedule of %lld workgroups and %lld state rows is too large", (long long)n_items,
                (long long)rows);
  out->B = B;
  out->H_Q = H_Q;
  out->H_KV = H_KV;
  out->L_K_max = L_K_max;
  out->pack_gqa = pack;
  out->heads_per_tile = hpt;
  out->tiles = B * tps;
  out->num_items = (int32_t)n_items;
  out->chunk_tiles = (int32_t)c;
  out->max_splits = max_s;
  out->state_rows = (int32_t)rows;
  out->num_cus = cus;
  {
    int64_t max_chunk = 0;  // tiles of the longest chunk
    for (int b = 0; b < B; ++b) max_chunk = std::max<int64_t>(max_chunk, (T[b] + split[b] - 1) / split[b]);
    out->kv_fetch = kv_fetch(n_items, cus, (max_chunk + 3) / 4);
  }
  out->seq_offset = (int32_t)seq_off;
  out->meta_bytes = (int32_t)need;
  out->combine = rows > 0 ? comb : 0;
  {
    double key_rows = 0.0;
    for (int b = 0; b < B; ++b) key_rows += (double)seq_lens[b] * H_KV;
    out->kv_nontemporal = kv_nontemporal(key_rows, g / hpt);
  }
  if (!meta) return fail(DA_ERR_NULL, "meta is NULL");
  if (meta_bytes < need)
    return fail(DA_ERR_WORKSPACE, "schedule needs %zu metadata bytes, got %zu", need, meta_bytes);

  // G head tiles read each KV head (G = 1 when a tile holds the whole
  // group).  Items are listed sequence, KV head, chunk, then those G tiles,
  // so the G workgroups that read the same keys are neighbours.
  const int G = g / hpt;
  std::vector<Item> items;
  items.reserve((size_t)n_items);
  for (int b = 0; b < B; ++b) {
    const int s = split[b];
    for (int kv = 0; kv < H_KV; ++kv)
      for (int i = 0; i < s; ++i)
        for (int m = 0; m < G; ++m) {
          Item it;
          it.tile = b * tps + kv * G + m;
          it.t0 = (int32_t)(T[b] * i / s);
          it.t1 = (int32_t)(T[b] * (i + 1) / s);
          it.row = s > 1 ? row0[b] + i : -1;
          items.push_back(it);
        }
  }
  // Longest chunks first, so that the tail of the launch holds short ones
  // (stable: neighbours that read the same keys stay neighbours).
  std::stable_sort(items.begin(), items.end(),
                   [](const Item& a, const Item& b) { return a.t1 - a.t0 > b.t1 - b.t0; });
  // The last chunk of a sequence runs to the end of the sequence as the
  // device sees it, so a length that grew after scheduling is still read.
  for (Item& it : items) {
    const int b = it.tile / tps;
    if (it.t1 == T[b]) it.t1 = INT32_MAX;
  }
  int32_t* w = static_cast<int32_t*>(meta);
  const int64_t n = n_items;
  // Workgroup i starts on XCD i % 8.  With G > 1, each block of 8G items is
  // transposed so that the G readers of one KV head and chunk take slots
  // j, j + 8, ..., j + 8(G-1) of the block: one XCD, one L2.  A last partial
  // block keeps list order.
  const int64_t blk = 8 * (int64_t)G;
  for (int64_t pos = 0; pos < n; ++pos) {
    int64_t bid = pos;
    if (G > 1 && pos < n - n % blk) {
      const int64_t base = pos - pos % blk, r = pos % blk;
      bid = base + (r % G) * 8 + r / G;
    }
    w[4 * bid + 0] = items[pos].tile;
    w[4 * bid + 1] = items[pos].t0;
    w[4 * bid + 2] = items[pos].t1;
    w[4 * bid + 3] = items[pos].row;
  }
  int32_t* sq = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(meta) + seq_off);
  for (int b = 0; b < B; ++b) {
    sq[2 * b] = row0[b];
    sq[2 * b + 1] = split[b];
  }
  return DA_OK;
}

WorkspaceLayout workspace_layout(int B, int H_Q, int d, int s) {
  WorkspaceLayout w{};
  const size_t rows = (size_t)B * H_Q;
  w.o_off = 0;
  w.m_off = align256(w.o_off + (size_t)s * rows * d * sizeof(float));
  w.l_off = align256(w.m_off + (size_t)s * rows * sizeof(float));
  w.states = align256(w.l_off + (size_t)s * rows * sizeof(float));
  w.total = w.states + DA_ARRIVAL_BYTES;
  return w;
}

}  // namespace da

extern "C" {

int da_choose_splits(int B, int H_Q, int H_KV, int L_K_max, int d, int num_cus, int cu_margin,
                     int policy, da_plan* out) {
  if (num_cus <= 0) {
    int is950 = 0;
    int rc = da_device_info(&num_cus, &is950);
    if (rc) return rc;
  }
  return da::plan(B, H_Q, H_KV, L_K_max, d, 0, -1, num_cus, cu_margin, policy, out);
}

int da_make_plan(int B, int H_Q, int H_KV, int L_K_max, int d, int num_splits, int pack_gqa,
                 int num_cus, int cu_margin, int policy, da_plan* out) {
  if (num_cus <= 0) {
    int is950 = 0;
    int rc = da_device_info(&num_cus, &is950);
    if (rc) return rc;
  }
  return da::plan(B, H_Q, H_KV, L_K_max, d, num_splits, pack_gqa, num_cus, cu_margin, policy, out);
}

double da_model_time(int policy, int B, int H_Q, int H_KV, int L_K, int heads_per_tile, int num_splits,
                     int v_slices, int combine, int num_cus) {
  if (B <= 0 || H_Q <= 0 || H_KV <= 0 || H_Q % H_KV != 0 || L_K < 0 || heads_per_tile <= 0 ||
      H_Q % heads_per_tile != 0 || num_splits < 1 || num_splits > da::kMaxSplits ||
      (v_slices != 1 && v_slices != 2 && v_slices != 4) || combine < 0 || combine > 1 || num_cus <= 0)
    return -1.0;
  const da::CostModel& m = policy == DA_POLICY_STREAMED || policy == DA_POLICY_TABLE_STREAMED
                               ? da::mi355x_streamed_model()
                               : da::mi355x_model();
  return da::model_time(m, B, H_Q, H_KV, L_K, heads_per_tile, num_splits, num_cus, v_slices, combine == 1);
}

size_t da_schedule_max_bytes(int B, int H_Q, int H_KV, int pack_gqa) {
  if (B <= 0 || H_Q <= 0 || H_KV <= 0 || H_Q % H_KV != 0) return 0;
  const int g = H_Q / H_KV;
  const int pack = pack_gqa >= 0 ? pack_gqa : (g > 1 ? 1 : 0);
  // the narrowest head tile the scheduler may choose
  const int64_t tps = H_Q / da::heads_per_tile(H_Q, H_KV, pack, da::kNarrowHeadsPerTile);
  return (size_t)B * tps * da::kMaxSplits * 16 + (size_t)B * 8;
}

int da_make_schedule(const int32_t* seq_lens, int B, int H_Q, int H_KV, int L_K_max, int d, int pack_gqa,
                     int num_cus, int cu_margin, int chunk_tiles, void* meta, size_t meta_bytes,
                     da_schedule* out) {
  da::clear_error();
  if (num_cus <= 0) {
    int is950 = 0;
    int rc = da_device_info(&num_cus, &is950);
    if (rc) return rc;
  }
  return da::make_schedule(seq_lens, B, H_Q, H_KV, L_K_max, d, pack_gqa, num_cus, cu_margin, chunk_tiles, meta,
                           meta_bytes, out);
}

size_t da_schedule_workspace_bytes(const da_schedule* s) {
  if (!s || s->state_rows <= 0 || s->H_Q <= 0) return 0;
  return da::workspace_layout(s->state_rows, s->H_Q, da::kHeadDim, 1).total;
}

size_t da_workspace_bytes(int B, int H_Q, int d, int num_splits) {
  if (B <= 0 || H_Q <= 0 || d <= 0 || num_splits <= 1) return 0;
  return da::workspace_layout(B, H_Q, d, num_splits).total;
}

int da_split_bounds(int L, int num_splits, int32_t* cuts) {
  if (!cuts) return da::fail(DA_ERR_NULL, "cuts is NULL");
  if (L < 0) return da::fail(DA_ERR_SHAPE, "L=%d is negative", L);
  if (num_splits <= 0 || num_splits > da::kMaxSplits)
    return da::fail(DA_ERR_SPLITS, "num_splits=%d not in [1, %d]", num_splits, da::kMaxSplits);
  for (int i = 0; i <= num_splits; ++i) cuts[i] = (int32_t)da::chunk_start(L, num_splits, i);
  return DA_OK;
}

const char* da_strerror(int code) {
  switch (code) {
    case DA_OK: return "ok";
    case DA_ERR_NULL: return "null pointer";
    case DA_ERR_SHAPE: return "invalid shape";
    case DA_ERR_UNSUPPORTED: return "unsupported head dim or device";
    case DA_ERR_SPLITS: return "num_splits out of range";
    case DA_ERR_ALIGN: return "misaligned pointer";
    case DA_ERR_WORKSPACE: return "workspace missing or too small";
    case DA_ERR_HIP: return "HIP runtime error";
    case DA_ERR_ARG: return "invalid argument";
    default: return "unknown error";
  }
}

const char* da_last_error(void) { return da::g_last_error; }

}  // extern "C"
