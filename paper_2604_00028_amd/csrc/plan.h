// Host-side planning shared by the C-ABI entry points: error state, the split
// policy, the sequence partition and workspace sizing.  No HIP calls here.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <vector>

#include "decode_attn.h"

namespace da {

constexpr int kHeadDim = DA_HEAD_DIM;
constexpr int kMaxSplits = DA_MAX_SPLITS;
constexpr int kMaxHeadsPerTile = 32;   // two 16-column MFMA head tiles per workgroup
constexpr int kNarrowHeadsPerTile = 16; // one 16-column MFMA head tile per workgroup
constexpr int64_t kL2Bytes = 8ll << 22;  // MI355X: 4 MiB of L2 on each of 8 XCDs
// K/V bytes of a call up to which V slices are considered: half the L2.  The
// slices of a chunk re-read its keys from their XCD's L2, which holds only
// that XCD's share of the chunks; at 32 MiB (B=16, H_KV=4, L_K=1024) four
// slices measured 19% slower than the best split.
constexpr int64_t kSliceKvBytes = kL2Bytes / 2;

// Records a printf-style message for da_last_error() and returns `code`.
int fail(int code, const char* fmt, ...);
void clear_error();

// Query heads one workgroup serves.  Packed: the whole GQA group of a KV head
// when it fits in `cap` columns, else the largest divisor of the group <= cap.
// Unpacked: one.
int heads_per_tile(int H_Q, int H_KV, int pack_gqa, int cap = kMaxHeadsPerTile);

// Whether a plan or schedule may serve `hpt` heads per workgroup in packing
// mode `pack` (0: one head; 1: the whole group up to 32 heads, or tiles of
// at most 16; 2: the whole group up to 32 heads).
bool heads_per_tile_valid(int H_Q, int H_KV, int pack, int hpt);

// First key of chunk i when L keys are cut into s balanced chunks.
inline int64_t chunk_start(int64_t L, int s, int i) { return (L * i) / s; }

// Constants of the MI355X cost model (times in microseconds, rates in bytes
// per microsecond), fitted to measured sweeps of every launch the planner
// can choose over 120-132 shapes (B, H_Q, H_KV, L_K).  Exposed so tests can
// check the model's properties.
struct CostModel {
  double base[2];          // launch, first loads and epilogue (16-column / 32-column head tiles)
  double t_tile[2];        // one 32-key tile on one wave, K fetched into the operand layout
  double t_tile_staged[2]; // ... K and V fetched straight into LDS (at most one workgroup per CU)
  double merge0;           // second launch that combines the chunk states, fixed part (s > 1)
  double merge1[2];        // ... per chunk
  double fused0;           // single-launch merge by the last workgroup of a tile, fixed part (s > 1)
  double fused1[2];        // ... per chunk and 8 heads of the tile (the state bytes that workgroup loads)
  double fused2;           // ... per batch of chunks after the first (kFusedBatch chunks per batch)
  double hbm_rate;         // sustained HBM bytes per microsecond, whole chip
  double hbm0;             // fixed part of the streaming bound
  double pnorm;            // the two bounds combine as (compute^p + stream^p)^(1/p)
  double contig_tile;      // tile times scale by this when a key row holds one KV head (H_KV = 1)
  double vs_tile[3];       // tile times scale by this with 1, 2 or 4 V slices per chunk
};
const CostModel& mi355x_model();
// The same model for K/V streamed from HBM on every call (policy STREAMED).
const CostModel& mi355x_streamed_model();

// A split count above one is chosen only if modelled faster than one launch
// by this factor.
constexpr double kSplitGain = 0.99;

// Modelled time (us) of one call with s splits (policy MI355X); `fused`:
// the chunk states are merged inside the split launch (da_plan.combine 1)
// rather than by a second launch.
double model_time(const CostModel& m, int B, int H_Q, int H_KV, int L_K, int hpt, int s, int cus, int vs = 1,
                  bool fused = false);

// Chunk states the merging workgroup of a single-launch merge loads at once
// (16-column / 32-column head tiles): one batch is merged in registers, more
// are staged through LDS batch by batch.
constexpr int kFusedBatch[2] = {8, 4};

// Modelled time (us) the merge of s chunk states of tiles of `hpt` heads adds
// to a call: a second launch, or inside the split launch (`fused`).
double merge_time(const CostModel& m, int hpt, int s, bool fused);

// Whether a plan of s chunks per sequence over `tiles` tiles of `hpt` heads
// merges the chunk states inside the split launch (da_plan.combine).
bool fused_merge(const CostModel& m, int hpt, int s, int64_t tiles);

// Whether `pl` may serve each chunk with pl.v_slices workgroups (1, 2 or 4):
// more than one only with K/V straight into LDS, packed tiles of either
// width (pack_gqa 1; not the paper's packing) or unpacked where one head is
// the group.
bool v_slices_valid(int H_Q, int H_KV, const da_plan& pl);

// Workgroups launched for `chunks` (tile, chunk) pairs with vs V slices:
// with slices, whole groups of 8 chunks, so that a chunk's slices share an
// XCD (the padding workgroups return at once).
inline int64_t launch_grid(int64_t chunks, int vs) {
  return vs == 1 ? chunks : (int64_t)vs * 8 * ((chunks + 7) / 8);
}

// Waves per workgroup (da_plan.group_waves) for a launch of `grid`
// workgroups on `cus` CUs over chunks of `chunk` keys of rows holding H_KV
// heads, each key row read by `readers` workgroups, with vs V slices and
// merge `combine`: 2 or 4.
int group_waves(int64_t grid, int cus, int64_t chunk, int H_KV, int readers, int vs, int combine);

// Whether a launch of `grid` workgroups that group_waves gives four waves
// runs faster as two-wave workgroups held to one per CU (da_plan.wg_per_cu),
// in 2-4 rounds over the CUs.
bool round_waves(int64_t grid, int cus, int64_t chunk, int H_KV, int readers, int vs, int combine);

// A plan made inside an entry point whose sequence lengths are read on the
// device (cu_seqlens_k, paged seq_lens): the sequences may be far shorter
// than L_K_max, so a two-wave plan, which pays only where every workgroup
// streams a long chunk, becomes the four-wave launch of the same grid (with
// the fetch path and merge policy MI355X gives four waves, sharing CUs).
void four_waves(da_plan* pl, int L_K_max);

// Time factor of a two-wave launch against the four-wave one where the
// two-wave rule applies: the least gain measured at 1-4 splits (1.8-2.5%),
// rounded up to what the planner counts on when it gives up the in-launch
// merge for two waves.
constexpr double kTwoWaveGain = 0.97;

// Whether a plan's wave count fits the rest of it: 4, or 2 with K/V through
// registers (kv_fetch 0 or 1), one V slice and no in-launch merge.
inline bool group_waves_valid(const da_plan& pl) {
  return pl.group_waves == 4 || (pl.group_waves == 2 && pl.kv_fetch != 2 && pl.v_slices == 1 && pl.combine == 0);
}

// How K/V tiles reach the matrix cores for a launch of `grid` workgroups on
// `cus` CUs whose waves walk up to `tiles_per_wave` 32-key tiles
// (da_plan.kv_fetch); kLoneFetch is the mode used when every workgroup has a
// CU to itself.
constexpr int kLoneFetch = 2;
int kv_fetch(int64_t grid, int cus, int64_t tiles_per_wave);

// Whether a launch reading `key_rows` key rows of one KV head (K and V,
// 512 bytes each), each row read by `readers` workgroups (the head tiles of
// one group), marks its K/V loads nontemporal (da_plan.kv_nontemporal): only
// when they exceed DA_RESIDENT_BYTES and one workgroup reads each row.
int kv_nontemporal(double key_rows, int readers);

// One entry of the configuration-specific split table (policies TABLE and
// TABLE_STREAMED): the launch measured fastest on one shape of a calibration
// sweep.
struct TableEntry {
  int32_t B, H_Q, H_KV, L_K;           // the shape
  int32_t hpt, s, vs, combine;         // heads per tile, num_splits, v_slices, combine
};
// The entry for exactly (B, H_Q, H_KV, L_K) in the resident (streamed =
// false) or streamed table, or nullptr.
const TableEntry* table_entry(bool streamed, int B, int H_Q, int H_KV, int L_K);

int plan(int B, int H_Q, int H_KV, int L_K_max, int d, int num_splits, int pack_gqa, int num_cus,
         int cu_margin, int policy, da_plan* out);

// Argument checks shared by the launch entry points (no HIP calls).
int check_shape(int B, int H_Q, int H_KV, int L_K_max, int d);

// Per-sequence schedule (da_make_schedule).  Split count of a sequence of T
// 32-key tiles for a target chunk of c tiles.
inline int seq_splits(int64_t T, int64_t c) {
  if (T <= 0) return 1;
  const int64_t s = (T + c - 1) / c;
  return s > kMaxSplits ? kMaxSplits : (int)s;
}

// Cost model of a per-sequence schedule (times in microseconds).  Chunks of
// unequal length make the tail of the launch matter, so the model follows
// the CUs one by one: each CU's share of the work, how many CUs are still
// busy as the shares run out, and the HBM rate they divide.
struct ScheduleModel {
  double base[2];           // fixed part (16-column / 32-column head tiles)
  double t_tile[2];         // one wave step (four 32-key tiles per workgroup), CU-bound
  double t_tile_staged[2];  // ... with K and V fetched straight into LDS
  double hbm_rate;          // bytes per microsecond the busy CUs divide
  double pnorm;             // a step costs (t_tile^p + (busy CUs x 64 KiB / hbm_rate)^p)^(1/p)
  double tail;              // scale of the summed steps
  double merge0;            // combine launch, fixed part (some sequence split)
  double merge1[2];         // ... per chunk of the most-split sequence
  double fused0;            // merge inside the split launch, fixed part (some sequence split)
  double fused1[2];         // ... per chunk of the most-split sequence and 8 heads of a tile
  double fused2;            // ... per batch of kFusedBatch chunks after the first
};
const ScheduleModel& mi355x_schedule_model();

// The merge term of a schedule whose most-split sequence has max_s chunks:
// a second launch (combine 0) or inside the split launch (combine 1).
double schedule_merge_time(const ScheduleModel& m, int hpt, int max_s, int combine);

// Cost of one wave step while `busy` CUs stream (index busy = 1..cus), for
// K through registers (direct) and straight into LDS (staged).
struct StepCost {
  std::vector<double> direct, staged;
  StepCost(const ScheduleModel& m, int wide, int cus);
};

// Modelled time (us) of a schedule with target chunk c tiles whose split
// sequences are merged as `combine` says; `tiles_of` holds the 32-key tile
// count of each sequence.
double schedule_time(const ScheduleModel& m, const StepCost& step, const int64_t* tiles_of, int B, int H_Q,
                     int hpt, int64_t c, int cus, int combine);

int make_schedule(const int32_t* seq_lens, int B, int H_Q, int H_KV, int L_K_max, int d, int pack_gqa,
                  int num_cus, int cu_margin, int chunk_tiles, void* meta, size_t meta_bytes, da_schedule* out);

// Workspace regions (256-byte aligned): chunk states Otilde | m | l from
// offset 0 (`states` ends them), and the arrival counters of single-launch
// merges in the last DA_ARRIVAL_BYTES of the caller's buffer, wherever its
// end is.  Chunk states of any shape stop before that region, so calls of
// different shapes can share one buffer without writing into the counters.
struct WorkspaceLayout {
  size_t o_off, m_off, l_off, states, total;
};
WorkspaceLayout workspace_layout(int B, int H_Q, int d, int s);
constexpr int kArrivalStride = DA_ARRIVAL_STRIDE / 4;  // uint32 words between two tiles' counters
constexpr int64_t kMaxArrivalTiles = DA_ARRIVAL_BYTES / DA_ARRIVAL_STRIDE;  // tiles a single-launch merge can count

// Offset of the arrival counters in a workspace of `bytes` bytes.
inline size_t arrival_offset(size_t bytes) { return (bytes - DA_ARRIVAL_BYTES) & ~(size_t)255; }

}  // namespace da
