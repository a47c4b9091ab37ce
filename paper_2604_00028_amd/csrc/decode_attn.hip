// Split-KV single-query decode attention for MI355X (gfx950): the split
// partial kernel, the log-sum-exp combine kernel, and the C-ABI launch entry
// points.
//
// What one workgroup computes (paper Sections 2.1, 2.2, 3.1): for one work
// tile -- a sequence b and the query heads that share one KV head when GQA
// packing is on (Sections 3.1 and 4: Batch x H_KV tiles for L_Q = 1), or a
// single query head when it is off -- and one chunk of that sequence's keys,
// the partial softmax state (running max m, sum l, unnormalised output
// Otilde).  With one split the state is normalised and written as the
// output; with several, the chunk states go to the workspace and the combine
// kernel merges them in chunk order (the paper's final reduction, Sections
// 3.1 and 5.3).
//
// gfx950 mapping:
//  * W wave64s per workgroup: 4, one per SIMD, or 2 where about one
//    workgroup per CU (up to three for pure MQA) streams long chunks over
//    most of the chip (fewer loads in flight read HBM faster there).  The chunk is cut into W contiguous key
//    ranges, one per wave, or, with two waves over key rows of at most
//    1 KiB (H_KV <= 4), its 32-key tiles alternate between the waves; each
//    wave walks its tiles in key order, and the W wave states are merged
//    through LDS in one step, each wave producing 128 / W of the output
//    dims.
//  * Scores S^T[key, head] = K . Q^T on MFMA v_mfma_f32_16x16x32_bf16: keys
//    are the 16 rows, the packed query heads the 16 columns (two column
//    tiles when a KV head serves up to 32 query heads).  K reaches the
//    A-operand layout one of three ways (FETCH): loaded straight into it
//    (each lane reads 64 bytes of one key row), row-contiguous into
//    registers and then through LDS, or row-contiguous straight into LDS
//    (buffer loads with the LDS destination), two tiles in flight per wave.
//  * Online softmax on the MFMA result layout: every lane holds 8 scores of
//    one head column; the tile max and sum over the 4 row groups take two
//    v_permlane16/32_swap steps; exp2 on the hardware v_exp_f32 with the
//    scale folded as scale*log2(e); fp32 running state; the output is only
//    rescaled when some column's running max moved.
//  * Output O^T[dim, head] += V^T . P^T on the same MFMA: the P operand is
//    the lane's own 8 probabilities (bf16), so softmax never moves data
//    across lanes; V^T comes from a per-wave LDS tile of 32 keys (16-byte
//    coalesced loads, 288-byte row pitch, ds_read_b64_tr_b16 transposing
//    reads: two per 16 output dims).
//  * K/V loads are raw buffer loads whose record count ends at the wave's
//    last key: keys past it read as zeros without touching memory, so ragged
//    tails cost no traffic and no load needs a mask or a branch.
//  * With packing off, workgroup ids are remapped so consecutive tiles land
//    on the same XCD (dispatch is round-robin over the 8 XCDs): the query
//    heads of one KV head then share that XCD's L2.  With packing on, each
//    KV head is read by one workgroup, and the round-robin spread measured
//    up to 12% faster at large grids.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <type_traits>

#include "decode_attn.h"
#include "plan.h"

namespace {

constexpr int D = DA_HEAD_DIM;
constexpr int kKeysPerTile = 32;
constexpr int kVPitch = 288;                 // bytes per staged V row (256 + 32 pad)
constexpr int kKPitch = 288;                 // bytes per staged K row (256 + 32 pad)
constexpr int kDeviceScope = 16;             // cache-policy field: sc1, device-scope coherent access
constexpr int kStateVals = 2 + 32;           // one wave's state per lane: m, l, 8 x 4 outputs

// How a tile's K and V reach the matrix cores.
enum Fetch : int {
  kFetchDirect = 0,  // K straight into the MFMA operand layout; V via registers to LDS
  kFetchStaged = 1,  // K and V row-contiguous into registers, then through LDS
  kFetchLds = 2,     // K and V row-contiguous straight into LDS (buffer_load ... lds), two stages
};

// Direct-to-LDS tiles: an instruction writes 64 lanes x 16 bytes = 4 rows
// contiguously, so a 32-key tile is 8 such blocks.  Blocks sit kBlockStride
// bytes apart and within a block the 16-byte chunks of row r are rotated
// by 2r positions, which places every chunk on the LDS banks a 288-byte row
// pitch would (the pitch the register-staged path uses): the operand reads
// below then measure no bank conflicts.
constexpr int kBlockStride = 4 * 288;
constexpr int kLdsTileBytes = 8 * kBlockStride;                 // one K or V tile
constexpr int kLdsStageBytes = 2 * kLdsTileBytes;                // K and V of one tile

// LDS of one workgroup of W waves with NT head tiles: the per-wave stages,
// reused after the tile loop for the wave-state merge (W slots, one wave
// state of NT x kStateVals x 64 floats each).
constexpr int merge_slot_bytes(int NT) { return NT * kStateVals * 64 * 4; }  // V slices use less
constexpr int stage_bytes(int FETCH) {
  return FETCH == kFetchLds ? 2 * kLdsStageBytes
                            : kKeysPerTile * (kVPitch + (FETCH == kFetchStaged ? kKPitch : 0));
}
constexpr int smem_bytes(int W, int NT, int FETCH) {
  return W * stage_bytes(FETCH) > W * merge_slot_bytes(NT) ? W * stage_bytes(FETCH) : W * merge_slot_bytes(NT);
}
static_assert(smem_bytes(4, 2, kFetchLds) <= 160 * 1024, "a workgroup must fit the LDS of one CU");
static_assert(smem_bytes(4, 1, kFetchDirect) >= (2 * (DA_MAX_SPLITS + 16) * 32 + 8 * 32) * 4,
              "the single-launch merge stages chunk maxima and sums in LDS");

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

// kDirect: one chunk per sequence, the normalised output is written.
// kPartials: chunk states go to the workspace for a separate combine launch.
// kFused: chunk states go to the workspace with device-scope stores, and
// the last workgroup of a tile to finish merges them (single launch).
enum Mode : int { kDirect = 0, kPartials = 1, kFused = 2 };

// Division by a launch constant d >= 1 as a multiply and a shift
// (Granlund and Montgomery, PLDI 1994, Theorem 4.2 with N = 32): with
// l = ceil(log2 d) and m = ceil(2^(32+l) / d) - 2^32, x / d = (x +
// mulhi(x, m)) >> l for every x < 2^32; for x < 2^31, the only numerators
// here, the sum does not overflow.  The host computes (m, l) once per launch.
struct Div {
  uint32_t m, l;
};

Div make_div(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  return Div{(uint32_t)((((1ull << (32 + l)) + d - 1) / d) - (1ull << 32)), l};
}

__device__ __forceinline__ int div_by(int x, Div d) {
  return (int)(((uint32_t)x + __umulhi((uint32_t)x, d.m)) >> d.l);
}

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* cu;    // nullable: fixed layout
  uint16_t* out;        // bf16 [B, H_Q, D]        (kDirect)
  float* lse;           // nullable, [B, H_Q]      (kDirect)
  float* o_part;        // [s, B, H_Q, D]          (kPartials)
  float* m_part;        // [s, B, H_Q]
  float* l_part;        // [s, B, H_Q]
  uint32_t* arrivals;   // kFused: one arrival counter per tile, zero between calls
  const int32_t* block_table;  // paged layout: [B, max_pages] page ids
  const int32_t* seq_lens;     // paged layout: [B] sequence lengths
  int page_size, max_pages, num_pages;
  Div div_page;         // page_size
  const int32_t* work;  // nullable: per-sequence schedule, int32x4 {tile, first, end, state row} per workgroup
  const int32_t* seqs;  // schedule, kFused: int32x2 [B] {first chunk-state row or -1, chunk count}
  int state_rows;       // chunk-state rows of the schedule
  int B, H_Q, H_KV, L_K, g, hpt, tiles_per_seq, tiles, s, mode;
  int xcd_group;        // 1: consecutive tiles share an XCD (packing off)
  Div div_s, div_tps, div_g;  // s, tiles_per_seq, g
  float scale_log2;     // softmax scale * log2(e)
};

// Max and sum over lanes {l, l^16, l^32, l^48}: the 4 row groups of one MFMA
// column.  permlane16_swap(x, x) hands every lane the pair (x[l], x[l^16])
// and permlane32_swap(x, x) the pair (x[l], x[l^32]), in the same order on
// both lanes of a pair, so every lane of a column ends with identical bits.
__device__ __forceinline__ float max_rows(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(c[0]), __uint_as_float(c[1]));
}

__device__ __forceinline__ float sum_rows(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto c = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(c[0]) + __uint_as_float(c[1]);
}

// Two floats to bf16 (round to nearest even), packed low/high in one dword:
// a single v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, bf16x2));
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 x) { return __builtin_bit_cast(bf16x8, x); }

// Byte offset of a shared-memory pointer within the workgroup's LDS.
__device__ __forceinline__ uint32_t lds_offset(const void* ptr) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)ptr;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Maximum over the 64 lanes of a wave (exact: the order does not matter).
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float lane_value(float x, int i) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), i));
}

// The log-sum-exp merge of s <= 64 chunk states (the paper's final
// reduction, Sections 3.1 and 5.3) for up to NR rows, by one wave: the lane
// holds output dims 2*lane and 2*lane + 1 of each row, and lane i holds the
// max and sum of chunk i.  Chunk i of row r is state row base[r] + i * srow
// (Otilde at o_part[row * D], m and l at m_part[row], l_part[row]).  Per
// row: M = max m_i over chunks with l_i > 0, w_i = exp(m_i - M) (0 for an
// empty chunk), then L = sum_i w_i l_i and O = sum_i w_i Otilde_i, both
// accumulated in chunk order i = 0..s-1, O / L rounded to bf16 and lse = M +
// ln L.  Every output element takes the same operations in the same order
// whichever kernel runs this, so the separate combine launch and the
// single-launch merge give the same bits.  COH: the states were written in
// this launch by other workgroups with device-scope stores and are read with
// device-scope loads.  State offsets are below 2 GiB (checked on the host).
template <int NR, bool COH>
__device__ __forceinline__ void merge_rows(const float* o_part, const float* m_part, const float* l_part,
                                           const int64_t (&base)[NR], const int64_t (&orow)[NR], int nr,
                                           int64_t srow, int s, uint16_t* out, float* lse, int lane) {
  constexpr int aux = COH ? kDeviceScope : 0;
  constexpr int CB = NR == 1 ? 16 : (32 / NR > 0 ? 32 / NR : 1);  // chunks loaded at once per row
  const __amdgpu_buffer_rsrc_t ors = make_rsrc(o_part, 0x7fffffff);
  const __amdgpu_buffer_rsrc_t mrs = make_rsrc(m_part, 0x7fffffff);
  const __amdgpu_buffer_rsrc_t lrs = make_rsrc(l_part, 0x7fffffff);
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  float mi[NR], li[NR];
  f32x2 a[NR][CB];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    mi[r] = -INFINITY;
    li[r] = 0.f;
    if (r < nr && lane < s) {
      const uint32_t off = (uint32_t)(base[r] + (int64_t)lane * srow) * 4u;
      mi[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, off, 0, aux));
      li[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(lrs, off, 0, aux));
    }
#pragma unroll
    for (int u = 0; u < CB; ++u)
      if (r < nr && u < s)
        a[r][u] = __builtin_bit_cast(
            f32x2, __builtin_amdgcn_raw_buffer_load_b64(
                       ors, (uint32_t)((base[r] + (int64_t)u * srow) * D + 2 * lane) * 4u, 0, aux));
  }
  float wi[NR], M[NR], L[NR], o0[NR], o1[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const bool live = li[r] > 0.f;
    M[r] = wave_max(live ? mi[r] : -INFINITY);
    wi[r] = live ? __builtin_amdgcn_exp2f((mi[r] - M[r]) * kLog2e) : 0.f;
    L[r] = 0.f;
    for (int i = 0; i < s; ++i) L[r] = fmaf(lane_value(wi[r], i), lane_value(li[r], i), L[r]);
    o0[r] = 0.f;
    o1[r] = 0.f;
  }
  for (int i0 = 0; i0 < s; i0 += CB) {
    if (i0 > 0) {
#pragma unroll
      for (int r = 0; r < NR; ++r)
#pragma unroll
        for (int u = 0; u < CB; ++u)
          if (r < nr && i0 + u < s)
            a[r][u] = __builtin_bit_cast(
                f32x2, __builtin_amdgcn_raw_buffer_load_b64(
                           ors, (uint32_t)((base[r] + (int64_t)(i0 + u) * srow) * D + 2 * lane) * 4u, 0, aux));
    }
#pragma unroll
    for (int u = 0; u < CB; ++u)
      if (i0 + u < s) {
#pragma unroll
        for (int r = 0; r < NR; ++r) {
          const float w = lane_value(wi[r], i0 + u);
          const bool live = lane_value(li[r], i0 + u) > 0.f;
          o0[r] = fmaf(w, live ? a[r][u].x : 0.f, o0[r]);
          o1[r] = fmaf(w, live ? a[r][u].y : 0.f, o1[r]);
        }
      }
  }
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    if (r >= nr) continue;
    const float inv = L[r] > 0.f ? 1.0f / L[r] : 0.f;
    *reinterpret_cast<uint32_t*>(out + orow[r] * D + 2 * lane) = pack_bf16x2(o0[r] * inv, o1[r] * inv);
    if (lse && lane == 0) lse[orow[r]] = L[r] > 0.f ? M[r] + logf(L[r]) : -INFINITY;
  }
}

// The single-launch merge: the last workgroup of a tile merges the tile's
// s chunk states for its hpt <= 32 rows (query heads), with every thread
// holding float4 output columns.  Chunk i of the tile's head h is state row
// srow0 + i * cstride + h (state_rows rows in all); its output row is orow0
// + h.  The states were written in this launch by
// other workgroups with device-scope stores and are read with device-scope
// loads.  Per output element the operations and their order are those of
// merge_rows (maximum over non-empty chunks, then the weights, L and O
// accumulated in chunk order), so both merges give the same bits.  The
// code is kept short and rolled: it runs once per tile, on cold
// instruction caches.  `lds` holds at least 3 x 64 x 32 floats.
template <int NT, int W>
__device__ __forceinline__ void merge_tile(const Params& p, float* lds, int64_t srow0, int64_t cstride, int s,
                                           int64_t orow0, int64_t state_rows, int tid) {
  constexpr int T = 64 * W;              // threads
  constexpr int R = T / 32;              // thread t stages row t % 32 of chunks t / 32 + R u
  constexpr int IPT = NT * 16 * 32 / T;  // float4 columns per thread (hpt * 32 items over T threads)
  constexpr int CB = 16 / IPT;           // chunks of columns loaded at once
  static_assert(CB == da::kFusedBatch[NT - 1], "the planner prices the merge in batches of CB chunks");
  constexpr uint32_t kOut = 0xfffffff0u; // an offset past every buffer: reads zero, touches nothing
  const int hpt = p.hpt;
  // 32-bit offsets: the chunk states of a call stay below 2 GiB (checked on the host), and the
  // buffer ranges end with them, so out-of-range rows and chunks read as zeros
  const uint32_t rows = (uint32_t)cstride;  // state rows between two chunks of one head
  const uint32_t r0 = (uint32_t)srow0;
  const uint32_t nrows = (uint32_t)state_rows;
  const __amdgpu_buffer_rsrc_t mrs = make_rsrc(p.m_part, nrows * 4u);
  const __amdgpu_buffer_rsrc_t lrs = make_rsrc(p.l_part, nrows * 4u);
  const __amdgpu_buffer_rsrc_t ors = make_rsrc(p.o_part, nrows * (uint32_t)D * 4u);
  // chunk rows are padded to 64 + CB so that a batch reads them unconditionally
  float* lm = lds;                               // [64 + CB chunks][32 rows] maxima
  float* ll = lds + (DA_MAX_SPLITS + CB) * 32;   // [64 + CB][32] sums
  float* lp = ll + (DA_MAX_SPLITS + CB) * 32;    // [R][32] maxima over each thread's live chunks
  // column items of this thread: item tid + T j is row item / 32, float4 column item % 32
  uint32_t ooff[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const uint32_t item = (uint32_t)(tid + T * j), h = item >> 5, c = item & 31u;
    ooff[j] = h < (uint32_t)hpt ? ((r0 + h) * D + 4u * c) * 4u : kOut;
  }
  const uint32_t ostride = rows * (uint32_t)D * 4u;  // bytes between two chunks of one row
  f32x4 a[IPT][CB];
  const int items = hpt * 32;  // column items of the tile; item groups j with T j >= items are skipped
  auto load_cols = [&](int i0) {
#pragma unroll
    for (int j = 0; j < IPT; ++j)
#pragma unroll
      for (int u = 0; u < CB; ++u)
        if (T * j < items && i0 + u < s)  // uniform
        a[j][u] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       ors, ooff[j] != kOut ? ooff[j] + (uint32_t)(i0 + u) * ostride : kOut, 0, kDeviceScope));
  };
  auto store_item = [&](int j, float M, float L, const f32x4& o) {
    const int item = tid + T * j, h = item >> 5, c = item & 31;
    if (h >= hpt) return;
    const int64_t row = orow0 + h;
    const float inv = L > 0.f ? 1.0f / L : 0.f;
    *reinterpret_cast<uint2*>(p.out + row * D + 4 * c) =
        make_uint2(pack_bf16x2(o[0] * inv, o[1] * inv), pack_bf16x2(o[2] * inv, o[3] * inv));
    if (p.lse && c == 0) p.lse[row] = L > 0.f ? M + logf(L) : -INFINITY;
  };
  if (s <= CB) {
    // one batch: every thread loads the maxima and sums of its own rows'
    // chunks with its columns and merges in registers (no LDS, no barrier)
    load_cols(0);
    float bm[IPT][CB], bl[IPT][CB];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint32_t h = (uint32_t)(tid + T * j) >> 5;
      const uint32_t moff = h < (uint32_t)hpt ? (r0 + h) * 4u : kOut;
#pragma unroll
      for (int u = 0; u < CB; ++u) {  // chunks past s read as l = 0, never live
        const uint32_t off = moff != kOut && u < s ? moff + (uint32_t)u * rows * 4u : kOut;
        bm[j][u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, off, 0, kDeviceScope));
        bl[j][u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(lrs, off, 0, kDeviceScope));
      }
    }
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      if (T * j >= items) break;  // uniform
      float M = -INFINITY, L = 0.f;
      f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int u = 0; u < CB; ++u) M = bl[j][u] > 0.f ? fmaxf(M, bm[j][u]) : M;
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        if (u < s) {
          const bool live = bl[j][u] > 0.f;
          const float w = live ? __builtin_amdgcn_exp2f((bm[j][u] - M) * kLog2e) : 0.f;
          L = fmaf(w, bl[j][u], L);
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = fmaf(w, a[j][u][e], o[e]);
        }
      }
      store_item(j, M, L, o);
    }
    return;
  }
  {
    const uint32_t h = (uint32_t)tid & 31u;
    const int i0 = tid >> 5;
    const uint32_t moff = h < (uint32_t)hpt ? (r0 + h) * 4u : kOut;
    float mv[DA_MAX_SPLITS / R], lv[DA_MAX_SPLITS / R];
#pragma unroll
    for (int u = 0; u < DA_MAX_SPLITS / R; ++u) {
      if (R * u >= s) break;  // uniform
      const int i = i0 + R * u;
      const uint32_t off = moff != kOut && i < s ? moff + (uint32_t)i * rows * 4u : kOut;
      mv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, off, 0, kDeviceScope));
      lv[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(lrs, off, 0, kDeviceScope));
    }
    load_cols(0);  // in flight while the maxima are staged
    float pm = -INFINITY;
#pragma unroll
    for (int u = 0; u < DA_MAX_SPLITS / R; ++u) {
      if (R * u >= s) break;
      const int i = i0 + R * u;  // < 64; rows and chunks out of range read as l = 0, never live
      lm[i * 32 + h] = mv[u];
      ll[i * 32 + h] = lv[u];
      pm = lv[u] > 0.f ? fmaxf(pm, mv[u]) : pm;
    }
    lp[i0 * 32 + h] = pm;
  }
  __syncthreads();
  float M[IPT], L[IPT];
  f32x4 o[IPT];
  int hh[IPT];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    hh[j] = ((tid + T * j) >> 5) & 31;
    M[j] = -INFINITY;
#pragma unroll
    for (int r = 0; r < R; ++r) M[j] = fmaxf(M[j], lp[r * 32 + hh[j]]);
    L[j] = 0.f;
    o[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int i0 = 0; i0 < s; i0 += CB) {
    if (i0 > 0) load_cols(i0);
    // the batch's maxima and sums, read at once (rows past s are read, never used)
    float bm[IPT][CB], bl[IPT][CB];
#pragma unroll
    for (int j = 0; j < IPT; ++j)
#pragma unroll
      for (int u = 0; u < CB; ++u) {
        bm[j][u] = lm[(i0 + u) * 32 + hh[j]];
        bl[j][u] = ll[(i0 + u) * 32 + hh[j]];
      }
#pragma unroll
    for (int u = 0; u < CB; ++u) {
      if (i0 + u < s) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
          if (T * j >= items) break;  // uniform
          const float mi = bm[j][u], li = bl[j][u];
          const bool live = li > 0.f;
          const float w = live ? __builtin_amdgcn_exp2f((mi - M[j]) * kLog2e) : 0.f;
          L[j] = fmaf(w, li, L[j]);
          // an empty chunk's output is exactly zero here (w = 0 and O~ = 0 add nothing), as the
          // combine's guard on empty chunks makes it
#pragma unroll
          for (int e = 0; e < 4; ++e) o[j][e] = fmaf(w, a[j][u][e], o[j][e]);
        }
      }
    }
  }
#pragma unroll
  for (int j = 0; j < IPT; ++j) store_item(j, M[j], L[j], o[j]);
}

// Waves per SIMD each variant must fit: three for the 16-column direct-fetch
// kernel (launches of many workgroups, several per CU), two otherwise.
template <int NT, int FETCH>
constexpr int kMinWaves = (NT == 1 && FETCH == 0) ? 3 : 2;

// NT: 16-column head tiles per workgroup (1: up to 16 query heads, 2: up to
// 32).  W: waves per workgroup.  FETCH: a Fetch value.  PG: paged K/V cache
// (pages of page_size rows, page_size a multiple of 32; chunks and wave
// ranges are then cut at 32-key tile boundaries, so every tile lies in one
// page).  SCH: per-sequence schedule (p.work lists every workgroup's head
// tile, 32-key tile range and chunk-state row).  Both are template
// parameters so that the uniform launch waits on no extra argument.
template <int NT, int W, int FETCH, bool PG, bool SCH, bool NTL, int VS>
__global__ void __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(kMinWaves<NT, FETCH>, 8)))
split_partial_kernel(Params p) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  // NTL: K/V loads carry the nontemporal hint (the cache-policy field of
  // the buffer instructions), for launches whose K/V cannot stay resident
  constexpr int kv_aux = NTL ? 2 : 0;
  // VS: the workgroup computes 128/VS of the output dims (its V slice); the
  // VS workgroups of a tile's chunk share its scores.  NB 16-dim blocks.
  static_assert(VS == 1 || (FETCH == kFetchLds && !SCH), "V slices only with direct-to-LDS fetch");
  constexpr int NB = 8 / VS;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int col = lane & 15;   // MFMA column: head within a 16-head tile
  const int quad = lane >> 4;  // MFMA row group

  // ---- which tile and chunk this workgroup owns (and which V slice)
  int bid = blockIdx.x;
  int nb0 = 0;  // first 16-dim output block of this workgroup
  if constexpr (VS > 1) {
    // Launched as VS x 8 x ceil(chunks / 8) workgroups: block ids 8i + x
    // hold slice i mod VS of chunk 8 (i / VS) + x, so the slices of a chunk
    // share an XCD and its L2 serves their repeated K reads.  Ids past the
    // last chunk have nothing to do (the whole workgroup leaves at once).
    const int vslice = (bid >> 3) % VS;
    bid = (bid & 7) + 8 * ((bid >> 3) / VS);
    if (bid >= p.tiles * p.s) return;
    nb0 = vslice * NB;
  }
  int tile, split = 0, prow = -1, w_first = 0, w_end = 0;
  if constexpr (SCH) {
    // scheduled: this workgroup's head tile, 32-key tile range and state row
    tile = p.work[4 * bid];
    w_first = p.work[4 * bid + 1];
    w_end = p.work[4 * bid + 2];
    prow = p.work[4 * bid + 3];
    if (tile < 0 || tile >= p.tiles || prow >= p.state_rows) return;  // not a schedule of this shape
  } else {
    const int nwg = p.tiles * p.s;
    const int logical = (p.xcd_group && nwg % 8 == 0) ? (bid % 8) * (nwg / 8) + bid / 8 : bid;
    tile = div_by(logical, p.div_s);
    split = logical - tile * p.s;
  }
  const int b = div_by(tile, p.div_tps);
  const int head0 = (tile - b * p.tiles_per_seq) * p.hpt;
  const int kvh = div_by(head0, p.div_g);

  int64_t row0 = 0;
  int L;
  if constexpr (PG) {
    L = p.seq_lens[b];
    L = L < 0 ? 0 : (L > p.L_K ? p.L_K : L);
  } else if (p.cu) {
    row0 = p.cu[b];
    L = p.cu[b + 1] - p.cu[b];
    L = L < 0 ? 0 : (L > p.L_K ? p.L_K : L);
  } else {
    row0 = (int64_t)b * p.L_K;
    L = p.L_K;
  }
  // Two waves over key rows of at most 1 KiB take the chunk's 32-key tiles
  // alternately (wave w: tiles w, w + 2, ...), so that a workgroup reads one
  // contiguous front.  Against contiguous halves on such rows (pure MQA and
  // 2-4 KV heads, 13 shapes of 192-320 workgroups): 2.1% faster on average
  // on one MI355X and 1.0% on another (0.94-1.04x per shape); on 2 KiB rows
  // (8 KV heads) 0.95-1.034x by shape, and with four waves 1.0-1.03x.
  // A wave then walks [key_lo, key_hi) in steps of `kstep` keys.
  const bool alternate = W == 2 && p.H_KV <= 4;
  const int kstep = alternate ? kKeysPerTile * W : kKeysPerTile;
  int key_lo, key_hi;
  if constexpr (PG || SCH) {
    // tiles of 32 keys cut into s chunks (or the scheduled range), each
    // chunk's tiles into W ranges
    const uint32_t T = (uint32_t)(L + kKeysPerTile - 1) / kKeysPerTile;
    uint32_t t0, nt;
    if constexpr (SCH) {
      const uint32_t f = (uint32_t)(w_first < 0 ? 0 : w_first);
      const uint32_t e = (uint32_t)(w_end < 0 ? 0 : w_end);
      t0 = f < T ? f : T;
      nt = (e < T ? e : T) > t0 ? (e < T ? e : T) - t0 : 0u;
    } else {
      t0 = (uint32_t)div_by((int)(T * (uint32_t)split), p.div_s);
      nt = (uint32_t)div_by((int)(T * (uint32_t)(split + 1)), p.div_s) - t0;
    }
    if (alternate) {
      key_lo = kKeysPerTile * (int)(t0 + (uint32_t)wave);
      key_hi = kKeysPerTile * (int)(t0 + nt);
    } else {
      key_lo = kKeysPerTile * (int)(t0 + nt * (uint32_t)wave / W);
      key_hi = kKeysPerTile * (int)(t0 + nt * (uint32_t)(wave + 1) / W);
    }
    key_hi = key_hi < L ? key_hi : L;
    key_lo = key_lo < key_hi ? key_lo : key_hi;
  } else {
    // L < 2^23 (one sequence's K spans < 2 GiB) and split < 64, so the
    // products fit 32 bits and the divisions stay 32-bit
    const int c0 = div_by(L * split, p.div_s);
    const int c1 = div_by(L * (split + 1), p.div_s);
    const int n = c1 - c0;
    if (alternate) {
      key_lo = c0 + kKeysPerTile * wave;
      key_hi = c1;
      key_lo = key_lo < key_hi ? key_lo : key_hi;
    } else {
      key_lo = c0 + (int)(((uint32_t)n * (uint32_t)wave) / W);
      key_hi = c0 + (int)(((uint32_t)n * (uint32_t)(wave + 1)) / W);
    }
  }

  // ---- K/V tile addressing.  Tile t holds keys [key_lo + kstep t, +32) of this
  //      (sequence, KV head); its buffer resource starts at that tile's first
  //      row (rows of H_KV*256 bytes) and ends at this wave's last key: any
  //      key >= key_hi is out of range and reads as zeros without touching
  //      memory, so no load needs a mask and ragged tails cost no traffic.
  //      Per-lane offsets below are relative to the tile's first row.
  const uint32_t rs = (uint32_t)p.H_KV * (D * 2);
  const int64_t base_elems = (row0 * p.H_KV + kvh) * D;
  // paged: this wave's page ids, 64 at a time, one per lane
  int pg_first = 0, pg_last = -1, pg_win = 0, pg_ids = 0;
  if constexpr (PG) {
    if (key_hi > key_lo) {
      pg_first = div_by(key_lo, p.div_page);
      pg_last = div_by(key_hi - 1, p.div_page);
    }
    pg_win = pg_first;
    const int j = pg_win + lane;
    pg_ids = j <= pg_last ? p.block_table[(int64_t)b * p.max_pages + j] : 0;
  }
  // element offset of tile t's first row and its record count in bytes
  auto tile_place = [&](int t, int64_t& elems, uint32_t& bytes) {
    const int first = key_lo + t * kstep;
    const int rows = key_hi - first;
    bytes = (uint32_t)__builtin_amdgcn_readfirstlane(rows > 0 ? (uint32_t)rows * rs : 0u);
    if constexpr (PG) {
      const int j = div_by(first, p.div_page);
      if (j - pg_win >= 64 && rows > 0) {  // next window of page ids (wave-uniform)
        pg_win = j;
        const int jj = pg_win + lane;
        pg_ids = jj <= pg_last ? p.block_table[(int64_t)b * p.max_pages + jj] : 0;
      }
      const int page = __builtin_amdgcn_readlane(pg_ids, (j - pg_win) & 63);
      // a page id outside the cache reads as zero keys and values
      if (page < 0 || page >= p.num_pages) bytes = 0u;
      const int64_t prow = (page < 0 || page >= p.num_pages ? 0 : (int64_t)page) * p.page_size +
                           (first - j * p.page_size);
      elems = (prow * p.H_KV + kvh) * D;
    } else {
      elems = base_elems + (int64_t)first * p.H_KV * D;
    }
  };

  // ---- Q^T as the MFMA B operand.  The reduction index of the product may
  //      map to head dims in any order as long as K and Q agree: k-step j,
  //      lane group `quad` covers dims [32j + 8*quad, +8).  Lane holds those
  //      dims of head column `col` (zeros for padding).
  bf16x8 qreg[NT][4];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int h = nt * 16 + col;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u32x4 x = {0u, 0u, 0u, 0u};
      if (h < p.hpt)
        x = *reinterpret_cast<const u32x4*>(p.q + ((int64_t)b * p.H_Q + head0 + h) * D + 32 * j + 8 * quad);
      qreg[nt][j] = as_bf16x8(x);
    }
  }

  float m_run[NT], l_run[NT];
  f32x4 acc_o[NT][NB];  // output blocks nb0 .. nb0 + NB - 1
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    m_run[nt] = -INFINITY;
    l_run[nt] = 0.f;
#pragma unroll
    for (int nn = 0; nn < NB; ++nn) acc_o[nt][nn] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  constexpr bool KS = FETCH == kFetchStaged;
  unsigned char* vstage = smem + wave * stage_bytes(FETCH);
  unsigned char* kstage = vstage + kKeysPerTile * kVPitch;
  const int ntiles = (key_hi - key_lo + kstep - 1) / kstep;

  // K/V of one 32-key tile.  V always comes as 8 rows-of-4 (16 consecutive
  // lanes read one 256-byte row) for its LDS stage.  K either comes the same
  // way and takes its own LDS stage (KS), from which it is read back in the
  // MFMA A layout, or is fetched straight into that layout: lane (row r,
  // group q) loads dims [32j + 8q, +8) of key r for j = 0..3 (64 bytes of
  // one row), so neighbouring lanes read different rows, which the memory pipeline
  // serves at about half the rate of row-contiguous lanes.  The per-lane
  // byte offsets are fixed; tile t moves the descriptor base by t*32 rows
  // and shrinks its record count to match (scalar work only).
  const uint32_t koff[2] = {(uint32_t)col * rs + 16u * quad, (uint32_t)(16 + col) * rs + 16u * quad};
  uint32_t voff[8];
#pragma unroll
  for (int jj = 0; jj < 8; ++jj) voff[jj] = (uint32_t)(4 * jj + quad) * rs + 16u * col;
  auto load_tile = [&](u32x4 (&kreg)[2][4], u32x4 (&vreg)[8], int t) {
    int64_t elems;
    uint32_t left;
    tile_place(t, elems, left);
    const __amdgpu_buffer_rsrc_t kt = make_rsrc(p.k + elems, left);
    const __amdgpu_buffer_rsrc_t vt = make_rsrc(p.v + elems, left);
    if constexpr (KS) {
      // kreg[mt][j]: rows 16mt + 4j + quad, bytes [16 col, +16)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          kreg[mt][j] = __builtin_amdgcn_raw_buffer_load_b128(kt, voff[4 * mt + j], 0, kv_aux);
    } else {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          kreg[mt][j] = __builtin_amdgcn_raw_buffer_load_b128(kt, koff[mt] + 64u * j, 0, kv_aux);
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) vreg[jj] = __builtin_amdgcn_raw_buffer_load_b128(vt, voff[jj], 0, kv_aux);
  };

  // S^T[16 keys x 16 heads] per (mt, nt) from the tile's 8 K operands.
  auto scores = [&](const bf16x8 (&kop)[2][4], f32x4 (&sc)[NT][2]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kop[mt][j], qreg[nt][j], acc, 0, 0, 0);
        sc[nt][mt] = acc;
      }
  };

  // Online softmax per head column, in log2 units of the scaled score: the
  // max is taken on raw scores (the scale is positive) and each exponent is
  // one fma, raw * scale*log2(e) - running max.  `last`: only the final tile
  // can be shorter than 32 keys and needs its scores masked.
  auto softmax = [&](f32x4 (&sc)[NT][2], int nvalid, auto last, bf16x8 (&pb)[NT]) {
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float x[8];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float r = sc[nt][mt][i];
          if constexpr (decltype(last)::value) r = (mt * 16 + quad * 4 + i) < nvalid ? r : -INFINITY;
          x[mt * 4 + i] = r;
        }
      const float rmax = max_rows(fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])),
                                        fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7]))));
      const float m_new = fmaxf(m_run[nt], rmax * p.scale_log2);
      const float alpha = __builtin_amdgcn_exp2f(m_run[nt] - m_new);
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        x[e] = __builtin_amdgcn_exp2f(fmaf(x[e], p.scale_log2, -m_new));
        psum += x[e];
      }
      l_run[nt] = l_run[nt] * alpha + psum;
      m_run[nt] = m_new;
      // alpha == 1 exactly when the column max did not move: skip the
      // multiply by one (a wave-uniform branch)
      if (__any(alpha != 1.0f)) {
#pragma unroll
        for (int nn = 0; nn < NB; ++nn) acc_o[nt][nn] *= alpha;
      }
      u32x4 pk;
      pk.x = pack_bf16x2(x[0], x[1]);
      pk.y = pack_bf16x2(x[2], x[3]);
      pk.z = pack_bf16x2(x[4], x[5]);
      pk.w = pack_bf16x2(x[6], x[7]);
      pb[nt] = as_bf16x8(pk);
    }
  };

  // O^T[16 dims x 16 heads] += V^T[16 dims x 32 keys] . P^T[32 keys x 16 heads]
  // The k index 8*quad + 4*mt + i of the product stands for key
  // 16*mt + 4*quad + i, matching the score layout.  The V^T operand comes
  // from transposing LDS reads (ds_read_b64_tr_b16): within each 16-lane
  // group, output lane j receives element j%4 of the 8-byte chunks that
  // lanes 4k + j/4 point at, k = 0..3.  Lane (quad, 4k + m) therefore points
  // at dims [16nn + 4m, +4) of key 16mt + 4quad + k -- vaddr(mt, nn) gives
  // that address for the stage layout in use -- and lane (quad, col)
  // receives V[16mt + 4quad + k][16nn + col] for k = 0..3.  All 16 reads are
  // issued before the first product so their LDS latency is paid once per
  // tile rather than once per 16 output dims.
  // With direct-to-LDS loads in flight (`opaque`; vaddr then gives LDS byte
  // offsets), the reads are written as inline assembly followed by an
  // explicit wait: the compiler cannot tell that they touch the other stage
  // and would otherwise drain every outstanding load before them.
  auto pv = [&](const bf16x8 (&pb)[NT], auto vaddr, auto opaque) {
    s16x4 vlo[NB], vhi[NB];
    if constexpr (decltype(opaque)::value) {
#pragma unroll
      for (int nn = 0; nn < NB; ++nn) {
        asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(vlo[nn]) : "v"((uint32_t)vaddr(0, nn)) : "memory");
        asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(vhi[nn]) : "v"((uint32_t)vaddr(1, nn)) : "memory");
      }
      // The wait names every result as an operand it updates, so nothing
      // that reads them can be scheduled before it.
      if constexpr (NB == 8)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(vlo[0]), "+v"(vlo[1]), "+v"(vlo[2]), "+v"(vlo[3]), "+v"(vlo[4]), "+v"(vlo[5]),
                       "+v"(vlo[6]), "+v"(vlo[7]), "+v"(vhi[0]), "+v"(vhi[1]), "+v"(vhi[2]), "+v"(vhi[3]),
                       "+v"(vhi[4]), "+v"(vhi[5]), "+v"(vhi[6]), "+v"(vhi[7])
                     :
                     : "memory");
      else if constexpr (NB == 4)
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(vlo[0]), "+v"(vlo[1]), "+v"(vlo[2]), "+v"(vlo[3]), "+v"(vhi[0]), "+v"(vhi[1]),
                       "+v"(vhi[2]), "+v"(vhi[3])
                     :
                     : "memory");
      else
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(vlo[0]), "+v"(vlo[1]), "+v"(vhi[0]), "+v"(vhi[1]) : : "memory");
    } else {
#pragma unroll
      for (int nn = 0; nn < NB; ++nn) {
        vlo[nn] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)vaddr(0, nn));
        vhi[nn] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)vaddr(1, nn));
      }
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * NB, 0);   // the DS reads first
    __builtin_amdgcn_sched_group_barrier(0x008, NB * NT, 0);  // then the MFMAs
#pragma unroll
    for (int nn = 0; nn < NB; ++nn) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, __builtin_shufflevector(vlo[nn], vhi[nn], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
        acc_o[nt][nn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[nt], acc_o[nt][nn], 0, 0, 0);
    }
  };

  constexpr std::true_type yes{};
  constexpr std::false_type no{};
  if constexpr (FETCH != kFetchLds) {
    // One tile held in (kreg, vreg).  `prefetch`: refill those registers
    // with tile t + 1 once K has been consumed (the loop refills
    // unconditionally, so the compiler waits for exactly the tile in use; the
    // final tile does not refill).  More tiles in flight per wave (a ring of
    // register buffers) measured slower: it needs more registers than a wave
    // may hold without spilling into accumulation registers.
    auto process = [&](u32x4 (&kreg)[2][4], u32x4 (&vreg)[8], int t, auto prefetch, auto last) {
      const int nvalid = key_hi - (key_lo + t * kstep);  // >= 1 (> 32: a full tile)
      bf16x8 kop[2][4];
      if constexpr (KS) {
        // row-major K tile in LDS (kKPitch bytes per key), read back so that
        // lane (col, quad) of operand (mt, j) holds dims [32j + 8quad, +8) of
        // key 16mt + col
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            *reinterpret_cast<u32x4*>(kstage + (16 * mt + 4 * j + quad) * kKPitch + 16 * col) = kreg[mt][j];
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            kop[mt][j] =
                as_bf16x8(*reinterpret_cast<const u32x4*>(kstage + (16 * mt + col) * kKPitch + 16 * (4 * j + quad)));
      } else {
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
#pragma unroll
          for (int j = 0; j < 4; ++j) kop[mt][j] = as_bf16x8(kreg[mt][j]);
      }
      f32x4 sc[NT][2];
      scores(kop, sc);

      // stage V rows in LDS (row-major, padded pitch)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        *reinterpret_cast<u32x4*>(vstage + (4 * jj + quad) * kVPitch + 16 * col) = vreg[jj];

      if constexpr (decltype(prefetch)::value) load_tile(kreg, vreg, t + 1);

      bf16x8 pb[NT];
      softmax(sc, nvalid, last, pb);
      __builtin_amdgcn_wave_barrier();
      const unsigned char* vrow = vstage + (quad * 4 + (col >> 2)) * kVPitch + 8 * (col & 3);
      pv(pb, [&](int mt, int nn) { return vrow + mt * 16 * kVPitch + 32 * nn; }, no);
      __builtin_amdgcn_wave_barrier();
    };

    u32x4 kreg[2][4], vreg[8];
    load_tile(kreg, vreg, 0);
    int t = 0;
    for (; t + 1 < ntiles; ++t) process(kreg, vreg, t, yes, no);
    if (t < ntiles) process(kreg, vreg, t, no, yes);
  } else {
    // Direct-to-LDS: each wave has two stages; tile t + 1 streams into one
    // while tile t is reduced from the other.  Lane l of a load instruction
    // for block b (rows 4b + l/16 of the tile) fills position l%16 of its
    // row, which holds chunk (l%16 - 2r) mod 16, r = l/16.
    const int rr = lane >> 4;
    const int cp = lane & 15;
    uint32_t dmaoff[8];
#pragma unroll
    for (int blk = 0; blk < 8; ++blk)
      dmaoff[blk] = (uint32_t)(4 * blk + rr) * rs + 16u * (uint32_t)((cp - 2 * rr) & 15);
    unsigned char* const sbase = smem + wave * stage_bytes(FETCH);
    // with V slices a lane loads its V chunk only if the chunk (8 dims) is
    // in this workgroup's slice: dims [16 nb0, 16 (nb0 + NB))
    const int vblock = ((cp - 2 * rr) & 15) >> 1;
    const bool vload = VS == 1 || (vblock >= nb0 && vblock < nb0 + NB);
    auto dma_tile = [&](int stage, int t) {
      int64_t elems;
      uint32_t left;
      tile_place(t, elems, left);
      const __amdgpu_buffer_rsrc_t kt = make_rsrc(p.k + elems, left);
      const __amdgpu_buffer_rsrc_t vt = make_rsrc(p.v + elems, left);
      unsigned char* ks = sbase + stage * kLdsStageBytes;
      unsigned char* vs = ks + kLdsTileBytes;
#pragma unroll
      for (int blk = 0; blk < 8; ++blk)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(kt, (lds_void*)(ks + blk * kBlockStride), 16, dmaoff[blk], 0, 0,
                                                 kv_aux);
      if (vload) {
#pragma unroll
        for (int blk = 0; blk < 8; ++blk)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(vt, (lds_void*)(vs + blk * kBlockStride), 16, dmaoff[blk], 0, 0,
                                                   kv_aux);
      }
    };
    // Operand reads.  K operand (mt, j), lane (col, quad): key 16mt + col is
    // row col%4 of block 4mt + col/4, dims [32j + 8quad, +8) are its chunk
    // 4j + quad.  V (see pv): key 16mt + 4quad + k is row k of block
    // 4mt + quad, dims [16nn + 4m, +4) sit in chunk 2nn + m/2.  The rotated
    // offsets differ per lane and per operand, so they are computed once.
    uint32_t kro[2][4], vro[2][NB];
    {
      const int kr = col & 3;
      const int vk = col >> 2;
      const int vm = col & 3;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          kro[mt][j] = lds_offset(sbase) + (uint32_t)((4 * mt + (col >> 2)) * kBlockStride + kr * 256 +
                                                      16 * ((4 * j + quad + 2 * kr) & 15));
#pragma unroll
        for (int nn = 0; nn < NB; ++nn)
          vro[mt][nn] = lds_offset(sbase) +
                        (uint32_t)(kLdsTileBytes + (4 * mt + quad) * kBlockStride + vk * 256 +
                                   16 * ((2 * (nb0 + nn) + (vm >> 1) + 2 * vk) & 15) + 8 * (vm & 1));
      }
    }
    // `stage` is a compile-time constant, so its offset folds into the LDS
    // instructions' immediate field.
    auto reduce = [&](auto stage, int t, auto last) {
      constexpr uint32_t so = decltype(stage)::value * kLdsStageBytes;
      bf16x8 kop[2][4];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          kop[mt][j] = as_bf16x8(*reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(
              (uintptr_t)(kro[mt][j] + so)));
      f32x4 sc[NT][2];
      scores(kop, sc);
      bf16x8 pb[NT];
      softmax(sc, key_hi - (key_lo + t * kstep), last, pb);
      pv(pb, [&](int mt, int nn) { return vro[mt][nn] + so; }, yes);
    };
    // The compiler cannot see that the LDS reads depend on the direct-to-LDS
    // loads, so the waits are explicit: 16 loads per tile, completing in
    // issue order.  Tile t lives in stage t % 2; the loop takes tiles in
    // pairs so that each stage is known at compile time.
    constexpr std::integral_constant<int, 0> s0{};
    constexpr std::integral_constant<int, 1> s1{};
    if (ntiles > 0) dma_tile(0, 0);
    int t = 0;
    for (; t + 2 < ntiles; t += 2) {
      dma_tile(1, t + 1);
      asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
      reduce(s0, t, no);
      dma_tile(0, t + 2);
      asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
      reduce(s1, t + 1, no);
    }
    if (t + 1 < ntiles) {
      dma_tile(1, t + 1);
      asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
      reduce(s0, t, no);
      ++t;
    }
    if (t < ntiles) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (t & 1)
        reduce(s1, t, yes);
      else
        reduce(s0, t, yes);
    }
  }

  // ---- merge the W wave states in one step.  Every wave publishes its
  //      state (per head column: running max, row-summed l, 8 x 4 output
  //      values; all waves share one lane layout) to LDS value-major
  //      ([value][lane], conflict-free).  After one barrier, wave w merges
  //      the W states for its 8/W blocks of 16 output dims -- maximum,
  //      weights, then sums taken in wave order, so the result is the same
  //      on every run -- and writes that slice of the output.
  // With fewer blocks than waves (V slices) waves 0 .. NB - 1 merge one
  // block each and the others only take part in the exchange.
  static_assert(NB % W == 0 || W % NB == 0, "blocks must divide among the waves");
  constexpr int NBW = NB >= W ? NB / W : 1;
  constexpr int SV = 2 + 4 * NB;  // state values per lane and head tile: m, l, NB x 4 outputs
  const bool merges = NB >= W || wave < NB;
  float lsum[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) lsum[nt] = sum_rows(l_run[nt]);
  auto slot = [&](int w) { return reinterpret_cast<float*>(smem) + (size_t)w * (NT * SV * 64); };
  __syncthreads();  // every wave is done with its stages
  {
    float* v0 = slot(wave) + lane;
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      float* v = v0 + nt * SV * 64;
      v[0] = m_run[nt];
      v[64] = lsum[nt];
#pragma unroll
      for (int nn = 0; nn < NB; ++nn)
#pragma unroll
        for (int i = 0; i < 4; ++i) v[(2 + nn * 4 + i) * 64] = acc_o[nt][nn][i];
    }
  }
  __syncthreads();

  const int64_t rows = (int64_t)p.B * p.H_Q;
  const int64_t row0_tile = (int64_t)b * p.H_Q + head0;
  const bool direct = SCH ? prow < 0 : p.mode == kDirect;
  // first chunk-state row of this workgroup's heads
  const int64_t srow0 = direct ? 0 : (SCH ? (int64_t)prow * p.H_Q + head0 : (int64_t)split * rows + row0_tile);
  const __amdgpu_buffer_rsrc_t ors = make_rsrc(p.o_part + srow0 * D, (uint32_t)p.hpt * D * 4);
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    float mk[W], wk[W];
    float M = -INFINITY;
#pragma unroll
    for (int k = 0; k < W; ++k) {
      mk[k] = slot(k)[nt * SV * 64 + lane];
      M = fmaxf(M, mk[k]);
    }
    float Lw = 0.f;
#pragma unroll
    for (int k = 0; k < W; ++k) {
      wk[k] = M == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mk[k] - M);  // all empty: stays empty
      Lw = fmaf(wk[k], slot(k)[(nt * SV + 1) * 64 + lane], Lw);
    }
    // lane (col, quad) owns dims 16(nb0 + nn) + 4quad + [0, 4) of head
    // 16nt + col, nn = wave * NBW + bb
    f32x4 o[NBW];
#pragma unroll
    for (int bb = 0; bb < NBW; ++bb) {
      const int nn = merges ? wave * NBW + bb : 0;
      o[bb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int k = 0; k < W; ++k)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[bb][i] = fmaf(wk[k], slot(k)[(nt * SV + 2 + nn * 4 + i) * 64 + lane], o[bb][i]);
    }
    const int h = nt * 16 + col;
    if (h >= p.hpt || !merges) continue;
    const int64_t row = row0_tile + h;
    const float mval = Lw > 0.f ? M * kLn2 : -INFINITY;
    if (direct) {
      const float inv = Lw > 0.f ? 1.0f / Lw : 0.f;
#pragma unroll
      for (int bb = 0; bb < NBW; ++bb) {
        const int nn = nb0 + wave * NBW + bb;
        *reinterpret_cast<uint2*>(p.out + row * D + 16 * nn + 4 * quad) =
            make_uint2(pack_bf16x2(o[bb][0] * inv, o[bb][1] * inv), pack_bf16x2(o[bb][2] * inv, o[bb][3] * inv));
      }
      if (p.lse && wave == 0 && quad == 0 && nb0 == 0) p.lse[row] = Lw > 0.f ? mval + logf(Lw) : -INFINITY;
    } else if (p.mode == kPartials) {
#pragma unroll
      for (int bb = 0; bb < NBW; ++bb) {
        const int nn = nb0 + wave * NBW + bb;
        const u32x4 bits = {__float_as_uint(o[bb][0]), __float_as_uint(o[bb][1]), __float_as_uint(o[bb][2]),
                            __float_as_uint(o[bb][3])};
        __builtin_amdgcn_raw_buffer_store_b128(bits, ors, (uint32_t)(h * D + 16 * nn + 4 * quad) * 4u, 0, 0);
      }
      if (wave == 0 && quad == 0 && nb0 == 0) {
        p.m_part[srow0 + h] = mval;
        p.l_part[srow0 + h] = Lw;
      }
    } else {
      // kFused: device-scope stores write the chunk state through L2, so
      // it is visible to every XCD once the stores have completed
#pragma unroll
      for (int bb = 0; bb < NBW; ++bb) {
        const int nn = nb0 + wave * NBW + bb;
        const u32x4 bits = {__float_as_uint(o[bb][0]), __float_as_uint(o[bb][1]), __float_as_uint(o[bb][2]),
                            __float_as_uint(o[bb][3])};
        __builtin_amdgcn_raw_buffer_store_b128(bits, ors, (uint32_t)(h * D + 16 * nn + 4 * quad) * 4u, 0,
                                               kDeviceScope);
      }
      if (wave == 0 && quad == 0 && nb0 == 0) {
        __hip_atomic_store(p.m_part + srow0 + h, mval, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(p.l_part + srow0 + h, Lw, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  // Two-wave kernels never merge in the launch (their plans use the second
  // launch; the merge's batches are sized for four waves).
  if constexpr (W == 4) if (p.mode == kFused && !direct) {
    // Single-launch merge.  Hand-off: every wave waits until its chunk
    // state stores have completed (they are device-scope, written through
    // L2), then thread 0 takes an arrival ticket for the tile.  The
    // workgroup that takes the last of the tile's tickets (s x VS, or a
    // scheduled sequence's chunk count) has seen every other workgroup's
    // ticket, each taken after that workgroup's stores completed, so
    // device-scope loads now return all the states.  This is the agent-scope
    // release/acquire sequence of the AMDGPU memory model without its L2
    // write-back and invalidate, which only non-atomic data needs; the chunk
    // states are written and read with device-scope (sc1) accesses only.  No
    // workgroup waits for another.  The last one sets the counter back to
    // zero for the next call.
    int s_m;
    int64_t srow_m, cstride, nrows;
    uint32_t n;
    if constexpr (SCH) {
      // the sequence's chunks are state rows first, first + 1, ... (uniform across the workgroup)
      const int first = p.seqs[2 * b], chunks = p.seqs[2 * b + 1];
      s_m = chunks;
      n = (uint32_t)chunks;
      srow_m = (int64_t)first * p.H_Q + head0;
      cstride = p.H_Q;
      nrows = (int64_t)p.state_rows * p.H_Q;
    } else {
      s_m = p.s;
      n = (uint32_t)p.s * VS;
      srow_m = row0_tile;
      cstride = rows;
      nrows = (int64_t)p.s * rows;
    }
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      // counters sit a cache line apart: atomics on one line are serialised
      uint32_t* counter = p.arrivals + (size_t)tile * da::kArrivalStride;
      const uint32_t prev = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const bool last = prev + 1u == n;
      if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_last = last ? 1 : 0;
    }
    __syncthreads();
    if (!s_last) return;
    merge_tile<NT, W>(p, reinterpret_cast<float*>(smem), srow_m, cstride, s_m, row0_tile, nrows, tid);
  }
}

// Log-sum-exp combine launch: one wave64 per (b, h) row, 2 dims per lane
// (merge_rows), so the result is bit-identical across runs, producers of the
// same chunk states, and the single-launch merge.  SEQ: per-sequence chunk
// counts and state rows from `seqs`.
template <bool SEQ>
__global__ void __launch_bounds__(256) split_combine_kernel(const float* __restrict__ o_part,
                                                            const float* __restrict__ m_part,
                                                            const float* __restrict__ l_part,
                                                            uint16_t* __restrict__ out, float* __restrict__ lse,
                                                            int s, int64_t rows,
                                                            const int32_t* __restrict__ seqs, int H_Q,
                                                            Div div_hq) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;  // waves are independent: no workgroup barrier below
  // Chunk i of this row sits at state row base + i * srow: uniform split
  // counts interleave the rows; a per-sequence schedule stores sequence b's
  // chunks from its first state row on (unsplit sequences are already done).
  int64_t base = row, srow = rows;
  if constexpr (SEQ) {
    const int b = div_by((int)row, div_hq);  // rows = B * H_Q < 2^24
    const int h = (int)row - b * H_Q;
    const int r0 = seqs[2 * b];
    s = seqs[2 * b + 1];
    if (r0 < 0 || s <= 1) return;
    s = s < DA_MAX_SPLITS ? s : DA_MAX_SPLITS;
    base = (int64_t)r0 * H_Q + h;
    srow = H_Q;
  }
  const int64_t bases[1] = {base};
  const int64_t orows[1] = {row};
  merge_rows<1, false>(o_part, m_part, l_part, bases, orows, 1, srow, s, out, lse, lane);
}

// ---------------------------------------------------------------- host side

constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];
std::atomic<int> g_lds[kMaxDevices];    // LDS bytes one workgroup may use
std::atomic<int> g_is950[kMaxDevices];  // 0 unknown, 1 yes, 2 no

int query_device(int* cus, int* is950, int* lds = nullptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return da::fail(DA_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return da::fail(DA_ERR_UNSUPPORTED, "device index %d", dev);
  if (g_is950[dev].load() == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return da::fail(DA_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    g_cus[dev].store(prop.multiProcessorCount);
    g_lds[dev].store((int)prop.sharedMemPerBlock);
    g_is950[dev].store(strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2);
  }
  *cus = g_cus[dev].load();
  *is950 = g_is950[dev].load() == 1;
  if (lds) *lds = g_lds[dev].load();
  return DA_OK;
}

bool aligned(const void* ptr, uintptr_t a) { return ((uintptr_t)ptr & (a - 1)) == 0; }

int check_inputs(const void* q, const void* k, const void* v, const int32_t* cu, int B, int H_Q, int H_KV,
                 int L_K_max, int d) {
  int rc = da::check_shape(B, H_Q, H_KV, L_K_max, d);
  if (!q) return da::fail(DA_ERR_NULL, "q must be non-NULL");
  // With L_K_max == 0 no key is ever read, so an empty cache may be NULL.
  if ((!k || !v) && !(rc == DA_OK && L_K_max == 0)) return da::fail(DA_ERR_NULL, "k and v must be non-NULL");
  if (rc) return rc;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16))
    return da::fail(DA_ERR_ALIGN, "q, k and v must be 16-byte aligned");
  if (cu && !aligned(cu, 4)) return da::fail(DA_ERR_ALIGN, "cu_seqlens_k must be 4-byte aligned");
  return DA_OK;
}

// Chunk states are addressed with 32-bit buffer offsets.
int check_state_size(int B, int H_Q, int s) {
  if ((int64_t)s * B * H_Q * D * 4 >= ((int64_t)1 << 31))
    return da::fail(DA_ERR_SHAPE, "num_splits*B*H_Q*D*4 = %lld bytes of chunk state exceed 2 GiB",
                    (long long)s * B * H_Q * D * 4);
  return DA_OK;
}

int ensure_gfx950(int* cus) {
  int is950 = 0;
  int rc = query_device(cus, &is950);
  if (rc) return rc;
  if (!is950) return da::fail(DA_ERR_UNSUPPORTED, "current device is not gfx950");
  return DA_OK;
}

template <int NT, int W, int FETCH, bool PG, bool SCH, bool NTL, int VS = 1>
const void* kernel_ptr() {
  return reinterpret_cast<const void*>(&split_partial_kernel<NT, W, FETCH, PG, SCH, NTL, VS>);
}

template <bool PG, bool SCH, bool NTL>
const void* pick_kernel(int NT, int FETCH, int VS, int W) {
  if (W == 2) {
    // two waves, K/V through registers: uniform and paged launches without V slices
    if constexpr (SCH) {
      return nullptr;
    } else {
      if (VS != 1) return nullptr;
      switch (FETCH * 2 + NT - 1) {
        case 0: return kernel_ptr<1, 2, kFetchDirect, PG, SCH, NTL>();
        case 1: return kernel_ptr<2, 2, kFetchDirect, PG, SCH, NTL>();
        case 2: return kernel_ptr<1, 2, kFetchStaged, PG, SCH, NTL>();
        case 3: return kernel_ptr<2, 2, kFetchStaged, PG, SCH, NTL>();
        default: return nullptr;
      }
    }
  }
  if (W != 4) return nullptr;
  if (VS != 1) {
    // V slices: direct-to-LDS fetch of uniform launches only
    if constexpr (SCH) {
      return nullptr;
    } else {
      if (FETCH != kFetchLds) return nullptr;
      if (VS == 2)
        return NT == 1 ? kernel_ptr<1, 4, kFetchLds, PG, SCH, NTL, 2>()
                       : kernel_ptr<2, 4, kFetchLds, PG, SCH, NTL, 2>();
      if (VS == 4)
        return NT == 1 ? kernel_ptr<1, 4, kFetchLds, PG, SCH, NTL, 4>()
                       : kernel_ptr<2, 4, kFetchLds, PG, SCH, NTL, 4>();
      return nullptr;
    }
  }
  switch (FETCH * 2 + NT - 1) {
    case 0: return kernel_ptr<1, 4, kFetchDirect, PG, SCH, NTL>();
    case 1: return kernel_ptr<2, 4, kFetchDirect, PG, SCH, NTL>();
    case 2: return kernel_ptr<1, 4, kFetchStaged, PG, SCH, NTL>();
    case 3: return kernel_ptr<2, 4, kFetchStaged, PG, SCH, NTL>();
    case 4: return kernel_ptr<1, 4, kFetchLds, PG, SCH, NTL>();
    case 5: return kernel_ptr<2, 4, kFetchLds, PG, SCH, NTL>();
    default: return nullptr;
  }
}

template <bool NTL>
const void* pick_kernel(bool paged, bool scheduled, int NT, int FETCH, int VS, int W) {
  if (paged)
    return scheduled ? pick_kernel<true, true, NTL>(NT, FETCH, VS, W)
                     : pick_kernel<true, false, NTL>(NT, FETCH, VS, W);
  return scheduled ? pick_kernel<false, true, NTL>(NT, FETCH, VS, W) : pick_kernel<false, false, NTL>(NT, FETCH, VS, W);
}

int launch_partial(const Params& prm, const da_plan& pl, hipStream_t stream) {
  const int W = pl.group_waves;
  const int NT = pl.heads_per_tile <= 16 ? 1 : 2;
  const int FETCH = pl.kv_fetch;
  if (W != 4 && W != 2) return da::fail(DA_ERR_ARG, "plan asks for %d waves per workgroup", W);
  if (W == 2 && (pl.combine != 0 || pl.v_slices != 1 || FETCH == kFetchLds))
    return da::fail(DA_ERR_ARG, "two-wave launches take K/V through registers, one V slice and no in-launch merge");
  if (pl.kv_nontemporal != 0 && pl.kv_nontemporal != 1)
    return da::fail(DA_ERR_ARG, "plan asks for K/V cache hint %d", pl.kv_nontemporal);
  const bool paged = prm.block_table != nullptr, scheduled = prm.work != nullptr;
  const void* fn = pl.kv_nontemporal ? pick_kernel<true>(paged, scheduled, NT, FETCH, pl.v_slices, W)
                                     : pick_kernel<false>(paged, scheduled, NT, FETCH, pl.v_slices, W);
  if (!fn)
    return da::fail(DA_ERR_ARG, "plan asks for K/V fetch mode %d with %d V slices and %d waves", FETCH, pl.v_slices, W);
  int cus = 0, is950 = 0, lds = 0;
  int rc = query_device(&cus, &is950, &lds);
  if (rc) return rc;
  int smem = smem_bytes(W, NT, FETCH);
  // one workgroup per CU at a time: ask for more than half of a CU's LDS
  // (a workgroup may use all of it, so the request still fits)
  if (pl.wg_per_cu == 1 && smem <= lds / 2) smem = lds / 2 + 1024 <= lds ? lds / 2 + 1024 : lds;
  if (smem > lds) return da::fail(DA_ERR_UNSUPPORTED, "workgroup needs %d bytes of LDS, device allows %d", smem, lds);
  void* args[] = {const_cast<Params*>(&prm)};
  hipError_t e = hipLaunchKernel(fn, dim3(pl.grid), dim3(64 * W), args, smem, stream);
  if (e != hipSuccess) return da::fail(DA_ERR_HIP, "split partial launch: %s", hipGetErrorString(e));
  return DA_OK;
}

int launch_combine(const float* o_part, const float* m_part, const float* l_part, uint16_t* out, float* lse,
                   int s, int64_t rows, hipStream_t stream, const int32_t* seqs = nullptr, int H_Q = 1) {
  const int grid = (int)((rows + 3) / 4);
  Div div_hq = make_div((uint32_t)H_Q);
  void* args[] = {&o_part, &m_part, &l_part, &out, &lse, &s, &rows, &seqs, &H_Q, &div_hq};
  const void* fn = seqs ? reinterpret_cast<const void*>(&split_combine_kernel<true>)
                        : reinterpret_cast<const void*>(&split_combine_kernel<false>);
  hipError_t e = hipLaunchKernel(fn, dim3(grid), dim3(256), args, 0, stream);
  if (e != hipSuccess) return da::fail(DA_ERR_HIP, "combine launch: %s", hipGetErrorString(e));
  return DA_OK;
}

// Shape and plan fields of the kernel arguments (the K/V layout fields are
// set by the caller).
void fill_params(Params& p, int B, int H_Q, int H_KV, int L_K_max, float scale, const da_plan& pl) {
  p.B = B;
  p.H_Q = H_Q;
  p.H_KV = H_KV;
  p.L_K = L_K_max;
  p.g = H_Q / H_KV;
  p.hpt = pl.heads_per_tile;
  p.tiles_per_seq = H_Q / pl.heads_per_tile;
  p.tiles = pl.tiles;
  p.s = pl.num_splits;
  p.div_s = make_div((uint32_t)p.s);
  p.div_tps = make_div((uint32_t)p.tiles_per_seq);
  p.div_g = make_div((uint32_t)p.g);
  p.xcd_group = pl.heads_per_tile < p.g ? 1 : 0;  // several workgroups read each KV head
  const float sigma = scale > 0.f ? scale : 1.0f / sqrtf((float)D);
  p.scale_log2 = sigma * kLog2e;
}

Params make_params(const void* q, const void* k, const void* v, const int32_t* cu, int B, int H_Q, int H_KV,
                   int L_K_max, float scale, const da_plan& pl) {
  Params p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.cu = cu;
  fill_params(p, B, H_Q, H_KV, L_K_max, scale, pl);
  return p;
}

// What the decode entry points share once their inputs are checked: the
// plan, the workspace check, then one launch (s == 1) or the chunk states
// followed by the log-sum-exp combine.  `p` carries the K/V layout.
// A plan made beforehand must describe a launch of this shape.
int check_plan(const da_plan* pl, int B, int H_Q, int H_KV) {
  if (!pl) return da::fail(DA_ERR_NULL, "plan is NULL");
  const int hpt = pl->heads_per_tile;
  if (pl->num_splits < 1 || pl->num_splits > DA_MAX_SPLITS || !da::heads_per_tile_valid(H_Q, H_KV, pl->pack_gqa, hpt) ||
      (int64_t)pl->tiles != (int64_t)B * (H_Q / hpt) ||
      (int64_t)pl->grid != da::launch_grid((int64_t)pl->tiles * pl->num_splits, pl->v_slices) ||
      !da::group_waves_valid(*pl) || pl->kv_fetch < 0 || pl->kv_fetch > 2 || pl->kv_nontemporal < 0 ||
      pl->kv_nontemporal > 1 || pl->num_cus < 1 || !da::v_slices_valid(H_Q, H_KV, *pl) || pl->combine < 0 ||
      pl->combine > 1 || (pl->combine == 1 && (pl->num_splits < 2 || pl->tiles > da::kMaxArrivalTiles)) ||
      pl->wg_per_cu < 0 || pl->wg_per_cu > 1)
    return da::fail(DA_ERR_ARG, "plan does not describe a launch of B=%d H_Q=%d H_KV=%d", B, H_Q, H_KV);
  return DA_OK;
}

// `given`: a plan made beforehand (checked), run as it is; NULL: plan here
// from (num_splits, pack_gqa) with the MI355X policy.
int run_decode(Params p, int B, int H_Q, int H_KV, int L_K_max, int d, float softmax_scale, int num_splits,
               int pack_gqa, void* out, float* lse_out, void* workspace, size_t workspace_bytes, void* stream,
               const da_plan* given = nullptr) {
  if (!out) return da::fail(DA_ERR_NULL, "out must be non-NULL");
  if (!aligned(out, 16)) return da::fail(DA_ERR_ALIGN, "out must be 16-byte aligned");
  if (lse_out && !aligned(lse_out, 4)) return da::fail(DA_ERR_ALIGN, "lse_out must be 4-byte aligned");
  if (num_splits > DA_MAX_SPLITS)
    return da::fail(DA_ERR_SPLITS, "num_splits=%d exceeds %d", num_splits, DA_MAX_SPLITS);
  if (pack_gqa < -1 || pack_gqa > 2) return da::fail(DA_ERR_ARG, "pack_gqa=%d not in {-1,0,1,2}", pack_gqa);
  if (workspace && !aligned(workspace, 16)) return da::fail(DA_ERR_ALIGN, "workspace must be 16-byte aligned");

  // A forced split count fixes the workspace need before any device access.
  // Every split call needs the counter region too, so that no call's chunk
  // states reach the counters another call on the same buffer relies on.
  auto check_workspace = [&](int s) {
    if (s <= 1) return (int)DA_OK;
    const size_t need = da::workspace_layout(B, H_Q, d, s).total;
    if (!workspace || workspace_bytes < need)
      return da::fail(DA_ERR_WORKSPACE, "num_splits=%d needs %zu workspace bytes, got %zu", s, need,
                      workspace ? workspace_bytes : (size_t)0);
    return check_state_size(B, H_Q, s);
  };
  int rc = check_workspace(given ? given->num_splits : num_splits);
  if (rc) return rc;
  int cus = 0;
  rc = ensure_gfx950(&cus);
  if (rc) return rc;
  da_plan pl;
  if (given) {
    pl = *given;
  } else {
    rc = da::plan(B, H_Q, H_KV, L_K_max, d, num_splits, pack_gqa, cus, 0, DA_POLICY_MI355X, &pl);
    if (rc) return rc;
    if (p.cu || p.seq_lens) da::four_waves(&pl, L_K_max);  // lengths known only on the device
  }
  const int s = pl.num_splits;
  const bool fused = s > 1 && pl.combine == 1;
  rc = check_workspace(s);
  if (rc) return rc;
  const da::WorkspaceLayout wl = da::workspace_layout(B, H_Q, d, s);

  fill_params(p, B, H_Q, H_KV, L_K_max, softmax_scale, pl);
  if (s == 1) {
    p.mode = kDirect;
    p.out = static_cast<uint16_t*>(out);
    p.lse = lse_out;
    return launch_partial(p, pl, static_cast<hipStream_t>(stream));
  }
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  p.mode = fused ? kFused : kPartials;
  p.o_part = reinterpret_cast<float*>(ws + wl.o_off);
  p.m_part = reinterpret_cast<float*>(ws + wl.m_off);
  p.l_part = reinterpret_cast<float*>(ws + wl.l_off);
  if (fused) {
    // one launch: the last workgroup of each tile merges its chunk states
    p.arrivals = reinterpret_cast<uint32_t*>(ws + da::arrival_offset(workspace_bytes));
    p.out = static_cast<uint16_t*>(out);
    p.lse = lse_out;
    return launch_partial(p, pl, static_cast<hipStream_t>(stream));
  }
  rc = launch_partial(p, pl, static_cast<hipStream_t>(stream));
  if (rc) return rc;
  return launch_combine(p.o_part, p.m_part, p.l_part, static_cast<uint16_t*>(out), lse_out, s, (int64_t)B * H_Q,
                        static_cast<hipStream_t>(stream));
}

// Checks of the paged layout arguments (shape already checked).
int check_paged(const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
                const int32_t* seq_lens, int B, int page_size, int max_pages, int num_pages, int L_K_max) {
  if (page_size < kKeysPerTile || page_size % kKeysPerTile != 0 || page_size > (1 << 20))
    return da::fail(DA_ERR_UNSUPPORTED, "page_size=%d must be a multiple of %d (at most 2^20)", page_size,
                    kKeysPerTile);
  if (max_pages < 1 || num_pages < 0 || (int64_t)max_pages * page_size < L_K_max)
    return da::fail(DA_ERR_SHAPE, "max_pages=%d pages of %d keys cannot hold L_K_max=%d (num_pages=%d)",
                    max_pages, page_size, L_K_max, num_pages);
  if ((int64_t)B * max_pages >= ((int64_t)1 << 31))
    return da::fail(DA_ERR_SHAPE, "block table of B*max_pages=%lld entries is too large",
                    (long long)B * max_pages);
  if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
    return da::fail(DA_ERR_ALIGN, "q, k_cache and v_cache must be 16-byte aligned");
  if (!aligned(block_table, 4) || !aligned(seq_lens, 4))
    return da::fail(DA_ERR_ALIGN, "block_table and seq_lens must be 4-byte aligned");
  return DA_OK;
}

// Shape, pointer and layout checks of the paged entry points.
int check_paged_inputs(const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
                       const int32_t* seq_lens, int B, int H_Q, int H_KV, int page_size, int max_pages,
                       int num_pages, int L_K_max, int d) {
  int rc = da::check_shape(B, H_Q, H_KV, L_K_max, d);
  if (!q) return da::fail(DA_ERR_NULL, "q must be non-NULL");
  if (!block_table || !seq_lens) return da::fail(DA_ERR_NULL, "block_table and seq_lens must be non-NULL");
  // With L_K_max == 0 no key is ever read, so empty pools may be NULL.
  if ((!k_cache || !v_cache) && !(rc == DA_OK && L_K_max == 0))
    return da::fail(DA_ERR_NULL, "k_cache and v_cache must be non-NULL");
  if (rc) return rc;
  return check_paged(q, k_cache, v_cache, block_table, seq_lens, B, page_size, max_pages, num_pages, L_K_max);
}

void set_paged(Params& p, const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
               const int32_t* seq_lens, int page_size, int max_pages, int num_pages) {
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_cache);
  p.v = static_cast<const uint16_t*>(v_cache);
  p.block_table = block_table;
  p.seq_lens = seq_lens;
  p.page_size = page_size;
  p.div_page = make_div((uint32_t)page_size);
  p.max_pages = max_pages;
  p.num_pages = num_pages;
}

// ---------------------------------------------------------------- no-allocation scratch

// Device memory for da_decode_attn_noalloc: one call's chunk states (up to
// DA_NOALLOC_STATE_BYTES) followed by the arrival-counter region, a file-scope
// array that each device holds from module load until the process ends.  In
// host code its name only stands in for the symbol: the device address comes
// from hipGetSymbolAddress, once per device, and only that address is used.
constexpr size_t kScratchBytes = (size_t)DA_NOALLOC_STATE_BYTES + DA_ARRIVAL_BYTES;

__global__ void __launch_bounds__(256) zero_words(uint32_t* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

std::atomic<unsigned char*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// The current device's address of `scratch`.  The first call on a device
// takes it with hipGetSymbolAddress and clears the arrival counters (they
// must start at zero) with a kernel on `stream`, not a memset, so that the
// first call may be captured in a graph.
int scratch_address(hipStream_t stream, unsigned char** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return da::fail(DA_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return da::fail(DA_ERR_UNSUPPORTED, "device index %d", dev);
  unsigned char* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (!ptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ptr = g_scratch[dev].load(std::memory_order_acquire);
    if (!ptr) {
      void* addr = nullptr;
      e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !addr)
        return da::fail(DA_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      uint32_t* counters = reinterpret_cast<uint32_t*>(static_cast<unsigned char*>(addr) +
                                                       da::arrival_offset(kScratchBytes));
      int words = DA_ARRIVAL_BYTES / 4;
      void* args[] = {&counters, &words};
      e = hipLaunchKernel(reinterpret_cast<const void*>(&zero_words), dim3(64), dim3(256), args, 0, stream);
      if (e != hipSuccess) return da::fail(DA_ERR_HIP, "scratch counter clear: %s", hipGetErrorString(e));
      ptr = static_cast<unsigned char*>(addr);
      g_scratch[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return DA_OK;
}

}  // namespace

extern "C" {

int da_device_info(int* num_cus, int* is_gfx950) {
  if (!num_cus || !is_gfx950) return da::fail(DA_ERR_NULL, "output pointers must be non-NULL");
  return query_device(num_cus, is_gfx950);
}

int da_decode_attn(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k, void* out,
                   float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d, float softmax_scale,
                   int num_splits, int pack_gqa, void* workspace, size_t workspace_bytes, void* stream) {
  da::clear_error();
  int rc = check_inputs(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  Params p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.cu = cu_seqlens_k;
  return run_decode(p, B, H_Q, H_KV, L_K_max, d, softmax_scale, num_splits, pack_gqa, out, lse_out, workspace,
                    workspace_bytes, stream);
}

int da_decode_attn_planned(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k, void* out,
                           float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d, float softmax_scale,
                           const da_plan* plan, void* workspace, size_t workspace_bytes, void* stream) {
  da::clear_error();
  int rc = check_inputs(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  rc = check_plan(plan, B, H_Q, H_KV);
  if (rc) return rc;
  Params p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.cu = cu_seqlens_k;
  return run_decode(p, B, H_Q, H_KV, L_K_max, d, softmax_scale, plan->num_splits, plan->pack_gqa, out, lse_out,
                    workspace, workspace_bytes, stream, plan);
}

int da_decode_attn_noalloc(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k, void* out,
                           float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d, float softmax_scale,
                           int num_splits, int pack_gqa, void* stream) {
  da::clear_error();
  int rc = check_inputs(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  if (!out) return da::fail(DA_ERR_NULL, "out must be non-NULL");
  if (!aligned(out, 16)) return da::fail(DA_ERR_ALIGN, "out must be 16-byte aligned");
  if (lse_out && !aligned(lse_out, 4)) return da::fail(DA_ERR_ALIGN, "lse_out must be 4-byte aligned");
  if (num_splits > DA_MAX_SPLITS)
    return da::fail(DA_ERR_SPLITS, "num_splits=%d exceeds %d", num_splits, DA_MAX_SPLITS);
  if (pack_gqa < -1 || pack_gqa > 2) return da::fail(DA_ERR_ARG, "pack_gqa=%d not in {-1,0,1,2}", pack_gqa);
  auto fits = [&](int s) {
    const size_t need = s > 1 ? da::workspace_layout(B, H_Q, d, s).total : 0;
    if (need > kScratchBytes)
      return da::fail(DA_ERR_WORKSPACE,
                      "num_splits=%d needs %zu bytes of chunk state and counters; the no-allocation scratch "
                      "holds %zu",
                      s, need, kScratchBytes);
    return (int)DA_OK;
  };
  rc = fits(num_splits);  // a forced split count is known before any device access
  if (rc) return rc;
  int cus = 0;
  rc = ensure_gfx950(&cus);
  if (rc) return rc;
  da_plan pl;
  rc = da::plan(B, H_Q, H_KV, L_K_max, d, num_splits, pack_gqa, cus, 0, DA_POLICY_MI355X, &pl);
  if (rc) return rc;
  if (cu_seqlens_k) da::four_waves(&pl, L_K_max);  // lengths known only on the device
  rc = fits(pl.num_splits);
  if (rc) return rc;
  unsigned char* ws = nullptr;
  if (pl.num_splits > 1) {
    rc = scratch_address(static_cast<hipStream_t>(stream), &ws);
    if (rc) return rc;
  }
  Params p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.cu = cu_seqlens_k;
  return run_decode(p, B, H_Q, H_KV, L_K_max, d, softmax_scale, pl.num_splits, pl.pack_gqa, out, lse_out, ws,
                    ws ? kScratchBytes : 0, stream, &pl);
}

int da_decode_attn_paged(const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
                         const int32_t* seq_lens, void* out, float* lse_out, int B, int H_Q, int H_KV,
                         int page_size, int max_pages, int num_pages, int L_K_max, int d, float softmax_scale,
                         int num_splits, int pack_gqa, void* workspace, size_t workspace_bytes, void* stream) {
  da::clear_error();
  int rc = check_paged_inputs(q, k_cache, v_cache, block_table, seq_lens, B, H_Q, H_KV, page_size, max_pages,
                              num_pages, L_K_max, d);
  if (rc) return rc;
  Params p{};
  set_paged(p, q, k_cache, v_cache, block_table, seq_lens, page_size, max_pages, num_pages);
  return run_decode(p, B, H_Q, H_KV, L_K_max, d, softmax_scale, num_splits, pack_gqa, out, lse_out, workspace,
                    workspace_bytes, stream);
}

int da_decode_attn_paged_planned(const void* q, const void* k_cache, const void* v_cache,
                                 const int32_t* block_table, const int32_t* seq_lens, void* out, float* lse_out,
                                 int B, int H_Q, int H_KV, int page_size, int max_pages, int num_pages, int L_K_max,
                                 int d, float softmax_scale, const da_plan* plan, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  da::clear_error();
  int rc = check_paged_inputs(q, k_cache, v_cache, block_table, seq_lens, B, H_Q, H_KV, page_size, max_pages,
                              num_pages, L_K_max, d);
  if (rc) return rc;
  rc = check_plan(plan, B, H_Q, H_KV);
  if (rc) return rc;
  Params p{};
  set_paged(p, q, k_cache, v_cache, block_table, seq_lens, page_size, max_pages, num_pages);
  return run_decode(p, B, H_Q, H_KV, L_K_max, d, softmax_scale, plan->num_splits, plan->pack_gqa, out, lse_out,
                    workspace, workspace_bytes, stream, plan);
}

int da_decode_attn_scheduled(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k,
                             const int32_t* block_table, const int32_t* seq_lens, int page_size, int max_pages,
                             int num_pages, void* out, float* lse_out, int d, float softmax_scale,
                             const da_schedule* sched, const void* meta_dev, void* workspace,
                             size_t workspace_bytes, void* stream) {
  da::clear_error();
  if (!sched) return da::fail(DA_ERR_NULL, "sched must be non-NULL");
  const int B = sched->B, H_Q = sched->H_Q, H_KV = sched->H_KV, L_K_max = sched->L_K_max;
  int rc = block_table ? da::check_shape(B, H_Q, H_KV, L_K_max, d)
                       : check_inputs(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  if (block_table) {
    if (!q) return da::fail(DA_ERR_NULL, "q must be non-NULL");
    if (!seq_lens) return da::fail(DA_ERR_NULL, "seq_lens must be non-NULL with a block table");
    if ((!k || !v) && L_K_max != 0) return da::fail(DA_ERR_NULL, "k_cache and v_cache must be non-NULL");
    rc = check_paged(q, k, v, block_table, seq_lens, B, page_size, max_pages, num_pages, L_K_max);
    if (rc) return rc;
  }
  // the schedule must describe a launch of this shape
  const int hpt = sched->heads_per_tile;
  if (!da::heads_per_tile_valid(H_Q, H_KV, sched->pack_gqa, hpt) ||
      sched->tiles != B * (H_Q / hpt) || sched->num_items < sched->tiles ||
      (int64_t)sched->num_items > (int64_t)sched->tiles * DA_MAX_SPLITS || sched->max_splits < 1 ||
      sched->max_splits > DA_MAX_SPLITS || sched->state_rows < 0 || sched->kv_fetch < 0 || sched->kv_fetch > 2 ||
      sched->kv_nontemporal < 0 || sched->kv_nontemporal > 1 ||
      (int64_t)sched->seq_offset != (int64_t)sched->num_items * 16 ||
      (sched->max_splits > 1) != (sched->state_rows > 0) || sched->combine < 0 || sched->combine > 1 ||
      (sched->combine == 1 && (sched->state_rows == 0 || sched->tiles > da::kMaxArrivalTiles)))
    return da::fail(DA_ERR_ARG, "schedule does not describe a launch of B=%d H_Q=%d H_KV=%d", B, H_Q, H_KV);
  if (!meta_dev) return da::fail(DA_ERR_NULL, "meta_dev must be non-NULL");
  if (!aligned(meta_dev, 16)) return da::fail(DA_ERR_ALIGN, "meta_dev must be 16-byte aligned");
  if (!out) return da::fail(DA_ERR_NULL, "out must be non-NULL");
  if (!aligned(out, 16)) return da::fail(DA_ERR_ALIGN, "out must be 16-byte aligned");
  if (lse_out && !aligned(lse_out, 4)) return da::fail(DA_ERR_ALIGN, "lse_out must be 4-byte aligned");
  const size_t need = da_schedule_workspace_bytes(sched);
  if (need) {
    if (!workspace || workspace_bytes < need)
      return da::fail(DA_ERR_WORKSPACE, "schedule needs %zu workspace bytes, got %zu", need,
                      workspace ? workspace_bytes : (size_t)0);
    if (!aligned(workspace, 16)) return da::fail(DA_ERR_ALIGN, "workspace must be 16-byte aligned");
  }
  int cus = 0;
  rc = ensure_gfx950(&cus);
  if (rc) return rc;

  Params p{};
  if (block_table) {
    set_paged(p, q, k, v, block_table, seq_lens, page_size, max_pages, num_pages);
  } else {
    p.q = static_cast<const uint16_t*>(q);
    p.k = static_cast<const uint16_t*>(k);
    p.v = static_cast<const uint16_t*>(v);
    p.cu = cu_seqlens_k;
  }
  da_plan pl{};
  pl.num_splits = 1;
  pl.pack_gqa = sched->pack_gqa;
  pl.heads_per_tile = hpt;
  pl.tiles = sched->tiles;
  pl.grid = sched->num_items;
  pl.num_cus = sched->num_cus;
  pl.group_waves = 4;
  pl.kv_fetch = sched->kv_fetch;
  pl.kv_nontemporal = sched->kv_nontemporal;
  pl.v_slices = 1;
  pl.combine = 0;
  fill_params(p, B, H_Q, H_KV, L_K_max, softmax_scale, pl);
  p.xcd_group = 0;  // the schedule orders its workgroups itself
  p.work = static_cast<const int32_t*>(meta_dev);
  p.state_rows = sched->state_rows;
  p.mode = sched->combine ? kFused : kPartials;
  p.out = static_cast<uint16_t*>(out);
  p.lse = lse_out;
  const int32_t* seqs =
      reinterpret_cast<const int32_t*>(static_cast<const unsigned char*>(meta_dev) + sched->seq_offset);
  p.seqs = seqs;
  if (need) {
    const da::WorkspaceLayout wl = da::workspace_layout(sched->state_rows, H_Q, D, 1);
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    p.o_part = reinterpret_cast<float*>(ws + wl.o_off);
    p.m_part = reinterpret_cast<float*>(ws + wl.m_off);
    p.l_part = reinterpret_cast<float*>(ws + wl.l_off);
    // the arrival counters: the fixed region at the end of the caller's buffer
    p.arrivals = reinterpret_cast<uint32_t*>(ws + da::arrival_offset(workspace_bytes));
  }
  rc = launch_partial(p, pl, static_cast<hipStream_t>(stream));
  if (rc || !need || sched->combine) return rc;
  return launch_combine(p.o_part, p.m_part, p.l_part, static_cast<uint16_t*>(out), lse_out, sched->max_splits,
                        (int64_t)B * H_Q, static_cast<hipStream_t>(stream), seqs, H_Q);
}

int da_split_partials(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k, float* o_part,
                      float* m_part, float* l_part, int B, int H_Q, int H_KV, int L_K_max, int d,
                      float softmax_scale, int num_splits, int pack_gqa, void* stream) {
  da::clear_error();
  int rc = check_inputs(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, d);
  if (rc) return rc;
  if (!o_part || !m_part || !l_part) return da::fail(DA_ERR_NULL, "o_part, m_part and l_part must be non-NULL");
  if (!aligned(o_part, 16) || !aligned(m_part, 4) || !aligned(l_part, 4))
    return da::fail(DA_ERR_ALIGN, "o_part must be 16-byte and m_part/l_part 4-byte aligned");
  if (num_splits < 1 || num_splits > DA_MAX_SPLITS)
    return da::fail(DA_ERR_SPLITS, "num_splits=%d not in [1, %d]", num_splits, DA_MAX_SPLITS);
  if (pack_gqa < 0 || pack_gqa > 2) return da::fail(DA_ERR_ARG, "pack_gqa=%d not in {0,1,2}", pack_gqa);
  rc = check_state_size(B, H_Q, num_splits);
  if (rc) return rc;
  int cus = 0;
  rc = ensure_gfx950(&cus);
  if (rc) return rc;
  da_plan pl;
  rc = da::plan(B, H_Q, H_KV, L_K_max, d, num_splits, pack_gqa, cus, 0, DA_POLICY_MI355X, &pl);
  if (rc) return rc;
  if (cu_seqlens_k) da::four_waves(&pl, L_K_max);  // lengths known only on the device
  Params p = make_params(q, k, v, cu_seqlens_k, B, H_Q, H_KV, L_K_max, softmax_scale, pl);
  p.mode = kPartials;
  p.o_part = o_part;
  p.m_part = m_part;
  p.l_part = l_part;
  return launch_partial(p, pl, static_cast<hipStream_t>(stream));
}

int da_combine_splits(const float* o_part, const float* m_part, const float* l_part, void* out, float* lse_out,
                      int num_splits, int B, int H_Q, int d, void* stream) {
  da::clear_error();
  if (!o_part || !m_part || !l_part || !out)
    return da::fail(DA_ERR_NULL, "o_part, m_part, l_part and out must be non-NULL");
  if (d != D) return da::fail(DA_ERR_UNSUPPORTED, "head dim %d unsupported (only %d)", d, D);
  if (B <= 0 || H_Q <= 0) return da::fail(DA_ERR_SHAPE, "B=%d H_Q=%d must be positive", B, H_Q);
  if (num_splits < 1 || num_splits > DA_MAX_SPLITS)
    return da::fail(DA_ERR_SPLITS, "num_splits=%d not in [1, %d]", num_splits, DA_MAX_SPLITS);
  if (!aligned(o_part, 8) || !aligned(m_part, 4) || !aligned(l_part, 4) || !aligned(out, 4) ||
      (lse_out && !aligned(lse_out, 4)))
    return da::fail(DA_ERR_ALIGN, "misaligned combine operand");
  int rc = check_state_size(B, H_Q, num_splits);
  if (rc) return rc;
  int cus = 0;
  rc = ensure_gfx950(&cus);
  if (rc) return rc;
  return launch_combine(o_part, m_part, l_part, static_cast<uint16_t*>(out), lse_out, num_splits, (int64_t)B * H_Q,
                        static_cast<hipStream_t>(stream));
}

}  // extern "C"
