/*
 * decode_attn.h - split-KV single-query decode attention on MI355X (gfx950).
 *
 * The operation (paper: Sections 2.1, 2.2, 3.1, 5.1): one decode step
 * (L_Q = 1) of softmax attention for Batch sequences, H_Q query heads that
 * share H_KV key/value heads (MQA when H_KV = 1, GQA otherwise; query head h
 * reads KV head h / (H_Q / H_KV)), head dimension D, over a KV cache of L_K
 * keys per sequence.  The sequence dimension is cut into num_splits chunks;
 * each chunk yields a partial softmax state (running max m, sum l and
 * unnormalised output Otilde) and a log-sum-exp combine merges them.  The
 * scheduling knobs (num_splits, pack_gqa, cu_margin) never change the
 * mathematical result (Section 3.1), only rounding order.
 *
 * Conventions for every entry point:
 *   - Tensors are dense, row-major, in device memory (hipMalloc'd or torch
 *     CUDA tensors), and owned by the caller.  The library never allocates or
 *     frees device memory and keeps no pointer after a call returns.
 *   - bf16 tensors are passed as raw 16-bit storage (IEEE bfloat16 bits).
 *   - Device pointers to bf16 data, partial outputs and the workspace must be
 *     16-byte aligned; fp32 lse/m/l pointers 4-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Work is
 *     enqueued asynchronously with no allocation, no host synchronisation and
 *     no device-to-host read, so calls can be captured in a HIP graph.
 *   - Return value 0 (DA_OK) or a negative da_status.  All argument checks
 *     run before any HIP call, so a rejected call touches no device state.
 *     Kernel faults surface at the caller's next synchronisation.
 *     da_last_error() gives a message for the calling thread's last failure.
 *   - Only D = 128 and only gfx950 devices are supported.
 */
#ifndef DECODE_ATTN_H
#define DECODE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DA_HEAD_DIM 128
#define DA_MAX_SPLITS 64
/* K/V bytes per call above which the planner marks K/V loads nontemporal:
 * MI355X's 256 MiB MALL plus 8 x 4 MiB of L2.  A call reading more cannot
 * find its K/V resident on the next call, and streaming hints then raise
 * the sustained HBM read rate. */
#define DA_RESIDENT_BYTES (288ull << 20)
/* Bytes at the end of a workspace that hold the arrival counters of
 * single-launch merges (da_plan.combine == 1): one uint32 per tile, 256 bytes
 * apart (atomics on one cache line are serialised, so counters of different
 * tiles must not share one), so such a plan has at most DA_ARRIVAL_BYTES /
 * 256 = 4096 tiles. */
#define DA_ARRIVAL_BYTES (1 << 20)
#define DA_ARRIVAL_STRIDE 256
/* Chunk-state bytes the scratch of da_decode_attn_noalloc holds (per device,
 * for the life of the process, with DA_ARRIVAL_BYTES of counters after it). */
#define DA_NOALLOC_STATE_BYTES (32 << 20)

typedef enum da_status {
  DA_OK = 0,
  DA_ERR_NULL = -1,        /* a required pointer is NULL */
  DA_ERR_SHAPE = -2,       /* B, H_Q, H_KV <= 0, H_Q % H_KV != 0, L_K_max < 0, sizes too large */
  DA_ERR_UNSUPPORTED = -3, /* D != 128, or the current device is not gfx950 */
  DA_ERR_SPLITS = -4,      /* num_splits > DA_MAX_SPLITS */
  DA_ERR_ALIGN = -5,       /* a pointer violates the alignment rules above */
  DA_ERR_WORKSPACE = -6,   /* workspace missing or smaller than da_workspace_bytes() */
  DA_ERR_HIP = -7,         /* a HIP runtime call failed (device query or launch) */
  DA_ERR_ARG = -8          /* another invalid argument (pack_gqa, policy, cu_margin, ...) */
} da_status;

typedef enum da_policy {
  DA_POLICY_MI355X = 0, /* CU-aware cost model over num_splits in [1, 64] (default) */
  DA_POLICY_PAPER = 1,  /* the paper's rule (Section 4): 128-key blocks, Batch*H_KV tiles;
                           at most 3 blocks -> 1; 4 blocks -> 1 with >= 4 tiles, else 3;
                           longer contexts fall through to the MI355X cost model */
  DA_POLICY_EVOLVED = 2, /* the evolved single-batch setting the paper's search found (Section 3,
                           Fig. 1): batch 1 -> 12 splits, 16 below 256 keys, GQA packing on;
                           larger batches use the MI355X cost model */
  DA_POLICY_STREAMED = 3, /* the MI355X cost model calibrated with K/V read from HBM on every call
                            (no cache reuse between calls, as in a decode step through all
                            layers); it splits earlier, e.g. 4 splits at B=1, H_KV=8, L_K=512,
                            and marks K/V loads nontemporal at any size where one workgroup
                            reads each key.  Its plans run through da_decode_attn_planned. */
  DA_POLICY_TABLE = 4,   /* configuration-specific split table learned offline (the paper's future
                            work, Sections 3.3, 4.1 and 4.2: split counts per configuration instead
                            of one rule): a shape (B, H_Q, H_KV, L_K_max) that the calibration
                            sweep with K/V resident timed gets the launch measured fastest on it
                            (split count, tile width, V slices, merge; a launch with fewer splits
                            within 1% of it preferred); every other shape, a forced num_splits,
                            pack_gqa 0 or 2, or a CU count other than the sweep's (after
                            cu_margin) is planned as DA_POLICY_MI355X plans it */
  DA_POLICY_TABLE_STREAMED = 5 /* the same over the sweep with K/V read from HBM on every call;
                            falls back to DA_POLICY_STREAMED, whose cache hint it uses */
} da_policy;

/* A launch plan: the scheduler metadata decided on the host before launch
 * (paper Section 5.1, precomputed scheduler metadata with an explicit
 * num_splits; Section 3.1, num_splits / pack_gqa / sm_margin). */
typedef struct da_plan {
  int32_t num_splits;     /* chunks per sequence, 1..64 */
  int32_t pack_gqa;       /* 0: one query head per workgroup; 1: the query heads of a KV head packed
                             into one workgroup, or for groups of more than 16 heads into tiles of at
                             most 16 when the policy's cost model predicts that faster; 2: packed,
                             the whole group in one workgroup (the paper's packing) */
  int32_t heads_per_tile; /* query heads one workgroup serves: 1 unpacked; packed, the group g = H_Q/H_KV
                             (its largest divisor <= 32 when g > 32), or with pack_gqa 1 possibly g's
                             largest divisor <= 16 */
  int32_t tiles;          /* work tiles = B * H_Q / heads_per_tile (Section 2.1: Batch x H_KV when packed) */
  int32_t grid;           /* workgroups launched: tiles * num_splits, or with V slices
                             v_slices * 8 * ceil(tiles * num_splits / 8) (a chunk's slices share an
                             XCD; the workgroups past the last chunk return at once) */
  int32_t num_cus;        /* compute units the plan was made for (after cu_margin) */
  int32_t group_waves;    /* wave64s per workgroup, each taking a contiguous part of the chunk (with 2
                             waves and H_KV <= 4, every other 32-key tile of it): 4, or 2
                             where the launch has between 3/4 and 5/4 as many workgroups as CUs (3
                             times as many for H_KV = 1 with chunks of >= 1024 keys, 4 times with
                             >= 2048), one
                             workgroup reads each key and chunks hold >= 512 keys (fewer loads
                             in flight read HBM faster there); with 2, kv_fetch is 0 or 1, v_slices
                             1 and combine 0.  Entry points that plan for themselves and read the
                             lengths on the device (cu_seqlens_k, paged seq_lens) launch four, as
                             their sequences may be far shorter than L_K_max. */
  int32_t kv_fetch;       /* how K/V tiles reach the matrix cores: 0 K straight into the operand
                             layout, V through registers to LDS (chunks of one 32-key tile per
                             wave, or two waves over rows of one KV head with at most one workgroup
                             per CU); 1 both row-contiguous into registers, then through LDS
                             (several workgroups per CU, or two waves); 2 both row-contiguous
                             straight into LDS, two tiles in flight per wave (four waves, at most
                             one workgroup per CU) */
  int32_t kv_nontemporal; /* 1: K/V loads carry the nontemporal (streaming) cache hint, chosen when
                             one call's K/V exceed DA_RESIDENT_BYTES and cannot stay in L2 and the
                             MALL between calls, and one workgroup reads each key (heads_per_tile
                             = H_Q/H_KV, v_slices = 1); 0: ordinary loads */
  int32_t v_slices;       /* workgroups that share each chunk: each computes the chunk's scores and
                             128/v_slices of the output dims (1, 2 or 4; more than 1 only with
                             kv_fetch 2 and pack_gqa 1, or pack_gqa 0 when H_Q = H_KV).  The
                             policies MI355X and STREAMED choose it where a launch keeps one
                             workgroup per CU and its K/V fit in L2 (the TABLE policies where
                             it was measured fastest); results are the same bits for every
                             value. */
  int32_t combine;        /* how num_splits > 1 chunk states are merged (the final reduction of
                             Sections 3.1 and 5.3): 0 a second kernel launch; 1 inside the split
                             launch, by the last workgroup of each tile to finish (an arrival
                             counter per tile in the workspace; no workgroup waits for another;
                             at most DA_ARRIVAL_BYTES / DA_ARRIVAL_STRIDE tiles).  Both give the same bits.  0 when
                             num_splits == 1.  The policies pick the merge their cost model
                             prices lower. */
  int32_t wg_per_cu;      /* 0: each CU holds as many of the launch's workgroups at once as its LDS
                             and registers allow; 1: one at a time (the launch asks for more than
                             half of a CU's LDS), so that a grid of a few times the CU count runs
                             in rounds of one workgroup per CU.  The policies set 1 on two-wave
                             plans of 2-4 such rounds over chunks of >= 2048 keys (4096 for four
                             rounds) with H_KV >= 2, where it keeps the chip's loads in flight at
                             the one-workgroup-per-CU level.  It changes where workgroups run,
                             never the result. */
} da_plan;

/* Choose num_splits and pack_gqa (paper Section 4: a sequence-aware split
 * policy that counts work tiles against the available compute units).
 * Policies MI355X, STREAMED and the two TABLE policies also choose the
 * packed tile width (see da_plan); PAPER and EVOLVED keep the whole group in
 * one tile.
 *   L_K_max  longest sequence in the batch (host-known, as with precomputed
 *            scheduler metadata, Section 5.1)
 *   num_cus  compute units to plan for; 0 = query the current device (one
 *            HIP attribute query, cached per device); > 0 = no device access
 *   cu_margin compute units to leave free (the paper's sm_margin, Section 3.1)
 *   policy   da_policy
 * Host-only integer/float arithmetic; deterministic for equal arguments.
 * The chosen split count keeps the chunk states below 2 GiB (they are
 * addressed with 32-bit offsets). */
int da_choose_splits(int B, int H_Q, int H_KV, int L_K_max, int d, int num_cus,
                     int cu_margin, int policy, da_plan* out);

/* The split policy's modelled time of one call, in microseconds: the cost
 * model that replaces the paper's H100 rule on MI355X (Section 4 counts work
 * tiles against the compute units; here the count of workgroups per CU, the
 * 32-key tiles each wave walks, the HBM rate and the merge of the chunk
 * states are priced with measured constants).  policy DA_POLICY_STREAMED
 * or DA_POLICY_TABLE_STREAMED uses the constants for K/V read from HBM on
 * every call, any other value those of DA_POLICY_MI355X.  heads_per_tile, v_slices and combine as in
 * da_plan; the launch is priced with four waves per workgroup (the planner
 * applies its two-wave rule to the model's choice); num_cus > 0.  Host only.  Returns -1 for arguments that describe
 * no launch (heads_per_tile not dividing H_Q, num_splits outside 1..64,
 * v_slices not 1, 2 or 4, combine not 0 or 1, non-positive sizes). */
double da_model_time(int policy, int B, int H_Q, int H_KV, int L_K, int heads_per_tile, int num_splits,
                     int v_slices, int combine, int num_cus);

/* Same as da_choose_splits with num_splits and/or pack_gqa forced
 * (num_splits <= 0 or pack_gqa == -1 leave that choice to the policy;
 * pack_gqa 0, 1 or 2 as in da_plan).
 * Fills every field of `out` for the resulting launch; num_cus as for
 * da_choose_splits.  Errors: DA_ERR_SHAPE for a shape the library does not
 * take, or a forced num_splits > 1 whose chunk states (num_splits x B x H_Q
 * x d x 4 bytes) would reach 2 GiB; DA_ERR_SPLITS for num_splits > 64;
 * DA_ERR_ARG for pack_gqa, policy, num_cus or cu_margin out of range. */
int da_make_plan(int B, int H_Q, int H_KV, int L_K_max, int d, int num_splits, int pack_gqa,
                 int num_cus, int cu_margin, int policy, da_plan* out);

/* Bytes of workspace da_decode_attn needs for num_splits chunks: the chunk
 * states (per-chunk max, sum and unnormalised output) that the paper's final
 * reduction merges (Sections 3.1 and 5.3), and the arrival counters of a
 * single-launch merge.  0 when num_splits == 1.  Layout: from offset 0,
 * Otilde fp32 [s,B,H_Q,D] | m fp32 [s,B,H_Q] | l fp32 [s,B,H_Q] (each
 * region 256-byte aligned); the arrival counters, one uint32 per tile every
 * DA_ARRIVAL_STRIDE bytes, start at (workspace_bytes - DA_ARRIVAL_BYTES)
 * rounded down to 256 bytes, i.e. in
 * the last DA_ARRIVAL_BYTES of the buffer the caller passes, whatever its
 * size.  Chunk states need no initialisation (every call writes what it
 * reads) and never reach the counter region.  The counters must be zero
 * before the first call whose plan has combine == 1 (zero the buffer once
 * when it is allocated); every such call leaves them zero, so one buffer
 * serves calls of any shape in turn.  A plan with combine == 0 does not
 * touch the counters, but every call with num_splits > 1 needs the full
 * da_workspace_bytes, so that no call's chunk states reach the counter
 * region of a buffer shared with single-launch calls. */
size_t da_workspace_bytes(int B, int H_Q, int d, int num_splits);

/* Cut points of sequence chunking: chunk i of a sequence of L keys is
 * [cuts[i], cuts[i+1]) with cuts[i] = floor(i*L/num_splits) (balanced,
 * key-granular; empty chunks when num_splits > L).  cuts has num_splits+1
 * entries, host memory.  The kernels partition each sequence this way. */
int da_split_bounds(int L, int num_splits, int32_t* cuts);

/* Decode attention, O = softmax(scale * q K^T) V per (sequence, query head)
 * (Section 2.1), computed in num_splits chunks per sequence and merged by
 * log-sum-exp (Sections 2.2, 3.1, 5.3).
 *   q            bf16 [B, H_Q, d]
 *   k, v         bf16 [B, L_K_max, H_KV, d] when cu_seqlens_k == NULL;
 *                bf16 [sum_b L_b, H_KV, d] otherwise; may be NULL when
 *                L_K_max == 0 (no key is read)
 *   cu_seqlens_k NULL (every sequence has L_K_max keys) or device int32
 *                [B+1] prefix sums: sequence b is rows [cu[b], cu[b+1]),
 *                cu[0] = 0, non-decreasing, each length <= L_K_max
 *   out          bf16 [B, H_Q, d], normalised output
 *   lse_out      NULL or fp32 [B, H_Q]: natural-log log-sum-exp of the
 *                scaled scores (-inf for an empty sequence, whose O is 0)
 *   softmax_scale <= 0 selects 1/sqrt(d)
 *   num_splits   <= 0: chosen by da_choose_splits (policy MI355X); else 1..64
 *   pack_gqa     -1: chosen by the policy; 0, 1 or 2 forced (da_plan)
 *   workspace    device memory of workspace_bytes >= da_workspace_bytes(B,
 *                H_Q, d, s) for the resolved s (unused when s == 1).  Calls
 *                that share a workspace must not overlap in time.
 * s == 1: one kernel launch.  s > 1: the split kernel writes the chunk
 * states to the workspace, and they are merged in chunk order either by the
 * combine kernel (exactly da_split_partials followed by da_combine_splits)
 * or, when the plan's combine is 1, inside the same launch by the last
 * workgroup of each tile (the workspace's arrival counters must then be
 * zero, see da_workspace_bytes).  Both merges give the same bits, and
 * results are bit-identical across runs on one device for a fixed
 * (num_splits, pack_gqa). */
int da_decode_attn(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k,
                   void* out, float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d,
                   float softmax_scale, int num_splits, int pack_gqa, void* workspace,
                   size_t workspace_bytes, void* stream);

/* Decode attention that runs a plan made beforehand instead of planning
 * again (Section 5.1: scheduler metadata precomputed on the host and
 * passed explicitly).  The plan comes from da_make_plan or da_choose_splits
 * for this B, H_Q and H_KV, with any policy and cu_margin, and may be edited
 * within its valid values. The launch uses exactly its split count, head
 * tiles, K/V fetch path, cache hint and workgroups per CU.  Other arguments and the workspace
 * need (for plan->num_splits) as in da_decode_attn.  Errors as there, plus
 * DA_ERR_NULL (plan NULL) and DA_ERR_ARG (the plan does not describe a launch
 * of this shape: num_splits outside 1..64, a heads_per_tile its pack_gqa
 * cannot produce, tiles != B*H_Q/heads_per_tile, a grid other than the one
 * the da_plan.grid comment gives for its tiles, num_splits and v_slices,
 * group_waves other than 4 or 2 (2 only with kv_fetch 0 or 1, v_slices 1 and
 * combine 0), kv_fetch outside 0..2, kv_nontemporal outside 0..1,
 * num_cus < 1, v_slices other than 1, 2 or 4, or v_slices > 1 with a
 * kv_fetch other than 2, with pack_gqa 2, or unpacked with H_Q != H_KV,
 * combine outside 0..1 or 1 with one split, wg_per_cu outside 0..1), all
 * before any device access. */
int da_decode_attn_planned(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k,
                           void* out, float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d,
                           float softmax_scale, const da_plan* plan, void* workspace,
                           size_t workspace_bytes, void* stream);

/* da_decode_attn for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * The same arguments without the workspace, the same plan (policy MI355X)
 * and the same bits as da_decode_attn for that plan.  The chunk states and
 * arrival counters of a split plan live in a fixed scratch array of
 * DA_NOALLOC_STATE_BYTES + DA_ARRIVAL_BYTES bytes that every device holds
 * from the library's load until the process ends; no call allocates or
 * frees anything.  The first call on a device looks up the array's address
 * and clears its counters with a kernel on `stream`.  Every call on a device
 * shares that array and leaves the previous call's chunk states in it:
 * calls that overlap in time on one device (other streams, other host
 * threads) race and must not be made.  Errors as for da_decode_attn, and
 * DA_ERR_WORKSPACE when the plan's chunk states exceed
 * DA_NOALLOC_STATE_BYTES (for a forced num_splits before any device
 * access), e.g. num_splits = 64 at B = 32, H_Q = 64. */
int da_decode_attn_noalloc(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k,
                           void* out, float* lse_out, int B, int H_Q, int H_KV, int L_K_max, int d,
                           float softmax_scale, int num_splits, int pack_gqa, void* stream);

/* Decode attention over a paged KV cache: the same computation as
 * da_decode_attn, with sequence b's keys held in fixed-size pages (the
 * serving layout whose per-batch scheduling metadata the paper's
 * deployment path precomputes, Section 5.1).
 *   k_cache, v_cache bf16 [num_pages, page_size, H_KV, d]: page n holds
 *                page_size consecutive keys of some sequence
 *   block_table  device int32 [B, max_pages]: key j of sequence b lives in
 *                page block_table[b*max_pages + j/page_size], row
 *                j % page_size; entries past the sequence are not read; a
 *                page id outside [0, num_pages) reads as zero keys/values
 *   seq_lens     device int32 [B]: sequence lengths, each clamped to
 *                [0, L_K_max]
 *   page_size    multiple of 32 (one 32-key tile never spans two pages)
 *   max_pages    columns of block_table; max_pages * page_size >= L_K_max
 * Chunks (and each workgroup's wave ranges) are cut at 32-key boundaries,
 * ceil(i * T / s) style over the T = ceil(L_b / 32) tiles, rather than at
 * da_split_bounds; the result does not depend on the cut.  Other arguments,
 * the workspace, error codes and launches are as for da_decode_attn. */
int da_decode_attn_paged(const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* block_table, const int32_t* seq_lens, void* out,
                         float* lse_out, int B, int H_Q, int H_KV, int page_size, int max_pages,
                         int num_pages, int L_K_max, int d, float softmax_scale, int num_splits,
                         int pack_gqa, void* workspace, size_t workspace_bytes, void* stream);

/* Paged decode attention that runs a plan made beforehand, as
 * da_decode_attn_planned does for contiguous K/V (Section 5.1: scheduler
 * metadata precomputed on the host).  Paged arguments as for
 * da_decode_attn_paged; plan, workspace and errors as for
 * da_decode_attn_planned.  This is how a STREAMED plan or one made with a
 * cu_margin reaches a paged cache with one split count for the batch. */
int da_decode_attn_paged_planned(const void* q, const void* k_cache, const void* v_cache,
                                 const int32_t* block_table, const int32_t* seq_lens, void* out,
                                 float* lse_out, int B, int H_Q, int H_KV, int page_size,
                                 int max_pages, int num_pages, int L_K_max, int d,
                                 float softmax_scale, const da_plan* plan, void* workspace,
                                 size_t workspace_bytes, void* stream);

/* Per-sequence scheduler metadata: the precomputed scheduling of Section 5.1
 * carried down to one split count per sequence, so that in a batch of mixed
 * lengths long sequences are cut into more chunks than short ones (the
 * sequence-aware rule of Section 4 applied to each sequence's own length).
 * Built on the host from host-known lengths; the caller copies the metadata
 * bytes to device memory and passes both to da_decode_attn_scheduled. */
typedef struct da_schedule {
  int32_t B, H_Q, H_KV, L_K_max; /* the shape it was made for */
  int32_t pack_gqa;              /* as in da_plan */
  int32_t heads_per_tile;        /* as in da_plan */
  int32_t tiles;                 /* head tiles = B * H_Q / heads_per_tile */
  int32_t num_items;             /* workgroups launched */
  int32_t chunk_tiles;           /* target chunk length in 32-key tiles */
  int32_t max_splits;            /* largest per-sequence split count (1..64) */
  int32_t state_rows;            /* chunk-state rows: sum of s_b over sequences with s_b > 1 */
  int32_t num_cus;               /* compute units planned for (after cu_margin) */
  int32_t kv_fetch;              /* as in da_plan */
  int32_t seq_offset;            /* byte offset of the per-sequence table in the metadata */
  int32_t meta_bytes;            /* metadata bytes written */
  int32_t kv_nontemporal;        /* as in da_plan, for the K/V of all B sequences */
  int32_t combine;               /* 1: the chunk states of each split sequence are merged inside
                                    the split launch by the last workgroup of each of its head
                                    tiles (arrival counters in the workspace, as in da_plan);
                                    0: by a second launch.  0 when no sequence is split */
} da_schedule;

/* Upper bound on the metadata bytes da_make_schedule writes for this shape
 * (every sequence at 64 chunks). */
size_t da_schedule_max_bytes(int B, int H_Q, int H_KV, int pack_gqa);

/* Build the per-sequence schedule.
 *   seq_lens   host int32 [B]: key counts, each in [0, L_K_max]
 *   pack_gqa   -1 (chosen as by the policy) or 0, 1, 2 as in da_plan
 *   num_cus    0 = query the current device, > 0 = no device access
 *   cu_margin  compute units to leave to concurrent work (Section 3.1's
 *              sm_margin): the schedule is sized for num_cus - cu_margin
 *   chunk_tiles <= 0: chosen by the MI355X cost model; > 0: every sequence
 *              is cut into ceil(T_b / chunk_tiles) chunks (at most 64), T_b
 *              = ceil(L_b / 32)
 *   meta       host buffer of meta_bytes >= the bytes needed (at most
 *              da_schedule_max_bytes); receives, 16-byte aligned:
 *                items int32x4 [num_items]: {head tile, first tile, end
 *                  tile, state row (-1: the chunk is the whole sequence and
 *                  writes the output directly)}, with the 32-key tile range
 *                  [first, end) of that workgroup's chunk; the last chunk of
 *                  each sequence has end = INT32_MAX (to the sequence end)
 *                sequences int32x2 [B] at seq_offset: {first state row or
 *                  -1, split count s_b}
 *   out        filled on success
 * Host-only; deterministic for equal arguments.  Errors: DA_ERR_NULL,
 * DA_ERR_SHAPE (a length outside [0, L_K_max]), DA_ERR_ARG (cu_margin,
 * pack_gqa), DA_ERR_WORKSPACE (meta_bytes too small; out->meta_bytes then
 * holds the size needed). */
int da_make_schedule(const int32_t* seq_lens, int B, int H_Q, int H_KV, int L_K_max, int d,
                     int pack_gqa, int num_cus, int cu_margin, int chunk_tiles, void* meta,
                     size_t meta_bytes, da_schedule* out);

/* Workspace bytes da_decode_attn_scheduled needs for `sched`: 0 when no
 * sequence is split.  Layout (256-byte aligned regions): Otilde fp32
 * [state_rows, H_Q, D] | m fp32 [state_rows, H_Q] | l fp32 [state_rows, H_Q],
 * and the DA_ARRIVAL_BYTES counter region at the end of the buffer passed,
 * as for da_decode_attn: zero before the first call, and every call leaves
 * it zero, so one zero-filled buffer serves uniform and scheduled calls. */
size_t da_schedule_workspace_bytes(const da_schedule* sched);

/* Decode attention driven by a per-sequence schedule: the same result as
 * da_decode_attn (or da_decode_attn_paged) up to rounding order.
 *   K/V layout: block_table == NULL -> contiguous (k, v, cu_seqlens_k as for
 *     da_decode_attn; page_size, max_pages, num_pages, seq_lens ignored);
 *     block_table != NULL -> paged (k, v are the page pools, with
 *     block_table, seq_lens, page_size, max_pages, num_pages as for
 *     da_decode_attn_paged; cu_seqlens_k ignored)
 *   sched      host struct from da_make_schedule for this B, H_Q, H_KV,
 *              L_K_max
 *   meta_dev   device copy of the metadata bytes (16-byte aligned).  The
 *              kernel reads the lengths on the device (cu_seqlens_k or
 *              seq_lens); where one differs from the length scheduled (up
 *              to L_K_max) every key is still read once, since chunks are
 *              clamped to the sequence and each sequence's last chunk runs
 *              to its end: only the balance changes
 *   workspace  >= da_schedule_workspace_bytes(sched)
 * One launch, or two (the combine launch when some sequence is split and
 * sched->combine is 0); no
 * allocation, graph-capturable; results bit-identical across runs for a
 * fixed schedule. */
int da_decode_attn_scheduled(const void* q, const void* k, const void* v,
                             const int32_t* cu_seqlens_k, const int32_t* block_table,
                             const int32_t* seq_lens, int page_size, int max_pages, int num_pages,
                             void* out, float* lse_out, int d, float softmax_scale,
                             const da_schedule* sched, const void* meta_dev, void* workspace,
                             size_t workspace_bytes, void* stream);

/* The split step alone: the partial softmax state of every chunk (the
 * per-chunk max, sum and unnormalised output the paper's final reduction
 * merges; Sections 3.1, 5.3).  Same inputs as da_decode_attn; num_splits
 * must be 1..64 and pack_gqa 0, 1 or 2 (no policy here).
 *   o_part fp32 [num_splits, B, H_Q, d]: sum_j exp(s_j - m_i) v_j over chunk i
 *   m_part fp32 [num_splits, B, H_Q]:    max scaled score of chunk i (natural
 *                                        log units), -inf for an empty chunk
 *   l_part fp32 [num_splits, B, H_Q]:    sum_j exp(s_j - m_i), 0 when empty
 * Chunks follow da_split_bounds.  Feeding the result to da_combine_splits
 * gives the same output as da_decode_attn up to rounding. */
int da_split_partials(const void* q, const void* k, const void* v, const int32_t* cu_seqlens_k,
                      float* o_part, float* m_part, float* l_part, int B, int H_Q, int H_KV,
                      int L_K_max, int d, float softmax_scale, int num_splits, int pack_gqa,
                      void* stream);

/* Log-sum-exp merge of num_splits partial states (the final reduction of
 * Sections 3.1 and 5.3): M = max_i m_i over non-empty chunks, w_i =
 * exp(m_i - M) (0 when l_i == 0), O = sum_i w_i Otilde_i / sum_i w_i l_i,
 * lse = M + ln(sum_i w_i l_i); summed in chunk order i = 0..s-1.
 * A row with every chunk empty gives O = 0 and lse = -inf.
 *   o_part, m_part, l_part as written by da_split_partials (any producer of
 *   that format works, e.g. partial states gathered from other devices)
 *   out bf16 [B, H_Q, d]; lse_out NULL or fp32 [B, H_Q].  One kernel launch. */
int da_combine_splits(const float* o_part, const float* m_part, const float* l_part, void* out,
                      float* lse_out, int num_splits, int B, int H_Q, int d, void* stream);

/* Compute units of the current device (hipDeviceAttributeMultiprocessorCount,
 * cached per device) and whether it is gfx950: the CU count the split policy
 * counts work tiles against (Section 4).  Errors: DA_ERR_NULL, DA_ERR_HIP. */
int da_device_info(int* num_cus, int* is_gfx950);

/* Static text for a da_status code.  No passage of the paper: library
 * infrastructure.  Never NULL; "unknown error" for a code not in da_status. */
const char* da_strerror(int code);

/* Message describing the calling thread's most recent failure ("" if none).
 * No passage of the paper: library infrastructure.  The text is owned by the
 * library and valid until the thread's next call into it. */
const char* da_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DECODE_ATTN_H */
