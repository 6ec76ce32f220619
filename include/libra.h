/*
 * libra: ragged paged-KV decode and append attention for MI355X (gfx950).
 *
 * The hot path underneath an agentic-RL rollout stage (arXiv 2606.03077): rollout is
 * autoregressive decoding that the paper calls memory- and bandwidth-bound (Sec. 1;
 * Sec. 2.1; App. A.1), over trajectories whose lengths are long-tailed (Sec. 2.2) and
 * grow when tool outputs are appended mid-trajectory (Sec. 1; Sec. 5, Phase 2 and the
 * migration steps).  The paper's engine keeps a per-request paged KV cache that can be
 * sharded along attention heads (Sec. 5, Step 2); the library keeps that head axis
 * separable in its layout.
 *
 * Conventions for every entry point
 * ---------------------------------
 * - All tensors are borrowed pointers owned by the caller.  "device" pointers must be
 *   HIP device memory of the current device; "host" pointers are ordinary host memory.
 * - Handles (libra_kv_layout, libra_plan, libra_trie) are created and destroyed by the
 *   library.  Layouts and plans are immutable after creation, except that a plan
 *   remembers (under a lock) which workspace its tables were last uploaded to, so calls
 *   on different streams with distinct workspaces and outputs may share a plan; a prefix
 *   tree grows by libra_trie_insert and must not be inserted into while another thread
 *   uses it.  A handle is destroyed only after the calls that use it were issued.
 * - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the null stream).
 *   No entry point synchronises the device or allocates device memory, except
 *   libra_xcd_read_weights (set-up) and libra_plan_destroy, which waits for the plan's
 *   own pending table upload (an event, not the device).  libra_splitkv_plan takes the
 *   plan's pinned host image of its tables and its events from a library-owned pool
 *   (allocating them only when the pool has none free), and the first plan with both
 *   single-token and chunk rows creates the device's auxiliary stream (default
 *   priority, kept until the process ends); libra_plan_destroy returns image and events
 *   to the pool.  Decode, append and upload calls allocate nothing.
 * - Host-only entry points (plan construction, cost evaluator, RolloutDP, prefix tree,
 *   routing, libra_kv_reshard_host) touch no GPU; the reshard may use up to 8 host
 *   threads for large runs.
 * - Every entry point returns a libra_status; nothing aborts, prints or throws.  On an
 *   error nothing has been enqueued, and libra_last_error() gives a per-thread message.
 * - Validation happens on the host before any launch.  Device-side contract violations
 *   (a block-table entry >= num_pages, a block table shorter than the plan's lengths)
 *   are undefined behaviour: the library does not read the block table on the host.
 *
 * Numerics: bf16 inputs, float32 accumulation, bf16 outputs rounded to nearest even,
 * log-sum-exp in float32 natural log.  Query head h reads KV head h / G with
 * G = num_q_heads / num_kv_heads (contiguous groups).
 */
#ifndef LIBRA_H_
#define LIBRA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum libra_status {
  LIBRA_OK = 0,
  LIBRA_E_INVAL = 1,        /* bad argument: null pointer, size, inconsistent plan */
  LIBRA_E_UNSUPPORTED = 2,  /* valid but not implemented: head_dim != 128, G > 16 ... */
  LIBRA_E_WORKSPACE = 3,    /* workspace smaller than libra_plan_workspace_bytes() */
  LIBRA_E_HIP = 4,          /* a HIP runtime call or kernel launch failed */
  LIBRA_E_NOMEM = 5         /* host allocation failed */
} libra_status;

enum {
  LIBRA_PAGE_SIZE = 16,     /* tokens per page */
  LIBRA_HEAD_DIM = 128,     /* channels per head */
  LIBRA_MAX_GROUP = 16,     /* largest supported num_q_heads / num_kv_heads */
  LIBRA_MAX_KV_HEADS = 1024, /* largest supported num_kv_heads (a page's K or V, all heads,
                                stays under 4 GiB of byte offsets) */
  LIBRA_UNIT_INTS = 12      /* int32 fields per plan unit */
};

enum { LIBRA_DTYPE_BF16 = 0 };
enum { LIBRA_MODE_DECODE = 0, LIBRA_MODE_APPEND = 1 };

typedef struct libra_kv_layout_s* libra_kv_layout;
typedef struct libra_plan_s* libra_plan;

/* Human-readable name of a status code (static storage). */
const char* libra_status_string(libra_status status);
/* Detail of the last error raised on the calling thread ("" if none). */
const char* libra_last_error(void);
/* Number of HIP calls this library has made, process-wide, that allocate or free device
 * or pinned host memory or create an event or a stream (hipMalloc, hipHostMalloc,
 * hipFree, hipEventCreate*, hipStreamCreate*).  Plan creation may make such calls (its
 * pinned staging image and events come from a pool that grows to the number of live
 * plans); decode and append calls with per-kernel timing off make none, which a caller
 * (or a test) can check by reading the count before and after. */
uint64_t libra_alloc_calls(void);

/* ------------------------------------------------------------------------------ */
/* Paged KV cache layout                                                           */
/* ------------------------------------------------------------------------------ */
/*
 * The cache is two caller-owned device buffers, K and V, each num_pages *
 * num_kv_heads tiles of 4096 bytes.  Tile (page, g) starts at byte
 * ((page * num_kv_heads) + g) * 4096 and holds the 16 token slots x 128 channels of
 * that page for KV head g as bf16, so the head axis stays separable per page (the
 * paper reshards KV along heads, Sec. 5, Step 2).  Inside a tile the element of
 * (slot s, channel d) sits at:
 *
 *   K: ((d / 8) * 16 + s) * 8 + d % 8
 *   V: (128 * ((s / 4) % 2) + d) * 8 + (s / 8) * 4 + s % 4
 *
 * i.e. the order in which a 64-lane wavefront consumes them as matrix-core operands:
 * a K granule (16 bytes) is one slot's 8 consecutive channels; V granule 128 h + d
 * holds channel d's slots {4h..4h+3, 8+4h..11+4h}, the 8 keys one lane of a 32x32x16
 * product takes, so one 16-byte load per lane reads 1 KiB contiguously.  Callers never address
 * elements directly: libra_kv_pack_pages / libra_kv_unpack_pages convert whole pages
 * from / to the logical format, and libra_append_attn writes new tokens.
 *
 * Logical page format (used by pack / unpack): [n_pages][num_kv_heads][16][128] bf16,
 * slot-major.  Token t of sequence b lives in page block_table[b * bt_stride + t / 16],
 * slot t % 16.
 */
typedef struct libra_kv_layout_desc {
  int64_t num_pages;     /* pages in each of k_cache / v_cache, > 0 */
  int32_t page_size;     /* must be LIBRA_PAGE_SIZE */
  int32_t num_kv_heads;  /* in [1, LIBRA_MAX_KV_HEADS] */
  int32_t head_dim;      /* must be LIBRA_HEAD_DIM */
  int32_t dtype;         /* must be LIBRA_DTYPE_BF16 */
  void* k_cache;         /* device, num_pages * num_kv_heads * 4096 bytes */
  void* v_cache;         /* device, same size */
} libra_kv_layout_desc;

/* Validates the descriptor and returns a handle (the buffers stay caller-owned). */
libra_status libra_kv_layout_create(const libra_kv_layout_desc* desc, libra_kv_layout* out);
void libra_kv_layout_destroy(libra_kv_layout layout);

/* Converts n_pages logical pages (device, [n_pages][Hkv][16][128] bf16) into the
 * layout's pages [first_page, first_page + n_pages).  k_src / v_src may be NULL to
 * skip one side.  Source and destination must not overlap. */
libra_status libra_kv_pack_pages(libra_kv_layout layout, const void* k_src, const void* v_src,
                                 int64_t first_page, int64_t n_pages, void* stream);

/* Inverse of libra_kv_pack_pages: pages [first_page, first_page + n_pages) to logical
 * format in k_dst / v_dst (device).  Used to offload or reshard a request's cache. */
libra_status libra_kv_unpack_pages(libra_kv_layout layout, void* k_dst, void* v_dst,
                                   int64_t first_page, int64_t n_pages, void* stream);

/* Copies the first seq_len tokens of each sequence out of the paged cache through the
 * block table: k_out / v_out (device) are [sum_b len_b][Hkv][128] bf16 with sequence b
 * starting at row cu_seq_lens[b].  cu_seq_lens (device, int32 [batch + 1]) is the
 * prefix sum of the lengths; max_pages bounds ceil(len_b / 16) and bt_stride >=
 * max_pages.  Bit-exact: it only moves bytes. */
libra_status libra_kv_gather(libra_kv_layout layout, const int32_t* block_table, int32_t bt_stride,
                             const int32_t* cu_seq_lens, int32_t batch, int32_t max_pages,
                             void* k_out, void* v_out, void* stream);

/* ------------------------------------------------------------------------------ */
/* Request migration: offload, head reshard, reload                                */
/* ------------------------------------------------------------------------------ */
/*
 * When a request pauses for a tool call, its KV pages are offloaded to host pinned
 * memory; while the tool runs they are resharded along the attention-head axis to the
 * target bucket's tensor-parallel degree; when the tool returns, each target GPU
 * reloads its head shard into pages of its own cache (Sec. 5, migration Steps 1-3).
 * Pages move as raw library-layout tiles, so no step re-encodes data.
 *
 * A page's tiles for all KV heads are contiguous: page p of K occupies bytes
 * [p * Hkv * 4096, (p + 1) * Hkv * 4096) of k_cache (likewise V).  A packed page run is
 * n_pages such blocks back to back.
 */

/* Gathers pages page_ids[0 .. n_pages) (device int32, n_pages <= num_pages) of the cache
 * into packed runs k_dst / v_dst of n_pages * Hkv * 4096 bytes each (either may be NULL).
 * A run is device memory, or pinned host memory (hipHostMalloc): then the kernel writes
 * it over PCIe itself, which offloads a request in one call.  Pageable host memory is
 * refused (LIBRA_E_INVAL).  Ids outside [0, num_pages) are skipped and leave their run
 * block unchanged.  Asynchronous on `stream`; the caller owns every buffer. */
libra_status libra_kv_copy_out(libra_kv_layout layout, const int32_t* page_ids, int64_t n_pages,
                               void* k_dst, void* v_dst, void* stream);

/* Scatters packed runs k_src / v_src (device or pinned host memory, as above; either may
 * be NULL) into pages page_ids[0 .. n_pages) of the cache: the reload of a request.  The
 * ids must be distinct (repeated ids race); ids outside [0, num_pages) are skipped. */
libra_status libra_kv_copy_in(libra_kv_layout layout, const int32_t* page_ids, int64_t n_pages,
                              const void* k_src, const void* v_src, void* stream);

/* Host-side reshard of packed page runs along the head axis (pure memory
 * rearrangement, no device work).  The n_src inputs hold heads_per_src heads each, in
 * head order (source shard i owns heads [i * heads_per_src, (i + 1) * heads_per_src));
 * their H = n_src * heads_per_src heads are dealt to n_dst outputs of H / n_dst
 * contiguous heads each.  A TP degree raised k-fold is (1 source, k outputs); lowered,
 * (k sources, 1 output).  All buffers are host memory of n_pages * heads * 4096 bytes
 * and must not overlap.  Returns LIBRA_E_INVAL if n_dst does not divide H. */
libra_status libra_kv_reshard_host(const void* const* src, int32_t n_src, int32_t heads_per_src,
                                   void* const* dst, int32_t n_dst, int64_t n_pages);

/* ------------------------------------------------------------------------------ */
/* Split-KV work plan (host)                                                       */
/* ------------------------------------------------------------------------------ */
/*
 * Partitions one batch step into work units so that a long-tailed batch keeps every
 * compute unit busy: the paper measures that the longest 10% of trajectories take over
 * half of rollout time (Sec. 2.2) and that stragglers set the makespan (Sec. 1).  The
 * paper gives no kernel-level rule; this one is the library's:
 *
 * 1. pages_b = ceil(L_b / 16), L_b = KV length after this step's new tokens.
 * 2. Rows with C_b = 1 query token are single rows, rows with C_b > 1 chunk rows.
 * 3. S = num_cus * units_per_cu, meant as one wave of decode workgroups (units_per_cu
 *    = workgroups resident per compute unit); R = floor(S / Hkv).
 * 4. One-wave apportionment: if there are at most R single rows, each starts with
 *    n_b = 1 and, while sum n_b < R, the single row with the largest pages_b / n_b (exact
 *    comparison, ties to the smaller b) among those that can still be split (n_b <
 *    max_splits and pages_b >= (n_b + 1) * min_split_pages) gets one more split; it
 *    stops early when none can.  This minimises the largest piece, max ceil(pages_b /
 *    n_b).  The result is used when 2 * (largest piece) * R <= 3 * sum pages_b (at most
 *    1.5 times the mean share); otherwise, or with more than R single rows, step 5.
 * 5. Chunk rule: W = sum over single rows of pages_b * Hkv; chunk = max(min_split_pages,
 *    ceil(W / S)) (min_split_pages if W = 0); n_b = min(max_splits, max(1,
 *    ceil(pages_b / chunk))).
 * 6. Split j of a single row covers pages [floor(j pages_b / n_b), floor((j+1) pages_b /
 *    n_b)), i.e. tokens [16 p0, min(16 p1, L_b)).  An empty sequence gets one empty unit.
 * 7. A chunk row is cut into query tiles of T tokens (T = q_tile, or floor(256 / G) if
 *    q_tile = 0): tile k holds new tokens [kT, min(kT + T, C_b)) and keys
 *    [0, P_b + min(kT + T, C_b)), P_b = L_b - C_b.  Tiles are not split along KV.
 * 8. Every unit is repeated for each KV head g.
 * 9. Single units come first, by descending KV tokens, ties by ascending (b, g, j).
 *    Chunk units follow, grouped per (b, g) and dealt to 8 per-XCD queues: a tile costs
 *    its key-loop steps, ceil((kv_end - kv_begin) / 64) (the kernel's time per step does
 *    not depend on the tile's query tokens), a group the sum of its tiles.  With
 *    F = ceil(total / 8), a group of cost c and m tiles is cut into n = min(m,
 *    ceil(c / F)) parts, tile i (ascending q_begin) going to part floor(S_i n / c), S_i =
 *    cost of the group's earlier tiles; empty parts are dropped.  Parts by descending
 *    cost (ties ascending (b, g, part)) go to the queue with the least accumulated cost
 *    (ties to the lowest queue); each queue then lists its parts by descending cost of
 *    their longest tile (ties ascending (b, g, part)), a part's tiles together by
 *    descending cost (ties ascending q_begin); queue 0's tiles are listed first, then
 *    queue 1's, ... (the chunk launch runs queue x's tiles on workgroups w with
 *    w % 8 = x, so the tiles of a part share an L2, and each CU takes the longest tiles
 *    first).
 * 10. Single rows with n_b > 1 own n_b float32 partial-result slots per KV head,
 *    allotted in ascending (b, g): part_base(b, g) = earlier split rows' slots + g n_b.
 * 11. The single units are placed on S slots.  The decode launch dispatches workgroup w
 *    to XCD w mod 8; when step 4 decided, all units are resident at once and workgroups
 *    w, w + num_cus, w + 2 num_cus, ... share one CU, so S = num_cus (CU slots);
 *    otherwise each XCD runs its workgroups as its CUs free up, so S = 8 (XCD queues).
 *    With n single units, slot c (0 <= c < S) holds the positions w < n with w mod S = c
 *    and has weight x_c = xcd_weight[c mod 8] (1000 for 0).  A unit costs the pages it
 *    reads, ceil(kv_end / 16) - floor(kv_begin / 16).  In step 9's order, each unit goes
 *    to the slot with room that minimises (load_c + cost) / x_c (exact cross-multiplied
 *    comparison, ties to the smaller c); the r-th unit a slot receives is listed at
 *    position c + r S.
 *
 * Unit fields (LIBRA_UNIT_INTS int32): b, g, kv_begin, kv_end, q_begin, q_end, split,
 * n_splits, part_base (-1 if unsplit), row0 (first query row of sequence b),
 * kind (0 single, 1 chunk), prior (P_b = L_b - C_b).
 * All arithmetic is exact 64-bit integer arithmetic; the table is deterministic.
 */
typedef struct libra_plan_params {
  int32_t num_cus;          /* compute units; 0 = query the current device */
  int32_t units_per_cu;     /* default 3 (decode workgroups resident per CU) */
  int32_t min_split_pages;  /* default 16 */
  int32_t max_splits;       /* default 64 */
  int32_t q_tile;           /* chunk query tile in tokens, at most floor(256 / G); 0 = that */
  int32_t xcd_weight[8];    /* step 11: relative HBM read rate of the CUs of XCD x, in
                               [1, 1000000]; 0 = 1000 (all equal when every entry is 0).
                               libra_xcd_read_weights measures it. */
} libra_plan_params;

typedef struct libra_plan_desc {
  int32_t mode;          /* LIBRA_MODE_DECODE (q_lens must be NULL) or LIBRA_MODE_APPEND */
  int32_t batch;         /* >= 0 sequences */
  int32_t num_q_heads;   /* Hq, a multiple of num_kv_heads */
  int32_t num_kv_heads;  /* Hkv */
} libra_plan_desc;

typedef struct libra_plan_info {
  int32_t n_units;          /* total units in the table */
  int32_t n_single;         /* units handled by the decode kernel */
  int32_t n_chunk;          /* units handled by the chunk kernel */
  int32_t n_partial_slots;  /* float32 partial results used by split rows */
  int64_t chunk_pages;      /* step 5's chunk size (computed even when step 4 decides) */
  int32_t q_tile;           /* step 7's tile size */
  int32_t n_rows;           /* query rows (sum C_b) */
  int32_t n_write_tiles;    /* (sequence, page) pairs an append writes */
  int32_t num_cus;          /* CUs the plan was cut for */
  int32_t n_merge_groups;   /* (sequence, KV head) pairs whose splits are merged */
  int32_t balanced;         /* 1 if step 4 set the split counts, 0 if step 5 did */
} libra_plan_info;

/* Builds the plan from host lengths.  seq_lens_host: int32 [batch], L_b >= 0 (>= C_b
 * for append).  q_lens_host: int32 [batch], C_b >= 1, for append; NULL for decode.
 * params may be NULL (defaults).  The tables are computed on the host (querying the
 * device only for num_cus = 0).  When a HIP device is visible, the plan also takes a
 * pinned host image of its tables and an upload event from the library's pool
 * (LIBRA_E_HIP if that allocation fails); without one, the plan serves inspection
 * (libra_plan_get_units / _info) and its decode / append / upload calls return
 * LIBRA_E_INVAL. */
libra_status libra_splitkv_plan(const libra_plan_desc* desc, const int32_t* seq_lens_host,
                                const int32_t* q_lens_host, const libra_plan_params* params,
                                libra_plan* out);
/* Measures the xcd_weight plan parameter on the current device.  With every CU
 * reading at once, the XCDs of one device may get unequal shares of HBM bandwidth, and a
 * decode launch then ends when the slowest XCD does.  2048 workgroups of 256 threads each
 * stream their own contiguous block of `buf` (device memory of any contents, 256-byte
 * aligned, bytes >= 1 GiB so that no block is read twice; only read) with 16-byte
 * non-temporal loads for 100 us of the device's constant clock and count the loads they
 * issue, per XCD; this runs reps + 1 times (1 <= reps <= 100), the first run not counted.
 * weights[x] (8 entries, host) = round(1000 * N_x / max_y N_y), N_x being the loads
 * issued on XCD x over the counted runs, clamped to [1, 1000]; an XCD that ran no
 * workgroup gets 0 (the plan's default).  Allocates 64 KiB of device memory for the call
 * and waits for `stream`: for set-up, not for graph capture. */
libra_status libra_xcd_read_weights(const void* buf, size_t bytes, int32_t reps,
                                    int32_t* weights, void* stream);
/* Measures the device's achievable HBM read rate, the ceiling a bandwidth-bound kernel is
 * compared with beside the vendor's peak.  `buf` (device memory of any contents, 256-byte
 * aligned, bytes >= 256 MiB, only read) is cut into 2048 contiguous blocks, one per
 * workgroup of 256 threads (8 per CU on 256 CUs), each streamed with 16-byte non-temporal
 * loads, four in flight per lane.  completion_gbps: one pass over the whole buffer timed
 * by events around the launch (ramp and tail included, as for any kernel that must finish
 * its bytes); interval_gbps: the loads issued while every workgroup reads for 100 us of
 * the device's constant clock (each workgroup re-reads the start of its block, so this
 * figure needs a buffer several times the 256 MB last-level cache, whose hits would
 * inflate it).  Each is the median of `reps` runs (1 <= reps <= 100)
 * after one warm-up run.  Allocates 64 KiB of device memory for the call and waits for
 * `stream`: for set-up and measurement, not for graph capture. */
libra_status libra_hbm_read_rate(const void* buf, size_t bytes, int32_t reps,
                                 double* interval_gbps, double* completion_gbps, void* stream);
/* Host view of the unit table (valid until libra_plan_destroy). */
libra_status libra_plan_get_units(libra_plan plan, const int32_t** units_host, int32_t* n_units);
libra_status libra_plan_get_info(libra_plan plan, libra_plan_info* info);
/* Bytes of device workspace the plan's calls need (unit, write, merge and XCD-queue tables
 * and the float32 partial results of split rows). */
size_t libra_plan_workspace_bytes(libra_plan plan);
/* Copies the plan's tables into `workspace` (device) on `stream`.  Decode / append calls
 * do this themselves unless this plan was the last one to upload to that address;
 * calling it explicitly once per batch step lets every layer's call skip it.  The
 * workspace then belongs to this plan until another plan uploads to it (plans may take
 * turns on one workspace; each call of another plan re-uploads).  Calls that share a
 * workspace must be ordered on one stream.  Memory that is freed and allocated again at
 * the same address, or written by anything but this library, no longer holds the tables:
 * call libra_plan_upload on it before the next decode / append call. */
libra_status libra_plan_upload(libra_plan plan, void* workspace, size_t ws_bytes, void* stream);
/* Waits for the plan's pending upload (if any), then frees it. */
void libra_plan_destroy(libra_plan plan);

/* ------------------------------------------------------------------------------ */
/* Attention                                                                       */
/* ------------------------------------------------------------------------------ */
/*
 * Decode: one query token per sequence attends all L_b cached tokens (the current
 * token's K/V is already in the cache).  This is the per-step operation of rollout,
 * autoregressive decoding that the paper finds bound by memory bandwidth and KV-cache
 * pressure (Sec. 1; Sec. 2.1; App. A.1), over a batch whose lengths are long-tailed
 * (Sec. 2.2).  For each query head h of sequence b:
 *   z_j = scale * <q_h, k_j>,  out = sum_j softmax(z)_j v_j,  lse = log sum_j exp(z_j)
 * over keys j in [0, L_b); L_b = 0 gives out = 0, lse = -inf.
 *
 * q, out: device bf16 [batch][num_q_heads][128].  lse: device float32
 * [batch][num_q_heads] or NULL.  block_table: device int32 [batch][bt_stride] with at
 * least ceil(L_b / 16) valid page ids per row.  The plan must be a decode plan built for
 * the same (batch, num_q_heads, num_kv_heads) and lengths; workspace: device, at least
 * libra_plan_workspace_bytes(plan) bytes, 256-byte aligned.  `scale` must be finite and
 * positive (LIBRA_E_INVAL otherwise).
 * Split rows write float32 partials; a second launch on the same stream merges them by
 * their log-sum-exps.
 *
 * HIP graphs: once the workspace holds the plan's tables (libra_plan_upload, or an
 * earlier call of the plan on that workspace), a decode or append call only enqueues
 * kernels (no allocation, host copy, memset or event), so it may be captured into a
 * HIP graph.  The graph keeps the workspace, buffers and layout pointers it was
 * captured with; while it may still be replayed, no other plan may use that workspace
 * (its upload would replace the tables the graph's kernels read).  Per-kernel timing
 * (libra_profile_enable) must be off during capture.
 */
libra_status libra_decode_attn(libra_kv_layout layout, libra_plan plan, const void* q,
                               const int32_t* block_table, int32_t bt_stride, int32_t batch,
                               int32_t num_q_heads, float scale, void* workspace, size_t ws_bytes,
                               void* out, float* lse, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): libra_decode_attn with the library's
 * static device scratch in place of a caller workspace.  Same arguments, layouts,
 * kernels and results as libra_decode_attn without `workspace` / `ws_bytes`.
 *
 * The scratch is a fixed array of 8 MiB per GPU (every GPU the library runs on holds its
 * own until the process ends); a plan whose libra_plan_workspace_bytes exceeds it is
 * refused with LIBRA_E_WORKSPACE before anything is enqueued.  No call allocates
 * (no hipMalloc, hipHostMalloc, hipFree or event creation); per-kernel timing is never
 * recorded for it.  The first call on a device looks up the scratch's device address
 * (hipGetSymbolAddress) with that device current; make one call before any capture.
 * A call copies the plan's tables into the scratch (from the plan's pinned image) unless
 * the scratch already holds that plan's tables, so repeated calls of one plan enqueue
 * kernels only.  All calls on one GPU share its scratch: calls that may overlap on that
 * GPU (other streams, other threads) race and must be ordered by the caller.  No kernel
 * of this call needs the scratch zeroed; stale contents are overwritten before use.
 */
libra_status libra_decode_attn_noalloc(libra_kv_layout layout, libra_plan plan, const void* q,
                                       const int32_t* block_table, int32_t bt_stride,
                                       int32_t batch, int32_t num_q_heads, float scale, void* out,
                                       float* lse, void* stream);

/*
 * Append: sequence b adds C_b tokens (a tool-output chunk, or C_b = 1 for an ordinary
 * decode step) after P_b = L_b - C_b cached tokens, as when a tool returns and its
 * output is incorporated before decoding resumes (Sec. 5, Phase 2 and Step 3).  The
 * call first writes k_new / v_new into the cache at positions [P_b, L_b), then new
 * token i attends keys [0, P_b + i] (causal, itself included) with the formula above.
 *
 * q, out: device bf16 [sum C_b][num_q_heads][128], rows of sequence b starting at
 * sum_{b' < b} C_b'.  k_new, v_new: device bf16 [sum C_b][num_kv_heads][128].  lse:
 * device float32 [sum C_b][num_q_heads] or NULL.  The block table must already map the
 * pages of positions [0, L_b).  The plan must be an append plan for the same shapes.
 *
 * When the plan has both single-token rows and chunk rows, the chunk tiles are
 * launched on `stream` and the single-token rows on the library's auxiliary stream of
 * the current device, forked from `stream` after the cache write and joined back before
 * the split merge (events only): the matrix-core bound chunk tiles and the HBM-bound
 * decode rows then share the device.  Work enqueued on `stream` after the call starts
 * after both.  Under HIP graph capture this is the usual fork / join, captured as such.
 */
libra_status libra_append_attn(libra_kv_layout layout, libra_plan plan, const void* q,
                               const void* k_new, const void* v_new, const int32_t* block_table,
                               int32_t bt_stride, int32_t batch, int32_t num_q_heads, float scale,
                               void* workspace, size_t ws_bytes, void* out, float* lse,
                               void* stream);

/* ------------------------------------------------------------------------------ */
/* Per-kernel timing                                                               */
/* ------------------------------------------------------------------------------ */
/*
 * When enabled (process-wide), every kernel the library enqueues is bracketed by a pair
 * of HIP events on the caller's stream.  libra_profile_collect waits for all recorded
 * events, adds up elapsed milliseconds per kernel kind into *out and clears the record.
 * Used to measure each kernel's own duration inside a multi-kernel call (and to fit
 * per-operator latency models from measured timings).  Off by default; enabling it
 * adds two event records per launch.  Not for use under HIP graph capture.
 */
enum {
  LIBRA_KERNEL_PACK = 0,
  LIBRA_KERNEL_UNPACK = 1,
  LIBRA_KERNEL_GATHER = 2,
  LIBRA_KERNEL_CACHE_WRITE = 3,
  LIBRA_KERNEL_DECODE = 4,
  LIBRA_KERNEL_MERGE = 5,
  LIBRA_KERNEL_CHUNK = 6,
  LIBRA_KERNEL_UPLOAD = 7,
  LIBRA_KERNEL_COPY_OUT = 8,
  LIBRA_KERNEL_COPY_IN = 9,
  LIBRA_KERNEL_KINDS = 10
};

typedef struct libra_kernel_times {
  double ms[LIBRA_KERNEL_KINDS];       /* summed elapsed time per kernel kind */
  int64_t launches[LIBRA_KERNEL_KINDS];
} libra_kernel_times;

libra_status libra_profile_enable(int enable);
libra_status libra_profile_collect(libra_kernel_times* out);

/* ------------------------------------------------------------------------------ */
/* Cost evaluator: per-operator latency polynomials (host)                         */
/* ------------------------------------------------------------------------------ */
/*
 * The cost evaluator models the time of an operator at sequence length L as a
 * polynomial, quadratic for attention, T(L) = gamma L^2 + eta L + theta, whose
 * coefficients come from timings measured offline (Sec. 4.5; App. B.1, "CE
 * calibration").  Its fidelity is reported as the mean absolute percentage error (MAPE)
 * of predicted against measured times (Sec. 7.5).  All functions here are pure host
 * arithmetic on caller memory.
 */
typedef struct libra_ce_poly {
  double gamma; /* coefficient of L^2 */
  double eta;   /* coefficient of L */
  double theta; /* constant */
} libra_ce_poly;

/* Least-squares fit of T(L) to n measured points (lengths[i], times[i]), minimising the
 * sum of squared RELATIVE errors ((T(L_i) - t_i) / t_i)^2, the quantity MAPE averages.
 * Needs n >= 3, at least 3 distinct lengths, finite lengths >= 0 and finite times > 0;
 * otherwise LIBRA_E_INVAL. */
libra_status libra_ce_fit(const double* lengths, const double* times, int32_t n,
                          libra_ce_poly* out);

/* MAPE in percent: 100 / n * sum |T(L_i) - t_i| / t_i (times > 0, n >= 1). */
libra_status libra_ce_mape(const libra_ce_poly* poly, const double* lengths, const double* times,
                           int32_t n, double* mape);

/* Sum of T(l) over the integers l = a .. b (0 if b < a), in closed form: the time of a
 * decode trajectory whose per-step operator time at context l is T(l).  Needs
 * 0 <= a, b <= 2^24. */
libra_status libra_ce_poly_sum(const libra_ce_poly* poly, int64_t a, int64_t b, double* out);

/* ------------------------------------------------------------------------------ */
/* Rollout partition: RolloutDP (host)                                             */
/* ------------------------------------------------------------------------------ */
/*
 * Splits n_gpus GPUs into inference instances of TP degrees from a set (e.g. {1,2,4,8})
 * and gives each instance a contiguous run of the requests sorted by length, minimising
 * the makespan (Sec. 4.2; Alg. 1, RolloutDP):
 *
 *   dp[0][0] = 0, dp[g][i] = min over tp <= g, 0 <= x <= i of
 *              max(dp[g - tp][i - x], Cost(tp, i - x + 1, i)),     answer dp[n_gpus][n_req].
 *
 * Cost(tp, a, b) is the cost evaluator's RolloutTime of one instance serving sorted
 * requests a..b (1-based; empty when x = 0, cost 0).  The library's model of it (the
 * paper leaves the aggregation to its simulator) is continuous batching of all the
 * instance's requests: the instance runs as many decode steps as its longest request,
 * each paying the non-attention time once, and every request pays its own trajectory's
 * attention time:
 *
 *   Cost(tp, a, b) = linear_step[tp] * len_b + attn_scale[tp] * sum_{j=a..b} A(len_j),
 *   A(len) = sum_{l=1..len} attn_step(l)          (libra_ce_poly_sum(attn_step, 1, len)).
 *
 * Ties: candidates are visited in increasing g, i, then tp in tp_set order, then x
 * ascending, and a candidate replaces the best only when strictly smaller.
 */
typedef struct libra_rollout_model {
  libra_ce_poly attn_step; /* attention time of one decode step of one request at context l */
  double linear_step[4];   /* non-attention time per decode step of an instance at TP 1,2,4,8 */
  double attn_scale[4];    /* attention time multiplier at TP 1, 2, 4, 8 */
} libra_rollout_model;

/* lengths: n_req request lengths (>= 0, <= 2^24).  tp_set: n_tp distinct degrees from
 * {1, 2, 4, 8}.  Outputs: *makespan (+inf if no partition uses exactly n_gpus GPUs);
 * order[n_req] = request indices sorted by (length, index); instances[3 * k] =
 * (tp, first sorted position, count) for the k-th instance, in backtracking order
 * (last-added first), *n_instances <= n_gpus.  Work O(n_gpus * n_req^2 * n_tp) with the
 * literal recurrence (exact = 1), or O(n_gpus * n_req * n_tp * log n_req) (exact = 0),
 * which uses that both arguments of the max are monotone in x and returns the same
 * makespan.  Limits: n_gpus <= 4096, n_req <= 65536. */
libra_status libra_rollout_dp(const int64_t* lengths, int32_t n_req, int32_t n_gpus,
                              const int32_t* tp_set, int32_t n_tp,
                              const libra_rollout_model* model, int32_t exact, double* makespan,
                              int32_t* order, int32_t* instances, int32_t* n_instances);

/* ------------------------------------------------------------------------------ */
/* Causality-guided bucket routing (host)                                          */
/* ------------------------------------------------------------------------------ */
/*
 * A prefix tree over tool-return histories (Sec. 5, "Causality-aware prefix tree").  A
 * node at depth k is the key (prompt_id, <s_1 .. s_k>), where s_i is the composite state
 * of the i-th tool call (tool type, payload size class, success or failure; encode it
 * with LIBRA_TOOL_STATE).  Every node counts the remaining trajectory length observed
 * from that point, in bins aligned to the bucket length thresholds: bin k holds lengths
 * in [edge[k-1], edge[k]) with edge[-1] = 0 and edge[n_edges] = infinity, so there are
 * n_edges + 1 bins.  A root above all prompts (depth -1) gathers every trace.
 */
#define LIBRA_TOOL_STATE(tool_type, large, failure) \
  ((int32_t)(((tool_type) << 2) | ((large) ? 2 : 0) | ((failure) ? 1 : 0)))

typedef struct libra_trie_s* libra_trie;

/* bin_edges: n_edges strictly increasing positive thresholds (n_edges in [0, 63]). */
libra_status libra_trie_create(const int64_t* bin_edges, int32_t n_edges, libra_trie* out);
void libra_trie_destroy(libra_trie trie);

/* Inserts one finished trajectory (Sec. 5, Phase 3; App. B.1 bootstrap): states[0 ..
 * n_states) are its tool returns in order, residual[k] (k = 0 .. n_states) the length
 * still to be generated after the k-th return (residual[0]: from the prompt on).  The
 * root, the prompt node and the node after each return record their residual. */
libra_status libra_trie_insert(libra_trie trie, int64_t prompt_id, const int32_t* states,
                               int32_t n_states, const int64_t* residual);

/* Walks (prompt_id, states[0 .. n_states)) and writes the residual-length distribution
 * F = {p_k} of the deepest node on that path that exists (an unseen node backs off to
 * its parent; an unseen prompt to the root) into hist[n_edges + 1], and that node's
 * depth into *depth (-1 = root).  An empty tree gives LIBRA_E_INVAL. */
libra_status libra_trie_lookup(libra_trie trie, int64_t prompt_id, const int32_t* states,
                               int32_t n_states, double* hist, int32_t* depth);

/* Phase 2 routing (Sec. 5): B* = argmin_B sum_k hist[k] * t_dec[B * n_bins + k] +
 * c_mig[current * n_buckets + B], with c_mig's diagonal taken as 0 whatever it holds.
 * Ties go to the lowest bucket index.  Writes *best and its cost *best_cost. */
libra_status libra_route_bucket(const double* hist, int32_t n_bins, const double* t_dec,
                                const double* c_mig, int32_t n_buckets, int32_t current,
                                int32_t* best, double* best_cost);

#ifdef __cplusplus
}
#endif

#endif /* LIBRA_H_ */
