/*
 * atp.h — C ABI of the MI355X state-preserving tensor-parallel reshard
 * (AnchorTP, arXiv 2511.11617: Sec. III-B elastic TP, Alg. 1 Continuous
 * Minimal Migration, Eq. 1 minimum reload, Sec. III-C execution scheduler).
 *
 * One surviving GPU's share of a TP change k -> k' with unequal widths:
 *   atp_plan             plan the change on the host (partitions, CMM tasks,
 *                        new arena layout, copy descriptors, in-place order)
 *   atp_reshard_weights  repack this GPU's retained weight slices into the
 *                        new shard layout and land the missing bytes
 *   atp_reshard_kv       the same for the paged KV cache (block ids kept)
 *   atp_sync             wait for both, report the first asynchronous error
 *
 * Conventions
 *   - Status: every int-returning call returns ATP_OK (0) or a negative
 *     ATP_E* code; atp_last_error() returns the message of the last failure
 *     on the calling thread.
 *   - Ownership: the caller owns every buffer (arenas, block table, pinned
 *     host buffers, staging).  The library allocates no device memory; it
 *     keeps its descriptors, prefix sums and landing ring inside the
 *     caller's staging buffer.  A plan is a library-owned host object,
 *     freed with atp_plan_free.
 *   - Streams: atp_stream is a hipStream_t.  Calls only enqueue work and
 *     return; atp_sync blocks.
 *   - Bytes are copied, never converted: any 16-bit payload (NaN, -0,
 *     denormals) arrives unchanged.
 *   - Threading: a plan is used by one host thread at a time.  Several
 *     plans may be pending on one device at once, each on buffers of its
 *     own; those issued on the same (compute, copy) pair run their side
 *     work in issue order.
 */
#ifndef ATP_H
#define ATP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
  ATP_OK = 0,
  ATP_EINVAL = -1,    /* malformed problem, bad argument, bad block table  */
  ATP_ECAPACITY = -2, /* an arena, staging or host buffer is too small     */
  ATP_EHIP = -3,      /* a HIP runtime call failed                         */
  ATP_EALIGN = -4,    /* a device buffer is not 256-byte aligned           */
  ATP_ESTATE = -5     /* call out of order (reshard again before atp_sync) */
};

typedef void *atp_stream; /* hipStream_t */

/* Half-open range [begin, end) in units of a partition space. */
typedef struct {
  int64_t begin, end;
} atp_range;

/* ---- partition spaces (Sec. III-B, Alg. 1) ------------------------------ */
/* How the old ranges (old_tp of them) or the new ranges (new_tp of them,
 * one per target, in target order) of a space are obtained; n is old_tp or
 * new_tp.
 *   EXPLICIT    given by the caller (old_ranges / new_ranges)
 *   FLOOR       Alg. 1: range j = [floor(j H / n), floor((j+1) H / n))
 *   CEIL_FIRST  Sec. III-B unequal widths: ceil(H/n) wide first, then
 *               floor(H/n) (the even split when n divides H)
 *   GQA         ranges follow the query-head space `gqa_space` (old ranges
 *               its old ranges, new ranges its new ones): query heads
 *               [a, b) need KV heads [floor(a/g), ceil(b/g)) with
 *               g = gqa_group; ranges may overlap (replicas)
 *   WIDTHS      consecutive ranges of the given widths (old_widths /
 *               new_widths), which must add up to H */
enum { ATP_RULE_EXPLICIT = 0, ATP_RULE_FLOOR = 1, ATP_RULE_CEIL_FIRST = 2, ATP_RULE_GQA = 3,
       ATP_RULE_WIDTHS = 4 };

/* One space: attention heads, KV heads, FFN column groups, experts.
 * total_units is H; with Alg. 1 it is the largest end of any old range,
 * dead ranks included.  Old rank i's range (dead ranks included) comes
 * from old_rule; the old ranges may overlap (replicated units) and must
 * together cover [0, H), and so must the new ranges. */
typedef struct {
  int64_t total_units;
  int32_t old_tp;
  int32_t new_tp;
  const atp_range *old_ranges; /* old_rule EXPLICIT: old_tp ranges   */
  int32_t new_rule;
  int32_t gqa_space; /* GQA: index of the query-head space     */
  int32_t gqa_group; /* GQA: query heads per KV head           */
  int32_t old_rule;  /* ATP_RULE_*; 0 = EXPLICIT (old_ranges)  */
  const atp_range *new_ranges; /* new_rule EXPLICIT: new_tp ranges   */
  const int64_t *old_widths;   /* old_rule WIDTHS: old_tp widths     */
  const int64_t *new_widths;   /* new_rule WIDTHS: new_tp widths     */
} atp_space;

/* ---- tensors (Sec. III-B layout invariants) ----------------------------- */
/* A weight is the full logical [rows, cols] row-major matrix; the space
 * shards its rows (ATP_ROWS: column-parallel Wq/Wk/Wv/W_gate/W_up/experts)
 * or its columns (ATP_COLS: row-parallel Wo/W_down); `unit` rows or
 * columns make one unit of the space.  old_offset is the byte offset of
 * this GPU's old shard in the old arena, or ATP_OFFSET_AUTO for the packed
 * layout (shards in tensor order, each at the next 256-byte boundary).
 * The new arena always uses the packed layout. */
enum { ATP_ROWS = 0, ATP_COLS = 1 };
#define ATP_OFFSET_AUTO UINT64_MAX

typedef struct {
  int32_t space;
  int32_t kind;
  int32_t layer;
  int32_t elem_bytes;
  int64_t rows, cols, unit;
  uint64_t old_offset;
} atp_tensor;

/* ---- paged KV cache (Sec. III-B: each token block keeps its heads apart) */
/* Arena of one rank: [layer][K,V][num_blocks][heads][block_tokens][head_dim]
 * (HEAD_MAJOR) or [layer][K,V][num_blocks][block_tokens][heads][head_dim]
 * (TOKEN_MAJOR), heads = the rank's KV-head range of `space`.  Physical
 * block ids are unchanged by the reshard; live_blocks is the number of
 * distinct ids the block table references.  With ATP_KV_COMPACT the new
 * arena has live_blocks blocks per (layer, K|V) plane instead of num_blocks,
 * and live block p lands at its rank among the live ids (ascending): the
 * caller renumbers its table the same way (atp_kv_evict_lru does). */
enum { ATP_KV_HEAD_MAJOR = 0, ATP_KV_TOKEN_MAJOR = 1 };

typedef struct {
  int32_t space;
  int32_t num_layers;
  int32_t block_tokens;
  int32_t head_dim;
  int32_t elem_bytes;
  int32_t layout;
  int64_t num_blocks;
  int64_t live_blocks;
} atp_kv;

/* ---- problem ------------------------------------------------------------ */
enum {
  ATP_ASSIGN_INORDER = 0,   /* target j hosted by the j-th survivor      */
  ATP_ASSIGN_MAXRETAIN = 1, /* survivor permutation keeping most bytes   */
  ATP_INPLACE = 1 << 4,     /* new layout overwrites the old arena       */
  ATP_PLAN_GREEDY = 1 << 8, /* Sec. V baseline: keep local, reload gaps  */
  ATP_PLAN_FULL = 1 << 9,   /* Sec. V baseline: reload every byte        */
  ATP_KV_COMPACT = 1 << 10, /* new KV arena holds only the live blocks,  */
                            /* block p at its rank among the live ids    */
                            /* (out of place only; see atp_kv_evict_lru) */
  ATP_NO_TAIL_STAGING = 1 << 11 /* in place: stage only what cycles need,  */
                            /* never the tail of a level chain (every     */
                            /* hazard then resolved by levels alone)      */
};

typedef struct {
  int32_t n_spaces;
  const atp_space *spaces;
  int32_t n_tensors;
  const atp_tensor *tensors;
  const atp_kv *kv;      /* NULL: no KV cache                          */
  const int32_t *failed; /* old ranks that died                        */
  int32_t n_failed;
  int32_t self_old_rank; /* this GPU's old rank (must survive)         */
  int32_t flags;
  int32_t reserved;
  uint64_t staging_cap;  /* in place: staging bytes the schedule may use */
} atp_problem;

typedef struct atp_plan_obj atp_plan_t;

/* Plan the reshard (Alg. 1 per space, Eq. 1 statistics, Sec. III-C
 * single-pass pre-allocation: new layout sizes and staging needs, and for
 * ATP_INPLACE a hazard-free level order with a bounded staging buffer; the
 * tail of a long level chain goes through the staging the cap leaves when
 * that saves launches, unless ATP_NO_TAIL_STAGING).
 * Errors: ATP_EINVAL (malformed problem), ATP_ECAPACITY (in-place schedule
 * needs more than staging_cap).  *out is set only on success. */
int atp_plan(const atp_problem *problem, atp_plan_t **out);
void atp_plan_free(atp_plan_t *plan);

/* Repack this GPU's weights (Sec. III-B parameter re-assignment/reload
 * primitive; Sec. III-C pipelined execution).
 *   arena        old shard (device, 256-B aligned), arena_bytes long; with
 *                ATP_INPLACE it must also hold the new layout
 *   new_arena    destination (device) of new_arena_bytes; NULL with ATP_INPLACE
 *   inflow_host  pinned host buffer of exactly stats.inflow_w bytes holding
 *                the bytes this GPU does not keep, in the plan's packing
 *                order (atp_plan_segments, ATP_SEG_INFLOW_W); stands in for
 *                peer P2P and host reload
 *   outbound_host pinned host buffer of stats.outbound_w bytes that receives
 *                (in place only) the old bytes peers need and this GPU drops,
 *                read before they are overwritten; may be NULL if 0 bytes
 *   staging      device scratch of at least stats.staging_w bytes
 * The copy kernel itself reads every inflow piece that is not a large
 * contiguous gap (those land by DMA) from inflow_host, and with ATP_INPLACE
 * writes the outbound bytes: both host buffers must come from hipHostMalloc
 * (device-accessible at the same address) and be 256-byte aligned, else
 * ATP_EINVAL / ATP_EALIGN.
 * Launch errors return ATP_EHIP once the work the call had already queued
 * has drained (the plan is then not pending); kernel-side errors surface in
 * atp_sync. */
int atp_reshard_weights(atp_plan_t *plan, void *arena, uint64_t arena_bytes,
                        void *new_arena, uint64_t new_arena_bytes,
                        const void *inflow_host, uint64_t inflow_bytes,
                        void *outbound_host, uint64_t outbound_bytes,
                        void *staging, uint64_t staging_bytes,
                        atp_stream compute, atp_stream copy);

/* Repack this GPU's paged KV cache (Sec. III-B KV operators with
 * variable-length shards).  block_table is a device int32
 * [n_seq][max_blocks], -1 = unused, read only; ids must be < num_blocks
 * and the distinct ids must number kv.live_blocks (else ATP_EINVAL from
 * atp_sync).  Buffers as for atp_reshard_weights, sizes from stats.*_kv.
 * With ATP_INPLACE the KV inflow lands only by DMA through the landing
 * ring (the copy kernel does not read it), so inflow_host may then be
 * ordinary pageable memory, at a lower copy rate; the outbound buffer must
 * still come from hipHostMalloc.
 * The weights and KV calls may be pending together if their staging
 * buffers do not overlap; with ATP_INPLACE the weights call must then come
 * first (a weights call after a pending KV call is ATP_ESTATE). */
int atp_reshard_kv(atp_plan_t *plan, void *kv_arena, uint64_t kv_bytes,
                   void *new_kv_arena, uint64_t new_kv_bytes,
                   const int32_t *block_table, int32_t n_seq, int32_t max_blocks,
                   const void *inflow_host, uint64_t inflow_bytes,
                   void *outbound_host, uint64_t outbound_bytes,
                   void *staging, uint64_t staging_bytes,
                   atp_stream compute, atp_stream copy);

/* atp_reshard_kv for callers that cannot allocate (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * reshard, with no staging argument.  Its descriptors, prefix sums, block
 * lists and landing ring live in a file-scope device array of the library
 * (atp_scratch_bytes() = 64 MiB, one copy per device, held until the process
 * ends), and the call allocates nothing: its events, pinned descriptor
 * buffers and side stream come from what atp_warmup(compute, copy, events)
 * pooled on this device for these streams (run it first; running short is
 * ATP_ESTATE, not an allocation).  A plan whose stats.staging_kv exceeds
 * atp_scratch_bytes() is ATP_ECAPACITY (in place, plan with a staging_cap
 * no larger).  Every such call of a process on one device shares that
 * device's array (each process loads its own), so two of them pending at
 * once would race on it: a second call before the first one's atp_sync is
 * refused with ATP_ESTATE.  Nothing in the array needs to start at zero.
 * Other arguments, results and errors as for atp_reshard_kv. */
int atp_reshard_kv_noalloc(atp_plan_t *plan, void *kv_arena, uint64_t kv_bytes,
                           void *new_kv_arena, uint64_t new_kv_bytes,
                           const int32_t *block_table, int32_t n_seq, int32_t max_blocks,
                           const void *inflow_host, uint64_t inflow_bytes,
                           void *outbound_host, uint64_t outbound_bytes,
                           atp_stream compute, atp_stream copy);
uint64_t atp_scratch_bytes(void);

/* Timing of the last reshard (HIP events; host clock for wall_ms). */
typedef struct {
  double plan_ms;      /* atp_plan host time                          */
  double wall_ms;      /* first reshard call -> atp_sync return        */
  double repack_w_ms;  /* weight repack kernels, summed launch times    */
  double repack_kv_ms; /* KV repack kernels, summed launch times        */
  double repack_span_ms; /* first -> last repack launch of each call,
                            summed; in place it includes the waits for
                            outbound reads                               */
  double h2d_ms;       /* copy-stream span of the inflow copies        */
  double d2h_ms;       /* span of the outbound copies (in place)       */
  double scatter_ms;   /* summed landing-ring scatter kernel time      */
  double overlap;      /* (repack + h2d - wall) / min(repack, h2d)     */
  uint64_t repack_bytes;  /* algorithmic bytes: 2 x moved retained    */
  uint64_t h2d_bytes, d2h_bytes, scatter_bytes;
  int32_t n_launches;
  int32_t reserved;
  double repack_union_ms; /* time during which any repack kernel of the
                             pending calls ran (their intervals' union):
                             the device repack time when the weights and
                             KV repacks overlap                          */
} atp_timing;

/* Wait for the pending reshard calls of `plan` and report them.  This ends
 * the reshard's freeze window (Sec. III-B: serving pauses while parameters
 * and KV are re-laid out, then resumes on the new layout): when it returns
 * ATP_OK, every retained byte is in its new place and every inflow byte has
 * landed (Sec. III-C: the reloads and transfers that were pipelined with the
 * repack are complete), so the caller may switch its views to the new
 * layout, reuse the host buffers and free staging.  Returns the first
 * asynchronous error: ATP_EINVAL for a bad block table (an id >= num_blocks,
 * or a live-block count other than kv.live_blocks), ATP_EHIP for a failure
 * on the GPU; ATP_ESTATE if nothing was issued.  Whatever it returns, no
 * work of the plan is still running afterwards.  `out` may be NULL. */
int atp_sync(atp_plan_t *plan, atp_timing *out);

/* Optional: do, before the first reshard on the current device, the
 * per-process set-up that reshard would otherwise pay (about 5 ms on the
 * 40-layer TP 4->3 workload): load the kernels, choose the library's side
 * stream for this (compute, copy) pair (a probe that waits for what those
 * streams already hold), and create `events` pooled HIP events of each kind
 * (0..4096; 256 covers the workloads here) and pinned descriptor buffers.
 * A process that may have to recover calls it ahead of time, e.g. right
 * after mapping the state plane's regions.  Calling it again is harmless.
 * Errors: ATP_EINVAL for `events` out of range, ATP_EHIP without a usable
 * device. */
int atp_warmup(atp_stream compute, atp_stream copy, int32_t events);

/* ---- inspection helpers (tests, benchmark) ------------------------------ */
typedef struct {
  int32_t self_new_rank;
  int32_t n_levels_w;   /* in-place levels (1 when out of place)      */
  int32_t n_levels_kv;
  int32_t n_desc_w, n_desc_kv;
  int32_t reserved;
  uint64_t old_arena_bytes, new_arena_bytes; /* weights, packed layouts */
  uint64_t old_kv_bytes, new_kv_bytes;
  uint64_t retained_w, inflow_w, outbound_w; /* this GPU, bytes          */
  uint64_t retained_kv, inflow_kv, outbound_kv;
  uint64_t moved_w, moved_kv;   /* retained bytes whose address changes */
  uint64_t staged_w, staged_kv; /* in place: bytes routed via staging   */
  uint64_t staging_w, staging_kv; /* staging bytes each call needs      */
  uint64_t global_keep, global_p2p, global_reload; /* all survivors     */
  uint64_t reload_min;          /* Eq. 1, bytes                         */
  uint64_t tail_w, tail_kv;     /* of staged: a level chain's tail,     */
                                /* moved through staging (in place)     */
} atp_stats;
int atp_plan_stats(const atp_plan_t *plan, atp_stats *out);

enum { ATP_KEEP = 0, ATP_P2P = 1, ATP_RELOAD = 2 };
typedef struct {
  int32_t kind;     /* ATP_KEEP / ATP_P2P / ATP_RELOAD                   */
  int32_t src;      /* old rank holding the units, -1 for a reload       */
  int32_t dst;      /* target index (new rank)                           */
  int32_t host;     /* old rank hosting the target                       */
  int64_t begin, end;
} atp_task;
/* Tasks of one space in plan order (Alg. 1). */
int atp_plan_tasks(const atp_plan_t *plan, int32_t space, atp_task *out,
                   int32_t cap, int32_t *n);
/* Resolved new ranges of one space, in target order. */
int atp_plan_ranges(const atp_plan_t *plan, int32_t space, atp_range *out,
                    int32_t cap, int32_t *n);
/* Resolved old ranges of one space, in old-rank order (dead ranks included). */
int atp_plan_old_ranges(const atp_plan_t *plan, int32_t space, atp_range *out,
                        int32_t cap, int32_t *n);
/* owner[j] = old rank hosting target j. */
int atp_plan_owner(const atp_plan_t *plan, int32_t *owner, int32_t cap, int32_t *n);
/* Old/new byte offsets and new shard bytes of tensor `t`. */
int atp_plan_layout(const atp_plan_t *plan, int32_t t, uint64_t *old_offset,
                    uint64_t *new_offset, uint64_t *new_bytes);

/* Packed host-buffer segments, in buffer order. */
enum { ATP_SEG_INFLOW_W = 0, ATP_SEG_OUTBOUND_W = 1, ATP_SEG_INFLOW_KV = 2,
       ATP_SEG_OUTBOUND_KV = 3 };
typedef struct {
  int32_t tensor;      /* tensor index, or -1 for KV                      */
  int32_t layer;       /* KV: layer                                       */
  int32_t which;       /* KV: 0 = K, 1 = V                                */
  int32_t kind;        /* ATP_P2P / ATP_RELOAD (inflow), ATP_P2P (outbound)*/
  int64_t unit_begin, unit_end; /* units of the tensor's / KV space      */
  uint64_t host_offset, bytes;  /* position in the packed host buffer   */
} atp_segment;
int atp_plan_segments(const atp_plan_t *plan, int32_t which, atp_segment *out,
                      int32_t cap, int32_t *n);

/* One kernel launch of the last reshard: kind 0 = weight repack,
 * 1 = KV repack, 2 = landing-ring scatter (in-place KV inflow), 3 = outbound
 * read into the host buffer (in place), 4 = inflow read from the host buffer;
 * `ms` from HIP events on the stream the launch ran on. */
typedef struct {
  int32_t kind, level;
  uint64_t bytes;
  double ms;
} atp_launch;
int atp_plan_launches(const atp_plan_t *plan, atp_launch *out, int32_t cap, int32_t *n);

/* The executable schedule of one call (which = 0 weights, 1 KV), in the
 * order the executor issues it, for replay on a host copy (tests):
 *   REPACK   device copy of level `level`; all copies of one level run
 *            concurrently, levels run in order
 *   H2D_RING host inflow -> landing-ring slot (staging), then the SCATTER
 *            copies that follow it; ring traffic starts after all levels
 *   H2D      host inflow -> arena, allowed once level `level` has
 *            finished (level -1: at any time) and the first `after_d2h`
 *            D2H copies of the list have finished
 *   D2H      arena or staging -> host outbound buffer; must finish
 *            before level `level` starts (-1: before any inflow landing
 *            that waits for it); issued one after another in list order
 *            (in place only)
 * A copy moves, for each item o in [item_begin, item_end) and line t in
 * [0, rows), `run` bytes from src_off + i(o) * src_stride + t * src_pitch
 * to dst_off + j(o) * dst_stride + t * dst_pitch, where i(o) / j(o) is
 * o - item_begin on a plain side and the o-th live block id (ascending)
 * on an indexed side; with ATP_COPY_BLOCK_RANGE the items are the live
 * blocks whose ids lie in [item_begin, item_end). */
enum { ATP_COPY_REPACK = 0, ATP_COPY_SCATTER = 1, ATP_COPY_H2D = 2, ATP_COPY_H2D_RING = 3,
       ATP_COPY_D2H = 4 };
enum { ATP_BUF_OLD = 0, ATP_BUF_NEW = 1, ATP_BUF_STAGING = 2, ATP_BUF_INFLOW = 3,
       ATP_BUF_OUTBOUND = 4 };
enum { ATP_COPY_SRC_INDEXED = 1, ATP_COPY_DST_INDEXED = 2, ATP_COPY_BLOCK_RANGE = 4 };
typedef struct {
  int32_t op, level;
  int32_t src_buf, dst_buf;
  int32_t flags;
  int32_t after_d2h; /* H2D, SCATTER: the first after_d2h D2H copies of
                        this list (issued in list order) must have
                        finished                                        */
  uint64_t src_off, dst_off, src_pitch, dst_pitch, src_stride, dst_stride;
  int64_t item_begin, item_end;
  uint64_t run, rows;
} atp_copy;
int atp_plan_copies(const atp_plan_t *plan, int32_t which, atp_copy *out, int32_t cap, int32_t *n);

/* Ranges of a partition of `total` units into `parts` (FLOOR or
 * CEIL_FIRST). */
int atp_partition(int64_t total, int32_t parts, int32_t rule, atp_range *out);

/* ---- range-read reload source (Sec. IV: the loader reads safetensors by
 * offsets, fetching only the byte intervals it needs) ---------------------- */
typedef struct atp_st_obj atp_st_t;

/* Open `n_paths` safetensors files and parse their headers: an 8-byte
 * little-endian header length, a JSON object of name -> {dtype, shape,
 * data_offsets}, then the data.  Every tensor is checked: known dtype,
 * offsets inside the data, size = product(shape) x dtype size, names unique
 * across the files.  Any violation gives ATP_EINVAL and *out stays unset.
 * The files stay open until atp_st_close. */
int atp_st_open(const char *const *paths, int32_t n_paths, atp_st_t **out);
void atp_st_close(atp_st_t *st);

typedef struct {
  int32_t file;        /* index into the paths given to atp_st_open      */
  int32_t elem_bytes;  /* bytes per element of the dtype                 */
  int32_t ndim;        /* rank of the shape (shape[] holds the first 8)  */
  int64_t shape[8];
  uint64_t offset, bytes; /* absolute byte range of the data in the file */
} atp_st_tensor;
/* Look a tensor up by name; ATP_EINVAL if no file holds it. */
int atp_st_find(const atp_st_t *st, const char *name, atp_st_tensor *out);

typedef struct {
  double read_ms;         /* wall time of the range reads                 */
  uint64_t bytes;         /* bytes read (= the plan's weight inflow)       */
  uint64_t reads;         /* pread calls issued                            */
  uint64_t tensor_bytes;  /* data bytes of the named tensors: what a full
                             reload of them would read                     */
  int32_t threads;        /* reader threads used                           */
} atp_load_stats;

/* Fill the plan's packed weight inflow buffer (atp_plan_segments,
 * ATP_SEG_INFLOW_W) from the files, reading only the needed intervals:
 *   names        one tensor name per problem tensor (problem order); the
 *                named tensor must be 2-D [rows, cols] with the problem
 *                tensor's rows, cols and elem_bytes (experts stacked as the
 *                problem states them)
 *   inflow_host  host buffer of exactly stats.inflow_w bytes (pinned for the
 *                reshard that follows); written in the plan's packing order:
 *                ATP_ROWS units [a, b) are rows [a*unit, b*unit), one
 *                interval; ATP_COLS units are columns, one interval per row,
 *                packed row after row
 *   n_threads    reader threads, <= 0 for min(16, hardware threads)
 *   stats        may be NULL
 * Synchronous; safe to call while a reshard of another plan runs.  A missing
 * name, a shape or element-size mismatch, a wrong buffer size or a failed
 * read gives ATP_EINVAL (the buffer is then partly written). */
int atp_load_weights(const atp_plan_t *plan, const atp_st_t *st, const char *const *names,
                     int32_t n_names, void *inflow_host, uint64_t inflow_bytes,
                     int32_t n_threads, atp_load_stats *stats);

/* The range-read reload pipelined with the weights reshard (Sec. III-C:
 * reloads overlapped with the rest of the recovery).  Runs the reads of
 * atp_load_weights on `n_threads` host threads (0: up to 16) into
 * inflow_host and enqueues the reshard of atp_reshard_weights (same
 * arguments and buffer rules), issuing each inflow piece only once the reads
 * under it have completed, so that the file reads overlap the landings; the
 * GPU never waits for the host.  Returns once every read is done and all the
 * work is enqueued; atp_sync as after atp_reshard_weights.  Out of place,
 * issue atp_reshard_kv first: its inflow then uses the link while the
 * weights are read.  Name or shape errors are ATP_EINVAL before anything
 * starts.  A failed read is ATP_EINVAL after the enqueued work has drained
 * (the plan is then not pending). */
int atp_load_reshard_weights(atp_plan_t *plan, const atp_st_t *st, const char *const *names,
                             int32_t n_names, void *arena, uint64_t arena_bytes,
                             void *new_arena, uint64_t new_arena_bytes,
                             void *inflow_host, uint64_t inflow_bytes,
                             void *outbound_host, uint64_t outbound_bytes,
                             void *staging, uint64_t staging_bytes,
                             atp_stream compute, atp_stream copy, int32_t n_threads,
                             atp_load_stats *stats);

/* The same pipelined reload, returning before the reads are done (Sec.
 * III-C: the reloads overlap the rest of the recovery, the KV move
 * included).  Queues the work that needs no inflow byte (prepare, outbound
 * reads, repack levels) and starts the reads; the inflow pieces are issued
 * by atp_sync, each once the reads under it have completed, and atp_sync
 * returns once they have landed.  Between the two calls the caller may
 * issue atp_reshard_kv (in place this is the order the library needs, and
 * its KV inflow then uses the link while the weights are read).  Every
 * buffer must stay valid until atp_sync returns; `st` and `names` only
 * during the call (the reads keep descriptors of their own).  Name or
 * shape errors are ATP_EINVAL before anything starts; a failed read is
 * atp_sync's ATP_EINVAL, after the queued work has drained.  The read
 * statistics come from atp_plan_load_stats after atp_sync. */
int atp_load_reshard_weights_async(atp_plan_t *plan, const atp_st_t *st, const char *const *names,
                                   int32_t n_names, void *arena, uint64_t arena_bytes,
                                   void *new_arena, uint64_t new_arena_bytes,
                                   void *inflow_host, uint64_t inflow_bytes,
                                   void *outbound_host, uint64_t outbound_bytes,
                                   void *staging, uint64_t staging_bytes,
                                   atp_stream compute, atp_stream copy, int32_t n_threads);
/* Read statistics of the plan's last atp_load_reshard_weights_async, once
 * atp_sync has returned ATP_OK for it; ATP_ESTATE before. */
int atp_plan_load_stats(const atp_plan_t *plan, atp_load_stats *out);

/* ---- KV budget under recovery (Sec. III-A: per-session recency; cold KV
 * released least recently used first when the demand exceeds the budget,
 * evicted sessions being rebuilt later by replay) ----------------------- */
typedef struct {
  int32_t kept_sessions, evicted_sessions;
  int64_t live_before, live_after;      /* distinct live block ids          */
  uint64_t demand_before, demand_after; /* live blocks x block_bytes        */
} atp_evict_stats;

/* Choose the sessions (rows of a host block table [n_seq][max_blocks], -1 =
 * unused, ids < num_blocks) that the new layout keeps under `budget_bytes`:
 *   last_use     per-session last-use time; larger = more recent
 *   block_bytes  bytes one block occupies in the new layout over all layers,
 *                K and V (stats.new_kv_bytes / num_blocks)
 * Sessions are evicted in ascending (last_use, session index) order while
 * (distinct live ids of the kept rows) x block_bytes > budget_bytes; a block
 * several rows share stays until its last row goes.  Outputs keep[n_seq]
 * (1 kept, 0 evicted) and new_table (may alias table): evicted rows become
 * all -1; with `compact` nonzero every kept id p becomes its rank among the
 * kept ids, the numbering of an ATP_KV_COMPACT arena.  Build the plan with
 * kv.live_blocks = stats.live_after and pass the kept rows (ids unchanged,
 * i.e. the table with compact = 0) to atp_reshard_kv.  ATP_EINVAL on an id
 * outside [-1, num_blocks) or NULL arrays. */
int atp_kv_evict_lru(const int32_t *table, int32_t n_seq, int32_t max_blocks, int64_t num_blocks,
                     const int64_t *last_use, uint64_t block_bytes, uint64_t budget_bytes,
                     int32_t compact, int32_t *keep, int32_t *new_table, atp_evict_stats *stats);

/* ---- state plane (Sec. III-A: a daemon, decoupled from the inference
 * process, keeps the GPU memory of the weights and the KV cache; inference
 * processes obtain handles to it over IPC and read and write it, so the
 * state survives a crashed inference process and a new one resumes on it;
 * the state plane also keeps each session's recency for the KV budget) ---- */
typedef struct atp_state_obj atp_state_t;

/* Run the daemon in the calling thread: listen on the Unix socket
 * `socket_path` (a stale socket file is replaced; a path another daemon
 * answers on is ATP_EINVAL), serve requests until atp_state_shutdown, then
 * free every region it holds and return ATP_OK.  The daemon owns each
 * region it allocates on `device` (hipMalloc + hipIpcGetMemHandle); it
 * touches the device only at the first allocation.  Regions are limited to
 * 2 GiB - 1 MiB each: larger IPC allocations have not opened reliably on
 * this platform. */
int atp_daemon_serve(const char *socket_path, int32_t device);

/* Connect to the daemon at `socket_path` (ATP_EINVAL if none answers).  One
 * connection belongs to one thread at a time.  atp_state_disconnect unmaps
 * every region the connection opened and closes it; the regions stay with
 * the daemon (as they do when the process dies). */
int atp_state_connect(const char *socket_path, atp_state_t **out);
void atp_state_disconnect(atp_state_t *state);

/* Ask the daemon for a new device region of `bytes` named `name` and map it
 * into this process at *dev_ptr (256-byte aligned, contents undefined).
 * ATP_EINVAL for an existing name or a size outside [1, 2 GiB - 1 MiB];
 * ATP_EHIP when the daemon or this process cannot allocate or map it. */
int atp_state_alloc(atp_state_t *state, const char *name, uint64_t bytes, void **dev_ptr);
/* Map the existing region `name`; *bytes (nullable) receives its size. */
int atp_state_open(atp_state_t *state, const char *name, void **dev_ptr, uint64_t *bytes);
/* Unmap a region this connection mapped (the daemon keeps it). */
int atp_state_release(atp_state_t *state, void *dev_ptr);
/* Unmap (here) and free (in the daemon) the region `name`. */
int atp_state_free(atp_state_t *state, const char *name);

/* Named host blobs kept by the daemon (block tables, per-session last use):
 * put replaces, get copies out.  atp_state_get with data = NULL only
 * reports the size in *bytes; a `cap` below the size is ATP_ECAPACITY with
 * *bytes set.  A missing name is ATP_EINVAL.  Blobs are at most 4 GiB. */
int atp_state_put(atp_state_t *state, const char *name, const void *data, uint64_t bytes);
int atp_state_get(atp_state_t *state, const char *name, void *data, uint64_t cap, uint64_t *bytes);

/* Text listing ("region <name> <bytes>" / "blob <name> <bytes>" lines,
 * NUL-terminated) of what the daemon holds; *bytes receives the size with
 * the terminator, text may be NULL to ask for it. */
int atp_state_list(atp_state_t *state, char *text, uint64_t cap, uint64_t *bytes);

/* Ask the daemon to free everything and stop.  A lost connection to the
 * daemon is ATP_ESTATE for every call. */
int atp_state_shutdown(atp_state_t *state);

const char *atp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* ATP_H */
