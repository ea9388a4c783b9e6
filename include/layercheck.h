/*
 * layercheck.h - C interface of the MI355X (gfx950) LayerCheck decision step.
 *
 * LayerCheck (adaptive layer-wise checkpointing for LLM post-training) keeps,
 * for every layer group of a model, a drift accumulator and the step at which
 * the layer was last persisted.  At each checkpoint opportunity it scores
 * every layer, selects the layers whose accumulated drift reached the
 * threshold or whose staleness reached the bound, and persists the full state
 * of exactly those layers (weights together with their optimizer tensors).
 * After a failure it assembles a mixed-timestamp composite state from the
 * newest persisted record of each layer.
 *
 * Every entry point returns an lc_status; nothing throws across this
 * interface.  All pointers to model arrays are DEVICE pointers owned by the
 * caller; the library never frees or reallocates them.  The library owns only
 * the opaque context and its small device tables.  Work is enqueued on the
 * HIP stream given at init; a context is single-stream and not thread-safe,
 * separate contexts are independent.  On any HIP failure the call returns
 * LC_ERR_HIP and the context is poisoned: later calls return
 * LC_ERR_BAD_STATE (lc_destroy still works).  Validation failures return
 * before anything is enqueued, leaving the context unchanged.  A message for
 * the last failure on the calling thread is available from lc_last_error().
 *
 * Tracing: with LAYERCHECK_ROCTX=1 in the environment when the first call is
 * made, every state-changing entry point (context, score, select, pack,
 * restore, optimizer steps, store) opens a roctx range named after itself
 * for the length of the call, so a marker trace (rocprofv3 --marker-trace)
 * places each call's host span beside its kernels.  The roctx library is
 * loaded at run time; without the variable, or without that library,
 * nothing is traced and nothing is loaded.
 *
 * Layer groups (Section 2.2): embed_tokens, each transformer block, the final
 * norm and lm_head.  A layer may consist of any number of tensors
 * ("segments"); a segment is one contiguous range of one tensor, so a ZeRO-3
 * shard of a layer is simply one segment (Section 4.1: each rank decides on
 * its own shard).
 */
#ifndef LAYERCHECK_H
#define LAYERCHECK_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LC_OK = 0,
  LC_ERR_INVALID_ARG = 1, /* bad pointer, size, id, order, value          */
  LC_ERR_BAD_STATE = 2,   /* call out of sequence, or poisoned context    */
  LC_ERR_CAPACITY = 3,    /* next record does not fit the staging buffer  */
  LC_ERR_NO_VERSION = 4,  /* a layer has no persisted record <= t_fail    */
  LC_ERR_HIP = 5,         /* a HIP runtime call failed                    */
  LC_ERR_OOM = 6,         /* host or device allocation of library tables  */
  LC_ERR_IO = 7           /* a file operation of the persistence store
                             failed (the message names it and its errno) */
} lc_status;

typedef enum { LC_DT_BF16 = 1, LC_DT_F32 = 2 } lc_dtype;

typedef enum {
  /* Eq. 1-2: the shadow holds W(t-1); each score adds u_l(t) to Delta_l and
   * the same pass refreshes the shadow of every layer to W(t). */
  LC_MODE_ACCUM = 0,
  /* Distance to the last persisted version: the shadow holds the weights as
   * last persisted; each score sets Delta_l = u_l(t); the pack of a selected
   * layer refreshes its shadow. */
  LC_MODE_SNAPSHOT = 1
} lc_mode;

typedef struct lc_ctx lc_ctx; /* opaque, library-owned */

/* One contiguous piece of one tensor of one layer.  All arrays hold `numel`
 * elements; weight and shadow have the layout's weight dtype, the others are
 * fp32.  Pointers must be naturally aligned (2 B for bf16, 4 B for fp32);
 * 16-byte alignment selects the vectorised fast path.  No two arrays of a
 * layout (over all its segments) may overlap in memory: LC_ERR_INVALID_ARG. */
typedef struct {
  uint32_t layer;     /* layer group id in [0, n_layers)                      */
  uint32_t reserved;  /* must be 0                                            */
  uint64_t numel;     /* > 0                                                  */
  void *weight;       /* device, live weights W (bf16 or fp32)                */
  void *shadow;       /* device, shadow copy S, same dtype; written by the lib.
                         May be NULL for every segment in LC_MODE_ACCUM when the
                         drift comes from lc_adamw_step_score (no S then)      */
  float *master;      /* device fp32 master copy; NULL iff !has_master        */
  float *exp_avg;     /* device fp32 Adam first moment m                      */
  float *exp_avg_sq;  /* device fp32 Adam second moment v.  Both may be NULL for
                         every segment: records then hold the weights (and
                         master) only, the SGD variant of Section 4.7          */
} lc_segment;

typedef struct {
  uint32_t n_layers;          /* N >= 1                                        */
  uint32_t n_segments;        /* >= n_layers                                   */
  const lc_segment *segments; /* host array; grouped by ascending layer id; the
                                 order inside a layer is the record order      */
  int32_t weight_dtype;       /* lc_dtype                                      */
  int32_t has_master;         /* 0 or 1                                        */
  int32_t mode;               /* lc_mode                                       */
  int32_t reserved;           /* must be 0                                     */
  const double *k0;           /* host [n_layers]: base thresholds K0_l >= 0
                                 (Section 3.4 uses 1e-3, 1e-2 for embeddings) */
  int64_t s_max;              /* staleness bound S_max >= 1 (Eq. 5)            */
  double eps_w;               /* Eq. 1 stabiliser, finite and >= 0 (e.g. 1e-8) */
  int64_t t_base;             /* step of the base full checkpoint (Sec. 3.4)   */
  void *stream;               /* hipStream_t, borrowed; NULL = null stream     */
} lc_layout_desc;

typedef struct {
  uint32_t n_selected;    /* layers persisted at this step                    */
  uint32_t n_forced;      /* selected by the staleness guard alone            */
  uint64_t payload_bytes; /* sum of record sizes of the selected layers       */
  int64_t max_age;        /* max_l (t - t_l) after the decision               */
  double weighted_age;    /* sum_l n_l (t - t_l) / sum_l n_l after the decision
                             (Section 3.3 size-weighted staleness), computed as
                             double(integer numerator) / double(integer denominator) */
} lc_select_stats;

typedef struct {
  uint64_t bytes_written; /* bytes of staging written by this call            */
  uint32_t n_packed;      /* records written by this call                     */
  uint32_t next_rank;     /* rank to pass as first_rank of the next call      */
  int32_t done;           /* 1 when every selected layer has been packed      */
  int32_t reserved;
} lc_pack_result;

typedef struct {
  int64_t step;           /* step the records were persisted at               */
  const uint8_t *mask;    /* host [n_layers]: 1 for each layer in the payload */
  const void *payload;    /* device memory, pinned host memory, or pageable
                             host memory: records of the masked layers in
                             ascending layer id (the lc_pack_selected format) */
  uint64_t payload_bytes; /* must equal the sum of their record sizes         */
} lc_version;

/* Tiles this build of the library works in (no GPU work).  A score chunk is
 * the run of one segment's weights that one score-kernel block reduces to one
 * fp64 pair (the fused optimizer steps use the same chunks); a piece is the
 * part of one record block that one pack or unpack block moves; every record
 * block starts record_align bytes aligned and is zero-padded to a multiple of
 * it. */
typedef struct {
  uint32_t chunk_bytes;  /* bytes of weights per score chunk                  */
  uint32_t piece_bytes;  /* bytes per pack / unpack piece                     */
  uint32_t record_align; /* block alignment and padding inside a record (256) */
  uint32_t reserved;
} lc_build_info;

lc_status lc_query_build(lc_build_info *out);

/* Layout query without any GPU work: validates `d` as lc_init_layout does and
 * reports per-layer element counts and record sizes (host arrays of n_layers
 * entries, either may be NULL). */
lc_status lc_query_layout(const lc_layout_desc *d, uint64_t *numel_out,
                          uint64_t *record_bytes_out);

/* Layer-aligned layout (Section 3.4: optimizer state laid out by layer):
 * builds the per-layer chunk and copy tables, allocates the small device
 * state, sets S <- W for every segment, Delta_l = 0 and t_l = t_base for every
 * layer (Section 3.2; the base full checkpoint of Section 3.4 counts as the
 * last persist).  The base selection (every layer, at t_base) is left
 * pending so the caller can pack the base version with lc_pack_selected.
 * Every array must be device (or managed) memory holding its segment's
 * numel elements, as far as HIP can report the allocation's extent;
 * otherwise LC_ERR_INVALID_ARG before any work is enqueued.  Work runs on
 * d->stream; returns once the device state is ready. */
lc_status lc_init_layout(const lc_layout_desc *d, lc_ctx **out);

/* Eq. 1-2 for every layer at decision step `step` (> every earlier step and
 * > t_base):  u_l = mean|W_l - S_l| / (mean|S_l| + eps_w), means taken jointly
 * over all elements of all segments of layer l, accumulated in fp64.
 * ACCUM: Delta_l += u_l and S <- W for all layers in the same pass.
 * SNAPSHOT: Delta_l = u_l.
 * A selection made by lc_select or lc_rebase has already reset Delta_l and
 * t_l of its layers (Eq. 4), so until every one of its records has been
 * packed this call returns LC_ERR_BAD_STATE with the state unchanged (a
 * dropped selection would let recovery fall back to older records and break
 * the staleness bound of Section 3.3).  The base that lc_init_layout leaves
 * pending resets nothing: in ACCUM mode a warm-up may leave it unpacked
 * (this call then drops it); SNAPSHOT mode needs it packed first.
 * Waits for the previous select kernel only when it must learn whether that
 * selection is packed (a selection whose mask was never read); otherwise
 * asynchronous. */
lc_status lc_score_layers(lc_ctx *c, int64_t step);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the score
 * of lc_score_layers with no context and no allocation.  For every layer of
 * the segment list, u_l = mean|W_l - S_l| / (mean|S_l| + eps_w) between its
 * `weight` and `shadow` arrays (the other segment fields are ignored), with
 * the same kernels, chunking and fixed-order sums as lc_score_layers, so u_l
 * is bit-identical to the u_l that lc_score_layers reports for the same
 * arrays.  Nothing is accumulated or written besides u_out: no Delta, no
 * shadow refresh, no state.
 *   segments:     host array, grouped by ascending layer, every layer in
 *                 [0, n_layers) present; weight and shadow device memory of
 *                 numel elements of weight_dtype each
 *   u_out:        device memory, n_layers doubles, written in full
 *   stream:       hipStream_t of the current device (NULL = null stream)
 * The device tables live in one fixed array per GPU of 16 MiB
 * (LC_NOALLOC_SCRATCH_BYTES), which the library holds from the first call
 * on that GPU until the process ends; a layout whose tables exceed it is
 * scored in consecutive batches of whole layers (about 6.9 GB of bf16
 * weights per batch), and a single layer whose tables alone exceed it is
 * refused with LC_ERR_CAPACITY before any work.  The call allocates no
 * device or pinned memory (small host-side tables live in ordinary heap
 * memory until it returns).  Every call on one GPU uses that GPU's array:
 * calls that overlap on one GPU (two host threads, or two streams whose
 * work overlaps) race and give wrong scores.  Argument errors:
 * LC_ERR_INVALID_ARG before any work.  Returns after u_out is written
 * (synchronises the stream). */
lc_status lc_score_layers_static(const lc_segment *segments, uint32_t n_segments, uint32_t n_layers,
                                 int32_t weight_dtype, double eps_w, double *u_out, void *stream);

/* Eq. 3-5 for every layer: K_l = K0_l * lr_scale (lr_scale = s(lr(t)) > 0,
 * finite); select l when Delta_l >= K_l or step - t_l >= S_max; a selected
 * layer gets Delta_l = 0 and t_l = step (Eq. 4), so its record must be packed
 * (lc_pack_selected) before the next score or optimizer step.  Must follow
 * lc_score_layers(step).  Writes the 0/1 mask (host [n_layers]) and stats
 * when the pointers are non-NULL, which waits for the select kernel (it
 * writes its result into pinned host memory, which the call polls; no
 * stream synchronisation); with both NULL the call is asynchronous. */
lc_status lc_select(lc_ctx *c, int64_t step, double lr_scale, uint8_t *mask_out,
                    lc_select_stats *stats_out);

/* Selective persistence (Section 3.2): writes the records of the selected
 * layers of rank >= first_rank (ranks count selected layers in ascending id)
 * into `staging` (device, 256-byte aligned), as many whole records as fit in
 * `capacity` bytes.  Record of layer l: its W blocks, then master (if
 * present), exp_avg and exp_avg_sq blocks (if present); one block per segment in layout
 * order holding the raw little-endian bytes, zero-padded to a multiple of 256
 * bytes.  Records are concatenated without gaps.  SNAPSHOT mode also sets
 * S <- W for the packed layers in the same pass.  Returns LC_ERR_CAPACITY if
 * the record at first_rank alone exceeds `capacity`, LC_ERR_INVALID_ARG if
 * `staging` is not device memory with room for the bytes to be written.  Waits for the
 * select kernel's result (polled in pinned host memory) when the mask is not
 * yet on the host; the copy itself is asynchronous. */
lc_status lc_pack_selected(lc_ctx *c, void *staging, uint64_t capacity, uint32_t first_rank,
                           lc_pack_result *out);

/* Composite recovery (Section 3.5, Eq. 8): for each layer the version with the
 * greatest step <= t_fail whose mask holds the layer is restored into W,
 * master, exp_avg, exp_avg_sq and S (<- W); Delta_l = 0, t_l = that step; the
 * next step must exceed t_fail.  A version newer than t_fail is ignored.  No
 * candidate for a layer: LC_ERR_NO_VERSION; two candidates at the same
 * greatest step: LC_ERR_INVALID_ARG.  `chosen_step_out` (host [n_layers] or
 * NULL) receives the step each layer was restored from.  A device payload
 * shorter than its payload_bytes is refused (LC_ERR_INVALID_ARG) before any
 * work is enqueued.  Returns after the restore has completed on the device. */
lc_status lc_restore_composite(lc_ctx *c, const lc_version *versions, uint32_t n_versions,
                               int64_t t_fail, int64_t *chosen_step_out);

/* Hyper-parameters of one AdamW step (decoupled weight decay, bias-corrected
 * moments).  The per-step scalars 1 - beta, 1 / (1 - beta^t) and
 * 1 - lr * weight_decay are formed in double and rounded to float once. */
typedef struct {
  double lr;           /* learning rate of this step, >= 0                     */
  double beta1;        /* first-moment decay, in [0, 1)                        */
  double beta2;        /* second-moment decay, in [0, 1)                       */
  double eps;          /* added to sqrt(v_hat), > 0                            */
  double weight_decay; /* decoupled decay for segments flagged in decay_mask   */
  int64_t adam_step;   /* bias-correction step count t >= 1                    */
} lc_adamw_params;

/* Full base checkpoint at `step` (Section 3.4: selective persistence stays
 * off during the warm-up window, which ends with a full checkpoint that is
 * the fallback for rarely updated layers).  Every layer counts as persisted
 * at `step`: Delta_l = 0, t_l = step, S <- W when the layout has a shadow.
 * Every layer is selected, as after lc_select, for lc_pack_selected to pack
 * (any selection still pending is replaced: the base holds every layer), and
 * the next score or optimizer step waits for that pack as after lc_select.  `step` must not precede the
 * last scored, optimizer or restore step; it may equal it (the warm-up's last
 * optimizer step, then its base).  Warm-up steps before it call
 * lc_adamw_step_score (or nothing) and skip lc_select.  Synchronises the
 * stream.  LC_ERR_BAD_STATE for an earlier step or a poisoned context. */
lc_status lc_rebase(lc_ctx *c, int64_t step);

/* The optimizer step with the drift taken from the update itself (Section 3.4
 * computes the drift inside the optimizer step; AdamW as trained in
 * Section 4.1).  For every element, in fp32 with one rounding per operation:
 *   m <- b1 m + (1-b1) g;  v <- b2 v + (1-b2) g*g;
 *   p_new = p * (1 - lr wd) - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)
 * where p is the fp32 master (or the weights themselves when there is no
 * master); the master, m, v and the weights (round-to-nearest-even image of
 * p_new) are written back.  Eq. 1 is applied to the parameters before and
 * after the update, u_l = mean|p_new - p| / (mean|p| + eps_w), and Eq. 2 adds
 * it to Delta_l.  One pass over the optimizer state: no shadow read or write.
 *   grads:      host array [n_segments] of device pointers, one gradient per
 *               segment, numel elements of grad_dtype (LC_DT_BF16 or LC_DT_F32)
 *   decay_mask: host array [n_segments] of 0/1 (weight decay applies), or
 *               NULL for all segments (the paper's with/without weight-decay
 *               parameter groups)
 * Requires LC_MODE_ACCUM and `step` greater than every earlier step; follows
 * the same call sequence as lc_score_layers (select and pack next) and, like
 * it, returns LC_ERR_BAD_STATE while a selection made by lc_select or
 * lc_rebase is not fully packed.  The
 * shadow is left as it was, so lc_score_layers is refused afterwards until a
 * restore or lc_rebase re-synchronises it.  Asynchronous. */
lc_status lc_adamw_step_score(lc_ctx *c, int64_t step, const void *const *grads, int32_t grad_dtype,
                              const uint8_t *decay_mask, const lc_adamw_params *p);

/* Hyper-parameters of one plain SGD step (decoupled weight decay). */
typedef struct {
  double lr;           /* learning rate of this step, >= 0                     */
  double weight_decay; /* decoupled decay for segments flagged in decay_mask   */
} lc_sgd_params;

/* The same for plain SGD, to which Section 4.7 notes the method carries over
 * (records then need no optimizer state: a layout without Adam moments).  For
 * every element, in fp32 with one rounding per operation:
 *   p_new = p * (1 - lr wd) - lr * g      (the decay only where decay_mask)
 * where p is the fp32 master (or the weights themselves when there is no
 * master); the master and the weights (round-to-nearest-even image of p_new)
 * are written back; Adam moments, if the layout has them, are not touched.
 * Eq. 1 on the parameters before and after the update, Eq. 2 into Delta_l.
 * Arguments, call sequence and errors as lc_adamw_step_score, except that no
 * moments are needed.  Asynchronous. */
lc_status lc_sgd_step_score(lc_ctx *c, int64_t step, const void *const *grads, int32_t grad_dtype,
                            const uint8_t *decay_mask, const lc_sgd_params *p);

/* ---- Persistence store (Section 3.5: reconstruction from persisted metadata) --
 * A directory of version files plus an append-only manifest recording the
 * persistence history: per version its step, its layer mask and its payload
 * (records in the lc_pack_selected format).  A version is visible once its
 * file is complete and fsync'ed and its manifest line ("LCV1 <step> <bytes>
 * <file> <mask as 0/1 characters>") is written and fsync'ed; on open, torn or
 * inconsistent lines, files of the wrong size and names other than a plain
 * "v*.lcr" file of the directory itself are ignored.  A store is
 * used from one thread; it owns a small pool of writer threads, and versions
 * become visible in the order they were appended.  A directory is open in at
 * most one store at a time (an exclusive lock on its "store.lock" file, held
 * until lc_store_close): a second lc_store_open of it, from this process or
 * another, returns LC_ERR_BAD_STATE.  Any failed file operation (create,
 * open, read, write, fsync, rename, lock) returns LC_ERR_IO with the path and
 * errno in lc_last_error().  A writer thread's failure drops the version it
 * was writing (the manifest never names it) and is reported by the call that
 * meets it and by every later append, lc_store_sync and compaction, all with
 * LC_ERR_IO; the history already durable stays readable. */
typedef struct lc_store lc_store;

/* Opens (creating the directory itself, not its parents) the store of a
 * layout with the given per-layer record sizes (lc_query_layout /
 * lc_record_bytes).  buffer_bytes is the size of the pinned drain ring
 * (0: 1 GiB; at least 1 MiB), cut into slots of at most 64 MiB: a device
 * payload that fits in it is copied out at host-link speed while the files
 * are written behind it.  The ring is allocated on the first device append. */
lc_status lc_store_open(const char *dir, uint32_t n_layers, const uint64_t *record_bytes, uint64_t buffer_bytes,
                        lc_store **out);

/* Appends one version: `payload` holds the records of the layers in `mask`
 * (host [n_layers], 0/1), payload_bytes their total size.  Device payloads
 * (e.g. the staging buffer of lc_pack_selected) are copied out through the
 * pinned buffers on a store-owned stream that first waits for the work
 * already enqueued on `stream` (hipStream_t, NULL = null stream); `stream`
 * then waits for those copies, so later work on it may reuse the buffer.  The
 * call returns once every copy is enqueued (it blocks while the ring is full);
 * the files are written by the writer threads.  Host payloads are
 * written before the call returns.  A layer may be stored at most once per
 * step (several versions of one step must have disjoint masks). */
lc_status lc_store_append(lc_store *s, int64_t step, const uint8_t *mask, const void *payload,
                          uint64_t payload_bytes, void *stream);

/* The same append, overlapped with the caller's next steps (the staging drain
 * of Section 3.5 runs beside training instead of in its stream): `stream`
 * does NOT wait for the copies out of a device payload.  Instead the store
 * records `reuse_event` (a hipEvent_t the caller created; required for a
 * device payload) on its own stream behind the last copy, and the caller must
 * order any later write to the payload after it (hipStreamWaitEvent, or
 * hipEventSynchronize) -- typically by alternating between two staging
 * buffers and waiting on the event of the one about to be packed again.  The
 * event is re-recorded by every call that is given it.  For a host payload
 * (written before the call returns) the event, if given, is recorded on
 * `stream`.  The call still blocks while the pinned ring is full.  Errors as
 * lc_store_append; after an error return nothing reads the payload any more. */
lc_status lc_store_append_async(lc_store *s, int64_t step, const uint8_t *mask, const void *payload,
                                uint64_t payload_bytes, void *stream, void *reuse_event);

/* Waits until every appended version is durable and visible.  After an I/O
 * failure of the writers (a full disk, say) the failed version is dropped and
 * this and every later append return LC_ERR_BAD_STATE with the error. */
lc_status lc_store_sync(lc_store *s);

/* Visible versions, in manifest order. */
lc_status lc_store_count(lc_store *s, uint32_t *n_out);
lc_status lc_store_entry(lc_store *s, uint32_t i, int64_t *step_out, uint8_t *mask_out /* [n_layers] or NULL */,
                         uint64_t *bytes_out);

/* The reconstruction plan (Section 3.5 step 1) over the visible versions:
 * per layer the greatest stored step <= t_fail holding it (host
 * [n_layers]); LC_ERR_NO_VERSION / LC_ERR_INVALID_ARG as for
 * lc_restore_composite. */
lc_status lc_store_plan(lc_store *s, int64_t t_fail, int64_t *chosen_step_out);

/* Composite recovery from the store (Section 3.5 steps 2-3): reads only the
 * chosen record of every layer and restores it into the context's arrays
 * exactly as lc_restore_composite does.  The records stream in 64 MiB pieces
 * through a 2 GiB pinned ring (allocated for the call) that eight reader
 * threads fill while the host-to-device copies of earlier pieces run.  The
 * context's layout must match the store's record sizes.  Returns after the
 * restore has completed on the device. */
lc_status lc_store_restore(lc_store *s, lc_ctx *c, int64_t t_fail, int64_t *chosen_step_out);

/* Storage reclamation: removes the versions that no reconstruction plan with
 * t_fail >= t_keep can choose (Section 3.5), i.e. keeps every non-empty
 * version after t_keep and, per layer, the newest version at or before t_keep
 * holding it; plans for t_fail >= t_keep are unchanged.  t_keep = the newest
 * stored step keeps exactly the latest record of every layer.  Waits for
 * pending writes first.  The manifest is replaced atomically (temporary file,
 * fsync, rename, directory fsync) before any version file is removed, so a
 * crash leaves either the old history or the new one; files that no manifest
 * line names are removed too.  `removed_out` (or NULL) receives the number of
 * files removed. */
lc_status lc_store_compact(lc_store *s, int64_t t_keep, uint32_t *removed_out);

/* Recovery timeline: after a restore at t_fail, training continues from
 * t_fail + 1 and versions persisted after t_fail belong to the abandoned run.
 * Removes every visible version with a step greater than `step` (the
 * manifest is rewritten atomically first, as for lc_store_compact) so the
 * resumed run can append its own versions of those steps.  Waits for pending
 * writes first.  `removed_out` (or NULL) receives the number of files
 * removed. */
lc_status lc_store_discard_after(lc_store *s, int64_t step, uint32_t *removed_out);

/* Waits for pending writes, stops the writer and frees the store. */
lc_status lc_store_close(lc_store *s);

/* Synchronises the stream and copies the per-layer state to host arrays of
 * n_layers entries (any may be NULL): the last scores u_l, accumulators
 * Delta_l and last-persist steps t_l. */
lc_status lc_read_state(lc_ctx *c, double *u_out, double *delta_out, int64_t *t_last_out);

/* Record size of one layer in bytes (0 for a bad id or NULL context). */
uint64_t lc_record_bytes(const lc_ctx *c, uint32_t layer);

/* Synchronises the stream and frees the context (NULL is a no-op). */
lc_status lc_destroy(lc_ctx *c);

/* Message for the last failing call on this thread ("" if none). */
const char *lc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LAYERCHECK_H */
