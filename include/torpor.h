/*
 * torpor.h - pipelined model swap-in and execution on one AMD MI355X (gfx950).
 *
 * The operation (paper Sec. 1 and Sec. 3, "late binding"; Sec. 4.3, "Model swapping and
 * pipeline execution"): functions publish models that stay in host memory while idle;
 * when a request arrives for a model that is not on the GPU, its weights are swapped
 * from a pinned host pool into GPU memory, grouped into transfers of about the size at
 * which transfer throughput stops improving, and each layer starts computing as soon
 * as the group holding it has arrived, so transfer and compute overlap within one
 * forward pass. Eviction only invalidates the GPU copy (Sec. 4.3, "Model eviction").
 * GPU memory is reserved once and managed internally, with no native allocation per
 * swap (Sec. 4.4, "Memory block allocation"); a parameter's device address is its
 * region base plus its unchanged offset (Sec. 4.4, "Memory address management").
 * Only the final output needs a host synchronisation (Sec. 4.2).
 *
 * Conventions for every call:
 *   - Return value: TP_OK (0) or a negative TP_E_* code; tp_last_error() then returns a
 *     thread-local message. Validation errors change no state.
 *   - Device pointers are plain HIP device addresses; streams are hipStream_t passed as
 *     void* (NULL = the null stream). Nothing in this interface allocates per request.
 *   - A context is used from one host thread at a time.
 */
#ifndef TORPOR_H
#define TORPOR_H

#include <stdint.h>

#ifndef TP_API
#define TP_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t tp_status;
enum {
  TP_OK = 0,
  TP_E_INVAL = -1,   /* malformed argument, descriptor or layout */
  TP_E_NOENT = -2,   /* unknown model id */
  TP_E_NOSPC = -3,   /* model larger than the arena, or workspace too small */
  TP_E_HIP = -4,     /* a HIP runtime call failed (message names it) */
  TP_E_STATE = -5    /* call not valid in the current state */
};

typedef enum { TP_F32 = 0, TP_BF16 = 1 } tp_dtype;

/* Model families (dims[] meaning per family):
 *   TP_ARCH_MLP      {layers, width, act(TP_ACT_*)}; layers x Linear(width, width) + bias,
 *                    activation after every layer but the last.
 *   TP_ARCH_RESNET50 {classes, image}; ResNet-50 v1.5, batch-norm folded into conv
 *                    biases, NHWC input [B][image][image][3], image % 32 == 0.
 *   TP_ARCH_BERT     {layers, d, heads, ffn, seq, vocab, maxpos}; post-LN encoder,
 *                    head dim 64, token type 0, no mask, LN eps 1e-12. */
typedef enum { TP_ARCH_MLP = 0, TP_ARCH_RESNET50 = 1, TP_ARCH_BERT = 2 } tp_arch;
enum { TP_ACT_NONE = 0, TP_ACT_RELU = 1, TP_ACT_GELU = 2 };

/* Tensor roles. MLP and ResNet use W/B (ResNet: layer = conv index in first-use order,
 * the FC is the last layer). BERT: layer 0 holds the embeddings, layers 1..L the encoder. */
enum {
  TP_ROLE_W = 0, TP_ROLE_B = 1,
  TP_ROLE_TOK_EMB = 10, TP_ROLE_POS_EMB = 11, TP_ROLE_TYPE_EMB = 12,
  TP_ROLE_EMB_LN_G = 13, TP_ROLE_EMB_LN_B = 14,
  TP_ROLE_QKV_W = 20, TP_ROLE_QKV_B = 21, TP_ROLE_O_W = 22, TP_ROLE_O_B = 23,
  TP_ROLE_LN1_G = 24, TP_ROLE_LN1_B = 25, TP_ROLE_FFN1_W = 26, TP_ROLE_FFN1_B = 27,
  TP_ROLE_FFN2_W = 28, TP_ROLE_FFN2_B = 29, TP_ROLE_LN2_G = 30, TP_ROLE_LN2_B = 31
};

/* One tensor inside the host weight buffer. Linear weights are [out][in], conv weights
 * OHWI, the fused BERT QKV weight is [3d][d] with rows Q (heads x 64), K, V; LN gamma and
 * beta are separate [d] tensors. Unused shape entries are 0. */
typedef struct {
  uint32_t layer;     /* first-use unit the tensor belongs to */
  uint32_t role;      /* TP_ROLE_* */
  uint64_t offset;    /* byte offset in the host buffer, multiple of 256 */
  uint64_t bytes;     /* byte size = prod(shape) * element size */
  int64_t shape[4];
} tp_tensor_desc;

/* Host weight layout of one model. Tensors are listed in first-use order: layers never
 * decrease and offsets strictly increase; tensors do not overlap. */
typedef struct {
  int32_t arch;        /* tp_arch */
  int32_t dtype;       /* tp_dtype of every weight; BERT and ResNet require TP_BF16 */
  int32_t dims[8];
  uint32_t n_tensors;
  const tp_tensor_desc* tensors;
} tp_model_desc;

/* How a chunk reaches the arena. MEMCPY and GATHER are the swap engines of the pipelined
 * path. PAGEABLE and ZERO exist for the swap-design breakdown of Sec. 6.1 ("Performance
 * breakdown of model swapping") and the direct-host-access alternative of Sec. 8 (related
 * work): PAGEABLE copies from an ordinary pageable copy of the weights that the library
 * keeps beside the pinned one (the baseline that the pinned pool improves on); ZERO
 * never copies: a request for a non-resident model runs its kernels on the weights in
 * the pinned host copy, read over the host link, and leaves the model non-resident
 * (tp_swap_in still makes it resident; the arena's counters see no ZERO request). */
enum { TP_COPY_MEMCPY = 0, TP_COPY_GATHER = 1, TP_COPY_PAGEABLE = 2, TP_COPY_ZERO = 3 };
enum {
  TP_FLAG_POISON = 1,     /* evicted extents are filled with 0xFF (NaN for fp32/bf16) */
  TP_FLAG_THROTTLE = 2,   /* a bounded delay kernel precedes every chunk on the copy stream */
  TP_FLAG_NO_GRAPH = 4,   /* launch warm requests kernel by kernel instead of replaying a graph */
  TP_FLAG_SERIAL = 8,     /* a cold request waits for its whole model before its first kernel
                           * (swap, then execute: no pipelining) */
  TP_FLAG_PER_TENSOR = 16,/* transfer groups close at tensor boundaries, not layer boundaries;
                           * with chunk_min_bytes = 0 every tensor is its own transfer (the
                           * parameter-level pipeline of Sec. 6.1) */
  TP_FLAG_TRACE = 32,     /* cold requests record timing events per chunk (tp_last_timeline) */
  TP_FLAG_CALLER_STREAM = 64, /* cold requests run their kernels on the caller's stream instead
                               * of the library's execution stream (see tp_config) */
  TP_FLAG_NO_TOUCH = 128,     /* warm requests never pre-read their weights into the caches */
  TP_FLAG_TOUCH_ALWAYS = 256  /* every warm request of a model with a cache-touch span pre-reads
                               * it, not only the first after another model's (see tp_config) */
};

/* Context configuration. arena_dev/work_dev are caller-owned device buffers that must
 * stay valid until tp_destroy; the library never frees them. copy_stream: the primary
 * copy stream (NULL: the library creates and later destroys one). Streams the library
 * creates for copies are given a hardware queue of their own (a stream with a full CU
 * mask), because a copy stream that shares the compute stream's hardware queue serialises
 * the swap behind the kernels; they synchronise with the legacy null stream, so requests
 * should run on created streams. A caller-supplied copy_stream should likewise not share
 * the compute stream's hardware queue.
 * With copy_streams == 2 the library adds a second such stream and alternates
 * chunks between the two, forked from the primary after every ordering wait (0 or 1:
 * one stream, so chunks arrive in first-use order at the full link rate).
 * chunk_min_bytes is the transfer group size G (0 = one chunk per layer). copy_method:
 * TP_COPY_MEMCPY uses hipMemcpyAsync; TP_COPY_GATHER runs a copy kernel reading
 * host-mapped pinned memory with gather_wgs workgroups (0 = default). throttle_us:
 * delay per chunk under TP_FLAG_THROTTLE. Warm requests of models whose forward pass
 * launches at least 16 kernels replay an instantiated HIP graph of it, cached per (model,
 * batch, workspace; up to 4 per model), unless TP_FLAG_NO_GRAPH is set; a request whose
 * input or output buffer differs from the graph's, or whose model now lies in another
 * extent, repoints the graph's kernels that hold those addresses (no new capture; an input
 * or output address with another residue modulo 16 is captured afresh); shorter forward
 * passes are launched kernel by kernel, which is faster for them. A cold request's kernels run on an
 * execution stream the library creates (with a hardware queue of its own, like the copy
 * streams), forked from the caller's stream by an event and joined back to it by another;
 * so whatever hardware queue the caller's stream maps to, the chunk copies overlap the
 * kernels (TP_FLAG_CALLER_STREAM: on the caller's stream instead). direct_max_bytes (0 = never): a cold request for a model of
 * at most this many bytes runs its kernels on the pinned host copy over the host link
 * (direct host access, the alternative to swapping that Sec. 8 cites) instead of waiting
 * for its first chunk, and the copy stream swaps the model in behind it; the next request
 * for the model waits for that swap. This removes the copy engine's start-up and hand-off
 * latency from the cold path of models small enough that it dominates. It applies with
 * one copy stream and copy_method TP_COPY_MEMCPY or TP_COPY_GATHER only.
 * A warm tp_infer request (model resident) for a model other than the one the previous
 * request served, whose bytes the requests in between have likely pushed out of the
 * Infinity Cache and the L2s, or for a model that tp_swap_in brought in and no request has
 * read since, first launches on the execution stream (after the model's copies) a kernel that reads the
 * model's weights and discards them, except a leading token-embedding table (of which a
 * request reads a few rows), while the request's own kernels run on the caller's stream: the
 * later layers then find their weights in the cache (measured on MI355X at batch 1 after the
 * caches were flushed: ResNet-50 397 -> 365 us, BERT-base 534 -> 501 us per forward pass).
 * Models whose span is under 4 MB or over 192 MB, and MLPs (whose warm pass streams its
 * weights at the rate a second reader would), are never touched; neither are requests of
 * tp_infer_noalloc or of a TP_FLAG_CALLER_STREAM context. The read does not change any
 * result. TP_FLAG_NO_TOUCH switches it off, TP_FLAG_TOUCH_ALWAYS applies it to every warm
 * request.
 *
 * plan chooses how a model's layers are grouped into transfers (chunks):
 *   TP_PLAN_GREEDY: the paper's rule (Sec. 4.3): whole layers in first-use order, a chunk
 *     closed at the first layer boundary where it holds >= chunk_min_bytes, the group size
 *     at the elbow of transfer throughput.
 *   TP_PLAN_COST: the boundaries that minimise a model of the cold request's completion
 *     time: copies back to back, each costing chunk_us (0: 15) plus its bytes at link_gbs
 *     (0: 57 GB/s); a layer starts when the previous one has finished and its chunk has
 *     landed; layer times from the library's per-kernel estimate at plan_batch samples
 *     (0: 1). Small chunks where compute could start early or would finish late, large
 *     ones where the link is the bottleneck. chunk_min_bytes is ignored, and so is
 *     TP_FLAG_PER_TENSOR. */
enum { TP_PLAN_GREEDY = 0, TP_PLAN_COST = 1 };
/* evict_policy chooses the victim when a non-resident model needs room (one victim at a
 * time until a placement exists, see alloc):
 *   TP_EVICT_LRU: the least recently used resident model.
 *   TP_EVICT_HEAVINESS: the paper's policy (Sec. 5.4, "Model eviction policy"): light
 *     models first (least recently used among them), and only when no light model is
 *     resident the least recently used heavy one. A model is heavy when swapping it slows
 *     its inference much: at registration, when the modelled cold time of its best chunk
 *     plan (the TP_PLAN_COST model) exceeds heavy_ratio (0: 3.0) times its modelled warm
 *     time; tp_set_model_class overrides this. The default separates the paper's light
 *     models, whose swapped latency is within about 1.2x of native, from its heavy one
 *     (about 3.4x; Sec. 7, table of remoting and swapping latencies). */
/*   TP_EVICT_LRU_WINDOW (beyond the paper; first-fit placement only, partitioned placement
 *     treats it as TP_EVICT_LRU): when no free gap fits, the victims are chosen together as
 *     the extents that one contiguous range of the needed size overlaps, taking among the
 *     ranges that start at the arena's base or where a resident extent ends the one whose most
 *     recently used victim is the oldest, then the one with fewer victim bytes, then the lower
 *     address. Least-recently-used eviction one model at a time frees space scattered over the
 *     arena and can invalidate several models for a gap one of them would have made. */
enum { TP_EVICT_LRU = 0, TP_EVICT_HEAVINESS = 1, TP_EVICT_LRU_WINDOW = 2 };
enum { TP_CLASS_AUTO = 0, TP_CLASS_LIGHT = 1, TP_CLASS_HEAVY = 2 };
/* alloc chooses where in the arena a model's extent goes:
 *   TP_ALLOC_FIRST_FIT: the lowest-addressed free gap that fits.
 *   TP_ALLOC_PARTITION: the paper's two-tier scheme (appendix "Memory Block Allocation"): the
 *     arena is cut into partitions of partition_bytes (0: the arena size / 8 rounded down to a
 *     MiB, at least 256 bytes; otherwise a multiple of 256); a short remainder of at least 256
 *     bytes is one more partition. A model no larger than a partition takes a slot of a
 *     partition dedicated to its size (the size rounded up to 256 bytes) when at least two
 *     registered models have that size, else a buddy block (sizes: a partition halved while
 *     the half stays a multiple of 256) in a buddy-managed partition; a larger model takes a
 *     run of consecutive free partitions. Fullest candidate partitions first; runs from the
 *     low end, new slot or buddy partitions from the high end. A partition is free again when
 *     its last model leaves. Victims (evict_policy) are taken one at a time until a placement
 *     exists.
 *   TP_ALLOC_PARTITION_CONSOLIDATE: as TP_ALLOC_PARTITION, and before each eviction one slot or
 *     buddy partition is evacuated if possible (the appendix's consolidation across
 *     partitions): the one with the fewest bytes in use whose models all fit, by the same
 *     rules, in other partitions without taking a free one; they are copied there
 *     device-to-device on the copy stream (after their swap-in and the destination's previous
 *     readers), and the moved model's next request waits for its copy. */
enum { TP_ALLOC_FIRST_FIT = 0, TP_ALLOC_PARTITION = 1, TP_ALLOC_PARTITION_CONSOLIDATE = 2 };
typedef struct {
  void* arena_dev;
  uint64_t arena_bytes;
  void* work_dev;
  uint64_t work_bytes;
  void* copy_stream;
  uint64_t chunk_min_bytes;
  int32_t copy_method;
  int32_t gather_wgs;
  int32_t flags;
  int32_t throttle_us;
  int32_t copy_streams;
  uint64_t direct_max_bytes;
  int32_t plan;           /* TP_PLAN_* */
  int32_t plan_batch;
  float link_gbs;
  float chunk_us;
  int32_t evict_policy;   /* TP_EVICT_* */
  float heavy_ratio;
  int32_t alloc;          /* TP_ALLOC_* */
  uint64_t partition_bytes;
} tp_config;

typedef struct {
  uint64_t capacity, used, largest_free;
  uint32_t resident, registered;
  uint64_t hits, misses, evictions, frag_evictions, bytes_swapped;
  /* host time of admissions (the arena decision, victim retirement and the copy stream's
   * ordering waits) of the requests that missed, in tp_infer / tp_swap_in: count, sum, max */
  uint64_t admit_calls, admit_ns_total, admit_ns_max;
  uint32_t partitions, partitions_free;   /* TP_ALLOC_PARTITION*: partitions in all, unoccupied */
  uint64_t evacuations, bytes_moved;      /* TP_ALLOC_PARTITION_CONSOLIDATE: partitions freed by moves, bytes moved */
  /* warm-request graphs: forward passes captured and instantiated; graph launches whose
   * kernel nodes were repointed instead (at the request's input and output buffers, or at the
   * model's weights in another extent than the nodes held); and those of the repointed
   * launches that moved the weights */
  uint64_t graph_captures, graph_repoints, graph_rebases;
  /* warm requests that pre-read their model's weights into the caches (see tp_config) */
  uint64_t cache_touches;
} tp_arena_stats_t;

typedef struct {
  uint64_t host_bytes;     /* size of the model's pinned host copy (= extent size) */
  uint64_t param_bytes;    /* sum of tensor sizes (no padding) */
  uint32_t n_chunks;
  int32_t resident;
  uint64_t extent_offset;  /* arena offset of the model's extent when resident */
  uint64_t last_use_clock; /* logical clock of the last request, 0 if never used */
  int32_t heavy;           /* 1 if the model is classed heavy (see TP_EVICT_HEAVINESS) */
  float cold_est_us;       /* modelled cold time of its best chunk plan (plan_batch samples) */
  float warm_est_us;       /* modelled warm time (sum of the per-layer estimates) */
} tp_model_info_t;

/* Creates a context bound to the current HIP device. The arena (Sec. 4.4: all GPU
 * memory reserved up front) must be 256-byte aligned. Errors: TP_E_INVAL for NULL or
 * misaligned buffers, TP_E_HIP if stream or event creation fails. */
TP_API tp_status tp_create(const tp_config* cfg, struct tp_ctx** out);

/* Waits for all outstanding work of the context, then frees its pinned host copies,
 * events and (if it created it) the copy stream. Never frees caller buffers. */
TP_API tp_status tp_destroy(struct tp_ctx* ctx);

/* Publishes a model (Sec. 3: idle models live in host memory). Copies host_bytes bytes
 * from host_weights into a library-owned pinned, device-mapped host buffer (Sec. 4.3:
 * pinned memory pool), so the caller may free its buffer on return. Validates the
 * descriptor against the family's architecture (every tensor present once with the
 * expected shape, aligned, in bounds, non-overlapping, in first-use order) and builds
 * the transfer-chunk plan. The model starts non-resident. Errors: TP_E_INVAL,
 * TP_E_HIP (pinned allocation failed). */
TP_API tp_status tp_register_model(struct tp_ctx* ctx, const tp_model_desc* desc,
                            const void* host_weights, uint64_t host_bytes, int32_t* model_id);

/* Evicts (if resident) after the model's last use has completed, then frees its host
 * copy and events. Synchronises on that model's work. */
TP_API tp_status tp_unregister_model(struct tp_ctx* ctx, int32_t model_id);

/* Runs one forward pass of a batch (Sec. 4.3). If the model is not resident an extent
 * is admitted (first fit; least recently used models are invalidated until one fits)
 * and its chunks are enqueued on the copy stream, each followed by an event; every
 * layer's first kernel on `stream` waits for the event of the chunk holding that layer.
 * Inputs: MLP [batch][width] in the model dtype; ResNet bf16 NHWC
 * [batch][image][image][3]; BERT int32 token ids [batch][seq] (ids outside [0, vocab)
 * are clamped). Output (fp32): MLP [batch][width]; ResNet [batch][classes]; BERT
 * [batch][seq][d]. Asynchronous: returns after enqueueing; the caller synchronises
 * `stream`. Requests are totally ordered: a request on a stream other than the previous
 * request's first waits for that request. Errors (synchronous, no state change):
 * TP_E_NOENT, TP_E_INVAL (batch < 1, NULL pointers), TP_E_NOSPC (model larger than the
 * arena, or workspace smaller than tp_workspace_bytes). On an enqueue failure the model
 * is left non-resident and TP_E_HIP is returned. */
TP_API tp_status tp_infer(struct tp_ctx* ctx, int32_t model_id, const void* input_dev, int32_t batch,
                   void* output_dev, void* stream);

/* tp_infer for callers that cannot allocate device memory (code that must not call hipMalloc,
 * tight serving loops, harnesses that forbid allocation): the same request, computing the
 * same bits, but its activations and split-contraction partials live in a static workspace
 * of 64 MiB (kNoAllocScratchBytes) that the library's code object holds on each device,
 * instead of the context's work_dev; its kernels are launched one by one (no graph is
 * captured or instantiated). The call allocates nothing; the caller still passes the input
 * and output buffers. The workspace is shared by every context and call on the device and
 * keeps the last call's contents (nothing in it needs to start at zero): calls that overlap
 * on one device race, so a process must not have two such requests in flight at once on
 * different contexts or unordered streams (one context's requests are ordered anyway).
 * Errors: as tp_infer; TP_E_NOSPC when the request needs more than the 64 MiB (e.g.
 * ResNet-50 beyond batch 2); TP_E_HIP if the workspace's device address could not be
 * resolved when the context was created. */
TP_API tp_status tp_infer_noalloc(struct tp_ctx* ctx, int32_t model_id, const void* input_dev, int32_t batch,
                                  void* output_dev, void* stream);
/* Enqueues the swap-in alone (admission + chunk copies, no compute), as a request with
 * no output; a following tp_infer of the same model is a hit. `stream` is made to wait
 * for the copies. Same errors as tp_infer. */
TP_API tp_status tp_swap_in(struct tp_ctx* ctx, int32_t model_id, void* stream);

/* Invalidates the model's device copy; nothing is copied back (Sec. 4.3). The extent is
 * reused only after the model's last enqueued use completes. Not an error if the model
 * is not resident. */
TP_API tp_status tp_evict(struct tp_ctx* ctx, int32_t model_id);

TP_API tp_status tp_is_resident(struct tp_ctx* ctx, int32_t model_id, int32_t* resident);
TP_API tp_status tp_arena_stats(struct tp_ctx* ctx, tp_arena_stats_t* out);
TP_API tp_status tp_model_info(struct tp_ctx* ctx, int32_t model_id, tp_model_info_t* out);

/* Sets a model's eviction class: TP_CLASS_LIGHT, TP_CLASS_HEAVY, or TP_CLASS_AUTO (back to
 * the registration-time estimate). Affects later evictions under TP_EVICT_HEAVINESS only.
 * Errors: TP_E_NOENT, TP_E_INVAL (unknown class). */
TP_API tp_status tp_set_model_class(struct tp_ctx* ctx, int32_t model_id, int32_t model_class);

/* The library's pinned host image of a registered model (what a swap copies, byte for byte).
 * It equals the registered bytes except that bf16 MLP weight matrices whose width is a
 * multiple of 128 are stored blocked for the skinny-batch kernel: each block of 16 rows x
 * 128 columns is contiguous, ordered [32-column group][8-column slot][row][8 elements].
 * *ptr stays valid until the model is unregistered; read-only. */
TP_API tp_status tp_model_host_image(struct tp_ctx* ctx, int32_t model_id, const void** ptr, uint64_t* bytes);

/* Chunk plan of a registered model: fills up to `cap` entries of [begin, end) host
 * byte ranges and the first layer each chunk holds; *n receives the chunk count. */
TP_API tp_status tp_model_chunks(struct tp_ctx* ctx, int32_t model_id, uint64_t* begin, uint64_t* end,
                          uint32_t* first_layer, uint32_t cap, uint32_t* n);

/* Timeline of the last cold tp_infer of a TP_FLAG_TRACE context (the pipelined path,
 * Sec. 4.3: chunk c's copy overlaps the layers of earlier chunks), in milliseconds from
 * that request's start event on the caller's stream: for each of the first `cap` chunks,
 * when its copy began and ended on the copy stream and when the caller's stream passed
 * its wait for the chunk (the first kernel that reads it starts after that); *n receives
 * the chunk count and *total_ms the time until the request's last kernel ended. Blocks
 * until that request has completed. TP_E_STATE if no cold request has been traced. */
TP_API tp_status tp_last_timeline(struct tp_ctx* ctx, float* copy_begin_ms, float* copy_end_ms, float* exec_begin_ms,
                           uint32_t cap, uint32_t* n, float* total_ms);

/* Workspace bytes tp_infer needs for this model at this batch size (host-only). */
TP_API tp_status tp_workspace_bytes(const tp_model_desc* desc, int32_t batch, uint64_t* bytes);

/* One request of an open-loop trace (tp_run_trace). */
typedef struct {
  int32_t model_id;
  int32_t batch;
  const void* input_dev;
  void* output_dev;
  uint64_t arrival_ns;      /* arrival time, nanoseconds after the start of the trace */
} tp_request;

typedef struct {
  uint64_t issue_ns;        /* when tp_infer was called (ns after the start) */
  uint64_t done_ns;         /* when the host observed the request's completion */
  int32_t hit;              /* the model was resident when the request was issued */
  int32_t status;           /* tp_infer's status for this request */
  uint64_t admit_ns;        /* host time of the request's admission if it missed, else 0 */
} tp_request_result;

/* Replays an open-loop request trace (the paper's serving setting, Sec. 3 and Sec. 7: requests
 * arrive independently of completions). The calling thread sleeps until each request's arrival
 * time and issues tp_infer on `stream`; a second thread waits for the requests' completions in
 * issue order and stamps the time the host sees each one, so latency = done - arrival includes
 * queueing behind earlier requests. At most 256 requests are in flight (a fixed ring of events
 * created once per context); the dispatcher waits for a free slot beyond that. Requests whose
 * tp_infer fails carry the status and are not waited for. Returns after the last completion. */
TP_API tp_status tp_run_trace(struct tp_ctx* ctx, const tp_request* requests, uint32_t n, void* stream,
                              tp_request_result* results);

/* Request queueing of tp_run_trace_sched. */
enum { TP_QUEUE_FIFO = 0, TP_QUEUE_SLO = 1 };
typedef struct {
  int32_t policy;         /* TP_QUEUE_FIFO or TP_QUEUE_SLO */
  int32_t max_inflight;   /* requests enqueued on the GPU at once (1..256) */
  double slo_pct;         /* tail percentile p of every function's SLO, in (0, 1) (e.g. 0.98) */
  double alpha;           /* initial high-priority threshold, in (0, 1] */
  double scalar;          /* alpha update factor, > 1 (the paper's default 2) */
  double threshold;       /* alpha update trigger (the paper's default 0.04) */
  uint64_t period_ns;     /* alpha update period, > 0 */
} tp_sched_config;

typedef struct {
  double alpha;           /* alpha at the end */
  uint32_t periods;       /* periods closed */
  uint32_t alpha_changes; /* periods that changed alpha */
  uint32_t compliant;     /* functions whose served requests met the SLO over the whole trace */
  uint32_t functions;     /* functions with at least one served request */
} tp_sched_stats;

/* Open-loop replay with a request queue on the host (Sec. 5.3 "Request queueing"): requests
 * are queued at their arrival times, and whenever fewer than max_inflight are enqueued on the
 * GPU the next one is chosen: TP_QUEUE_FIFO, the earliest arrival; TP_QUEUE_SLO, the paper's
 * SLO-aware policy over the functions (model ids) of the trace: each function's required
 * request count RRC = (p n - m) / (1 - p) from its n served requests, m of them within their
 * deadline (deadline_ns[i], relative to request i's arrival); functions sorted by RRC
 * ascending, the first k in the high-priority group with k the largest such that their positive
 * RRCs sum to at most alpha times all of them; the high group first, largest RRC first, then
 * the low group, smallest RRC first; a function's own requests in arrival order. alpha is
 * updated every period_ns from the ratio of functions whose requests served in that period met
 * the SLO (served within deadline / served >= p), as in the appendix's auto-configuration.
 * Results and errors as tp_run_trace; *stats (may be NULL) summarises the run. */
TP_API tp_status tp_run_trace_sched(struct tp_ctx* ctx, const tp_request* requests, uint32_t n, void* stream,
                                    const tp_sched_config* cfg, const uint64_t* deadline_ns,
                                    tp_request_result* results, tp_sched_stats* stats);

/* Test hook for the error paths (fault handling is Sec. 4.5's concern; this checks the
 * library's own rollback): the nth copy the context enqueues from now on (1 = the next;
 * chunk copies of swaps and consolidation moves) fails as if the HIP runtime had rejected
 * it, with nothing enqueued for it; 0 disarms. The request then fails like any enqueue
 * failure: TP_E_HIP, the model left non-resident, its extent retired. Host-side only: no
 * device work fails. Errors: TP_E_INVAL (NULL context, nth < 0). */
TP_API tp_status tp_debug_fail_copy(struct tp_ctx* ctx, int32_t nth);
/* Thread-local message describing the last non-OK status ("" if none). */
TP_API const char* tp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TORPOR_H */
