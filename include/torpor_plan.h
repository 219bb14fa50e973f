/*
 * torpor_plan.h - host-only planning calls of libtorpor (no GPU needed).
 *
 * They expose the bookkeeping the runtime uses, so that capacity planners (and the
 * test suite) can ask what a request sequence would do without touching a device:
 * descriptor validation, the transfer-chunk plan (paper Sec. 4.3: parameters grouped
 * into transfers of about the throughput-elbow size, whole layers per group), and an
 * arena model with first-fit placement and least-recently-used eviction that only
 * invalidates (Sec. 4.3 "Model eviction"; Sec. 4.4 "Memory block allocation"; Sec. 5.4).
 * Same status codes and tp_last_error() as torpor.h.
 */
#ifndef TORPOR_PLAN_H
#define TORPOR_PLAN_H

#include "torpor.h"

#ifndef TP_API
#define TP_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* Validates a descriptor exactly as tp_register_model does. */
TP_API tp_status tph_validate(const tp_model_desc* desc, uint64_t host_bytes);

/* Whether a warm request of this model pre-reads its weights into the caches (the cache touch
 * of tp_config), and which bytes of its extent: *applies = 1 and [*lo, *hi) (offsets into the
 * extent) or *applies = 0 and both 0. The extent minus a leading token-embedding table, for
 * ResNet-50 and BERT models whose span is 4 MB to 192 MB; never for an MLP. */
TP_API tp_status tph_touch_span(const tp_model_desc* desc, uint64_t host_bytes, int32_t* applies, uint64_t* lo,
                                uint64_t* hi);

/* Chunk plan for group size chunk_min_bytes under context flags `flags` (only
 * TP_FLAG_PER_TENSOR matters); same outputs as tp_model_chunks. */
TP_API tp_status tph_plan(const tp_model_desc* desc, uint64_t host_bytes, uint64_t chunk_min_bytes, int32_t flags,
                   uint64_t* begin, uint64_t* end, uint32_t* first_layer, uint32_t cap, uint32_t* n);

/* The cost-model chunk plan of TP_PLAN_COST for this model at plan_batch samples, with
 * link_gbs and chunk_us as in tp_config (0: defaults); same outputs as tph_plan, plus the
 * modelled completion time in *est_us (may be NULL). */
TP_API tp_status tph_plan_cost_model(const tp_model_desc* desc, uint64_t host_bytes, int32_t plan_batch, float link_gbs,
                              float chunk_us, uint64_t* begin, uint64_t* end, uint32_t* first_layer, uint32_t cap,
                              uint32_t* n, double* est_us);

/* The grouping of TP_PLAN_COST over explicit units: n_units units starting at host offsets
 * unit_begin[] (increasing, unit_begin[0] = 0) of a buffer of total_bytes bytes, running
 * for unit_us[] microseconds each; link_bytes_per_us, chunk_us and wait_us model the copies
 * and hand-offs (all > 0 except wait_us >= 0). Writes the first unit of each chunk (up to
 * cap), the chunk count and the modelled completion time. */
TP_API tp_status tph_plan_cost(const uint64_t* unit_begin, const double* unit_us, uint32_t n_units, uint64_t total_bytes,
                        double link_bytes_per_us, double chunk_us, double wait_us, uint32_t* first_unit, uint32_t cap,
                        uint32_t* n_chunks, double* est_us);

/* Per-layer time estimate (us) of the cost model at `batch` samples; *n receives the layer
 * count, up to cap values are written. */
TP_API tp_status tph_layer_costs(const tp_model_desc* desc, uint64_t host_bytes, int32_t batch, double* us, uint32_t cap,
                          uint32_t* n);

/* SLO-aware queueing (Sec. 5.3 "Request queueing"; appendix "Function request
 * prioritization"), as used by tp_run_trace_sched. tph_rrc: *out = (p n - m) / (1 - p), the
 * required request count of a function with n requests served, m of them within the deadline,
 * tail percentile p in (0, 1). */
TP_API tp_status tph_rrc(uint64_t n, uint64_t m, double p, double* out);

/* The request to run next among n_pending queued requests (pending_func: the function of
 * each, in arrival order) of n_funcs functions with counters n[], m[]: functions sorted by
 * RRC ascending (ties: lower index), the first k forming the high-priority group with k the
 * largest such that the positive RRCs of the first k sum to at most alpha times those of all;
 * a high-priority function with the largest RRC first, else the low-priority one with the
 * smallest RRC (ties: lower index), its earliest queued request. *pick receives the index in
 * pending_func (-1 if none is queued); high_out (n_funcs entries, may be NULL) the group. */
TP_API tp_status tph_sched_pick(uint32_t n_funcs, const uint64_t* n, const uint64_t* m, double p, double alpha,
                         uint32_t n_pending, const int32_t* pending_func, int32_t* pick, uint8_t* high_out);

/* One period of the alpha auto-configuration (appendix "Function request prioritization"):
 * *out = min(alpha * scalar^d, 1), where d is +1 when the compliant share rose by more than
 * |threshold| (new_ratio - last_ratio), -1 when it fell by more than |threshold|, else 0.
 * alpha in (0, 1], scalar > 1; TP_E_INVAL otherwise. */
TP_API tp_status tph_alpha_update(double alpha, double last_ratio, double new_ratio, double scalar, double threshold,
                           double* out);

struct tph_arena;
/* An arena of `capacity` bytes whose extents are rounded up to `align` (power of two). */
TP_API tp_status tph_arena_create(uint64_t capacity, uint64_t align, struct tph_arena** out);
TP_API tp_status tph_arena_destroy(struct tph_arena* a);
TP_API tp_status tph_arena_register(struct tph_arena* a, int32_t model_id, uint64_t bytes);
TP_API tp_status tph_arena_unregister(struct tph_arena* a, int32_t model_id);
/* One request: *hit, the extent *offset, and up to `cap` victims in eviction order
 * (*n_victims receives their count). TP_E_NOSPC (no state change) if the model is
 * larger than the arena. */
TP_API tp_status tph_arena_request(struct tph_arena* a, int32_t model_id, int32_t* hit, uint64_t* offset,
                            int32_t* victims, uint32_t cap, uint32_t* n_victims);
TP_API tp_status tph_arena_evict(struct tph_arena* a, int32_t model_id);
/* Eviction policy (TP_EVICT_*, default LRU) and a model's class for TP_EVICT_HEAVINESS. */
TP_API tp_status tph_arena_set_policy(struct tph_arena* a, int32_t policy);
TP_API tp_status tph_arena_set_heavy(struct tph_arena* a, int32_t model_id, int32_t heavy);
/* Placement: partition_bytes > 0 switches to the two-tier partition scheme of TP_ALLOC_PARTITION
 * (torpor.h) with partitions of that size (a multiple of the alignment), with consolidation
 * (TP_ALLOC_PARTITION_CONSOLIDATE) if `consolidate`; 0 back to first fit. TP_E_STATE while
 * any model is resident, TP_E_INVAL for a size that is not a multiple. tph_arena_request
 * reports the victims alone; tph_arena_steps gives the last request's victims and moves in
 * the order made. */
TP_API tp_status tph_arena_set_partitioned(struct tph_arena* a, uint64_t partition_bytes, int32_t consolidate);
/* The steps of the last tph_arena_request in the order made: up to `cap` entries of a model,
 * whether it was moved (1; consolidation) or evicted (0), its old offset and (moves) its new
 * one; *n receives the count. The device replays them in this order. */
TP_API tp_status tph_arena_steps(struct tph_arena* a, int32_t* model_id, int32_t* moved, uint64_t* from, uint64_t* to,
                                 uint32_t cap, uint32_t* n);
TP_API tp_status tph_arena_stats(struct tph_arena* a, tp_arena_stats_t* out);

#ifdef __cplusplus
}
#endif
#endif /* TORPOR_PLAN_H */
