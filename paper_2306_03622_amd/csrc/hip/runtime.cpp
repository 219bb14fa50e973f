// The C ABI of libtorpor (torpor.h): registration into a pinned host pool, admission
// into the HBM arena, the chunked swap-in on the copy stream with one event per chunk,
// and the per-layer handoff to the caller's compute stream.
#include "runtime.hpp"

#include <algorithm>
#include <chrono>
#include <cstring>
#include <new>
#include <thread>

#include <hip/hip_ext.h>

#include "../core/errors.hpp"
#include "../kernels/kernels.hpp"
#include "../kernels/touch.hpp"
#include "scratch.hpp"

using namespace tp;

thread_local std::vector<tp::k::LaunchRecord>* tp::k::launch_log = nullptr;

namespace {

tp_status hip_fail(hipError_t e, const std::string& what) {
  return fail(TP_E_HIP, what + ": " + hipGetErrorString(e));
}

#define TP_HIP(call)                                  \
  do {                                                \
    hipError_t e_ = (call);                           \
    if (e_ != hipSuccess) return hip_fail(e_, #call); \
  } while (0)

Model* find(tp_ctx* c, int32_t id) {
  auto it = c->models.find(id);
  return it == c->models.end() ? nullptr : it->second.get();
}

// A copy stream of the library's own. The runtime maps streams onto a few hardware queues;
// when a copy stream lands on the compute stream's queue, its event packets and the
// kernels execute in one order, so a chunk's copy waits for the kernels enqueued before
// it and the swap no longer overlaps the forward pass (measured on MI355X: BERT-base at
// batch 8, 5.6 ms cold instead of 4.3 ms). A stream with an explicit CU mask is given a
// hardware queue of its own; the mask names every CU, and copies do not run on CUs anyway
// (gather copies do, on any of them). Such a stream is not created non-blocking, so it
// synchronises with the legacy null stream: callers should run requests on streams of
// their own.
hipError_t create_copy_stream(int device, hipStream_t* s) {
  int cus = 0;
  hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device);
  if (e != hipSuccess || cus < 1) return e != hipSuccess ? e : hipErrorInvalidDevice;
  std::vector<uint32_t> mask((cus + 31) / 32, 0xffffffffu);
  if (cus % 32) mask.back() = (1u << (cus % 32)) - 1;
  return hipExtStreamCreateWithCUMask(s, (uint32_t)mask.size(), mask.data());
}

hipError_t sync_copies(tp_ctx* c) {
  hipError_t e = hipSuccess;
  for (int i = 0; i < 2; ++i)
    if (c->copy[i] && e == hipSuccess) e = hipStreamSynchronize(c->copy[i]);
  return e;
}

void destroy_streams(tp_ctx* c) {
  if (c->own_copy && c->copy[0]) (void)hipStreamDestroy(c->copy[0]);
  if (c->exec) (void)hipStreamDestroy(c->exec);
  if (c->exec_fork) (void)hipEventDestroy(c->exec_fork);
  if (c->exec_join) (void)hipEventDestroy(c->exec_join);
  if (c->touch_sink) (void)hipFree(c->touch_sink);
  if (c->copy[1]) (void)hipStreamDestroy(c->copy[1]);
  if (c->capture) (void)hipStreamDestroy(c->capture);
  if (c->req_done) (void)hipEventDestroy(c->req_done);
  for (auto* v : {&c->tl.copy_begin, &c->tl.copy_end, &c->tl.exec_begin})
    for (hipEvent_t e : *v)
      if (e) (void)hipEventDestroy(e);
  if (c->tl.start) (void)hipEventDestroy(c->tl.start);
  if (c->tl.done) (void)hipEventDestroy(c->tl.done);
  if (c->fork) (void)hipEventDestroy(c->fork);
  if (c->claim_ev) (void)hipEventDestroy(c->claim_ev);
  for (hipEvent_t e : c->trace_ev)
    if (e) (void)hipEventDestroy(e);
}

k::Split make_split(char* work, const Model* m, int batch) {
  k::Split sp;
  if (m->spec.dtype != TP_BF16) return sp;
  sp.partials = reinterpret_cast<float*>(work + activation_bytes(m->spec, batch));
  sp.partial_bytes = kSplitScratch;
  return sp;
}

void destroy_graph(GraphEntry& g) {
  if (g.exec) (void)hipGraphExecDestroy(g.exec);
  if (g.graph) (void)hipGraphDestroy(g.graph);
  g.exec = nullptr;
  g.graph = nullptr;
}

void drop_graphs(Model* m) {
  for (auto& g : m->graphs) destroy_graph(g);
  m->graphs.clear();
}

// tp_debug_fail_copy: true when the copy about to be enqueued is the one chosen to fail
bool injected_failure(tp_ctx* c) { return c->fail_copy > 0 && --c->fail_copy == 0; }

void free_model(Model* m) {
  drop_graphs(m);
  for (hipEvent_t e : m->chunk_ev)
    if (e) (void)hipEventDestroy(e);
  if (m->last_use) (void)hipEventDestroy(m->last_use);
  if (m->host) (void)hipHostFree(m->host);
}

// The extent [off, off + len) of model `id` was invalidated; its old owner's enqueued
// work may still read it, so whoever writes it next must first wait for that work.
tp_status retire(tp_ctx* c, int32_t id, uint64_t off, uint64_t len) {
  c->retired.push_back({off, len, id});
  if (c->cfg.flags & TP_FLAG_POISON) {
    Model* m = find(c, id);
    if (m && m->used) TP_HIP(hipStreamWaitEvent(c->copy[0], m->last_use, 0));
    TP_HIP(hipMemsetAsync(c->arena + off, 0xFF, len, c->copy[0]));
  }
  return ok();
}

// Orders the copy stream after every retired owner of bytes in [off, off + len) and
// drops those bytes from the retired set (the new owner's own last use guards them now).
tp_status claim(tp_ctx* c, uint64_t off, uint64_t len) {
  std::vector<tp_ctx::Retired> keep;
  const uint64_t end = off + len;
  for (const auto& r : c->retired) {
    const uint64_t rend = r.off + r.len;
    if (rend <= off || r.off >= end) {
      keep.push_back(r);
      continue;
    }
    // (an owner whose last use has already completed needs no wait packet on the copy stream)
    Model* m = find(c, r.model);
    if (m && m->used && hipEventQuery(m->last_use) != hipSuccess)
      TP_HIP(hipStreamWaitEvent(c->copy[0], m->last_use, 0));
    if (r.off < off) keep.push_back({r.off, off - r.off, r.model});
    if (rend > end) keep.push_back({end, rend - end, r.model});
  }
  c->retired.swap(keep);
  return ok();
}

// Enqueues the copy of chunk i of `m` into the extent at arena offset `off`, then its event.
hipError_t enqueue_chunk(tp_ctx* c, const Model* m, uint64_t off, size_t i) {
  if (injected_failure(c)) return hipErrorInvalidValue;     // nothing enqueued for this chunk
  const size_t n = m->chunks.size();
  const int ns = (c->ncopy == 2 && n > 1) ? 2 : 1;
  hipError_t e = hipSuccess;
  if (i == 0 && ns == 2) {
    // everything ordered on copy[0] so far (victim waits, poison) precedes copy[1]'s chunks
    e = hipEventRecord(c->fork, c->copy[0]);
    if (e == hipSuccess) e = hipStreamWaitEvent(c->copy[1], c->fork, 0);
  }
  const Chunk& ch = m->chunks[i];
  const uint64_t nb = ch.end - ch.begin;
  char* dst = c->arena + off + ch.begin;
  hipStream_t s = c->copy[i % ns];
  if (e == hipSuccess && (c->cfg.flags & TP_FLAG_THROTTLE)) e = k::delay(c->cfg.throttle_us, s);
  const bool traced = c->tl.active && i < c->tl.copy_begin.size();
  if (e == hipSuccess && traced) e = hipEventRecord(c->tl.copy_begin[i], s);
  if (e == hipSuccess) {
    if (c->cfg.copy_method == TP_COPY_GATHER)
      e = k::gather_copy(static_cast<char*>(m->host_dev) + ch.begin, dst, nb, c->cfg.gather_wgs, s);
    else if (c->cfg.copy_method == TP_COPY_PAGEABLE)
      e = hipMemcpyAsync(dst, m->pageable.get() + ch.begin, nb, hipMemcpyHostToDevice, s);
    else
      e = hipMemcpyAsync(dst, static_cast<char*>(m->host) + ch.begin, nb, hipMemcpyHostToDevice, s);
  }
  // the traced end precedes the chunk's event, so that a kernel released by that event
  // starts after the recorded end
  if (e == hipSuccess && traced) e = hipEventRecord(c->tl.copy_end[i], s);
  if (e == hipSuccess) e = hipEventRecord(m->chunk_ev[i], s);
  return e;
}

// A consolidation move of resident model `x` from arena offset `from` to `to`, on the primary
// copy stream: after the destination's retired owners and x's own swap-in (its last chunk
// on each copy stream), a device-to-device copy of x's image; x's last chunk event is then
// recorded after the copy and x marked pending, so x's next request waits for it (settle).
// The old extent is retired under x, like an eviction: whoever writes it next waits for x's
// enqueued readers; the copy itself precedes any later write on the copy streams.
tp_status move_extent(tp_ctx* c, Model* x, uint64_t from, uint64_t to) {
  const uint64_t len = c->policy->bytes(x->id);
  tp_status s = claim(c, to, len);
  if (s != TP_OK) return s;
  const size_t n = x->chunk_ev.size();
  if (injected_failure(c)) return hip_fail(hipErrorInvalidValue, "consolidation move (injected)");
  TP_HIP(hipStreamWaitEvent(c->copy[0], x->chunk_ev[n - 1], 0));
  if (c->ncopy == 2 && n > 1) TP_HIP(hipStreamWaitEvent(c->copy[0], x->chunk_ev[n - 2], 0));
  TP_HIP(hipMemcpyAsync(c->arena + to, c->arena + from, x->spec.host_bytes, hipMemcpyDeviceToDevice, c->copy[0]));
  TP_HIP(hipEventRecord(x->chunk_ev.back(), c->copy[0]));
  x->bg_pending = true;
  return retire(c, x->id, from, len);
}

// One request's admission: a hit, or consolidation moves made and victims invalidated, in
// the arena's order, with their readers waited for on the primary copy stream; the chunk
// copies are then issued by the request's Waiter. On failure the model is left
// non-resident.
tp_status admit(tp_ctx* c, Model* m, bool* swapped) {
  const auto t0 = std::chrono::steady_clock::now();
  Arena::Decision d = c->policy->request(m->id);
  *swapped = !d.hit;
  if (d.hit) return ok();
  struct Timer {              // host time of this (missing) admission, on every return path
    tp_ctx* c;
    std::chrono::steady_clock::time_point t0;
    ~Timer() {
      const uint64_t ns = (uint64_t)std::chrono::duration_cast<std::chrono::nanoseconds>(
                              std::chrono::steady_clock::now() - t0).count();
      ++c->admit_calls;
      c->last_admit_ns = ns;
      c->admit_ns_total += ns;
      c->admit_ns_max = std::max(c->admit_ns_max, ns);
    }
  } timer{c, t0};
  m->bg_pending = false;         // a new swap supersedes an earlier one
  tp_status s = TP_OK;
  // the arena's victims and moves, in the order it made them; also when it then found no
  // placement, so that the extents it invalidated are retired like any other
  for (const auto& st : d.steps) {
    if (s != TP_OK) break;
    s = st.move ? move_extent(c, find(c, st.id), st.from, st.to) : retire(c, st.id, st.from, c->policy->bytes(st.id));
  }
  if (s == TP_OK && !d.placed) return fail(TP_E_NOSPC, "model cannot be placed in the arena");
  if (s == TP_OK) s = claim(c, d.offset, m->spec.host_bytes);
  if (s != TP_OK) {
    const std::string msg = last_error();
    for (const auto& mv : d.moves) {       // a move may not have been copied: drop the moved models
      const uint64_t len = c->policy->bytes(mv.id);
      c->policy->evict(mv.id);
      (void)retire(c, mv.id, mv.from, len);
      (void)retire(c, mv.id, mv.to, len);
    }
    if (d.placed) {
      c->policy->evict(m->id);
      (void)retire(c, m->id, d.offset, m->spec.host_bytes);
    }
    return fail(s, msg);
  }
  return ok();
}

}  // namespace

hipError_t tp::Waiter::trace_exec(int c) {
  if (!ctx || !ctx->tl.active || c >= (int)ctx->tl.exec_begin.size()) return hipSuccess;
  return hipEventRecord(ctx->tl.exec_begin[c], stream);
}

hipError_t tp::Waiter::hand_back() {
  hipError_t e = hipEventRecord(ctx->exec_join, stream);
  if (e == hipSuccess) e = hipStreamWaitEvent(caller, ctx->exec_join, 0);
  stream = caller;
  if (slot) *slot = caller;
  caller = nullptr;
  return e;
}

hipError_t tp::Waiter::issue_through(int c) {
  hipError_t e = hipSuccess;
  while (e == hipSuccess && issued <= c && issued < (int)m->chunks.size()) e = enqueue_chunk(ctx, m, base_off, issued++);
  return e;
}

namespace {

hipError_t run_forward(ExecCtx& x) {
  switch (x.m->spec.arch) {
    case TP_ARCH_MLP: return run_mlp(x);
    case TP_ARCH_RESNET50: return run_resnet(x);
    case TP_ARCH_BERT: return run_bert(x);
  }
  return hipErrorInvalidValue;
}

// Warm request: replay the model's forward pass as one graph launch. A graph is captured
// from the same kernel sequence (on a private stream, nothing executes) the first time a
// (batch, workspace) combination is seen; up to kGraphs combinations stay instantiated per
// model. A request whose weights lie elsewhere than the graph's nodes hold (the model came
// back into another extent) or with other input or output buffers repoints those nodes in
// place; an input or output whose address has another residue modulo 16 than the captured
// one is captured afresh instead, since a launcher may choose its kernel by that alignment.
// If capture fails the model falls back to launching its kernels one by one, which computes
// the same bits.
constexpr size_t kGraphs = 4;

// A graph launch costs more host and device time than a few direct kernel launches
// (measured on MI355X: a 4-kernel forward takes 36 us as a graph, 26 us launched one by
// one), so only forward passes of at least this many kernels are replayed as graphs.
constexpr int kGraphMinLaunches = 16;

int forward_launches(const ModelSpec& s) {
  switch (s.arch) {
    case TP_ARCH_MLP: return s.dims[0];
    case TP_ARCH_BERT: return 7 * s.dims[0] + 1;
    default: return 1 << 20;      // ResNet-50: > 50 convolutions
  }
}

// The kernel nodes of a captured single-stream graph in launch order: the graph must be one
// chain of `n` kernel nodes whose kernels are those of the recorded launches.
bool chain_nodes(hipGraph_t g, const std::vector<k::LaunchRecord>& rec, std::vector<hipGraphNode_t>* out) {
  size_t n = 0;
  if (hipGraphGetRootNodes(g, nullptr, &n) != hipSuccess || n != 1) return false;
  hipGraphNode_t cur = nullptr;
  if (hipGraphGetRootNodes(g, &cur, &n) != hipSuccess) return false;
  out->clear();
  while (cur) {
    hipGraphNodeType t;
    if (hipGraphNodeGetType(cur, &t) != hipSuccess || t != hipGraphNodeTypeKernel) return false;
    if (out->size() >= rec.size()) return false;
    hipKernelNodeParams p{};
    if (hipGraphKernelNodeGetParams(cur, &p) != hipSuccess || p.func != rec[out->size()].func) return false;
    out->push_back(cur);
    size_t nd = 0;
    if (hipGraphNodeGetDependentNodes(cur, nullptr, &nd) != hipSuccess || nd > 1) return false;
    hipGraphNode_t next = nullptr;
    if (nd == 1 && hipGraphNodeGetDependentNodes(cur, &next, &nd) != hipSuccess) return false;
    cur = nd == 1 ? next : nullptr;
  }
  return out->size() == rec.size();
}

// Points the graph's nodes at the weights at `base` and at `in` and `out`: each node that
// holds a pointer into the captured extent, input or output gets its recorded arguments
// with those pointers moved by the same displacement (weights) or replaced (buffers). Only
// the nodes whose pointers change are set.
hipError_t repoint(GraphEntry& g, const char* base, const void* in, void* out) {
  const bool moved = base != g.cur_base, io = in != g.cur_in || out != g.cur_out;
  const uintptr_t b0 = (uintptr_t)g.cap_base, b1 = b0 + g.extent_bytes;
  std::vector<uint8_t> b;
  std::vector<void*> argv;
  for (uint32_t i = 0; i < g.launches.size(); ++i) {
    const uint8_t use = g.use[i];
    if (!((moved && (use & kUsesWeights)) || (io && (use & kUsesBuffers)))) continue;
    const k::LaunchRecord& r = g.launches[i];
    b = r.bytes;
    for (uint32_t at : r.ptr_at) {
      uintptr_t v;
      std::memcpy(&v, b.data() + at, sizeof v);
      if (v == (uintptr_t)g.cap_in) v = (uintptr_t)in;
      else if (v == (uintptr_t)g.cap_out) v = (uintptr_t)out;
      else if (v >= b0 && v < b1) v = (uintptr_t)base + (v - b0);
      else continue;
      std::memcpy(b.data() + at, &v, sizeof v);
    }
    argv.resize(r.arg_at.size());
    for (size_t j = 0; j < argv.size(); ++j) argv[j] = b.data() + r.arg_at[j];
    hipKernelNodeParams p{};
    p.func = const_cast<void*>(r.func);
    p.gridDim = r.grid;
    p.blockDim = r.block;
    p.sharedMemBytes = r.shmem;
    p.kernelParams = argv.data();
    p.extra = nullptr;
    const hipError_t e = hipGraphExecKernelNodeSetParams(g.exec, g.nodes[i], &p);
    if (e != hipSuccess) return e;
  }
  g.cur_base = base;
  g.cur_in = in;
  g.cur_out = out;
  return hipSuccess;
}

// Captures and instantiates the forward pass of `m` into `g` (its key fields set).
hipError_t capture_graph(tp_ctx* c, Model* m, GraphEntry& g) {
  Waiter w;
  w.m = m;
  char* base = const_cast<char*>(g.cap_base);
  char* work = const_cast<char*>(g.work);
  ExecCtx x{m, base, work, g.cap_in, g.cap_out, g.batch, c->capture, &w, make_split(work, m, g.batch)};
  g.launches.clear();
  k::launch_log = &g.launches;
  hipError_t e = hipStreamBeginCapture(c->capture, hipStreamCaptureModeThreadLocal);
  if (e == hipSuccess) {
    hipError_t er = run_forward(x);
    e = hipStreamEndCapture(c->capture, &g.graph);
    if (er != hipSuccess) e = er;
  }
  k::launch_log = nullptr;
  if (e == hipSuccess) e = hipGraphInstantiate(&g.exec, g.graph, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    destroy_graph(g);
    return e;
  }
  ++c->graph_captures;
  g.cur_base = g.cap_base;
  g.cur_in = g.cap_in;
  g.cur_out = g.cap_out;
  g.patchable = chain_nodes(g.graph, g.launches, &g.nodes);
  g.use.assign(g.launches.size(), 0);
  const uintptr_t b0 = (uintptr_t)g.cap_base, b1 = b0 + g.extent_bytes;
  for (uint32_t i = 0; g.patchable && i < g.launches.size(); ++i) {
    const k::LaunchRecord& r = g.launches[i];
    for (uint32_t at : r.ptr_at) {
      uintptr_t v;
      std::memcpy(&v, r.bytes.data() + at, sizeof v);
      if (v == (uintptr_t)g.cap_in || v == (uintptr_t)g.cap_out) g.use[i] |= kUsesBuffers;
      else if (v >= b0 && v < b1) g.use[i] |= kUsesWeights;
    }
  }
  return hipSuccess;
}

hipError_t launch_graph(tp_ctx* c, Model* m, char* base, char* work, const void* in, int batch, void* out,
                        hipStream_t stream) {
  GraphEntry* hit = nullptr;
  for (auto& g : m->graphs)
    if (g.batch == batch && g.work == work) hit = &g;
  if (hit && (hit->cur_base != base || hit->cur_in != in || hit->cur_out != out)) {
    const bool same_align = ((uintptr_t)in & 15) == ((uintptr_t)hit->cap_in & 15) &&
                            ((uintptr_t)out & 15) == ((uintptr_t)hit->cap_out & 15);
    const bool moved = hit->cur_base != base;
    hipError_t e = hit->patchable && same_align ? repoint(*hit, base, in, out) : hipErrorNotSupported;
    if (e == hipSuccess) {
      ++c->graph_repoints;
      if (moved) ++c->graph_rebases;
    } else {
      (void)hipGetLastError();
      destroy_graph(*hit);                 // captured again below, for these buffers
      m->graphs.erase(m->graphs.begin() + (hit - m->graphs.data()));
      hit = nullptr;
    }
  }
  if (!hit) {
    if (m->graphs.size() >= kGraphs) {
      auto oldest = std::min_element(m->graphs.begin(), m->graphs.end(),
                                     [](const GraphEntry& a, const GraphEntry& b) { return a.stamp < b.stamp; });
      destroy_graph(*oldest);
      m->graphs.erase(oldest);
    }
    GraphEntry g;
    g.batch = batch;
    g.cap_base = base;
    g.extent_bytes = m->spec.host_bytes;
    g.work = work;
    g.cap_in = in;
    g.cap_out = out;
    if (capture_graph(c, m, g) != hipSuccess) {
      (void)hipGetLastError();
      m->graph_failed = true;
      Waiter w2;
      w2.m = m;
      ExecCtx x2{m, base, work, in, out, batch, stream, &w2, make_split(work, m, batch)};
      return run_forward(x2);
    }
    m->graphs.push_back(std::move(g));
    hit = &m->graphs.back();
  }
  hit->stamp = ++c->graph_clock;
  return hipGraphLaunch(hit->exec, stream);
}

// A request that finds the model resident: if a direct-access request left its swap
// running behind it, wait for the swap's last chunk (once; later requests are ordered
// after this one).
hipError_t settle(Model* m, hipStream_t stream) {
  if (!m->bg_pending) return hipSuccess;
  m->bg_pending = false;
  return hipStreamWaitEvent(stream, m->chunk_ev.back(), 0);
}

tp_status begin_request(tp_ctx* c, hipStream_t stream) {
  if (c->any_request && stream != c->last_stream) TP_HIP(hipStreamWaitEvent(stream, c->req_done, 0));
  return ok();
}

tp_status end_request(tp_ctx* c, Model* m, hipStream_t stream) {
  if (c->tl.active) {
    c->tl.active = false;
    TP_HIP(hipEventRecord(c->tl.done, stream));
    c->tl.valid = true;
  }
  TP_HIP(hipEventRecord(m->last_use, stream));
  m->used = true;
  TP_HIP(hipEventRecord(c->req_done, stream));
  c->last_stream = stream;
  c->any_request = true;
  return ok();
}

tp_status check_request(tp_ctx* c, int32_t id, Model** out) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  if (!c->policy->fits_at_all(id))
    return fail(TP_E_NOSPC, "model of " + std::to_string(m->spec.host_bytes) + " bytes exceeds the arena of " +
                                std::to_string(c->cfg.arena_bytes) + " bytes");
  *out = m;
  return ok();
}

// A warm request for a model other than the one the previous request served (whose bytes the
// requests in between have likely pushed out of the Infinity Cache and the L2s), or for one
// that tp_swap_in brought in and no request has read since (the copy engine's writes leave it
// out of the caches; every warm request under TP_FLAG_TOUCH_ALWAYS) reads the model's touch
// span on the execution stream while its own kernels run on the caller's stream: its later
// layers then find their weights in the cache. The read waits for the model's last copies
// (a tp_swap_in's may still be in flight) and for nothing else; reading bytes that a later swap
// overwrites meanwhile is harmless (they are discarded), and the read stays inside the arena,
// which outlives the context. A failure only forgoes the touch.
void maybe_touch(tp_ctx* c, Model* m, uint64_t off) {
  if (!c->exec || !c->touch_sink || (c->cfg.flags & TP_FLAG_NO_TOUCH) || m->bg_pending) return;
  if (!(c->cfg.flags & TP_FLAG_TOUCH_ALWAYS) && c->last_served == m->id && !m->touch_due) return;
  uint64_t lo = 0, hi = 0;
  if (!touch_span(m->spec, &lo, &hi)) return;
  const size_t n = m->chunk_ev.size();
  hipError_t e = n ? hipStreamWaitEvent(c->exec, m->chunk_ev[n - 1], 0) : hipSuccess;
  if (e == hipSuccess && c->ncopy == 2 && n > 1) e = hipStreamWaitEvent(c->exec, m->chunk_ev[n - 2], 0);
  if (e == hipSuccess) e = k::touch(c->arena + off + lo, hi - lo, c->touch_sink, c->exec);
  if (e == hipSuccess) ++c->cache_touches;
  else (void)hipGetLastError();
}

// One request (tp_infer and its variants), with the workspace `work` of `work_bytes`.
// allow_graphs: warm forward passes may replay a graph; allow_touch: a warm request may
// pre-read its weights on the execution stream (maybe_touch).
tp_status infer_request(tp_ctx* c, int32_t id, const void* input_dev, int32_t batch, void* output_dev,
                        hipStream_t stream, char* work, uint64_t work_bytes, const char* who, bool allow_graphs = true,
                        bool allow_touch = true) {
  Model* m = nullptr;
  tp_status s = check_request(c, id, &m);
  if (s != TP_OK) return s;
  if (batch < 1 || !input_dev || !output_dev) return fail(TP_E_INVAL, std::string(who) + ": batch < 1 or NULL buffer");
  const uint64_t need = workspace_bytes(m->spec, batch);
  if (need > work_bytes)
    return fail(TP_E_NOSPC, std::string(who) + ": workspace of " + std::to_string(work_bytes) + " bytes, need " +
                                std::to_string(need));
  if ((s = begin_request(c, stream)) != TP_OK) return s;
  if (c->cfg.copy_method == TP_COPY_ZERO && !c->policy->resident(id)) {
    // direct host access: the kernels read the weights from the pinned host copy
    Waiter w;
    w.m = m;
    ExecCtx x{m, static_cast<char*>(m->host_dev), work, input_dev, output_dev, batch, stream, &w,
              make_split(work, m, batch)};
    hipError_t e = run_forward(x);
    if (e != hipSuccess) {
      (void)end_request(c, m, stream);
      return hip_fail(e, std::string(who) + ": kernel launch");
    }
    return end_request(c, m, stream);
  }
  const bool direct = c->cfg.direct_max_bytes && m->spec.host_bytes <= c->cfg.direct_max_bytes &&
                      !c->policy->resident(id) && c->ncopy == 1 &&
                      (c->cfg.copy_method == TP_COPY_MEMCPY || c->cfg.copy_method == TP_COPY_GATHER);
  bool swapped = false;
  if ((s = admit(c, m, &swapped)) != TP_OK) return s;
  const uint64_t off = c->policy->offset(id);
  if (!swapped && allow_touch) maybe_touch(c, m, off);
  c->last_served = id;
  m->touch_due = false;          // this request reads the weights (a cold one as they land)
  const bool graphs = allow_graphs && !(c->cfg.flags & TP_FLAG_NO_GRAPH) && !m->graph_failed &&
                      forward_launches(m->spec) >= kGraphMinLaunches;
  // a swapping request's kernels run on the library's execution stream (see tp_create),
  // all but its last chunk's (a single-chunk request stays on the caller's stream)
  const bool forked = swapped && !direct && c->exec && m->chunks.size() > 1;
  // a small fp32 MLP's cold request swaps it in with its own first kernel (run_mlp_swapin)
  const bool swapin = direct && swapped && !graphs && !(c->cfg.flags & TP_FLAG_POISON) &&
                      mlp_swapin_fits(m->spec, batch);
  hipError_t e = swapped ? hipSuccess : settle(m, stream);
  if (e != hipSuccess) {
    // fall through to the failure handling below
  } else if (swapin) {
    // The extent is written from the caller's stream, so that stream first waits for what the
    // copy stream must finish before the extent may be written (the waits for its retired
    // readers that admission enqueued there, earlier copies), unless all of it is done.
    const hipError_t q = hipStreamQuery(c->copy[0]);
    if (q == hipErrorNotReady) {
      e = hipEventRecord(c->claim_ev, c->copy[0]);
      if (e == hipSuccess) e = hipStreamWaitEvent(stream, c->claim_ev, 0);
    } else if (q != hipSuccess) {
      e = q;
    }
    if (e == hipSuccess && injected_failure(c)) e = hipErrorInvalidValue;   // counts as the copy
    if (e == hipSuccess) {
      Waiter w;
      w.m = m;
      ExecCtx x{m, c->arena + off, work, input_dev, output_dev, batch, stream, &w, make_split(work, m, batch)};
      e = run_mlp_swapin(x, m->host_dev);
    }
    if (e == hipSuccess && (s = end_request(c, m, stream)) == TP_OK) {
      // the chunk events (which later copies and moves order themselves on) complete with
      // the request, on the copy stream: recorded on the caller's stream, the completion of
      // that stream measured ~15 us later on MI355X
      e = hipStreamWaitEvent(c->copy[0], c->req_done, 0);
      for (size_t i = 0; e == hipSuccess && i < m->chunk_ev.size(); ++i) e = hipEventRecord(m->chunk_ev[i], c->copy[0]);
      if (e == hipSuccess) return ok();
      c->policy->evict(id);
      (void)retire(c, id, off, m->spec.host_bytes);
      return hip_fail(e, std::string(who) + ": swap-in events");
    }
    if (s != TP_OK) {
      c->policy->evict(id);
      (void)retire(c, id, off, m->spec.host_bytes);
      return s;
    }
  } else if (direct) {
    // The request's kernels read the host copy and own the host link while they run; the
    // swap is enqueued after the request's completion event, on the copy stream that
    // waits for it, so neither the link nor (when the runtime maps both streams onto one
    // hardware queue) the caller's synchronisation waits for the copy.
    char* host = static_cast<char*>(m->host_dev);
    if (graphs) {
      e = launch_graph(c, m, host, work, input_dev, batch, output_dev, stream);
    } else {
      Waiter w;
      w.m = m;
      ExecCtx x{m, host, work, input_dev, output_dev, batch, stream, &w, make_split(work, m, batch)};
      e = run_forward(x);
    }
    if (e == hipSuccess && (s = end_request(c, m, stream)) == TP_OK) {
      Waiter bg;
      bg.m = m;
      bg.ctx = c;
      bg.base_off = off;
      e = hipStreamWaitEvent(c->copy[0], c->req_done, 0);
      if (e == hipSuccess) e = bg.issue_through((int)m->chunks.size() - 1);
      if (e == hipSuccess) {
        m->bg_pending = true;
        return ok();
      }
      c->policy->evict(id);
      (void)retire(c, id, off, m->spec.host_bytes);
      return hip_fail(e, std::string(who) + ": swap enqueue");
    }
    if (s != TP_OK) {
      c->policy->evict(id);
      (void)retire(c, id, off, m->spec.host_bytes);
      return s;
    }
  } else if (!swapped && graphs) {
    e = launch_graph(c, m, c->arena + off, work, input_dev, batch, output_dev, stream);
  } else {
    const hipStream_t xs = forked ? c->exec : stream;
    Waiter w;
    w.m = m;
    w.stream = xs;
    w.swapping = swapped;
    w.ctx = c;
    w.base_off = off;
    ExecCtx x{m, c->arena + off, work, input_dev, output_dev, batch, xs, &w, make_split(work, m, batch)};
    if (swapped && (c->cfg.flags & TP_FLAG_TRACE)) {
      c->tl.active = true;
      c->tl.valid = false;
      c->tl.n = (uint32_t)m->chunks.size();
      e = hipEventRecord(c->tl.start, stream);
    }
    // the first chunk's copy goes out before anything else is enqueued
    if (e == hipSuccess && swapped) e = w.issue_through(0);
    if (e == hipSuccess && forked) {
      // the execution stream waits for the caller's earlier work, unless all of it has
      // already completed (then the hand-over would only add a cross-queue wait)
      const hipError_t q = hipStreamQuery(stream);
      if (q == hipErrorNotReady) {
        e = hipEventRecord(c->exec_fork, stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(c->exec, c->exec_fork, 0);
      } else if (q != hipSuccess) {
        e = q;
      }
      w.caller = stream;
      w.slot = &x.stream;
    }
    // swap, then execute: every chunk is waited for before the first kernel
    if (e == hipSuccess && swapped && (c->cfg.flags & TP_FLAG_SERIAL)) e = w.need(m->spec.n_layers - 1);
    if (e == hipSuccess) e = run_forward(x);
    // every layer asks for its chunk; issue any the forward pass did not reach
    if (e == hipSuccess && swapped) e = w.issue_through((int)m->chunks.size() - 1);
    if (w.caller) {
      // not handed back (a failure before the last chunk): join whatever was enqueued on
      // the execution stream, so that the request's completion (and the model's last use)
      // covers it
      const hipError_t ej = w.hand_back();
      if (e == hipSuccess) e = ej;
    }
  }
  if (e != hipSuccess) {
    // keep the ordering intact, then leave the model non-resident
    (void)end_request(c, m, stream);
    c->policy->evict(id);
    (void)retire(c, id, off, m->spec.host_bytes);
    return hip_fail(e, std::string(who) + ": enqueue");
  }
  return end_request(c, m, stream);
}

}  // namespace

extern "C" {

tp_status tp_create(const tp_config* cfg, tp_ctx** out) {
  if (!cfg || !out) return fail(TP_E_INVAL, "tp_create: NULL argument");
  if (!cfg->arena_dev || cfg->arena_bytes == 0) return fail(TP_E_INVAL, "tp_create: empty arena");
  if ((uintptr_t)cfg->arena_dev % 256) return fail(TP_E_INVAL, "tp_create: arena must be 256-byte aligned");
  if (cfg->work_bytes && (!cfg->work_dev || (uintptr_t)cfg->work_dev % 256))
    return fail(TP_E_INVAL, "tp_create: workspace must be non-NULL and 256-byte aligned");
  if (cfg->copy_method < TP_COPY_MEMCPY || cfg->copy_method > TP_COPY_ZERO)
    return fail(TP_E_INVAL, "tp_create: unknown copy_method");
  if (cfg->gather_wgs < 0 || cfg->gather_wgs > 4096 || cfg->throttle_us < 0 || cfg->throttle_us > 100000)
    return fail(TP_E_INVAL, "tp_create: gather_wgs or throttle_us out of range");
  if (cfg->copy_streams < 0 || cfg->copy_streams > 2) return fail(TP_E_INVAL, "tp_create: copy_streams must be 0, 1 or 2");
  if (cfg->plan < TP_PLAN_GREEDY || cfg->plan > TP_PLAN_COST || cfg->plan_batch < 0 || cfg->plan_batch > 65536 ||
      !(cfg->link_gbs >= 0) || cfg->link_gbs > 1e4 || !(cfg->chunk_us >= 0) || cfg->chunk_us > 1e5)
    return fail(TP_E_INVAL, "tp_create: plan, plan_batch, link_gbs or chunk_us out of range");
  if ((cfg->evict_policy != TP_EVICT_LRU && cfg->evict_policy != TP_EVICT_HEAVINESS &&
       cfg->evict_policy != TP_EVICT_LRU_WINDOW) || !(cfg->heavy_ratio >= 0) ||
      cfg->heavy_ratio > 1e6)
    return fail(TP_E_INVAL, "tp_create: evict_policy or heavy_ratio out of range");
  if (cfg->alloc < TP_ALLOC_FIRST_FIT || cfg->alloc > TP_ALLOC_PARTITION_CONSOLIDATE ||
      (cfg->alloc != TP_ALLOC_FIRST_FIT && cfg->partition_bytes % 256))
    return fail(TP_E_INVAL, "tp_create: alloc or partition_bytes out of range");
  std::unique_ptr<tp_ctx> c(new (std::nothrow) tp_ctx);
  if (!c) return fail(TP_E_NOSPC, "out of host memory");
  c->cfg = *cfg;
  if (c->cfg.gather_wgs == 0) c->cfg.gather_wgs = 64;
  c->arena = static_cast<char*>(cfg->arena_dev);
  c->work = static_cast<char*>(cfg->work_dev);
  c->policy.reset(new Arena(cfg->arena_bytes, 256, cfg->evict_policy));
  if (cfg->alloc != TP_ALLOC_FIRST_FIT) {
    uint64_t part = cfg->partition_bytes;
    if (!part) part = std::max<uint64_t>(cfg->arena_bytes / 8 / (1u << 20) * (1u << 20), 256);
    // nothing is resident yet and part is a multiple of 256: cannot fail
    (void)c->policy->set_partitioned(part, cfg->alloc == TP_ALLOC_PARTITION_CONSOLIDATE);
  }
  TP_HIP(hipGetDevice(&c->device));
  c->ncopy = cfg->copy_streams == 2 ? 2 : 1;
  hipError_t e = hipSuccess;
  // One small device copy on the legacy null stream before the library creates its CU-masked
  // streams (which synchronise with the null stream). Measured on MI355X: when a process had
  // made no such copy before they were created, synchronising the caller's stream after a
  // direct-access request also waited for the swap enqueued behind it on the copy stream
  // (1 MB fp32 MLP cold: 145 us instead of 54 us, for as long as the process ran); a copy
  // made after the streams exist did not help, one made before did. It copies the arena's
  // first 256 bytes over the next 256, which nothing has been placed in yet.
  if (cfg->arena_bytes >= 512) {
    e = hipMemcpyAsync(c->arena + 256, c->arena, 256, hipMemcpyDeviceToDevice, nullptr);
    if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
  }
  if (cfg->copy_stream) {
    c->copy[0] = static_cast<hipStream_t>(cfg->copy_stream);
  } else {
    e = create_copy_stream(c->device, &c->copy[0]);
    c->own_copy = e == hipSuccess;
  }
  if (e == hipSuccess && c->ncopy == 2) e = create_copy_stream(c->device, &c->copy[1]);
  if (e == hipSuccess && !(cfg->flags & TP_FLAG_CALLER_STREAM)) {
    // the execution stream of swapping requests: a hardware queue of its own, like the copy
    // streams, so that whatever queue the caller's stream lands on, chunk copies and layer
    // kernels are never serialised behind each other in one queue
    e = create_copy_stream(c->device, &c->exec);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->exec_fork, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&c->exec_join, hipEventDisableTiming);
    // the cache touch's sink (written only in the impossible case, see k::touch)
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&c->touch_sink), 64 * sizeof(uint32_t));
  }
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&c->capture, hipStreamNonBlocking);
  // tp_infer_noalloc's workspace on this device (a failure only disables that entry point,
  // which then reports it)
  if (e == hipSuccess && scratch_init(c->device) != hipSuccess) (void)hipGetLastError();

  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->req_done, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->claim_ev, hipEventDisableTiming);
  if (e == hipSuccess && (cfg->flags & TP_FLAG_TRACE)) e = hipEventCreate(&c->tl.start);
  if (e == hipSuccess && (cfg->flags & TP_FLAG_TRACE)) e = hipEventCreate(&c->tl.done);
  if (e != hipSuccess) {
    destroy_streams(c.get());
    return hip_fail(e, "tp_create: stream or event creation");
  }
  *out = c.release();
  return ok();
}

tp_status tp_destroy(tp_ctx* c) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  hipError_t e = sync_copies(c);
  if (e == hipSuccess && c->exec) e = hipStreamSynchronize(c->exec);
  if (e == hipSuccess && c->any_request) e = hipEventSynchronize(c->req_done);
  for (auto& kv : c->models) {
    if (kv.second->used) (void)hipEventSynchronize(kv.second->last_use);
    free_model(kv.second.get());
  }
  destroy_streams(c);
  delete c;
  return e == hipSuccess ? ok() : hip_fail(e, "tp_destroy synchronisation");
}

tp_status tp_register_model(tp_ctx* c, const tp_model_desc* desc, const void* host_weights, uint64_t host_bytes,
                            int32_t* model_id) {
  if (!c || !desc || !host_weights || !model_id || host_bytes == 0) return fail(TP_E_INVAL, "tp_register_model: NULL argument");
  std::unique_ptr<Model> m(new (std::nothrow) Model);
  if (!m) return fail(TP_E_NOSPC, "out of host memory");
  std::string err;
  tp_status s = validate_model(desc, host_bytes, &m->spec, &err);
  if (s != TP_OK) return fail(s, err);
  m->id = c->next_id;
  {
    // cost-model estimates: the plan of TP_PLAN_COST and the heaviness class
    LinkModel lm;
    if (c->cfg.link_gbs > 0) lm.link_bytes_per_us = c->cfg.link_gbs * 1e3;
    if (c->cfg.chunk_us > 0) lm.chunk_us = c->cfg.chunk_us;
    const int pb = c->cfg.plan_batch > 0 ? c->cfg.plan_batch : 1;
    double cold = 0, warm = 0;
    std::vector<Chunk> best = plan_chunks_cost(m->spec, pb, lm, &cold);
    for (double t : layer_cost_us(m->spec, pb)) warm += t;
    m->cold_est_us = (float)cold;
    m->warm_est_us = (float)warm;
    m->heavy_auto = cold > (c->cfg.heavy_ratio > 0 ? c->cfg.heavy_ratio : 3.0) * warm;
    if (c->cfg.plan == TP_PLAN_COST) m->chunks = std::move(best);
  }
  if (c->cfg.plan != TP_PLAN_COST) {
    m->chunks = plan_chunks(m->spec, c->cfg.chunk_min_bytes, (c->cfg.flags & TP_FLAG_PER_TENSOR) != 0);
  }
  m->chunk_of_layer.assign(m->spec.n_layers, 0);
  for (size_t i = 0; i < m->chunks.size(); ++i)
    for (uint32_t l = m->chunks[i].first_layer; l <= m->chunks[i].last_layer; ++l) m->chunk_of_layer[l] = (uint32_t)i;
  const uint64_t nb = m->spec.host_bytes;
  hipError_t e = hipHostMalloc(&m->host, nb, hipHostMallocMapped);
  if (e != hipSuccess) { m->host = nullptr; return hip_fail(e, "hipHostMalloc (pinned model copy)"); }
  std::memcpy(m->host, host_weights, host_bytes);
  if (nb > host_bytes) std::memset(static_cast<char*>(m->host) + host_bytes, 0, nb - host_bytes);
  if (m->spec.packed_mlp) {
    // weight matrices in the skinny-GEMM block order, one thread per group of layers
    std::vector<std::thread> th;
    const int L = m->spec.dims[0], W = m->spec.dims[1];
    const int nt = std::max(1, std::min(8, L));
    for (int w = 0; w < nt; ++w)
      th.emplace_back([&, w] {
        for (int l = w; l < L; l += nt) {
          const tp_tensor_desc& t = m->spec.t(l, TP_ROLE_W);
          pack_rows16x128(reinterpret_cast<const uint16_t*>(static_cast<const char*>(host_weights) + t.offset),
                          reinterpret_cast<uint16_t*>(static_cast<char*>(m->host) + t.offset), W, W);
        }
      });
    for (auto& t : th) t.join();
  }
  if (c->cfg.copy_method == TP_COPY_PAGEABLE) {
    m->pageable.reset(new (std::nothrow) char[nb]);
    if (!m->pageable) {
      free_model(m.get());
      return fail(TP_E_NOSPC, "out of host memory (pageable model copy)");
    }
    std::memcpy(m->pageable.get(), m->host, nb);
  }
  e = hipHostGetDevicePointer(&m->host_dev, m->host, 0);
  if (c->cfg.flags & TP_FLAG_TRACE) {
    // timing events for as many chunks as the largest plan so far (made once, kept)
    for (auto* v : {&c->tl.copy_begin, &c->tl.copy_end, &c->tl.exec_begin})
      while (e == hipSuccess && v->size() < m->chunks.size()) {
        hipEvent_t ev = nullptr;
        e = hipEventCreate(&ev);
        if (e == hipSuccess) v->push_back(ev);
      }
  }
  m->chunk_ev.assign(m->chunks.size(), nullptr);
  for (size_t i = 0; e == hipSuccess && i < m->chunks.size(); ++i)
    e = hipEventCreateWithFlags(&m->chunk_ev[i], hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&m->last_use, hipEventDisableTiming);
  if (e != hipSuccess) {
    free_model(m.get());
    return hip_fail(e, "tp_register_model: event or mapping setup");
  }
  if (c->policy->add_model(m->id, nb, m->heavy_auto) != TP_OK) {
    free_model(m.get());
    return fail(TP_E_STATE, "model id collision");
  }
  *model_id = m->id;
  c->models[m->id] = std::move(m);
  ++c->next_id;
  return ok();
}

tp_status tp_unregister_model(tp_ctx* c, int32_t id) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  // the copy streams may still read the host copy; the last use may still read the extent
  TP_HIP(sync_copies(c));
  if (m->used) TP_HIP(hipEventSynchronize(m->last_use));
  if (c->policy->resident(id)) c->policy->evict(id);
  c->retired.erase(std::remove_if(c->retired.begin(), c->retired.end(),
                                  [&](const tp_ctx::Retired& r) { return r.model == id; }),
                   c->retired.end());
  c->policy->remove_model(id);
  free_model(m);
  c->models.erase(id);
  return ok();
}

tp_status tp_infer(tp_ctx* c, int32_t id, const void* input_dev, int32_t batch, void* output_dev, void* stream_) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  return infer_request(c, id, input_dev, batch, output_dev, static_cast<hipStream_t>(stream_), c->work,
                       c->cfg.work_bytes, "tp_infer");
}

tp_status tp_infer_noalloc(tp_ctx* c, int32_t id, const void* input_dev, int32_t batch, void* output_dev,
                           void* stream_) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  char* work = scratch_region(c->device);
  if (!work) return fail(TP_E_HIP, "tp_infer_noalloc: the static workspace's address could not be resolved on device " +
                                        std::to_string(c->device) + " at tp_create");
  Model* m = find(c, id);
  if (m && batch >= 1 && workspace_bytes(m->spec, batch) > kNoAllocScratchBytes)
    return fail(TP_E_NOSPC, "tp_infer_noalloc: the request needs " + std::to_string(workspace_bytes(m->spec, batch)) +
                                " bytes of workspace; the static workspace holds " +
                                std::to_string(kNoAllocScratchBytes));
  // kernels launched one by one: instantiating a graph may allocate device memory
  return infer_request(c, id, input_dev, batch, output_dev, static_cast<hipStream_t>(stream_), work,
                       kNoAllocScratchBytes, "tp_infer_noalloc", false, false);
}

tp_status tp_swap_in(tp_ctx* c, int32_t id, void* stream_) {
  Model* m = nullptr;
  tp_status s = check_request(c, id, &m);
  if (s != TP_OK) return s;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  if ((s = begin_request(c, stream)) != TP_OK) return s;
  bool swapped = false;
  if ((s = admit(c, m, &swapped)) != TP_OK) return s;
  if (!swapped) TP_HIP(settle(m, stream));
  if (swapped) {
    Waiter w;
    w.m = m;
    w.ctx = c;
    w.base_off = c->policy->offset(id);
    hipError_t e = w.issue_through((int)m->chunks.size() - 1);
    if (e != hipSuccess) {
      c->policy->evict(id);
      (void)retire(c, id, w.base_off, m->spec.host_bytes);
      return hip_fail(e, "tp_swap_in: copy enqueue");
    }
    const size_t n = m->chunk_ev.size();
    TP_HIP(hipStreamWaitEvent(stream, m->chunk_ev[n - 1], 0));
    if (c->ncopy == 2 && n > 1) TP_HIP(hipStreamWaitEvent(stream, m->chunk_ev[n - 2], 0));
    m->touch_due = true;
  }
  return end_request(c, m, stream);
}

tp_status tp_evict(tp_ctx* c, int32_t id) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  if (!find(c, id)) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  if (!c->policy->resident(id)) return ok();
  const uint64_t off = c->policy->offset(id), len = c->policy->bytes(id);
  c->policy->evict(id);
  return retire(c, id, off, len);
}

tp_status tp_last_timeline(tp_ctx* c, float* copy_begin, float* copy_end, float* exec_begin, uint32_t cap,
                           uint32_t* n, float* total_ms) {
  if (!c || !n) return fail(TP_E_INVAL, "NULL argument");
  if (!(c->cfg.flags & TP_FLAG_TRACE) || !c->tl.valid) return fail(TP_E_STATE, "no traced cold request");
  TP_HIP(hipEventSynchronize(c->tl.done));
  *n = c->tl.n;
  if (total_ms) TP_HIP(hipEventElapsedTime(total_ms, c->tl.start, c->tl.done));
  const uint32_t k = std::min<uint32_t>(std::min<uint32_t>(cap, c->tl.n), (uint32_t)c->tl.copy_begin.size());
  for (uint32_t i = 0; i < k; ++i) {
    if (copy_begin) TP_HIP(hipEventElapsedTime(&copy_begin[i], c->tl.start, c->tl.copy_begin[i]));
    if (copy_end) TP_HIP(hipEventElapsedTime(&copy_end[i], c->tl.start, c->tl.copy_end[i]));
    if (exec_begin) TP_HIP(hipEventElapsedTime(&exec_begin[i], c->tl.start, c->tl.exec_begin[i]));
  }
  return ok();
}

tp_status tp_is_resident(tp_ctx* c, int32_t id, int32_t* resident) {
  if (!c || !resident) return fail(TP_E_INVAL, "NULL argument");
  if (!find(c, id)) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  *resident = c->policy->resident(id) ? 1 : 0;
  return ok();
}

tp_status tp_arena_stats(tp_ctx* c, tp_arena_stats_t* out) {
  if (!c || !out) return fail(TP_E_INVAL, "NULL argument");
  c->policy->stats(out);
  out->admit_calls = c->admit_calls;
  out->admit_ns_total = c->admit_ns_total;
  out->admit_ns_max = c->admit_ns_max;
  out->graph_captures = c->graph_captures;
  out->graph_repoints = c->graph_repoints;
  out->graph_rebases = c->graph_rebases;
  out->cache_touches = c->cache_touches;
  return ok();
}

tp_status tp_debug_fail_copy(tp_ctx* c, int32_t nth) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  if (nth < 0) return fail(TP_E_INVAL, "tp_debug_fail_copy: nth < 0");
  c->fail_copy = nth;
  return ok();
}

tp_status tp_model_info(tp_ctx* c, int32_t id, tp_model_info_t* out) {
  if (!c || !out) return fail(TP_E_INVAL, "NULL argument");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  out->host_bytes = m->spec.host_bytes;
  out->param_bytes = m->spec.param_bytes;
  out->n_chunks = (uint32_t)m->chunks.size();
  out->resident = c->policy->resident(id) ? 1 : 0;
  out->extent_offset = c->policy->offset(id);
  out->last_use_clock = c->policy->last_use(id);
  out->heavy = c->policy->heavy(id) ? 1 : 0;
  out->cold_est_us = m->cold_est_us;
  out->warm_est_us = m->warm_est_us;
  return ok();
}

tp_status tp_set_model_class(tp_ctx* c, int32_t id, int32_t cls) {
  if (!c) return fail(TP_E_INVAL, "NULL context");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  if (cls < TP_CLASS_AUTO || cls > TP_CLASS_HEAVY) return fail(TP_E_INVAL, "unknown model class");
  c->policy->set_heavy(id, cls == TP_CLASS_AUTO ? m->heavy_auto : cls == TP_CLASS_HEAVY);
  return ok();
}

tp_status tp_model_host_image(tp_ctx* c, int32_t id, const void** ptr, uint64_t* bytes) {
  if (!c || !ptr || !bytes) return fail(TP_E_INVAL, "NULL argument");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  *ptr = m->host;
  *bytes = m->spec.host_bytes;
  return ok();
}

tp_status tp_model_chunks(tp_ctx* c, int32_t id, uint64_t* begin, uint64_t* end, uint32_t* first_layer,
                          uint32_t cap, uint32_t* n) {
  if (!c || !n) return fail(TP_E_INVAL, "NULL argument");
  Model* m = find(c, id);
  if (!m) return fail(TP_E_NOENT, "unknown model id " + std::to_string(id));
  *n = (uint32_t)m->chunks.size();
  for (uint32_t i = 0; i < m->chunks.size() && i < cap; ++i) {
    if (begin) begin[i] = m->chunks[i].begin;
    if (end) end[i] = m->chunks[i].end;
    if (first_layer) first_layer[i] = m->chunks[i].first_layer;
  }
  return ok();
}

tp_status tp_workspace_bytes(const tp_model_desc* desc, int32_t batch, uint64_t* bytes) {
  if (!desc || !bytes || batch < 1) return fail(TP_E_INVAL, "tp_workspace_bytes: bad argument");
  if (!desc->tensors || desc->n_tensors == 0) return fail(TP_E_INVAL, "descriptor has no tensors");
  uint64_t host = 0;
  for (uint32_t i = 0; i < desc->n_tensors; ++i)
    host = std::max(host, desc->tensors[i].offset + desc->tensors[i].bytes);
  ModelSpec m;
  std::string err;
  tp_status s = validate_model(desc, host, &m, &err);
  if (s != TP_OK) return fail(s, err);
  *bytes = workspace_bytes(m, batch);
  return ok();
}

}  // extern "C"
