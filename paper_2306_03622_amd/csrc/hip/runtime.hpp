// Runtime state of a context: registered models with their pinned host copies and
// events, the arena bookkeeping, the copy stream, and the per-request ordering state.
#pragma once
#include <hip/hip_runtime_api.h>

#include <memory>
#include <string>
#include <unordered_map>
#include <vector>

#include "../core/arena.hpp"
#include "../core/model.hpp"
#include "../kernels/kernels.hpp"
#include "torpor.h"

namespace tp {

// An instantiated graph of one warm forward pass of a model at one batch size, over one
// arena extent and one workspace. Its kernels' arguments name the input and output buffers
// of the request it was captured from; `launches` holds every kernel's recorded arguments, so
// a later request with other buffers repoints the kernel nodes that hold those two addresses
// in place (hipGraphExecKernelNodeSetParams) instead of capturing the pass again.
// Which pointers a recorded launch of a graph holds (GraphEntry::use).
enum : uint8_t { kUsesWeights = 1, kUsesBuffers = 2 };

struct GraphEntry {
  int batch = 0;
  const char* cap_base = nullptr;   // the weights' extent at capture, and its size
  uint64_t extent_bytes = 0;
  const char* cur_base = nullptr;   // the extent the instantiated nodes point into now
  const char* work = nullptr;
  const void* cap_in = nullptr;   // buffers of the captured request
  void* cap_out = nullptr;
  const void* cur_in = nullptr;   // buffers the instantiated nodes hold now
  void* cur_out = nullptr;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  std::vector<hipGraphNode_t> nodes;        // kernel nodes in launch order
  std::vector<k::LaunchRecord> launches;    // the same launches as recorded at capture
  std::vector<uint8_t> use;                 // per launch: kUsesWeights | kUsesBuffers
  bool patchable = false;                   // nodes and records matched one to one
  uint64_t stamp = 0;
};

struct Model {
  int32_t id = 0;
  ModelSpec spec;
  std::vector<Chunk> chunks;
  std::vector<uint32_t> chunk_of_layer;
  void* host = nullptr;          // pinned, device-mapped copy of the weights
  void* host_dev = nullptr;      // its device-visible address
  std::unique_ptr<char[]> pageable;  // ordinary host copy (TP_COPY_PAGEABLE contexts only)
  std::vector<hipEvent_t> chunk_ev;
  hipEvent_t last_use = nullptr;
  bool used = false;             // last_use has been recorded at least once
  bool bg_pending = false;       // swapped in behind a direct-access request: the next
                                 // request must wait for the last chunk's event
  bool touch_due = false;        // swapped in by tp_swap_in and read by no request since, so
                                 // its bytes are not in the caches (see maybe_touch)
  std::vector<GraphEntry> graphs;
  bool graph_failed = false;     // capture failed once: launch this model kernel by kernel
  float cold_est_us = 0, warm_est_us = 0;   // cost-model estimates at the context's plan batch
  bool heavy_auto = false;       // heaviness class from the estimates
};

// Drives a cold request's swap from the layer loop. Before the first kernel of a layer,
// need() issues the copies of every chunk up to the one holding that layer (each copy
// followed by its event on a copy stream) and makes `stream` wait for those events.
// Copies are thus issued interleaved with the layer kernels: copy c+1 is enqueued after
// the kernels of chunk c. When the runtime maps the copy stream onto the same hardware
// queue as the compute stream, this order keeps each chunk's event packet behind the
// kernels that precede it instead of ahead of all of them.
//
// A forked request runs the layers of every chunk but the last on the library's execution
// stream and hands back to the caller's stream (`caller`) for the last chunk's layers: the
// caller's stream then waits for the execution stream's work so far (which is done long
// before the last chunk lands in a transfer-bound request) and for the last chunk itself,
// so the hand-back adds no latency at the end. `slot` is the stream the layer kernels are
// launched on (the request's ExecCtx::stream), switched at the hand-back.
struct Waiter {
  const Model* m = nullptr;
  hipStream_t stream = nullptr;
  bool swapping = false;
  int waited = -1;
  tp_ctx* ctx = nullptr;
  uint64_t base_off = 0;
  int issued = 0;                // chunks whose copies are enqueued
  hipStream_t caller = nullptr;  // forked requests: the caller's stream, else null
  hipStream_t* slot = nullptr;
  hipError_t issue_through(int c);
  hipError_t hand_back();
  hipError_t need(uint32_t layer) {
    if (!swapping) return hipSuccess;
    const int c = (int)m->chunk_of_layer[layer];
    hipError_t e = issue_through(c);
    if (e == hipSuccess && caller && c == (int)m->chunks.size() - 1) e = hand_back();
    while (e == hipSuccess && waited < c) {
      ++waited;
      e = hipStreamWaitEvent(stream, m->chunk_ev[waited], 0);
      if (e == hipSuccess) e = trace_exec(waited);
    }
    return e;
  }
  hipError_t trace_exec(int c);
};

// Device addresses of the running request.
struct ExecCtx {
  const Model* m;
  char* base;        // arena extent base of the model
  char* work;        // workspace
  const void* in;
  void* out;
  int batch;
  hipStream_t stream;
  Waiter* wait;
  k::Split split;    // scratch for contractions split over k
  template <typename T>
  const T* t(uint32_t layer, uint32_t role) const {
    return reinterpret_cast<const T*>(base + m->spec.t(layer, role).offset);
  }
};

hipError_t run_mlp(ExecCtx& x);
// An fp32 MLP's cold forward that is also its swap-in: the first layer reads its weights from
// the pinned host image and, in the same launch, the whole image is copied into the extent at
// x.base; the other layers then run from the extent. Same results as run_mlp.
bool mlp_swapin_fits(const ModelSpec& s, int batch);
hipError_t run_mlp_swapin(ExecCtx& x, const void* host_image);
hipError_t run_resnet(ExecCtx& x);
hipError_t run_bert(ExecCtx& x);

}  // namespace tp

struct tp_ctx {
  int device = 0;
  tp_config cfg{};
  char* arena = nullptr;
  char* work = nullptr;
  hipStream_t copy[2] = {nullptr, nullptr};   // copy[0] carries all ordering waits
  int ncopy = 1;
  bool own_copy = false;
  hipEvent_t fork = nullptr;                   // copy[1] starts a swap after copy[0]
  hipEvent_t claim_ev = nullptr;               // a swap-in kernel's stream waits for copy[0]
  hipStream_t capture = nullptr;               // private stream for graph capture
  uint64_t graph_clock = 0;
  uint64_t graph_captures = 0, graph_repoints = 0, graph_rebases = 0;
  // warm requests' cache touch (see maybe_touch): 64 words the touch kernel may write, the
  // model the previous request served (0: none yet), touches launched
  uint32_t* touch_sink = nullptr;
  int32_t last_served = 0;
  uint64_t cache_touches = 0;
  // cold (swapping) requests run on the library's execution stream, forked from and joined
  // back to the caller's stream (null under TP_FLAG_CALLER_STREAM)
  hipStream_t exec = nullptr;
  hipEvent_t exec_fork = nullptr, exec_join = nullptr;
  int32_t fail_copy = 0;                       // tp_debug_fail_copy countdown (0: off)
  std::unique_ptr<tp::Arena> policy;
  std::unordered_map<int32_t, std::unique_ptr<tp::Model>> models;
  int32_t next_id = 1;
  // request ordering across caller streams
  hipEvent_t req_done = nullptr;
  hipStream_t last_stream = nullptr;
  bool any_request = false;
  std::vector<hipEvent_t> trace_ev;            // completion ring of tp_run_trace
  uint64_t admit_calls = 0, admit_ns_total = 0, admit_ns_max = 0;   // admissions that missed
  uint64_t last_admit_ns = 0;                                         // the latest of them
  // extents invalidated but possibly still read by enqueued work of their old owner
  struct Retired {
    uint64_t off, len;
    int32_t model;
  };
  std::vector<Retired> retired;
  // TP_FLAG_TRACE: timing events of the last traced cold request
  struct Timeline {
    hipEvent_t start = nullptr, done = nullptr;
    std::vector<hipEvent_t> copy_begin, copy_end, exec_begin;   // per chunk
    uint32_t n = 0;                  // chunks of the traced request
    bool active = false;             // the request being enqueued is traced
    bool valid = false;
  } tl;
};
