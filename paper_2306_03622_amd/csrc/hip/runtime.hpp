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
#include "torpor.h"

namespace tp {

struct Model {
  int32_t id = 0;
  ModelSpec spec;
  std::vector<Chunk> chunks;
  std::vector<uint32_t> chunk_of_layer;
  void* host = nullptr;          // pinned, device-mapped copy of the weights
  void* host_dev = nullptr;      // its device-visible address
  std::vector<hipEvent_t> chunk_ev;
  hipEvent_t last_use = nullptr;
  bool used = false;             // last_use has been recorded at least once
};

// Makes `stream` wait for the chunk holding a layer, once per chunk, in first-use order.
// Chunks complete in order on the single copy stream, so waiting for chunk c covers all
// earlier chunks.
struct Waiter {
  const Model* m = nullptr;
  hipStream_t stream = nullptr;
  bool swapping = false;
  int waited = -1;
  hipError_t need(uint32_t layer) {
    if (!swapping) return hipSuccess;
    const int c = (int)m->chunk_of_layer[layer];
    if (c <= waited) return hipSuccess;
    waited = c;
    return hipStreamWaitEvent(stream, m->chunk_ev[c], 0);
  }
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
  template <typename T>
  const T* t(uint32_t layer, uint32_t role) const {
    return reinterpret_cast<const T*>(base + m->spec.t(layer, role).offset);
  }
};

hipError_t run_mlp(ExecCtx& x);
hipError_t run_resnet(ExecCtx& x);
hipError_t run_bert(ExecCtx& x);

}  // namespace tp

struct tp_ctx {
  int device = 0;
  tp_config cfg{};
  char* arena = nullptr;
  char* work = nullptr;
  hipStream_t copy = nullptr;
  bool own_copy = false;
  std::unique_ptr<tp::Arena> policy;
  std::unordered_map<int32_t, std::unique_ptr<tp::Model>> models;
  int32_t next_id = 1;
  // request ordering across caller streams
  hipEvent_t req_done = nullptr;
  hipStream_t last_stream = nullptr;
  bool any_request = false;
  // extents invalidated but possibly still read by enqueued work of their old owner
  struct Retired {
    uint64_t off, len;
    int32_t model;
  };
  std::vector<Retired> retired;
};
