// Model descriptors: validation against each family's architecture, the transfer-chunk
// plan and workspace sizing. Host-only C++ (no HIP).
#pragma once
#include <cstdint>
#include <string>
#include <vector>

#include "torpor.h"

namespace tp {

struct ConvShape {      // one convolution of the ResNet family, in first-use order
  int cout, k, cin, stride, pad;
};

// The 53 convolutions of ResNet-50 v1.5 (per bottleneck: 1x1, 3x3 carrying the stage
// stride, 1x1, then the projection shortcut in each stage's first block).
std::vector<ConvShape> resnet50_convs();

struct ConvGeom {       // a convolution with its input and output spatial size
  ConvShape c;
  int hin, hout;
};
// Geometry of every convolution at a square input of `image` pixels (conv1, then the
// 3x3/2 pad-1 max-pool, then the bottlenecks; the shortcut reads the block input).
std::vector<ConvGeom> resnet50_geometry(int image);

struct Chunk {
  uint64_t begin, end;          // host byte range [begin, end)
  uint32_t first_layer, last_layer;
};

struct ModelSpec {
  int32_t arch = 0, dtype = 0;
  int32_t dims[8] = {};
  std::vector<tp_tensor_desc> tensors;
  uint64_t host_bytes = 0;      // rounded up to 256
  uint64_t param_bytes = 0;
  uint32_t n_layers = 0;
  std::vector<int32_t> lookup;  // (layer * kRoles + role) -> tensor index, -1 if absent
  static constexpr int kRoles = 32;
  bool packed_mlp = false;      // bf16 MLP weights stored in 16 x 128 blocks (see pack_rows16x128)

  const tp_tensor_desc& t(uint32_t layer, uint32_t role) const {
    return tensors[lookup[layer * kRoles + role]];
  }
};

// Validates `d` against its family (see torpor.h) and fills `out`. Returns TP_OK or
// TP_E_INVAL with a message in *err.
tp_status validate_model(const tp_model_desc* d, uint64_t host_bytes, ModelSpec* out, std::string* err);

// Greedy grouping in first-use order: whole layers (or, with per_tensor, whole tensors); a
// chunk is closed at the first layer (tensor) boundary where it holds >= min_bytes. Chunks
// tile [0, host_bytes). With per_tensor a layer may span several chunks: first_layer and
// last_layer are the layers of a chunk's first and last tensor.
std::vector<Chunk> plan_chunks(const ModelSpec& m, uint64_t min_bytes, bool per_tensor = false);

// Pipeline-aware grouping. Model of a cold request: chunk copies run back to back on one
// copy stream, each costing chunk_us plus its bytes at link_bytes_per_us; a layer's kernels
// start when the previous layer has finished and, for the first layer of a chunk, wait_us
// after that chunk has landed; layer l then runs for layer_us[l]. Over the units (layers)
// starting at host offsets unit_begin[0..n) (unit 0 at byte 0) of a buffer of total_bytes,
// plan_cost picks the chunk boundaries that minimise the modelled completion time (ties:
// fewer chunks) by dynamic programming, and returns the first unit of every chunk.
struct LinkModel {
  double link_bytes_per_us = 57.0e3;   // bytes per microsecond (57 GB/s)
  double chunk_us = 15.0;              // fixed cost of one copy and its event
  double wait_us = 5.0;                // from a chunk's event to the first kernel that waits for it
};
std::vector<uint32_t> plan_cost(const std::vector<uint64_t>& unit_begin, uint64_t total_bytes,
                                const std::vector<double>& layer_us, const LinkModel& lm, double* est_us);

// Modelled completion time of a given grouping (chunk c starts at unit first[c]).
double plan_time(const std::vector<uint64_t>& unit_begin, uint64_t total_bytes, const std::vector<double>& layer_us,
                 const LinkModel& lm, const std::vector<uint32_t>& first);

// Estimated time (us) of each layer's kernels for a batch of `batch` samples: per kernel a
// fixed launch-and-drain cost plus its FLOPs and bytes at sustained rates of the layer
// kernels. Coarse by design: the plan only needs compute and transfer in proportion.
std::vector<double> layer_cost_us(const ModelSpec& m, int32_t batch);

// plan_cost over the model's layers with layer_cost_us(batch), as chunks tiling the buffer.
std::vector<Chunk> plan_chunks_cost(const ModelSpec& m, int32_t batch, const LinkModel& lm, double* est_us = nullptr);

// Activation buffers of the executors for `batch` samples (each buffer 256-aligned).
uint64_t activation_bytes(const ModelSpec& m, int32_t batch);

// fp32 partial tiles for contractions split over k (bf16 families only); placed after
// the activation buffers.
constexpr uint64_t kSplitScratch = 32ull << 20;

// Workspace needed by tp_infer: activations, then the split scratch.
uint64_t workspace_bytes(const ModelSpec& m, int32_t batch);

inline uint64_t round_up(uint64_t n, uint64_t a) { return (n + a - 1) / a * a; }

// Bounds of the bytes a warm request pre-reads into the caches (a span smaller is not missed
// for long enough to matter; one larger would not stay in the 256 MB Infinity Cache beside
// everything else).
constexpr uint64_t kTouchMinBytes = 4ull << 20, kTouchMaxBytes = 192ull << 20;

// The part [*lo, *hi) of a model's extent that a warm request pre-reads into the caches: all
// of it but a leading token-embedding table, of which a request reads only its ids' rows
// (BERT-base: 47 of 218 MB). False for an MLP, whose warm pass streams its weights at the rate
// a second reader would (the two would only compete for the same bytes), and for a span
// outside [kTouchMinBytes, kTouchMaxBytes].
bool touch_span(const ModelSpec& s, uint64_t* lo, uint64_t* hi);

// Blocked copy of a bf16 [N][K] matrix (N % 16 == 0, K % 128 == 0): block (n/16, k/128) is
// 2048 contiguous elements ordered [(k%128)/32][(k%32)/8][n%16][k%8], so that one 16-byte load
// per lane of a 64-lane wave reads a whole 1 KB run of a skinny-GEMM operand.
void pack_rows16x128(const uint16_t* src, uint16_t* dst, int64_t N, int64_t K);

}  // namespace tp
