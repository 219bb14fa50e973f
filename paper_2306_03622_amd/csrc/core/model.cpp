#include "model.hpp"

#include <algorithm>
#include <cstdio>

namespace tp {

std::vector<ConvShape> resnet50_convs() {
  std::vector<ConvShape> v;
  v.push_back({64, 7, 3, 2, 3});
  const int blocks[4] = {3, 4, 6, 3}, mids[4] = {64, 128, 256, 512};
  int cin = 64;
  for (int s = 0; s < 4; ++s) {
    const int mid = mids[s], out = 4 * mid;
    for (int b = 0; b < blocks[s]; ++b) {
      const int stride = (s > 0 && b == 0) ? 2 : 1;
      v.push_back({mid, 1, cin, 1, 0});
      v.push_back({mid, 3, mid, stride, 1});
      v.push_back({out, 1, mid, 1, 0});
      if (b == 0) v.push_back({out, 1, cin, stride, 0});
      cin = out;
    }
  }
  return v;
}

std::vector<ConvGeom> resnet50_geometry(int image) {
  const auto convs = resnet50_convs();
  std::vector<ConvGeom> g;
  auto out = [](int h, const ConvShape& c) { return (h + 2 * c.pad - c.k) / c.stride + 1; };
  const int h1 = out(image, convs[0]);
  g.push_back({convs[0], image, h1});
  int cur = (h1 + 2 - 3) / 2 + 1;   // max-pool
  size_t i = 1;
  const int blocks[4] = {3, 4, 6, 3};
  for (int s = 0; s < 4; ++s) {
    for (int b = 0; b < blocks[s]; ++b) {
      const int h_in = cur;
      const int h_a = out(h_in, convs[i]);
      g.push_back({convs[i], h_in, h_a}); ++i;                       // 1x1
      const int h_b = out(h_a, convs[i]);
      g.push_back({convs[i], h_a, h_b}); ++i;                        // 3x3 (stride)
      g.push_back({convs[i], h_b, out(h_b, convs[i])}); ++i;         // 1x1
      if (b == 0) { g.push_back({convs[i], h_in, out(h_in, convs[i])}); ++i; }   // shortcut
      cur = h_b;
    }
  }
  return g;
}

namespace {

struct Want {
  uint32_t layer, role;
  int64_t shape[4];
};

std::string fmt(const char* f, long long a = 0, long long b = 0, long long c = 0, long long d = 0) {
  char buf[256];
  std::snprintf(buf, sizeof buf, f, a, b, c, d);
  return buf;
}

bool expected(const tp_model_desc* d, std::vector<Want>* w, uint32_t* n_layers, std::string* err) {
  const int32_t* D = d->dims;
  auto add = [&](uint32_t l, uint32_t r, int64_t a, int64_t b = 0, int64_t c = 0, int64_t e = 0) {
    w->push_back({l, r, {a, b, c, e}});
  };
  switch (d->arch) {
    case TP_ARCH_MLP: {
      const int L = D[0], W = D[1], act = D[2];
      if (L < 1 || L > 4096 || W < 8 || W % 8 || W > 65536 || act < 0 || act > 2) {
        *err = fmt("MLP dims {layers=%lld, width=%lld, act=%lld}: need layers>=1, width%%8==0, act in 0..2",
                   L, W, act);
        return false;
      }
      if (d->dtype != TP_F32 && d->dtype != TP_BF16) { *err = "MLP dtype must be TP_F32 or TP_BF16"; return false; }
      for (int l = 0; l < L; ++l) { add(l, TP_ROLE_W, W, W); add(l, TP_ROLE_B, W); }
      *n_layers = L;
      return true;
    }
    case TP_ARCH_RESNET50: {
      const int classes = D[0], image = D[1];
      if (classes < 1 || classes > 65536 || image < 32 || image % 32 || image > 1024) {
        *err = fmt("ResNet dims {classes=%lld, image=%lld}: need classes>=1, image%%32==0, 32<=image<=1024",
                   classes, image);
        return false;
      }
      if (d->dtype != TP_BF16) { *err = "ResNet dtype must be TP_BF16"; return false; }
      auto convs = resnet50_convs();
      uint32_t l = 0;
      for (auto& c : convs) { add(l, TP_ROLE_W, c.cout, c.k, c.k, c.cin); add(l, TP_ROLE_B, c.cout); ++l; }
      add(l, TP_ROLE_W, classes, 2048); add(l, TP_ROLE_B, classes);
      *n_layers = l + 1;
      return true;
    }
    case TP_ARCH_BERT: {
      const int L = D[0], dm = D[1], H = D[2], F = D[3], S = D[4], V = D[5], P = D[6];
      if (L < 1 || H < 1 || dm != 64 * H || dm > 1024 || F < 8 || F % 8 || F > 16384 || S < 32 || S % 32 ||
          S > 256 || P < S || V < 1) {
        *err = "BERT dims {layers, d, heads, ffn, seq, vocab, maxpos}: need d == 64*heads <= 1024, "
               "ffn%8==0, seq%32==0, 32<=seq<=256, maxpos>=seq, vocab>=1";
        return false;
      }
      if (d->dtype != TP_BF16) { *err = "BERT dtype must be TP_BF16"; return false; }
      add(0, TP_ROLE_TOK_EMB, V, dm); add(0, TP_ROLE_POS_EMB, P, dm); add(0, TP_ROLE_TYPE_EMB, 2, dm);
      add(0, TP_ROLE_EMB_LN_G, dm); add(0, TP_ROLE_EMB_LN_B, dm);
      for (int l = 1; l <= L; ++l) {
        add(l, TP_ROLE_QKV_W, 3 * dm, dm); add(l, TP_ROLE_QKV_B, 3 * dm);
        add(l, TP_ROLE_O_W, dm, dm); add(l, TP_ROLE_O_B, dm);
        add(l, TP_ROLE_LN1_G, dm); add(l, TP_ROLE_LN1_B, dm);
        add(l, TP_ROLE_FFN1_W, F, dm); add(l, TP_ROLE_FFN1_B, F);
        add(l, TP_ROLE_FFN2_W, dm, F); add(l, TP_ROLE_FFN2_B, dm);
        add(l, TP_ROLE_LN2_G, dm); add(l, TP_ROLE_LN2_B, dm);
      }
      *n_layers = L + 1;
      return true;
    }
    default:
      *err = fmt("unknown arch %lld", d->arch);
      return false;
  }
}

}  // namespace

tp_status validate_model(const tp_model_desc* d, uint64_t host_bytes, ModelSpec* out, std::string* err) {
  if (!d || !out) { *err = "NULL descriptor"; return TP_E_INVAL; }
  if (d->n_tensors == 0 || !d->tensors) { *err = "descriptor has no tensors"; return TP_E_INVAL; }
  std::vector<Want> want;
  uint32_t n_layers = 0;
  if (!expected(d, &want, &n_layers, err)) return TP_E_INVAL;
  if (d->n_tensors != want.size()) {
    *err = fmt("descriptor lists %lld tensors, the architecture has %lld", d->n_tensors, (long long)want.size());
    return TP_E_INVAL;
  }
  const uint64_t esz = d->dtype == TP_F32 ? 4 : 2;
  ModelSpec m;
  m.arch = d->arch;
  m.dtype = d->dtype;
  std::copy(d->dims, d->dims + 8, m.dims);
  m.n_layers = n_layers;
  m.lookup.assign((size_t)n_layers * ModelSpec::kRoles, -1);
  m.tensors.assign(d->tensors, d->tensors + d->n_tensors);
  uint64_t prev_end = 0;
  uint32_t prev_layer = 0;
  for (uint32_t i = 0; i < d->n_tensors; ++i) {
    const tp_tensor_desc& t = d->tensors[i];
    if (t.layer >= n_layers || t.role >= (uint32_t)ModelSpec::kRoles) {
      *err = fmt("tensor %lld: layer %lld / role %lld out of range", i, t.layer, t.role);
      return TP_E_INVAL;
    }
    int32_t& slot = m.lookup[t.layer * ModelSpec::kRoles + t.role];
    if (slot >= 0) { *err = fmt("tensor %lld: duplicate (layer %lld, role %lld)", i, t.layer, t.role); return TP_E_INVAL; }
    slot = (int32_t)i;
    if (i > 0 && t.layer < prev_layer) {
      *err = fmt("tensor %lld: layers must not decrease (first-use order)", i);
      return TP_E_INVAL;
    }
    if (t.offset % 256) { *err = fmt("tensor %lld: offset %lld not 256-byte aligned", i, (long long)t.offset); return TP_E_INVAL; }
    if (i > 0 && t.offset < prev_end) { *err = fmt("tensor %lld overlaps or precedes the previous one", i); return TP_E_INVAL; }
    if (t.offset + t.bytes > host_bytes || t.offset + t.bytes < t.offset) {
      *err = fmt("tensor %lld: [%lld, +%lld) exceeds the host buffer", i, (long long)t.offset, (long long)t.bytes);
      return TP_E_INVAL;
    }
    prev_end = t.offset + t.bytes;
    prev_layer = t.layer;
    m.param_bytes += t.bytes;
  }
  for (const Want& w : want) {
    const int32_t idx = m.lookup[w.layer * ModelSpec::kRoles + w.role];
    if (idx < 0) { *err = fmt("missing tensor (layer %lld, role %lld)", w.layer, w.role); return TP_E_INVAL; }
    const tp_tensor_desc& t = m.tensors[idx];
    uint64_t n = 1;
    for (int k = 0; k < 4; ++k) {
      if (t.shape[k] != w.shape[k]) {
        *err = fmt("tensor (layer %lld, role %lld): shape[%lld] = %lld differs from the architecture",
                   w.layer, w.role, k, t.shape[k]);
        return TP_E_INVAL;
      }
      if (w.shape[k]) n *= (uint64_t)w.shape[k];
    }
    if (t.bytes != n * esz) {
      *err = fmt("tensor (layer %lld, role %lld): %lld bytes, shape needs %lld", w.layer, w.role,
                 (long long)t.bytes, (long long)(n * esz));
      return TP_E_INVAL;
    }
  }
  m.host_bytes = round_up(host_bytes, 256);
  m.packed_mlp = m.arch == TP_ARCH_MLP && m.dtype == TP_BF16 && m.dims[1] % 128 == 0;
  *out = std::move(m);
  return TP_OK;
}

void pack_rows16x128(const uint16_t* src, uint16_t* dst, int64_t N, int64_t K) {
  const int64_t nkb = K / 128;
  for (int64_t t = 0; t < N / 16; ++t)
    for (int64_t kb = 0; kb < nkb; ++kb) {
      uint16_t* blk = dst + (t * nkb + kb) * 2048;
      for (int j = 0; j < 4; ++j)
        for (int q = 0; q < 4; ++q)
          for (int r = 0; r < 16; ++r) {
            const uint16_t* s8 = src + (t * 16 + r) * K + kb * 128 + j * 32 + q * 8;
            std::copy(s8, s8 + 8, blk + j * 512 + (q * 16 + r) * 8);
          }
    }
}

std::vector<Chunk> plan_chunks(const ModelSpec& m, uint64_t min_bytes, bool per_tensor) {
  // byte spans in first-use order: one per layer, or one per tensor
  struct Span { uint32_t layer; uint64_t begin, end; };
  std::vector<Span> spans;
  for (const auto& t : m.tensors) {
    if (!per_tensor && !spans.empty() && spans.back().layer == t.layer) spans.back().end = t.offset + t.bytes;
    else spans.push_back({t.layer, t.offset, t.offset + t.bytes});
  }
  std::vector<Chunk> out;
  bool open = false;
  Chunk cur{};
  for (const Span& s : spans) {
    if (!open) {
      cur.begin = out.empty() ? 0 : s.begin;
      cur.first_layer = s.layer;
      open = true;
    }
    cur.end = s.end;
    cur.last_layer = s.layer;
    if (cur.end - cur.begin >= min_bytes) { out.push_back(cur); open = false; }
  }
  if (open) out.push_back(cur);
  for (size_t i = 0; i + 1 < out.size(); ++i) out[i].end = out[i + 1].begin;
  out.back().end = m.host_bytes;
  return out;
}

double plan_time(const std::vector<uint64_t>& unit_begin, uint64_t total_bytes, const std::vector<double>& layer_us,
                 const LinkModel& lm, const std::vector<uint32_t>& first) {
  const size_t n = unit_begin.size(), nc = first.size();
  double copy_end = 0.0, done = 0.0;
  for (size_t c = 0; c < nc; ++c) {
    const uint32_t u0 = first[c], u1 = c + 1 < nc ? first[c + 1] : (uint32_t)n;
    const uint64_t b0 = c == 0 ? 0 : unit_begin[u0], b1 = c + 1 < nc ? unit_begin[u1] : total_bytes;
    copy_end += lm.chunk_us + (double)(b1 - b0) / lm.link_bytes_per_us;
    done = std::max(done, copy_end + lm.wait_us);
    for (uint32_t u = u0; u < u1; ++u) done += layer_us[u];
  }
  return done;
}

std::vector<uint32_t> plan_cost(const std::vector<uint64_t>& unit_begin, uint64_t total_bytes,
                                const std::vector<double>& layer_us, const LinkModel& lm, double* est_us) {
  // F[k][j]: earliest modelled finish of units [0, j) split into k chunks, the k-th ending
  // at unit j. The k-th chunk lands at A = k * chunk_us + begin(j) / rate whatever its own
  // start, so F[k][j] = min_i max(F[k-1][i], A + wait) + T(i, j).
  const size_t n = unit_begin.size();
  std::vector<double> T(n + 1, 0.0);
  for (size_t u = 0; u < n; ++u) T[u + 1] = T[u] + layer_us[u];
  auto bytes_to = [&](size_t j) { return j == n ? total_bytes : unit_begin[j]; };
  const double inf = 1e300;
  std::vector<double> F((n + 1) * (n + 1), inf);
  std::vector<uint32_t> arg((n + 1) * (n + 1), 0);
  auto at = [&](size_t k, size_t j) -> size_t { return k * (n + 1) + j; };
  F[at(0, 0)] = 0.0;
  for (size_t k = 1; k <= n; ++k)
    for (size_t j = k; j <= n; ++j) {
      const double land = (double)k * lm.chunk_us + (double)bytes_to(j) / lm.link_bytes_per_us + lm.wait_us;
      double best = inf;
      uint32_t bi = 0;
      for (size_t i = k - 1; i < j; ++i) {
        const double f = F[at(k - 1, i)];
        if (f >= inf) continue;
        const double v = std::max(f, land) + (T[j] - T[i]);
        if (v < best) { best = v; bi = (uint32_t)i; }
      }
      F[at(k, j)] = best;
      arg[at(k, j)] = bi;
    }
  double best = inf;
  for (size_t k = 1; k <= n; ++k) best = std::min(best, F[at(k, n)]);
  size_t kb = 1;
  while (F[at(kb, n)] > best + 1e-6 * (1.0 + best)) ++kb;   // fewest chunks among the optima
  std::vector<uint32_t> first(kb);
  size_t j = n;
  for (size_t k = kb; k >= 1; --k) {
    const uint32_t i = arg[at(k, j)];
    first[k - 1] = i;
    j = i;
  }
  if (est_us) *est_us = F[at(kb, n)];
  return first;
}

namespace {

// sustained rates of the layer kernels for the cost model (MI355X, bf16 MFMA kernels of
// this library at the shapes of the model families; measured per kernel)
constexpr double kKernelUs = 7.0;            // launch, fill and drain of one dependent kernel
constexpr double kFlopPerUs = 200.0e6;       // 200 TFLOP/s
constexpr double kBytePerUs = 3.5e6;         // 3.5 TB/s

double kernel_us(double flops, double bytes) { return kKernelUs + flops / kFlopPerUs + bytes / kBytePerUs; }

}  // namespace

std::vector<double> layer_cost_us(const ModelSpec& m, int32_t batch) {
  const double B = std::max(batch, 1);
  std::vector<double> t(m.n_layers, 0.0);
  switch (m.arch) {
    case TP_ARCH_MLP: {
      const double W = m.dims[1], esz = m.dtype == TP_F32 ? 4 : 2;
      for (auto& v : t) v = kernel_us(2 * B * W * W, W * W * esz + 2 * B * W * esz);
      break;
    }
    case TP_ARCH_RESNET50: {
      const auto g = resnet50_geometry(m.dims[1]);
      for (size_t l = 0; l < g.size() && l < t.size(); ++l) {
        const ConvGeom& c = g[l];
        const double hw_in = (double)c.hin * c.hin, hw_out = (double)c.hout * c.hout;
        const double k2 = (double)c.c.k * c.c.k;
        t[l] = kernel_us(2 * B * hw_out * c.c.cout * k2 * c.c.cin,
                         2 * (c.c.cout * k2 * c.c.cin + B * hw_in * c.c.cin + B * hw_out * c.c.cout));
      }
      // conv1 is followed by the max-pool; the FC by nothing but is preceded by the avg-pool
      const ConvGeom& c0 = g[0];
      const int hp = (c0.hout + 2 - 3) / 2 + 1;
      t[0] += kernel_us(0, 2 * B * c0.c.cout * ((double)c0.hout * c0.hout + (double)hp * hp));
      const double cls = m.dims[0];
      const ConvGeom& gl = g.back();
      t.back() = kernel_us(0, 2 * B * 2048 * ((double)gl.hout * gl.hout + 1)) +
                 kernel_us(2 * B * 2048 * cls, 2 * (2048 * cls + B * 2048) + 4 * B * cls);
      break;
    }
    case TP_ARCH_BERT: {
      const double d = m.dims[1], F = m.dims[3], S = m.dims[4], M = B * S;
      t[0] = kernel_us(0, M * d * 8);
      for (size_t l = 1; l < t.size(); ++l)
        t[l] = kernel_us(2 * M * d * 3 * d, 2 * (3 * d * d + M * d + 3 * M * d)) +        // QKV
               kernel_us(4 * B * S * S * d, 2 * (3 * M * d + M * d)) +                    // attention
               kernel_us(2 * M * d * d, 2 * (d * d + M * d) + 8 * M * d) +                 // O + residual
               kernel_us(0, 6 * M * d) +                                                 // LN
               kernel_us(2 * M * d * F, 2 * (d * F + M * d + M * F)) +                   // FFN1
               kernel_us(2 * M * F * d, 2 * (d * F + M * F) + 8 * M * d) +               // FFN2 + residual
               kernel_us(0, 6 * M * d);                                                  // LN
      break;
    }
  }
  return t;
}

std::vector<Chunk> plan_chunks_cost(const ModelSpec& m, int32_t batch, const LinkModel& lm, double* est_us) {
  // one unit per layer, starting at the layer's first tensor (unit 0 at byte 0)
  std::vector<uint64_t> begin;
  std::vector<uint32_t> layer_of;
  for (const auto& t : m.tensors)
    if (begin.empty() || layer_of.back() != t.layer) {
      begin.push_back(begin.empty() ? 0 : t.offset);
      layer_of.push_back(t.layer);
    }
  const std::vector<double> all = layer_cost_us(m, batch);
  std::vector<double> us(layer_of.size());
  for (size_t u = 0; u < us.size(); ++u) us[u] = all[layer_of[u]];
  const std::vector<uint32_t> first = plan_cost(begin, m.host_bytes, us, lm, est_us);
  std::vector<Chunk> out(first.size());
  for (size_t c = 0; c < first.size(); ++c) {
    const uint32_t u1 = c + 1 < first.size() ? first[c + 1] : (uint32_t)begin.size();
    out[c].begin = c == 0 ? 0 : begin[first[c]];
    out[c].end = c + 1 < first.size() ? begin[u1] : m.host_bytes;
    out[c].first_layer = layer_of[first[c]];
    out[c].last_layer = layer_of[u1 - 1];
  }
  return out;
}

uint64_t workspace_bytes(const ModelSpec& m, int32_t batch) {
  return activation_bytes(m, batch) + (m.dtype == TP_BF16 ? kSplitScratch : 0);
}

uint64_t activation_bytes(const ModelSpec& m, int32_t batch) {
  const uint64_t B = (uint64_t)std::max(batch, 1);
  switch (m.arch) {
    case TP_ARCH_MLP: {
      const uint64_t esz = m.dtype == TP_F32 ? 4 : 2;
      return 2 * round_up(B * m.dims[1] * esz, 256);
    }
    case TP_ARCH_RESNET50: {
      // five activation buffers sized for the largest per-sample activation, plus the
      // pooled features
      uint64_t best = 0;
      for (const auto& g : resnet50_geometry(m.dims[1]))
        best = std::max(best, (uint64_t)g.hout * g.hout * g.c.cout);
      return 5 * round_up(B * best * 2, 256) + round_up(B * 2048 * 2, 256);
    }
    case TP_ARCH_BERT: {
      const uint64_t M = B * m.dims[4], d = m.dims[1], F = m.dims[3];
      return round_up(M * d * 2, 256) * 2 + round_up(M * 3 * d * 2, 256) + round_up(M * d * 4, 256) +
             round_up(M * F * 2, 256);
    }
  }
  return 0;
}

bool touch_span(const ModelSpec& s, uint64_t* lo, uint64_t* hi) {
  if (s.arch == TP_ARCH_MLP) return false;
  uint64_t a = 0;
  for (const tp_tensor_desc& t : s.tensors)
    if (t.role == TP_ROLE_TOK_EMB && t.offset == 0) a = round_up(t.bytes, 256);
  const uint64_t b = s.host_bytes;
  if (a >= b || b - a < kTouchMinBytes || b - a > kTouchMaxBytes) return false;
  *lo = a;
  *hi = b;
  return true;
}

}  // namespace tp
