// Forward passes of the three model families as kernel sequences on the caller's
// stream. Every layer first asks the Waiter for the chunk holding its weights, so a
// cold request computes layer l while later chunks are still being copied. Kernel
// choice and launch shapes depend only on the model and the batch, never on residency
// or extent address, so pipelined, preloaded and relocated runs are bit-identical.
#include <algorithm>

#include "../kernels/kernels.hpp"
#include "../kernels/swapin.hpp"
#include "runtime.hpp"

namespace tp {

#define TP_TRY(expr)                       \
  do {                                     \
    hipError_t e_ = (expr);                \
    if (e_ != hipSuccess) return e_;       \
  } while (0)

hipError_t run_mlp(ExecCtx& x) {
  const ModelSpec& s = x.m->spec;
  const int L = s.dims[0], W = s.dims[1], act = s.dims[2], B = x.batch;
  const bool f32 = s.dtype == TP_F32;
  const uint64_t bytes = round_up((uint64_t)B * W * (f32 ? 4 : 2), 256);
  char* buf[2] = {x.work, x.work + bytes};
  const void* cur = x.in;
  for (int l = 0; l < L; ++l) {
    TP_TRY(x.wait->need(l));
    const bool last = l == L - 1;
    void* dst = last ? x.out : buf[l & 1];
    const int a = last ? k::ACT_NONE : act;
    if (f32) {
      TP_TRY(k::linear_f32(static_cast<const float*>(cur), B, W, x.t<float>(l, TP_ROLE_W), W,
                           x.t<float>(l, TP_ROLE_B), a, static_cast<float*>(dst), x.stream));
    } else {
      k::Epilogue ep;
      ep.bias = x.t<uint16_t>(l, TP_ROLE_B);
      ep.act = a;
      ep.out = dst;
      ep.out_f32 = last;
      ep.w_packed = s.packed_mlp;
      TP_TRY(k::linear_bf16(static_cast<const uint16_t*>(cur), B, W, x.t<uint16_t>(l, TP_ROLE_W), W, ep, x.split,
                             x.stream));
    }
    cur = dst;
  }
  return hipSuccess;
}

bool mlp_swapin_fits(const ModelSpec& s, int batch) {
  return s.arch == TP_ARCH_MLP && s.dtype == TP_F32 && batch <= 8 && s.dims[1] <= 1024 &&
         s.t(0, TP_ROLE_W).offset % 16 == 0;
}

hipError_t run_mlp_swapin(ExecCtx& x, const void* host_image) {
  const ModelSpec& s = x.m->spec;
  const int L = s.dims[0], W = s.dims[1], act = s.dims[2], B = x.batch;
  const uint64_t bytes = round_up((uint64_t)B * W * 4, 256);
  char* buf[2] = {x.work, x.work + bytes};
  void* dst = L == 1 ? x.out : buf[0];
  TP_TRY(k::linear_f32_swap(static_cast<const float*>(x.in), B, W, W, L == 1 ? k::ACT_NONE : act,
                            static_cast<float*>(dst), host_image, x.base, s.host_bytes, s.t(0, TP_ROLE_W).offset,
                            s.t(0, TP_ROLE_B).offset, x.stream));
  const void* cur = dst;
  for (int l = 1; l < L; ++l) {
    const bool last = l == L - 1;
    dst = last ? x.out : buf[l & 1];
    TP_TRY(k::linear_f32(static_cast<const float*>(cur), B, W, x.t<float>(l, TP_ROLE_W), W, x.t<float>(l, TP_ROLE_B),
                         last ? k::ACT_NONE : act, static_cast<float*>(dst), x.stream));
    cur = dst;
  }
  return hipSuccess;
}

hipError_t run_resnet(ExecCtx& x) {
  const ModelSpec& s = x.m->spec;
  const int classes = s.dims[0], image = s.dims[1], B = x.batch;
  const std::vector<ConvGeom> g = resnet50_geometry(image);
  uint64_t best = 0;
  for (const auto& c : g) best = std::max(best, (uint64_t)c.hout * c.hout * c.c.cout);
  const uint64_t bsz = round_up((uint64_t)B * best * 2, 256);
  uint16_t* buf[5];
  for (int i = 0; i < 5; ++i) buf[i] = reinterpret_cast<uint16_t*>(x.work + i * bsz);
  uint16_t* pooled = reinterpret_cast<uint16_t*>(x.work + 5 * bsz);

  auto conv = [&](uint32_t layer, const uint16_t* in, uint16_t* out, const void* res, int act) -> hipError_t {
    const ConvGeom& c = g[layer];
    TP_TRY(x.wait->need(layer));
    k::Epilogue ep;
    ep.bias = x.t<uint16_t>(layer, TP_ROLE_B);
    ep.res = res;
    ep.act = act;
    ep.out = out;
    return k::conv_bf16(in, B, c.hin, c.hin, c.c.cin, x.t<uint16_t>(layer, TP_ROLE_W), c.c.cout, c.c.k, c.c.k,
                        c.c.stride, c.c.pad, ep, x.split, x.stream);
  };

  TP_TRY(conv(0, static_cast<const uint16_t*>(x.in), buf[0], nullptr, k::ACT_RELU));
  TP_TRY(k::maxpool3s2(buf[0], B, g[0].hout, g[0].hout, g[0].c.cout, buf[1], x.stream));
  int cur = 1;
  uint32_t li = 1;
  const int blocks[4] = {3, 4, 6, 3};
  int hw = g[1].hin;
  for (int st = 0; st < 4; ++st) {
    for (int b = 0; b < blocks[st]; ++b) {
      int o[4], n = 0;
      for (int i = 0; i < 5; ++i)
        if (i != cur) o[n++] = i;
      const bool proj = b == 0;
      TP_TRY(conv(li, buf[cur], buf[o[0]], nullptr, k::ACT_RELU));          // 1x1
      TP_TRY(conv(li + 1, buf[o[0]], buf[o[1]], nullptr, k::ACT_RELU));     // 3x3, stage stride
      const uint16_t* res = buf[cur];
      if (proj) {                                                           // projection shortcut
        TP_TRY(conv(li + 3, buf[cur], buf[o[2]], nullptr, k::ACT_NONE));
        res = buf[o[2]];
      }
      TP_TRY(conv(li + 2, buf[o[1]], buf[o[3]], res, k::ACT_RELU));         // 1x1 + shortcut, ReLU
      hw = g[li + 2].hout;
      cur = o[3];
      li += proj ? 4 : 3;
    }
  }
  TP_TRY(k::avgpool(buf[cur], B, hw * hw, 2048, pooled, x.stream));
  TP_TRY(x.wait->need(li));
  k::Epilogue ep;
  ep.bias = x.t<uint16_t>(li, TP_ROLE_B);
  ep.out = x.out;
  ep.out_f32 = 1;
  return k::linear_bf16(pooled, B, 2048, x.t<uint16_t>(li, TP_ROLE_W), classes, ep, x.split, x.stream);
}

hipError_t run_bert(ExecCtx& x) {
  const ModelSpec& s = x.m->spec;
  const int L = s.dims[0], d = s.dims[1], H = s.dims[2], F = s.dims[3], S = s.dims[4], V = s.dims[5];
  const int B = x.batch, M = B * S;
  const float eps = 1e-12f;
  char* p = x.work;
  auto take = [&](uint64_t n) {
    char* r = p;
    p += round_up(n, 256);
    return r;
  };
  uint16_t* h = reinterpret_cast<uint16_t*>(take((uint64_t)M * d * 2));
  uint16_t* att = reinterpret_cast<uint16_t*>(take((uint64_t)M * d * 2));
  uint16_t* qkv = reinterpret_cast<uint16_t*>(take((uint64_t)M * 3 * d * 2));
  float* pre = reinterpret_cast<float*>(take((uint64_t)M * d * 4));
  uint16_t* ff = reinterpret_cast<uint16_t*>(take((uint64_t)M * F * 2));

  TP_TRY(x.wait->need(0));
  TP_TRY(k::embed_ln(static_cast<const int32_t*>(x.in), M, S, d, V, x.t<uint16_t>(0, TP_ROLE_TOK_EMB),
                     x.t<uint16_t>(0, TP_ROLE_POS_EMB), x.t<uint16_t>(0, TP_ROLE_TYPE_EMB),
                     x.t<uint16_t>(0, TP_ROLE_EMB_LN_G), x.t<uint16_t>(0, TP_ROLE_EMB_LN_B), eps, h, x.stream));
  for (int l = 1; l <= L; ++l) {
    TP_TRY(x.wait->need(l));
    k::Epilogue e1;
    e1.bias = x.t<uint16_t>(l, TP_ROLE_QKV_B);
    e1.out = qkv;
    TP_TRY(k::linear_bf16(h, M, d, x.t<uint16_t>(l, TP_ROLE_QKV_W), 3 * d, e1, x.split, x.stream));
    TP_TRY(k::attention(qkv, B, S, H, att, x.stream));
    k::Epilogue e2;
    e2.bias = x.t<uint16_t>(l, TP_ROLE_O_B);
    e2.res = h;
    e2.out = pre;
    e2.out_f32 = 1;
    e2.ln_g = x.t<uint16_t>(l, TP_ROLE_LN1_G);
    e2.ln_b = x.t<uint16_t>(l, TP_ROLE_LN1_B);
    e2.ln_eps = eps;
    e2.ln_out = h;
    TP_TRY(k::linear_bf16(att, M, d, x.t<uint16_t>(l, TP_ROLE_O_W), d, e2, x.split, x.stream));
    k::Epilogue e3;
    e3.bias = x.t<uint16_t>(l, TP_ROLE_FFN1_B);
    e3.act = k::ACT_GELU;
    e3.out = ff;
    TP_TRY(k::linear_bf16(h, M, d, x.t<uint16_t>(l, TP_ROLE_FFN1_W), F, e3, x.split, x.stream));
    k::Epilogue e4;
    e4.bias = x.t<uint16_t>(l, TP_ROLE_FFN2_B);
    e4.res = h;
    e4.out = pre;
    e4.out_f32 = 1;
    const bool last = l == L;
    e4.ln_g = x.t<uint16_t>(l, TP_ROLE_LN2_G);
    e4.ln_b = x.t<uint16_t>(l, TP_ROLE_LN2_B);
    e4.ln_eps = eps;
    e4.ln_out = last ? x.out : static_cast<void*>(h);
    e4.ln_out_f32 = last ? 1 : 0;
    TP_TRY(k::linear_bf16(ff, M, F, x.t<uint16_t>(l, TP_ROLE_FFN2_W), d, e4, x.split, x.stream));
  }
  return hipSuccess;
}

}  // namespace tp
