// Host optimizer step for the output layer's FP32 master weights (Layer-Adam).
//
// The paper updates each layer on the CPU while the GPU runs the next layer's backward (Section
// 3.1, "Asynchronous Parameter Updating"), with a CPU-Adam variant whose states live in host memory
// (Section 3.2, "Layer-Adam Optimizer"), from 16-bit gradients offloaded to a pinned buffer, and it
// converts the updated parameters to 16 bits in a shared pinned buffer before the next h2d copy
// (Section 3.2, "Optimized CPU Memory Layout with Shared Buffers"). This is that update: AdamW with
// bias correction, fp32 states, the 16-bit conversion fused into the same pass, split over threads
// in contiguous ranges and compiled for the host's widest vector unit (AVX-512, AVX2 or baseline
// x86-64, chosen at load time).
#include <immintrin.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "lce.h"

namespace {

inline float bf16_to_f32(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Round to nearest even; NaN stays a (quiet) NaN.
inline uint16_t f32_to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

inline float f16_to_f32(uint16_t b) {
  _Float16 h;
  std::memcpy(&h, &b, 2);
  return (float)h;
}

inline uint16_t f32_to_f16(float f) {
  const _Float16 h = (_Float16)f;
  uint16_t b;
  std::memcpy(&b, &h, 2);
  return b;
}

struct Coefs {
  float lr, b1, b2, eps, wd, c1, c2;  // c1 = 1 / (1 - b1^t), c2 = 1 / (1 - b2^t)
};

// DT: element type of the gradient and of the optional 16-bit parameter copy. Inlined into one
// multiversioned function per type below, so that each vector-width clone compiles its own copy.
template <int DT>
__attribute__((always_inline)) inline void adam_body(float* __restrict p, const void* __restrict gv,
                                                      float* __restrict m, float* __restrict v,
                                                      void* __restrict outv, int64_t i0, int64_t i1, Coefs c) {
  const uint16_t* g16 = (const uint16_t*)gv;
  const float* g32 = (const float*)gv;
  uint16_t* out = (uint16_t*)outv;
  for (int64_t i = i0; i < i1; ++i) {
    float g;
    if constexpr (DT == LCE_DTYPE_BF16) g = bf16_to_f32(g16[i]);
    else if constexpr (DT == LCE_DTYPE_FP16) g = f16_to_f32(g16[i]);
    else g = g32[i];
    const float mi = c.b1 * m[i] + (1.f - c.b1) * g;
    const float vi = c.b2 * v[i] + (1.f - c.b2) * g * g;
    m[i] = mi;
    v[i] = vi;
    const float pi = p[i];
    const float pn = pi - c.lr * ((mi * c.c1) / (std::sqrt(vi * c.c2) + c.eps) + c.wd * pi);
    p[i] = pn;
    if constexpr (DT == LCE_DTYPE_BF16) {
      if (out) out[i] = f32_to_bf16(pn);
    } else if constexpr (DT == LCE_DTYPE_FP16) {
      if (out) out[i] = f32_to_f16(pn);
    }
  }
}

__attribute__((target_clones("avx512f", "avx2", "default"))) void adam_bf16(
    float* p, const void* g, float* m, float* v, void* out, int64_t i0, int64_t i1, Coefs c) {
  adam_body<LCE_DTYPE_BF16>(p, g, m, v, out, i0, i1, c);
}
__attribute__((target_clones("avx512f", "avx2", "default"))) void adam_f16(
    float* p, const void* g, float* m, float* v, void* out, int64_t i0, int64_t i1, Coefs c) {
  adam_body<LCE_DTYPE_FP16>(p, g, m, v, out, i0, i1, c);
}
__attribute__((target_clones("avx512f", "avx2", "default"))) void adam_f32(
    float* p, const void* g, float* m, float* v, void* out, int64_t i0, int64_t i1, Coefs c) {
  adam_body<LCE_DTYPE_FP32>(p, g, m, v, out, i0, i1, c);
}

// bf16 gradients on AVX-512: 16 parameters per step, the same update and the same integer
// round-to-nearest-even (NaN kept quiet) as the generic body, with the four outputs written by
// streaming stores. The update is bound by host memory traffic, and an ordinary store first reads
// its cache line (parameter, moments and 16-bit copy: 14 of the 42 bytes a parameter would cost);
// none of these lines is read again before the next step. Needs p, m, v 64-byte aligned and out
// 32-byte aligned at i0, and i1 - i0 a multiple of 16; the caller checks.
__attribute__((target("avx512f,avx512bw"))) void adam_bf16_stream(float* __restrict p, const uint16_t* __restrict g,
                                                                  float* __restrict m, float* __restrict v,
                                                                  uint16_t* __restrict out, int64_t i0, int64_t i1,
                                                                  Coefs c) {
  const __m512 b1 = _mm512_set1_ps(c.b1), nb1 = _mm512_set1_ps(1.f - c.b1);
  const __m512 b2 = _mm512_set1_ps(c.b2), nb2 = _mm512_set1_ps(1.f - c.b2);
  const __m512 c1 = _mm512_set1_ps(c.c1), c2 = _mm512_set1_ps(c.c2), eps = _mm512_set1_ps(c.eps);
  const __m512 lr = _mm512_set1_ps(c.lr), wd = _mm512_set1_ps(c.wd);
  const __m512i one = _mm512_set1_epi32(1), bias = _mm512_set1_epi32(0x7fff);
  const __m512i absmask = _mm512_set1_epi32(0x7fffffff), inf = _mm512_set1_epi32(0x7f800000);
  const __m512i quiet = _mm512_set1_epi32(0x0040);
  for (int64_t i = i0; i < i1; i += 16) {
    const __m512 gv = _mm512_castsi512_ps(
        _mm512_slli_epi32(_mm512_cvtepu16_epi32(_mm256_loadu_si256((const __m256i*)(g + i))), 16));
    const __m512 mi = _mm512_add_ps(_mm512_mul_ps(b1, _mm512_load_ps(m + i)), _mm512_mul_ps(nb1, gv));
    const __m512 vi = _mm512_add_ps(_mm512_mul_ps(b2, _mm512_load_ps(v + i)), _mm512_mul_ps(_mm512_mul_ps(nb2, gv), gv));
    const __m512 pi = _mm512_load_ps(p + i);
    const __m512 den = _mm512_add_ps(_mm512_sqrt_ps(_mm512_mul_ps(vi, c2)), eps);
    const __m512 upd = _mm512_add_ps(_mm512_div_ps(_mm512_mul_ps(mi, c1), den), _mm512_mul_ps(wd, pi));
    const __m512 pn = _mm512_sub_ps(pi, _mm512_mul_ps(lr, upd));
    _mm512_stream_ps(m + i, mi);
    _mm512_stream_ps(v + i, vi);
    _mm512_stream_ps(p + i, pn);
    if (out) {
      const __m512i u = _mm512_castps_si512(pn);
      const __m512i lsb = _mm512_and_si512(_mm512_srli_epi32(u, 16), one);
      __m512i r = _mm512_srli_epi32(_mm512_add_epi32(_mm512_add_epi32(u, bias), lsb), 16);
      const __mmask16 nan = _mm512_cmpgt_epu32_mask(_mm512_and_si512(u, absmask), inf);
      r = _mm512_mask_mov_epi32(r, nan, _mm512_or_si512(_mm512_srli_epi32(u, 16), quiet));
      _mm256_stream_si256((__m256i*)(out + i), _mm512_cvtepi32_epi16(r));
    }
  }
  _mm_sfence();  // streaming stores are weakly ordered: visible before the range is reported done
}

bool has_avx512() {
  static const bool ok = __builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw");
  return ok;
}

template <int DT>
void adam_range(float* p, const void* g, float* m, float* v, void* out, int64_t i0, int64_t i1, Coefs c) {
  if constexpr (DT == LCE_DTYPE_BF16) {
    // The streaming body on the 16-aligned middle of the range, the generic one around it.
    int64_t a = i0;
    while (a < i1 && ((uintptr_t)(p + a) & 63)) ++a;
    const int64_t b = a + (i1 - a) / 16 * 16;
    const bool aligned = ((uintptr_t)(m + a) & 63) == 0 && ((uintptr_t)(v + a) & 63) == 0 &&
                         (!out || ((uintptr_t)((uint16_t*)out + a) & 31) == 0);
    if (has_avx512() && aligned && b > a) {
      adam_bf16(p, g, m, v, out, i0, a, c);
      adam_bf16_stream(p, (const uint16_t*)g, m, v, (uint16_t*)out, a, b, c);
      adam_bf16(p, g, m, v, out, b, i1, c);
    } else {
      adam_bf16(p, g, m, v, out, i0, i1, c);
    }
  } else if constexpr (DT == LCE_DTYPE_FP16) {
    adam_f16(p, g, m, v, out, i0, i1, c);
  } else {
    adam_f32(p, g, m, v, out, i0, i1, c);
  }
}

template <int DT>
void adam_threads(float* p, const void* g, float* m, float* v, void* out, int64_t n, Coefs c, int threads) {
  if (threads <= 1 || n < (int64_t)1 << 16) {
    adam_range<DT>(p, g, m, v, out, 0, n, c);
    return;
  }
  // Contiguous ranges, 64-element aligned, one per thread (the calling thread takes the first).
  const int64_t per = ((n + threads - 1) / threads + 63) / 64 * 64;
  std::vector<std::thread> pool;
  for (int k = 1; k < threads; ++k) {
    const int64_t a = k * per, b = std::min<int64_t>(n, a + per);
    if (a >= b) break;
    pool.emplace_back([=] { adam_range<DT>(p, g, m, v, out, a, b, c); });
  }
  adam_range<DT>(p, g, m, v, out, 0, std::min<int64_t>(n, per), c);
  for (auto& t : pool) t.join();
}

bool finite(float x) { return x == x && x > -3.0e38f && x < 3.0e38f; }

}  // namespace

extern "C" lce_status_t lce_host_adam_step(float* param, const void* grad, int dtype, float* exp_avg,
                                           float* exp_avg_sq, int64_t n, const lce_adam_config_t* cfg,
                                           int64_t step, void* param16, int n_threads) {
  if (!param || !grad || !exp_avg || !exp_avg_sq || !cfg || n < 0 || step < 1 || n_threads < 0)
    return LCE_ERR_INVALID_ARGUMENT;
  if (dtype != LCE_DTYPE_BF16 && dtype != LCE_DTYPE_FP16 && dtype != LCE_DTYPE_FP32) return LCE_ERR_INVALID_ARGUMENT;
  if (dtype == LCE_DTYPE_FP32 && param16) return LCE_ERR_INVALID_ARGUMENT;
  if (!finite(cfg->lr) || cfg->lr < 0.f || !(cfg->beta1 >= 0.f && cfg->beta1 < 1.f) ||
      !(cfg->beta2 >= 0.f && cfg->beta2 < 1.f) || !finite(cfg->eps) || cfg->eps <= 0.f ||
      !finite(cfg->weight_decay) || cfg->weight_decay < 0.f)
    return LCE_ERR_INVALID_ARGUMENT;
  Coefs c;
  c.lr = cfg->lr;
  c.b1 = cfg->beta1;
  c.b2 = cfg->beta2;
  c.eps = cfg->eps;
  c.wd = cfg->weight_decay;
  c.c1 = (float)(1.0 / (1.0 - std::pow((double)cfg->beta1, (double)step)));
  c.c2 = (float)(1.0 / (1.0 - std::pow((double)cfg->beta2, (double)step)));
  int threads = n_threads;
  if (threads == 0) threads = (int)std::max(1u, std::thread::hardware_concurrency());
  if (dtype == LCE_DTYPE_BF16) adam_threads<LCE_DTYPE_BF16>(param, grad, exp_avg, exp_avg_sq, param16, n, c, threads);
  else if (dtype == LCE_DTYPE_FP16) adam_threads<LCE_DTYPE_FP16>(param, grad, exp_avg, exp_avg_sq, param16, n, c, threads);
  else adam_threads<LCE_DTYPE_FP32>(param, grad, exp_avg, exp_avg_sq, nullptr, n, c, threads);
  return LCE_OK;
}
