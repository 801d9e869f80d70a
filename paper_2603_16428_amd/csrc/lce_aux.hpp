// Bandwidth-bound kernels around the three contractions of the fused linear + cross-entropy step.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "lce_gemm.hpp"

namespace lce {

__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(f16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(float v) { return v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }
template <> __device__ __forceinline__ f16 from_f32<f16>(float v) { return (f16)v; }
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }

// The call's first job (aux_kernel). Blocks 0 .. ceil(N/4) - 1: the target logit z_{i, y_i} =
// x_i . w_{y_i} in fp32, one wave per token; ignored tokens get 0, a label outside [0, V) gets NaN
// (so that the token's loss is NaN) and reads nothing; ref (optional) receives the reference of the
// target-referenced logits epilogue, z_{i, y_i} for a valid label and NaN otherwise. Block
// ceil(N/4): n_valid = the number of labels different from ignore_index over all N tokens (the
// mean's divisor is global, never per chunk; fixed-order tree), and clears the chunks' fallback
// flags (see combine_kernel).
// Blocks: ceil(N/4) + 1.
struct PrepareJob {
  const void* X;
  const void* W;
  const int64_t* y;
  int64_t N, H, V, ignore_index;
  float* tgt;
  float* ref;
  int* n_valid;
  int* flags;
  int64_t nflags;
};

template <typename T>
__device__ __forceinline__ void prepare_block(int64_t b, const PrepareJob& a) {
  const int64_t ntok = (a.N + 3) / 4;
  if (b == ntok) {
    __shared__ int part[256];
    for (int64_t k = threadIdx.x; k < a.nflags; k += 256) a.flags[k] = 0;
    int c = 0;
    for (int64_t i = threadIdx.x; i < a.N; i += 256) c += (a.y[i] != a.ignore_index);
    part[threadIdx.x] = c;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
      if ((int)threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
      __syncthreads();
    }
    if (threadIdx.x == 0) *a.n_valid = part[0];
    return;
  }
  const int64_t i = b * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= a.N) return;
  const int64_t lab = a.y[i];
  if (lab == a.ignore_index || lab < 0 || lab >= a.V) {
    if (lane == 0) {
      a.tgt[i] = lab == a.ignore_index ? 0.f : __builtin_nanf("");
      if (a.ref != nullptr) a.ref[i] = __builtin_nanf("");
    }
    return;
  }
  constexpr int kVec = 16 / sizeof(T);
  const T* xr = (const T*)a.X + i * a.H;
  const T* wr = (const T*)a.W + lab * a.H;
  float s = 0.f;
  for (int64_t h = (int64_t)lane * kVec; h < a.H; h += 64 * kVec) {
#pragma unroll
    for (int e = 0; e < kVec; ++e) s = fmaf(to_f32(xr[h + e]), to_f32(wr[h + e]), s);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) {
    a.tgt[i] = s;
    if (a.ref != nullptr) a.ref[i] = s;
  }
}

// Sum of the token losses tl[0 .. N) by one block of 256 threads: in fp64, in a fixed order (1024
// strided partial sums, then a tree over them), divided by n_valid for the mean (0 when no token
// is valid).
__device__ __forceinline__ void loss_sum_block(const float* __restrict__ tl, int64_t N, const int* __restrict__ n_valid,
                                               int mean, float* __restrict__ loss) {
  __shared__ double part[1024];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int v = threadIdx.x + 256 * u;
    double s = 0.0;
    for (int64_t i = v; i < N; i += 1024) s += (double)tl[i];
    part[v] = s;
  }
  __syncthreads();
  for (int k = 512; k > 0; k >>= 1) {
    for (int v = threadIdx.x; v < k; v += 256) part[v] += part[v + k];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    double r = part[0];
    if (mean) {
      const int nv = *n_valid;
      r = nv > 0 ? r / (double)nv : 0.0;
    }
    *loss = (float)r;
  }
}

// Row combine. For each token of the chunk: M = max_t m_t, lse = M + log sum_t s_t exp(m_t - M),
// and the token loss lse - z_target (0 for ignored tokens). A block takes 16 tokens x 16 slice
// groups: thread (token j, group k) merges slices k, k + 16, ... in increasing order (a 64-byte
// coalesced row of partials per slice), then group 0 merges the 16 groups in a fixed order.
//
// Backward, the per-token factor that the dH epilogue and the dW operand apply (scale_out):
//   CMB_TREF  : e holds exp(z - z_target) for valid tokens (label in [0, V), not ignored), and the
//               partials were taken relative to z_target, so S = sum_v exp(z_v - z_target) =
//               exp(lse - z_target) is the merged sum. dZ = g (p - onehot) = (g / S) (e - S onehot):
//               the factor is g / S (0 for other tokens) and the label's entry of e becomes e - S.
//               A token whose S exceeds kTrefMaxSum (loss above 60) or is not at least kTrefMinSum
//               (NaN included: inputs that are not finite) sets *flag: its e may have overflowed,
//               so the chunk is redone with slice-maximum references. The lower bound is loose on
//               purpose: the target's own term is exp(z_y - z_target) = 1 only up to the difference
//               between the GEMM's and the fp32 dot's rounding of z_y, so a confident token
//               (p_y close to 1) has S slightly below 1 as often as above it.
//   CMB_SLICE : dlogits forms dZ with g inside; the factor is 1.
// run_if: do nothing unless *run_if != 0 (nullptr: always run).
enum CombineMode { CMB_FORWARD = 0, CMB_TREF = 1, CMB_SLICE = 2 };
constexpr float kTrefMaxSum = 1.1420073898e26f;  // exp(60)
constexpr float kTrefMinSum = 0.5f;
constexpr int kCombineTokens = 16;
template <typename T>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ pmax, const float* __restrict__ psum,
                                                      int64_t ldp, int slices, int rows,
                                                      const int64_t* __restrict__ y, int64_t ignore_index,
                                                      const float* __restrict__ tgt,
                                                      float* __restrict__ lse_out,     // [rows] (chunk-offset)
                                                      float* __restrict__ loss_out,    // [rows] (chunk-offset)
                                                      int mode, float* __restrict__ scale_out,
                                                      const int* __restrict__ n_valid, int mean, T* __restrict__ ez,
                                                      int64_t KP, int64_t V, int* __restrict__ flag,
                                                      const int* __restrict__ run_if) {
  if (run_if != nullptr && *run_if == 0) return;
  __shared__ float sm[16][kCombineTokens], ss[16][kCombineTokens];
  const int t = threadIdx.x % kCombineTokens, grp = threadIdx.x / kCombineTokens;
  const int i = blockIdx.x * kCombineTokens + t;
  float m = -INFINITY, s = 0.f;
  // Target-referenced partials all share one reference per token (its target logit, or 0 for a
  // token without one), so the maxima are not read: the merge below runs with 0 in their place,
  // where every factor exp(m - mn) is exactly 1 as it would be with the reference itself, and the
  // reference is added back to the merged maximum.
  const bool shared_ref = mode == CMB_TREF;
  if (i < rows) {
    // Eight slices' partials are requested before any is merged (the merge order is unchanged).
    constexpr int kAhead = 8;
    for (int k0 = grp; k0 < slices; k0 += 16 * kAhead) {
      float mk[kAhead], sk[kAhead];
#pragma unroll
      for (int u = 0; u < kAhead; ++u) {
        const int k = min(k0 + 16 * u, slices - 1);
        mk[u] = shared_ref ? 0.f : pmax[(size_t)k * ldp + i];
        sk[u] = psum[(size_t)k * ldp + i];
      }
#pragma unroll
      for (int u = 0; u < kAhead; ++u) {
        if (k0 + 16 * u >= slices) break;
        const float mn = fmaxf(m, mk[u]);
        s = s * __expf(m - mn) + sk[u] * __expf(mk[u] - mn);
        m = mn;
      }
    }
  }
  sm[grp][t] = m;
  ss[grp][t] = s;
  __syncthreads();
  if (grp == 0 && i < rows) {
    float M = sm[0][t];
    for (int k = 1; k < 16; ++k) M = fmaxf(M, sm[k][t]);
    float S = 0.f;
    for (int k = 0; k < 16; ++k) S += ss[k][t] * __expf(sm[k][t] - M);
    const int64_t lab = y[i];
    if (shared_ref) {
      // The logits epilogue's reference: the target logit of a valid token when finite, else 0.
      const float r = tgt[i];
      M = (lab != ignore_index && lab >= 0 && lab < V && __builtin_isfinite(r)) ? r : 0.f;
    }
    const float lse = M + __logf(S);
    lse_out[i] = lse;
    loss_out[i] = (lab == ignore_index) ? 0.f : lse - tgt[i];
    if (mode == CMB_TREF) {
      float sc = 0.f;
      if (lab != ignore_index && lab >= 0 && lab < V) {
        const float sum = S * __expf(M - tgt[i]);  // every m_t is tgt[i] here, so this is S
        if (sum >= kTrefMinSum && sum <= kTrefMaxSum) {  // (NaN fails both)
          const int nv = *n_valid;
          const float g = mean ? (nv > 0 ? 1.f / (float)nv : 0.f) : 1.f;
          sc = g / sum;
          // Element (token i, id lab) of the blocked layout.
          const int64_t byte = lab * (int64_t)sizeof(T);
          const int ln = (i & 31) + 32 * (int)((byte >> 4) & 1);
          T* p = (T*)((char*)ez + ((size_t)(i >> 5) * KP + (size_t)(byte >> 5)) * 1024 + ln * 16 + (byte & 15));
          *p = from_f32<T>(to_f32(*p) - sum);
        } else {
          *flag = 1;
        }
      }
      scale_out[i] = sc;
    } else if (mode == CMB_SLICE) {
      scale_out[i] = 1.f;
    }
  }
}

// dlogits, in place, on e's blocked layout: fragment (jb, q), 1 KB at byte (jb KP + q) 1024, holds
// tokens 32 jb .. 32 jb + 31 by the q-th 32 bytes of the vocabulary; lane l's 16 bytes are token
// 32 jb + l%32, ids from (32 q + 16 (l/32)) / sizeof(T). For token i of the chunk and id v
// (slice t = v / 128):
//   dZ[i][v] = g_i exp(m_t,i - lse_i) e[i][v] - g_i [v == y_i],   g_i = valid_i / n_valid (mean) or valid_i,
// where e = exp(z - m_t,i) was stored by the logits GEMM. Every piece of the buffer is written:
// tokens at or beyond `rows` and ids at or beyond V as zeros (the dW GEMM sums over the last token
// block, the dH GEMM reads the id padding). Block (b, jb) covers K-pairs 16 b .. 16 b + 15 of token
// block jb (KP is a multiple of 16); wave w takes K-pairs 16 b + 4 w .. + 3, which lie in one
// slice, so each lane has one token and one scale. For fp16 both e and dZ carry the storage
// scales of Storage<f16> (dZ = (p - onehot) kDz for valid tokens; g is applied later).
template <typename T>
__device__ __forceinline__ void dlogits_block(T* __restrict__ ez, int64_t KP, int64_t bx, int jb,
                                              const float* __restrict__ pmax, int64_t ldp,
                                              const float* __restrict__ lse, const int64_t* __restrict__ y,
                                              int64_t ignore_index, const int* __restrict__ n_valid, int mean,
                                              int rows, int V) {
  constexpr int kVec = 16 / sizeof(T);          // ids per piece
  const int l = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t q0 = 16 * bx + 4 * w;
  char* piece = (char*)ez + ((size_t)jb * KP + q0) * 1024 + l * 16;
  // All four pieces are read before any is written: HBM needs the loads in flight together. Tokens
  // at or beyond `rows` read stale data that the select below discards.
  uint4 raw[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) raw[k] = *(const uint4*)(piece + k * 1024);
  const int i = 32 * jb + (l & 31);
  const int ic = min(i, rows - 1);
  const int64_t lab = y[ic];
  const bool active = i < rows && lab != ignore_index;
  const int v0 = (int)((q0 * 32 + 16 * (l >> 5)) / (int)sizeof(T));
  const int slice = min(v0, V - 1) / kLseSlice;
  const int nv = *n_valid;
  const float g = Storage<T>::kDzUnscaled ? Storage<T>::kDz : (mean ? (nv > 0 ? 1.f / (float)nv : 0.f) : 1.f);
  constexpr float kInvE = 1.f / Storage<T>::kE;
  const float c = g * kInvE * __expf(pmax[(size_t)slice * ldp + i] - lse[ic]);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int v = v0 + k * (32 / (int)sizeof(T));
    T ev[kVec], outv[kVec];
    *(uint4*)ev = raw[k];
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
      float d = (active && v + e < V) ? c * to_f32(ev[e]) : 0.f;
      if (active && v + e == lab) d -= g;
      outv[e] = from_f32<T>(d);
    }
    *(uint4*)(piece + k * 1024) = *(const uint4*)outv;
  }
}

// The job's `blocks` blocks walk the (b, jb) pairs b fastest (as many blocks as pairs take one
// each); run_if: do nothing unless *run_if != 0 (nullptr: always run).
struct DlogitsJob {
  void* ez;
  int64_t KP, NB;
  const float* pmax;
  int64_t ldp;
  const float* lse;
  const int64_t* y;
  int64_t ignore_index;
  const int* n_valid;
  int mean, rows, V;
  const int* run_if;
};

template <typename T>
__device__ __forceinline__ void dlogits_job(int64_t b, int64_t blocks, const DlogitsJob& a) {
  if (a.run_if != nullptr && *a.run_if == 0) return;
  const int64_t nbx = a.KP / 16;
  for (int64_t idx = b; idx < nbx * a.NB; idx += blocks)
    dlogits_block<T>((T*)a.ez, a.KP, idx % nbx, (int)(idx / nbx), a.pmax, a.ldp, a.lse, a.y, a.ignore_index,
                     a.n_valid, a.mean, a.rows, a.V);
}

// out[i][h] = sum_s part[s][i][h] (fixed order), times the dz storage scale's inverse of the
// operand type TS (1 unless dz is stored unscaled), converted to the output type T.
template <typename T, typename TS = T>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int splits,
                                                           int64_t count, T* __restrict__ out,
                                                           const int* __restrict__ n_valid, int mean) {
  const int64_t idx = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (idx >= count) return;
  float4 s = *(const float4*)(part + idx);
  for (int k = 1; k < splits; ++k) {
    const float4 v = *(const float4*)(part + (size_t)k * count + idx);
    s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
  }
  if constexpr (Storage<TS>::kDzUnscaled) {
    const float sc = dz_epilogue_scale<TS>(n_valid, mean);
    s.x *= sc; s.y *= sc; s.z *= sc; s.w *= sc;
  }
  out[idx] = from_f32<T>(s.x);
  out[idx + 1] = from_f32<T>(s.y);
  out[idx + 2] = from_f32<T>(s.z);
  out[idx + 3] = from_f32<T>(s.w);
}

// One launch for several independent bandwidth-bound jobs, each on its own consecutive range of
// blocks of 256 threads (a job with 0 blocks is absent), in this order: prepare_block,
// block_k_block, block_mn_block, dlogits_job, loss_sum_block (one block). Jobs in one launch touch
// disjoint buffers; what orders them against the other kernels is the stream order of the
// launches (the loss sum goes into a launch after the call's last combine_kernel).
struct BlockKJob {
  const void* src;
  int64_t ld;
  int N, K, KP, NB;
  void* dst;
};
struct BlockMnJob {
  const void* src;
  int64_t ld;
  int N, K, KP, NB;  // NB column blocks by ceil(KP / 4) K-pair groups, column block fastest
  void* dst;
  const float* row_scale;
};
struct LossJob {
  const float* tl;
  int64_t N;
  const int* n_valid;
  int mean;
  float* loss;
};
struct AuxJobs {
  int64_t prep_blocks, bk_blocks, bmn_blocks, dl_blocks, loss_blocks;
  PrepareJob prep;
  BlockKJob bk;
  BlockMnJob bmn;
  DlogitsJob dl;
  LossJob ls;
};

template <typename T>
__global__ __launch_bounds__(256) void aux_kernel(const AuxJobs j) {
  int64_t b = blockIdx.x;
  if (b < j.prep_blocks) {
    prepare_block<T>(b, j.prep);
    return;
  }
  b -= j.prep_blocks;
  if (b < j.bk_blocks) {
    block_k_block<T>(b, (const T*)j.bk.src, j.bk.ld, j.bk.N, j.bk.K, j.bk.KP, j.bk.NB, (T*)j.bk.dst);
    return;
  }
  b -= j.bk_blocks;
  if (b < j.bmn_blocks) {
    block_mn_block<T>((int)(b % j.bmn.NB), (int)(b / j.bmn.NB), (const T*)j.bmn.src, j.bmn.ld, j.bmn.N, j.bmn.K,
                      j.bmn.KP, (T*)j.bmn.dst, j.bmn.row_scale);
    return;
  }
  b -= j.bmn_blocks;
  if (b < j.dl_blocks) {
    dlogits_job<T>(b, j.dl_blocks, j.dl);
    return;
  }
  b -= j.dl_blocks;
  if (b < j.loss_blocks) loss_sum_block(j.ls.tl, j.ls.N, j.ls.n_valid, j.ls.mean, j.ls.loss);
}

}  // namespace lce

namespace lce {

// ---- final RMSNorm around the step (x_i = gamma . h_i r_i, r_i = 1 / sqrt(mean_j h_ij^2 + eps)) ----

// One wave per token: r_i, and the normalised row x_i in the input dtype (fp32 arithmetic).
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_rows_kernel(const T* __restrict__ h, const T* __restrict__ gamma,
                                                           int64_t N, int64_t H, float eps, T* __restrict__ x,
                                                           float* __restrict__ r_out) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  constexpr int kVec = 16 / sizeof(T);
  const T* hr = h + i * H;
  float ss = 0.f;
  for (int64_t j = (int64_t)lane * kVec; j < H; j += 64 * kVec) {
    T v[kVec];
    *(uint4*)v = *(const uint4*)(hr + j);
#pragma unroll
    for (int e = 0; e < kVec; ++e) ss = fmaf(to_f32(v[e]), to_f32(v[e]), ss);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const float r = 1.f / sqrtf(ss / (float)H + eps);
  T* xr = x + i * H;
  for (int64_t j = (int64_t)lane * kVec; j < H; j += 64 * kVec) {
    T v[kVec], gv[kVec], o[kVec];
    *(uint4*)v = *(const uint4*)(hr + j);
    *(uint4*)gv = *(const uint4*)(gamma + j);
#pragma unroll
    for (int e = 0; e < kVec; ++e) o[e] = from_f32<T>(to_f32(gv[e]) * (to_f32(v[e]) * r));
    *(uint4*)(xr + j) = *(const uint4*)o;
  }
  if (lane == 0) r_out[i] = r;
}

// One wave per token: s_i = sum_k h_ik gamma_k dX_ik (fp32, fixed order; dX in fp32).
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_rowdot_kernel(const T* __restrict__ h, const T* __restrict__ gamma,
                                                             const float* __restrict__ dx, int64_t N, int64_t H,
                                                             float* __restrict__ s_out) {
  const int64_t i = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (i >= N) return;
  constexpr int kVec = 16 / sizeof(T);
  float s = 0.f;
  for (int64_t j = (int64_t)lane * kVec; j < H; j += 64 * kVec) {
    T hv[kVec], gv[kVec];
    *(uint4*)hv = *(const uint4*)(h + i * H + j);
    *(uint4*)gv = *(const uint4*)(gamma + j);
#pragma unroll
    for (int e = 0; e < kVec; ++e) s = fmaf(to_f32(hv[e]) * to_f32(gv[e]), dx[i * H + j + e], s);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  if (lane == 0) s_out[i] = s;
}

// The Jacobian, from the fp32 dX rows into the gradient rows, kRmsRows tokens x 256 features per block:
//   dh_ij = r_i gamma_j dX_ij - r_i^3 h_ij s_i / H,   and the block's share of
//   dgamma_j = sum_i dX_ij h_ij r_i, written to part[blockIdx.y][j] (summed in a fixed order later).
constexpr int kRmsRows = 64;
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_backward_kernel(const T* __restrict__ h, const T* __restrict__ gamma,
                                                               const float* __restrict__ r, const float* __restrict__ s,
                                                               const float* __restrict__ dx, T* __restrict__ g,
                                                               int64_t N, int64_t H, float* __restrict__ part) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t i0 = (int64_t)blockIdx.y * kRmsRows;
  if (j >= H) return;
  const float gj = to_f32(gamma[j]);
  const float invH = 1.f / (float)H;
  float dg = 0.f;
  const int64_t i1 = i0 + kRmsRows < N ? i0 + kRmsRows : N;
  for (int64_t i = i0; i < i1; ++i) {
    const float ri = r[i];
    const float hij = to_f32(h[i * H + j]);
    const float dxij = dx[i * H + j];
    dg = fmaf(dxij * hij, ri, dg);
    g[i * H + j] = from_f32<T>(ri * gj * dxij - ri * ri * ri * hij * s[i] * invH);
  }
  part[(size_t)blockIdx.y * H + j] = dg;
}

// dgamma_j = sum over row blocks of part[b][j], in block order.
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_gamma_reduce_kernel(const float* __restrict__ part, int blocks,
                                                                   int64_t H, T* __restrict__ dgamma) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j >= H) return;
  float acc = 0.f;
  for (int b = 0; b < blocks; ++b) acc += part[(size_t)b * H + j];
  dgamma[j] = from_f32<T>(acc);
}

}  // namespace lce
