// MFMA GEMM core for the three contractions of the fused linear + cross-entropy step.
//
//   C[m, n] = sum_k A[m, k] * B[n, k]      A: [M, K] pitch lda, B: [N, K] pitch ldb (K contiguous)
//
// One workgroup computes a 256 x 256 tile of C with four waves (2 x 2), each wave a 128 x 128
// sub-tile held as 4 x 4 blocks of the 32x32 MFMA accumulator (256 fp32 per lane). K advances in
// tiles of 128 bytes per row (64 bf16 or 32 fp32). Both operand tiles are streamed from global
// memory straight into LDS with buffer_load ... lds (16 bytes per lane), double buffered, and the
// buffer descriptors' range check turns rows beyond M/N into zeros. LDS rows are XOR-swizzled in
// 16-byte units so that the MFMA fragment reads (ds_read_b128) are free of bank conflicts.
//
// The epilogue decides what the tile becomes:
//   LSE_FWD / LSE_BWD : C = logits^T tile (rows = vocabulary, columns = tokens). Per token and per
//                       128-row vocabulary slice: the maximum m and sum exp(z - m) (the vocabulary-
//                       tiled online log-sum-exp); LSE_BWD also stores e = exp(z - m) token-major.
//   STORE             : C written as the output dtype (or as fp32 split-K partials).
//   DW                : C added into the fp32 dW accumulator (first / middle / last chunk).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lce {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTile = 256;                       // BM = BN
constexpr int kRowBytes = 128;                   // bytes of K per row per K-tile
constexpr int kOperandBytes = kTile * kRowBytes; // 32 KB
constexpr int kStageBytes = 2 * kOperandBytes;   // A + B
constexpr int kGemmSmem = 2 * kStageBytes;       // two stages: 128 KB
constexpr int kGemmThreads = 256;
constexpr int kLseSlice = 128;                   // vocabulary rows per log-sum-exp partial
constexpr uint32_t kOOB = 0x80000000u;           // a buffer offset beyond every range check
constexpr float kLog2e = 1.4426950408889634f;

enum Epilogue { EPI_LSE_FWD = 0, EPI_LSE_BWD = 1, EPI_STORE = 2, EPI_DW = 3 };
enum DwMode { DW_FIRST = 0, DW_MID = 1, DW_LAST = 2, DW_ONLY = 3 };

struct GemmArgs {
  const void* A;
  const void* B;
  int64_t lda, ldb;   // pitches in elements
  int M, N, K;        // K: elements, a multiple of 16 bytes' worth
  int tiles_m, tiles_n, splits, k_per_split;  // k_per_split: a multiple of the K-tile
  int group_m;        // tile rows per raster group
  // epilogue
  void* out;          // LSE_BWD: e (token-major, pitch ldo); STORE: output or fp32 partials; DW: dW
  int64_t ldo;
  float* acc;         // DW: fp32 accumulator [M, ldacc]
  int64_t ldacc;
  float* pmax;        // LSE: [slices, ldp]
  float* psum;
  int64_t ldp;
  int mode;           // DW: DwMode; STORE: 1 = fp32 split-K partials at out + split * M * ldo
};

__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// Tile coordinates of linear block `bid`. The dispatcher places block b on XCD b % 8, so blocks
// are first renumbered to make each XCD's share a contiguous range, then rastered in groups of
// group_m tile rows (columns advance every group_m blocks), so that the blocks resident on one XCD
// share A and B slices in that XCD's L2.
__device__ __forceinline__ void tile_coords(int bid, int total, int tiles_m, int group_m,
                                            int& tm, int& rest) {
  const int per = total >> 3, rem = total & 7;
  const int x = bid & 7, q = bid >> 3;
  const int b2 = x * per + (x < rem ? x : rem) + q;
  const int width = group_m * (total / tiles_m);  // total = tiles_m * tiles_n * splits
  const int grp = b2 / width;
  const int first = grp * group_m;
  const int gm = min(group_m, tiles_m - first);
  const int in = b2 - grp * width;
  tm = first + in % gm;
  rest = in / gm;
}

template <typename T>
__device__ __forceinline__ void mfma_pair(f32x16& c, const f32x4& a, const f32x4& b);

template <>
__device__ __forceinline__ void mfma_pair<bf16>(f32x16& c, const f32x4& a, const f32x4& b) {
  // 16 bf16 of K per lane pair (lanes l and l+32 hold the two halves of K).
  c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                              __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

template <>
__device__ __forceinline__ void mfma_pair<float>(f32x16& c, const f32x4& a, const f32x4& b) {
  // 8 fp32 of K: each 32x32x2 step takes element s of both lanes' 4-vectors.
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], c, 0, 0, 0);
  c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], c, 0, 0, 0);
}

__device__ __forceinline__ void store_out(bf16* p, float v) { *p = (bf16)v; }
__device__ __forceinline__ void store_out(float* p, float v) { *p = v; }

template <typename T, int EPI>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_kernel(const GemmArgs g) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kChunk = 16 / kEsz;        // elements per 16-byte chunk
  constexpr int kBK = kRowBytes / kEsz;    // elements per K-tile

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;

  const int total = g.tiles_m * g.tiles_n * g.splits;
  int tm, rest;
  tile_coords(blockIdx.x, total, g.tiles_m, g.group_m, tm, rest);
  const int tn = rest % g.tiles_n;
  const int split = rest / g.tiles_n;
  const int m0 = tm * kTile, n0 = tn * kTile;
  const int kb = split * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);

  const int rows_a = min(kTile, g.M - m0), rows_b = min(kTile, g.N - n0);
  const __amdgpu_buffer_rsrc_t ra =
      make_rsrc((const char*)g.A + (size_t)m0 * g.lda * kEsz, (uint32_t)rows_a * (uint32_t)g.lda * kEsz);
  const __amdgpu_buffer_rsrc_t rb =
      make_rsrc((const char*)g.B + (size_t)n0 * g.ldb * kEsz, (uint32_t)rows_b * (uint32_t)g.ldb * kEsz);

  // Loader: wave w fills LDS bytes [(8w + j) * 1 KB, +1 KB) of each operand tile with instruction
  // j; lane l lands in row 8(8w + j) + l/8, 16-byte slot l%8, and so fetches logical chunk
  // (l%8) ^ swz(row) of that row.
  uint32_t off_a[8], off_b[8];
  int kc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int r = (w * 8 + j) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ swz(r);
    kc[j] = c * kChunk;
    off_a[j] = (uint32_t)r * (uint32_t)g.lda * kEsz + (uint32_t)(c * 16);
    off_b[j] = (uint32_t)r * (uint32_t)g.ldb * kEsz + (uint32_t)(c * 16);
  }

  auto issue = [&](int k0, int stage) {
    char* sa = smem + stage * kStageBytes + w * 8 * 1024;
    char* sb = sa + kOperandBytes;
    const bool tail = k0 + kBK > ke;
    const uint32_t koff = (uint32_t)k0 * kEsz;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t oa = off_a[j] + koff, ob = off_b[j] + koff;
      if (tail && k0 + kc[j] >= ke) { oa = kOOB; ob = kOOB; }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(sa + j * 1024), 16, oa, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void*)(sb + j * 1024), 16, ob, 0, 0, 0);
    }
  };

  // Fragment reads: block mb covers rows wm*128 + 32mb + (l%32); K-pair p reads logical chunk
  // 2p + l/32 (lanes l and l+32 carry the two 16-byte halves of 32 bytes of K).
  int frag_a[4], frag_b[4], swz_a[4], swz_b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int ra_row = wm * 128 + i * 32 + (lane & 31);
    const int rb_row = wn * 128 + i * 32 + (lane & 31);
    frag_a[i] = ra_row * kRowBytes;
    frag_b[i] = kOperandBytes + rb_row * kRowBytes;
    swz_a[i] = swz(ra_row);
    swz_b[i] = swz(rb_row);
  }
  const int khalf = lane >> 5;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x16){};

  const int nk = (ke - kb + kBK - 1) / kBK;
  if (nk > 0) {
    issue(kb, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) issue(kb + (kt + 1) * kBK, cur ^ 1);
    const char* st = smem + cur * kStageBytes;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      f32x4 fa[4], fb[4];
      const int c = 2 * p + khalf;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        fa[i] = *(const f32x4*)(st + frag_a[i] + ((c ^ swz_a[i]) << 4));
        fb[i] = *(const f32x4*)(st + frag_b[i] + ((c ^ swz_b[i]) << 4));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) mfma_pair<T>(acc[i][j], fa[i], fb[j]);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // ---- epilogue. Accumulator element r of block (i, j) sits at
  //      row = 32i + 8(r/4) + 4(l/32) + r%4, col = 32j + l%32 of the wave's 128 x 128 sub-tile.
  const int mw = m0 + wm * 128, nw = n0 + wn * 128;
  const int rsub = 4 * (lane >> 5);
  const int csub = lane & 31;

  if constexpr (EPI == EPI_LSE_FWD || EPI == EPI_LSE_BWD) {
    if (mw >= g.M) return;
    const int slice = mw / kLseSlice;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = nw + 32 * j + csub;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = mw + 32 * i + 8 * (r >> 2) + rsub + (r & 3);
          if (row < g.M) mx = fmaxf(mx, acc[i][j][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float ml = mx * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = mw + 32 * i + 8 * (r >> 2) + rsub + (r & 3);
          const float e = row < g.M ? __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, -ml)) : 0.f;
          s += e;
          acc[i][j][r] = e;
        }
      s += __shfl_xor(s, 32);
      if (col < g.N) {
        if constexpr (EPI == EPI_LSE_BWD) {
          T* e_row = (T*)g.out + (size_t)col * g.ldo;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int row = mw + 32 * i + 8 * q + rsub;
              if (row < g.M) {
                if constexpr (sizeof(T) == 2) {
                  bf16x4 v = {(bf16)acc[i][j][4 * q], (bf16)acc[i][j][4 * q + 1],
                              (bf16)acc[i][j][4 * q + 2], (bf16)acc[i][j][4 * q + 3]};
                  *(bf16x4*)(e_row + row) = v;
                } else {
                  f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                             acc[i][j][4 * q + 3]};
                  *(f32x4*)(e_row + row) = v;
                }
              }
            }
        }
        if (lane < 32) {
          g.pmax[(size_t)slice * g.ldp + col] = mx;
          g.psum[(size_t)slice * g.ldp + col] = s;
        }
      }
    }
  } else if constexpr (EPI == EPI_STORE) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = mw + 32 * i + 8 * (r >> 2) + rsub + (r & 3);
        if (row >= g.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = nw + 32 * j + csub;
          if (col >= g.N) continue;
          if (g.mode == 1) {
            float* o = (float*)g.out + (size_t)split * g.M * g.ldo;
            o[(size_t)row * g.ldo + col] = acc[i][j][r];
          } else {
            store_out((T*)g.out + (size_t)row * g.ldo + col, acc[i][j][r]);
          }
        }
      }
  } else {  // EPI_DW
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = mw + 32 * i + 8 * (r >> 2) + rsub + (r & 3);
        if (row >= g.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int col = nw + 32 * j + csub;
          if (col >= g.N) continue;
          float* a = g.acc + (size_t)row * g.ldacc + col;
          const float v = acc[i][j][r];
          switch (g.mode) {
            case DW_FIRST: *a = v; break;
            case DW_MID: *a += v; break;
            case DW_LAST: store_out((T*)g.out + (size_t)row * g.ldo + col, *a + v); break;
            default: store_out((T*)g.out + (size_t)row * g.ldo + col, v); break;
          }
        }
      }
  }
}

}  // namespace lce
