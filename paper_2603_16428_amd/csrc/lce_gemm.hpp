// MFMA GEMM core for the three contractions of the fused linear + cross-entropy step.
//
//   C[m, n] = sum_k A[m, k] * B[n, k]      A: [M, K] pitch lda, B: [N, K] pitch ldb (K contiguous)
//
// One workgroup computes a 256 x 256 tile of C with four waves (2 x 2), each wave a 128 x 128
// sub-tile held as 4 x 4 blocks of the 32x32 MFMA accumulator (256 fp32 per lane, in AGPRs). K
// advances in tiles of one 128-byte cache line per row (64 bf16 or 32 fp32); eight lanes load one
// line (16 bytes each). Every K-tile is requested about two K-tiles ahead of its MFMAs: a single
// K-tile in flight per CU leaves the MFMAs waiting on this access pattern's load latency, and three
// LDS stages of both operands (192 KB) do not fit. So operand A streams straight into a ring of
// three LDS slots (buffer_load ... lds) while operand B is parked in one of two register buffers
// (buffer_load_dwordx4) and written (ds_write_b128) into one of two LDS slots during the preceding
// K-tile: 160 KB of LDS and 64 VGPRs. The buffer descriptors' range check turns rows beyond M/N,
// and K-tiles past the end, into zeros. LDS rows are XOR-swizzled in
// 16-byte units so that the fragment reads (ds_read_b128) are free of bank conflicts. Fragments
// are double-buffered in registers: the reads for the next 32 bytes of K are in flight while the
// MFMAs of the current ones run.
//
// The epilogue decides what the tile becomes:
//   LSE_FWD / LSE_BWD : C = logits^T tile (rows = vocabulary, columns = tokens). Per token and per
//                       128-row vocabulary slice: the maximum m and sum exp(z - m) (the vocabulary-
//                       tiled online log-sum-exp); LSE_BWD also stores e = exp(z - m) token-major.
//   STORE             : C written as the output dtype (or as fp32 split-K partials).
//   DW                : C added into the fp32 dW accumulator (first / middle / last chunk).
// STORE and DW issue the MFMAs with the operands swapped, so each lane holds four consecutive
// columns of C and writes them as one vector.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace lce {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kTile = 256;                       // BM = BN
constexpr int kRowBytes = 128;                   // bytes of K per row per K-tile (one cache line)
constexpr int kSlots = kRowBytes / 16;           // 16-byte chunks per row
constexpr int kPairs = kSlots / 2;               // 32-byte K-pairs (one MFMA step) per K-tile
constexpr int kOperandBytes = kTile * kRowBytes; // 32 KB: one operand's K-tile
constexpr int kASlots = 3;                       // A: ring of K-tiles filled by LDS-DMA
constexpr int kBSlots = 2;                       // B: LDS slots filled from registers
constexpr int kBBase = kASlots * kOperandBytes;  // B slots follow the A ring
constexpr int kGemmSmem = (kASlots + kBSlots) * kOperandBytes;  // 160 KB, all of a CU's LDS
constexpr int kLoadsPerOperand = kSlots;         // 16-byte loads per lane per operand K-tile
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

// 16-byte slot of logical chunk c (0..7) of LDS row r is c ^ swz(r): conflict-free fragment reads
// whether the LDS serves 8 or 16 lanes' 16-byte reads per cycle.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ const void* uniform_ptr(const void* p) {
  const uint64_t v = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (const void*)(((uint64_t)hi << 32) | lo);
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
  // 16 bf16 of K per lane pair (lanes l and l+32 hold the two halves of 32 bytes of K).
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

__device__ __forceinline__ void store4(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *(bf16x4*)p = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *(f32x4*)p = v;
}

template <typename T, int EPI>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_kernel(const GemmArgs g) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kChunk = 16 / kEsz;        // elements per 16-byte chunk
  constexpr int kBK = kRowBytes / kEsz;    // elements per K-tile
  constexpr bool kSwap = (EPI == EPI_STORE || EPI == EPI_DW);

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;

  const int total = g.tiles_m * g.tiles_n * g.splits;
  int tm, rest;
  tile_coords(blockIdx.x, total, g.tiles_m, g.group_m, tm, rest);
  tm = __builtin_amdgcn_readfirstlane(tm);
  rest = __builtin_amdgcn_readfirstlane(rest);
  const int tn = rest % g.tiles_n;
  const int split = rest / g.tiles_n;
  const int m0 = tm * kTile, n0 = tn * kTile;
  const int kb = split * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);

  const int rows_a = min(kTile, g.M - m0), rows_b = min(kTile, g.N - n0);
  const __amdgpu_buffer_rsrc_t ra =
      make_rsrc(uniform_ptr((const char*)g.A + (size_t)m0 * g.lda * kEsz),
                __builtin_amdgcn_readfirstlane((uint32_t)rows_a * (uint32_t)g.lda * kEsz));
  const __amdgpu_buffer_rsrc_t rb =
      make_rsrc(uniform_ptr((const char*)g.B + (size_t)n0 * g.ldb * kEsz),
                __builtin_amdgcn_readfirstlane((uint32_t)rows_b * (uint32_t)g.ldb * kEsz));

  // Loader: load j of wave w covers LDS bytes [(8w + j) * 1 KB, +1 KB) of an operand K-tile; lane
  // l holds row 8(8w + j) + l/8, 16-byte slot l%8, which is logical chunk (l%8) ^ swz(row) of the
  // row. Each group of eight lanes reads one whole 128-byte line.
  uint32_t off_a[kSlots], off_b[kSlots];
  int kc[kSlots];
#pragma unroll
  for (int j = 0; j < kSlots; ++j) {
    const int r = (w * kSlots + j) * (64 / kSlots) + lane / kSlots;
    const int c = (lane % kSlots) ^ swz(r);
    kc[j] = c * kChunk;
    off_a[j] = (uint32_t)r * (uint32_t)g.lda * kEsz + (uint32_t)(c * 16);
    off_b[j] = (uint32_t)r * (uint32_t)g.ldb * kEsz + (uint32_t)(c * 16);
  }

  // A K-tile t: LDS-DMA into ring slot t % 3. Chunks at or beyond ke, including whole K-tiles past
  // the end, read zeros without touching memory, so every iteration issues the same number of
  // loads and the wait counts below are constants.
  auto load_a = [&](int t) {
    const int k0 = kb + t * kBK;
    const uint32_t koff = (uint32_t)k0 * kEsz;
    char* st = smem + (t % kASlots) * kOperandBytes + w * kSlots * 1024;
#pragma unroll
    for (int j = 0; j < kSlots; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void*)(st + j * 1024), 16,
                                               k0 + kc[j] < ke ? off_a[j] + koff : kOOB, 0, 0, 0);
  };
  // B K-tile t: into register buffer t % 2 (the caller passes that parity as a constant, so that
  // the buffers stay in registers) ...
  u32x4 vb[2][kSlots];
  auto load_b = [&](int t, auto par) {
    const int k0 = kb + t * kBK;
    const uint32_t koff = (uint32_t)k0 * kEsz;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) vb[par][j] = load16(rb, k0 + kc[j] < ke ? off_b[j] + koff : kOOB);
  };
  // ... then from there into LDS slot t % 2.
  auto write_b = [&](auto par) {
    char* st = smem + kBBase + par * kOperandBytes + w * kSlots * 1024 + lane * 16;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) *(u32x4*)(st + j * 1024) = vb[par][j];
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;

  // Fragment reads: block i covers rows wm*128 + 32i + (l%32) of A (wn*... of B); K-pair p reads
  // logical chunk 2p + l/32 (lanes l and l+32 carry the two 16-byte halves of 32 bytes of K).
  // swz(row) depends on row % 64 only: it is the same for a lane's A and B rows of block i.
  int frag_a[4], frag_b[4], swi[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    frag_a[i] = (wm * 128 + i * 32 + (lane & 31)) * kRowBytes;
    frag_b[i] = (wn * 128 + i * 32 + (lane & 31)) * kRowBytes;
    swi[i] = swz(i * 32 + (lane & 31));
  }
  const int khalf = lane >> 5;

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x16){};

  f32x4 fa[2][4], fb[2][4];
  // Fragments of K-pair p of K-tile t into fragment buffer `buf`.
  auto read_frags = [&](int t, int p, int buf) {
    const char* sa = smem + (t % kASlots) * kOperandBytes;
    const char* sb = smem + kBBase + (t & 1) * kOperandBytes;
    const int c = 2 * p + khalf;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa[buf][i] = *(const f32x4*)(sa + frag_a[i] + ((c ^ swi[i]) << 4));
      fb[buf][i] = *(const f32x4*)(sb + frag_b[i] + ((c ^ swi[i]) << 4));
    }
  };
  auto mma = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (kSwap) mfma_pair<T>(acc[i][j], fb[buf][j], fa[buf][i]);
        else mfma_pair<T>(acc[i][j], fa[buf][i], fb[buf][j]);
      }
  };

  // Main loop, one K-tile per iteration. On entry to iteration kt: A K-tile kt and B K-tile kt are
  // in LDS, A K-tile kt + 1 and B K-tiles kt + 1, kt + 2 are in flight. Section p runs the 16
  // MFMAs of K-pair p on fragments read during the previous section while the fragments of K-pair
  // p + 1 are read. Section 0 also starts A K-tile kt + 2 (into the ring slot freed by the previous
  // barrier); section 2 writes B K-tile kt + 1 into the other B slot and reloads its register
  // buffer with B K-tile kt + 3. Then barrier, and section 3 reads K-pair 0 of K-tile kt + 1.
  // Loads retire in issue order, which per iteration is A(kt + 2), B(kt + 3); the prologue issues
  // B(0) A(0) B(1) A(1) B(2) so that "the K-tile needed next has landed" is always "at most 24
  // loads outstanding". The scheduling-group hints pin the interleaving; fragment reads precede
  // LDS-bound loads in program order (the compiler keeps LDS reads before LDS writes that follow).
  constexpr int kAfter = 3 * kLoadsPerOperand;
  auto sched = [](int n_ds_read, int n_ds_write, int n_vmem, bool vmem_first) {
    if constexpr (kEsz != 2) return;  // fp32: four MFMAs per K-pair; left to the compiler
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                       // one MFMA
      if (i < n_ds_read) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
      if (i < n_ds_write) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // one LDS write
      if (vmem_first ? i < n_vmem : i >= 16 - n_vmem)
        __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);                     // one global load
    }
    __builtin_amdgcn_sched_barrier(0);  // each section is scheduled on its own
  };
  // One iteration for K-tile kt, whose parity is `par` (a constant).
  auto iteration = [&](int kt, auto par) {
    constexpr int q = decltype(par)::value ^ 1;
    read_frags(kt, 1, 1);
    load_a(kt + 2);
    mma(0);
    sched(8, 0, kLoadsPerOperand, false);
    read_frags(kt, 2, 0);
    mma(1);
    sched(8, 0, 0, false);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kAfter) : "memory");  // B(kt + 1) landed
    read_frags(kt, 3, 1);
    write_b(std::integral_constant<int, q>{});
    load_b(kt + 3, std::integral_constant<int, q>{});
    mma(0);
    sched(8, kLoadsPerOperand, kLoadsPerOperand, false);
    // A(kt + 1) landed (vmcnt) for every wave (barrier); every wave wrote B(kt + 1) and finished
    // reading the slots that the next iteration refills (lgkmcnt before the barrier).
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kAfter) : "memory");
    read_frags(kt + 1, 0, 0);
    mma(1);
    sched(8, 0, 0, false);
  };
  // An odd count runs one more K-tile of zeros (past the end every load reads zeros).
  const int nk = (ke - kb + kBK - 1) / kBK;
  if (nk > 0) {
    load_b(0, P0{});
    load_a(0);
    load_b(1, P1{});
    load_a(1);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kLoadsPerOperand) : "memory");  // B(0) landed
    write_b(P0{});
    load_b(2, P0{});
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(kAfter) : "memory");    // A(0) landed
    __syncthreads();
    read_frags(0, 0, 0);
    for (int kt = 0; kt < nk; kt += 2) {
      iteration(kt, P0{});
      iteration(kt + 1, P1{});
    }
    // Loads of K-tiles past the end may still be in flight (they target no memory); their LDS and
    // registers must not be reused before they retire.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  // ---- epilogue. Without the swap, accumulator element r of block (i, j) sits at
  //      row = 32i + 8(r/4) + 4(l/32) + r%4, col = 32j + l%32 of the wave's 128 x 128 sub-tile;
  //      with it, at row = 32i + l%32, col = 32j + 8(r/4) + 4(l/32) + r%4.
  const int mw = m0 + wm * 128, nw = n0 + wn * 128;
  const int sub4 = 4 * (lane >> 5);
  const int l32 = lane & 31;

  if constexpr (EPI == EPI_LSE_FWD || EPI == EPI_LSE_BWD) {
    if (mw >= g.M) return;
    const int slice = mw / kLseSlice;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = nw + 32 * j + l32;
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = mw + 32 * i + 8 * (r >> 2) + sub4 + (r & 3);
          if (row < g.M) mx = fmaxf(mx, acc[i][j][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float ml = mx * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = mw + 32 * i + 8 * (r >> 2) + sub4 + (r & 3);
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
              const int row = mw + 32 * i + 8 * q + sub4;
              if (row < g.M)
                store4(e_row + row, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                       acc[i][j][4 * q + 3]);
            }
        }
        if (lane < 32) {
          g.pmax[(size_t)slice * g.ldp + col] = mx;
          g.psum[(size_t)slice * g.ldp + col] = s;
        }
      }
    }
  } else {
    // Swapped layout: lane owns rows mw + 32i + l%32 and 4 consecutive columns per (j, q).
    // N (the output pitch) is a multiple of 4 here, so a 4-column group is all in or all out.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = mw + 32 * i + l32;
      if (row >= g.M) continue;
      if constexpr (EPI == EPI_STORE) {
        if (g.mode == 1) {
          float* o = (float*)g.out + (size_t)split * g.M * g.ldo + (size_t)row * g.ldo;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = nw + 32 * j + 8 * q + sub4;
              if (col < g.N)
                store4(o + col, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
            }
        } else {
          T* o = (T*)g.out + (size_t)row * g.ldo;
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = nw + 32 * j + 8 * q + sub4;
              if (col < g.N)
                store4(o + col, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
            }
        }
      } else {  // EPI_DW
        float* a = g.acc + (size_t)row * g.ldacc;
        T* o = (T*)g.out + (size_t)row * g.ldo;
        if (g.mode == DW_MID || g.mode == DW_LAST) {
          // Load the whole row group first so that the loads are in flight together.
          f32x4 prev[4][4];
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = nw + 32 * j + 8 * q + sub4;
              prev[j][q] = col < g.N ? *(const f32x4*)(a + col) : (f32x4){};
            }
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = nw + 32 * j + 8 * q + sub4;
              if (col >= g.N) continue;
              const float v0 = prev[j][q][0] + acc[i][j][4 * q], v1 = prev[j][q][1] + acc[i][j][4 * q + 1];
              const float v2 = prev[j][q][2] + acc[i][j][4 * q + 2], v3 = prev[j][q][3] + acc[i][j][4 * q + 3];
              if (g.mode == DW_MID) store4(a + col, v0, v1, v2, v3);
              else store4(o + col, v0, v1, v2, v3);
            }
        } else {
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int col = nw + 32 * j + 8 * q + sub4;
              if (col >= g.N) continue;
              if (g.mode == DW_FIRST)
                store4(a + col, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              else
                store4(o + col, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
            }
        }
      }
    }
  }
}

}  // namespace lce
