// MFMA GEMM core for the three contractions of the fused linear + cross-entropy step.
//
//   C[m, n] = sum_k A(m, k) * B(n, k)
//
// Each operand is stored either K-contiguous (element (m, k) at P[m * ld + k]) or MN-contiguous
// (element (m, k) at P[k * ld + m]). The three contractions use:
//   logits^T = W . X_c^T     A = W [V, H] K-contig,        B = X_c [n_c, H] K-contig
//   dH_c     = dZ_c . W      A = dZ_c [n_c, V] K-contig,   B = W [V, H] MN-contig
//   dW      += dZ_c^T . X_c  A = dZ_c [n_c, V] MN-contig,  B = X_c [n_c, H] MN-contig
// so W and dZ are never transposed in memory. Two main loops share the tile, waves, fragment
// reads and epilogues: gemm_kernel (below) takes both operands through LDS and runs dH;
// gemm_xb_kernel (at the end of this file) reads B from a fragment-blocked copy straight into
// registers and runs the logits and dW contractions, whose B is the small X chunk.
//
// gemm_kernel. One workgroup computes a 256 x 256 tile of C with four waves (2 x 2), each wave a
// 128 x 128 sub-tile held as 4 x 4 blocks of the 32x32 MFMA accumulator (256 fp32 per lane). K
// advances in K-tiles of 64 bf16 (32 fp32); an operand's K-tile is 32 KB of LDS either way:
// 256 rows of 128 bytes (K-contig) or 64 (32) K-rows of 512 (1024) bytes (MN-contig). Global loads
// are 16 bytes per lane and read whole 128-byte lines.
//
// Every K-tile is requested about two K-tiles ahead of its MFMAs: with a single K-tile in flight per
// CU the MFMAs wait on this access pattern's load latency, and three LDS stages of both operands
// (192 KB) do not fit in the 160 KB of LDS. So operand A streams straight into a ring of three LDS
// slots (buffer_load ... lds) while operand B is parked in one of two register buffers
// (buffer_load_dwordx4, 64 VGPRs) and written (ds_write_b128) into one of two LDS slots during the
// preceding K-tile. Buffer descriptors turn rows beyond M/N (K-contig) or K-rows beyond the K
// range (MN-contig, one descriptor per K-tile), and K-tiles past the end, into zeros.
//
// Fragments: for the 32x32x16 bf16 MFMA a lane supplies 8 consecutive K of one row/column.
// K-contig tiles give them with one ds_read_b128; MN-contig bf16 tiles with two ds_read_b64_tr_b16
// (each 16-lane group reads four K-rows of 16 columns and the LDS transposes them so that lane j
// receives column j of the four rows); MN-contig fp32 tiles with four ds_read_b32. The 16-byte
// slots of every LDS row are XOR-swizzled so that these reads are free of bank conflicts.
// Fragments are double-buffered in registers: the reads for the next 32 bytes of K are in flight
// while the MFMAs of the current ones run.
//
// The epilogue decides what the tile becomes:
//   LSE_FWD / LSE_BWD : C = logits^T tile (rows = vocabulary, columns = tokens). Per token and per
//                       128-row vocabulary slice: the maximum m and sum exp(z - m) (the vocabulary-
//                       tiled online log-sum-exp); LSE_BWD also stores e = exp(z - m) token-major.
//   STORE             : C written as the output dtype (or as fp32 split-K partials).
//   DW                : C written into dW (first chunk) or added to it (later chunks).
// STORE and DW issue the MFMAs with the operands swapped, so each lane holds four consecutive
// columns of C (LSE_BWD: four consecutive vocabulary rows of e's token-major row). bf16 results
// are regrouped between lanes l and l + 32 so that each store writes 32 contiguous bytes per row.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace lce {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef f16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kTile = 256;                       // BM = BN
constexpr int kTileBytes = 128;                  // bytes of K per row of a K-contig K-tile
constexpr int kOperandBytes = 32 * 1024;         // one operand's K-tile in LDS
constexpr int kASlots = 3;                       // A: ring of K-tiles filled by LDS-DMA
constexpr int kBSlots = 2;                       // B: LDS slots filled from registers
constexpr int kBBase = kASlots * kOperandBytes;  // B slots follow the A ring
constexpr int kGemmSmem = (kASlots + kBSlots) * kOperandBytes;  // 160 KB, all of a CU's LDS
constexpr int kLoadsPerOperand = 8;              // 16-byte loads per lane per operand K-tile
constexpr int kGemmThreads = 256;
constexpr int kLseSlice = 128;                   // vocabulary rows per log-sum-exp partial
constexpr uint32_t kOOB = 0x80000000u;           // a buffer offset beyond every range check
constexpr float kLog2e = 1.4426950408889634f;

enum Epilogue { EPI_LSE_FWD = 0, EPI_LSE_BWD = 1, EPI_STORE = 2, EPI_DW = 3 };
enum DwMode { DW_STORE = 0, DW_ACCUMULATE = 1 };

struct GemmArgs {
  const void* A;
  const void* B;
  int64_t lda, ldb;   // pitches in elements
  int M, N, K;        // K-contig operands need K to be a multiple of 16 bytes' worth
  int tiles_m, tiles_n, splits, k_per_split;  // k_per_split: a multiple of the K-tile
  int group_m;        // tile rows per raster group
  // epilogue
  void* out;          // LSE_BWD: e (token-major, pitch ldo >= M rounded up to 128); STORE: output or
                      // fp32 partials; DW: dW
  int64_t ldo;
  float* pmax;        // LSE: [slices, ldp]
  float* psum;
  int64_t ldp;
  int mode;           // DW: DwMode; STORE: 1 = fp32 split-K partials at out + split * M * ldo
  const int* n_valid; // STORE (mode 0) / DW of 16-bit types whose dz is stored unscaled: the
  int mean;           // valid-token count and reduction that give g (see Storage)
};

// K-contig tiles: logical 16-byte chunk c (0..7) of LDS row r sits in slot c ^ swz_k(r).
__device__ __forceinline__ int swz_k(int r) { return (r ^ (r >> 3)) & 7; }
// MN-contig bf16 tiles: logical 16-byte slot s (0..31) of K-row k sits in slot s ^ swz_mn(k).
__device__ __forceinline__ int swz_mn(int k) { return ((k & 1) ? 4 : 0) ^ ((k & 2) ? 10 : 0) ^ ((k & 8) ? 16 : 0); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// voff: per-lane byte offset; soff: uniform byte offset (an SGPR).
__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff = 0) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, char* lds, uint32_t voff, uint32_t soff = 0) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)lds, 16, voff, soff, 0, 0);
}

__device__ __forceinline__ i16x4 read_tr(const char* lds) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)lds);
}

__device__ __forceinline__ uint64_t uniform64(uint64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
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
__device__ __forceinline__ void mfma_pair<f16>(f32x16& c, const f32x4& a, const f32x4& b) {
  c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
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
__device__ __forceinline__ void store4(f16* p, float a, float b, float c, float d) {
  f16x4 v = {(f16)a, (f16)b, (f16)c, (f16)d};
  *(f16x4*)p = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  f32x4 v = {a, b, c, d};
  *(f32x4*)p = v;
}
__device__ __forceinline__ f32x4 load4(const bf16* p) {
  const bf16x4 v = *(const bf16x4*)p;
  return (f32x4){(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}
__device__ __forceinline__ f32x4 load4(const f16* p) {
  const f16x4 v = *(const f16x4*)p;
  return (f32x4){(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
}
__device__ __forceinline__ f32x4 load4(const float* p) { return *(const f32x4*)p; }

// Storage scales of the 16-bit types. fp16 has a 5-bit exponent: with the mean's 1/n_valid the
// gradient entries of a large vocabulary (~1e-9) would flush to zero, so for fp16 e is stored as
// exp(z - m) 2^15 and dz as (p - [v == y]) 2^10, and the dH / dW epilogues apply
// g 2^-10 (g = 1/n_valid for the mean, 1 for the sum). bf16 (fp32's exponent range) and fp32
// store e and dz = g (p - [v == y]) as they are.
template <typename T>
struct Storage {
  static constexpr float kE = 1.f;           // e is stored times kE
  static constexpr bool kDzUnscaled = false;  // dz holds (p - onehot) kDz instead of g (p - onehot)
  static constexpr float kDz = 1.f;
};
template <>
struct Storage<f16> {
  static constexpr float kE = 32768.f;
  static constexpr bool kDzUnscaled = true;
  static constexpr float kDz = 1024.f;
};

// The factor the dH / dW epilogues apply to their accumulators (1 unless dz is stored unscaled).
template <typename T>
__device__ __forceinline__ float dz_epilogue_scale(const int* n_valid, int mean) {
  if constexpr (!Storage<T>::kDzUnscaled) {
    return 1.f;
  } else {
    const int nv = *n_valid;
    const float g = mean ? (nv > 0 ? 1.f / (float)nv : 0.f) : 1.f;
    return g * (1.f / Storage<T>::kDz);
  }
}

// A 16-bit output row segment of 32 elements held by lanes l and l + 32 (half = l / 32): lane l has
// the 4-element groups at 8q + 4 half, q = 0..3, as v[4q + e]. One v_permlane32_swap per dword
// regroups them so that lane l ends with elements 0-7 and 16-23 and lane l + 32 with 8-15 and
// 24-31, and each store instruction writes 32 contiguous bytes of the row instead of 16 (the
// stores of a tile's epilogue are a burst that every CU issues at about the same time).
// in0 / in1: whether this lane's first / second 8 elements lie inside the output.
// The lane index, recomputed where it is needed: values derived from it early and kept alive
// through the main loop for the epilogue would be spilled.
__device__ __forceinline__ int lane_id() {
  uint32_t ln;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
  return (int)ln;
}

template <typename T>
__device__ __forceinline__ void store_row32(T* p, const f32x16& v, bool in0, bool in1) {
  typedef T t4 __attribute__((ext_vector_type(4)));
  const int half = lane_id() >> 5;
  uint32_t a[4], b[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const t4 x = {(T)v[4 * q], (T)v[4 * q + 1], (T)v[4 * q + 2], (T)v[4 * q + 3]};
    const u32x2 u = __builtin_bit_cast(u32x2, x);
    uint32_t* d = (q & 1) ? b : a;
    d[(q >> 1) * 2] = u[0];
    d[(q >> 1) * 2 + 1] = u[1];
  }
  // a = (q0, q2), b = (q1, q3); swap a's upper 32 lanes with b's lower 32 lanes.
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const auto r = __builtin_amdgcn_permlane32_swap(a[e], b[e], false, false);
    a[e] = r[0];
    b[e] = r[1];
  }
  if (in0) *(u32x4*)(p + 8 * half) = (u32x4){a[0], a[1], b[0], b[1]};
  if (in1) *(u32x4*)(p + 16 + 8 * half) = (u32x4){a[2], a[3], b[2], b[3]};
}

// Loads and fragment reads of one operand (the tile's 256 rows/columns starting at mn0).
template <typename T, bool MN>
struct Operand {
  static constexpr int kEsz = (int)sizeof(T);
  static constexpr int kBK = kTileBytes / kEsz;       // K per K-tile
  static constexpr int kMnRowBytes = kTile * kEsz;    // MN-contig: bytes per K-row

  const char* base;   // element (mn0, 0)
  int64_t ld;
  int kb, ke;         // K range of this split
  // Byte offset of load j within a K-tile = row_off + j * row_step + (slot_x ^ xor_j(j)): a lane
  // term, a uniform term and a compile-time XOR. Two registers per lane instead of eight offsets.
  uint32_t row_off, slot_x, row_step;
  int frag[4];        // per 32-row block: this lane's LDS byte offset at K-pair 0
  __amdgpu_buffer_rsrc_t rsrc_k;  // K-contig: one descriptor for the whole run

  __device__ __forceinline__ void init(const void* p, int64_t ld_, int mn0, int rows, int kb_, int ke_,
                                       int w, int lane, int wsub) {
    ld = ld_;
    kb = kb_;
    ke = ke_;
    if constexpr (!MN) {
      base = (const char*)p + (size_t)mn0 * ld * kEsz;
      rsrc_k = make_rsrc((const void*)uniform64((uint64_t)base),
                         __builtin_amdgcn_readfirstlane((uint32_t)rows * (uint32_t)ld * kEsz));
      // Load j of wave w covers LDS bytes [(8w + j) KB, +1 KB): lane l holds row
      // r = 64w + 8j + l/8, slot l%8, which is logical chunk c = (l%8) ^ swz_k(r) of the row, and
      // swz_k(r) = (l/8) ^ j. So the byte offset is (64w + l/8) ld + 8j ld + 16 (((l%8) ^ (l/8)) ^ j).
      row_off = (uint32_t)(64 * w + (lane >> 3)) * (uint32_t)ld * kEsz;
      row_step = 8u * (uint32_t)ld * kEsz;
      slot_x = (uint32_t)(((lane & 7) ^ (lane >> 3)) << 4);
      // Fragment of block i: row wsub + 32i + l%32, logical chunk 2p + l/32.
#pragma unroll
      for (int i = 0; i < 4; ++i) frag[i] = (wsub + 32 * i + (lane & 31)) * kTileBytes;
    } else {
      base = (const char*)p + (size_t)mn0 * kEsz;
      if constexpr (kEsz == 2) {
        // Load j of wave w: lane l holds K-row kr = 16w + 2j + l/32, slot l%32, which is logical
        // slot (l%32) ^ swz_mn(kr), and swz_mn(kr) = 4 (l/32) ^ 10 (j&1) ^ 16 ((j>>2)&1).
        row_off = (uint32_t)(16 * w + (lane >> 5)) * (uint32_t)ld * 2;
        row_step = 2u * (uint32_t)ld * 2;
        slot_x = (uint32_t)(((lane & 31) ^ (4 * (lane >> 5))) << 4);
        // Transposed reads: 16-lane group g, lane i' = l%16 reads K-row 16p + 8(g/2) + 4s + i'/4
        // at column wsub + 32i + 16(g%2) + 4(i'%4). The swizzle depends only on row bits 0, 1
        // and 3, all fixed by the lane, so the address is this base plus (16p + 4s) * 512.
        // Block i only flips address bits 6-7: its 16-byte slot is block 0's XOR 4i (the column's
        // slot bits 2-3 come from 32i alone), so frag[i] = frag[0] ^ (i << 6).
        const int g = lane >> 4, ip = lane & 15;
        const int r0 = 8 * (g >> 1) + (ip >> 2);
        const int col = wsub + 16 * (g & 1) + 4 * (ip & 3);
        frag[0] = r0 * kMnRowBytes + (((col >> 3) ^ swz_mn(r0)) << 4) + 8 * ((col >> 2) & 1);
      } else {
        // fp32: load j of wave w: lane l holds K-row 8w + j, slot l; fragment reads are plain.
        row_off = (uint32_t)(8 * w) * (uint32_t)ld * 4;
        row_step = (uint32_t)ld * 4;
        slot_x = (uint32_t)(lane * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) frag[i] = (4 * (lane >> 5)) * kMnRowBytes + (wsub + 32 * i + (lane & 31)) * 4;
      }
    }
  }

  // The compile-time XOR part of load j's offset.
  static __device__ __forceinline__ constexpr uint32_t xor_j(int j) {
    if constexpr (!MN) return (uint32_t)(j << 4);
    else if constexpr (kEsz == 2) return (uint32_t)((((j & 1) ? 10 : 0) ^ (((j >> 2) & 1) ? 16 : 0)) << 4);
    else return 0u;
  }

  // Descriptor for K-tile t. MN-contig: its valid K-rows only, so that rows at or beyond ke,
  // including whole K-tiles past the end, read zeros without touching memory.
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(int t) const {
    if constexpr (!MN) {
      return rsrc_k;
    } else {
      const int k0 = kb + t * kBK;
      const int nrows = max(0, min(kBK, ke - k0));
      const char* p = base + (size_t)(k0 < ke ? k0 : kb) * ld * kEsz;
      return make_rsrc((const void*)uniform64((uint64_t)p),
                       __builtin_amdgcn_readfirstlane((uint32_t)nrows * (uint32_t)ld * kEsz));
    }
  }

  // Byte offset of load j of K-tile t, in two parts: a per-lane part, formed by one v_xad_u32 where
  // it is used (hoisted out of the main loop, the sixteen offsets of two operands would outgrow the
  // registers and be spilled, and spill traffic would upset the vmcnt waits), and a uniform part in
  // soffset: j row_step plus, K-contig, the K-tile's start (kOOB for a K-tile at or past ke). A
  // chain of dependent address instructions in front of each load stalls the in-order issue, and
  // the MFMAs queued behind it, for tens of cycles per load. K-contig, this reads whole K-tiles:
  // only for K ranges made of whole K-tiles, or rows whose padding up to the next K-tile is zeros
  // (or meets zeros in the other operand); otherwise offset() below checks every chunk.
  __device__ __forceinline__ uint32_t lane_offset(int j) const {
    uint32_t o;
    asm volatile("v_xad_u32 %0, %1, %2, %3" : "=v"(o) : "v"(slot_x), "s"(xor_j(j)), "v"(row_off));
    return o;
  }
  __device__ __forceinline__ uint32_t uniform_offset(int t, int j) const {
    uint32_t o = (uint32_t)j * row_step;
    if constexpr (!MN) {
      const int k0 = kb + t * kBK;
      o = k0 < ke ? o + (uint32_t)k0 * kEsz : kOOB;
    }
    return __builtin_amdgcn_readfirstlane(o);
  }

  // The whole offset with a per-chunk K check (kOOB where a K-contig chunk lies at or beyond ke),
  // for K-contig operands whose K range ends inside a K-tile.
  __device__ __forceinline__ uint32_t offset(int t, int j) const {
    uint32_t o;
    asm volatile("v_xor_b32 %0, %2, %1\n\tv_add3_u32 %0, %0, %3, %4"
                 : "=&v"(o)
                 : "v"(slot_x), "s"(xor_j(j)), "v"(row_off), "s"((uint32_t)j * row_step));
    if constexpr (!MN) {
      const int k0 = kb + t * kBK;
      const int kc = (int)(((slot_x ^ xor_j(j)) >> 4) * (16 / kEsz));  // first K of the chunk
      return k0 + kc < ke ? o + (uint32_t)k0 * kEsz : kOOB;
    } else {
      return o;
    }
  }

  // Fragment of K-pair p of block i from the LDS tile at `st`.
  __device__ __forceinline__ f32x4 fragment(const char* st, int p, int i, int khalf, int sw) const {
    if constexpr (!MN) {
      return *(const f32x4*)(st + frag[i] + (((2 * p + khalf) ^ sw) << 4));
    } else if constexpr (kEsz == 2) {
      // Issued as inline assembly: the compiler cannot tell which LDS bytes the transposing read
      // builtin touches, and so would wait for every outstanding LDS-DMA load before it. The
      // caller waits for these reads itself (see sync_frags). The address, (frag[0] ^ (i << 6)) +
      // tile base, is formed here too: hoisted, the per-block addresses of two such operands would
      // be spilled.
      i16x4 lo, hi;
      uint32_t a;
      asm volatile(
          "v_xor_b32 %2, %3, %4\n\t"
          "v_add_u32 %2, %5, %2\n\t"
          "ds_read_b64_tr_b16 %0, %2 offset:%6\n\t"
          "ds_read_b64_tr_b16 %1, %2 offset:%7"
          : "=v"(lo), "=v"(hi), "=&v"(a)
          : "s"(i << 6), "v"(frag[0]), "s"((uint32_t)(uintptr_t)(lds_void*)st), "i"((16 * p) * kMnRowBytes),
            "i"((16 * p + 4) * kMnRowBytes));
      const i16x4 v[2] = {lo, hi};
      return __builtin_bit_cast(f32x4, v);
    } else {
      const char* q = st + frag[i] + (8 * p) * kMnRowBytes;
      return (f32x4){*(const float*)q, *(const float*)(q + kMnRowBytes), *(const float*)(q + 2 * kMnRowBytes),
                     *(const float*)(q + 3 * kMnRowBytes)};
    }
  }
};

// 16-bit dW accumulation (chunks after the first): the wave's current dW values in the swapped
// accumulator layout, loaded raw while the pipeline fills, then the accumulators' starting values.
// They enter divided by the factor the epilogue will apply (the dz storage scale, 1 for bf16), so
// that the epilogue's one multiply gives dW + factor * (this chunk's sum); a zero factor (a mean
// over no valid token) starts them at zero.
template <typename T>
using vec4_t = T __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ void load_dw_prev(const GemmArgs& g, vec4_t<T> (&prev)[4][4][4], int mw, int nw, int lane) {
  typedef vec4_t<T> t4;
  const int sub4 = 4 * (lane >> 5);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = mw + 32 * i + (lane & 31);
    const T* o = (const T*)g.out + (size_t)row * g.ldo;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int col = nw + 32 * j + 8 * q + sub4;
        prev[i][j][q] = (row < g.M && col < g.N) ? *(const t4*)(o + col) : (t4){};
      }
  }
}

template <typename T>
__device__ __forceinline__ void apply_dw_prev(f32x16 (&acc)[4][4], const vec4_t<T> (&prev)[4][4][4], float inv_scale) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float x = (float)prev[i][j][q][e];
          acc[i][j][4 * q + e] = Storage<T>::kDzUnscaled ? x * inv_scale : x;
        }
}

// The epilogue factor's reciprocal for apply_dw_prev (0 when the factor is 0).
template <typename T>
__device__ __forceinline__ float dw_prev_scale(const GemmArgs& g) {
  if constexpr (!Storage<T>::kDzUnscaled) {
    return 1.f;
  } else {
    const float sc = dz_epilogue_scale<T>(g.n_valid, g.mean);
    return sc > 0.f ? 1.f / sc : 0.f;
  }
}

// The epilogue: what a wave's 128 x 128 accumulator sub-tile at (mw, nw) becomes. Without the
// operand swap, accumulator element r of block (i, j) sits at row = 32i + 8(r/4) + 4(l/32) + r%4,
// col = 32j + l%32 of the sub-tile; with it, at row = 32i + l%32, col = 32j + 8(r/4) + 4(l/32) + r%4.
// PRELOADED (DW): the accumulators started from the tile's current dW values.
template <typename T, int EPI, bool PRELOADED>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x16 (&acc)[4][4], int mw, int nw, int split,
                                              bool accumulate) {
  constexpr int kEsz = (int)sizeof(T);
  const int lane = lane_id();
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
          acc[i][j][r] = e * Storage<T>::kE;
        }
      s += __shfl_xor(s, 32);
      if (col < g.N) {
        if constexpr (EPI == EPI_LSE_BWD) {
          T* e_row = (T*)g.out + (size_t)col * g.ldo;
          if constexpr (kEsz == 2) {
            // Whole 128-row wave slices: e's pitch is M rounded up to 128, and rows at or beyond M
            // hold exp = 0 here.
#pragma unroll
            for (int i = 0; i < 4; ++i) store_row32(e_row + mw + 32 * i, acc[i][j], true, true);
          } else {
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
    const float sc = dz_epilogue_scale<T>(g.n_valid, g.mean);
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
          if constexpr (kEsz == 2) {
            // N is a multiple of 8 for 16-bit types, so an 8-column piece is all in or all out.
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              if constexpr (Storage<T>::kDzUnscaled) acc[i][j] *= sc;
              const int c0 = nw + 32 * j + 8 * (lane >> 5);
              store_row32(o + nw + 32 * j, acc[i][j], c0 < g.N, c0 + 16 < g.N);
            }
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                const int col = nw + 32 * j + 8 * q + sub4;
                if (col < g.N)
                  store4(o + col, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
              }
          }
        }
      } else if constexpr (PRELOADED) {  // EPI_DW, 16-bit: the accumulators already hold the earlier chunks' sum
        T* o = (T*)g.out + (size_t)row * g.ldo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if constexpr (Storage<T>::kDzUnscaled) acc[i][j] *= sc;
          const int c0 = nw + 32 * j + 8 * (lane >> 5);
          store_row32(o + nw + 32 * j, acc[i][j], c0 < g.N, c0 + 16 < g.N);
        }
      } else {  // EPI_DW, fp32: add the earlier chunks' sum here
        T* o = (T*)g.out + (size_t)row * g.ldo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f32x4 base[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = nw + 32 * j + 8 * q + sub4;
            base[q] = (!PRELOADED && accumulate && col < g.N) ? load4(o + col) : (f32x4){};
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = nw + 32 * j + 8 * q + sub4;
            if (col < g.N)
              store4(o + col, base[q][0] + sc * acc[i][j][4 * q], base[q][1] + sc * acc[i][j][4 * q + 1],
                     base[q][2] + sc * acc[i][j][4 * q + 2], base[q][3] + sc * acc[i][j][4 * q + 3]);
          }
        }
      }
    }
  }
}

// KCHECK: K-contig operands check every chunk against the K range (see Operand::offset).
template <typename T, int EPI, bool A_MN, bool B_MN, bool KCHECK>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_kernel(const GemmArgs g) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kBK = kTileBytes / kEsz;   // elements per K-tile
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

  Operand<T, A_MN> opa;
  Operand<T, B_MN> opb;
  opa.init(g.A, g.lda, m0, min(kTile, g.M - m0), kb, ke, w, lane, wm * 128);
  opb.init(g.B, g.ldb, n0, min(kTile, g.N - n0), kb, ke, w, lane, wn * 128);
  const int khalf = lane >> 5;
  // K-contig fragments: swz_k(row) depends on row % 64 only, the same for a lane's A and B rows.
  int swi[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) swi[i] = swz_k(i * 32 + (lane & 31));

  // A K-tile t: LDS-DMA into ring slot t % 3.
  auto load_a = [&](int t) {
    const __amdgpu_buffer_rsrc_t r = opa.rsrc(t);
    char* st = smem + (t % kASlots) * kOperandBytes + w * 8 * 1024;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if constexpr (KCHECK && !A_MN) dma16(r, st + j * 1024, opa.offset(t, j));
      else dma16(r, st + j * 1024, opa.lane_offset(j), opa.uniform_offset(t, j));
    }
  };
  // B K-tile t: into register buffer t % 2 (the caller passes that parity as a constant, so that
  // the buffers stay in registers) ...
  u32x4 vb[2][8];
  auto load_b = [&](int t, auto par) {
    const __amdgpu_buffer_rsrc_t r = opb.rsrc(t);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if constexpr (KCHECK && !B_MN) vb[par][j] = load16(r, opb.offset(t, j));
      else vb[par][j] = load16(r, opb.lane_offset(j), opb.uniform_offset(t, j));
    }
  };
  // ... then from there into LDS slot t % 2, at the same place LDS-DMA would have put it.
  auto write_b = [&](auto par) {
    char* st = smem + kBBase + par * kOperandBytes + w * 8 * 1024 + lane * 16;
#pragma unroll
    for (int j = 0; j < 8; ++j) *(u32x4*)(st + j * 1024) = vb[par][j];
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;

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
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa[buf][i] = opa.fragment(sa, p, i, khalf, swi[i]);
      fb[buf][i] = opb.fragment(sb, p, i, khalf, swi[i]);
    }
  };
  // Fragment reads issued as inline assembly are invisible to the compiler's wait insertion: at
  // the start of each section wait for all earlier LDS traffic (the previous section's reads, long
  // since done), with the fragment registers as operands so that no MFMA moves above the wait.
  auto sync_frags = [&]() {
    if constexpr ((A_MN || B_MN) && kEsz == 2) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(fa[0][0]), "+v"(fa[0][1]), "+v"(fa[0][2]), "+v"(fa[0][3]), "+v"(fb[0][0]),
                     "+v"(fb[0][1]), "+v"(fb[0][2]), "+v"(fb[0][3]), "+v"(fa[1][0]), "+v"(fa[1][1]),
                     "+v"(fa[1][2]), "+v"(fa[1][3]), "+v"(fb[1][0]), "+v"(fb[1][1]), "+v"(fb[1][2]),
                     "+v"(fb[1][3])
                   :
                   : "memory");
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
  constexpr int kReads = (A_MN ? 0 : 4) + (B_MN ? 0 : 4);  // compiler-visible LDS reads per K-pair
  auto sched = [](int n_ds_write, int n_vmem) {
    if constexpr (kEsz != 2) return;  // fp32: four MFMAs per K-pair; left to the compiler
    // The section's LDS reads go one after each of its first MFMAs.
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                                  // one MFMA
      if (i < kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);                 // one LDS read
      if (i < n_ds_write) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);             // one LDS write
      if (i >= 16 - n_vmem) __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);           // one global load
    }
    __builtin_amdgcn_sched_barrier(0);  // each section is scheduled on its own
  };
  // One iteration for K-tile kt, whose parity is `par` (a constant).
  auto iteration = [&](int kt, auto par) {
    constexpr int q = decltype(par)::value ^ 1;
    sync_frags();
    read_frags(kt, 1, 1);
    load_a(kt + 2);
    mma(0);
    sched(0, kLoadsPerOperand);
    sync_frags();
    read_frags(kt, 2, 0);
    mma(1);
    sched(0, 0);
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kAfter) : "memory");  // B(kt + 1) landed
    sync_frags();
    read_frags(kt, 3, 1);
    write_b(std::integral_constant<int, q>{});
    load_b(kt + 3, std::integral_constant<int, q>{});
    mma(0);
    sched(kLoadsPerOperand, kLoadsPerOperand);
    // A(kt + 1) landed (vmcnt) for every wave (barrier); every wave wrote B(kt + 1) and finished
    // reading the slots that the next iteration refills (lgkmcnt before the barrier).
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kAfter) : "memory");
    read_frags(kt + 1, 0, 0);
    mma(1);
    sched(0, 0);
  };
  // 16-bit dW accumulation (chunks after the first): the tile's current dW values are loaded here,
  // raw, in flight together with the loads that fill the pipeline, and become the accumulators'
  // starting values, so the epilogue only stores. (fp32 adds them in the epilogue instead: its
  // 256 values per lane would not fit next to the pipeline's registers.)
  const int mw = m0 + wm * 128, nw = n0 + wn * 128;
  constexpr bool kPreload = EPI == EPI_DW && kEsz == 2;
  const bool accumulate = EPI == EPI_DW && g.mode == DW_ACCUMULATE;
  vec4_t<T> prev[kPreload ? 4 : 1][4][4];
  if constexpr (kPreload) {
    if (accumulate) load_dw_prev<T>(g, prev, mw, nw, lane);
  }
  // An odd count runs one more K-tile of zeros (past the end every load reads zeros).
  const int nk = (ke - kb + kBK - 1) / kBK;
  if (nk > 0) {
    load_b(0, P0{});
    load_a(0);
    load_b(1, P1{});
    load_a(1);
    if constexpr (kPreload) {
      if (accumulate) apply_dw_prev<T>(acc, prev, dw_prev_scale<T>(g));
    }
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kLoadsPerOperand) : "memory");  // B(0) landed
    write_b(P0{});
    load_b(2, P0{});
    // A(0) landed and B(0) written, for every wave. (Not __syncthreads: it would also wait for
    // every load in flight.)
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kAfter) : "memory");
    read_frags(0, 0, 0);
    for (int kt = 0; kt < nk; kt += 2) {
      iteration(kt, P0{});
      iteration(kt + 1, P1{});
    }
    // Loads of K-tiles past the end may still be in flight (they target no memory); their LDS and
    // registers must not be reused before they retire.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  gemm_epilogue<T, EPI, kPreload>(g, acc, mw, nw, split, accumulate);
}

// ---- Operand B straight to registers ---------------------------------------------------------
//
// gemm_xb_kernel computes the same tile with the same waves and epilogues, but reads operand B from
// a fragment-blocked copy straight into the registers the MFMAs take it from: every B load is one
// whole 1 KB fragment, and B never passes through LDS, which halves a K-tile's LDS traffic (A's
// 32 KB written, 64 KB read). A streams into a ring of four LDS slots by LDS-DMA, three K-tiles
// ahead; B circulates through a ring of eight K-pairs of fragments (128 VGPRs), seven K-pairs ahead.
// A K-tile is four sections of 16 MFMAs; each section issues one quarter of A's K-tile three ahead
// (two LDS-DMA loads) and the four B fragments of the K-pair seven ahead, between its MFMAs.
//
// Blocked layout of B (N columns, reduction K, element type T): fragment (jb, q) -- 32 columns by
// K-pair q, the q-th 32 bytes of every column's K run -- is 1 KB at byte (jb KP + q) 1024, and lane
// l of it holds column 32 jb + l%32, bytes [32 q + 16 (l/32), +16): the 16 bytes that lane feeds
// the MFMA. KP counts the K-pairs per column block with K rounded up to a whole K-tile; columns at
// or beyond N and K at or beyond K are zeros. (The A fragments read from LDS cover the same K bytes:
// K-pair p of K-tile t, lane half h, bytes [32 p + 16 h, +16) of the K-tile.)
constexpr int kXbASlots = 4;
constexpr int kXbAhead = kXbASlots - 1;
constexpr int kXbSmem = kXbASlots * kOperandBytes;  // 128 KB

// Blocked copy of a K-contiguous source (element (n, k) at src[n * ld + k]; K a multiple of 16
// bytes' worth): one thread per 16-byte piece. Grid: NB * KP * 64 threads.
template <typename T>
__global__ __launch_bounds__(256) void block_k_kernel(const T* __restrict__ src, int64_t ld, int N, int K, int KP,
                                                      int NB, T* __restrict__ dst) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t frag = t >> 6;
  if (frag >= (int64_t)NB * KP) return;
  const int l = (int)(t & 63);
  const int jb = (int)(frag / KP), q = (int)(frag - (int64_t)jb * KP);
  const int n = 32 * jb + (l & 31);
  const int k = (32 * q + 16 * (l >> 5)) / (int)sizeof(T);
  u32x4 v = {0u, 0u, 0u, 0u};
  if (n < N && k < K) v = *(const u32x4*)(src + (size_t)n * ld + k);
  *(u32x4*)((char*)dst + (size_t)frag * 1024 + l * 16) = v;
}

// Blocked copy of an MN-contiguous source (element (n, k) at src[k * ld + n]; N a multiple of 16
// bytes' worth): block (jb, g) stages the 128 bytes' worth of K rows of K-pairs 4g .. 4g + 3 by 32
// columns in LDS, then each thread gathers one 16-byte piece down a column. Grid: (NB, ceil(KP / 4)).
template <typename T>
__global__ __launch_bounds__(256) void block_mn_kernel(const T* __restrict__ src, int64_t ld, int N, int K, int KP,
                                                       T* __restrict__ dst) {
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kVec = 16 / kEsz;            // elements per piece
  constexpr int kRows = 128 / kEsz;          // K rows of four K-pairs
  constexpr int kPieces = 32 / kVec;         // pieces per K row of 32 columns
  static_assert(kRows * kPieces == 256, "one piece per thread");
  typedef T vec_t __attribute__((ext_vector_type(kVec)));
  __shared__ __attribute__((aligned(16))) T tile[kRows][32];
  const int jb = blockIdx.x, grp = blockIdx.y;
  const int t = threadIdx.x;
  {
    const int r = t / kPieces, pc = t % kPieces;
    const int k = grp * kRows + r, n = 32 * jb + pc * kVec;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (k < K && n < N) v = *(const u32x4*)(src + (size_t)k * ld + n);
    *(u32x4*)&tile[r][pc * kVec] = v;
  }
  __syncthreads();
  const int q = grp * 4 + (t >> 6);
  if (q >= KP) return;
  const int l = t & 63;
  const int kr = (t >> 6) * (32 / kEsz) + (l >> 5) * kVec;
  vec_t v;
#pragma unroll
  for (int e = 0; e < kVec; ++e) v[e] = tile[kr + e][l & 31];
  *(vec_t*)((char*)dst + ((size_t)jb * KP + q) * 1024 + l * 16) = v;
}

// g.B: the blocked copy of B; g.ldb: its KP. Splits must start at whole K-tiles (k_per_split).
template <typename T, int EPI, bool A_MN, bool KCHECK>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_xb_kernel(const GemmArgs g) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kBK = kTileBytes / kEsz;
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

  Operand<T, A_MN> opa;
  opa.init(g.A, g.lda, m0, min(kTile, g.M - m0), kb, ke, w, lane, wm * 128);
  const int khalf = lane >> 5;
  int swi[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) swi[i] = swz_k(i * 32 + (lane & 31));

  // B: this wave's four column blocks start at jb0; K-pair q of this split is fragment q0 + q.
  const int KP = (int)g.ldb;
  const int NB = (g.N + 31) >> 5;
  const __amdgpu_buffer_rsrc_t rb =
      make_rsrc(g.B, __builtin_amdgcn_readfirstlane((uint32_t)NB * (uint32_t)KP * 1024u));
  const int jb0 = (n0 + wn * 128) >> 5;
  const uint32_t bvoff = (uint32_t)lane * 16u;
  const int q0 = kb * kEsz / 32;
  const int qend = ((ke - kb) * kEsz + 31) / 32;

  // Quarter pc of A K-tile t (loads 2 pc, 2 pc + 1) into ring slot t % 4.
  auto load_a_q = [&](int t, auto pc) {
    constexpr int pq = decltype(pc)::value;
    const __amdgpu_buffer_rsrc_t r = opa.rsrc(t);
    char* st = smem + (t & (kXbASlots - 1)) * kOperandBytes + w * 8 * 1024;
#pragma unroll
    for (int j = 2 * pq; j < 2 * pq + 2; ++j) {
      if constexpr (KCHECK && !A_MN) dma16(r, st + j * 1024, opa.offset(t, j));
      else dma16(r, st + j * 1024, opa.lane_offset(j), opa.uniform_offset(t, j));
    }
  };
  auto load_a = [&](int t) {
    load_a_q(t, std::integral_constant<int, 0>{});
    load_a_q(t, std::integral_constant<int, 1>{});
    load_a_q(t, std::integral_constant<int, 2>{});
    load_a_q(t, std::integral_constant<int, 3>{});
  };
  f32x4 vb[8][4];
  // B K-pair q into ring slot `slot` (a constant, so that the ring stays in registers).
  auto load_b = [&](int q, auto slot) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t so = q < qend ? (uint32_t)((jb0 + j) * KP + q0 + q) * 1024u : kOOB;
      vb[decltype(slot)::value][j] = __builtin_bit_cast(f32x4, load16(rb, bvoff, __builtin_amdgcn_readfirstlane(so)));
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (f32x16){};

  f32x4 fa[2][4];
  auto read_frags = [&](int t, int p, int buf) {
    const char* sa = smem + (t & (kXbASlots - 1)) * kOperandBytes;
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[buf][i] = opa.fragment(sa, p, i, khalf, swi[i]);
  };
  // See gemm_kernel: transposing reads are invisible to the compiler's waits.
  auto sync_frags = [&]() {
    if constexpr (A_MN && kEsz == 2) {
      asm volatile("s_waitcnt lgkmcnt(0)"
                   : "+v"(fa[0][0]), "+v"(fa[0][1]), "+v"(fa[0][2]), "+v"(fa[0][3]), "+v"(fa[1][0]),
                     "+v"(fa[1][1]), "+v"(fa[1][2]), "+v"(fa[1][3])
                   :
                   : "memory");
    }
  };
  auto mma = [&](int buf, auto slot) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (kSwap) mfma_pair<T>(acc[i][j], vb[decltype(slot)::value][j], fa[buf][i]);
        else mfma_pair<T>(acc[i][j], fa[buf][i], vb[decltype(slot)::value][j]);
      }
  };
  constexpr int kReads = A_MN ? 0 : 4;  // compiler-visible LDS reads per section
  // The section's LDS reads after its first MFMAs, its six loads after MFMAs 1, 3, .., 11.
  auto sched = []() {
    if constexpr (kEsz != 2) return;  // fp32: 64 MFMAs per section; left to the compiler
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (i < kReads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      if ((i & 1) && i < 12) __builtin_amdgcn_sched_group_barrier(0x010, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  // Section s (0..7) of the K-tile pair starting at kt (even): K-tile kt' = kt + s/4, K-pair
  // p = s%4, K-pair q = 4 kt + s of the split. The compiler waits for B's registers itself. At
  // p == 3, A(kt' + 1) has landed in LDS for every wave before K-pair 0 of it is read: its last
  // quarter went out in section 4 (kt' + 1 - ahead) + 3, and each of the 4 ahead - 5 sections
  // since issued six loads (loads retire in order; whichever order a section issues its own two
  // kinds in, all six of a later section come after).
  constexpr int kAWait = 6 * (4 * kXbAhead - 5);
  static_assert(kXbAhead >= 2 && kAWait <= 63, "vmcnt range");
  auto section = [&](int kt, auto sc) {
    constexpr int s = decltype(sc)::value;
    constexpr int p = s & 3;
    const int ktp = kt + (s >> 2);
    if constexpr (p == 3) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(kAWait) : "memory");
    sync_frags();
    if constexpr (p == 3) read_frags(ktp + 1, 0, (s + 1) & 1);
    else read_frags(ktp, p + 1, (s + 1) & 1);
    // Loads retire in issue order, so a B load waits for every A load issued before it. With A
    // K-contiguous (W, streamed from HBM) the section issues its B fragments first (measured 4%
    // faster on the logits GEMM); with A MN-contiguous (dZ^T) the order made no difference.
    if constexpr (!A_MN) {
      mma(s & 1, std::integral_constant<int, s>{});
      load_b(4 * kt + s + 7, std::integral_constant<int, (s + 7) & 7>{});
      load_a_q(ktp + kXbAhead, std::integral_constant<int, p>{});
    } else {
      load_a_q(ktp + kXbAhead, std::integral_constant<int, p>{});
      mma(s & 1, std::integral_constant<int, s>{});
      load_b(4 * kt + s + 7, std::integral_constant<int, (s + 7) & 7>{});
    }
    sched();
  };

  const int mw = m0 + wm * 128, nw = n0 + wn * 128;
  constexpr bool kPreload = EPI == EPI_DW && kEsz == 2;
  const bool accumulate = EPI == EPI_DW && g.mode == DW_ACCUMULATE;
  vec4_t<T> prev[kPreload ? 4 : 1][4][4];
  if constexpr (kPreload) {
    if (accumulate) load_dw_prev<T>(g, prev, mw, nw, lane);
  }
  // An odd count runs one more K-tile of zeros (past the end every load reads zeros).
  const int nk = (ke - kb + kBK - 1) / kBK;
  if (nk > 0) {
    // Prologue: A(0 .. ahead-1), then B(0 .. 6). A(0) has landed for every wave (issued after it:
    // the other A K-tiles and 28 B loads) before its first fragments are read; the first waits at
    // p == 3 find at least as many loads after A(1), A(2) as they allow. The dW values (128 VGPRs
    // raw) become accumulators once the first three K-pairs of B are on their way, before the rest
    // of B's ring fills the registers.
#pragma unroll
    for (int t = 0; t < kXbAhead; ++t) load_a(t);
    load_b(0, std::integral_constant<int, 0>{});
    load_b(1, std::integral_constant<int, 1>{});
    load_b(2, std::integral_constant<int, 2>{});
    if constexpr (kPreload) {
      if (accumulate) apply_dw_prev<T>(acc, prev, dw_prev_scale<T>(g));
    }
    load_b(3, std::integral_constant<int, 3>{});
    load_b(4, std::integral_constant<int, 4>{});
    load_b(5, std::integral_constant<int, 5>{});
    load_b(6, std::integral_constant<int, 6>{});
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(8 * (kXbAhead - 1) + 28) : "memory");
    read_frags(0, 0, 0);
    for (int kt = 0; kt < nk; kt += 2) {
      section(kt, std::integral_constant<int, 0>{});
      section(kt, std::integral_constant<int, 1>{});
      section(kt, std::integral_constant<int, 2>{});
      section(kt, std::integral_constant<int, 3>{});
      section(kt, std::integral_constant<int, 4>{});
      section(kt, std::integral_constant<int, 5>{});
      section(kt, std::integral_constant<int, 6>{});
      section(kt, std::integral_constant<int, 7>{});
    }
    // Loads past the end may still be in flight (they target no memory); their LDS and registers
    // must not be reused before they retire.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  gemm_epilogue<T, EPI, kPreload>(g, acc, mw, nw, split, accumulate);
}

}  // namespace lce
