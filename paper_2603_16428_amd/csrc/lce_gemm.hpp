// MFMA GEMM core for the three contractions of the fused linear + cross-entropy step.
//
//   C[m, n] = sum_k A(m, k) * B(n, k)
//
// Operand A is stored K-contiguous (element (m, k) at P[m * ld + k]), MN-contiguous (element
// (m, k) at P[k * ld + m]) or fragment-blocked; operand B is always fragment-blocked (the layout is
// defined above gemm_xb_kernel). The three contractions use:
//   logits^T = W . X_c^T      A = W [V, H] K-contig,    B = X_c blocked (columns tokens, K = H)
//   dH_c^T   = W^T . dZ_c^T   A = W [V, H] MN-contig,   B = dZ_c blocked (columns tokens, K = V)
//   dW      += dZ_c^T . X_c   A = dZ_c blocked,         B = X_c blocked (columns H, K = tokens)
// The logits epilogue stores e, and dlogits then dZ, in the blocked layout itself, so W is never
// transposed or copied and only the small X chunk is rearranged (twice per chunk).
//
// One workgroup computes a 256 x 256 tile of C with four waves (2 x 2), each wave a 128 x 128
// sub-tile held as 4 x 4 blocks of the 32x32 MFMA accumulator (256 fp32 per lane). K advances in
// K-tiles of 64 bf16 (32 fp32); A's K-tile is 32 KB of LDS either way: 256 rows of 128 bytes
// (K-contig) or 64 (32) K-rows of 512 (1024) bytes (MN-contig and blocked). Global loads are 16
// bytes per lane. Buffer descriptors turn rows beyond M (K-contig) or K-rows beyond the K range
// (MN-contig and blocked, one descriptor per K-tile), and K-tiles past the end, into zeros.
//
// A's fragments: for the 32x32x16 bf16 MFMA a lane supplies 8 consecutive K of one row. K-contig
// tiles give them with one ds_read_b128; MN-contig bf16 tiles with two ds_read_b64_tr_b16 (each
// 16-lane group reads four K-rows of 16 columns and the LDS transposes them so that lane j
// receives column j of the four rows); MN-contig fp32 tiles with four ds_read_b32. The 16-byte
// slots of every LDS row are XOR-swizzled so that these reads are free of bank conflicts. A
// blocked A is fetched into the very LDS slots an MN-contig one would occupy. Fragments are
// double-buffered in registers: the reads for the next 32 bytes of K are in flight while the
// MFMAs of the current ones run.
//
// The epilogue decides what the tile becomes:
//   LSE_FWD / LSE_BWD : C = logits^T tile (rows = vocabulary, columns = tokens). Per token and per
//                       128-row vocabulary slice: the maximum m and sum exp(z - m) (the vocabulary-
//                       tiled online log-sum-exp); LSE_BWD also stores e = exp(z - m), blocked.
//   STORE             : C^T written token-major as the output dtype (or as fp32 split-K partials):
//                       the chunk's dH rows from dH^T tiles.
//   DW                : C written into dW (first chunk) or added to it (later chunks).
// DW issues the MFMAs with the operands swapped, so each lane holds four consecutive columns of C;
// LSE and STORE keep four consecutive rows of C (vocabulary ids, hidden units) per lane. 16-bit
// results are regrouped between lanes l and l + 32 so that each lane stores 16 contiguous bytes.
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
constexpr int kGemmThreads = 256;
constexpr int kLseSlice = 128;                   // vocabulary rows per log-sum-exp partial
constexpr uint32_t kOOB = 0x80000000u;           // a buffer offset beyond every range check
constexpr float kLog2e = 1.4426950408889634f;

enum Epilogue { EPI_LSE_FWD = 0, EPI_LSE_BWD = 1, EPI_STORE = 2, EPI_DW = 3 };
// Layouts of operand A: K-contiguous, MN-contiguous, fragment-blocked (MN pieces, see Operand).
enum ALayout { A_K = 0, A_MN = 1, A_BLK = 2 };
// DW epilogue: the first chunk writes dW, later ones add to it (the running sum carried in dW's own
// type); or, with an fp32 cross-chunk accumulator (acc32), the first chunk writes acc32, the middle
// ones add to it and the last one adds and writes dW.
enum DwMode { DW_STORE = 0, DW_ACCUMULATE = 1, DW_ACC32_FIRST = 2, DW_ACC32_MID = 3, DW_ACC32_LAST = 4 };

struct GemmArgs {
  const void* A;
  const void* B;
  int64_t lda, ldb;   // pitches in elements
  int M, N, K;        // K-contig operands need K to be a multiple of 16 bytes' worth
  int tiles_m, tiles_n, splits, k_per_split;  // k_per_split: a multiple of the K-tile
  int group_m;        // tile rows per raster group
  // epilogue
  void* out;          // LSE_BWD: e, blocked (ldo = K-pairs per token block, covering M rounded up
                      // to 256); STORE: token-major output or fp32 partials; DW: dW
  int64_t ldo;
  float* pmax;        // LSE: [slices, ldp]
  float* psum;
  int64_t ldp;
  int mode;           // DW: DwMode; STORE: 1 = fp32 split-K partials at out + split * M * ldo
  const int* n_valid; // STORE (mode 0) / DW of 16-bit types whose dz is stored unscaled: the
  int mean;           // valid-token count and reduction that give g (see Storage)
  // LSE_BWD, target-referenced (ref != nullptr; chunk-offset, like the columns): ref[col] is the
  // token's target logit if it has a valid label, else NaN. A token with a finite ref has its e
  // stored relative to it instead of the slice maximum, and its partials use the same reference;
  // every other token (ignored, label outside [0, M), padding) has its e stored as 0.
  const float* ref;
  const float* col_scale;  // STORE: per-column factor on the accumulators (nullptr = none)
  const int* run_if;       // nullptr, or: the launch does nothing unless *run_if != 0
  float* acc32;            // DW with mode DW_ACC32_*: fp32 accumulator [M, ldo]
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

// The lane index, recomputed where it is needed: values derived from it early and kept alive
// through the main loop for the epilogue would be spilled.
__device__ __forceinline__ int lane_id() {
  uint32_t ln;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(ln));
  return (int)ln;
}

// A 16-bit segment of 32 consecutive elements held by lanes l and l + 32 (half = l / 32): lane l
// has the 4-element groups at 8q + 4 half, q = 0..3, as v[4q + e]. One v_permlane32_swap per dword
// regroups them so that lane l ends with elements 0-7 (lo) and 16-23 (hi) and lane l + 32 with
// 8-15 and 24-31: whole 16-byte pieces, so that each store instruction writes 32 contiguous bytes
// of a row instead of 16, or one whole 1 KB fragment of the blocked layout.
template <typename T>
__device__ __forceinline__ void regroup32(const f32x16& v, u32x4& lo, u32x4& hi) {
  typedef T t4 __attribute__((ext_vector_type(4)));
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
  lo = (u32x4){a[0], a[1], b[0], b[1]};
  hi = (u32x4){a[2], a[3], b[2], b[3]};
}

// Row-major: the segment starts at p; in0 / in1: whether this lane's first / second 8 elements lie
// inside the output.
template <typename T>
__device__ __forceinline__ void store_row32(T* p, const f32x16& v, bool in0, bool in1) {
  const int half = lane_id() >> 5;
  u32x4 lo, hi;
  regroup32<T>(v, lo, hi);
  if (in0) *(u32x4*)(p + 8 * half) = lo;
  if (in1) *(u32x4*)(p + 16 + 8 * half) = hi;
}

// Blocked: the segment is 32 vocabulary ids of one token, which fill this lane's 16-byte piece of
// two consecutive fragments; p is the piece in the first.
template <typename T>
__device__ __forceinline__ void store_frag32(char* p, const f32x16& v) {
  u32x4 lo, hi;
  regroup32<T>(v, lo, hi);
  *(u32x4*)p = lo;
  *(u32x4*)(p + 1024) = hi;
}

// Loads and fragment reads of operand A (the tile's 256 rows starting at mn0) in layout AL.
//
// Blocked A (AL = A_BLK) is dZ as the logits epilogue and dlogits leave it: M = vocabulary ids,
// K = tokens, in the fragment-blocked layout with the tokens as its columns and the ids as its K
// (ld = K-pairs per 32-token block). Element (m, k) is at byte (k / 32 ld + m s / 32) 1024 +
// (k % 32 + 32 ((m s / 16) % 2)) 16 + (m s) % 16, s = sizeof(T): a 16-byte piece holds 16 / s
// consecutive ids of one token. 16-bit: each load fetches one whole fragment (1 KB, 32 tokens by
// 16 ids) into LDS as it is, up to a permutation of its pieces, and the transposing fragment reads
// find each lane's four ids of a token inside a piece. fp32: each load fetches the MN-contig
// pieces (4 ids of one token at 512 c + 16 (k % 32) past the token block's start of the tile's
// ids, c the MN slot), 32 scattered pieces per load, into the MN-contig LDS layout.
template <typename T, int AL>
struct Operand {
  static constexpr int kEsz = (int)sizeof(T);
  static constexpr int kBK = kTileBytes / kEsz;       // K per K-tile
  static constexpr int kMnRowBytes = kTile * kEsz;    // MN-contig: bytes per K-row
  static constexpr bool MN = AL != A_K;                // the MN-contig LDS layout and fragment reads
  static constexpr bool BLK = AL == A_BLK;

  const char* base;   // element (mn0, 0)
  int64_t ld;
  int kb, ke;         // K range of this split
  // Byte offset of load j within a K-tile = row_off + j * row_step + (slot_x ^ xor_j(j)): a lane
  // term, a uniform term and a compile-time XOR (the kernel forms the eight per-lane terms once).
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
      base = BLK ? (const char*)p + (size_t)mn0 * 32 * kEsz : (const char*)p + (size_t)mn0 * kEsz;
      if constexpr (kEsz == 2) {
        const int g = lane >> 4, ip = lane & 15;
        if constexpr (BLK) {
          // The LDS K-tile holds the 32 fragments of the K-tile's two token blocks b by the
          // tile's 16 id fragments c, fragment (b, c) in 1 KB slot 16 b + c. Piece P of a fragment
          // (token P%32, id half P/32) sits at 16 Q, Q = P ^ 4 (P/32) ^ 8 (c%2), so that the
          // fragment reads below are free of bank conflicts. Load j of wave w fills slot 8w + j:
          // token block w/2, c = 8 (w%2) + j; lane l fetches piece l ^ 4 (l/32) ^ 8 (j%2).
          row_off = (uint32_t)(w >> 1) * (uint32_t)ld * 1024u + (uint32_t)(w & 1) * 8192u;
          row_step = 1024u;
          slot_x = (uint32_t)((lane ^ (4 * (lane >> 5))) << 4);
          // Transposed reads: 16-lane group g, lane i' = l%16 reads token 16p + 8(g/2) + 4s + i'/4
          // of the K-tile, ids wsub + 32i + 16(g%2) + 4(i'%4) .. + 3: slot 16 (p/2) + (wsub +
          // 32i)/16 + g%2, Q = i'/4 + 4 (s ^ h) + 8 ((g/2) ^ (g%2)) + 16 (p%2) + 32 h with
          // h = (i'%4)/2, byte 8 (i'%2) of the piece. frag[0] is the address at p = s = i = 0;
          // s flips bit 6, p and i add 16384 (p/2) + 256 (p%2) + 2048 i.
          const int h = (ip & 3) >> 1;
          frag[0] = (wsub / 16 + (g & 1)) * 1024 + 16 * ((ip >> 2) + 4 * h + 8 * ((g >> 1) ^ (g & 1)) + 32 * h) +
                    8 * (ip & 1);
        } else {
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
          const int r0 = 8 * (g >> 1) + (ip >> 2);
          const int col = wsub + 16 * (g & 1) + 4 * (ip & 3);
          frag[0] = r0 * kMnRowBytes + (((col >> 3) ^ swz_mn(r0)) << 4) + 8 * ((col >> 2) & 1);
        }
      } else {
        // fp32: load j of wave w: lane l holds K-row 8w + j, slot l; fragment reads are plain.
        // Blocked: K-row 8w + j is token 8w + j of the K-tile's one token block; slot l at 512 l.
        if constexpr (BLK) {
          row_off = (uint32_t)(8 * w) * 16u;
          row_step = 16u;
          slot_x = (uint32_t)lane << 9;
        } else {
          row_off = (uint32_t)(8 * w) * (uint32_t)ld * 4;
          row_step = (uint32_t)ld * 4;
          slot_x = (uint32_t)(lane * 16);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) frag[i] = (4 * (lane >> 5)) * kMnRowBytes + (wsub + 32 * i + (lane & 31)) * 4;
      }
    }
  }

  // The compile-time XOR part of load j's offset.
  static __device__ __forceinline__ constexpr uint32_t xor_j(int j) {
    if constexpr (!MN) return (uint32_t)(j << 4);
    else if constexpr (kEsz == 2 && BLK) return (uint32_t)((j & 1) ? 128 : 0);
    else if constexpr (kEsz == 2) return (uint32_t)((((j & 1) ? 10 : 0) ^ (((j >> 2) & 1) ? 16 : 0)) << 4);
    else return 0u;
  }

  // Descriptor for K-tile t. MN-contig: its valid K-rows only, so that rows at or beyond ke,
  // including whole K-tiles past the end, read zeros without touching memory. Blocked: the token
  // blocks that hold tokens below ke (the rest of the last one is zeros in memory), up to the end
  // of the tile's ids in the last of them.
  __device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(int t) const {
    if constexpr (!MN) {
      return rsrc_k;
    } else if constexpr (BLK) {
      // Branch-free (a branch here would split the main loop's scheduled sections): a K-tile at or
      // past the end gets no blocks and an empty range, whatever its base.
      const int k0 = kb + t * kBK;
      const int nblk = min(kBK / 32, (max(ke - k0, 0) + 31) >> 5);
      const uint32_t blk = (uint32_t)ld * 1024u;
      const uint32_t bytes = (uint32_t)nblk * blk - (uint32_t)min(nblk, 1) * (blk - (uint32_t)(kTile * kEsz * 32));
      const char* p = base + (size_t)(k0 >> 5) * blk;
      return make_rsrc((const void*)uniform64((uint64_t)p), __builtin_amdgcn_readfirstlane(bytes));
    } else {
      const int k0 = kb + t * kBK;
      const int nrows = max(0, min(kBK, ke - k0));
      const char* p = base + (size_t)(k0 < ke ? k0 : kb) * ld * kEsz;
      return make_rsrc((const void*)uniform64((uint64_t)p),
                       __builtin_amdgcn_readfirstlane((uint32_t)nrows * (uint32_t)ld * kEsz));
    }
  }

  // Byte offset of load j of K-tile t, in two parts: a per-lane part, computed once per tile for
  // the eight loads of a K-tile and held in registers through the main loop (lane_offset), and a
  // uniform part in soffset: j row_step plus, K-contig, the K-tile's start (kOOB for a K-tile at or
  // past ke). Address arithmetic in front of each load stalls the in-order issue, and the MFMAs
  // queued behind it; with operand B straight to registers the eight lane offsets fit beside the
  // pipeline without spills (a build test checks). K-contig, this reads whole K-tiles: only for K
  // ranges made of whole K-tiles, or rows whose padding up to the next K-tile is zeros (or meets
  // zeros in the other operand); otherwise offset() below checks every chunk.
  __device__ __forceinline__ uint32_t lane_offset(int j) const { return (slot_x ^ xor_j(j)) + row_off; }
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

  // 16-bit MN-contig and blocked A: the fragment reads address LDS through per-lane registers that
  // hold the whole address in the current pair of ring slots (slots 0-1 or 2-3), so that the slot
  // within the pair, the K-pair and the block enter as the read's immediate offset and no address
  // arithmetic sits between the MFMAs. MN: xa[i] for block i (frag[0] ^ (i << 6)); blocked: xa[0]
  // and xa[1] for the two reads of a fragment (frag[0], frag[0] ^ 64). All plus the ring's base.
  static constexpr int kXa = (kEsz == 2 && MN) ? (BLK ? 2 : 4) : 0;
  uint32_t xa[kXa > 0 ? kXa : 1];
  __device__ __forceinline__ void init_xa(uint32_t ring_base) {
    if constexpr (kXa > 0) {
#pragma unroll
      for (int k = 0; k < kXa; ++k)
        xa[k] = ring_base + (uint32_t)(frag[0] ^ (k << 6));
    }
  }
  // Moves the addresses to the other pair of slots (delta = +-2 slots).
  __device__ __forceinline__ void shift_xa(int delta) {
    if constexpr (kXa > 0) {
#pragma unroll
      for (int k = 0; k < kXa; ++k) xa[k] += (uint32_t)delta;
    }
  }
  // Fragment of K-pair KPR of block i in slot SIP (0, 1) of the pair that the addresses `a` point at.
  template <int SIP, int KPR>
  static __device__ __forceinline__ f32x4 fragment_x(const uint32_t (&a)[kXa > 0 ? kXa : 1], int i) {
    i16x4 lo, hi;
    if constexpr (BLK) {
      // Block i adds 2048 i; K-pair p adds 16384 (p/2) + 256 (p%2); the second read is at frag ^ 64.
      asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%4\n\tds_read_b64_tr_b16 %1, %3 offset:%4"
                   : "=v"(lo), "=v"(hi)
                   : "v"(a[0]), "v"(a[1]), "i"(SIP * kOperandBytes + 16384 * (KPR >> 1) + 256 * (KPR & 1) + 2048 * i));
    } else {
      asm volatile("ds_read_b64_tr_b16 %0, %2 offset:%3\n\tds_read_b64_tr_b16 %1, %2 offset:%4"
                   : "=v"(lo), "=v"(hi)
                   : "v"(a[i]), "i"(SIP * kOperandBytes + (16 * KPR) * kMnRowBytes),
                     "i"(SIP * kOperandBytes + (16 * KPR + 4) * kMnRowBytes));
    }
    const i16x4 v[2] = {lo, hi};
    return __builtin_bit_cast(f32x4, v);
  }

  // Fragment of K-pair p of block i from the LDS tile at `st`.
  __device__ __forceinline__ f32x4 fragment(const char* st, int p, int i, int khalf, int sw) const {
    if constexpr (!MN) {
      return *(const f32x4*)(st + frag[i] + (((2 * p + khalf) ^ sw) << 4));
    } else if constexpr (kEsz == 2 && BLK) {
      // As below; the two reads of a fragment differ in address bit 6 (s), which the tile base
      // (a multiple of 1 KB) leaves alone, and p and i only add an immediate offset.
      i16x4 lo, hi;
      uint32_t a, b;
      asm volatile(
          "v_add_u32 %2, %4, %5\n\t"
          "v_xor_b32 %3, 64, %2\n\t"
          "ds_read_b64_tr_b16 %0, %2 offset:%6\n\t"
          "ds_read_b64_tr_b16 %1, %3 offset:%6"
          : "=v"(lo), "=v"(hi), "=&v"(a), "=&v"(b)
          : "s"((uint32_t)(uintptr_t)(lds_void*)st), "v"(frag[0]), "i"(16384 * (p >> 1) + 256 * (p & 1) + 2048 * i));
      const i16x4 v[2] = {lo, hi};
      return __builtin_bit_cast(f32x4, v);
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

// 16-bit dW accumulation (chunks after the first): the wave's current dW values, loaded raw while
// the pipeline fills, then the accumulators' starting values. Each lane loads the two 16-byte row
// pieces that store_row32 writes from it (lanes l and l + 32 cover 32 contiguous bytes of a row per
// load), and one v_permlane32_swap per dword -- the inverse of regroup32's, which is its own
// inverse -- returns the elements to the swapped accumulator layout. They enter divided by the
// factor the epilogue will apply (the dz storage scale, 1 for bf16), so that the epilogue's one
// multiply gives dW + factor * (this chunk's sum); a zero factor (a mean over no valid token)
// starts them at zero.
template <typename T>
__device__ __forceinline__ void load_dw_prev(const GemmArgs& g, u32x4 (&prev)[4][4][2], int mw, int nw, int lane) {
  const int half = lane >> 5;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = mw + 32 * i + (lane & 31);
    const T* o = (const T*)g.out + (size_t)row * g.ldo;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // N (the output pitch) is a multiple of 8: a 16-byte piece is all in or all out.
      const int c0 = nw + 32 * j + 8 * half;
      prev[i][j][0] = (row < g.M && c0 < g.N) ? *(const u32x4*)(o + c0) : (u32x4){};
      prev[i][j][1] = (row < g.M && c0 + 16 < g.N) ? *(const u32x4*)(o + c0 + 16) : (u32x4){};
    }
  }
}

template <typename T>
__device__ __forceinline__ void apply_dw_prev(f32x16 (&acc)[4][4], const u32x4 (&prev)[4][4][2], float inv_scale) {
  typedef T t4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const u32x4 lo = prev[i][j][0], hi = prev[i][j][1];
      // regroup32 left lo = (a0, a1, b0, b1), hi = (a2, a3, b2, b3) after its swap.
      uint32_t a[4] = {lo[0], lo[1], hi[0], hi[1]};
      uint32_t b[4] = {lo[2], lo[3], hi[2], hi[3]};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const auto r = __builtin_amdgcn_permlane32_swap(a[e], b[e], false, false);
        a[e] = r[0];
        b[e] = r[1];
      }
      // Now a = (q0, q2), b = (q1, q3): the lane's 4-element groups at 8q + 4 (l / 32).
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t* d = (q & 1) ? b : a;
        const t4 x = __builtin_bit_cast(t4, (u32x2){d[(q >> 1) * 2], d[(q >> 1) * 2 + 1]});
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float v = (float)x[e];
          acc[i][j][4 * q + e] = Storage<T>::kDzUnscaled ? v * inv_scale : v;
        }
      }
      // One block at a time: interleaved, the conversions' temporaries outgrow the registers.
      __builtin_amdgcn_sched_barrier(0);
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
// operand swap (LSE, STORE), accumulator element r of block (i, j) sits at row = 32i + 8(r/4) +
// 4(l/32) + r%4, col = 32j + l%32 of the sub-tile; with it (DW), at row = 32i + l%32,
// col = 32j + 8(r/4) + 4(l/32) + r%4.
// PRELOADED (DW): the accumulators started from the tile's current dW values.
template <typename T, int EPI, bool PRELOADED>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, f32x16 (&acc)[4][4], int mw, int nw, int split,
                                              bool accumulate, int n0, const char* refs_lds) {
  constexpr int kEsz = (int)sizeof(T);
  const int lane = lane_id();
  const int sub4 = 4 * (lane >> 5);
  const int l32 = lane & 31;
  if constexpr (EPI == EPI_LSE_FWD || EPI == EPI_LSE_BWD) {
    if (mw >= g.M) return;
    const int slice = mw / kLseSlice;
    const bool tref = EPI == EPI_LSE_BWD && g.ref != nullptr;
    // Each logit costs a few VALU instructions and an exponential here. Only the last tile row has
    // rows at or beyond M; every other wave runs the body without the per-value bound check (a
    // uniform branch), and each block's exponentials go from VGPRs straight to the e' store
    // instead of back through the accumulator registers.
    auto body = [&](auto full_c) {
      constexpr bool FULL = decltype(full_c)::value;
      auto inside = [&](int i, int r) { return FULL || mw + 32 * i + 8 * (r >> 2) + sub4 + (r & 3) < g.M; };
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int col = nw + 32 * j + l32;
        const bool in = col < g.N;
        float m_ref, ml, s = 0.f;
        if (tref) {
          // Target-referenced: the token's reference (the tile's references were copied to LDS
          // while the pipeline filled). A token without one (ignored, invalid label, padding) takes
          // +inf, so its e is exactly 0 and its partial sum 0: a backward call reports no lse, and
          // such a token's loss does not depend on it.
          const float ref = *(const float*)(refs_lds + 4 * (col - n0));
          const bool keep = in && __builtin_isfinite(ref);
          m_ref = keep ? ref : 0.f;
          ml = keep ? ref * kLog2e : INFINITY;
        } else {
          // The slice maximum as the reference.
          float mx = -INFINITY;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r)
              if (inside(i, r)) mx = fmaxf(mx, acc[i][j][r]);
          mx = fmaxf(mx, __shfl_xor(mx, 32));
          m_ref = mx;
          ml = mx * kLog2e;
        }
        // Every token block that holds a token of the chunk is written whole: target-referenced,
        // the lanes of tokens at or beyond N store zeros (the dW GEMM sums over the last block).
        // e blocked: the token is column l%32 of token block col/32, so this lane's piece of every
        // fragment of that block is at lane * 16; 32 ids fill the lane's pieces of two fragments.
        const bool store = EPI == EPI_LSE_BWD && nw + 32 * j < g.N;
        char* e_blk = (char*)g.out + (size_t)((nw + 32 * j) >> 5) * g.ldo * 1024 + lane * 16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          f32x16 ev;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float e = inside(i, r) ? __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], kLog2e, -ml)) : 0.f;
            s += e;
            ev[r] = e * Storage<T>::kE;
          }
          if constexpr (EPI == EPI_LSE_BWD) {
            if (store) {
              if constexpr (kEsz == 2) {
                // Whole 128-row wave slices: the blocked rows cover M rounded up to 256, and rows
                // at or beyond M hold exp = 0 here.
                store_frag32<T>(e_blk + (size_t)((mw + 32 * i) >> 4) * 1024, ev);
              } else {
                // fp32: a K-pair is 8 ids, half of it per lane half. The dH GEMM reads every K-pair
                // that holds an id below M whole, so such a K-pair is stored whole: its ids at or
                // beyond M hold exp = 0 here, and nothing stale from the workspace reaches it.
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                  const int kp_row = mw + 32 * i + 8 * q;
                  if (FULL || kp_row < g.M)
                    store4((T*)(e_blk + (size_t)(kp_row >> 3) * 1024), ev[4 * q], ev[4 * q + 1], ev[4 * q + 2],
                           ev[4 * q + 3]);
                }
              }
            }
          }
        }
        s += __shfl_xor(s, 32);
        if (in && lane < 32) {
          g.pmax[(size_t)slice * g.ldp + col] = m_ref;
          g.psum[(size_t)slice * g.ldp + col] = s;
        }
      }
    };
    if (mw + 128 <= g.M) body(std::true_type{});
    else body(std::false_type{});
  } else if constexpr (EPI == EPI_STORE) {
    // C^T token-major: column n = nw + 32j + l%32 of C is row n of the output, and the lane's four
    // consecutive rows of C per (i, q) are four consecutive elements of it. M (the output's row
    // length) is a multiple of 8 for 16-bit types and of 4 for fp32, so pieces are all in or out.
    // mode 1: fp32 partials, split s at out + s * N * ldo.
    const float sc = dz_epilogue_scale<T>(g.n_valid, g.mean);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = nw + 32 * j + l32;
      if (col >= g.N) continue;
      if (g.col_scale) {
        const float cs = g.col_scale[col];
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i][j] *= cs;
      }
      if (g.mode == 1) {
        float* o = (float*)g.out + ((size_t)split * g.N + col) * g.ldo;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int row = mw + 32 * i + 8 * q + sub4;
            if (row < g.M)
              store4(o + row, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
          }
      } else {
        T* o = (T*)g.out + (size_t)col * g.ldo;
        if constexpr (kEsz == 2) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            if constexpr (Storage<T>::kDzUnscaled) acc[i][j] *= sc;
            const int r0 = mw + 32 * i + 8 * (lane >> 5);
            store_row32(o + mw + 32 * i, acc[i][j], r0 < g.M, r0 + 16 < g.M);
          }
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const int row = mw + 32 * i + 8 * q + sub4;
              if (row < g.M)
                store4(o + row, acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
            }
        }
      }
    }
  } else {
    // DW, swapped layout: lane owns rows mw + 32i + l%32 and 4 consecutive columns per (j, q).
    // N (the output pitch) is a multiple of 4 here, so a 4-column group is all in or all out.
    const float sc = dz_epilogue_scale<T>(g.n_valid, g.mean);
    if (g.mode >= DW_ACC32_FIRST) {
      // fp32 cross-chunk accumulator: acc32 (+)= sc * C, or at the last chunk dW = acc32 + sc * C
      // rounded once. A block's four 16-byte pieces are requested together before any is used.
      const bool read = g.mode != DW_ACC32_FIRST, last = g.mode == DW_ACC32_LAST;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int row = mw + 32 * i + l32;
        if (row >= g.M) continue;
        float* a = g.acc32 + (size_t)row * g.ldo;
        T* o = (T*)g.out + (size_t)row * g.ldo;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          f32x4 base[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = nw + 32 * j + 8 * q + sub4;
            base[q] = (read && col < g.N) ? *(const f32x4*)(a + col) : (f32x4){};
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int col = nw + 32 * j + 8 * q + sub4;
            if (col >= g.N) continue;
            const f32x4 v = base[q] + sc * (f32x4){acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                                   acc[i][j][4 * q + 3]};
            if (last) store4(o + col, v[0], v[1], v[2], v[3]);
            else store4(a + col, v[0], v[1], v[2], v[3]);
          }
        }
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = mw + 32 * i + l32;
      if (row >= g.M) continue;
      if constexpr (PRELOADED) {  // EPI_DW, 16-bit: the accumulators already hold the earlier chunks' sum
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

// ---- The main loop: operand B straight to registers -------------------------------------------
//
// gemm_xb_kernel reads operand B from its fragment-blocked layout straight into the registers the
// MFMAs take it from: every B load is one whole 1 KB fragment, and B never passes through LDS, so
// a K-tile's LDS traffic is A's alone (32 KB written, 64 KB read). A streams into a ring of four
// LDS slots by LDS-DMA, three K-tiles ahead; B circulates through a ring of eight K-pairs of
// fragments (128 VGPRs), seven K-pairs ahead. A K-tile is four sections of 16 MFMAs; each section
// issues one quarter of A's K-tile three ahead (two LDS-DMA loads) and the four B fragments of the
// K-pair seven ahead, between its MFMAs.
//
// Blocked layout (N columns, reduction K, element type T): fragment (jb, q) -- 32 columns by
// K-pair q, the q-th 32 bytes of every column's K run -- is 1 KB at byte (jb KP + q) 1024, and lane
// l of it holds column 32 jb + l%32, bytes [32 q + 16 (l/32), +16): the 16 bytes that lane feeds
// the MFMA. KP counts the K-pairs per column block with K rounded up to a whole K-tile at least;
// columns at or beyond N and K at or beyond K are zeros. (The A fragments read from LDS cover the
// same K bytes: K-pair p of K-tile t, lane half h, bytes [32 p + 16 h, +16) of the K-tile.)
constexpr int kXbASlots = 4;
constexpr int kXbAhead = kXbASlots - 1;
// The A ring, then 1 KB for the tile's 256 per-token references (target-referenced LSE_BWD).
constexpr int kXbRefs = kXbASlots * kOperandBytes;
constexpr int kXbSmem = kXbRefs + 1024;  // 129 KB

// Blocked copy of a K-contiguous source (element (n, k) at src[n * ld + k]; K a multiple of 16
// bytes' worth): one thread per 16-byte piece, block b of 256 threads taking pieces 256 b ..
// 256 b + 255. Blocks: ceil(NB * KP * 64 / 256).
template <typename T>
__device__ __forceinline__ void block_k_block(int64_t b, const T* __restrict__ src, int64_t ld, int N, int K,
                                              int KP, int NB, T* __restrict__ dst) {
  const int64_t t = b * 256 + threadIdx.x;
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
// columns in LDS, then each thread gathers one 16-byte piece down a column. Blocks: NB x
// ceil(KP / 4). row_scale (nullptr = none): K row k is multiplied by row_scale[k] on the way
// (rounded once to T).
template <typename T>
__device__ __forceinline__ void block_mn_block(int jb, int grp, const T* __restrict__ src, int64_t ld, int N, int K,
                                               int KP, T* __restrict__ dst, const float* __restrict__ row_scale) {
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kVec = 16 / kEsz;            // elements per piece
  constexpr int kRows = 128 / kEsz;          // K rows of four K-pairs
  constexpr int kPieces = 32 / kVec;         // pieces per K row of 32 columns
  static_assert(kRows * kPieces == 256, "one piece per thread");
  typedef T vec_t __attribute__((ext_vector_type(kVec)));
  __shared__ __attribute__((aligned(16))) T tile[kRows][32];
  const int t = threadIdx.x;
  {
    const int r = t / kPieces, pc = t % kPieces;
    const int k = grp * kRows + r, n = 32 * jb + pc * kVec;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (k < K && n < N) {
      v = *(const u32x4*)(src + (size_t)k * ld + n);
      if (row_scale != nullptr) {
        const float c = row_scale[k];
        vec_t x = __builtin_bit_cast(vec_t, v);
#pragma unroll
        for (int e = 0; e < kVec; ++e) x[e] = (T)((float)x[e] * c);
        v = __builtin_bit_cast(u32x4, x);
      }
    }
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

// g.A: operand A in layout AL (ALayout); g.B: operand B blocked, g.ldb its KP. KCHECK: a K-contig
// A checks every chunk against the K range (see Operand::offset). Splits must start at whole
// K-tiles (k_per_split).
template <typename T, int EPI, int AL, bool KCHECK>
__device__ __forceinline__ void gemm_xb_tile(const GemmArgs& g, int bid, char* smem) {
  constexpr int kEsz = (int)sizeof(T);
  constexpr int kBK = kTileBytes / kEsz;
  constexpr bool kSwap = EPI == EPI_DW;
  constexpr bool kAmn = AL != A_K;  // MN-contig LDS layout (MN-contig or blocked A)

  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;

  const int total = g.tiles_m * g.tiles_n * g.splits;
  int tm, rest;
  tile_coords(bid, total, g.tiles_m, g.group_m, tm, rest);
  tm = __builtin_amdgcn_readfirstlane(tm);
  rest = __builtin_amdgcn_readfirstlane(rest);
  const int tn = rest % g.tiles_n;
  const int split = rest / g.tiles_n;
  const int m0 = tm * kTile, n0 = tn * kTile;
  const int kb = split * g.k_per_split;
  const int ke = min(g.K, kb + g.k_per_split);

  Operand<T, AL> opa;
  opa.init(g.A, g.lda, m0, min(kTile, g.M - m0), kb, ke, w, lane, wm * 128);
  const int khalf = lane >> 5;
  int swi[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) swi[i] = swz_k(i * 32 + (lane & 31));

  // B: this wave's four column blocks start at jb0 (the descriptor's base; blocks at or beyond
  // NB read zeros); K-pair q of this split is fragment q0 + q of a block.
  const int KP = (int)g.ldb;
  const int NB = (g.N + 31) >> 5;
  const int jb0 = (n0 + wn * 128) >> 5;
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(
      (const void*)uniform64((uint64_t)((const char*)g.B + (size_t)jb0 * KP * 1024)),
      __builtin_amdgcn_readfirstlane((uint32_t)max(0, min(4, NB - jb0)) * (uint32_t)KP * 1024u));
  const uint32_t bvoff = (uint32_t)lane * 16u;
  const int q0 = kb * kEsz / 32;
  const int qend = ((ke - kb) * kEsz + 31) / 32;

  uint32_t aoff[8];  // per-lane parts of the eight loads of an A K-tile
#pragma unroll
  for (int j = 0; j < 8; ++j) aoff[j] = opa.lane_offset(j);
  // Quarter pc of A K-tile t (loads 2 pc, 2 pc + 1) into ring slot t % 4.
  auto load_a_q = [&](int t, auto pc) {
    constexpr int pq = decltype(pc)::value;
    const __amdgpu_buffer_rsrc_t r = opa.rsrc(t);
    char* st = smem + (t & (kXbASlots - 1)) * kOperandBytes + w * 8 * 1024;
#pragma unroll
    for (int j = 2 * pq; j < 2 * pq + 2; ++j) {
      if constexpr (KCHECK && AL == A_K) dma16(r, st + j * 1024, opa.offset(t, j));
      else dma16(r, st + j * 1024, aoff[j], opa.uniform_offset(t, j));
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
      const uint32_t so = q < qend ? (uint32_t)(j * KP + q0 + q) * 1024u : kOOB;
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
  // 16-bit MN-contig / blocked A: reads through the address registers. NEXT: the pair of slots after
  // the current one (the addresses moved by pair_delta for these reads only).
  constexpr bool kXread = Operand<T, AL>::kXa > 0;
  int pair_delta = 2 * kOperandBytes;  // current pair 0-1: the next is 2 slots up, then down
  if constexpr (kXread) opa.init_xa((uint32_t)(uintptr_t)(lds_void*)smem);
  auto read_frags_x = [&](auto sip, auto kpr, auto next, int buf) {
    constexpr int SIP = decltype(sip)::value, KPR = decltype(kpr)::value;
    if constexpr (decltype(next)::value) {
      uint32_t a[Operand<T, AL>::kXa > 0 ? Operand<T, AL>::kXa : 1];
#pragma unroll
      for (int k = 0; k < Operand<T, AL>::kXa; ++k) a[k] = opa.xa[k] + (uint32_t)pair_delta;
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[buf][i] = Operand<T, AL>::template fragment_x<SIP, KPR>(a, i);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) fa[buf][i] = Operand<T, AL>::template fragment_x<SIP, KPR>(opa.xa, i);
    }
  };
  // Fragment reads issued as inline assembly are invisible to the compiler's wait insertion: at
  // the start of each section wait for all earlier LDS traffic (the previous section's reads, long
  // since done), with the fragment registers as operands so that no MFMA moves above the wait.
  auto sync_frags = [&]() {
    if constexpr (kAmn && kEsz == 2) {
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
  constexpr int kReads = kAmn ? 0 : 4;  // compiler-visible LDS reads per section
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
    if constexpr (kXread) {
      // Section s reads K-tile kt + s/4 (slot s/4 of the current pair), or at p == 3 the next
      // K-tile: kt + 1 (slot 1) from section 3, kt + 2 (slot 0 of the next pair) from section 7.
      using I = std::integral_constant<int, 0>;
      using One = std::integral_constant<int, 1>;
      if constexpr (s == 3) read_frags_x(One{}, I{}, std::false_type{}, (s + 1) & 1);
      else if constexpr (s == 7) read_frags_x(I{}, I{}, std::true_type{}, (s + 1) & 1);
      else read_frags_x(std::integral_constant<int, (s >> 2)>{}, std::integral_constant<int, p + 1>{},
                        std::false_type{}, (s + 1) & 1);
    } else {
      if constexpr (p == 3) read_frags(ktp + 1, 0, (s + 1) & 1);
      else read_frags(ktp, p + 1, (s + 1) & 1);
    }
    // Loads retire in issue order, so a B load waits for every A load issued before it. With A
    // K-contiguous (W, streamed from HBM) the section issues its B fragments first (measured 4%
    // faster on the logits GEMM); with A MN-contiguous (dZ^T) the order made no difference.
    if constexpr (!kAmn) {
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

  // 16-bit dW accumulation (chunks after the first): the tile's current dW values are loaded here,
  // raw, in flight together with the loads that fill the pipeline, and become the accumulators'
  // starting values, so the epilogue only stores. (fp32 adds them in the epilogue instead: its
  // 256 values per lane would not fit next to the pipeline's registers.)
  const int mw = m0 + wm * 128, nw = n0 + wn * 128;
  constexpr bool kPreload = EPI == EPI_DW && kEsz == 2;
  const bool accumulate = EPI == EPI_DW && g.mode == DW_ACCUMULATE;
  u32x4 prev[kPreload ? 4 : 1][4][2];
  if constexpr (kPreload) {
    if (accumulate) load_dw_prev<T>(g, prev, mw, nw, lane);
  }
  // An odd count runs one more K-tile of zeros (past the end every load reads zeros).
  const int nk = (ke - kb + kBK - 1) / kBK;
  // Target-referenced LSE_BWD: the tile's 256 references into LDS, one LDS-DMA load issued before
  // the prologue's (so that none of its hand-counted waits counts it); past N it reads zeros. The
  // first barrier of the main loop comes after this wave's wait for it.
  const bool tref = EPI == EPI_LSE_BWD && g.ref != nullptr;
  if (tref && w == 0) {
    const __amdgpu_buffer_rsrc_t rr = make_rsrc((const void*)uniform64((uint64_t)(g.ref + n0)),
                                                __builtin_amdgcn_readfirstlane((uint32_t)max(0, g.N - n0) * 4u));
    dma16(rr, smem + kXbRefs, (uint32_t)lane * 16u);
  }
  if (nk > 0) {
    // Prologue: A(0 .. ahead-1), then B(0 .. 6). A(0) has landed for every wave (issued after it:
    // the other A K-tiles and 28 B loads) before its first fragments are read; the first waits at
    // p == 3 find at least as many loads after A(1), A(2) as they allow. The dW values (128 VGPRs
    // raw) become accumulators before the rest of B's ring fills the registers: bf16's once the
    // first three K-pairs of B are on their way, fp16's before any.
#pragma unroll
    for (int t = 0; t < kXbAhead; ++t) load_a(t);
    // fp16's values are also scaled as they enter: its temporaries fit only before B's ring fills.
    if constexpr (kPreload && Storage<T>::kDzUnscaled) {
      if (accumulate) apply_dw_prev<T>(acc, prev, dw_prev_scale<T>(g));
    }
    load_b(0, std::integral_constant<int, 0>{});
    load_b(1, std::integral_constant<int, 1>{});
    load_b(2, std::integral_constant<int, 2>{});
    if constexpr (kPreload && !Storage<T>::kDzUnscaled) {
      if (accumulate) apply_dw_prev<T>(acc, prev, dw_prev_scale<T>(g));
    }
    load_b(3, std::integral_constant<int, 3>{});
    load_b(4, std::integral_constant<int, 4>{});
    load_b(5, std::integral_constant<int, 5>{});
    load_b(6, std::integral_constant<int, 6>{});
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(8 * (kXbAhead - 1) + 28) : "memory");
    if constexpr (kXread) {
      read_frags_x(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{}, std::false_type{}, 0);
    } else {
      read_frags(0, 0, 0);
    }
    for (int kt = 0; kt < nk; kt += 2) {
      section(kt, std::integral_constant<int, 0>{});
      section(kt, std::integral_constant<int, 1>{});
      section(kt, std::integral_constant<int, 2>{});
      section(kt, std::integral_constant<int, 3>{});
      section(kt, std::integral_constant<int, 4>{});
      section(kt, std::integral_constant<int, 5>{});
      section(kt, std::integral_constant<int, 6>{});
      section(kt, std::integral_constant<int, 7>{});
      if constexpr (kXread) {
        opa.shift_xa(pair_delta);
        pair_delta = -pair_delta;
      }
    }
    // Loads past the end may still be in flight (they target no memory); their LDS and registers
    // must not be reused before they retire.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  gemm_epilogue<T, EPI, kPreload>(g, acc, mw, nw, split, accumulate, n0, smem + kXbRefs);
}

// One 256 x 256 tile per workgroup. With g.run_if set, the whole grid does nothing unless
// *g.run_if is nonzero: work that a flag set on the device may or may not ask for.
template <typename T, int EPI, int AL, bool KCHECK>
__global__ __launch_bounds__(kGemmThreads, 1) void gemm_xb_kernel(const GemmArgs g) {
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  if (g.run_if != nullptr && __builtin_amdgcn_readfirstlane(*g.run_if) == 0) return;
  gemm_xb_tile<T, EPI, AL, KCHECK>(g, blockIdx.x, smem);
}

}  // namespace lce
