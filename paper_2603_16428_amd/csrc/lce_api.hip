// C ABI of the fused linear + cross-entropy step: argument checks, workspace plan, chunk loop.
//
// Per call (Section 3.3, "Optimized Triton Kernels": projection fused with the loss, gradients in
// token chunks, the N x V logits never held):
//   count valid labels (global mean divisor) -> target logits
//   for each chunk of n_c tokens:
//     fragment-blocked copies of X_c (operand B of the logits and dW GEMMs)
//     logits^T tile GEMM with the log-sum-exp epilogue  (stores e = exp(z - m_slice) for backward,
//                                                       fragment-blocked)
//     row combine -> lse, token losses
//     [backward] dlogits in place -> dH rows GEMM (dH^T = W^T dZ^T: reads W as it is) -> dW GEMM
//                (reads the blocked dZ as it is; the first chunk writes dW, later chunks add to it)
//   loss reduction (fp64, fixed order)
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "lce.h"
#include "lce_aux.hpp"
#include "lce_gemm.hpp"

// Scratch memory of lce_forward_no_alloc: the workspace of a forward call, in a static device array
// that every device the library runs on holds (its own copy, at its own address) until the process
// ends. Host code never passes this name to a kernel: the name is a host-side stand-in, and the
// device address comes from hipGetSymbolAddress (lce::no_alloc_scratch below).
static __device__ __align__(256) char scratch[LCE_NO_ALLOC_SCRATCH_BYTES];

namespace lce {
namespace {

constexpr int64_t kAlign = 256;
constexpr int kMaxDevices = 64;

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// ---- optional per-kernel timing (events on the launch stream) ----
enum TimingKind { T_LOGITS = 0, T_DH = 1, T_DW = 2, T_DLOGITS = 3, T_OTHER = 5, T_KINDS = 6 };
struct TimedLaunch {
  int kind;
  hipEvent_t start, stop;
};
std::mutex g_timing_mu;
bool g_timing_on = false;
std::vector<TimedLaunch> g_timed;

// Brackets the launches made during its lifetime with events when timing is enabled.
class KernelTimer {
 public:
  KernelTimer(int kind, hipStream_t s) : kind_(kind), s_(s) {
    std::lock_guard<std::mutex> lk(g_timing_mu);
    if (!g_timing_on) return;
    if (hipEventCreate(&start_) != hipSuccess) return;
    if (hipEventCreate(&stop_) != hipSuccess) { (void)hipEventDestroy(start_); return; }
    active_ = hipEventRecord(start_, s_) == hipSuccess;
  }
  ~KernelTimer() {
    if (!active_) return;
    std::lock_guard<std::mutex> lk(g_timing_mu);
    if (hipEventRecord(stop_, s_) == hipSuccess) {
      g_timed.push_back({kind_, start_, stop_});
    } else {
      (void)hipEventDestroy(start_);
      (void)hipEventDestroy(stop_);
    }
  }

 private:
  int kind_;
  hipStream_t s_;
  hipEvent_t start_ = nullptr, stop_ = nullptr;
  bool active_ = false;
};
int64_t cdiv(int64_t x, int64_t m) { return (x + m - 1) / m; }

// The device address of `scratch` on the current device, looked up on the first call per device
// (with that device current) and kept.
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

lce_status_t no_alloc_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LCE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LCE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return LCE_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return LCE_OK;
}

struct Plan {
  int64_t N = 0, H = 0, V = 0;
  int esz = 0, dtype = 0;
  bool backward = false;
  // Backward with target-referenced e (bf16, fp32): the logits epilogue stores exp(z - z_target),
  // combine folds the one-hot term into e and leaves a per-token factor for the dH epilogue and
  // the dW operand, and no dlogits pass runs unless a chunk's flag asks for the slice-maximum
  // path. fp16 (whose exponent range cannot hold exp(z - z_target)) keeps the dlogits pass.
  bool tref = false;
  int64_t nc = 0, chunks = 0;     // tokens per chunk, number of chunks
  int64_t ncp = 0;                // tokens per chunk rounded up to 64
  int64_t slices = 0;
  int dh_splits = 1;
  int64_t dh_kps = 0;             // K (vocabulary) per dH split, multiple of the K-tile
  // dW's running sum over chunks in an fp32 accumulator instead of dW's own 16-bit type (more
  // chunks than carry_chunks() allows for the type).
  bool dw_acc32 = false;
  // Fragment-blocked copies of a chunk's X: operand B of the logits GEMM (columns = tokens,
  // K = H) and of the dW GEMM (columns = H, K = tokens): column blocks and K-pairs per block.
  int64_t xk_nb = 0, xk_kp = 0, xm_nb = 0, xm_kp = 0;
  // e / dZ of a chunk, blocked (columns = tokens, K = vocabulary rounded up to the tile): operand
  // B of the dH GEMM and blocked operand A of the dW GEMM.
  int64_t ez_nb = 0, ez_kp = 0;
  // workspace offsets (bytes)
  size_t o_nvalid = 0, o_tgt = 0, o_lse = 0, o_tl = 0, o_pmax = 0, o_psum = 0, o_e = 0, o_dhp = 0;
  size_t o_scale = 0, o_flags = 0, o_ref = 0, o_acc32 = 0;
  size_t o_xk = 0, o_xm = 0;
  size_t total = 0;
};

int num_cus() {
  static std::atomic<int> cached{0};
  int c = cached.load();
  if (c > 0) return c;
  int dev = 0;
  hipDeviceProp_t p;
  if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&p, dev) == hipSuccess &&
      p.multiProcessorCount > 0) {
    c = p.multiProcessorCount;
  } else {
    c = 256;
  }
  cached.store(c);
  return c;
}

constexpr int64_t kFwdChunk = 16384;  // automatic forward chunk (a multiple of 64)

// Chunks up to which dW's running sum may be carried in dW's own 16-bit type. Each boundary
// between chunks rounds the running sum once (relative error at most the unit roundoff u, on a
// partial sum of about the size of the final one), so c chunks add at most (c - 1) u; with the
// rounding of e' and of the output (2 u) the total stays within the gradient bar of the type
// (bf16: 2e-2 = 5.1 u with u = 2^-8, so c <= 4; fp16: 5e-3 = 10.2 u with u = 2^-11, so c <= 9).
// Beyond it the sum is carried in an fp32 accumulator of V x H in the workspace.
int carry_chunks(int esz, int dtype) { return esz == 4 ? 0 : dtype == LCE_DTYPE_BF16 ? 4 : 9; }

int64_t auto_chunk(int64_t N, int64_t H) {
  const int64_t half = cdiv(N, 2);
  int64_t nc = std::min(H, half) / 64 * 64;
  return std::max<int64_t>(64, nc);
}

bool dtype_ok(int dtype) { return dtype == LCE_DTYPE_FP32 || dtype == LCE_DTYPE_BF16 || dtype == LCE_DTYPE_FP16; }

// Fills `p`; returns LCE_OK or the status that the sizes deserve.
// dx_f32: the caller wants d loss / d hidden in fp32 (through the split-K partials even with one
// split), as the RMSNorm variant does.
lce_status_t make_plan(int64_t N, int64_t H, int64_t V, int dtype, bool backward, int64_t chunk_tokens,
                       Plan& p, bool query_device, bool dx_f32 = false) {
  if (N < 1 || H < 1 || V < 1 || !dtype_ok(dtype) || chunk_tokens < 0) return LCE_ERR_INVALID_ARGUMENT;
  p.N = N; p.H = H; p.V = V;
  p.esz = dtype == LCE_DTYPE_FP32 ? 4 : 2;
  p.backward = backward;
  p.dtype = dtype;
  p.tref = backward && dtype != LCE_DTYPE_FP16;
  if (H % (16 / p.esz) != 0) return LCE_ERR_UNSUPPORTED;
  // Automatic chunks: a training step keeps one chunk's e/dZ, so its chunks stay small; a forward
  // call keeps only per-slice partials (N V / 16 bytes), so it takes up to 16384 tokens at once
  // (one launch of the logits GEMM instead of several, each with a partly empty last wave).
  int64_t nc = chunk_tokens != 0 ? chunk_tokens
               : backward      ? auto_chunk(N, H)
               : N <= kFwdChunk ? N
                                : std::max(auto_chunk(N, H), kFwdChunk);
  // An automatic backward chunk grows, when that keeps the chunk count within the type's carry
  // limit, up to 2 H tokens: its e buffer then grows by less than the fp32 accumulator (V x H x 4
  // bytes) it makes unnecessary.
  if (chunk_tokens == 0 && backward) {
    const int lim = carry_chunks(p.esz, dtype);
    if (lim > 0 && cdiv(N, nc) > lim) {
      const int64_t grown = round_up(cdiv(N, lim), 64);
      if (grown <= 2 * H) nc = grown;
    }
  }
  if (nc >= N) nc = N;
  else if (nc % 64 != 0) return LCE_ERR_INVALID_ARGUMENT;
  p.nc = nc;
  p.chunks = cdiv(N, nc);
  p.ncp = round_up(nc, 64);
  p.slices = cdiv(V, kLseSlice);
  // 32-bit limits: buffer ranges of one 256-row operand slice (and of four column blocks of a
  // blocked operand), and int tile/element indices.
  const int64_t lim = (int64_t(1) << 31) - 1;
  const int64_t maxpitch = std::max({H, round_up(V, kTile)});
  if ((int64_t)kTile * maxpitch * p.esz > lim || N > lim / 2 || V > lim / 2 || H > lim / 2) return LCE_ERR_UNSUPPORTED;
  if (cdiv(V, kTile) * cdiv(H, kTile) > lim / 16) return LCE_ERR_UNSUPPORTED;
  p.xk_nb = cdiv(p.ncp, 32);
  p.xk_kp = round_up(H * p.esz, kTileBytes) / 32;
  p.xm_nb = cdiv(H, 32);
  p.xm_kp = round_up(p.ncp * p.esz, kTileBytes) / 32;
  if (p.xk_nb * p.xk_kp * 1024 > lim || p.xm_nb * p.xm_kp * 1024 > lim) return LCE_ERR_UNSUPPORTED;
  p.ez_nb = p.ncp / 32;
  p.ez_kp = round_up(V, kTile) * p.esz / 32;

  if (backward) {
    // dH tiles of one chunk: split the vocabulary (K) so that the grid fills the device.
    const int64_t tiles = cdiv(nc, kTile) * cdiv(H, kTile);
    const int cus = query_device ? num_cus() : 256;
    const int64_t kbk = kTileBytes / p.esz;
    const int64_t kblocks = cdiv(V, kbk);
    double best = 1e30;
    int best_s = 1;
    for (int s = 1; s <= 8; ++s) {
      if (s > kblocks) break;
      const double waves = (double)cdiv(tiles * s, cus);
      const double cost = waves / s + (s > 1 ? 0.03 * s : 0.0);
      if (cost < best - 1e-9) { best = cost; best_s = s; }
    }
    p.dh_splits = best_s;
    p.dh_kps = cdiv(kblocks, best_s) * kbk;
    p.dw_acc32 = p.esz == 2 && p.chunks > carry_chunks(p.esz, dtype);
  }

  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (size_t)round_up((int64_t)bytes, kAlign);
    return o;
  };
  p.o_nvalid = take(64);
  p.o_tgt = take((size_t)N * 4);
  p.o_lse = take((size_t)N * 4);
  p.o_tl = take((size_t)N * 4);
  p.o_pmax = take((size_t)p.slices * p.ncp * 4);
  p.o_psum = take((size_t)p.slices * p.ncp * 4);
  p.o_xk = take((size_t)(p.xk_nb * p.xk_kp * 1024));
  if (backward) {
    p.o_xm = take((size_t)(p.xm_nb * p.xm_kp * 1024));
    p.o_e = take((size_t)(p.ez_nb * p.ez_kp * 1024));
    p.o_scale = take((size_t)N * 4);
    p.o_ref = take((size_t)N * 4);  // used by target-referenced plans (kept for all: one layout per element size)
    p.o_flags = take((size_t)p.chunks * 4);
    if (p.dh_splits > 1 || dx_f32) p.o_dhp = take((size_t)p.dh_splits * p.nc * H * 4);
    if (p.dw_acc32) p.o_acc32 = take((size_t)V * H * 4);
  }
  p.total = off;
  return LCE_OK;
}

// The forward plan of lce_forward_no_alloc: the automatic chunk if it is valid and its workspace
// fits the static scratch, else the largest multiple of 64 tokens below it that is and does (both
// the workspace and the 32-bit limits of make_plan grow with the chunk, so a binary search finds
// it). An error at 64 tokens per chunk does not depend on the chunk and is returned as it is;
// LCE_ERR_WORKSPACE_TOO_SMALL when 64 tokens per chunk are valid but do not fit.
lce_status_t make_no_alloc_plan(int64_t N, int64_t H, int64_t V, int dtype, Plan& p) {
  const size_t cap = (size_t)LCE_NO_ALLOC_SCRATCH_BYTES;
  lce_status_t st = make_plan(N, H, V, dtype, false, 0, p, true);
  if (st == LCE_OK && p.total <= cap) return LCE_OK;
  const int64_t top = st == LCE_OK ? p.nc : N;
  Plan q;
  st = make_plan(N, H, V, dtype, false, 64, q, true);
  if (st != LCE_OK) return st;
  if (q.total > cap) return LCE_ERR_WORKSPACE_TOO_SMALL;
  int64_t lo = 1, hi = (top - 1) / 64;  // chunks of 64 lo tokens are valid and fit
  while (lo < hi) {
    const int64_t mid = (lo + hi + 1) / 2;
    if (make_plan(N, H, V, dtype, false, mid * 64, q, true) == LCE_OK && q.total <= cap) lo = mid;
    else hi = mid - 1;
  }
  return make_plan(N, H, V, dtype, false, lo * 64, p, true);
}

// AL: operand A's layout (ALayout); operand B is blocked. KCHECK: a K-contig A's K range may end
// inside a K-tile and its rows are not zero-padded up to the next one (see Operand::offset).
template <typename T, int EPI, int AL, bool KCHECK = false>
hipError_t launch_gemm(GemmArgs g, hipStream_t s) {
  const void* fn = (const void*)gemm_xb_kernel<T, EPI, AL, KCHECK>;
  static std::atomic<uint64_t> configured[kMaxDevices / 64 + 1];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < kMaxDevices) {
    const uint64_t bit = uint64_t(1) << (dev & 63);
    if (!(configured[dev >> 6].load() & bit)) {
      e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, kXbSmem);
      if (e != hipSuccess) return e;
      configured[dev >> 6].fetch_or(bit);
    }
  }
  g.tiles_m = (int)cdiv(g.M, kTile);
  g.tiles_n = (int)cdiv(g.N, kTile);
  const int blocks = g.tiles_m * g.tiles_n * g.splits;
  if (blocks <= 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_xb_kernel<T, EPI, AL, KCHECK>), dim3(blocks), dim3(kGemmThreads), kXbSmem, s, g);
  return hipGetLastError();
}

// Optional events for a caller that streams dW out as it is produced: the last chunk's dW GEMM runs
// as `blocks` launches over consecutive ranges of vocabulary rows (multiples of the tile), each
// followed by dw_done[b]; dh_done is recorded after the last chunk's dH (W is not read after it).
struct DwBlocks {
  int blocks = 0;
  hipEvent_t* dw_done = nullptr;
  int64_t* row0 = nullptr;     // [blocks + 1] row boundaries, filled by run
  hipEvent_t dh_done = nullptr;
};

// dx32 (optional): receives d loss / d hidden in fp32 instead of dH (the plan must have dx_f32).
template <typename T>
lce_status_t run(const Plan& p, const T* X, const T* W, const int64_t* y, int64_t ignore_index, int reduction,
                 float* loss, float* lse_user, T* dH, T* dW, char* ws, hipStream_t s, float* dx32 = nullptr,
                 DwBlocks* hook = nullptr) {
  const int64_t N = p.N, H = p.H, V = p.V;
  int* nvalid = (int*)(ws + p.o_nvalid);
  float* tgt = (float*)(ws + p.o_tgt);
  float* lse = lse_user ? lse_user : (float*)(ws + p.o_lse);
  float* tl = (reduction == LCE_REDUCTION_NONE) ? loss : (float*)(ws + p.o_tl);
  float* pmax = (float*)(ws + p.o_pmax);
  float* psum = (float*)(ws + p.o_psum);
  T* ez = p.backward ? (T*)(ws + p.o_e) : nullptr;
  T* xk = (T*)(ws + p.o_xk);
  T* xm = p.backward ? (T*)(ws + p.o_xm) : nullptr;
  float* dhp = (p.backward && (p.dh_splits > 1 || dx32)) ? (float*)(ws + p.o_dhp) : nullptr;
  float* scale = p.backward ? (float*)(ws + p.o_scale) : nullptr;
  float* tref = p.tref ? (float*)(ws + p.o_ref) : nullptr;
  int* flags = p.backward ? (int*)(ws + p.o_flags) : nullptr;
  float* acc32 = p.dw_acc32 ? (float*)(ws + p.o_acc32) : nullptr;
  const int mean = reduction == LCE_REDUCTION_MEAN;

  // Small bandwidth-bound jobs share launches (aux_kernel): each launch boundary costs ~10 us of
  // the step. The fragment-blocked copies of X_c: operand B of the logits GEMM (block_k) and,
  // backward, of the dW GEMM (block_mn; target-referenced: scaled per token, so made once the
  // factors are known).
  auto bk_job = [&](AuxJobs& j, int64_t c) {
    const int64_t t0 = c * p.nc;
    j.bk_blocks = cdiv(p.xk_nb * p.xk_kp * 64, 256);
    j.bk = BlockKJob{X + t0 * H, H, (int)std::min(p.nc, N - t0), (int)H, (int)p.xk_kp, (int)p.xk_nb, xk};
  };
  auto bmn_job = [&](AuxJobs& j, int64_t c, const float* row_scale) {
    const int64_t t0 = c * p.nc;
    j.bmn_blocks = p.xm_nb * cdiv(p.xm_kp, 4);
    j.bmn = BlockMnJob{X + t0 * H, H, (int)H, (int)std::min(p.nc, N - t0), (int)p.xm_kp, (int)p.xm_nb, xm,
                       row_scale};
  };
  auto dl_job = [&](AuxJobs& j, int64_t c, const int* run_if, int64_t blocks) {
    const int64_t t0 = c * p.nc;
    j.dl_blocks = blocks;
    j.dl = DlogitsJob{ez, p.ez_kp, p.ez_nb, pmax, p.ncp, lse + t0, y + t0, ignore_index, nvalid, mean,
                      (int)std::min(p.nc, N - t0), (int)V, run_if};
  };
  // The call's loss (reduction mean or sum): one block, in a launch after the last combine_kernel.
  auto loss_job = [&](AuxJobs& j) {
    if (reduction == LCE_REDUCTION_NONE) return;
    j.loss_blocks = 1;
    j.ls = LossJob{tl, N, nvalid, mean, loss};
  };
  auto aux = [&](const AuxJobs& j, TimingKind kind) {
    KernelTimer t(kind, s);
    const int64_t blocks = j.prep_blocks + j.bk_blocks + j.bmn_blocks + j.dl_blocks + j.loss_blocks;
    hipLaunchKernelGGL((aux_kernel<T>), dim3((unsigned)blocks), dim3(256), 0, s, j);
    return hipGetLastError();
  };
  {
    // prepare (target logits, references, n_valid, flags) and chunk 0's copies.
    AuxJobs j{};
    j.prep_blocks = cdiv(N, 4) + 1;
    j.prep = PrepareJob{X, W, y, N, H, V, ignore_index, tgt, tref, nvalid, flags, (int64_t)(flags ? p.chunks : 0)};
    bk_job(j, 0);
    if (p.backward && !p.tref) bmn_job(j, 0, nullptr);
    if (aux(j, T_OTHER) != hipSuccess) return LCE_ERR_HIP;
  }
  bool bk_ready = true;  // X_c's block_k copy was made by an earlier launch

  for (int64_t c = 0; c < p.chunks; ++c) {
    const int64_t t0 = c * p.nc;
    const int rows = (int)std::min(p.nc, N - t0);
    const bool last_chunk = c == p.chunks - 1;
    // fp16 (not target-referenced): the unscaled dW operand copy, after the previous chunk's dW.
    const bool bmn_now = c > 0 && p.backward && !p.tref;
    if (!bk_ready || bmn_now) {
      AuxJobs j{};
      if (!bk_ready) bk_job(j, c);
      if (bmn_now) bmn_job(j, c, nullptr);
      if (aux(j, T_OTHER) != hipSuccess) return LCE_ERR_HIP;
    }
    bk_ready = false;
    // logits^T tile = W . X_c^T with the log-sum-exp epilogue.
    GemmArgs g{};
    g.A = W; g.lda = H; g.M = (int)V;
    g.B = xk; g.ldb = p.xk_kp; g.N = rows;
    g.K = (int)H;
    g.splits = 1; g.k_per_split = (int)round_up(H, kTileBytes / p.esz);
    g.group_m = 4;
    g.pmax = pmax; g.psum = psum; g.ldp = p.ncp;
    hipError_t e;
    {
    KernelTimer t(T_LOGITS, s);
    // W's rows end at H: whole K-tiles read them unchecked only when H is made of whole K-tiles.
    const bool whole = H % (kTileBytes / p.esz) == 0;
    if (p.backward) {
      g.out = ez; g.ldo = p.ez_kp;
      if (p.tref) g.ref = tref + t0;
      e = whole ? launch_gemm<T, EPI_LSE_BWD, A_K, false>(g, s) : launch_gemm<T, EPI_LSE_BWD, A_K, true>(g, s);
    } else {
      e = whole ? launch_gemm<T, EPI_LSE_FWD, A_K, false>(g, s) : launch_gemm<T, EPI_LSE_FWD, A_K, true>(g, s);
    }
    }
    if (e != hipSuccess) return LCE_ERR_HIP;

    auto combine = [&](int mode, const int* run_if) {
      KernelTimer t(T_OTHER, s);
      hipLaunchKernelGGL((combine_kernel<T>), dim3((unsigned)cdiv(rows, kCombineTokens)), dim3(256), 0, s, pmax, psum,
                         p.ncp, (int)p.slices, rows, y + t0, ignore_index, tgt + t0, lse + t0, tl + t0, mode,
                         scale ? scale + t0 : nullptr, (const int*)nvalid, mean, ez, p.ez_kp, V,
                         flags ? flags + c : nullptr, run_if);
      return hipGetLastError();
    };
    if (combine(p.tref ? CMB_TREF : CMB_FORWARD, nullptr) != hipSuccess) return LCE_ERR_HIP;
    if (!p.backward) {
      if (last_chunk) {
        AuxJobs j{};
        loss_job(j);
        if (j.loss_blocks > 0 && aux(j, T_OTHER) != hipSuccess) return LCE_ERR_HIP;
      }
      continue;
    }

    // One launch after the chunk's combines: dlogits (in place, blocked), the dW operand's copy of
    // X_c (target-referenced), and the next chunk's block_k copy (the logits GEMMs that read the
    // current one have run) or, after the last chunk, the loss sum.
    AuxJobs tail{};
    if (!last_chunk) {
      bk_job(tail, c + 1);
      bk_ready = true;
    } else {
      loss_job(tail);
    }
    if (p.tref) {
      // Only when combine flagged a token whose exp(z - z_target) may have overflowed: the chunk's
      // logits again with slice-maximum references, combine, and dlogits (work that returns at
      // once when the flag is clear).
      const int* flag = flags + c;
      GemmArgs gf = g;
      gf.ref = nullptr; gf.run_if = flag;
      {
      KernelTimer t(T_OTHER, s);
      const bool whole = H % (kTileBytes / p.esz) == 0;
      e = whole ? launch_gemm<T, EPI_LSE_BWD, A_K, false>(gf, s) : launch_gemm<T, EPI_LSE_BWD, A_K, true>(gf, s);
      }
      if (e != hipSuccess) return LCE_ERR_HIP;
      if (combine(CMB_SLICE, flag) != hipSuccess) return LCE_ERR_HIP;
      dl_job(tail, c, flag, std::min<int64_t>(p.ez_kp / 16 * p.ez_nb, (int64_t)num_cus()));
      bmn_job(tail, c, scale + t0);
      if (aux(tail, T_OTHER) != hipSuccess) return LCE_ERR_HIP;
    } else {
      // dlogits on every piece: a block per (K-pair group, token block).
      dl_job(tail, c, nullptr, p.ez_kp / 16 * p.ez_nb);
      if (aux(tail, T_DLOGITS) != hipSuccess) return LCE_ERR_HIP;
    }

    // dH rows of the chunk, as dH_c^T = W^T . dZ_c^T (A = W [V, H] MN-contig over H, B = dZ_c
    // blocked over the chunk's tokens), stored token-major.
    GemmArgs gh{};
    gh.A = W; gh.lda = H; gh.M = (int)H;
    gh.B = ez; gh.ldb = p.ez_kp; gh.N = rows;
    gh.K = (int)V;
    gh.splits = p.dh_splits; gh.k_per_split = (int)p.dh_kps;
    gh.group_m = 4;
    if (p.dh_splits > 1 || dx32) {
      gh.out = dhp; gh.ldo = H; gh.mode = 1;
    } else {
      gh.out = dH + t0 * H; gh.ldo = H; gh.mode = 0;
    }
    gh.n_valid = nvalid; gh.mean = mean;
    if (p.tref) gh.col_scale = scale + t0;
    {
    KernelTimer t(T_DH, s);
    if (launch_gemm<T, EPI_STORE, A_MN>(gh, s) != hipSuccess) return LCE_ERR_HIP;
    if (dx32) {
      const int64_t count = (int64_t)rows * H;
      hipLaunchKernelGGL((split_reduce_kernel<float, T>), dim3((unsigned)cdiv(count / 4, 256)), dim3(256), 0, s, dhp,
                         p.dh_splits, count, dx32 + t0 * H, (const int*)nvalid, mean);
      if (hipGetLastError() != hipSuccess) return LCE_ERR_HIP;
    } else if (p.dh_splits > 1) {
      const int64_t count = (int64_t)rows * H;
      hipLaunchKernelGGL((split_reduce_kernel<T>), dim3((unsigned)cdiv(count / 4, 256)), dim3(256), 0, s, dhp,
                         p.dh_splits, count, dH + t0 * H, (const int*)nvalid, mean);
      if (hipGetLastError() != hipSuccess) return LCE_ERR_HIP;
    }
    }

    // dW (+)= dZ_c^T . X_c  (A = dZ_c blocked, rows = vocabulary; B = X_c blocked over H).
    GemmArgs gw{};
    gw.A = ez; gw.lda = p.ez_kp; gw.M = (int)V;
    gw.B = xm; gw.ldb = p.xm_kp; gw.N = (int)H;
    gw.K = rows;
    gw.splits = 1; gw.k_per_split = (int)round_up(rows, kTileBytes / p.esz);
    gw.group_m = 4;
    gw.out = dW; gw.ldo = H;
    const bool last = c == p.chunks - 1;
    gw.mode = c == 0 ? DW_STORE : DW_ACCUMULATE;
    if (acc32) {
      gw.acc32 = acc32;
      gw.mode = c == 0 ? DW_ACC32_FIRST : last ? DW_ACC32_LAST : DW_ACC32_MID;
    }
    gw.n_valid = nvalid; gw.mean = mean;
    if (hook && last) {
      if (hipEventRecord(hook->dh_done, s) != hipSuccess) return LCE_ERR_HIP;
      const int64_t tiles = cdiv(V, kTile);
      for (int b = 0; b < hook->blocks; ++b) {
        const int64_t r0 = std::min(V, tiles * b / hook->blocks * kTile);
        const int64_t r1 = std::min(V, tiles * (b + 1) / hook->blocks * kTile);
        hook->row0[b] = r0;
        hook->row0[b + 1] = r1;
        if (r1 > r0) {
          GemmArgs gb = gw;
          gb.A = ez + 32 * r0;          // blocked: vocabulary id r0 starts 32 r0 elements in
          gb.M = (int)(r1 - r0);
          gb.out = dW + r0 * H;
          if (gb.acc32) gb.acc32 += r0 * H;
          KernelTimer t(T_DW, s);
          if (launch_gemm<T, EPI_DW, A_BLK>(gb, s) != hipSuccess) return LCE_ERR_HIP;
        }
        if (hipEventRecord(hook->dw_done[b], s) != hipSuccess) return LCE_ERR_HIP;
      }
    } else {
    KernelTimer t(T_DW, s);
    if (launch_gemm<T, EPI_DW, A_BLK>(gw, s) != hipSuccess) return LCE_ERR_HIP;
    }
  }

  return hipGetLastError() == hipSuccess ? LCE_OK : LCE_ERR_HIP;
}

// The RMSNorm variant: the LCE plan, then x [N,H], r [N] and, for backward, dX [N,H] fp32, s [N]
// and the dgamma partials [row blocks, H] (fp32) after it in the same workspace.
struct RmsPlan {
  Plan lce;
  int64_t row_blocks = 0;
  size_t o_x = 0, o_r = 0, o_dx = 0, o_s = 0, o_part = 0;
  size_t total = 0;
};

lce_status_t make_rms_plan(int64_t N, int64_t H, int64_t V, int dtype, bool backward, int64_t chunk_tokens,
                           RmsPlan& rp, bool query_device) {
  lce_status_t st = make_plan(N, H, V, dtype, backward, chunk_tokens, rp.lce, query_device, backward);
  if (st != LCE_OK) return st;
  size_t off = rp.lce.total;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (size_t)round_up((int64_t)bytes, kAlign);
    return o;
  };
  rp.o_x = take((size_t)N * H * rp.lce.esz);
  rp.o_r = take((size_t)N * 4);
  if (backward) {
    rp.row_blocks = cdiv(N, kRmsRows);
    if (rp.row_blocks > 65535) return LCE_ERR_UNSUPPORTED;  // rmsnorm_backward_kernel's grid y
    rp.o_dx = take((size_t)N * H * 4);
    rp.o_s = take((size_t)N * 4);
    rp.o_part = take((size_t)rp.row_blocks * H * 4);
  }
  rp.total = off;
  return LCE_OK;
}

bool eps_ok(float eps) { return eps >= 0.f && eps <= 3.0e38f; }  // rejects NaN and inf

template <typename T>
lce_status_t run_rms(const RmsPlan& rp, const T* h, const T* gamma, const T* W, const int64_t* y, float eps,
                     int64_t ignore_index, int reduction, float* loss, float* lse, T* normed, T* dh, T* dgamma,
                     T* dW, char* ws, hipStream_t s) {
  const int64_t N = rp.lce.N, H = rp.lce.H;
  T* x = normed ? normed : (T*)(ws + rp.o_x);
  float* r = (float*)(ws + rp.o_r);
  {
    KernelTimer t(T_OTHER, s);
    hipLaunchKernelGGL((rmsnorm_rows_kernel<T>), dim3((unsigned)cdiv(N, 4)), dim3(256), 0, s, h, gamma, N, H, eps, x,
                       r);
  }
  if (hipGetLastError() != hipSuccess) return LCE_ERR_HIP;
  // The LCE step on the normalised rows; its hidden gradient dX stays in fp32.
  float* dx = rp.lce.backward ? (float*)(ws + rp.o_dx) : nullptr;
  lce_status_t st = run<T>(rp.lce, x, W, y, ignore_index, reduction, loss, lse, nullptr, dW, ws, s, dx);
  if (st != LCE_OK || !rp.lce.backward) return st;
  KernelTimer t(T_OTHER, s);
  float* srow = (float*)(ws + rp.o_s);
  float* part = (float*)(ws + rp.o_part);
  hipLaunchKernelGGL((rmsnorm_rowdot_kernel<T>), dim3((unsigned)cdiv(N, 4)), dim3(256), 0, s, h, gamma,
                     (const float*)dx, N, H, srow);
  hipLaunchKernelGGL((rmsnorm_backward_kernel<T>), dim3((unsigned)cdiv(H, 256), (unsigned)rp.row_blocks), dim3(256),
                     0, s, h, gamma, (const float*)r, (const float*)srow, (const float*)dx, dh, N, H, part);
  hipLaunchKernelGGL((rmsnorm_gamma_reduce_kernel<T>), dim3((unsigned)cdiv(H, 256)), dim3(256), 0, s,
                     (const float*)part, (int)rp.row_blocks, H, dgamma);
  return hipGetLastError() == hipSuccess ? LCE_OK : LCE_ERR_HIP;
}

// ---- one training step of the output layer with its weights kept in host memory ----
//
// Section 3.1 ("Asynchronous Parameter Updating"): once a layer's backward finishes, its gradient
// goes d2h on a side stream while the CPU updates the previous piece and the GPU keeps computing;
// Section 3.2: FP32 masters in host memory, gradients in a pinned 16-bit buffer, the updated
// parameters converted to 16 bits in a pinned buffer before the h2d copy. For the output layer
// alone the pieces are blocks of vocabulary rows: the last chunk's dW GEMM runs block by block, each
// block's gradient is copied out as soon as it is done, the host updates it while later blocks are
// still being computed or copied, and the updated block is copied back on a second side stream.
// The step's two side streams (gradient copies out, parameter copies in), one pair per device,
// created (default priority, non-blocking) on the first call on that device and kept until the
// process ends; calls on one device share them.
std::mutex g_side_mu;
hipStream_t g_side_d2h[kMaxDevices] = {}, g_side_h2d[kMaxDevices] = {};

lce_status_t side_streams(hipStream_t& sd, hipStream_t& su) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return LCE_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return LCE_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_side_mu);
  for (hipStream_t* p : {&g_side_d2h[dev], &g_side_h2d[dev]}) {
    if (*p == nullptr && hipStreamCreateWithFlags(p, hipStreamNonBlocking) != hipSuccess) {
      *p = nullptr;
      return LCE_ERR_HIP;
    }
  }
  sd = g_side_d2h[dev];
  su = g_side_h2d[dev];
  return LCE_OK;
}

struct StepClock {
  hipEvent_t a = nullptr, b = nullptr;
  bool ok() const { return a && b; }
};

double event_ms(hipEvent_t a, hipEvent_t b) {
  float ms = 0.f;
  return hipEventElapsedTime(&ms, a, b) == hipSuccess ? (double)ms : 0.0;
}

template <typename T>
lce_status_t run_head(const Plan& p, const T* X, const int64_t* y, int64_t ignore_index, int reduction,
                      T* W, T* dH, T* dW, float* loss, float* master, float* m, float* v, T* grad_host,
                      T* param_host, const lce_adam_config_t* adam, int64_t step, int blocks, int threads,
                      bool overlap, char* ws, hipStream_t s, lce_head_step_timing_t* timing) {
  const auto t_start = std::chrono::steady_clock::now();
  const int64_t H = p.H, V = p.V;
  const int dt = std::is_same<T, bf16>::value ? LCE_DTYPE_BF16 : LCE_DTYPE_FP16;
  hipStream_t sd = nullptr, su = nullptr;
  std::vector<hipEvent_t> evs;
  auto ev = [&]() -> hipEvent_t {
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    evs.push_back(e);
    return e;
  };
  lce_status_t st = LCE_OK;
  double update_ms = 0.0;
  std::vector<hipEvent_t> dw_done(blocks), d2h_a(blocks), d2h_b(blocks), h2d_a(blocks), h2d_b(blocks);
  std::vector<int64_t> row0(blocks + 1, 0);
  hipEvent_t g0 = nullptr, g1 = nullptr, dh_done = nullptr, upd_end = nullptr;
  do {
    if ((st = side_streams(sd, su)) != LCE_OK) break;
    g0 = ev(); g1 = ev(); dh_done = ev(); upd_end = ev();
    for (int b = 0; b < blocks; ++b) {
      dw_done[b] = ev(); d2h_a[b] = ev(); d2h_b[b] = ev(); h2d_a[b] = ev(); h2d_b[b] = ev();
    }
    if (!g0 || !g1 || !dh_done || !upd_end || !h2d_b[blocks - 1]) { st = LCE_ERR_HIP; break; }
    if (hipEventRecord(g0, s) != hipSuccess) { st = LCE_ERR_HIP; break; }
    DwBlocks hook;
    hook.blocks = blocks;
    hook.dw_done = dw_done.data();
    hook.row0 = row0.data();
    hook.dh_done = dh_done;
    st = run<T>(p, X, W, y, ignore_index, reduction, loss, nullptr, dH, dW, ws, s, nullptr, &hook);
    if (st != LCE_OK) break;
    if (hipEventRecord(g1, s) != hipSuccess) { st = LCE_ERR_HIP; break; }
    if (!overlap) {
      // Sequential reference schedule: all of the step, then all copies and the whole update.
      if (hipStreamWaitEvent(sd, g1, 0) != hipSuccess || hipStreamWaitEvent(su, g1, 0) != hipSuccess) {
        st = LCE_ERR_HIP; break;
      }
    } else if (hipStreamWaitEvent(su, dh_done, 0) != hipSuccess) {  // W is free once the last dH is done
      st = LCE_ERR_HIP; break;
    }
    // Gradient blocks out, in order, each as soon as its GEMM block is done.
    for (int b = 0; b < blocks && st == LCE_OK; ++b) {
      const size_t off = (size_t)row0[b] * H, n = (size_t)(row0[b + 1] - row0[b]) * H;
      if ((overlap && hipStreamWaitEvent(sd, dw_done[b], 0) != hipSuccess) || hipEventRecord(d2h_a[b], sd) != hipSuccess ||
          (n && hipMemcpyAsync(grad_host + off, dW + off, n * sizeof(T), hipMemcpyDeviceToHost, sd) != hipSuccess) ||
          hipEventRecord(d2h_b[b], sd) != hipSuccess)
        st = LCE_ERR_HIP;
    }
    if (st != LCE_OK) break;
    // Sequential schedule: every gradient block is in host memory before the update starts.
    if (!overlap && hipStreamSynchronize(sd) != hipSuccess) { st = LCE_ERR_HIP; break; }
    // Host update of each block when its gradient has landed, then its parameters back in (the
    // sequential schedule holds the copies back until the whole update is done).
    for (int b = 0; b < blocks && st == LCE_OK; ++b) {
      const size_t off = (size_t)row0[b] * H, n = (size_t)(row0[b + 1] - row0[b]) * H;
      if (hipEventSynchronize(d2h_b[b]) != hipSuccess) { st = LCE_ERR_HIP; break; }
      const auto u0 = std::chrono::steady_clock::now();
      if (n) st = lce_host_adam_step(master + off, grad_host + off, dt, m + off, v + off, (int64_t)n, adam, step,
                                     param_host + off, threads);
      update_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - u0).count();
      if (st != LCE_OK) break;
      if (!overlap) continue;
      if (hipEventRecord(h2d_a[b], su) != hipSuccess ||
          (n && hipMemcpyAsync(W + off, param_host + off, n * sizeof(T), hipMemcpyHostToDevice, su) != hipSuccess) ||
          hipEventRecord(h2d_b[b], su) != hipSuccess)
        st = LCE_ERR_HIP;
    }
    for (int b = 0; b < blocks && st == LCE_OK && !overlap; ++b) {
      const size_t off = (size_t)row0[b] * H, n = (size_t)(row0[b + 1] - row0[b]) * H;
      if (hipEventRecord(h2d_a[b], su) != hipSuccess ||
          (n && hipMemcpyAsync(W + off, param_host + off, n * sizeof(T), hipMemcpyHostToDevice, su) != hipSuccess) ||
          hipEventRecord(h2d_b[b], su) != hipSuccess)
        st = LCE_ERR_HIP;
    }
    if (st != LCE_OK) break;
    // The caller's stream sees the updated weights; the call returns when everything is done.
    if (hipEventRecord(upd_end, su) != hipSuccess || hipStreamWaitEvent(s, upd_end, 0) != hipSuccess ||
        hipStreamSynchronize(su) != hipSuccess || hipStreamSynchronize(sd) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      st = LCE_ERR_HIP;
  } while (false);
  if (st == LCE_OK && timing) {
    timing->step_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    timing->gpu_ms = event_ms(g0, g1);
    timing->d2h_ms = timing->h2d_ms = 0.0;
    for (int b = 0; b < blocks; ++b) {
      timing->d2h_ms += event_ms(d2h_a[b], d2h_b[b]);
      timing->h2d_ms += event_ms(h2d_a[b], h2d_b[b]);
    }
    timing->update_ms = update_ms;
    timing->tail_ms = event_ms(g1, upd_end);
  }
  if (st != LCE_OK) {  // leave no work behind on the side streams before releasing them
    if (sd) (void)hipStreamSynchronize(sd);
    if (su) (void)hipStreamSynchronize(su);
  }
  for (auto e : evs) (void)hipEventDestroy(e);
  return st;
}

}  // namespace
}  // namespace lce

extern "C" {

size_t lce_workspace_size(int64_t N, int64_t H, int64_t V, int dtype, int with_backward, int64_t chunk_tokens) {
  lce::Plan p;
  if (lce::make_plan(N, H, V, dtype, with_backward != 0, chunk_tokens, p, true) != LCE_OK) return 0;
  return p.total;
}

int64_t lce_auto_chunk_tokens(int64_t N, int64_t H, int64_t V, int dtype) {
  lce::Plan p;
  if (lce::make_plan(N, H, V, dtype, true, 0, p, false) != LCE_OK) return 0;
  return p.nc;
}

lce_status_t lce_plan_info(int64_t N, int64_t H, int64_t V, int dtype, int with_backward, int64_t chunk_tokens,
                           lce_plan_info_t* info) {
  if (!info) return LCE_ERR_INVALID_ARGUMENT;
  lce::Plan p;
  const lce_status_t st = lce::make_plan(N, H, V, dtype, with_backward != 0, chunk_tokens, p, true);
  if (st != LCE_OK) return st;
  std::memset(info, 0, sizeof(*info));
  info->chunk_tokens = p.nc;
  info->chunks = p.chunks;
  info->dh_splits = p.backward ? p.dh_splits : 0;
  info->target_referenced = p.tref ? 1 : 0;
  info->dw_fp32_carry = p.dw_acc32 ? 1 : 0;
  info->workspace_bytes = p.total;
  info->fallback_flags_offset = p.backward ? p.o_flags : 0;
  return LCE_OK;
}

lce_status_t lce_forward(const void* hidden, const void* weight, const int64_t* labels, int64_t N, int64_t H,
                         int64_t V, int dtype, int64_t ignore_index, int reduction, float* loss, float* lse,
                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!hidden || !weight || !labels || !loss) return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_NONE && reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM)
    return LCE_ERR_INVALID_ARGUMENT;
  lce::Plan p;
  lce_status_t st = lce::make_plan(N, H, V, dtype, false, 0, p, true);
  if (st != LCE_OK) return st;
  if (!workspace || workspace_bytes < p.total) return LCE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run<lce::bf16>(p, (const lce::bf16*)hidden, (const lce::bf16*)weight, labels, ignore_index,
                               reduction, loss, lse, nullptr, nullptr, (char*)workspace, s);
  if (dtype == LCE_DTYPE_FP16)
    return lce::run<lce::f16>(p, (const lce::f16*)hidden, (const lce::f16*)weight, labels, ignore_index,
                              reduction, loss, lse, nullptr, nullptr, (char*)workspace, s);
  return lce::run<float>(p, (const float*)hidden, (const float*)weight, labels, ignore_index, reduction, loss, lse,
                         nullptr, nullptr, (char*)workspace, s);
}

lce_status_t lce_forward_no_alloc(const void* hidden, const void* weight, const int64_t* labels, int64_t N,
                                  int64_t H, int64_t V, int dtype, int64_t ignore_index, int reduction, float* loss,
                                  float* lse, void* stream) {
  if (!hidden || !weight || !labels || !loss) return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_NONE && reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM)
    return LCE_ERR_INVALID_ARGUMENT;
  lce::Plan p;
  lce_status_t st = lce::make_no_alloc_plan(N, H, V, dtype, p);
  if (st != LCE_OK) return st;
  void* ws = nullptr;
  st = lce::no_alloc_scratch(&ws);
  if (st != LCE_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run<lce::bf16>(p, (const lce::bf16*)hidden, (const lce::bf16*)weight, labels, ignore_index,
                               reduction, loss, lse, nullptr, nullptr, (char*)ws, s);
  if (dtype == LCE_DTYPE_FP16)
    return lce::run<lce::f16>(p, (const lce::f16*)hidden, (const lce::f16*)weight, labels, ignore_index,
                              reduction, loss, lse, nullptr, nullptr, (char*)ws, s);
  return lce::run<float>(p, (const float*)hidden, (const float*)weight, labels, ignore_index, reduction, loss, lse,
                         nullptr, nullptr, (char*)ws, s);
}

lce_status_t lce_forward_backward(const void* hidden, const void* weight, const int64_t* labels, int64_t N,
                                  int64_t H, int64_t V, int dtype, int64_t ignore_index, int reduction, float* loss,
                                  void* grad_hidden, void* grad_weight, int64_t chunk_tokens, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  if (!hidden || !weight || !labels || !loss || !grad_hidden || !grad_weight) return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM) return LCE_ERR_INVALID_ARGUMENT;
  lce::Plan p;
  lce_status_t st = lce::make_plan(N, H, V, dtype, true, chunk_tokens, p, true);
  if (st != LCE_OK) return st;
  if (!workspace || workspace_bytes < p.total) return LCE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run<lce::bf16>(p, (const lce::bf16*)hidden, (const lce::bf16*)weight, labels, ignore_index,
                               reduction, loss, nullptr, (lce::bf16*)grad_hidden, (lce::bf16*)grad_weight,
                               (char*)workspace, s);
  if (dtype == LCE_DTYPE_FP16)
    return lce::run<lce::f16>(p, (const lce::f16*)hidden, (const lce::f16*)weight, labels, ignore_index,
                              reduction, loss, nullptr, (lce::f16*)grad_hidden, (lce::f16*)grad_weight,
                              (char*)workspace, s);
  return lce::run<float>(p, (const float*)hidden, (const float*)weight, labels, ignore_index, reduction, loss,
                         nullptr, (float*)grad_hidden, (float*)grad_weight, (char*)workspace, s);
}

size_t lce_rmsnorm_workspace_size(int64_t N, int64_t H, int64_t V, int dtype, int with_backward,
                                  int64_t chunk_tokens) {
  lce::RmsPlan rp;
  if (lce::make_rms_plan(N, H, V, dtype, with_backward != 0, chunk_tokens, rp, true) != LCE_OK) return 0;
  return rp.total;
}

lce_status_t lce_rmsnorm_forward(const void* hidden, const void* gamma, const void* weight, const int64_t* labels,
                                 int64_t N, int64_t H, int64_t V, int dtype, float eps, int64_t ignore_index,
                                 int reduction, float* loss, float* lse, void* normed, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  if (!hidden || !gamma || !weight || !labels || !loss || !lce::eps_ok(eps)) return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_NONE && reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM)
    return LCE_ERR_INVALID_ARGUMENT;
  lce::RmsPlan rp;
  lce_status_t st = lce::make_rms_plan(N, H, V, dtype, false, 0, rp, true);
  if (st != LCE_OK) return st;
  if (!workspace || workspace_bytes < rp.total) return LCE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run_rms<lce::bf16>(rp, (const lce::bf16*)hidden, (const lce::bf16*)gamma, (const lce::bf16*)weight,
                                   labels, eps, ignore_index, reduction, loss, lse, (lce::bf16*)normed, nullptr,
                                   nullptr, nullptr, ws, s);
  if (dtype == LCE_DTYPE_FP16)
    return lce::run_rms<lce::f16>(rp, (const lce::f16*)hidden, (const lce::f16*)gamma, (const lce::f16*)weight,
                                  labels, eps, ignore_index, reduction, loss, lse, (lce::f16*)normed, nullptr,
                                  nullptr, nullptr, ws, s);
  return lce::run_rms<float>(rp, (const float*)hidden, (const float*)gamma, (const float*)weight, labels, eps,
                             ignore_index, reduction, loss, lse, (float*)normed, nullptr, nullptr, nullptr, ws, s);
}

lce_status_t lce_rmsnorm_forward_backward(const void* hidden, const void* gamma, const void* weight,
                                          const int64_t* labels, int64_t N, int64_t H, int64_t V, int dtype,
                                          float eps, int64_t ignore_index, int reduction, float* loss,
                                          void* grad_hidden, void* grad_gamma, void* grad_weight,
                                          int64_t chunk_tokens, void* workspace, size_t workspace_bytes,
                                          void* stream) {
  if (!hidden || !gamma || !weight || !labels || !loss || !grad_hidden || !grad_gamma || !grad_weight ||
      !lce::eps_ok(eps))
    return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM) return LCE_ERR_INVALID_ARGUMENT;
  lce::RmsPlan rp;
  lce_status_t st = lce::make_rms_plan(N, H, V, dtype, true, chunk_tokens, rp, true);
  if (st != LCE_OK) return st;
  if (!workspace || workspace_bytes < rp.total) return LCE_ERR_WORKSPACE_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  char* ws = (char*)workspace;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run_rms<lce::bf16>(rp, (const lce::bf16*)hidden, (const lce::bf16*)gamma, (const lce::bf16*)weight,
                                   labels, eps, ignore_index, reduction, loss, nullptr, nullptr,
                                   (lce::bf16*)grad_hidden, (lce::bf16*)grad_gamma, (lce::bf16*)grad_weight, ws, s);
  if (dtype == LCE_DTYPE_FP16)
    return lce::run_rms<lce::f16>(rp, (const lce::f16*)hidden, (const lce::f16*)gamma, (const lce::f16*)weight,
                                  labels, eps, ignore_index, reduction, loss, nullptr, nullptr,
                                  (lce::f16*)grad_hidden, (lce::f16*)grad_gamma, (lce::f16*)grad_weight, ws, s);
  return lce::run_rms<float>(rp, (const float*)hidden, (const float*)gamma, (const float*)weight, labels, eps,
                             ignore_index, reduction, loss, nullptr, nullptr, (float*)grad_hidden,
                             (float*)grad_gamma, (float*)grad_weight, ws, s);
}

lce_status_t lce_head_train_step(const void* hidden, const int64_t* labels, int64_t N, int64_t H, int64_t V,
                                 int dtype, int64_t ignore_index, int reduction, int64_t chunk_tokens,
                                 void* weight, void* grad_hidden, void* grad_weight, float* loss, float* master,
                                 float* exp_avg, float* exp_avg_sq, void* grad_host, void* param_host,
                                 const lce_adam_config_t* adam, int64_t step, int vocab_blocks, int n_threads,
                                 int overlap, void* workspace, size_t workspace_bytes, void* stream,
                                 lce_head_step_timing_t* timing) {
  if (!hidden || !labels || !weight || !grad_hidden || !grad_weight || !loss || !master || !exp_avg ||
      !exp_avg_sq || !grad_host || !param_host || !adam || step < 1 || vocab_blocks < 1 || vocab_blocks > 256 ||
      n_threads < 0)
    return LCE_ERR_INVALID_ARGUMENT;
  if (reduction != LCE_REDUCTION_MEAN && reduction != LCE_REDUCTION_SUM) return LCE_ERR_INVALID_ARGUMENT;
  if (dtype != LCE_DTYPE_BF16 && dtype != LCE_DTYPE_FP16) return dtype == LCE_DTYPE_FP32 ? LCE_ERR_UNSUPPORTED
                                                                                        : LCE_ERR_INVALID_ARGUMENT;
  lce::Plan p;
  lce_status_t st = lce::make_plan(N, H, V, dtype, true, chunk_tokens, p, true);
  if (st != LCE_OK) return st;
  if (!workspace || workspace_bytes < p.total) return LCE_ERR_WORKSPACE_TOO_SMALL;
  // The optimizer settings are checked before any GPU work.
  const lce_adam_config_t& a = *adam;
  if (!(a.lr >= 0.f && a.lr < 3.0e38f) || !(a.beta1 >= 0.f && a.beta1 < 1.f) || !(a.beta2 >= 0.f && a.beta2 < 1.f) ||
      !(a.eps > 0.f && a.eps < 3.0e38f) || !(a.weight_decay >= 0.f && a.weight_decay < 3.0e38f))
    return LCE_ERR_INVALID_ARGUMENT;
  hipStream_t s = (hipStream_t)stream;
  if (dtype == LCE_DTYPE_BF16)
    return lce::run_head<lce::bf16>(p, (const lce::bf16*)hidden, labels, ignore_index, reduction, (lce::bf16*)weight,
                                    (lce::bf16*)grad_hidden, (lce::bf16*)grad_weight, loss, master, exp_avg, exp_avg_sq,
                                    (lce::bf16*)grad_host, (lce::bf16*)param_host, adam, step, vocab_blocks,
                                    n_threads, overlap != 0, (char*)workspace, s, timing);
  return lce::run_head<lce::f16>(p, (const lce::f16*)hidden, labels, ignore_index, reduction, (lce::f16*)weight,
                                 (lce::f16*)grad_hidden, (lce::f16*)grad_weight, loss, master, exp_avg, exp_avg_sq,
                                 (lce::f16*)grad_host, (lce::f16*)param_host, adam, step, vocab_blocks, n_threads,
                                 overlap != 0, (char*)workspace, s, timing);
}

lce_status_t lce_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(lce::g_timing_mu);
  for (auto& t : lce::g_timed) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  lce::g_timed.clear();
  lce::g_timing_on = enable != 0;
  return LCE_OK;
}

lce_status_t lce_timing_read(double* ms, int64_t* launches, int n_kinds) {
  if (!ms || !launches || n_kinds < 1) return LCE_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lk(lce::g_timing_mu);
  for (int k = 0; k < n_kinds; ++k) { ms[k] = 0.0; launches[k] = 0; }
  lce_status_t st = LCE_OK;
  for (auto& t : lce::g_timed) {
    float e = 0.f;
    if (hipEventSynchronize(t.stop) != hipSuccess || hipEventElapsedTime(&e, t.start, t.stop) != hipSuccess) {
      st = LCE_ERR_HIP;
    } else if (t.kind < n_kinds) {
      ms[t.kind] += e;
      launches[t.kind] += 1;
    }
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  lce::g_timed.clear();
  return st;
}

const char* lce_status_string(int status) {
  switch (status) {
    case LCE_OK: return "LCE_OK";
    case LCE_ERR_INVALID_ARGUMENT: return "LCE_ERR_INVALID_ARGUMENT";
    case LCE_ERR_UNSUPPORTED: return "LCE_ERR_UNSUPPORTED";
    case LCE_ERR_WORKSPACE_TOO_SMALL: return "LCE_ERR_WORKSPACE_TOO_SMALL";
    case LCE_ERR_HIP: return "LCE_ERR_HIP";
    default: return "LCE_ERR_UNKNOWN";
  }
}

}  // extern "C"
