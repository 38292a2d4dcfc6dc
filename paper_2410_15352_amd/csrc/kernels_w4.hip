// The persistent four-wave bf16 GEMM, the G^ and the decompression kernels and
// their launchers.  Built as its
// own translation unit with -mllvm -enable-misched=false and
// -mllvm -enable-post-misched=false: the K-step code in gemm_w4.hpp is written
// in issue order and must not be rescheduled.
#include "gemm_w4_launch.hpp"

#include <atomic>

namespace compact {

// One instantiation per use, so that profiles report the forward and the dx
// GEMM separately; KMASK: K % 8 != 0, ODD: an odd output width (the LLaMA-1B
// widths of 5461); PAIRS: A copied in 64-deep slots, two 32-deep K tiles at a
// time.
template <int USE, bool KMASK = false, bool ODD = false, bool PAIRS = false>
__global__ __launch_bounds__(kW4Threads, 1) void k_gemm_w4(W4Gemm g) {
  gemm_w4_persistent<KMASK, ODD, PAIRS>(g);
}

template <int SHAPE>
__global__ __launch_bounds__(256, 1) void k_ghat_w4(GhatW4Params p) {
  ghat_w4<SHAPE>(p);
}

// Four workgroups per CU for bf16 W (at most 128 registers per lane), two for fp32 W.
template <bool WF32>
__global__ __launch_bounds__(256, WF32 ? 2 : 4) void k_dec_w4(DecW4Batch d) {
  const int b = static_cast<int>(xcd_remap(blockIdx.x, gridDim.x));
  const int l = batch_layer_of(d.begin, d.count, b);
  dec_w4_tile<WF32>(d.layer[l], b - d.begin[l]);
}

namespace {

constexpr int kMaxDevices = 64;
std::atomic<int> g_cus[kMaxDevices];        // CU count per device, 0 until queried
constexpr int kGemmVariants = 16;
std::atomic<bool> g_lds_set[kMaxDevices][kGemmVariants + 3];  // dynamic LDS limit raised: k_gemm_w4, k_ghat_w4

bool fits_offsets(int64_t ld, int64_t K) {
  // 32-bit buffer offsets: 256 rows of ld elements plus K, in bytes
  return ld > 0 && (int64_t(kW4Tile) * ld + K) * 2 < (int64_t(1) << 31);
}

}  // namespace

// Rows of tiles per band of the walk order (gemm_w4.hpp).  Measured on the
// LLaMA-350M shapes (65536 tokens; 4 to 23 column tiles; band_rows 1, 3, 4, 6,
// 8, 16): 4 is the best or within 2% of the best for every forward and dx
// shape, and 2.6 ms per step faster than the row-major walk (band_rows 1).
int w4_band_rows(int tiles_m) { return tiles_m < 4 ? (tiles_m > 0 ? tiles_m : 1) : 4; }

bool gemm_w4_eligible(int64_t M, int64_t K, int64_t lda, int64_t ldb, int64_t rows_b, int64_t ldc0,
                      int64_t cols0, int64_t ldc1, int64_t cols1, bool b_tiled) {
  if (M < 1 || K < int64_t(kW4MinKTiles) * kW4K) return false;
  if (K % 8 != 0 && !b_tiled) return false;  // B's padding past K must be zero (staged here)
  if (lda % 8 != 0 || ldb % 8 != 0 || lda < K || ldb < K) return false;
  if (!fits_offsets(lda, K) || !fits_offsets(ldb, K) || !fits_offsets(ldc0, 0)) return false;
  if (cols0 < 1) return false;
  if (cols1 != 0 && !fits_offsets(ldc1, 0)) return false;
  const int64_t limit = int64_t(1) << 30;
  if (M > limit || rows_b > limit || ldc0 > limit || ldc1 > limit) return false;
  return true;
}

hipError_t gemm_w4_launch(const W4Gemm& g, W4Use use, hipStream_t stream) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  int cus = g_cus[dev].load(std::memory_order_relaxed);
  if (cus == 0) {
    e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    cus = cus > 0 ? cus : 1;
    g_cus[dev].store(cus, std::memory_order_relaxed);
  }
  const bool kmask = g.K % 8 != 0;
  const bool odd = g.seg[0].cols % 2 != 0 || (g.seg[1].tiles > 0 && g.seg[1].cols % 2 != 0);
  // A in 64-deep slots (at least kW4PMinKTiles K tiles): an odd number of K
  // tiles is padded by one (a zero K tile, 1/kt more matrix work), which pays
  // from about 40 K tiles on
  const int64_t kt = ceil_div(g.K, kW4K);
  const bool pairs = kt >= kW4PMinKTiles && (kt % 2 == 0 || kt >= 41);
  const int u = (use == W4Use::kForward ? 0 : 8) + (pairs ? 4 : 0) + (kmask ? 2 : 0) + (odd ? 1 : 0);
  static const void* const fns[kGemmVariants] = {
      reinterpret_cast<const void*>(k_gemm_w4<0, false, false, false>),
      reinterpret_cast<const void*>(k_gemm_w4<0, false, true, false>),
      reinterpret_cast<const void*>(k_gemm_w4<0, true, false, false>),
      reinterpret_cast<const void*>(k_gemm_w4<0, true, true, false>),
      reinterpret_cast<const void*>(k_gemm_w4<0, false, false, true>),
      reinterpret_cast<const void*>(k_gemm_w4<0, false, true, true>),
      reinterpret_cast<const void*>(k_gemm_w4<0, true, false, true>),
      reinterpret_cast<const void*>(k_gemm_w4<0, true, true, true>),
      reinterpret_cast<const void*>(k_gemm_w4<1, false, false, false>),
      reinterpret_cast<const void*>(k_gemm_w4<1, false, true, false>),
      reinterpret_cast<const void*>(k_gemm_w4<1, true, false, false>),
      reinterpret_cast<const void*>(k_gemm_w4<1, true, true, false>),
      reinterpret_cast<const void*>(k_gemm_w4<1, false, false, true>),
      reinterpret_cast<const void*>(k_gemm_w4<1, false, true, true>),
      reinterpret_cast<const void*>(k_gemm_w4<1, true, false, true>),
      reinterpret_cast<const void*>(k_gemm_w4<1, true, true, true>)};
  const size_t lds = pairs ? kW4PLds : kW4Lds;
  if (!g_lds_set[dev][u].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(fns[u], hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
    if (e != hipSuccess) return e;
    g_lds_set[dev][u].store(true, std::memory_order_release);
  }
  if (g.tiles <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(g.tiles < cus ? g.tiles : cus));
  W4Gemm gg = g;
  gg.band_rows = w4_band_rows(g.tiles / g.tiles_n);
  void* args[] = {&gg};
  e = hipLaunchKernel(fns[u], grid, dim3(kW4Threads), args, lds, stream);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

bool dec_w4_eligible(int64_t n, int64_t m, int64_t r, int64_t ldw, int64_t ldn, int64_t ldpt, bool w_f32) {
  const int64_t esz = w_f32 ? 4 : 2, lim = int64_t(1) << 31;
  if (n < 1 || m < 1 || r < 1 || ldn % 8 != 0 || ldpt % 8 != 0 || ldw % 4 != 0) return false;
  if (ldw < m || ldn < m || ldpt < n) return false;
  // 32-bit offsets: a W tile (128 rows), and every K tile of N and P^T
  if (int64_t(kDecT) * ldw * esz >= lim) return false;
  if ((r + 2 * kDecK) * ldn * 2 >= lim || (r + 2 * kDecK) * ldpt * 2 >= lim) return false;
  return n < lim && m < lim;
}

hipError_t dec_w4_launch(const DecW4Batch& d, bool w_f32, hipStream_t stream) {
  const int blocks = d.begin[d.count];
  if (d.count <= 0 || blocks <= 0) return hipSuccess;
  if (w_f32)
    hipLaunchKernelGGL(k_dec_w4<true>, dim3(static_cast<uint32_t>(blocks)), dim3(256), kDecLds, stream, d);
  else
    hipLaunchKernelGGL(k_dec_w4<false>, dim3(static_cast<uint32_t>(blocks)), dim3(256), kDecLds, stream, d);
  return hipGetLastError();
}

hipError_t ghat_w4_launch(const GhatW4Params& p, hipStream_t stream) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (p.shape < 0 || p.shape > 2) return hipErrorInvalidValue;
  static const void* const fns[3] = {reinterpret_cast<const void*>(k_ghat_w4<0>),
                                     reinterpret_cast<const void*>(k_ghat_w4<1>),
                                     reinterpret_cast<const void*>(k_ghat_w4<2>)};
  static const size_t lds[3] = {GhShape<0>::kLds, GhShape<1>::kLds, GhShape<2>::kLds};
  if (!g_lds_set[dev][kGemmVariants + p.shape].load(std::memory_order_acquire)) {
    e = hipFuncSetAttribute(fns[p.shape], hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds[p.shape]));
    if (e != hipSuccess) return e;
    g_lds_set[dev][kGemmVariants + p.shape].store(true, std::memory_order_release);
  }
  const int64_t blocks = int64_t(p.tile_begin[p.count]) * p.splits;
  if (blocks <= 0) return hipSuccess;
  const dim3 grid(static_cast<uint32_t>(blocks));
  if (p.shape == 1)
    hipLaunchKernelGGL(k_ghat_w4<1>, grid, dim3(256), lds[1], stream, p);
  else if (p.shape == 2)
    hipLaunchKernelGGL(k_ghat_w4<2>, grid, dim3(256), lds[2], stream, p);
  else
    hipLaunchKernelGGL(k_ghat_w4<0>, grid, dim3(256), lds[0], stream, p);
  return hipGetLastError();
}

}  // namespace compact
