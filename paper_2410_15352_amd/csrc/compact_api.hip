// Host side of the C ABI declared in include/compact.h: argument validation,
// workspace sizing and kernel launches.  See the header for the contract.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>
#include <algorithm>
#include <mutex>

#include "../../include/compact.h"
#include "gemm_w4_launch.hpp"
#include "kernels_bf16.hpp"
#include "kernels_common.hpp"

using namespace compact;

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  std::vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return COMPACT_OK;
}

int check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(COMPACT_EHIP, "%s: %s", what, hipGetErrorString(e));
  return COMPACT_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t elem_size(int dtype) { return dtype == COMPACT_BF16 ? 2 : 4; }

bool valid_dtype(int d) { return d == COMPACT_F32 || d == COMPACT_BF16; }

// Leading-dimension rule: ld >= cols and rows start on 16-byte boundaries.
int check_matrix(const char* name, const void* p, int64_t ld, int64_t cols, int dtype) {
  if (p == nullptr) return fail(COMPACT_EINVAL, "%s is NULL", name);
  if (ld < cols) return fail(COMPACT_EINVAL, "%s: ld %lld < columns %lld", name, (long long)ld, (long long)cols);
  if (!aligned16(p)) return fail(COMPACT_EALIGN, "%s: pointer not 16-byte aligned", name);
  const int64_t q = dtype == COMPACT_BF16 ? 8 : 4;
  if (ld % q != 0) return fail(COMPACT_EALIGN, "%s: ld %lld not a multiple of %lld", name, (long long)ld, (long long)q);
  return COMPACT_OK;
}

int check_dense(const char* name, const void* p) {
  if (p == nullptr) return fail(COMPACT_EINVAL, "%s is NULL", name);
  if (!aligned16(p)) return fail(COMPACT_EALIGN, "%s: pointer not 16-byte aligned", name);
  return COMPACT_OK;
}

int check_shape(int64_t tokens, int64_t n, int64_t m, int64_t r, int proj) {
  if (tokens < 0 || n < 1 || m < 1) return fail(COMPACT_EINVAL, "bad shape tokens=%lld n=%lld m=%lld", (long long)tokens, (long long)n, (long long)m);
  if (r < 1 || r > n) return fail(COMPACT_EINVAL, "rank r=%lld must satisfy 1 <= r <= n=%lld", (long long)r, (long long)n);
  const int kind = proj & 0xFF, draws = (proj >> 8) & 0xFF, flags = proj >> 16;
  if (proj < 0 || (kind != COMPACT_PROJ_GAUSSIAN && kind != COMPACT_PROJ_IDENTITY && kind != COMPACT_PROJ_SPARSE_JL))
    return fail(COMPACT_EINVAL, "unknown projection %d", proj);
  if (kind != COMPACT_PROJ_SPARSE_JL && (draws != 0 || flags != 0))
    return fail(COMPACT_EINVAL, "unknown projection %d", proj);
  if (flags & ~(COMPACT_PROJ_GATHER >> 16)) return fail(COMPACT_EINVAL, "unknown projection %d", proj);
  if (kind == COMPACT_PROJ_SPARSE_JL && draws > kSjltMaxS)
    return fail(COMPACT_EINVAL, "sparse projection: %d draws per row (at most %d)", draws, kSjltMaxS);
  if ((proj & COMPACT_PROJ_GATHER) && (draws != 0 ? draws : COMPACT_SPARSE_JL_DEFAULT_S) > COMPACT_GATHER_MAX_S)
    return fail(COMPACT_EUNSUPPORTED, "gather-add forward: %d draws per row (at most %d)",
                draws != 0 ? draws : COMPACT_SPARSE_JL_DEFAULT_S, COMPACT_GATHER_MAX_S);
  if ((proj & COMPACT_PROJ_GATHER) && r >= int64_t(kGatherSkip))
    return fail(COMPACT_EUNSUPPORTED, "gather-add forward: r=%lld (below %u)", (long long)r, kGatherSkip);
  if (kind == COMPACT_PROJ_IDENTITY && r != n) return fail(COMPACT_EINVAL, "identity projection needs r == n (r=%lld, n=%lld)", (long long)r, (long long)n);
  if (n > (int64_t(1) << 31) || r > (int64_t(1) << 31)) return fail(COMPACT_EUNSUPPORTED, "n and r must be below 2^31");
  return COMPACT_OK;
}

constexpr size_t kWsAlign = 256;
constexpr int kMaxScratchDevices = 64;

void* align_ws(void* ws) {
  const uintptr_t a = (reinterpret_cast<uintptr_t>(ws) + kWsAlign - 1) & ~uintptr_t(kWsAlign - 1);
  return reinterpret_cast<void*>(a);
}

// Tile shapes of the bf16 kernels.  Forward and dx: 256 x 256 tiles, 8 waves
// in a 4 x 2 grid (64 x 128 per wave), two LDS stages of 64 KB.  G^: 128 x 128
// tiles, 4 waves (r is often 128 or less).
constexpr int kBM = 256, kBN = 256, kWGM = 4, kWGN = 2;
constexpr int kThreads = kWGM * kWGN * kWave;
constexpr size_t kGemmLds = 2u * (kBM + kBN) * kBK * sizeof(uint16_t);
constexpr int kGBM = 128, kGBN = 128, kGWGM = 2, kGWGN = 2;
constexpr int kGThreads = kGWGM * kGWGN * kWave;
constexpr size_t kGhatLds = 2u * (kGBM + kGBN) * kBK * sizeof(uint16_t);

// Split-K plan for G^ = z^T dL/do (K = tokens).
struct SplitPlan {
  int tiles_r, tiles_m, splits;
  int64_t split_len;
};

SplitPlan ghat_plan(int64_t tokens, int64_t r, int64_t m) {
  SplitPlan s;
  s.tiles_r = static_cast<int>(ceil_div(r, kGBM));
  s.tiles_m = static_cast<int>(ceil_div(m, kGBN));
  const int64_t tiles = int64_t(s.tiles_r) * s.tiles_m;
  const int64_t ktiles = ceil_div(tokens > 0 ? tokens : 1, kBK);
  int64_t splits = ceil_div(512, tiles);
  if (splits < 1) splits = 1;
  if (splits > ktiles) splits = ktiles;
  s.split_len = ceil_div(ktiles, splits) * kBK;
  s.splits = static_cast<int>(ceil_div(tokens > 0 ? tokens : 1, s.split_len));
  return s;
}

// Split-K plan of the transposing-read G^ kernel (gemm_ghat.hpp) for one or
// more projections of the same tokens (one launch): tm x tn tiles (256 x 256
// when every projection of the launch has r >= 1024, or r >= 256 and 256-row
// tiles pad r no further than 128-row ones; else 384 x 128 when 256 < r and
// 384-row tiles pad no further; else 128 x 256), one split count for all of them,
// at most one workgroup per CU (256 on MI355X), splits of whole 32-token K
// tiles.  Projection j's partial sums take splits x (tiles_r tm) x
// (tiles_m tn) fp32 at byte offset part_off[j].
struct GhatGroupPlan {
  int count;
  int shape, tm, tn;
  int tiles_r[kGhMaxLayers], tiles_m[kGhMaxLayers];
  int tiles, splits;
  int64_t split_len;
  size_t part_off[kGhMaxLayers], bytes;
};

bool ghat_tall_fits(int64_t r) {
  return r > 256 && round_up(r, kGhTallTm) <= round_up(r, kGhTm);
}

// From r = 1024 on the 256 x 256 tiles are taken whatever their padding (at
// most 1280 rows for 1152, 11%): there G^ is bound by the MFMAs and their
// fragment reads, not by HBM, and these tiles read a third fewer fragments per
// MFMA than the 128-row ones (LLaMA-1B's down at r = 1365: G^ phase 42.9 ->
// 41.0 ms per step, measured on one box).
bool ghat_square_fits(int64_t r) {
  return r >= 1024 || (r >= 256 && round_up(r, kGhSqTm) <= round_up(r, kGhTm));
}

GhatGroupPlan ghat_group_plan(int64_t tokens, int count, const int64_t* r, const int64_t* m) {
  GhatGroupPlan g{};
  g.count = count;
  bool square = count > 0, tall = count > 0;
  for (int j = 0; j < count; ++j) {
    square = square && ghat_square_fits(r[j]);
    tall = tall && ghat_tall_fits(r[j]);
  }
  g.shape = square ? 2 : tall ? 1 : 0;
  g.tm = square ? kGhSqTm : tall ? kGhTallTm : kGhTm;
  g.tn = square ? kGhSqTn : tall ? kGhTallTn : kGhTn;
  int64_t tiles = 0;
  for (int j = 0; j < count; ++j) {
    g.tiles_r[j] = static_cast<int>(ceil_div(r[j], g.tm));
    g.tiles_m[j] = static_cast<int>(ceil_div(m[j], g.tn));
    tiles += int64_t(g.tiles_r[j]) * g.tiles_m[j];
  }
  g.tiles = static_cast<int>(tiles);
  const int64_t ktiles = ceil_div(tokens > 0 ? tokens : 1, kGhK);
  int64_t splits = tiles > 0 ? 256 / tiles : 1;
  if (splits < 1) splits = 1;
  if (splits > ktiles) splits = ktiles;
  g.split_len = ceil_div(ktiles, splits) * kGhK;
  g.splits = static_cast<int>(ceil_div(tokens > 0 ? tokens : 1, g.split_len));
  size_t off = 0;
  for (int j = 0; j < count; ++j) {
    g.part_off[j] = off;
    const size_t b = size_t(g.splits) * size_t(g.tiles_r[j]) * g.tm * size_t(g.tiles_m[j]) * g.tn * sizeof(float);
    off += size_t(round_up(static_cast<int64_t>(b), kWsAlign));
  }
  g.bytes = off;
  return g;
}

// The transposing-read kernel takes projection (z, dL/do) of the plan:
// 32-bit buffer offsets over a split plus one K tile.
bool ghat_w4_eligible(const GhatGroupPlan& g, int64_t tokens, int64_t ldz, int64_t lddy) {
  if (tokens < 1 || tokens > (int64_t(1) << 30)) return false;
  const int64_t span = g.split_len + 2 * kGhK;
  const int64_t lim = int64_t(1) << 31;
  return span * ldz * 2 < lim && span * lddy * 2 < lim && ldz < lim / 4 && lddy < lim / 4;
}

size_t ghat_ws_bytes(int64_t tokens, int64_t r, int64_t m) {
  const SplitPlan s = ghat_plan(tokens, r, m);
  const size_t a = size_t(s.splits) * size_t(s.tiles_r) * kGBM * size_t(s.tiles_m) * kGBN * sizeof(float);
  const size_t b = ghat_group_plan(tokens, 1, &r, &m).bytes;
  return a > b ? a : b;  // either path may run (the choice depends on the leading dimensions)
}

int64_t pt_ld(int64_t n) { return round_up(n, kBK); }

// G[j][c] = sum over splits, in order, of part[s][j][c].
int launch_splitk_reduce(const float* part, int splits, int64_t ldp, int64_t plane, int64_t r, int64_t m, float* G,
                         int accumulate, hipStream_t s) {
  if (m % 4 == 0 && aligned16(G)) {
    hipLaunchKernelGGL(k_splitk_reduce4, dim3(static_cast<uint32_t>(ceil_div(r * (m / 4), 256))), dim3(256), 0, s,
                       part, splits, ldp, plane, r, m, G, accumulate);
  } else {
    hipLaunchKernelGGL(k_splitk_reduce, dim3(static_cast<uint32_t>(ceil_div(r * m, 256))), dim3(256), 0, s, part,
                       splits, ldp, plane, r, m, G, accumulate);
  }
  return check_launch("G^ reduce");
}

// G^_j = z_j^T dL/do_j for the projections of a plan: one split-K launch over
// the layer table and one reduction launch.  z[j], dy[j] may be column slices.
int launch_ghat_group(const GhatGroupPlan& g, int64_t tokens, const void* const* z, const int64_t* ldz,
                      const void* const* dy, const int64_t* lddy, float* const* G, const int64_t* r,
                      const int64_t* m, int accumulate, void* ws, hipStream_t s) {
  GhatW4Params p{};
  ReduceBatch rb{};
  rb.accumulate = accumulate;
  char* base = static_cast<char*>(align_ws(ws));
  p.count = rb.count = g.count;
  p.T = static_cast<int>(tokens);
  p.splits = rb.splits = g.splits;
  p.split_len = static_cast<int>(g.split_len);
  p.shape = g.shape;
  int tb = 0, rbk = 0;
  for (int j = 0; j < g.count; ++j) {
    GhatW4Layer& L = p.layer[j];
    L.z = static_cast<const uint16_t*>(z[j]); L.ldz = static_cast<int>(ldz[j]);
    L.dy = static_cast<const uint16_t*>(dy[j]); L.lddy = static_cast<int>(lddy[j]);
    L.part = reinterpret_cast<float*>(base + g.part_off[j]);
    L.r = static_cast<int>(r[j]); L.m = static_cast<int>(m[j]);
    L.tiles_r = g.tiles_r[j]; L.tiles_m = g.tiles_m[j];
    p.tile_begin[j] = tb;
    tb += g.tiles_r[j] * g.tiles_m[j];
    ReduceLayer& R = rb.layer[j];
    R.part = L.part;
    R.G = G[j];
    R.ldp = int64_t(g.tiles_m[j]) * g.tn;
    R.plane = int64_t(g.tiles_r[j]) * g.tm * R.ldp;
    R.r = L.r; R.m = L.m;
    R.mq = static_cast<int>(ceil_div(m[j], 4));
    R.vec = (m[j] % 4 == 0 && aligned16(G[j])) ? 1 : 0;
    rb.begin[j] = rbk;
    rbk += static_cast<int>(ceil_div(r[j] * R.mq, 256));
  }
  p.tile_begin[g.count] = tb;
  rb.begin[g.count] = rbk;
  const hipError_t e = ghat_w4_launch(p, s);
  if (e != hipSuccess) return fail(COMPACT_EHIP, "G^ split-K (bf16): %s", hipGetErrorString(e));
  if (rbk > 0) hipLaunchKernelGGL(k_splitk_reduce_batched, dim3(static_cast<uint32_t>(rbk)), dim3(256), 0, s, rb);
  return check_launch("G^ reduce");
}

// Forward operand of the persistent GEMM, K = n contiguous: rows 0 .. m-1 hold
// W^T, rows round_up(m, 256) .. + r - 1 hold P^T (rows in between are never
// read into a stored output).
// Rows of the forward's staged B operand [W^T; pad; P^T; pad]: y and z each
// start on a 256-row tile.
int64_t stacked_rows(int64_t m, int64_t r) { return round_up(m, kW4Tile) + round_up(r, kW4Tile); }

// Gather-add tables (COMPACT_PROJ_GATHER): [n][s] entries per projection,
// each 256-byte aligned.
size_t gather_table_bytes(int64_t n, int s) {
  return size_t(round_up(n * s * int64_t(sizeof(uint32_t)), int64_t(kWsAlign)));
}

// Forward workspace of `count` projections of widths msum and ranks rsum in
// total: the stacked operand, or with the gather flag W^T alone followed by
// the tables (at most kGatherMaxS draws per row), whichever is larger.
size_t fwd_ws_bytes(int64_t n, int64_t msum, int64_t rsum, int count) {
  const size_t stacked = size_t(stacked_rows(msum, rsum)) * size_t(pt_ld(n)) * sizeof(uint16_t);
  const size_t gathered = size_t(round_up(msum, kW4Tile)) * size_t(pt_ld(n)) * sizeof(uint16_t) +
                          size_t(count) * gather_table_bytes(n, kGatherMaxS);
  return std::max(stacked, gathered) + kWsAlign;
}

// A K-tiled B operand of `rows` rows and K columns fits the persistent GEMM's
// 32-bit buffer offsets.
bool tiled_fits(int64_t rows, int64_t K) { return ceil_div(K, kW4K) * rows * 64 < (int64_t(1) << 31); }

// Workspace of the dx GEMM's K-tiled copy of W: n rows padded to 256, K = m.
size_t dx_stage_bytes(int64_t n, int64_t m) { return size_t(round_up(n, kW4Tile)) * size_t(round_up(m, kW4K)) * 2; }

int w4_tiles(int64_t cols) { return static_cast<int>(ceil_div(cols, kW4Tile)); }
int64_t n_ld(int64_t m) { return round_up(m, 8); }

// The projection of a (validated) compact_proj code: kind, rank and, for the
// sparse projection, the draws per row (0 in the code means the default).
ProjDesc proj_desc(int proj, int64_t r) {
  ProjDesc d{};
  d.kind = proj & 0xFF;
  d.r = static_cast<int>(r);
  const int draws = (proj >> 8) & 0xFF;
  d.s = d.kind == COMPACT_PROJ_SPARSE_JL ? (draws != 0 ? draws : COMPACT_SPARSE_JL_DEFAULT_S) : 0;
  return d;
}

// The forward computes z of a sparse projection by the gather-add launch.
bool proj_gather(int proj) {
  return (proj & 0xFF) == COMPACT_PROJ_SPARSE_JL && (proj & COMPACT_PROJ_GATHER) != 0;
}

// P = scale x the unscaled stream: 1/sqrt(r) for the Gaussian, 1/sqrt(s) for
// the sparse projection, 1 for the identity.
double proj_scale64(int proj, int64_t r) {
  const ProjDesc d = proj_desc(proj, r);
  if (d.kind == COMPACT_PROJ_IDENTITY) return 1.0;
  return 1.0 / std::sqrt(static_cast<double>(d.kind == COMPACT_PROJ_SPARSE_JL ? d.s : r));
}

float proj_scale(int proj, int64_t r) { return static_cast<float>(proj_scale64(proj, r)); }

int set_lds(const void* fn, size_t bytes) {
  if (bytes <= 65536) return COMPACT_OK;
  const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(bytes));
  if (e != hipSuccess) return fail(COMPACT_EHIP, "hipFuncSetAttribute(%zu B LDS): %s", bytes, hipGetErrorString(e));
  return COMPACT_OK;
}

__global__ void k_fill_f32(float* p, int64_t count, float v) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e < count) p[e] = v;
}

int launch_gemm_f32(const GemmF32Params& gp, hipStream_t s, const char* what) {
  GemmF32Params p = gp;
  const int64_t tm = ceil_div(p.M, 64), tn = ceil_div(p.N, 64);
  if (tm == 0 || tn == 0) return COMPACT_OK;
  p.tiles_n = static_cast<int>(tn);
  hipLaunchKernelGGL(k_gemm_f32, dim3(static_cast<uint32_t>(tm * tn)), dim3(256), 0, s, p);
  return check_launch(what);
}

OperandF32 mem_operand(const float* p, int64_t su, int64_t sv, int64_t U, int64_t V) {
  OperandF32 o{};
  o.p = p;
  o.su = su;
  o.sv = sv;
  o.U = U;
  o.V = V;
  return o;
}

OperandF32 pgen_operand(uint64_t seed, int64_t n, int64_t r, int proj) {
  OperandF32 o{};
  o.pgen = 1;
  o.proj = proj_desc(proj, r);
  o.key = philox_key(seed);
  o.U = n;
  o.V = r;
  return o;
}

}  // namespace

extern "C" {

int compact_version(void) { return 100; }

const char* compact_last_error(void) { return g_last_error.c_str(); }

const char* compact_status_string(int status) {
  switch (status) {
    case COMPACT_OK: return "ok";
    case COMPACT_EINVAL: return "invalid argument";
    case COMPACT_EALIGN: return "misaligned pointer or leading dimension";
    case COMPACT_EUNSUPPORTED: return "unsupported configuration";
    case COMPACT_EWORKSPACE: return "workspace missing or too small";
    case COMPACT_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

uint64_t compact_next_seed(uint64_t seed, int64_t t, int64_t T) {
  if (T > 0 && t >= 1 && t % T == 0) return seed + 1u;
  return seed;
}

int64_t compact_saved_activation_elems(int64_t tokens, int64_t n, int64_t r) {
  (void)n;
  return tokens * r;
}

size_t compact_fwd_workspace_bytes(int64_t n, int64_t m, int64_t r, int dtype) {
  if (dtype != COMPACT_BF16 || n < 1 || m < 1 || r < 1) return 0;
  return fwd_ws_bytes(n, m, r, 1);
}

size_t compact_bwd_workspace_bytes(int64_t tokens, int64_t n, int64_t m, int64_t r, int dtype) {
  if (dtype != COMPACT_BF16 || tokens < 0 || n < 1 || m < 1 || r < 1) return 0;
  // the dx GEMM's copy of W, then (after it) the G^ partial sums
  return std::max(ghat_ws_bytes(tokens, r, m), dx_stage_bytes(n, m)) + kWsAlign;
}

// Step scratch of one layer: N [r][n_ld(m)] (compute dtype), then for bf16
// compute the P^T panel [r][pt_ld(n)] bf16.
static size_t step_layer_bytes(int64_t n, int64_t m, int64_t r, int dtype) {
  size_t b = round_up(static_cast<int64_t>(size_t(r) * size_t(n_ld(m)) * elem_size(dtype)), kWsAlign);
  if (dtype == COMPACT_BF16) b += round_up(static_cast<int64_t>(size_t(r) * size_t(pt_ld(n)) * 2), kWsAlign);
  return b;
}

size_t compact_step_workspace_bytes(int64_t n, int64_t m, int64_t r, int dtype) {
  if (n < 1 || m < 1 || r < 1) return 0;
  return step_layer_bytes(n, m, r, dtype) + kWsAlign;
}

}  // extern "C"

namespace {

// Projections that share one input: W = [W_0 | W_1 | ...] (n x msum), y the
// same columns, z = [z_0 | z_1 | ...] (rsum columns).
struct FwdGroup {
  int count;
  int64_t m[kMaxGroup], r[kMaxGroup];
  uint64_t seed[kMaxGroup];
  int64_t msum, rsum;
};

size_t fwd_group_ws_bytes(int64_t n, const FwdGroup& G) { return fwd_ws_bytes(n, G.msum, G.rsum, G.count); }

// The persistent bf16 forward over the stacked operand [W^T; pad to 256;
// P_0^T; P_1^T; ...]: y in the first column tiles, z after.  Sets `taken`
// to false (and launches nothing) when the persistent kernel does not take
// the shape.
int fwd_group_w4(const void* x, int64_t ldx, const void* W, int64_t ldw, void* y, int64_t ldy, void* z,
                 int64_t ldz, int64_t tokens, int64_t n, const FwdGroup& G, int proj, void* ws,
                 hipStream_t s, bool& taken) {
  int st;
  const int64_t ldb = pt_ld(n);
  // gather-add z: the GEMM computes y alone and its B operand is W^T alone
  const bool gather = proj_gather(proj);
  const int64_t rows_b = gather ? round_up(G.msum, kW4Tile) : stacked_rows(G.msum, G.rsum);
  taken = ws != nullptr &&
          gemm_w4_eligible(tokens, n, ldx, ldb, rows_b, ldy, G.msum, gather ? 0 : ldz, gather ? 0 : G.rsum, true) &&
          tiled_fits(rows_b, n);
  if (!taken) return COMPACT_OK;
  uint16_t* bs = static_cast<uint16_t*>(align_ws(ws));
  const int64_t mp = round_up(G.msum, kW4Tile);
  const int sparse_s = proj_desc(proj, 1).s;
  char* tables = reinterpret_cast<char*>(bs) + round_up(rows_b * ldb * int64_t(sizeof(uint16_t)), int64_t(kWsAlign));
  FwdStage fs{};
  fs.W = static_cast<const uint16_t*>(W); fs.ldw = ldw; fs.n = n; fs.m = G.msum;
  fs.b = PanelOut{bs, ldb, rows_b}; fs.ldb = ldb;
  fs.count = G.count;
  fs.kind = proj_desc(proj, 1).kind;
  fs.sparse_s = proj_desc(proj, 1).s;
  fs.tiles_c = static_cast<int>(ceil_div(G.msum, 64));
  fs.pt_begin[0] = 0;
  int64_t row = mp;
  for (int j = 0; j < G.count; ++j) {
    fs.row_off[j] = row;
    fs.r[j] = G.r[j];
    fs.key[j] = philox_key(G.seed[j]);
    fs.pscale[j] = proj_scale(proj, G.r[j]);
    if (gather) {  // a table row per thread
      fs.table[j] = reinterpret_cast<uint32_t*>(tables + size_t(j) * gather_table_bytes(n, sparse_s));
      fs.pt_begin[j + 1] = fs.pt_begin[j] + static_cast<int>(ceil_div(n, 256));
    } else {
      fs.pt_begin[j + 1] = fs.pt_begin[j] + pt_blocks(fs.kind, G.r[j], ldb);
    }
    row += G.r[j];
  }
  const int64_t stage_blocks = fs.pt_begin[G.count] + ceil_div(n, 64) * fs.tiles_c;
  if (stage_blocks > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "staging grid too large");
  hipLaunchKernelGGL(k_fwd_stage_bf16, dim3(static_cast<uint32_t>(stage_blocks)), dim3(256), 0, s, fs);
  if ((st = check_launch("W^T and P^T staging (bf16)"))) return st;
  W4Gemm g{};
  g.A = static_cast<const uint16_t*>(x); g.lda = static_cast<int>(ldx);
  g.M = static_cast<int>(tokens); g.K = static_cast<int>(n);
  g.B = bs; g.ldb = static_cast<int>(ldb); g.rows_b = static_cast<int>(rows_b); g.b_tiled = 1;
  g.seg[0] = W4Seg{static_cast<uint16_t*>(y), static_cast<int>(ldy), static_cast<int>(G.msum), w4_tiles(G.msum)};
  if (!gather)
    g.seg[1] = W4Seg{static_cast<uint16_t*>(z), static_cast<int>(ldz), static_cast<int>(G.rsum), w4_tiles(G.rsum)};
  g.tiles_n = g.seg[0].tiles + g.seg[1].tiles;
  const int64_t tiles = ceil_div(tokens, kW4Tile) * g.tiles_n;
  if (tiles > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "grid too large");
  g.tiles = static_cast<int>(tiles);
  const hipError_t e = gemm_w4_launch(g, W4Use::kForward, s);
  if (e != hipSuccess) return fail(COMPACT_EHIP, "forward GEMM (bf16): %s", hipGetErrorString(e));
  if (!gather) return COMPACT_OK;
  GatherParams gp{};
  gp.x = static_cast<const uint16_t*>(x); gp.ldx = ldx; gp.T = tokens; gp.ldz = ldz;
  gp.n = static_cast<int>(n); gp.s = sparse_s;
  gp.count = G.count;
  int64_t ro = 0;
  gp.chunk_begin[0] = 0;
  for (int j = 0; j < G.count; ++j) {
    gp.layer[j] = GatherLayer{fs.table[j], static_cast<uint16_t*>(z) + ro, static_cast<int>(G.r[j])};
    gp.chunk_begin[j + 1] = gp.chunk_begin[j] + static_cast<int>(ceil_div(G.r[j], kGatherChunk));
    ro += G.r[j];
  }
  const int64_t blocks = ceil_div(tokens, kGatherTok) * gp.chunk_begin[G.count];
  if (blocks > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "gather grid too large");
  hipLaunchKernelGGL(k_sjl_gather, dim3(static_cast<uint32_t>(blocks)), dim3(kGatherTok), 0, s, gp);
  return check_launch("gather-add z (bf16)");
}

}  // namespace

extern "C" {

int compact_fwd(const void* x, int64_t ldx, const void* W, int64_t ldw, void* y, int64_t ldy,
                void* z, int64_t ldz, int64_t tokens, int64_t n, int64_t m, int64_t r,
                uint64_t seed, int proj, int dtype, void* ws, size_t ws_bytes, void* stream) {
  int st;
  if (!valid_dtype(dtype)) return fail(COMPACT_EINVAL, "unknown dtype %d", dtype);
  if ((st = check_shape(tokens, n, m, r, proj))) return st;
  if ((st = check_matrix("x", x, ldx, n, dtype))) return st;
  if ((st = check_matrix("W", W, ldw, m, dtype))) return st;
  if ((st = check_matrix("y", y, ldy, m, dtype))) return st;
  if ((st = check_matrix("z", z, ldz, r, dtype))) return st;
  if (ws != nullptr && ws_bytes < compact_fwd_workspace_bytes(n, m, r, dtype))
    return fail(COMPACT_EWORKSPACE, "forward workspace %zu B < %zu B", ws_bytes, compact_fwd_workspace_bytes(n, m, r, dtype));
  if (tokens == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);

  if (dtype == COMPACT_F32) {
    GemmF32Params gp{};
    gp.A = mem_operand(static_cast<const float*>(x), ldx, 1, tokens, n);
    gp.B = mem_operand(static_cast<const float*>(W), ldw, 1, n, m);
    gp.M = tokens; gp.N = m; gp.K = n; gp.mode = 0;
    gp.out = static_cast<float*>(y); gp.ldo = ldy; gp.scale = 1.0f;
    if ((st = launch_gemm_f32(gp, s, "forward y (fp32)"))) return st;
    gp.B = pgen_operand(seed, n, r, proj);
    gp.N = r; gp.out = static_cast<float*>(z); gp.ldo = ldz; gp.scale = proj_scale(proj, r);
    if ((st = launch_gemm_f32(gp, s, "forward z (fp32)"))) return st;
    return ok();
  }

  const PhiloxKey key = philox_key(seed);
  const float pscale = proj_scale(proj, r);
  const int64_t ldb = pt_ld(n);
  {
    FwdGroup G{};
    G.count = 1; G.m[0] = m; G.r[0] = r; G.seed[0] = seed; G.msum = m; G.rsum = r;
    bool taken = false;
    if ((st = fwd_group_w4(x, ldx, W, ldw, y, ldy, z, ldz, tokens, n, G, proj, ws, s, taken))) return st;
    if (taken) return ok();
  }

  FwdParams p{};
  p.x = static_cast<const uint16_t*>(x); p.ldx = ldx;
  p.W = static_cast<const uint16_t*>(W); p.ldw = ldw;
  p.y = static_cast<uint16_t*>(y); p.ldy = ldy;
  p.z = static_cast<uint16_t*>(z); p.ldz = ldz;
  p.T = tokens; p.n = n; p.m = m; p.r = r;
  p.key = key;
  p.proj = proj_desc(proj, r);
  p.pscale = pscale;
  p.tiles_y = static_cast<int>(ceil_div(m, kBN));
  p.tiles_z = static_cast<int>(ceil_div(r, kBN));
  if (ws != nullptr) {
    uint16_t* pt = static_cast<uint16_t*>(align_ws(ws));
    const int64_t units = proj_t_units(proj_desc(proj, r).kind, r, ldb);
    hipLaunchKernelGGL(k_pstream_t_bf16, dim3(static_cast<uint32_t>(ceil_div(units, 256))), dim3(256), 0, s,
                       proj_desc(proj, r), key, n, pscale, pt, ldb);
    if ((st = check_launch("P panel (bf16)"))) return st;
    p.pt = pt;
    p.ldpt = ldb;
  }
  const int64_t blocks = ceil_div(tokens, kBM) * (p.tiles_y + p.tiles_z);
  if (blocks > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "grid too large");
  {
    auto fn = k_fwd_bf16<kBM, kBN, kWGM, kWGN>;
    if ((st = set_lds(reinterpret_cast<const void*>(fn), kGemmLds))) return st;
    hipLaunchKernelGGL(fn, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), kGemmLds, s, p);
  }
  if ((st = check_launch("fused forward (bf16)"))) return st;
  return ok();
}

size_t compact_fwd_group_workspace_bytes(int64_t n, int32_t count, const int64_t* m, const int64_t* r, int dtype) {
  if (dtype != COMPACT_BF16 || n < 1 || count < 1 || count > kMaxGroup || m == nullptr || r == nullptr) return 0;
  FwdGroup G{};
  G.count = count;
  for (int j = 0; j < count; ++j) {
    if (m[j] < 1 || r[j] < 1) return 0;
    G.msum += m[j];
    G.rsum += r[j];
  }
  return fwd_group_ws_bytes(n, G);
}

int compact_fwd_group(const void* x, int64_t ldx, const void* W, int64_t ldw, void* y, int64_t ldy, void* z,
                      int64_t ldz, int64_t tokens, int64_t n, int32_t count, const int64_t* m, const int64_t* r,
                      const uint64_t* seeds, int proj, int dtype, void* ws, size_t ws_bytes, void* stream) {
  int st;
  if (!valid_dtype(dtype)) return fail(COMPACT_EINVAL, "unknown dtype %d", dtype);
  if (count < 1 || count > kMaxGroup) return fail(COMPACT_EINVAL, "count %d not in [1, %d]", count, kMaxGroup);
  if (m == nullptr || r == nullptr || seeds == nullptr) return fail(COMPACT_EINVAL, "m, r or seeds is NULL");
  FwdGroup G{};
  G.count = count;
  for (int j = 0; j < count; ++j) {
    if ((st = check_shape(tokens, n, m[j], r[j], proj))) {
      const std::string msg = g_last_error;
      return fail(st, "projection %d: %s", j, msg.c_str());
    }
    // every column slice but the last starts on a 16-byte boundary
    if (j + 1 < count && (m[j] % 8 != 0 || r[j] % 8 != 0))
      return fail(COMPACT_EALIGN, "projection %d: m=%lld and r=%lld must be multiples of 8 (all but the last)", j,
                  (long long)m[j], (long long)r[j]);
    G.m[j] = m[j];
    G.r[j] = r[j];
    G.seed[j] = seeds[j];
    G.msum += m[j];
    G.rsum += r[j];
  }
  if ((st = check_matrix("x", x, ldx, n, dtype))) return st;
  if ((st = check_matrix("W", W, ldw, G.msum, dtype))) return st;
  if ((st = check_matrix("y", y, ldy, G.msum, dtype))) return st;
  if ((st = check_matrix("z", z, ldz, G.rsum, dtype))) return st;
  const size_t need = compact_fwd_group_workspace_bytes(n, count, m, r, dtype);
  if (ws != nullptr && ws_bytes < need) return fail(COMPACT_EWORKSPACE, "forward workspace %zu B < %zu B", ws_bytes, need);
  if (tokens == 0) return ok();
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == COMPACT_BF16) {
    bool taken = false;
    if ((st = fwd_group_w4(x, ldx, W, ldw, y, ldy, z, ldz, tokens, n, G, proj, ws, s,
                           taken)))
      return st;
    if (taken) return ok();
  }
  // otherwise one compact_fwd per projection on the column slices
  const size_t esz = elem_size(dtype);
  int64_t mo = 0, ro = 0;
  for (int j = 0; j < count; ++j) {
    if ((st = compact_fwd(x, ldx, static_cast<const char*>(W) + mo * esz, ldw, static_cast<char*>(y) + mo * esz,
                          ldy, static_cast<char*>(z) + ro * esz, ldz, tokens, n, m[j], r[j], seeds[j], proj, dtype,
                          ws, ws_bytes, stream)))
      return st;
    mo += m[j];
    ro += r[j];
  }
  return ok();
}

}  // extern "C"

namespace {

// Alg. 2 for one projection; accumulate: G <- G + z^T dL/do.
int bwd_impl(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z, int64_t ldz, void* dx,
             int64_t lddx, float* G, int64_t tokens, int64_t n, int64_t m, int64_t r, int dtype, int accumulate,
             void* ws, size_t ws_bytes, void* stream) {
  int st;
  if (!valid_dtype(dtype)) return fail(COMPACT_EINVAL, "unknown dtype %d", dtype);
  if ((st = check_shape(tokens, n, m, r, COMPACT_PROJ_GAUSSIAN))) return st;
  if (dx == nullptr && G == nullptr) return fail(COMPACT_EINVAL, "dx and G are both NULL");
  if ((st = check_matrix("dy", dy, lddy, m, dtype))) return st;
  if (dx != nullptr) {
    if ((st = check_matrix("W", W, ldw, m, dtype))) return st;
    if ((st = check_matrix("dx", dx, lddx, n, dtype))) return st;
  }
  if (G != nullptr) {
    if ((st = check_matrix("z", z, ldz, r, dtype))) return st;
    if ((st = check_dense("G", G))) return st;
    const size_t need = compact_bwd_workspace_bytes(tokens, n, m, r, dtype);
    if (need > 0 && (ws == nullptr || ws_bytes < need))
      return fail(COMPACT_EWORKSPACE, "backward workspace %zu B < %zu B", ws_bytes, need);
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (tokens == 0) {
    if (G != nullptr && !accumulate) {  // a sum over no tokens
      hipLaunchKernelGGL(k_fill_f32, dim3(static_cast<uint32_t>(ceil_div(r * m, 256))), dim3(256), 0, s, G, r * m, 0.0f);
      if ((st = check_launch("zero G"))) return st;
    }
    return ok();
  }

  if (dtype == COMPACT_F32) {
    if (dx != nullptr) {
      GemmF32Params gp{};
      gp.A = mem_operand(static_cast<const float*>(dy), lddy, 1, tokens, m);
      gp.B = mem_operand(static_cast<const float*>(W), 1, ldw, m, n);
      gp.M = tokens; gp.N = n; gp.K = m; gp.mode = 0;
      gp.out = static_cast<float*>(dx); gp.ldo = lddx; gp.scale = 1.0f;
      if ((st = launch_gemm_f32(gp, s, "dx (fp32)"))) return st;
    }
    if (G != nullptr) {
      GemmF32Params gp{};
      gp.A = mem_operand(static_cast<const float*>(z), 1, ldz, r, tokens);
      gp.B = mem_operand(static_cast<const float*>(dy), lddy, 1, tokens, m);
      gp.M = r; gp.N = m; gp.K = tokens; gp.mode = accumulate ? 2 : 0;
      gp.out = G; gp.ldo = m; gp.scale = 1.0f;
      if ((st = launch_gemm_f32(gp, s, "G^ (fp32)"))) return st;
    }
    return ok();
  }

  const int64_t npad = round_up(n, kW4Tile);
  const bool stage_w = ws != nullptr && ws_bytes >= dx_stage_bytes(n, m) + kWsAlign && tiled_fits(npad, m);
  if (dx != nullptr && gemm_w4_eligible(tokens, m, lddy, ldw, n, lddx, n, 0, 0, stage_w)) {
    // persistent GEMM: dx = dL/do W^T with W [n][m] as the K-contiguous B,
    // copied into the K-tiled layout first when the workspace holds it
    // (always when m % 8 != 0: the copy is zero past m)
    W4Gemm g{};
    g.A = static_cast<const uint16_t*>(dy); g.lda = static_cast<int>(lddy);
    g.M = static_cast<int>(tokens); g.K = static_cast<int>(m);
    g.B = static_cast<const uint16_t*>(W); g.ldb = static_cast<int>(ldw); g.rows_b = static_cast<int>(n);
    if (stage_w) {
      uint16_t* wt = static_cast<uint16_t*>(align_ws(ws));
      const int64_t units = n * ceil_div(m, 8);
      hipLaunchKernelGGL(k_stage_rows_bf16, dim3(static_cast<uint32_t>(ceil_div(units, 256))), dim3(256), 0, s,
                         static_cast<const uint16_t*>(W), ldw, n, m, PanelOut{wt, 0, npad});
      if ((st = check_launch("W K-tile staging (bf16)"))) return st;
      g.B = wt; g.rows_b = static_cast<int>(npad); g.b_tiled = 1;
    }
    g.seg[0] = W4Seg{static_cast<uint16_t*>(dx), static_cast<int>(lddx), static_cast<int>(n), w4_tiles(n)};
    g.seg[1] = W4Seg{static_cast<uint16_t*>(dx), static_cast<int>(lddx), 0, 0};
    g.tiles_n = g.seg[0].tiles;
    const int64_t tiles = ceil_div(tokens, kW4Tile) * g.tiles_n;
    if (tiles > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "grid too large");
    g.tiles = static_cast<int>(tiles);
    const hipError_t e = gemm_w4_launch(g, W4Use::kDx, s);
    if (e != hipSuccess) return fail(COMPACT_EHIP, "dx GEMM (bf16): %s", hipGetErrorString(e));
  } else if (dx != nullptr) {
    DxParams p{};
    p.dy = static_cast<const uint16_t*>(dy); p.lddy = lddy;
    p.W = static_cast<const uint16_t*>(W); p.ldw = ldw;
    p.dx = static_cast<uint16_t*>(dx); p.lddx = lddx;
    p.T = tokens; p.n = n; p.m = m;
    p.tiles_n = static_cast<int>(ceil_div(n, kBN));
    const int64_t blocks = ceil_div(tokens, kBM) * p.tiles_n;
    auto fn = k_dx_bf16<kBM, kBN, kWGM, kWGN>;
    if ((st = set_lds(reinterpret_cast<const void*>(fn), kGemmLds))) return st;
    hipLaunchKernelGGL(fn, dim3(static_cast<uint32_t>(blocks)), dim3(kThreads), kGemmLds, s, p);
    if ((st = check_launch("dx (bf16)"))) return st;
  }
  const GhatGroupPlan gp = ghat_group_plan(tokens, 1, &r, &m);
  if (G != nullptr && ghat_w4_eligible(gp, tokens, ldz, lddy)) {
    if ((st = launch_ghat_group(gp, tokens, &z, &ldz, &dy, &lddy, &G, &r, &m, accumulate, ws, s))) return st;
  } else if (G != nullptr) {
    const SplitPlan sp = ghat_plan(tokens, r, m);
    GhatParams p{};
    p.z = static_cast<const uint16_t*>(z); p.ldz = ldz;
    p.dy = static_cast<const uint16_t*>(dy); p.lddy = lddy;
    p.part = static_cast<float*>(align_ws(ws));
    p.T = tokens; p.r = r; p.m = m;
    p.tiles_r = sp.tiles_r; p.tiles_m = sp.tiles_m; p.splits = sp.splits; p.split_len = sp.split_len;
    const int64_t blocks = int64_t(sp.tiles_r) * sp.tiles_m * sp.splits;
    hipLaunchKernelGGL((k_ghat_bf16<kGBM, kGBN, kGWGM, kGWGN>), dim3(static_cast<uint32_t>(blocks)),
                       dim3(kGThreads), kGhatLds, s, p);
    if ((st = check_launch("G^ split-K (bf16)"))) return st;
    const int64_t ldp = int64_t(sp.tiles_m) * kGBN, plane = int64_t(sp.tiles_r) * kGBM * ldp;
    if ((st = launch_splitk_reduce(p.part, sp.splits, ldp, plane, r, m, G, accumulate, s))) return st;
  }
  return ok();
}

}  // namespace

extern "C" {

int compact_bwd(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z,
                int64_t ldz, void* dx, int64_t lddx, float* G, int64_t tokens, int64_t n,
                int64_t m, int64_t r, int dtype, void* ws, size_t ws_bytes, void* stream) {
  return bwd_impl(dy, lddy, W, ldw, z, ldz, dx, lddx, G, tokens, n, m, r, dtype, 0, ws, ws_bytes, stream);
}

size_t compact_bwd_group_workspace_bytes(int64_t tokens, int64_t n, int32_t count, const int64_t* m,
                                         const int64_t* r, int dtype) {
  if (dtype != COMPACT_BF16 || tokens < 0 || count < 1 || count > kGhMaxLayers || m == nullptr || r == nullptr)
    return 0;
  for (int j = 0; j < count; ++j)
    if (m[j] < 1 || r[j] < 1) return 0;
  // the one-launch plan, or compact_bwd on each slice when it does not apply
  size_t need = ghat_group_plan(tokens, count, r, m).bytes;
  int64_t msum = 0;
  for (int j = 0; j < count; ++j) {
    need = std::max(need, ghat_ws_bytes(tokens, r[j], m[j]));
    msum += m[j];
  }
  if (n >= 1) need = std::max(need, dx_stage_bytes(n, msum));  // the dx GEMM's copy of W
  return need + kWsAlign;
}

int compact_bwd_group(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z, int64_t ldz,
                      void* dx, int64_t lddx, float* const* G, int64_t tokens, int64_t n, int32_t count,
                      const int64_t* m, const int64_t* r, int dtype, int accumulate, void* ws, size_t ws_bytes,
                      void* stream) {
  int st;
  if (accumulate != 0 && accumulate != 1) return fail(COMPACT_EINVAL, "accumulate must be 0 or 1");
  if (!valid_dtype(dtype)) return fail(COMPACT_EINVAL, "unknown dtype %d", dtype);
  if (count < 1 || count > kGhMaxLayers) return fail(COMPACT_EINVAL, "group of %d projections (1 .. %d)", count, kGhMaxLayers);
  if (m == nullptr || r == nullptr) return fail(COMPACT_EINVAL, "m or r array is NULL");
  if (dx == nullptr && G == nullptr) return fail(COMPACT_EINVAL, "dx and G are both NULL");
  int64_t msum = 0, rsum = 0;
  for (int j = 0; j < count; ++j) {
    if ((st = check_shape(tokens, n, m[j], r[j], COMPACT_PROJ_GAUSSIAN))) return st;
    if (j + 1 < count && (m[j] % 8 != 0 || r[j] % 8 != 0))
      return fail(COMPACT_EALIGN, "group member %d: m and r of all but the last projection must be multiples of 8", j);
    if (G != nullptr && G[j] == nullptr) return fail(COMPACT_EINVAL, "G[%d] is NULL", j);
    if (G != nullptr && (st = check_dense("G", G[j]))) return st;
    msum += m[j];
    rsum += r[j];
  }
  if ((st = check_matrix("dy", dy, lddy, msum, dtype))) return st;
  if (dx != nullptr) {
    if ((st = check_matrix("W", W, ldw, msum, dtype))) return st;
    if ((st = check_matrix("dx", dx, lddx, n, dtype))) return st;
  }
  if (G != nullptr) {
    if ((st = check_matrix("z", z, ldz, rsum, dtype))) return st;
    const size_t need = compact_bwd_group_workspace_bytes(tokens, n, count, m, r, dtype);
    if (need > 0 && (ws == nullptr || ws_bytes < need))
      return fail(COMPACT_EWORKSPACE, "backward workspace %zu B < %zu B", ws_bytes, need);
  }
  // dL/dx summed over the projections: one GEMM over the concatenated weight
  if (dx != nullptr) {
    if ((st = compact_bwd(dy, lddy, W, ldw, nullptr, ldz, dx, lddx, nullptr, tokens, n, msum, 1, dtype, ws,
                          ws_bytes, stream)))
      return st;
  }
  if (G == nullptr) return ok();
  const size_t esz = elem_size(dtype);
  const void* zs[kGhMaxLayers];
  const void* dys[kGhMaxLayers];
  int64_t ldzs[kGhMaxLayers], lddys[kGhMaxLayers];
  int64_t mo = 0, ro = 0;
  for (int j = 0; j < count; ++j) {
    zs[j] = static_cast<const char*>(z) + ro * esz;
    dys[j] = static_cast<const char*>(dy) + mo * esz;
    ldzs[j] = ldz;
    lddys[j] = lddy;
    mo += m[j];
    ro += r[j];
  }
  const GhatGroupPlan gp = ghat_group_plan(tokens, count, r, m);
  if (dtype == COMPACT_BF16 && tokens > 0 && ghat_w4_eligible(gp, tokens, ldz, lddy)) {
    if ((st = launch_ghat_group(gp, tokens, zs, ldzs, dys, lddys, G, r, m, accumulate, ws,
                                static_cast<hipStream_t>(stream))))
      return st;
    return ok();
  }
  // otherwise G^ of each projection on its own
  for (int j = 0; j < count; ++j)
    if ((st = bwd_impl(dys[j], lddy, nullptr, ldw, zs[j], ldz, nullptr, lddx, G[j], tokens, n, m[j], r[j], dtype,
                       accumulate, ws, ws_bytes, stream)))
      return st;
  return ok();
}

}  // extern "C"

namespace {

// Per-layer launch description of Alg. 3 (Adam + P^T staging, decompression).
struct StepPlan {
  AdamLayer al;
  int adam_blocks, pt_blocks;
  DecW4Layer dl;
  int dec_tiles;
};

int validate_step(const void* W, int64_t ldw, const float* G, const float* M, const float* V, int64_t n,
                  int64_t m, int64_t r, int64_t t, double lr, double beta1, double beta2, double eps,
                  double alpha, int proj, int dtype, int w_dtype) {
  int st;
  if (!valid_dtype(dtype) || !valid_dtype(w_dtype)) return fail(COMPACT_EINVAL, "unknown dtype");
  if ((st = check_shape(0, n, m, r, proj))) return st;
  if ((st = check_matrix("W", W, ldw, m, w_dtype))) return st;
  if ((st = check_dense("G", G)) || (st = check_dense("M", M)) || (st = check_dense("V", V))) return st;
  if (t < 1) return fail(COMPACT_EINVAL, "step index t=%lld must be >= 1", (long long)t);
  if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0))
    return fail(COMPACT_EINVAL, "betas must lie in [0, 1)");
  if (!(eps > 0.0) || !std::isfinite(eps)) return fail(COMPACT_EINVAL, "eps must be > 0");
  if (!(lr >= 0.0) || !std::isfinite(lr) || !std::isfinite(alpha)) return fail(COMPACT_EINVAL, "bad lr or alpha");
  if (dtype == COMPACT_F32 && w_dtype != COMPACT_F32)
    return fail(COMPACT_EUNSUPPORTED, "fp32 decompression needs fp32 W");
  if (dtype == COMPACT_BF16 && !dec_w4_eligible(n, m, r, ldw, n_ld(m), pt_ld(n), w_dtype == COMPACT_F32))
    return fail(COMPACT_EUNSUPPORTED, "decompression: shape too large for 32-bit offsets (n=%lld m=%lld r=%lld ldw=%lld)",
                (long long)n, (long long)m, (long long)r, (long long)ldw);
  return COMPACT_OK;
}

// Adam constants of one step: 1 - beta and the bias corrections formed in fp64
// and rounded once.
AdamConsts adam_consts(int64_t t, double beta1, double beta2, double eps, int proj, int dtype) {
  AdamConsts c{};
  c.b1 = static_cast<float>(beta1);
  c.b2 = static_cast<float>(beta2);
  c.omb1 = static_cast<float>(1.0 - beta1);
  c.omb2 = static_cast<float>(1.0 - beta2);
  c.bc1 = static_cast<float>(1.0 - std::pow(beta1, static_cast<double>(t)));
  c.bc2 = static_cast<float>(1.0 - std::pow(beta2, static_cast<double>(t)));
  c.eps = static_cast<float>(eps);
  c.n_f32 = dtype == COMPACT_F32;
  c.kind = proj_desc(proj, 1).kind;
  c.sparse_s = proj_desc(proj, 1).s;
  return c;
}

// `ws` is this layer's scratch (step_layer_bytes, 256-byte aligned).
void plan_step(void* W, int64_t ldw, const float* G, float* M, float* V, int64_t n, int64_t m, int64_t r,
               uint64_t seed, double lr, double alpha, int proj, int dtype, void* ws, StepPlan& P) {
  const int64_t ldn = n_ld(m), ldpt = pt_ld(n);
  char* base = static_cast<char*>(ws);
  AdamLayer& a = P.al;
  a = AdamLayer{};
  a.G = G; a.M = M; a.V = V; a.N = base;
  a.ldn = static_cast<int>(ldn);
  a.r = static_cast<int>(r);
  a.m = static_cast<int>(m);
  a.n = static_cast<int>(n);
  a.key = philox_key(seed);
  P.adam_blocks = adam_blocks(r, m);
  P.pt_blocks = 0;
  P.dec_tiles = 0;
  const double coef64 = lr * alpha * proj_scale64(proj, r);
  DecW4Layer& d = P.dl;
  d = DecW4Layer{};
  d.coef = static_cast<float>(coef64);
  if (dtype != COMPACT_BF16) return;
  uint16_t* pt = reinterpret_cast<uint16_t*>(
      base + round_up(static_cast<int64_t>(size_t(r) * size_t(ldn) * elem_size(dtype)), kWsAlign));
  a.pt = pt;
  a.ldpt = static_cast<int>(ldpt);
  P.pt_blocks = pt_blocks(proj_desc(proj, r).kind, r, ldpt);
  d.W = W; d.ldw = static_cast<int>(ldw);
  d.N = static_cast<const uint16_t*>(a.N); d.ldn = static_cast<int>(ldn);
  d.pt = pt; d.ldpt = static_cast<int>(ldpt);
  d.n = static_cast<int>(n); d.m = static_cast<int>(m); d.r = static_cast<int>(r);
  d.tiles_c = static_cast<int>(ceil_div(m, kDecT));
  P.dec_tiles = static_cast<int>(ceil_div(n, kDecT) * d.tiles_c);
}

// Adam (+ P^T staging) for every layer of `plans`, then the decompression, in
// equal groups of at most kStepBatch layers per launch.
int launch_step_groups(const std::vector<StepPlan>& plans, const AdamConsts& c, int dtype, int w_dtype,
                       hipStream_t s) {
  int st;
  const int count = static_cast<int>(plans.size());
  const int groups = (count + kStepBatch - 1) / kStepBatch;
  const int per = (count + groups - 1) / groups;
  for (int i0 = 0; i0 < count; i0 += per) {
    StepBatch b{};
    b.c = c;
    b.count = std::min(per, count - i0);
    b.adam_begin[0] = 0;
    b.pt_begin[0] = 0;
    for (int j = 0; j < b.count; ++j) {
      const StepPlan& P = plans[i0 + j];
      b.layer[j] = P.al;
      b.adam_begin[j + 1] = b.adam_begin[j] + P.adam_blocks;
      b.pt_begin[j + 1] = b.pt_begin[j] + P.pt_blocks;
    }
    const int blocks = b.adam_begin[b.count] + b.pt_begin[b.count];
    hipLaunchKernelGGL(k_adam_pt_batched, dim3(static_cast<uint32_t>(blocks)), dim3(256), 0, s, b);
    if ((st = check_launch("Adam and P^T staging"))) return st;
  }
  if (dtype != COMPACT_BF16) return COMPACT_OK;
  static_assert(kDecBatch >= kStepBatch, "one decompression launch per Adam launch");
  for (int i0 = 0; i0 < count; i0 += per) {
    DecW4Batch d{};
    d.count = std::min(per, count - i0);
    d.begin[0] = 0;
    for (int j = 0; j < d.count; ++j) {
      d.layer[j] = plans[i0 + j].dl;
      d.begin[j + 1] = d.begin[j] + plans[i0 + j].dec_tiles;
    }
    const hipError_t e = dec_w4_launch(d, w_dtype == COMPACT_F32, s);
    if (e != hipSuccess) return fail(COMPACT_EHIP, "decompression launch: %s", hipGetErrorString(e));
  }
  return COMPACT_OK;
}

}  // namespace

extern "C" {

int compact_step(void* W, int64_t ldw, const float* G, float* M, float* V, int64_t n,
                 int64_t m, int64_t r, uint64_t seed, int64_t t, double lr, double beta1,
                 double beta2, double eps, double alpha, int proj, int dtype, int w_dtype,
                 void* ws, size_t ws_bytes, void* stream) {
  int st;
  if ((st = validate_step(W, ldw, G, M, V, n, m, r, t, lr, beta1, beta2, eps, alpha, proj, dtype, w_dtype)))
    return st;
  const size_t need = compact_step_workspace_bytes(n, m, r, dtype);
  if (ws == nullptr || ws_bytes < need) return fail(COMPACT_EWORKSPACE, "step workspace %zu B < %zu B", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<StepPlan> plans(1);
  plan_step(W, ldw, G, M, V, n, m, r, seed, lr, alpha, proj, dtype, align_ws(ws), plans[0]);
  if ((st = launch_step_groups(plans, adam_consts(t, beta1, beta2, eps, proj, dtype), dtype, w_dtype, s))) return st;
  if (dtype == COMPACT_F32) {
    GemmF32Params gp{};
    gp.A = pgen_operand(seed, n, r, proj);
    gp.B = mem_operand(static_cast<const float*>(plans[0].al.N), plans[0].al.ldn, 1, r, m);
    gp.M = n; gp.N = m; gp.K = r; gp.mode = 1;
    gp.out = static_cast<float*>(W); gp.ldo = ldw; gp.coef = plans[0].dl.coef;
    if ((st = launch_gemm_f32(gp, s, "decompress (fp32)"))) return st;
  }
  return ok();
}

size_t compact_step_batched_workspace_bytes(const compact_layer* layers, int32_t count, int dtype) {
  if (layers == nullptr || count <= 0) return 0;
  size_t total = kWsAlign;
  for (int32_t i = 0; i < count; ++i) total += step_layer_bytes(layers[i].n, layers[i].m, layers[i].r, dtype);
  return total;
}

int compact_step_batched(const compact_layer* layers, int32_t count, int64_t t, double lr,
                         double beta1, double beta2, double eps, int proj, int dtype, int w_dtype,
                         void* ws, size_t ws_bytes, void* stream) {
  int st;
  if (count < 0 || (count > 0 && layers == nullptr)) return fail(COMPACT_EINVAL, "bad layer list");
  if (count == 0) return ok();
  if (dtype != COMPACT_BF16) return fail(COMPACT_EUNSUPPORTED, "batched step supports bf16 compute only");
  for (int32_t i = 0; i < count; ++i) {
    const compact_layer& L = layers[i];
    if ((st = validate_step(L.W, L.ldw, L.G, L.M, L.V, L.n, L.m, L.r, t, lr, beta1, beta2, eps, L.alpha, proj,
                            dtype, w_dtype))) {
      const std::string msg = g_last_error;
      return fail(st, "layer %d: %s", static_cast<int>(i), msg.c_str());
    }
  }
  const size_t need = compact_step_batched_workspace_bytes(layers, count, dtype);
  if (ws == nullptr || ws_bytes < need) return fail(COMPACT_EWORKSPACE, "batched step workspace %zu B < %zu B", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  std::vector<StepPlan> plans(static_cast<size_t>(count));
  char* cursor = static_cast<char*>(align_ws(ws));
  for (int32_t i = 0; i < count; ++i) {
    const compact_layer& L = layers[i];
    plan_step(L.W, L.ldw, L.G, L.M, L.V, L.n, L.m, L.r, L.seed, lr, L.alpha, proj, dtype, cursor, plans[i]);
    cursor += step_layer_bytes(L.n, L.m, L.r, dtype);
  }
  if ((st = launch_step_groups(plans, adam_consts(t, beta1, beta2, eps, proj, dtype), dtype, w_dtype, s))) return st;
  return ok();
}

// Scratch of compact_bwd_noalloc: one array per GPU, part of the library's
// code object (allocated by the runtime when the module is loaded on a device,
// held until the process ends).  Host code never passes `scratch` itself to a
// kernel: its name is a host-side stand-in; the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[COMPACT_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];

// The device address of this device's `scratch` (the current device), looked
// up on the first call on the device.
int scratch_ptr(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(COMPACT_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices) return fail(COMPACT_EUNSUPPORTED, "device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(COMPACT_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return COMPACT_OK;
}

}  // namespace

int compact_bwd_noalloc(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z, int64_t ldz,
                        void* dx, int64_t lddx, float* G, int64_t tokens, int64_t n, int64_t m, int64_t r,
                        int dtype, void* stream) {
  int st;
  if (!valid_dtype(dtype)) return fail(COMPACT_EINVAL, "unknown dtype %d", dtype);
  if ((st = check_shape(tokens, n, m, r, COMPACT_PROJ_GAUSSIAN))) return st;
  const size_t need = G != nullptr ? compact_bwd_workspace_bytes(tokens, n, m, r, dtype) : 0;
  if (need > COMPACT_NOALLOC_SCRATCH_BYTES)
    return fail(COMPACT_EUNSUPPORTED, "backward needs %zu B of scratch; compact_bwd_noalloc has %zu B (use compact_bwd)",
                need, static_cast<size_t>(COMPACT_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws))) return st;
  // with a whole scratch (not only `need` bytes) compact_bwd also stages W
  // for dx whenever that fits, as it does with a caller workspace this large
  return compact_bwd(dy, lddy, W, ldw, z, ldz, dx, lddx, G, tokens, n, m, r, dtype, ws,
                     COMPACT_NOALLOC_SCRATCH_BYTES, stream);
}

int compact_pstream(uint64_t seed, int64_t n, int64_t r, float* out, int64_t ld, void* stream) {
  if (n < 1 || r < 1) return fail(COMPACT_EINVAL, "bad shape n=%lld r=%lld", (long long)n, (long long)r);
  if (out == nullptr) return fail(COMPACT_EINVAL, "out is NULL");
  if (ld < r) return fail(COMPACT_EINVAL, "ld < r");
  if (n > (int64_t(1) << 31) || r > (int64_t(1) << 31)) return fail(COMPACT_EUNSUPPORTED, "n and r must be below 2^31");
  const int64_t quads = ceil_div(n, 4) * r;
  hipLaunchKernelGGL(k_pstream_f32, dim3(static_cast<uint32_t>(ceil_div(quads, 256))), dim3(256), 0,
                     static_cast<hipStream_t>(stream), philox_key(seed), n, r, out, ld);
  int st;
  if ((st = check_launch("P stream"))) return st;
  return ok();
}

int compact_projection(uint64_t seed, int64_t n, int64_t r, int proj, float* out, int64_t ld, void* stream) {
  int st;
  if ((st = check_shape(0, n, 1, r, proj))) return st;
  if (out == nullptr) return fail(COMPACT_EINVAL, "out is NULL");
  if (ld < r) return fail(COMPACT_EINVAL, "ld < r");
  const int64_t quads = ceil_div(n, 4) * r;
  if (ceil_div(quads, 256) > 0x7FFFFFFF) return fail(COMPACT_EUNSUPPORTED, "n x r too large");
  hipLaunchKernelGGL(k_projection_f32, dim3(static_cast<uint32_t>(ceil_div(quads, 256))), dim3(256), 0,
                     static_cast<hipStream_t>(stream), proj_desc(proj, r), philox_key(seed), n, out, ld);
  if ((st = check_launch("projection stream"))) return st;
  return ok();
}

int compact_pstream_boxmuller(const uint32_t* a, const uint32_t* b, float* g_even, float* g_odd,
                              int64_t count, void* stream) {
  if (count < 0) return fail(COMPACT_EINVAL, "count < 0");
  if (count == 0) return ok();
  if (!a || !b || !g_even || !g_odd) return fail(COMPACT_EINVAL, "NULL pointer");
  if (count > (int64_t(1) << 40)) return fail(COMPACT_EUNSUPPORTED, "count too large");
  hipLaunchKernelGGL(k_boxmuller, dim3(static_cast<uint32_t>(ceil_div(count, 256))), dim3(256), 0,
                     static_cast<hipStream_t>(stream), a, b, g_even, g_odd, count);
  int st;
  if ((st = check_launch("Box-Muller"))) return st;
  return ok();
}

}  // extern "C"
