/*
 * compact.h — C ABI of the CompAct compressed linear layer on AMD MI355X (gfx950).
 *
 * CompAct (Shamshoum et al., "CompAct: Compressed Activations for
 * Memory-Efficient LLM Training") replaces the activation a linear layer saves
 * for its backward pass, x in R^{T x n} (T = b*l tokens), by the projection
 * z = x P in R^{T x r}, where P in R^{n x r} is a Gaussian random matrix with
 * entries N(0, 1/r) drawn from a per-layer seed and never stored (§3.2, §3.3).
 * The weight gradient is then computed compressed, G^ = z^T dL/do (r x m),
 * Adam runs on r x m moments, and the update is decompressed as P N (§3.2,
 * Alg. 1-3).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - All matrices are row-major with an explicit leading dimension (ld, in
 *    elements).  W is n x m as in the paper (input features by output
 *    features), NOT the out x in layout of torch.nn.Linear.
 *  - All tensor pointers are DEVICE pointers owned by the caller; the library
 *    allocates nothing and frees nothing.  Scratch memory comes from a
 *    caller-provided workspace whose size is given by the matching
 *    *_workspace_bytes function (compact_bwd_noalloc alone uses a scratch
 *    array of the library's device code instead, see there).
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Every call is asynchronous and ordered on that stream; the call returns
 *    after the launches are enqueued.
 *  - dtype COMPACT_BF16: x, W, y, z, dL/do, dx are bfloat16, stored as 16-bit
 *    patterns; accumulation is fp32 (MFMA); results are rounded to nearest-even.
 *    The compressed gradient G^ and the Adam moments M, V are always fp32.
 *    dtype COMPACT_F32: every tensor is fp32.
 *  - Alignment: tensor base pointers must be 16-byte aligned; bf16 leading
 *    dimensions must be multiples of 8 and fp32 leading dimensions multiples
 *    of 4 (rows start on 16-byte boundaries).  A row of n = 5461 bf16 values,
 *    for instance, needs ld >= 5464.
 *  - Errors: every entry point validates its arguments on the host before any
 *    launch and returns a compact_status; nothing is launched when the result
 *    is not COMPACT_OK.  A failed launch returns COMPACT_EHIP.  A fault while a
 *    kernel runs surfaces at the caller's next synchronisation.  The library
 *    never aborts, throws or prints; compact_last_error() gives a description
 *    of the last failure on the calling thread.
 *  - Projection: the caller passes the same seed to compact_fwd and to
 *    compact_step of the same iteration (Alg. 1 and Alg. 3 re-sample P from
 *    the layer seed); compact_bwd needs no seed (Alg. 2 uses only z and W).
 *  - Non-finite values are not checked for and never masked: a NaN or an
 *    infinity in an input reaches exactly the outputs that depend on it under
 *    IEEE arithmetic (a NaN in token t of x: row t of y and z; a NaN in
 *    dL/do at (t, c): row t of dx, column c of G^, M, V and of W).  Other
 *    elements are unaffected.
 */
#ifndef COMPACT_H_
#define COMPACT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  COMPACT_OK = 0,
  COMPACT_EINVAL = -1,        /* bad size, pointer, rank or hyper-parameter */
  COMPACT_EALIGN = -2,        /* pointer or leading dimension misaligned    */
  COMPACT_EUNSUPPORTED = -3,  /* valid request the library does not support */
  COMPACT_EWORKSPACE = -4,    /* workspace missing or too small             */
  COMPACT_EHIP = -5           /* a HIP runtime call or launch failed        */
} compact_status;

typedef enum { COMPACT_F32 = 0, COMPACT_BF16 = 1 } compact_dtype;

typedef enum {
  COMPACT_PROJ_GAUSSIAN = 0,  /* P = G / sqrt(r), G the seeded N(0,1) stream  */
  COMPACT_PROJ_IDENTITY = 1,  /* P = I (requires r == n): uncompressed layer  */
  COMPACT_PROJ_SPARSE_JL = 2  /* P = S / sqrt(s), S the seeded sparse JL
                                 stream with s signed draws per row (below)  */
} compact_proj;

/*
 * Sparse Johnson-Lindenstrauss projection (the ablation's sparse JL matrices,
 * §5, after Dasgupta, Kumar and Sarlos 2010; the paper gives no parameters).
 * The `proj` argument COMPACT_PROJ_SPARSE_JL_S(s) selects s draws per row,
 * 1 <= s <= 64; plain COMPACT_PROJ_SPARSE_JL means s = 8.  Row i of S receives
 * s unit draws with random signs at hashed columns (draws on one column add):
 *   draw q of row i, 0 <= q < s:
 *     (w0, w1, w2, w3) = Philox4x32-10((i, q >> 1, 0x4A4C5350, 0), key(seed))
 *     (a, b) = (w0, w1) for even q, (w2, w3) for odd q
 *     column floor(a r / 2^32), sign +1 if b < 2^31 else -1
 * with key(seed) as for the Gaussian stream (compact_pstream).  E[P P^T] = I
 * as for the Gaussian, so Alg. 3's decompression stays unbiased.  S holds
 * small integers; the forward rounds P = S / sqrt(s) to bf16 once (exact for
 * s = 1, 4, 16, 64) and the update applies 1/sqrt(s) in fp32.
 */
#define COMPACT_SPARSE_JL_DEFAULT_S 8
#define COMPACT_PROJ_SPARSE_JL_S(s) (COMPACT_PROJ_SPARSE_JL | ((s) << 8))

/*
 * Gather-add forward for the sparse projection (the sparse JL route of §6-§7
 * to cheaper projections: z as sums of signed input features rather than a
 * dense product).  OR-ed into a sparse code with at most
 * COMPACT_GATHER_MAX_S draws per row, it changes how compact_fwd and
 * compact_fwd_group compute z on the bf16 path with a workspace: y comes from
 * the persistent GEMM over W^T alone, and z from one gather launch in which
 * the lane of token t adds, in order of the input feature i and then of the
 * draw, x[t][i] * bf16(S[i][c] / sqrt(s)) into an fp32 sum per column c (draws
 * of row i that share a column are merged first, and entries with S[i][c] = 0
 * are skipped), rounded once to bf16.  y is bitwise the same as without the
 * flag; z differs from the GEMM paths only in the order of the fp32 additions.
 * A NaN or infinity at x[t][i] then reaches z[t][c] only where S[i][c] != 0.
 * The flag is ignored on the fp32 path, without a workspace and by every
 * other entry point (the backward and Alg. 3 do not depend on it), so one
 * code can be passed to all of them.  It is an alternative for measurement,
 * not a faster path: on MI355X the LDS float additions it is built on make
 * it much slower than the MFMA columns of the fused GEMM at every s.
 */
#define COMPACT_PROJ_GATHER (1 << 16)
#define COMPACT_GATHER_MAX_S 16

/*
 * Forward pass, Alg. 1:  y = x W  and  z = x P.
 *
 *   x  [tokens x n]  (ld ldx)  input activations
 *   W  [n x m]       (ld ldw)  weight
 *   y  [tokens x m]  (ld ldy)  output o = x W
 *   z  [tokens x r]  (ld ldz)  compressed activation saved for the backward pass
 *   seed  layer seed; P[i][j] = G(seed, i, j) / sqrt(r) (the P stream, below)
 *   proj  COMPACT_PROJ_GAUSSIAN, COMPACT_PROJ_IDENTITY with r == n, or
 *         COMPACT_PROJ_SPARSE_JL[_S(s)] (P = S / sqrt(s), above)
 *   ws, ws_bytes  optional workspace of at least
 *         compact_fwd_workspace_bytes(n, m, r, dtype) bytes (bf16 path).  With
 *         it the call stages W^T and this call's P^T (r x n, P rounded to
 *         bf16 once) in the workspace and runs one persistent GEMM over both
 *         (when n % 8 == 0, n >= 320 and m, r are even; otherwise the fused
 *         GEMM reads the staged P^T and W directly); with ws == NULL the fused
 *         GEMM regenerates every P tile in LDS.  All paths give bitwise
 *         identical y and z.  The workspace is scratch: it is dead when the
 *         call's kernels have finished.
 * Requirements: tokens >= 0, n >= 1, m >= 1, 1 <= r <= n.
 * Errors: COMPACT_EINVAL (shapes, a NULL tensor, ld smaller than the row,
 * an unknown dtype or projection code, the identity with r != n),
 * COMPACT_EALIGN, COMPACT_EWORKSPACE (a workspace smaller than the size
 * above), COMPACT_EUNSUPPORTED (n or r of 2^31 or more; the gather flag with
 * more than COMPACT_GATHER_MAX_S draws or r >= 65535), COMPACT_EHIP; nothing
 * is launched on a validation error, and tokens = 0 launches nothing.
 */
int compact_fwd(const void* x, int64_t ldx, const void* W, int64_t ldw, void* y, int64_t ldy,
                void* z, int64_t ldz, int64_t tokens, int64_t n, int64_t m, int64_t r,
                uint64_t seed, int proj, int dtype, void* ws, size_t ws_bytes, void* stream);

size_t compact_fwd_workspace_bytes(int64_t n, int64_t m, int64_t r, int dtype);

/*
 * Forward pass of several projections that read the same input, Alg. 1 per
 * projection (the paper compresses q, k, v of attention and gate, up of the
 * MLP, each with its own P; they share the block input x):
 *
 *   for j = 0 .. count-1:  y_j = x W_j  and  z_j = x P_j
 *
 *   W  [n x M]       (ld ldw)  W = [W_0 | W_1 | ...]: W_j is columns
 *                              mo_j .. mo_j + m[j] - 1, mo_j = m[0] + .. + m[j-1]
 *   y  [tokens x M]  (ld ldy)  y_j in the same columns as W_j
 *   z  [tokens x R]  (ld ldz)  z_j is columns ro_j .. ro_j + r[j] - 1,
 *                              ro_j = r[0] + .. + r[j-1]
 *   M = m[0] + .. + m[count-1], R = r[0] + .. + r[count-1]
 *   m, r, seeds   HOST arrays of count entries (read during the call);
 *                 P_j[i][k] = G(seeds[j], i, k) / sqrt(r[j])
 *   count  1 .. 8; every m[j], r[j] but the last a multiple of 8 (so each
 *          column slice starts on a 16-byte boundary)
 *   ws, ws_bytes  optional workspace of at least
 *          compact_fwd_group_workspace_bytes(n, count, m, r, dtype) bytes (bf16
 *          path).  With it the call stages [W^T; P_0^T; P_1^T; ...] once and runs
 *          one persistent GEMM for all projections (x is read once; the z
 *          columns of all projections share output tiles); otherwise, and for
 *          fp32, it runs compact_fwd on each column slice.
 * Results are bitwise identical to compact_fwd on each (W_j, y_j, z_j) slice.
 * The backward of the group is compact_bwd_group (or compact_bwd with W and
 * the concatenated dL/do for dx, and on the column slices z_j, dL/do_j for
 * each G^_j).
 * Errors: COMPACT_EINVAL (count, NULL arrays, shapes), COMPACT_EALIGN,
 * COMPACT_EWORKSPACE, COMPACT_EHIP; nothing is launched on a validation error.
 */
int compact_fwd_group(const void* x, int64_t ldx, const void* W, int64_t ldw, void* y, int64_t ldy, void* z,
                      int64_t ldz, int64_t tokens, int64_t n, int32_t count, const int64_t* m, const int64_t* r,
                      const uint64_t* seeds, int proj, int dtype, void* ws, size_t ws_bytes, void* stream);

size_t compact_fwd_group_workspace_bytes(int64_t n, int32_t count, const int64_t* m, const int64_t* r, int dtype);

/*
 * Backward pass, Alg. 2:  G^ = z^T dL/do  and  dx = dL/do W^T.
 *
 *   dy [tokens x m]  (ld lddy)  gradient of the loss with respect to y
 *   W  [n x m]       (ld ldw)
 *   z  [tokens x r]  (ld ldz)   the activation saved by compact_fwd
 *   dx [tokens x n]  (ld lddx)  input gradient (exact: it does not involve P);
 *                               may be NULL to skip it (e.g. the first layer)
 *   G  [r x m] fp32, dense (ld = m): compressed weight gradient; may be NULL
 *                               to skip it (not both NULL)
 *   ws, ws_bytes  workspace of at least
 *         compact_bwd_workspace_bytes(tokens, n, m, r, dtype) bytes (bf16
 *         path), required when G is computed: it holds the split-K partial
 *         sums of G^ (the sum over tokens is split and reduced in a fixed
 *         order, so G^ is deterministic) and, before them, a K-tiled copy of W
 *         that the dx GEMM reads (with NULL or a smaller workspace dx reads W
 *         itself; dx is bitwise the same either way).
 * Requirements as compact_fwd.  tokens = 0: dx has no rows and G^ = 0 is
 * written.
 * Errors: COMPACT_EINVAL (shapes, dx and G both NULL, a NULL operand of a
 * requested output, ld smaller than the row, an unknown dtype),
 * COMPACT_EALIGN, COMPACT_EWORKSPACE (G requested on the bf16 path without a
 * workspace of the size above), COMPACT_EUNSUPPORTED (n or r of 2^31 or
 * more), COMPACT_EHIP; nothing is launched on a validation error.
 */
int compact_bwd(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z,
                int64_t ldz, void* dx, int64_t lddx, float* G, int64_t tokens, int64_t n,
                int64_t m, int64_t r, int dtype, void* ws, size_t ws_bytes, void* stream);

size_t compact_bwd_workspace_bytes(int64_t tokens, int64_t n, int64_t m, int64_t r, int dtype);

/*
 * Backward pass of an input group (the projections of one compact_fwd_group
 * call), Alg. 2 per projection:
 *
 *   dx = sum over j of dL/do_j W_j^T = dL/do W^T   (the input is shared)
 *   G^_j = z_j^T dL/do_j,  j = 0 .. count-1
 *
 *   dy [tokens x M]  (ld lddy)  dL/do = [dL/do_0 | dL/do_1 | ...], columns as W
 *   W  [n x M]       (ld ldw)   W = [W_0 | W_1 | ...] (needed only for dx)
 *   z  [tokens x R]  (ld ldz)   z = [z_0 | z_1 | ...] from compact_fwd_group
 *   dx [tokens x n]  (ld lddx)  may be NULL to skip it
 *   G  HOST array of count device pointers, G[j] [r[j] x m[j]] fp32 dense; the
 *      array may be NULL to skip every G^ (not together with dx == NULL)
 *   m, r  HOST arrays of count entries (as in compact_fwd_group: every m[j],
 *      r[j] but the last a multiple of 8), count 1 .. 8
 *   ws, ws_bytes  workspace of at least
 *      compact_bwd_group_workspace_bytes(tokens, n, count, m, r, dtype) bytes
 *   accumulate  0: G[j] = G^_j;  1: G[j] = G[j] + G^_j (gradient accumulation
 *      over several backward passes before one optimizer step: the sum over
 *      the splits is formed first and added to G[j] in one fp32 addition, so
 *      the result is bitwise G[j] + (the G^_j of accumulate = 0))
 * bf16: one dx GEMM, then one split-K launch for every G^_j (one grid of about
 * one workgroup per CU over all projections) and one reduction launch; the
 * splits are summed in a fixed order, so each G^_j is deterministic (it may
 * differ in the last bits from compact_bwd on the slices, whose token splits
 * differ).  dx is bitwise compact_bwd's.  fp32: compact_bwd per slice.
 * Errors: COMPACT_EINVAL (also accumulate not 0 or 1), COMPACT_EALIGN,
 * COMPACT_EWORKSPACE, COMPACT_EHIP; nothing is launched on a validation error.
 */
int compact_bwd_group(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z, int64_t ldz,
                      void* dx, int64_t lddx, float* const* G, int64_t tokens, int64_t n, int32_t count,
                      const int64_t* m, const int64_t* r, int dtype, int accumulate, void* ws, size_t ws_bytes,
                      void* stream);

size_t compact_bwd_group_workspace_bytes(int64_t tokens, int64_t n, int32_t count, const int64_t* m,
                                         const int64_t* r, int dtype);

/*
 * compact_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Arguments, results and errors as compact_bwd; the
 * G^ split-K partial sums (and the K-tiled copy of W for dx, when it fits)
 * live in a library-owned scratch array of COMPACT_NOALLOC_SCRATCH_BYTES per
 * GPU, part of the library's device code: the runtime reserves it on every
 * GPU the library runs on when the library is first used there, and it stays
 * reserved until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library call).  Results are bitwise those of
 * compact_bwd with a workspace of that size.
 * Every call on one GPU shares that GPU's scratch and leaves its contents
 * behind: calls that may overlap on one GPU (different streams, or threads
 * without ordering between them) race and must be serialised by the caller.
 * Errors: as compact_bwd, and COMPACT_EUNSUPPORTED when G is requested and
 * compact_bwd_workspace_bytes(tokens, n, m, r, dtype) exceeds the scratch
 * (then nothing is launched).  The size, 64 MiB and the 256-byte alignment
 * allowance every workspace size includes, covers every layer of the
 * LLaMA-60M, RoBERTa-Base, LLaMA-350M and LLaMA-1B shapes at any token count
 * (the most, 64 MiB of G^ partial sums, at n = m = 2048, r = 512 or 256).
 */
#define COMPACT_NOALLOC_SCRATCH_BYTES ((64u << 20) + 256u)

int compact_bwd_noalloc(const void* dy, int64_t lddy, const void* W, int64_t ldw, const void* z, int64_t ldz,
                        void* dx, int64_t lddx, float* G, int64_t tokens, int64_t n, int64_t m, int64_t r,
                        int dtype, void* stream);

/*
 * Optimizer step, Alg. 3 (Adam on the compressed gradient, then decompression):
 *
 *   M <- b1 M + (1 - b1) G^,   V <- b2 V + (1 - b2) G^2     (stored uncorrected)
 *   N  = (M / (1 - b1^t)) / (sqrt(V / (1 - b2^t)) + eps)
 *   W <- W - lr * alpha * P N,  P re-sampled from `seed` (same as the forward)
 *
 *   W  [n x m] (ld ldw)  updated in place; w_dtype COMPACT_BF16 or COMPACT_F32
 *                        (fp32 master weights; allowed with either dtype)
 *   G  [r x m] fp32 dense   compressed gradient from compact_bwd
 *   M, V [r x m] fp32 dense Adam moments, updated in place (zero before t = 1)
 *   t     1-based step index used in the bias correction (t >= 1)
 *   lr, beta1, beta2, eps, alpha   Adam hyper-parameters and the scale alpha
 *         (0 <= beta < 1, eps > 0, lr >= 0), as doubles: 1 - beta, the bias
 *         corrections 1 - beta^t and lr alpha / sqrt(r) are formed in fp64 on
 *         the host and rounded once to fp32 (rounding beta2 = 0.999 to fp32
 *         first would move 1 - beta2 by 1.3e-5 relative)
 *   dtype compute type of the decompression P N: COMPACT_BF16 (bf16 P and N,
 *         MFMA, fp32 accumulate) or COMPACT_F32
 *   ws, ws_bytes  workspace of at least compact_step_workspace_bytes(n, m, r,
 *         dtype) bytes (holds N between the two kernels)
 * The seed schedule of Alg. 3 (t <- t+1, new seed every T steps) is host logic:
 * compact_next_seed.
 * Errors: COMPACT_EINVAL (shapes, NULL tensors, t < 1, a beta outside [0, 1),
 * eps not positive and finite, lr negative or not finite, alpha not finite,
 * an unknown dtype or projection code), COMPACT_EALIGN, COMPACT_EWORKSPACE,
 * COMPACT_EUNSUPPORTED (fp32 compute into bf16 W; a bf16 shape whose tiles
 * need offsets of 2^31 bytes or more), COMPACT_EHIP; nothing is launched on a
 * validation error.
 */
int compact_step(void* W, int64_t ldw, const float* G, float* M, float* V, int64_t n,
                 int64_t m, int64_t r, uint64_t seed, int64_t t, double lr, double beta1,
                 double beta2, double eps, double alpha, int proj, int dtype, int w_dtype,
                 void* ws, size_t ws_bytes, void* stream);

size_t compact_step_workspace_bytes(int64_t n, int64_t m, int64_t r, int dtype);

/*
 * One layer of compact_step_batched.  Pointers as in compact_step.
 */
typedef struct {
  void* W;          /* [n x m], ld ldw, w_dtype of the call          */
  int64_t ldw;
  const float* G;   /* [r x m] fp32 dense                           */
  float* M;         /* [r x m] fp32 dense                           */
  float* V;         /* [r x m] fp32 dense                           */
  int64_t n, m, r;
  uint64_t seed;    /* the seed this layer's forward used            */
  double alpha;     /* per-layer scale alpha (Alg. 3)               */
} compact_layer;

/*
 * Alg. 3 for `count` layers at once (same step t and hyper-parameters lr,
 * beta1, beta2, eps; per-layer seed and alpha): one Adam launch and one
 * decompression launch per 16 layers instead of two launches per layer.
 * `layers` is a HOST array, read during the call.  Results are bitwise equal
 * to calling compact_step on each layer.  bf16 compute only (dtype
 * COMPACT_BF16); w_dtype bf16 or fp32.  Workspace: at least
 * compact_step_batched_workspace_bytes(layers, count, dtype) bytes.
 */
int compact_step_batched(const compact_layer* layers, int32_t count, int64_t t, double lr,
                         double beta1, double beta2, double eps, int proj, int dtype, int w_dtype,
                         void* ws, size_t ws_bytes, void* stream);

size_t compact_step_batched_workspace_bytes(const compact_layer* layers, int32_t count, int dtype);

/*
 * The P stream (§3.3: P sampled from the layer seed, re-sampled with the same
 * seed, never stored), exported for tests: writes the UNSCALED normals
 * G(seed, i, j), 0 <= i < n, 0 <= j < r, as fp32 into out [n x r] (ld >= r,
 * device pointer).  P = G / sqrt(r).
 *
 * Definition: key = (seed mod 2^32, seed >> 32); counter = (i >> 2, j, 0, 0);
 * (w0, w1, w2, w3) = Philox4x32-10(counter, key) [Salmon et al., SC'11];
 * (a, b) = (w0, w1) for rows 4p, 4p+1 and (w2, w3) for rows 4p+2, 4p+3;
 * Box-Muller with radius sqrt(-2 ln u), u = (2 (a >> 9) + 1) 2^-24, and angle
 * 2 pi ((b >> 8) + 1/2) 2^-24; even rows take the cosine, odd rows the sine.
 * ln, sin and cos are fixed fp32 series (atanh series, Taylor series), so the
 * stream is reproducible bit for bit on any IEEE fp32 machine.
 */
int compact_pstream(uint64_t seed, int64_t n, int64_t r, float* out, int64_t ld, void* stream);

/*
 * The unscaled stream of any projection, exported for tests: out [n x r]
 * (ld >= r, device pointer, fp32) receives G(seed, i, j) for
 * COMPACT_PROJ_GAUSSIAN (as compact_pstream), the identity for
 * COMPACT_PROJ_IDENTITY (r == n), or the integer matrix S(seed, i, j) for
 * COMPACT_PROJ_SPARSE_JL[_S(s)].  P = scale x out with scale 1/sqrt(r),
 * 1 and 1/sqrt(s).
 */
int compact_projection(uint64_t seed, int64_t n, int64_t r, int proj, float* out, int64_t ld, void* stream);

/*
 * Test export: the Box-Muller step of the P stream applied to arbitrary word
 * pairs, g_even[e] = rho(a[e]) cos(theta(b[e])), g_odd[e] = rho(a[e]) sin(theta(b[e])),
 * for 0 <= e < count (all device pointers, count >= 0).  Lets a test sweep every
 * radius and angle code exhaustively.
 */
int compact_pstream_boxmuller(const uint32_t* a, const uint32_t* b, float* g_even, float* g_odd,
                              int64_t count, void* stream);

/*
 * Seed schedule, end of Alg. 3: after step t (1-based) taken with `seed`,
 * returns the seed of step t+1: seed + 1 when T > 0 and t mod T == 0, else
 * seed (T <= 0: never re-sample).  Host-only, no GPU work.
 */
uint64_t compact_next_seed(uint64_t seed, int64_t t, int64_t T);

/* Activation elements saved per layer (Table 1): tokens * r, against tokens * n. */
int64_t compact_saved_activation_elems(int64_t tokens, int64_t n, int64_t r);

const char* compact_status_string(int status);

/* Description of the last failure on the calling thread ("" if none). */
const char* compact_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int compact_version(void);

#ifdef __cplusplus
}
#endif

#endif /* COMPACT_H_ */
