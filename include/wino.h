/*
 * wino.h -- region-wise multi-channel Winograd / Cook-Toom 3x3 convolution on
 * AMD MI355X (gfx950): F(2x2,3x3) (m = 2) and F(4x4,3x3) (m = 4), stride 1.
 *
 * The method (Sec. 2 of Maji et al., "Efficient Winograd or Cook-Toom
 * Convolution Kernel Implementation on Widely Used Mobile CPUs"): a layer is
 * Eq. 1 applied region by region -- every (m+2)x(m+2) input region of every
 * channel is taken to the transform domain, multiplied elementwise with the
 * transformed filter of each (output, input) channel pair, summed over the input
 * channels, and taken back once per output region.  The work splits into an
 * offline weight transform and three per-inference stages (Sec. 2, the
 * three-step list): input transform (scatter into per-position matrices),
 * T = (m+2)^2 independent GEMMs contracting over C (Sec. 2.2), and output
 * transform (gather, inverse transform, write).
 *
 * Conventions for every entry point
 *   - Data pointers are DEVICE pointers owned by the caller.  The library never
 *     allocates, frees or keeps a pointer after the call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *     asynchronously: a return of WINO_OK means "enqueued", not "finished".
 *   - Arguments are validated before any HIP call.  On failure the call returns
 *     a negative status, enqueues nothing and leaves all outputs untouched.
 *   - Launch failures return WINO_ERR_HIP (the HIP error is consumed); faults
 *     during execution surface at the caller's next synchronisation.
 *   - Stateless, reentrant and thread-safe; results are bitwise deterministic
 *     from run to run (no atomics; every reduction has a fixed order).
 *   - Filter 3x3, stride 1 and symmetric zero padding `pad` >= 0 are fixed by
 *     the method; Ho = H + 2*pad - 2 and Wo = W + 2*pad - 2 must be >= 1.
 *     The operation is cross-correlation (no kernel flip):
 *       y[n,k,i,j] = sum_c sum_{r,s<3} x[n,c,i+r-pad,j+s-pad] * g[k,c,r,s]
 *     with x read as zero outside [0,H) x [0,W).
 *   - Floating point is IEEE fp32 storage and fp32 arithmetic (the paper's
 *     precision, Sec. 3); FMA contraction is allowed; the GEMMs run on fp32 MFMA.
 *   - Size limits of the NCHW (channel-first) paths, from the kernels' 32-bit
 *     offsets into x: one image's input, C*H*W*4 bytes, must be below 1 GiB for
 *     the fused and split algorithms, and (16 / (th*tw) + 2) such images below
 *     1 GiB for the staged input transform (the images one 16-tile block
 *     spans).  The fused and split kernels also read the channels past C (up
 *     to whole channel steps) as zeros through offsets past the image, so
 *     1 GiB + P*H*W*4 must stay below 4 GiB, with P = S * (steps + 3) for the
 *     fused kernel (S = 32 channels a step for m = 2 and 3x3, 16 otherwise;
 *     steps = ceil(channels of one slice / S)) and P = 16 * ceil(C/16) for
 *     the split one.  A layer past a limit of an
 *     explicitly chosen algorithm returns WINO_ERR_UNSUPPORTED; WINO_ALGO_AUTO
 *     moves on to one that fits (fused, then split, then staged) and returns
 *     WINO_ERR_UNSUPPORTED only when none does.  Split larger inputs along C
 *     or the image.
 *
 * Tiling (Sec. 2, region decomposition)
 *   alpha = m + 2, T = alpha^2, th = ceil(Ho/m), tw = ceil(Wo/m),
 *   P = N*th*tw tiles, tile p = (n*th + ti)*tw + tj covers output rows
 *   ti*m .. ti*m+m-1 and cols tj*m .. tj*m+m-1 and reads the input region whose
 *   top-left corner is (ti*m - pad, tj*m - pad).  Outputs past Ho x Wo are
 *   computed on zero-extended input and discarded.
 *   Transform-domain element (xi, nu) of a region has index t = xi*alpha + nu.
 *
 * Transform-domain layouts (MFMA-native blocking; Cp = roundup(C,4),
 * Kp = roundup(K,16), Pp = roundup(P,16), CQ = Cp/4, KB = Kp/16, PB = Pp/16)
 *   U (filters):  float U[KB][CQ][T/4][64][4], element (t,c,k) at lane
 *                 (c%4)*16 + k%16, slot t%4, of group (k/16, c/4, t/4).
 *                 Padding is zero.
 *   V (inputs):   float V[PB][CQ][T/4][64][4], element (t,c,p) at lane
 *                 (c%4)*16 + p%16, slot t%4, of group (p/16, c/4, t/4).
 *                 Padding is zero.
 *   M (products): float M[PB][KB][T][64][4], element (t,k,p) at lane
 *                 16*((k%16)/4) + p%16, slot k%4, of block (p/16, k/16, t).
 *   For one position t, the 64 lanes of a U or V group are exactly one wave's
 *   operand of a 16x16x4 fp32 MFMA, and a lane's 4 consecutive positions are
 *   one 16-byte word; each 256-float block of M is one wave's accumulator tile.
 */
#ifndef WINO_H
#define WINO_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define WINO_OK                0
#define WINO_ERR_INVALID_ARG  (-1)   /* null pointer, non-positive size, Ho/Wo < 1, overflow, aliasing */
#define WINO_ERR_UNSUPPORTED  (-2)   /* m not in {2, 4}, an unknown flag bit, or past a size limit */
#define WINO_ERR_WORKSPACE    (-3)   /* workspace missing or smaller than required */
#define WINO_ERR_HIP          (-4)   /* a HIP launch or query failed */

/* ---- flags -------------------------------------------------------------- */
#define WINO_FLAG_RELU     0x001u   /* y = max(y, 0), applied in the output transform */
#define WINO_ALGO_AUTO     0x000u   /* let the planner choose (default) */
#define WINO_ALGO_FUSED    0x100u   /* one kernel: input transform -> GEMMs -> output transform */
#define WINO_ALGO_STAGED   0x200u   /* three kernels through the workspace (V, then M) */
#define WINO_ALGO_SPLIT    0x300u   /* two kernels: input transform into a tile-blocked
                                       workspace, then the GEMMs with the output
                                       transform in their epilogue (large layers) */
#define WINO_ALGO_LOWC     0x400u   /* one kernel for C <= 4 (a network's first layer): a
                                       lane per tile, vector FMAs over the channels */
#define WINO_ALGO_MASK     0xF00u
/* Reduced-precision GEMM operands (3x3 NCHW layers only): U and V rounded to
 * fp16 or bf16 (nearest, ties to even), the T per-position GEMMs on 16-bit MFMA
 * with fp32 accumulation, the output transform in fp32.  Algorithms: the three
 * stages (WINO_ALGO_STAGED; fp32 M through the workspace) or the split path
 * (WINO_ALGO_SPLIT; the GEMM kernel applies the output transform to its
 * accumulators); AUTO takes split on layers with at least two rounds of its
 * work items on the CUs, else the three stages.  U must come from
 * wino_filter_transform_p with the same format.  Not
 * within the fp32 gates: measured normwise errors against the exact result are
 * about 5e-4 (fp16) and 4e-3 (bf16) for m = 2, 7e-3 and 6e-2 for m = 4. */
#define WINO_PREC_F16      0x010u
#define WINO_PREC_BF16     0x020u
#define WINO_PREC_MASK     0x030u
/* Optional overrides of the fused kernel's variant (0 = planner's choice):
 *   WINO_BLOCK_1x16 / WINO_BLOCK_4x4: a workgroup's 16 tiles are one row of 16
 *                  tiles, or a 4 x 4 square of tiles;
 *   WINO_CSPLIT(n) n in {1,2,4,8} (F(2x2,3x3)) or {1,2,4} (F(4x4,3x3),
 *                  F(2x2,5x5)): waves of a workgroup that split the input
 *                  channels of one filter block, reduced in a fixed order.
 * Results of every variant agree to fp32 rounding; unsupported combinations
 * return WINO_ERR_UNSUPPORTED. */
#define WINO_BLOCK_1x16    0x1000u
#define WINO_BLOCK_4x4     0x2000u
#define WINO_CSPLIT(n)     (((unsigned)(n) & 0xFu) << 16)
/* WINO_CSLICES(n), n in 1..8 and at most ceil(C/4), with WINO_ALGO_FUSED: the
 * channels in n slices over separate workgroups (quads split as evenly as
 * ceil(CQ/n) allows), each writing a partial output to the workspace
 * ([slices][N][K][Ho][Wo] fp32), summed in slice order by one more launch
 * (ReLU applied there).  WINO_ALGO_AUTO picks it for fused layers whose
 * workgroups fill less than half of the 256 CUs with long channel loops (deep
 * layers at batch 1), if the caller passes the workspace that
 * wino_workspace_bytes then reports; without it the layer runs unsliced.
 * WINO_CSLICES(1) keeps AUTO from slicing. */
#define WINO_CSLICES(n)    (((unsigned)(n) & 0xFu) << 20)

/* Human-readable text of a status code (static storage, never NULL). */
const char* wino_status_string(int status);

/* Library version, 100*major + minor. */
int wino_version(void);

/* Bytes of the transformed-filter buffer U for (C, K, m): 4*T*Cp*Kp.
 * Returns 0 if C or K <= 0, m is not 2 or 4, or the size overflows. */
size_t wino_filter_bytes(int C, int K, int m);

/* Bytes of V (input transform output) and of M (GEMM output) for a layer.
 * Return 0 on invalid arguments (same rules as wino_conv2d). */
size_t wino_input_tf_bytes(int N, int C, int H, int W, int pad, int m);
size_t wino_gemm_out_bytes(int N, int K, int H, int W, int pad, int m);

/* Workspace bytes wino_conv2d needs for this layer and flags word.  The
 * result depends on the whole word as wino_conv2d reads it: the algorithm
 * (and, for WINO_ALGO_AUTO, the planner's choice of split, channel slices or
 * staged), WINO_PREC_* (16-bit V plus fp32 M, or the split path's 16-bit V), WINO_CSLICES(n) (the partial
 * outputs) and the variant overrides.  0 means the plan needs none (workspace
 * may then be NULL).  Returns (size_t)-1 for invalid arguments and for flag
 * sets or layers that wino_conv2d would reject as WINO_ERR_UNSUPPORTED. */
size_t wino_workspace_bytes(int N, int C, int H, int W, int K, int pad, int m, unsigned flags);

/* Offline filter transform (Eq. 1's W w W^T; Sec. 2, the GEMM step's 'B'
 * matrices, computed once per weight set and reused).
 *   g : [K][C][3][3] fp32 (KCRS), read only.
 *   U : wino_filter_bytes(C,K,m) bytes, written in the U layout above.  Each
 *       element is G g G^T evaluated in fp64 and rounded to fp32.
 * Errors: INVALID_ARG (null, C/K <= 0, overflow), UNSUPPORTED (m), HIP. */
int wino_filter_transform(const float* g, float* U, int C, int K, int m, void* stream);

/* The planner's choice for a layer (r = 3, or 5 with m = 2), for callers that
 * pass the workspace wino_workspace_bytes(_r) reports: *algo = the
 * WINO_ALGO_* value that runs (FUSED, SPLIT, STAGED or LOWC), *slices = the
 * fused kernel's channel slices (1 when unsliced or not fused).  Errors as for
 * wino_workspace_bytes_r's arguments (INVALID_ARG, UNSUPPORTED); null outputs
 * are INVALID_ARG. */
int wino_plan_r(int N, int C, int H, int W, int K, int pad, int m, int r, unsigned flags, unsigned* algo,
                int* slices);

/* One 3x3 stride-1 convolution layer (Eq. 1 over all regions; Sec. 2).
 *   x : [N][C][H][W] fp32 (NCHW), read only.
 *   U : output of wino_filter_transform with the same (C, K, m), read only.
 *   y : [N][K][Ho][Wo] fp32 (NCHW), written; must not overlap x.
 *   flags : WINO_FLAG_RELU and/or one WINO_ALGO_* value.
 *   workspace / workspace_bytes : device scratch of at least
 *       wino_workspace_bytes(N,C,H,W,K,pad,m,flags) bytes (V and M of the staged
 *       algorithm, the tile-blocked V of the split one, the partial outputs of
 *       channel slices); may be NULL/0 when that is 0.  With WINO_ALGO_AUTO the
 *       planner uses the split algorithm or channel slices only if the
 *       workspace given is large enough, else the plain fused kernel (or
 *       WINO_ERR_WORKSPACE where the fused kernel's offsets would not fit, see
 *       the size limits above).  Contents on
 *       return are unspecified; calls sharing one workspace must not overlap in
 *       time.
 * Errors: INVALID_ARG, UNSUPPORTED, WORKSPACE, HIP. */
int wino_conv2d(const float* x, const float* U, float* y,
                int N, int C, int H, int W, int K, int pad, int m,
                unsigned flags, void* workspace, size_t workspace_bytes, void* stream);

/* Stage 1 alone, input transform (Sec. 2.1.1 for m = 2; Eq. 1's X^T x X):
 * every region of every channel to the transform domain, scattered into the
 * per-position matrices.
 *   x : [N][C][H][W] fp32; V : wino_input_tf_bytes(...) bytes, V layout.
 * For m = 2 each element is computed with the paper's printed add/sub order
 * (a pass over rows, then the same pass over columns) and is bit-exact. */
int wino_input_transform(const float* x, float* V, int N, int C, int H, int W,
                         int pad, int m, void* stream);

/* Stage 2 alone, the T per-position GEMMs (Sec. 2.2):
 *   M_t[k][p] = sum_c U_t[c][k] * V_t[c][p]  for every t < T.
 *   U : filter layout for (C, K, m); V : input layout for (N,C,H,W,pad,m);
 *   M : wino_gemm_out_bytes(N,K,H,W,pad,m) bytes, M layout. */
int wino_batched_gemm(const float* U, const float* V, float* M,
                      int N, int C, int H, int W, int K, int pad, int m, void* stream);

/* Stage 3 alone, output transform (Eq. 1's Z^T ( . ) Z; Sec. 2, third step):
 * gather the T values of every (tile, output channel), inverse-transform, write
 * the m x m block into y (NCHW), cropped to Ho x Wo.  flags: WINO_FLAG_RELU. */
int wino_output_transform(const float* M, float* y, int N, int K, int H, int W,
                          int pad, int m, unsigned flags, void* stream);

/* Transformed filters in a 16-bit GEMM format (prec = WINO_PREC_F16 or
 * WINO_PREC_BF16; 0 gives the fp32 calls above):
 *   UH[KB][C32][T][64][8] 16-bit values, C32 = ceil(C/32): element (t,c,k) at
 *   lane ((c%16)/4)*16 + k%16, half ((c%32)/16)*4 + c%4 of block (k/16, c/32,
 *   t) -- one 16-byte word per lane, the lane's A operand of
 *   v_mfma_f32_16x16x32 (four consecutive channels of each 16-channel half of
 *   the 32-channel chunk; padding zero).  Each value is G g G^T in fp64,
 *   rounded to fp32, then to the 16-bit format.
 *   Bytes: 2*T*roundup(C,32)*roundup(K,16). */
size_t wino_filter_bytes_p(int C, int K, int m, unsigned prec);
int wino_filter_transform_p(const float* g, void* U, int C, int K, int m, unsigned prec, void* stream);

/* ---- 5x5 filters: F(2x2,5x5) ----------------------------------------------
 * The same method for r x r filters (Eq. 1 with a 5x5 filter; the paper's
 * Table 2 benchmarks 5x5 layers with its F(2x2,5x5,6x6) variant).  Supported
 * (m, r): (2, 3), (4, 3) -- identical to the 3x3 calls above -- and (2, 5).
 * For r = 5: alpha = m + r - 1 = 6, T = 36, Ho = H + 2*pad - 4, Wo = W + 2*pad - 4;
 * points {0, 1, -1, 2, -2, inf} (the same B^T as F(4x4,3x3)):
 *   G   = [1/4 0 0 0 0; -1/6 -1/6 -1/6 -1/6 -1/6; -1/6 1/6 -1/6 1/6 -1/6;
 *          1/24 1/12 1/6 1/3 2/3; 1/24 -1/12 1/6 -1/3 2/3; 0 0 0 0 1]
 *   A^T = [1 1 1 1 1 0; 0 1 -1 2 -2 1]
 *   y[n,k,i,j] = sum_c sum_{r,s<5} x[n,c,i+r-pad,j+s-pad] * g[k,c,r,s].
 * Layouts of U, V and M are the ones above with T = 36.  g is [K][C][5][5].
 * 5x5 layers run the fused kernel (WINO_ALGO_AUTO or _FUSED, no workspace;
 * WINO_BLOCK_* and WINO_CSPLIT(n), n in {1,2,4}, as for m = 4) or the three
 * stages (WINO_ALGO_STAGED, with the workspace), plus WINO_FLAG_RELU.
 * Errors as for the 3x3 calls; UNSUPPORTED for other (m, r), for
 * WINO_ALGO_SPLIT and _LOWC, and for the 16-bit formats. */
size_t wino_filter_bytes_r(int C, int K, int m, int r);
int wino_filter_transform_r(const float* g, float* U, int C, int K, int m, int r, void* stream);
size_t wino_workspace_bytes_r(int N, int C, int H, int W, int K, int pad, int m, int r, unsigned flags);
int wino_conv2d_r(const float* x, const float* U, float* y,
                  int N, int C, int H, int W, int K, int pad, int m, int r,
                  unsigned flags, void* workspace, size_t workspace_bytes, void* stream);
/* The three stages alone for r x r filters (the calls above with r = 3). */
size_t wino_input_tf_bytes_r(int N, int C, int H, int W, int pad, int m, int r);
size_t wino_gemm_out_bytes_r(int N, int K, int H, int W, int pad, int m, int r);
int wino_input_transform_r(const float* x, float* V, int N, int C, int H, int W,
                           int pad, int m, int r, void* stream);
int wino_batched_gemm_r(const float* U, const float* V, float* M,
                        int N, int C, int H, int W, int K, int pad, int m, int r, void* stream);
int wino_output_transform_r(const float* M, float* y, int N, int K, int H, int W,
                            int pad, int m, int r, unsigned flags, void* stream);

/* ---- 1-D layers: F(1xm, 1xr, 1x8) ------------------------------------------
 * 1 x r filters (axis WINO_AXIS_W: correlation along rows) or r x 1 filters
 * (WINO_AXIS_H: along columns) -- the paper applies the method to 1xN and Nx1
 * layers (Table 2's 1x7 and 7x1 Inception-v3 layers) with the variants
 * F(1x6,1x3,1x8), F(1x4,1x5,1x8) and F(1x2,1x7,1x8): (m, r) in {(6,3), (4,5),
 * (2,7)}.  alpha = 8 inputs per region, T = 8 positions, points
 * {0, 1, -1, 2, -2, 1/2, -1/2, inf}.
 *   g : [K][C][r] fp32 (the taps of a [K][C][1][r] or [K][C][r][1] filter).
 *   pad : zero padding along the filtered axis only (the other extent is 1).
 *   Axis W: y[n,k,i,j] = sum_c sum_{s<r} x[n,c,i,j+s-pad] * g[k,c,s],
 *           Ho = H, Wo = W + 2*pad - (r-1); tiles of 1 x m outputs.
 *   Axis H: y[n,k,i,j] = sum_c sum_{s<r} x[n,c,i+s-pad,j] * g[k,c,s],
 *           Ho = H + 2*pad - (r-1), Wo = W; tiles of m x 1 outputs.
 * Tile p = (n*th + ti)*tw + tj as above (th = Ho, tw = ceil(Wo/m) along W;
 * th = ceil(Ho/m), tw = Wo along H); U, V and M use the blocked layouts above
 * with T = 8.  The three stages run (flags: WINO_ALGO_AUTO or _STAGED, and
 * WINO_FLAG_RELU); the workspace is always required.  Errors as for
 * wino_conv2d; UNSUPPORTED for other (m, r) or axis values. */
#define WINO_AXIS_W 1
#define WINO_AXIS_H 2
size_t wino_filter_bytes_1d(int C, int K, int m, int r);
int wino_filter_transform_1d(const float* g, float* U, int C, int K, int m, int r, void* stream);
size_t wino_workspace_bytes_1d(int N, int C, int H, int W, int K, int pad, int m, int r, int axis,
                               unsigned flags);
int wino_conv2d_1d(const float* x, const float* U, float* y,
                   int N, int C, int H, int W, int K, int pad, int m, int r, int axis,
                   unsigned flags, void* workspace, size_t workspace_bytes, void* stream);

/* ---- channel-last tensors ---------------------------------------------------
 * The 3x3 layer of wino_conv2d with x as [N][H][W][C] and y as [N][Ho][Wo][K]
 * (NHWC, the layout the paper chooses for its channel-vectorised transforms,
 * Sec. 2.1).  U comes from wino_filter_transform as before.  Flags:
 * WINO_ALGO_STAGED runs the three stages through the workspace (V and M);
 * WINO_ALGO_SPLIT the split path (input transform into the tile-blocked V
 * workspace, then GEMMs with the output transform storing y channel-last);
 * WINO_ALGO_AUTO takes split on layers with at least two rounds of its work
 * items on the CUs (e.g. N=64, 256 channels, 56x56), else the three stages;
 * and WINO_FLAG_RELU.  wino_workspace_bytes_nhwc gives the workspace of the
 * plan the flags choose.  Errors as for wino_conv2d. */
size_t wino_workspace_bytes_nhwc(int N, int C, int H, int W, int K, int pad, int m, unsigned flags);
int wino_conv2d_nhwc(const float* x, const float* U, float* y,
                     int N, int C, int H, int W, int K, int pad, int m,
                     unsigned flags, void* workspace, size_t workspace_bytes, void* stream);

/* ---- allocation-free variant ------------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the layer of
 * wino_conv2d with the same arguments and flags, its workspace taken from a
 * static device array of WINO_NOALLOC_SCRATCH_BYTES bytes that the library
 * holds on every GPU it runs on until the process ends (no hipMalloc, hipFree
 * or other allocation; the caller passes x, U and y as before).
 *   - WINO_ALGO_AUTO plans as wino_conv2d does with a workspace of that size:
 *     the split algorithm, channel slices or the staged one where their
 *     workspace fits, else the fused kernel (WINO_ERR_WORKSPACE only when no
 *     algorithm that fits is left, see the size limits above).
 *   - An explicit algorithm or WINO_CSLICES(n) whose workspace
 *     (wino_workspace_bytes with the same flags) exceeds the array returns
 *     WINO_ERR_WORKSPACE before any HIP call.
 *   - Every call on one GPU shares that GPU's array, which keeps the last
 *     call's contents (every algorithm writes all the workspace it reads):
 *     calls that overlap in time on one GPU, from any stream or thread, race
 *     and must be serialised by the caller.
 * Errors: as for wino_conv2d. */
#define WINO_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int wino_conv2d_noalloc(const float* x, const float* U, float* y,
                        int N, int C, int H, int W, int K, int pad, int m,
                        unsigned flags, void* stream);

/* Glue between the blocks of a VGG-style stack (not part of the method):
 * 2x2 window, stride 2 max-pool, y: [N][C][H/2][W/2] (floor). */
int wino_maxpool2x2(const float* x, float* y, int N, int C, int H, int W, void* stream);

/* Measurement aid (not part of the method): the fp32 matrix-core rate the chip
 * sustains, to set beside the published peak when reading roofline fractions.
 * One launch of 2048 waves (2 per SIMD of 256 CUs), each running 8 independent
 * chains of iters v_mfma_f32_16x16x4_f32 on operands of 1.0.  out: 2048 floats
 * (device, caller-owned); out[w] = 32 * iters exactly for every wave w (a check
 * that the work ran).  iters in [1, 2^21], else WINO_ERR_INVALID_ARG; null out
 * is invalid too.  wino_probe_mfma_f32_flops(iters) gives the launch's FLOPs
 * (0 outside that range); FLOPs / elapsed time is the sustained rate. */
int wino_probe_mfma_f32(int iters, float* out, void* stream);
size_t wino_probe_mfma_f32_flops(int iters);

#ifdef __cplusplus
}
#endif

#endif /* WINO_H */
