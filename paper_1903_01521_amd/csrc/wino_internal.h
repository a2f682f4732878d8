// Host-side plan of one layer and the launchers the C-ABI calls.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "wino.h"

namespace wino {

// The NCHW input kernels address x through 32-bit buffer offsets, and any
// offset at or past this limit reads as zero: the fused and split kernels
// within one image, the staged input transforms (fp32 and 16-bit) across the
// images one 16-tile block spans.  The planner rejects inputs that would need
// larger offsets.
constexpr uint32_t kInvalidOffset = 1u << 30;

// Geometry of an r x r (3x3, or 5x5 with m = 2) stride-1 layer tiled into
// m x m output regions, and the blocked transform-domain extents (see the
// layout notes in wino.h).
struct Geom {
    int N, C, H, W, K, pad, m;
    int Ho, Wo, th, tw;
    int P;          // tiles, N*th*tw
    int A, T;       // alpha = m + r - 1; T = alpha^2 (2-D) or alpha (1-D)
    int r;          // filter side (the filter's length for 1-D layers)
    int axis;       // 0: r x r filter; 1: 1 x r (along W); 2: r x 1 (along H)
    int nhwc;       // 1: x is [N][H][W][C] and y is [N][Ho][Wo][K] (three-stage path)
    int CQ, KB, PB; // 4-channel quads, 16-filter blocks, 16-tile blocks
};

// Kernel variant of the fused algorithm.
struct FusedCfg {
    int csplit;     // waves of one workgroup splitting the channel quads of a unit
    int bw;         // tile-block width: 16 (1 x 16 tiles) or 4 (4 x 4 tiles)
    int nsl;        // channel slices over workgroups (1: none), summed by k_slice_sum
};

// Division of n < 2^31 by a fixed d >= 1 as ((mulhi(n, m) + n) >> l), with
// l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1 (Granlund and
// Montgomery's round-up method; mulhi(n, m) + n < 2^32 for such n).
struct FastDiv {
    uint32_t m;
    int l;
};

// Runtime part of the fused kernel's work decomposition (host-computed).
struct FusedTiling {
    int nbh, nbw;   // tile blocks per image along rows / columns
    int nt;         // tile blocks in the batch
    int nkg;        // filter groups (each 16 * 8/(row groups * csplit) filters)
    int per;        // work items per XCD, ceil(nt * nkg / 8)
    int nsteps;     // channel steps, ceil(CQ / csplit)
    int kfast;      // item order: 1 = filter group fastest (tile major), 0 = group major
    int bw;         // split path: tile-block width (16 or 4)
    FastDiv d_item; // fused path: item -> (quotient, remainder) by nkg (kfast) or nt
    FastDiv d_img;  // by nbh * nbw (tile blocks per image)
    FastDiv d_nbw;  // by nbw
    int nsl;        // channel slices: workgroup items nt * nkg per slice
    int qsl;        // channel quads per slice
    FastDiv d_sl;   // by nt * nkg
    long long ysz;  // N*K*Ho*Wo: floats of one slice's partial output
};

size_t filter_elems(int C, int K, int m, int r);         // T*Cp*Kp
size_t v_elems(const Geom& g);                           // PB*CQ*T*64
size_t m_elems(const Geom& g);                           // PB*KB*T*256

hipError_t launch_filter_transform(const float* g, float* U, int C, int K, int m, int r, hipStream_t s);
hipError_t launch_input_transform(const float* x, float* V, const Geom& g, hipStream_t s);
hipError_t launch_batched_gemm(const float* U, const float* V, float* M, const Geom& g, hipStream_t s);
hipError_t launch_output_transform(const float* M, float* y, const Geom& g, bool relu, hipStream_t s);
// cfg.nsl > 1: the channels in cfg.nsl slices over workgroups, partial outputs
// to part ([nsl][N][K][Ho][Wo]), then summed in slice order into y.
hipError_t launch_fused(const float* x, const float* U, float* y, const Geom& g, FusedCfg cfg,
                        bool relu, hipStream_t s, float* part = nullptr);
// Channel quads per slice, and the slices that hold any, for a requested count.
int slice_quads(const Geom& g, int nsl);
int slices_used(const Geom& g, int nsl);
// Split path: input transform into a workspace of 16-tile blocks, then the
// GEMMs with the output transform in their epilogue.
long split_blocks(const Geom& g);            // ceil(P / 16)
size_t vblk_elems(const Geom& g);
// Work items of the GEMM kernel: (pair of tile blocks, filter group).  When
// the last round of items would leave most CUs idle (items % 256, at most
// 256 / units of them), those items run as units of one tile block and one
// filter block each.
constexpr long kSplitCus = 256;
struct SplitTail {
    long items;     // (tile-block pair, filter group) items
    long tail;      // of them, run as units
    int units;      // units per item: 2 tile blocks x filter blocks per group
};
SplitTail split_tail(const Geom& g);
// The split path's input transform by whole tile rows: R rows of the batch
// per workgroup (0: the 16-tile patch kernel instead, always for vec = 0,
// i.e. a width that is not a multiple of 4 or an unaligned x), LDS row pitch
// in floats, dynamic LDS bytes.
constexpr size_t kVrowsLds = 64 << 10;
struct VrowsPlan {
    int R, pitch;
    size_t lds;
};
VrowsPlan vrows_plan(const Geom& g, int vec);
// The split path on fp16 (prec 1) / bf16 (prec 2) operands: VH = the workspace
// of split16_workspace bytes, UH from the 16-bit filter transform.
hipError_t launch_split16(const float* x, const void* UH, float* y, void* VH, const Geom& g, int prec, bool relu,
                          hipStream_t s);
hipError_t launch_split(const float* x, const float* U, float* y, float* Vb, const Geom& g, int bw, bool relu,
                        hipStream_t s);
// Low-C path (C <= 4): a lane per tile, vector FMAs over the few channels.
hipError_t launch_lowc(const float* x, const float* U, float* y, const Geom& g, bool relu, hipStream_t s);
hipError_t launch_maxpool2x2(const float* x, float* y, int N, int C, int H, int W, hipStream_t s);
// Waves of the matrix-core peak probe: 256 CUs x 4 SIMDs x 2 waves.
constexpr int kProbeWaves = 2048;
// Up to 2^21 iterations every partial sum of the probe's check value is an
// integer below 2^24, so the check is exact.
constexpr int kProbeMaxIters = 1 << 21;
hipError_t launch_mfma_probe(int iters, float* out, hipStream_t s);
// Scratch of wino_conv2d_noalloc: a static device array of this many bytes
// per GPU; *out = its address on the current device (looked up once per
// device and kept).
constexpr size_t kNoAllocScratchBytes = WINO_NOALLOC_SCRATCH_BYTES;
hipError_t noalloc_scratch(void** out);
// 1-D layers (1 x r or r x 1 filters, F(1xm, 1xr, 1x8)): filter transform; the
// input and output transforms dispatch on g.axis inside launch_input_transform
// and launch_output_transform.
hipError_t launch_filter_transform_1d(const float* g, float* U, int C, int K, int m, int r, hipStream_t s);
// 16-bit GEMM operands (prec 1: fp16, 2: bf16): filter transform into UH, and
// the three stages through VH (16-bit) and M (fp32).
hipError_t launch_filter_transform16(const float* g, void* UH, int C, int K, int m, int prec, hipStream_t s);
hipError_t launch_staged16(const float* x, const void* UH, float* y, void* VH, float* M, const Geom& g, int prec,
                           bool relu, hipStream_t s);

}  // namespace wino
