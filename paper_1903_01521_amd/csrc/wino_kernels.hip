// HIP kernels for gfx950 (MI355X): region-wise multi-channel Winograd
// F(2x2,3x3) / F(4x4,3x3) convolution, stride 1.
//
// Work split (Sec. 2, the three-step decomposition, plus the offline weight
// transform):
//   k_filter  : U = G g G^T per (output, input) channel pair, fp64 inside.
//   k_input   : V = B^T d B per (tile, channel) region           (staged path)
//   k_gemm    : M_t = U_t^T V_t for each of the T positions       (staged path)
//   k_output  : y = A^T M A per (tile, output channel)            (staged path)
//   k_fused   : all three per-inference stages in one kernel; the input
//               transform writes straight into MFMA operand registers and the
//               output transform reads straight from the accumulators.
//
// MFMA mapping (v_mfma_f32_16x16x4_f32, one wave):
//   D[i][j] += sum_{q<4} A[i][q] * B[q][j],  i, j < 16
//   A operand: lane l holds A[l%16][l/16];  B operand: lane l holds B[l/16][l%16];
//   D: lane l holds D[4*(l/16) + r][l%16] in slot r.
// With A = U_t (i = output channel, q = input channel), B = V_t (q = input
// channel, j = tile) and D = M_t (i = output channel, j = tile), a lane that
// transforms the region of tile l%16, channel l/16 holds exactly its B operand
// for all T positions, and after the channel loop holds the T accumulators of
// tile l%16 for output channels 4*(l/16) .. 4*(l/16)+3 -- everything the output
// transform of those four (tile, channel) pairs needs, in its own registers.
#include "wino_internal.h"
#include "wino_transforms.h"

namespace wino {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------ helpers

struct TileCoord {
    int n, ti, tj;
    bool valid;
};

__device__ __forceinline__ TileCoord decode_tile(int p, const Geom& g) {
    TileCoord t;
    t.valid = p < g.P;
    const int pp = t.valid ? p : 0;
    const int per = g.th * g.tw;
    t.n = pp / per;
    const int rem = pp - t.n * per;
    t.ti = rem / g.tw;
    t.tj = rem - t.ti * g.tw;
    return t;
}

// ---- region loads through a per-wave buffer resource -----------------------
// Offsets are 32-bit byte offsets from the first image a 16-tile block touches.
// Any offset >= kInvalid lies past the resource's record count, and the buffer
// unit returns 0 for it: a padded row, column, channel or tile is read as zero
// without a select.  The host guarantees that every valid offset is below
// kInvalid (the images one block spans hold < 1 GiB of input).
constexpr uint32_t kInvalid = 1u << 30;
constexpr int kRsrcWord3 = 0x00020000;   // raw (unformatted) 32-bit buffer

template <int MT>
struct RegionPlan {
    __amdgpu_buffer_rsrc_t rsrc;     // wave-uniform
    uint32_t row[MT + 2];            // lane's channel-plane + row byte offset, or kInvalid
    uint32_t col[MT + 2];            // column byte offset, or kInvalid
    uint32_t plane_bytes;            // H*W*4: step between channels (soffset units)
};

// p0 = first tile of the wave's 16-tile block (wave-uniform); tc = lane's tile;
// cl = lane's channel within a quad.
template <int MT>
__device__ __forceinline__ RegionPlan<MT> make_region_plan(const float* __restrict__ x, const Geom& g,
                                                           int p0, const TileCoord& tc, int cl) {
    constexpr int A = MT + 2;
    RegionPlan<MT> rp;
    const int n0 = __builtin_amdgcn_readfirstlane(min(p0, g.P - 1) / (g.th * g.tw));
    const size_t img = (size_t)g.C * g.H * g.W;
    const size_t left = ((size_t)g.N - n0) * img * 4;
    rp.rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(x + (size_t)n0 * img), (short)0,
                                                (int)(left < kInvalid ? left : kInvalid), kRsrcWord3);
    rp.plane_bytes = (uint32_t)g.H * g.W * 4;
    const uint32_t plane = ((uint32_t)(tc.n - n0) * g.C + cl) * rp.plane_bytes;
    const int r0 = tc.ti * MT - g.pad, c0 = tc.tj * MT - g.pad;
#pragma unroll
    for (int u = 0; u < A; ++u) {
        const int row = r0 + u;
        rp.row[u] = (tc.valid && row >= 0 && row < g.H) ? plane + (uint32_t)row * g.W * 4 : kInvalid;
    }
#pragma unroll
    for (int v = 0; v < A; ++v) {
        const int col = c0 + v;
        rp.col[v] = (col >= 0 && col < g.W) ? (uint32_t)col * 4 : kInvalid;
    }
    return rp;
}

// d = the region of channel quad cq for this lane (channel cq*4 + cl), zero
// outside the image, past the last channel, and for tiles past P.
template <int MT>
__device__ __forceinline__ void load_region(const RegionPlan<MT>& rp, const Geom& g, int cq, int cl,
                                            float (&d)[MT + 2][MT + 2]) {
    constexpr int A = MT + 2;
    const uint32_t chan = (cq * 4 + cl < g.C) ? 0u : kInvalid;
    const int soff = __builtin_amdgcn_readfirstlane(cq * 4 * (int)rp.plane_bytes);
#pragma unroll
    for (int u = 0; u < A; ++u) {
        const uint32_t rowq = rp.row[u] + chan;
#pragma unroll
        for (int v = 0; v < A; ++v)
            d[u][v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                          rp.rsrc, (int)(rowq + rp.col[v]), soff, 0));
    }
}

// Write the m x m output block of (tile tc, output channel k), cropped to Ho x Wo.
template <int MT>
__device__ __forceinline__ void store_block(float* __restrict__ y, const Geom& g,
                                            const TileCoord& tc, int k,
                                            const float (&o)[MT][MT], bool relu, bool vec_ok) {
    if (!tc.valid || k >= g.K) return;
    const int oi0 = tc.ti * MT, oj0 = tc.tj * MT;
    float* base = y + ((size_t)tc.n * g.K + k) * (size_t)g.Ho * (size_t)g.Wo;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
        const int oi = oi0 + i;
        if (oi >= g.Ho) break;
        float* row = base + (size_t)oi * g.Wo + oj0;
        float v[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) v[j] = relu ? fmaxf(o[i][j], 0.0f) : o[i][j];
        if (vec_ok && oj0 + MT <= g.Wo) {
            if constexpr (MT == 4) {
                *(float4*)row = make_float4(v[0], v[1], v[2], v[3]);
            } else {
                *(float2*)row = make_float2(v[0], v[1]);
            }
        } else {
#pragma unroll
            for (int j = 0; j < MT; ++j)
                if (oj0 + j < g.Wo) row[j] = v[j];
        }
    }
}

// ------------------------------------------------------------------ filter
// One wave per (16-filter block, 4-channel quad); lane = (c%4)*16 + k%16.
template <int MT>
__global__ __launch_bounds__(256) void k_filter(const float* __restrict__ gw, float* __restrict__ U,
                                                int C, int K, int CQ, int KB) {
    constexpr int T = (MT + 2) * (MT + 2);
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (long)KB * CQ) return;
    const int kb = (int)(w / CQ), cq = (int)(w % CQ);
    const int k = kb * 16 + (lane & 15), c = cq * 4 + (lane >> 4);
    float gg[3][3];
    const bool ok = k < K && c < C;
    const float* src = gw + ((size_t)(ok ? k : 0) * C + (ok ? c : 0)) * 9;
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int s = 0; s < 3; ++s) gg[r][s] = ok ? src[r * 3 + s] : 0.0f;
    float u[T];
    filter_tf<MT>(gg, u);
    float* dst = U + ((size_t)w * T) * 64 + lane;
#pragma unroll
    for (int t = 0; t < T; ++t) dst[t * 64] = u[t];
}

// ------------------------------------------------------------------ input
// One wave per (16-tile block, 4-channel quad); neighbouring waves take
// neighbouring tile blocks so their overlapping regions share cache lines.
template <int MT>
__global__ __launch_bounds__(256) void k_input(const float* __restrict__ x, float* __restrict__ V, Geom g) {
    constexpr int A = MT + 2, T = A * A;
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * g.CQ) return;
    const int cq = (int)(w / g.PB), pb = (int)(w % g.PB);
    const int cl = lane >> 4;
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const RegionPlan<MT> rp = make_region_plan<MT>(x, g, pb * 16, tc, cl);
    float d[A][A];
    load_region<MT>(rp, g, cq, cl, d);
    float v[T];
    input_tf<MT>(d, v);
    float* dst = V + (((size_t)pb * g.CQ + cq) * T) * 64 + lane;
#pragma unroll
    for (int t = 0; t < T; ++t) dst[t * 64] = v[t];
}

// ------------------------------------------------------------------ GEMM
// Per transform position t: M_t[k][p] = sum_c U_t[c][k] V_t[c][p].
// Workgroup tile: 4 k-blocks x 4 p-blocks (64 x 64), four waves each 2 x 2
// blocks of 16 x 16.  Channels advance 16 at a time (4 quads) through a double
// buffer in LDS; the next chunk is fetched into registers while the current
// one feeds the MFMAs.
__global__ __launch_bounds__(256) void k_gemm(const float* __restrict__ U, const float* __restrict__ V,
                                              float* __restrict__ M, Geom g) {
    __shared__ float As[2][4][4][64];   // [buf][quad][k-block][lane]
    __shared__ float Bs[2][4][4][64];   // [buf][quad][p-block][lane]
    const int t = blockIdx.y;
    const int KB4 = (g.KB + 3) >> 2;
    const int pb0 = (int)(blockIdx.x / KB4) * 4;
    const int kb0 = (int)(blockIdx.x % KB4) * 4;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wk = wave >> 1, wp = wave & 1;
    const int lblk = tid >> 4, lq = tid & 15, lcq = lblk >> 2, lbi = lblk & 3;
    const int nchunks = (g.CQ + 3) >> 2;
    const int T = g.T;

    float4 ra, rb;
    auto fetch = [&](int chunk) {
        const int cq = chunk * 4 + lcq;
        const int kb = kb0 + lbi, pb = pb0 + lbi;
        ra = make_float4(0.f, 0.f, 0.f, 0.f);
        rb = ra;
        if (cq < g.CQ && kb < g.KB)
            ra = *(const float4*)(U + (((size_t)kb * g.CQ + cq) * T + t) * 64 + lq * 4);
        if (cq < g.CQ && pb < g.PB)
            rb = *(const float4*)(V + (((size_t)pb * g.CQ + cq) * T + t) * 64 + lq * 4);
    };
    auto stage = [&](int buf) {
        *(float4*)&As[buf][lcq][lbi][lq * 4] = ra;
        *(float4*)&Bs[buf][lcq][lbi][lq * 4] = rb;
    };

    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    fetch(0);
    stage(0);
    __syncthreads();
    for (int ch = 0; ch < nchunks; ++ch) {
        const int buf = ch & 1;
        if (ch + 1 < nchunks) fetch(ch + 1);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float a0 = As[buf][q][wk * 2 + 0][lane];
            const float a1 = As[buf][q][wk * 2 + 1][lane];
            const float b0 = Bs[buf][q][wp * 2 + 0][lane];
            const float b1 = Bs[buf][q][wp * 2 + 1][lane];
            acc[0][0] = mfma16x16x4(a0, b0, acc[0][0]);
            acc[0][1] = mfma16x16x4(a0, b1, acc[0][1]);
            acc[1][0] = mfma16x16x4(a1, b0, acc[1][0]);
            acc[1][1] = mfma16x16x4(a1, b1, acc[1][1]);
        }
        if (ch + 1 < nchunks) stage(buf ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int kb = kb0 + wk * 2 + i, pb = pb0 + wp * 2 + j;
            if (kb < g.KB && pb < g.PB)
                *(f32x4*)(M + (((size_t)pb * g.KB + kb) * T + t) * 256 + lane * 4) = acc[i][j];
        }
    }
}

// ------------------------------------------------------------------ output
// One wave per (16-tile block, 16-filter block): each lane gathers the T
// accumulators of its four (tile, output channel) pairs and writes four m x m
// blocks.
template <int MT>
__global__ __launch_bounds__(256) void k_output(const float* __restrict__ M, float* __restrict__ y, Geom g,
                                                int relu, int vec_ok) {
    constexpr int T = (MT + 2) * (MT + 2);
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (long)g.PB * g.KB) return;
    const int pb = (int)(w / g.KB), kb = (int)(w % g.KB);
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const float* src = M + ((size_t)w * T) * 256 + lane * 4;
    f32x4 mv[T];
#pragma unroll
    for (int t = 0; t < T; ++t) mv[t] = *(const f32x4*)(src + t * 256);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float m1[T];
#pragma unroll
        for (int t = 0; t < T; ++t) m1[t] = mv[t][r];
        float o[MT][MT];
        output_tf<MT>(m1, o);
        store_block<MT>(y, g, tc, kb * 16 + 4 * (lane >> 4) + r, o, relu != 0, vec_ok != 0);
    }
}

// ------------------------------------------------------------------ fused
// Output unit of a wave: 16 tiles (one p-block) x 16*KSUB output channels, all
// T positions.  CSPLIT waves of a workgroup share one unit and take every
// CSPLIT-th channel quad; their partial results are output-transformed (the
// transform is linear) and summed through LDS in wave order 0, 1, ...
template <int MT, int KSUB, int CSPLIT>
__global__ __launch_bounds__(256) void k_fused(const float* __restrict__ x, const float* __restrict__ U,
                                               float* __restrict__ y, Geom g, int relu, int vec_ok) {
    constexpr int A = MT + 2, T = A * A;
    constexpr int UNITS = 4 / CSPLIT;            // output units per workgroup
    constexpr int NB = KSUB * 4;                 // (k-block, slot) output groups per lane
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cs = wave % CSPLIT;
    const int uw = wave / CSPLIT;
    const int KG = (g.KB + KSUB - 1) / KSUB;
    const long unit = (long)blockIdx.x * UNITS + uw;
    const bool active = unit < (long)g.PB * KG;
    const int pb = active ? (int)(unit / KG) : 0;
    const int kg = active ? (int)(unit % KG) : 0;
    const int cl = lane >> 4;
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);

    f32x4 acc[KSUB][T];
#pragma unroll
    for (int s = 0; s < KSUB; ++s)
#pragma unroll
        for (int t = 0; t < T; ++t) acc[s][t] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Channel quads of this wave: cs, cs + CSPLIT, ...  (nq of them).
    const int nq = (active && cs < g.CQ) ? (g.CQ - cs + CSPLIT - 1) / CSPLIT : 0;
    if (nq > 0) {
        const RegionPlan<MT> rp = make_region_plan<MT>(x, g, pb * 16, tc, cl);
        // U block of (k-block kb, quad cq) starts at ((kb*CQ + cq)*T)*64.  A k-block
        // past KB (only the last group when KSUB > 1) re-reads block KB-1; its
        // results belong to filters >= K and are never stored.
        const float* ublk[KSUB];
#pragma unroll
        for (int s = 0; s < KSUB; ++s)
            ublk[s] = U + ((size_t)min(kg * KSUB + s, g.KB - 1) * g.CQ * T) * 64 + lane;
        // Region values run one quad ahead in two register stages; each quad's
        // filter values are requested at the top of its step, so their latency
        // hides behind the input transform.
        float xa[A][A], xb[A][A];
        float ur[KSUB][T];
        auto load_x = [&](int i, float (&xr)[A][A]) { load_region<MT>(rp, g, cs + i * CSPLIT, cl, xr); };
        auto load_u = [&](int i) {
            const size_t q = (size_t)(cs + i * CSPLIT) * T * 64;
#pragma unroll
            for (int s = 0; s < KSUB; ++s)
#pragma unroll
                for (int t = 0; t < T; ++t) ur[s][t] = ublk[s][q + t * 64];
        };
        auto compute = [&](float (&xr)[A][A]) {
            float v[T];
            input_tf<MT>(xr, v);
#pragma unroll
            for (int s = 0; s < KSUB; ++s)
#pragma unroll
                for (int t = 0; t < T; ++t) acc[s][t] = mfma16x16x4(ur[s][t], v[t], acc[s][t]);
        };
        load_x(0, xa);
        int i = 0;
        for (; i + 1 < nq; i += 2) {
            load_u(i);
            load_x(i + 1, xb);
            compute(xa);
            load_u(i + 1);
            load_x(min(i + 2, nq - 1), xa);      // past the end: a harmless repeat load
            compute(xb);
        }
        if (i < nq) {
            load_u(i);
            compute(xa);
        }
    }

    if constexpr (CSPLIT == 1) {
        if (!active) return;
#pragma unroll
        for (int s = 0; s < KSUB; ++s) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float m1[T];
#pragma unroll
                for (int t = 0; t < T; ++t) m1[t] = acc[s][t][r];
                float o[MT][MT];
                output_tf<MT>(m1, o);
                store_block<MT>(y, g, tc, (kg * KSUB + s) * 16 + 4 * cl + r, o, relu != 0, vec_ok != 0);
            }
        }
    } else {
        static_assert(NB % CSPLIT == 0, "each wave must own whole output groups");
        __shared__ float red[UNITS][CSPLIT][NB][MT * MT][64];
#pragma unroll
        for (int s = 0; s < KSUB; ++s) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                float m1[T];
#pragma unroll
                for (int t = 0; t < T; ++t) m1[t] = acc[s][t][r];
                float o[MT][MT];
                output_tf<MT>(m1, o);
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < MT; ++j) red[uw][cs][s * 4 + r][i * MT + j][lane] = o[i][j];
            }
        }
        __syncthreads();
        if (!active) return;
        constexpr int PER = NB / CSPLIT;
#pragma unroll
        for (int b = 0; b < PER; ++b) {
            const int grp = cs * PER + b;        // (k-block s, slot r) = (grp / 4, grp % 4)
            float o[MT][MT];
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j) {
                    float sum = red[uw][0][grp][i * MT + j][lane];
#pragma unroll
                    for (int q = 1; q < CSPLIT; ++q) sum += red[uw][q][grp][i * MT + j][lane];
                    o[i][j] = sum;
                }
            store_block<MT>(y, g, tc, (kg * KSUB + grp / 4) * 16 + 4 * cl + (grp % 4), o,
                            relu != 0, vec_ok != 0);
        }
    }
}

// ------------------------------------------------------------------ maxpool
__global__ __launch_bounds__(256) void k_maxpool2x2(const float* __restrict__ x, float* __restrict__ y,
                                                    long total, int H, int W, int Ho, int Wo) {
    const long i = (long)blockIdx.x * 256 + threadIdx.x;
    if (i >= total) return;
    const int oj = (int)(i % Wo);
    const long r = i / Wo;
    const int oi = (int)(r % Ho);
    const long plane = r / Ho;
    const float* s = x + (size_t)plane * H * W + (size_t)(2 * oi) * W + 2 * oj;
    y[i] = fmaxf(fmaxf(s[0], s[1]), fmaxf(s[W], s[W + 1]));
}

// ------------------------------------------------------------------ launchers

static inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

hipError_t launch_filter_transform(const float* gw, float* U, int C, int K, int m, hipStream_t s) {
    const int CQ = (C + 3) / 4, KB = (K + 15) / 16;
    const long waves = (long)KB * CQ;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    if (m == 2)
        hipLaunchKernelGGL(k_filter<2>, grid, block, 0, s, gw, U, C, K, CQ, KB);
    else
        hipLaunchKernelGGL(k_filter<4>, grid, block, 0, s, gw, U, C, K, CQ, KB);
    return hipGetLastError();
}

hipError_t launch_input_transform(const float* x, float* V, const Geom& g, hipStream_t s) {
    const long waves = (long)g.PB * g.CQ;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    if (g.m == 2)
        hipLaunchKernelGGL(k_input<2>, grid, block, 0, s, x, V, g);
    else
        hipLaunchKernelGGL(k_input<4>, grid, block, 0, s, x, V, g);
    return hipGetLastError();
}

hipError_t launch_batched_gemm(const float* U, const float* V, float* M, const Geom& g, hipStream_t s) {
    const long tiles = (long)((g.PB + 3) / 4) * ((g.KB + 3) / 4);
    const dim3 grid((unsigned)tiles, (unsigned)g.T), block(256);
    hipLaunchKernelGGL(k_gemm, grid, block, 0, s, U, V, M, g);
    return hipGetLastError();
}

hipError_t launch_output_transform(const float* M, float* y, const Geom& g, bool relu, hipStream_t s) {
    const long waves = (long)g.PB * g.KB;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    const int vec_ok = (g.Wo % g.m == 0) && aligned(y, 4 * g.m);
    if (g.m == 2)
        hipLaunchKernelGGL(k_output<2>, grid, block, 0, s, M, y, g, (int)relu, vec_ok);
    else
        hipLaunchKernelGGL(k_output<4>, grid, block, 0, s, M, y, g, (int)relu, vec_ok);
    return hipGetLastError();
}

template <int MT, int KSUB, int CSPLIT>
static hipError_t fused_instance(const float* x, const float* U, float* y, const Geom& g, bool relu,
                                 hipStream_t s) {
    const int KG = (g.KB + KSUB - 1) / KSUB;
    const long units = (long)g.PB * KG;
    constexpr int UNITS = 4 / CSPLIT;
    const dim3 grid((unsigned)((units + UNITS - 1) / UNITS)), block(256);
    const int vec_ok = (g.Wo % MT == 0) && aligned(y, 4 * MT);
    hipLaunchKernelGGL((k_fused<MT, KSUB, CSPLIT>), grid, block, 0, s, x, U, y, g, (int)relu, vec_ok);
    return hipGetLastError();
}

hipError_t launch_fused(const float* x, const float* U, float* y, const Geom& g, FusedCfg c, bool relu,
                        hipStream_t s) {
#define WINO_FUSED_CASE(MT, KS, CS) \
    if (g.m == MT && c.ksub == KS && c.csplit == CS) return fused_instance<MT, KS, CS>(x, U, y, g, relu, s);
    WINO_FUSED_CASE(2, 1, 1)
    WINO_FUSED_CASE(2, 1, 2)
    WINO_FUSED_CASE(2, 1, 4)
    WINO_FUSED_CASE(2, 2, 1)
    WINO_FUSED_CASE(2, 2, 2)
    WINO_FUSED_CASE(2, 2, 4)
    WINO_FUSED_CASE(4, 1, 1)
    WINO_FUSED_CASE(4, 1, 2)
    WINO_FUSED_CASE(4, 1, 4)
#undef WINO_FUSED_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_maxpool2x2(const float* x, float* y, int N, int C, int H, int W, hipStream_t s) {
    const int Ho = H / 2, Wo = W / 2;
    const long total = (long)N * C * Ho * Wo;
    const dim3 grid((unsigned)((total + 255) / 256)), block(256);
    hipLaunchKernelGGL(k_maxpool2x2, grid, block, 0, s, x, y, total, H, W, Ho, Wo);
    return hipGetLastError();
}

size_t filter_elems(int C, int K, int m) {
    const size_t T = (size_t)(m + 2) * (m + 2);
    return T * (size_t)((C + 3) / 4) * 4 * (size_t)((K + 15) / 16) * 16;
}
size_t v_elems(const Geom& g) { return (size_t)g.PB * g.CQ * g.T * 64; }
size_t m_elems(const Geom& g) { return (size_t)g.PB * g.KB * g.T * 256; }

}  // namespace wino
