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
#include <atomic>
#include <mutex>
#include <type_traits>

#include "wino_internal.h"
#include "wino_transforms.h"

namespace wino {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma16x16x4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// The 16-bit form: fp16 (PREC 1) or bf16 (PREC 2), eight reduction slots per
// lane in a 16-byte operand, fp32 accumulation.
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

template <int PREC>
__device__ __forceinline__ f32x4 mfma16x16x32(uint4 a, uint4 b, f32x4 c) {
    if constexpr (PREC == 1)
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b),
                                                       c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                        __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv d) { return (__umulhi(n, d.m) + n) >> d.l; }

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
constexpr uint32_t kInvalid = kInvalidOffset;
constexpr int kRsrcWord3 = 0x00020000;   // raw (unformatted) 32-bit buffer

// Transformed filters as a raw buffer (the host keeps U below 2 GiB for the
// fused kernels).  A lane's 16-byte word of a U group sits at the constant
// per-lane offset lane*16 plus a wave-uniform group offset, so filter loads
// need no per-load address registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t u_rsrc(const float* U, const Geom& g) {
    const size_t ub = (size_t)g.KB * g.CQ * g.T * 256;
    return __builtin_amdgcn_make_buffer_rsrc((void*)U, (short)0, (int)(ub < 0x7fffffffu ? ub : 0x7fffffffu),
                                             kRsrcWord3);
}
__device__ __forceinline__ f32x4 u_load(__amdgpu_buffer_rsrc_t r, uint32_t lane_off, uint32_t group_off) {
    return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)lane_off, (int)group_off, 0));
}

// Regions of side A (MT + 2 for 3x3 filters, MT + 4 for 5x5) stepping by MT.
template <int MT, int A = MT + 2>
struct RegionPlan {
    __amdgpu_buffer_rsrc_t rsrc;     // wave-uniform
    uint32_t row[A];                 // lane's channel-plane + row byte offset, or kInvalid
    uint32_t col[A];                 // column byte offset, or kInvalid
    uint32_t plane_bytes;            // H*W*4: step between channels (soffset units)
};

// p0 = first tile of the wave's 16-tile block (wave-uniform); tc = lane's tile;
// cl = lane's channel within a quad.
template <int MT, int A = MT + 2>
__device__ __forceinline__ RegionPlan<MT, A> make_region_plan(const float* __restrict__ x, const Geom& g,
                                                              int p0, const TileCoord& tc, int cl) {
    RegionPlan<MT, A> rp;
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
template <int MT, int A = MT + 2>
__device__ __forceinline__ void load_region(const RegionPlan<MT, A>& rp, const Geom& g, int cq, int cl,
                                            float (&d)[A][A]) {
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

// Output rows leave through streaming (non-temporal) stores where a kernel
// writes whole cache lines: y is not read back, so it need not displace cached
// inputs.  Where the lines of a row are completed by several store
// instructions (rows narrower than a line run, or not line-aligned), plain
// stores let L2 merge the pieces before they go to HBM; streaming stores of
// such pieces run at half the bandwidth or less.
template <bool NT>
__device__ __forceinline__ void store_out(float* p, float a, float b, float c, float d) {
    const f32x4 q = {a, b, c, d};
    if constexpr (NT) __builtin_nontemporal_store(q, (f32x4*)p);
    else *(f32x4*)p = q;
}
template <bool NT>
__device__ __forceinline__ void store_out(float* p, float a, float b) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 q = {a, b};
    if constexpr (NT) __builtin_nontemporal_store(q, (f32x2*)p);
    else *(f32x2*)p = q;
}

// Write output row i (MT values) of the block of (tile tc, output channel k),
// cropped to Ho x Wo.
template <int MT, bool NT = true>
__device__ __forceinline__ void store_row(float* __restrict__ y, const Geom& g, const TileCoord& tc, int k,
                                          int i, const float (&o)[MT], bool relu, bool vec_ok) {
    const int oi = tc.ti * MT + i, oj0 = tc.tj * MT;
    if (!tc.valid || k >= g.K || oi >= g.Ho) return;
    float* row = y + (((size_t)tc.n * g.K + k) * (size_t)g.Ho + oi) * (size_t)g.Wo + oj0;
    float v[MT];
#pragma unroll
    for (int j = 0; j < MT; ++j) v[j] = relu ? fmaxf(o[j], 0.0f) : o[j];
    if (vec_ok && oj0 + MT <= g.Wo) {
        if constexpr (MT == 4) {
            store_out<NT>(row, v[0], v[1], v[2], v[3]);
        } else {
            store_out<NT>(row, v[0], v[1]);
        }
    } else {
        // Plain 4-byte stores, whatever NT says: they merge into whole lines
        // in L2, where non-temporal ones went out as partial-line writes
        // (25-30% of the split and fused calls on 26-30 pixel wide layers).
#pragma unroll
        for (int j = 0; j < MT; ++j)
            if (oj0 + j < g.Wo) row[j] = v[j];
    }
}

// Write the m x m output block of (tile tc, output channel k), cropped to Ho x Wo.
template <int MT, bool NT = true>
__device__ __forceinline__ void store_block(float* __restrict__ y, const Geom& g,
                                            const TileCoord& tc, int k,
                                            const float (&o)[MT][MT], bool relu, bool vec_ok) {
#pragma unroll
    for (int i = 0; i < MT; ++i) store_row<MT, NT>(y, g, tc, k, i, o[i], relu, vec_ok);
}

// Channel-last y [N][Ho][Wo][K]: the m x m outputs of (tile tc, output channels
// k0 .. k0+3), cropped to Ho x Wo and K; one 16-byte store per pixel when vec
// (K % 4 == 0 and y 16-byte aligned), streaming when NT.
template <int MT, bool NT = false>
__device__ __forceinline__ void store_tile_nhwc(float* __restrict__ y, const Geom& g, const TileCoord& tc, int k0,
                                                const float (&o)[4][MT][MT], bool relu, bool vec) {
    if (!tc.valid || k0 >= g.K) return;
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int oi = tc.ti * MT + i, oj = tc.tj * MT + j;
            if (oi >= g.Ho || oj >= g.Wo) continue;
            float* py = y + (((size_t)tc.n * g.Ho + oi) * g.Wo + oj) * g.K + k0;
            float v[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = relu ? fmaxf(o[r][i][j], 0.0f) : o[r][i][j];
            if (vec && k0 + 4 <= g.K) {
                store_out<NT>(py, v[0], v[1], v[2], v[3]);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (k0 + r < g.K) py[r] = v[r];
            }
        }
}

// Store a lane's T transform-domain values into one (block, quad) group of the
// U/V layout [T/4][64][4]: one 16-byte store per group of four positions, the
// wave writing whole 1 KiB runs.  NT: streaming stores (measured: faster for
// the staged input transform, slower for the split path's).
template <int T, bool NT>
__device__ __forceinline__ void store_t4(float* __restrict__ blk, int lane, const float (&v)[T]) {
#pragma unroll
    for (int g4 = 0; g4 < T / 4; ++g4)
        store_out<NT>(blk + ((size_t)g4 * 64 + lane) * 4, v[4 * g4], v[4 * g4 + 1], v[4 * g4 + 2], v[4 * g4 + 3]);
}

// ------------------------------------------------------------------ filter
// Filter pairs (16 filters x 4 channels) from which one wave per pair computes
// all positions.
constexpr long kFilterAllPairs = 256;

// The 4-position group tg (wave-uniform) of a lane's filter transform: a
// branch per group, each computing only its own positions.
template <int MT, int R, int... G>
__device__ __forceinline__ float4 filter_pick(int tg, const float (&g)[R][R], std::integer_sequence<int, G...>) {
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    ((tg == G ? (void)(o = filter_tf4<MT, 4 * G, R>(g)) : (void)0), ...);
    return o;
}

// All position groups of a lane's filter transform, group G to U + G*256.
template <int MT, int R, int... G>
__device__ __forceinline__ void filter_all(const float (&g)[R][R], float* __restrict__ u,
                                           std::integer_sequence<int, G...>) {
    ((*(float4*)(u + G * 256) = filter_tf4<MT, 4 * G, R>(g)), ...);
}

// One wave per (16-filter block, 4-channel quad) -- or, for layers with few
// filter pairs, per (block, quad, group of four positions), which widens the
// grid T/4 times and keeps the latency of the small case down.  Lane =
// (c%4)*16 + k%16, so each group the wave writes is one contiguous 1 KiB run of
// U with a 16-byte store per lane.  Four waves per workgroup.  With STAGE (one
// wave per pair and CQ % 4 == 0) the workgroup's four quads are 16 consecutive
// channels of the same 16 filters: it reads their 16 runs of 16*R*R contiguous
// floats of g with coalesced loads into LDS first.  R: filter side (3 or 5).
template <int MT, bool ALL, bool STAGE, int R = 3>
__global__ __launch_bounds__(256) void k_filter(const float* __restrict__ gw, float* __restrict__ U,
                                                int C, int K, int CQ, long nw) {
    constexpr int A = MT + R - 1, T = A * A, TG = T / 4, RR = R * R, RUN = 16 * RR;
    static_assert(ALL || !STAGE, "staging needs one wave per pair");
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    float gg[R][R];
    long pair;
    if constexpr (STAGE) {
        __shared__ float gs[16 * RUN];                // [filter][16 channels x R*R]
        const long p0 = (long)blockIdx.x * 4;         // nw % 4 == 0: every wave is valid
        const int kb = (int)(p0 / CQ), c0 = (int)(p0 % CQ) * 4;
#pragma unroll
        for (int i = 0; i < RR; ++i) {
            const int e = (int)threadIdx.x + 256 * i, row = e / RUN, off = e - row * RUN;
            const int k = kb * 16 + row, c = c0 + off / RR;
            gs[e] = (k < K && c < C) ? gw[((size_t)k * C + c0) * RR + off] : 0.0f;
        }
        __syncthreads();
        pair = w;
        const float* src = gs + (lane & 15) * RUN + ((int)(w - p0) * 4 + (lane >> 4)) * RR;
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int s = 0; s < R; ++s) gg[r][s] = src[r * R + s];
    } else {
        if (w >= nw) return;
        pair = ALL ? w : w / TG;                      // kb * CQ + cq
        const int kb = (int)(pair / CQ), cq = (int)(pair % CQ);
        const int k = kb * 16 + (lane & 15), c = cq * 4 + (lane >> 4);
        const bool ok = k < K && c < C;
        const float* src = gw + ((size_t)(ok ? k : 0) * C + (ok ? c : 0)) * RR;
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int s = 0; s < R; ++s) gg[r][s] = ok ? src[r * R + s] : 0.0f;
    }
    if constexpr (ALL) {
        filter_all<MT, R>(gg, U + ((size_t)pair * TG * 64 + lane) * 4, std::make_integer_sequence<int, TG>{});
    } else {
        *(float4*)(U + ((size_t)w * 64 + lane) * 4) =
            filter_pick<MT, R>((int)(w % TG), gg, std::make_integer_sequence<int, TG>{});
    }
}

// ------------------------------------------------------------------ input
// One wave per (16-tile block, 4-channel quad); neighbouring waves take
// neighbouring tile blocks so their overlapping regions share cache lines, and
// each XCD takes one contiguous run of workgroups (workgroup b runs item
// (b % 8) * per + b / 8), so those neighbours meet in the same L2.
template <int MT, int R = 3>
__global__ __launch_bounds__(256) void k_input(const float* __restrict__ x, float* __restrict__ V, Geom g,
                                               long nwg) {
    constexpr int A = MT + R - 1, T = A * A;
    const int lane = threadIdx.x & 63;
    const long per = (nwg + 7) / 8, item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nwg) return;
    const long w = item * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * g.CQ) return;
    const int cq = (int)(w / g.PB), pb = (int)(w % g.PB);
    const int cl = lane >> 4;
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const RegionPlan<MT, A> rp = make_region_plan<MT, A>(x, g, pb * 16, tc, cl);
    float d[A][A];
    load_region<MT, A>(rp, g, cq, cl, d);
    float v[T];
    input_tf<A - 2>(d, v);                 // B^T depends only on the region side (the points)
    store_t4<T, true>(V + ((size_t)pb * g.CQ + cq) * T * 64, lane, v);
}

// ------------------------------------------------------------------ output
// A workgroup owns whole rows of tiles of one image (R rows of tw <= 64 tiles,
// or a 64-tile piece of one row) for one 16-filter block: wave = filter quad,
// lane = tile.  Each lane gathers the T values of its four (tile, filter) pairs
// from the blocked M and writes four m x m blocks, so the workgroup writes, per
// filter, output rows that together cover whole rows of y -- the pieces of a
// cache line come from the same wave, moments apart, and merge in L2.
template <int MT, int RF = 3>
__global__ __launch_bounds__(256) void k_output(const float* __restrict__ M, float* __restrict__ y, Geom g,
                                                int relu, int vec_ok, int R, int segs, int ipi, int nitems) {
    constexpr int T = (MT + RF - 1) * (MT + RF - 1);
    const int lane = threadIdx.x & 63, kq = threadIdx.x >> 6;
    const int item = (int)(blockIdx.x % (unsigned)nitems), kb = (int)(blockIdx.x / (unsigned)nitems);
    const int n = item / ipi, it = item - n * ipi;
    TileCoord tc;
    tc.n = n;
    if (segs == 0) {                        // R whole rows of tw tiles
        tc.ti = it * R + lane / g.tw;
        tc.tj = lane % g.tw;
        tc.valid = lane < R * g.tw && tc.ti < g.th;
    } else {                                // piece it % segs of row it / segs
        tc.ti = it / segs;
        tc.tj = (it % segs) * 64 + lane;
        tc.valid = tc.tj < g.tw;
    }
    const int p = tc.valid ? (n * g.th + tc.ti) * g.tw + tc.tj : 0;
    // element (t, k, p) of M: lane 16*((k%16)/4) + p%16, slot k%4 of block (p/16, k/16, t)
    const float* src = M + (((size_t)(p / 16) * g.KB + kb) * T) * 256 + (16 * kq + p % 16) * 4;
    f32x4 mv[T];
#pragma unroll
    for (int t = 0; t < T; ++t) mv[t] = tc.valid ? *(const f32x4*)(src + t * 256) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float m1[T];
#pragma unroll
        for (int t = 0; t < T; ++t) m1[t] = mv[t][r];
        float o[MT][MT];
        output_tf<MT, RF>(m1, o);
        store_block<MT, false>(y, g, tc, kb * 16 + 4 * kq + r, o, relu != 0, vec_ok != 0);
    }
}

// ------------------------------------------------------------------ fused
// One workgroup of 8 waves computes one tile block (16 tiles: 1 x 16 or 4 x 4)
// for KGW 16-filter blocks, over all channels, all T positions, start to end.
// RF is the filter side: 3, or 5 with m = 2 (6 x 6 regions like m = 4's).
// The 8 waves are (filter block kw) x (row group h of TS) x (channel split cs
// of CS): wave h owns transform-domain rows [h*A/TS, (h+1)*A/TS), i.e. T/TS
// accumulators per lane.
//
// The channel loop advances QS = KGW*CS = 8/TS quads per step.  Within a step,
// quad j = kw*CS + cs is input-transformed by wave (kw, h, cs) for its rows --
// every wave transforms exactly one region set per step -- and each wave then
// multiplies the KGW quads of its channel split (j = kw'*CS + cs) with its own
// filter block.  With KGW > 1 the transforms are exchanged through one LDS
// stage, written for step s+1 after step s's products; with KGW = 1 they stay
// in registers.
//
// The halo'd input patch of a step comes straight into LDS (buffer loads with
// an LDS destination, no register round trip) two steps ahead (three with
// KGW > 1, whose transform runs a step early), in three stages
// that are distinct LDS objects, so the compiler can see that reading one stage
// never waits for loads still landing in another.  Rows, columns and channels
// outside the image and the alignment columns are offsets past the buffer
// record and read as 0.  Filters go straight to registers ahead of their use
// (no other wave uses them), one 16-byte load per 4 positions.  The region's input
// transform gives exactly the B operand of v_mfma_f32_16x16x4_f32.  At the end
// the CS channel parts of a (filter block, row group) first sum their
// accumulators through LDS, each wave keeping a 1/CS share of the (filter,
// position) values; each wave then applies its row group's part of A^T M A
// (linear in M) to its share, and the row groups' partial outputs are summed
// through LDS once more.  Both sums run in a fixed order.
template <int MT, int TS, int CS, int BW, int VEC, int R = 3>
struct FusedShape {
    static constexpr int A = MT + R - 1, T = A * A, RN = A / TS, TH = RN * A;
    static constexpr int PARTS = TS * CS, KGW = 8 / PARTS, BH = 16 / BW;
    static constexpr int QS = KGW * CS;                    // quads per step (= 8 / TS)
    static constexpr bool SHARE = KGW > 1;                 // transforms exchanged through LDS
    static constexpr int PR = BH * MT + R - 1;             // patch rows
    static constexpr int PC = BW * MT + R - 1;             // patch columns
    // VEC: the patch rows come as 16-byte chunks starting at the 4-aligned column
    // at or before the patch (up to 3 columns early); else one float per load.
    static constexpr int EW = VEC ? 4 : 1;                 // floats per load
    static constexpr int PCP = VEC ? (PC + 6) / 4 * 4 : (PC + 3) / 4 * 4;   // row pitch, 16-byte aligned
    static constexpr int NE = PCP / EW;                    // loads per patch row
    static constexpr int XS = 4 * QS * PR * PCP;           // patch floats per step
    static constexpr int JX = (XS / EW + 511) / 512;       // patch loads per thread per step
    static constexpr int XSP = JX * 512 * EW;
    // PRIV (one filter block per workgroup, row blocks, 16-byte loads, one row
    // group): each wave loads its own quad's patch into a region of its own, so
    // the channel loop needs no workgroup barrier (F(2x2,3x3) on the N=1
    // 32-channel 56x56 layer: 4.99 -> 4.86 us).  With two row groups a wave
    // would need 5 of the 6 region rows (Bt rows 0-2 use region rows 0-4,
    // rows 3-5 use 1-5), 1.7x the shared patch bytes, and that cost what the
    // barriers did (10.05 against 10.12 us on the N=1 64-channel layer).
    static constexpr bool PRIV = !SHARE && BH == 1 && VEC && TS == 1;
    static constexpr int XW = 4 * A * PCP;                 // floats of a wave's patch (PRIV)
    static constexpr int JXW = (XW / EW + 63) / 64;        // its loads per lane per step
    static constexpr int XSTW = JXW * 64 * EW + 4 * VEC;   // floats of a wave's stage region
    static constexpr int NJ = PRIV ? JXW : JX;             // patch loads per lane per step
    static constexpr int XST = PRIV ? 8 * XSTW : XSP + 4 * VEC;   // floats of one patch stage
    static constexpr int VSZ = TS * QS * TH * 64;          // floats of one transform stage
    // Epilogue.  Channel sum: value f = r*TH + t of a lane (filter slot r,
    // position t of its row group) goes to wave f / V1 of the CS channel parts;
    // a wave then owns NF whole filters (CS <= 4) or one filter's rows of one of
    // PH halves of the row group (CS = 8).  Output sum: the G2 waves holding
    // partial outputs of one filter set (row groups x halves) keep NR2 of its NR
    // output rows each.  Only runs bound for another wave pass through LDS
    // (G2*(G2-1) blocks per filter set; CS*(CS-1) per (filter block, row
    // group) when CS <= 4); with CS = 8 every run does, so that the sum needs
    // no per-wave copy of its code (measured faster there).
    static constexpr int NFG = CS < 4 ? CS : 4, NF = 4 / NFG, PH = CS > 4 ? CS / 4 : 1;
    static constexpr int V1 = 4 * TH / CS, VW1 = V1 % 4 == 0 ? 4 : 2;
    static constexpr int G2 = TS * PH, NR = NF * MT, NR2 = NR / G2;
    static constexpr bool OWN1 = CS <= 4;                                    // own run kept in registers
    static constexpr int NB1 = OWN1 ? CS - 1 : CS;                           // channel-sum blocks per run
    static constexpr int EX1 = KGW * TS * CS * NB1 * V1 * 64;                // floats of the channel sum
    static constexpr int EX2 = KGW * NFG * G2 * (G2 - 1) * NR2 * MT * 64;    // floats of the output sum
    static constexpr int EXF = EX1 + EX2;                                    // disjoint ranges
    // LDS: three patch stages, then the transform stage (SHARE); the epilogue
    // reuses the whole allocation, which the last object is sized to cover.
    static constexpr int VSN0 = SHARE ? VSZ : 0;
    static constexpr int VSN1 = EXF > 3 * XST + VSN0 ? EXF - 3 * XST : VSN0;
    static constexpr int VSN = VSN1 > 4 ? VSN1 : 4;
    static constexpr int LDS_FLOATS = 3 * XST + VSN;
    static constexpr int LDS_BYTES = 4 * LDS_FLOATS;
    static_assert(KGW * PARTS == 8, "8 waves per workgroup");
    static_assert(T % 4 == 0, "positions come in groups of 4");
    static_assert(CS == 1 || CS == 2 || CS == 4 || CS == 8, "channel parts");
    static_assert(PH == 1 || (TS == 1 && RN % PH == 0), "row halves of a single row group");
    static_assert(V1 % 2 == 0 && NR % G2 == 0, "exchange granularity");
    static_assert(XST % 4 == 0 && VSN % 4 == 0, "16-byte LDS objects");
};

// s_waitcnt immediate: vmcnt <= n, lgkmcnt = 0, expcnt unconstrained.
template <int n>
__device__ __forceinline__ void wait_vm_lds() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((n & 15) | (7 << 4) | (0 << 8) | (((n >> 4) & 3) << 14));
}

// Workgroup barrier without the release fence of __syncthreads(): that fence
// would also wait for the direct-to-LDS loads still in flight for later steps.
// Callers first wait for exactly the loads (vmcnt) and LDS operations
// (lgkmcnt) the other waves need; the memory clobber keeps the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void wg_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int R> using IC = std::integral_constant<int, R>;

// f(IC<I>) for I = I0 .. I1-1, in order.
template <int I0, int I1, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (I0 < I1) {
        f(IC<I0>{});
        static_for<I0 + 1, I1>(f);
    }
}

// f(IC<v>) for the runtime value v in [0, N) (wave-uniform): one instance per value.
template <typename F, int... I>
__device__ __forceinline__ void with_ic(int v, F&& f, std::integer_sequence<int, I...>) {
    ((v == I ? (f(IC<I>{}), 0) : 0), ...);
}

template <int MT, int TS, int CS, int BW, int VEC, int H, int RF>
__device__ __forceinline__ void fused_steps(const __amdgpu_buffer_rsrc_t xr,
                                            const uint32_t (&xoff)[FusedShape<MT, TS, CS, BW, VEC, RF>::NJ],
                                            uint32_t step_b, const float* __restrict__ U, const Geom& g,
                                            const FusedTiling& ft, int kb, int wave, int lane, int kw, int cs,
                                            int bi, int bj, float* xs0, float* xs1, float* xs2, float* vs,
                                            f32x4 (&acc)[FusedShape<MT, TS, CS, BW, VEC, RF>::TH], int xlo,
                                            int cq0, int cqn, int nsteps) {
    using S = FusedShape<MT, TS, CS, BW, VEC, RF>;
    constexpr int A = S::A, RN = S::RN, X0 = H * RN, TH = S::TH, T = S::T, QS = S::QS, KGW = S::KGW;
    constexpr int G0 = X0 * A / 4, NG = (X0 * A + TH - 1) / 4 - G0 + 1;   // this row group's position groups
    const int cl = lane >> 4;
    const int jt = kw * CS + cs;          // the quad this wave transforms in every step

    auto xstage = [&](auto rc) -> float* {
        constexpr int R = decltype(rc)::value % 3;
        if constexpr (R == 0) return xs0;
        else if constexpr (R == 1) return xs1;
        else return xs2;
    };
    // Patch of step j -> stage j % 3 (with KGW > 1 a step past the last reads
    // zeros into a stage nobody reads, so every step issues exactly JX loads).
    auto issue_x = [&](auto rc, int j) {
        float* xs = xstage(rc);
        const uint32_t cbase = (uint32_t)j * step_b;
        if constexpr (S::PRIV) {
#pragma unroll
            for (int i = 0; i < S::JXW; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, xs + wave * S::XSTW + xlo + i * 64 * S::EW, 4 * S::EW,
                                                         xoff[i] + cbase, 0, 0, 0);
        } else {
#pragma unroll
            for (int i = 0; i < S::JX; ++i)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, xs + xlo + (i * 512 + wave * 64) * S::EW, 4 * S::EW,
                                                         xoff[i] + cbase, 0, 0, 0);
        }
    };
    // Filters of (step j, quad slot q) of the channel slice [cq0, cq0 + cqn): a
    // quad past the slice repeats a valid block (it meets zero regions, the
    // patch buffer ending at the slice); past the last step it repeats the last.
    const __amdgpu_buffer_rsrc_t ur = u_rsrc(U, g);
    const uint32_t ulane = (uint32_t)lane * 16u;
    auto load_u = [&](int j, int q, f32x4 (&ug)[NG]) {
        const int cq = cq0 + min(min(j, nsteps - 1) * QS + q, cqn - 1);
        const uint32_t go = __builtin_amdgcn_readfirstlane((uint32_t)(((kb * g.CQ + cq) * (T / 4) + G0) * 1024));
#pragma unroll
        for (int i = 0; i < NG; ++i) ug[i] = u_load(ur, ulane, go + i * 1024u);
    };
    auto transform = [&](auto rc, float (&v)[TH]) {
        // VEC: the patch's first column sits 4 floats in (or at 0 when the
        // chunks start on it), so region rows stay 16-byte aligned (8-byte
        // aligned for m = 2).
        const float* wp = S::PRIV ? xstage(rc) + wave * S::XSTW + cl * A * S::PCP + bj * MT + (xlo ? 4 : 0)
                                  : xstage(rc) + ((jt * 4 + cl) * S::PR + bi * MT) * S::PCP + bj * MT + (xlo ? 4 : 0);
        float d[A][A];
#pragma unroll
        for (int u = 0; u < A; ++u) {
            const float* row = wp + u * S::PCP;
            if constexpr (MT == 4) {
                const float4 a4 = *(const float4*)row;
                const float2 b2 = *(const float2*)(row + 4);
                d[u][0] = a4.x; d[u][1] = a4.y; d[u][2] = a4.z; d[u][3] = a4.w; d[u][4] = b2.x; d[u][5] = b2.y;
            } else {
#pragma unroll
                for (int v2 = 0; v2 < A / 2; ++v2) {
                    const float2 a2 = *(const float2*)(row + 2 * v2);
                    d[u][2 * v2] = a2.x; d[u][2 * v2 + 1] = a2.y;
                }
            }
        }
        // B^T depends only on the region side (the points): F(2x2,5x5) uses F(4x4,3x3)'s.
        input_tf_rows<A - 2, X0, RN>(d, v);
    };
    auto mfma_quad = [&](const float (&v)[TH], const f32x4 (&ug)[NG]) {
#pragma unroll
        for (int t = 0; t < TH; ++t) {
            const int idx = X0 * A + t;
            acc[t] = mfma16x16x4(ug[idx / 4 - G0][idx % 4], v[t], acc[t]);
        }
    };

    f32x4 ua[NG], ub[NG];
    if constexpr (!S::SHARE) {
        // Step s: transform quad cs of step s (patch landed two steps ago), one
        // quad of MFMAs.  Filters also come two steps ahead, into a ring of three
        // register sets that follows the three patch stages.
        constexpr int WAITN = S::NJ + NG;     // loads issued in the previous step
        f32x4 uc[NG];
        auto uring = [&](auto rc) -> f32x4 (&)[NG] {
            constexpr int R = decltype(rc)::value % 3;
            if constexpr (R == 0) return ua;
            else if constexpr (R == 1) return ub;
            else return uc;
        };
        // No loads past the last step: the last step waits for everything.
        issue_x(IC<0>{}, 0);
        load_u(0, cs, ua);
        if (nsteps > 1) {
            issue_x(IC<1>{}, 1);
            load_u(1, cs, ub);
        }
        auto step = [&](auto rc, int s) {  // s % 3 == R
            constexpr int R = decltype(rc)::value;
            // patch and filters of step s have landed (for this wave)
            if (s + 1 < nsteps) wait_vm_lds<WAITN>();
            else wait_vm_lds<0>();
            // ... for every wave; step s-1 is fully consumed (PRIV: the wave's
            // own loads are all it reads)
            if constexpr (!S::PRIV) wg_barrier();
            // The patch DMA goes out first; the filters of step s+2 only after this
            // step's MFMAs, so the two bursts do not queue together at the step start.
            if (s + 2 < nsteps) issue_x(IC<(R + 2) % 3>{}, s + 2);   // that stage held step s-1's patch
            __builtin_amdgcn_sched_barrier(0);   // keep the prefetch ahead of this step's work
            float v[TH];
            transform(IC<R>{}, v);
            mfma_quad(v, uring(IC<R>{}));
            __builtin_amdgcn_sched_barrier(0);
            if (s + 2 < nsteps) load_u(s + 2, cs, uring(IC<(R + 2) % 3>{}));
        };
        int s = 0;
        for (; s + 3 <= nsteps; s += 3) {   // straight-line body: exact wait analysis
            step(IC<0>{}, s);
            step(IC<1>{}, s + 1);
            step(IC<2>{}, s + 2);
        }
        if (s < nsteps) step(IC<0>{}, s);
        if (s + 1 < nsteps) step(IC<1>{}, s + 1);
    } else {
        // Step s: for each filter-block slot kw' the MFMAs of quad kw'*CS + cs
        // from the V stage, then (after every wave has read it) the transform of
        // quad jt of step s+1 into the same stage.  One V stage [(h*QS + quad)][t][64]:
        // VALU and MFMA work of one SIMD do not overlap on this chip, so a second
        // stage would only buy scheduling freedom, and without it the patch
        // stages fit LDS with 16-byte loads.
        // The loads of a step, in issue order: the filters of its quad slots
        // (KGW * NG, the last NG for the next step's first slot), then at its
        // end the patch DMA three steps ahead (JX).  A filter load waits (by
        // its register) for every older load, so the DMA goes last: the
        // filters of step s then wait only for the DMA issued at the end of
        // step s-1.  Before transforming patch s+1 (DMA'd at the end of step
        // s-2, or in the prologue) at most WAITT newer loads may be pending.
        constexpr int WAITT = S::JX + NG + KGW * NG < 63 ? S::JX + NG + KGW * NG : 63;
        float* vbase = vs + (H * QS) * TH * 64 + lane;
        auto put_v = [&](const float (&v)[TH]) {
            float* p = vbase + jt * TH * 64;
#pragma unroll
            for (int t = 0; t < TH; ++t) p[t * 64] = v[t];
        };
        issue_x(IC<0>{}, 0);
        issue_x(IC<1>{}, 1);
        issue_x(IC<2>{}, 2);
        load_u(0, cs, ua);
        wait_vm_lds<2 * S::JX + NG>();       // step 0's patch has landed
        wg_barrier();
        {
            float v[TH];
            transform(IC<0>{}, v);
            put_v(v);
        }
        auto step = [&](auto rc, int s) {  // s % 3 == R
            constexpr int R = decltype(rc)::value;
            wait_vm_lds<63>();             // this wave's V(s) writes are done (LDS only)
            wg_barrier();                  // ... every wave's
            // Quad slots k2 = 0 .. KGW-1: the V values and filters of slot k2+1
            // are requested before slot k2's MFMAs (scheduling barriers keep the
            // compiler from sinking them back next to their uses).
            const float* vp = vbase + cs * TH * 64;
            float va[TH], vb[TH];
#pragma unroll
            for (int t = 0; t < TH; ++t) va[t] = vp[t * 64];
#pragma unroll
            for (int k2 = 0; k2 < KGW; ++k2) {
                f32x4 (&ucur)[NG] = (k2 & 1) ? ub : ua;
                f32x4 (&unext)[NG] = (k2 & 1) ? ua : ub;
                float (&vcur)[TH] = (k2 & 1) ? vb : va;
                float (&vnext)[TH] = (k2 & 1) ? va : vb;
                if (k2 + 1 < KGW) {
                    load_u(s, (k2 + 1) * CS + cs, unext);
                    const float* p = vp + (k2 + 1) * CS * TH * 64;
#pragma unroll
                    for (int t = 0; t < TH; ++t) vnext[t] = p[t * 64];
                } else {
                    load_u(s + 1, cs, unext);
                }
                __builtin_amdgcn_sched_barrier(0);
                mfma_quad(vcur, ucur);
                __builtin_amdgcn_sched_barrier(0);
            }
            if constexpr (KGW & 1) {       // keep "ua holds the current filters" at step starts
#pragma unroll
                for (int i = 0; i < NG; ++i) ua[i] = ub[i];
            }
            if (s + 1 < nsteps) {
                wait_vm_lds<WAITT>();      // patch s+1 has landed and V(s) is read (this wave)
                wg_barrier();              // ... every wave
                float v[TH];
                transform(IC<(R + 1) % 3>{}, v);
                put_v(v);
            }
            issue_x(IC<R>{}, s + 3);       // stage R held patch s, transformed at the end of step s-1
        };
        int s = 0;
        for (; s + 3 <= nsteps; s += 3) {   // straight-line body: exact wait analysis
            step(IC<0>{}, s);
            step(IC<1>{}, s + 1);
            step(IC<2>{}, s + 2);
        }
        if (s < nsteps) step(IC<0>{}, s);
        if (s + 1 < nsteps) step(IC<1>{}, s + 1);
    }
    __builtin_amdgcn_s_waitcnt(0);         // no load outlives the loop
}

// o[r] = this wave's share of the m x m output of (tile, filter 16*kb + 4*cl + r)
template <int MT, int TS, int CS, int BW, int VEC, int H>
__device__ __forceinline__ void fused_share(const f32x4 (&acc)[FusedShape<MT, TS, CS, BW, VEC>::TH],
                                            float (&o)[4][MT][MT]) {
    using S = FusedShape<MT, TS, CS, BW, VEC>;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float m1[S::TH];
#pragma unroll
        for (int t = 0; t < S::TH; ++t) m1[t] = acc[t][r];
        output_tf_rows<MT, H * S::RN, S::RN>(m1, o[r]);
    }
}

template <int MT, int TS, int CS, int BW, int VEC, int RF = 3>
__global__ __launch_bounds__(512) void k_fused(const float* __restrict__ x, const float* __restrict__ U,
                                               float* __restrict__ y, Geom g, FusedTiling ft, int relu,
                                               int vec_ok, int nts, float* __restrict__ ypart) {
    using S = FusedShape<MT, TS, CS, BW, VEC, RF>;
    constexpr int PARTS = S::PARTS, KGW = S::KGW;
    __shared__ float4 xs0[S::XST / 4], xs1[S::XST / 4], xs2[S::XST / 4];   // patch stages
    __shared__ float4 vs[S::VSN / 4];                      // transform stages (SHARE)

    // Work item, XCD-aware: workgroups go round-robin to the 8 XCDs, so XCD
    // (b % 8) gets the contiguous run [xcd*per, (xcd+1)*per) of the item order.
    // Filter-group-major order keeps one or two groups' filters in an XCD's L2;
    // tile-major order (kfast) keeps the XCD's input patches there instead, and
    // every filter group of a patch reads it from L2.
    // With channel slices the slice is the slowest index of the item.
    const int b = blockIdx.x;
    const int per_sl = ft.nt * ft.nkg;
    const int item0 = (b & 7) * ft.per + (b >> 3);
    if (item0 >= per_sl * ft.nsl) return;
    const int sl = ft.nsl > 1 ? (int)fdiv((uint32_t)item0, ft.d_sl) : 0;
    const int item = item0 - sl * per_sl;
    const int iq = (int)fdiv((uint32_t)item, ft.d_item), ir = item - iq * (ft.kfast ? ft.nkg : ft.nt);
    const int kgi = ft.kfast ? ir : iq;
    const int tb = ft.kfast ? iq : ir;
    const int n = (int)fdiv((uint32_t)tb, ft.d_img), r2 = tb - n * (ft.nbh * ft.nbw);
    const int bq = (int)fdiv((uint32_t)r2, ft.d_nbw);
    const int ti0 = bq * S::BH, tj0 = (r2 - bq * ft.nbw) * BW;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int kw = wave / PARTS, part = wave % PARTS, h = part % TS, cs = part / TS;
    const int kb = min(kgi * KGW + kw, g.KB - 1);    // a block past KB only re-reads KB-1; never stored
    const int l16 = lane & 15, bi = l16 / BW, bj = l16 % BW, cl = lane >> 4;
    TileCoord tc;
    tc.n = n;
    tc.ti = ti0 + bi;
    tc.tj = tj0 + bj;
    tc.valid = tc.ti < g.th && tc.tj < g.tw;

    // Patch load e = j*512 + tid of [4*QS channels][PR][NE loads]: its byte
    // offset in image n for step 0 (kInvalid outside the image or past the
    // row).  VEC: loads are 16-byte chunks from column col0, which is the patch's
    // first column moved back by xsh to a multiple of 4; with W % 4 == 0 every
    // chunk lies wholly inside or wholly outside the row.
    // The buffer covers this slice's channels of image n only: channels past
    // the slice (or past C) read as zeros.
    const int cq0 = sl * ft.qsl, cqn = min(ft.qsl, g.CQ - cq0);
    const int c0 = cq0 * 4, cn = min(g.C - c0, cqn * 4);
    const int nsteps = (cqn + S::QS - 1) / S::QS;
    const size_t img = (size_t)g.C * g.H * g.W;
    const size_t sl_b = (size_t)cn * g.H * g.W * 4;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + (size_t)n * img + (size_t)c0 * g.H * g.W), (short)0, (int)(sl_b < kInvalid ? sl_b : kInvalid),
        kRsrcWord3);
    const uint32_t plane_b = (uint32_t)g.H * g.W * 4;
    // In LDS the chunks start xlo floats past the stage base, which puts the
    // patch's first column (xsh floats into its chunk) on a 16-byte boundary.
    const int xsh = VEC ? (4 - g.pad % 4) % 4 : 0, xlo = (4 - xsh) % 4;
    const int row0 = ti0 * MT - g.pad, col0 = tj0 * MT - g.pad - xsh;
    uint32_t xoff[S::NJ];
    if constexpr (S::PRIV) {
        // load e = j*64 + lane of the wave's [4 channels of its quad][A rows][NE]
#pragma unroll
        for (int j = 0; j < S::JXW; ++j) {
            const int e = j * 64 + lane;
            const int ch = e / (S::A * S::NE), rem = e - ch * (S::A * S::NE);
            const int r = rem / S::NE, c = (rem - r * S::NE) * S::EW;
            const int row = row0 + r, col = col0 + c;
            const bool ok = (e * S::EW < S::XW) & ((unsigned)row < (unsigned)g.H) & ((unsigned)col < (unsigned)g.W);
            const uint32_t off =
                (uint32_t)((kw * CS + cs) * 4 + ch) * plane_b + ((uint32_t)row * (uint32_t)g.W + (uint32_t)col) * 4u;
            xoff[j] = ok ? off : kInvalid;
        }
    } else {
#pragma unroll
        for (int j = 0; j < S::JX; ++j) {
            const int e = j * 512 + tid;
            const int ch = e / (S::PR * S::NE), rem = e - ch * (S::PR * S::NE);
            const int r = rem / S::NE, c = (rem - r * S::NE) * S::EW;
            const int row = row0 + r, col = col0 + c;
            const bool ok = (e * S::EW < S::XS) & (VEC || c < S::PC) & ((unsigned)row < (unsigned)g.H) &
                            ((unsigned)col < (unsigned)g.W);
            const uint32_t off = (uint32_t)ch * plane_b + ((uint32_t)row * (uint32_t)g.W + (uint32_t)col) * 4u;
            xoff[j] = ok ? off : kInvalid;
        }
    }
    const uint32_t step_b = 4u * S::QS * plane_b;

    f32x4 acc[S::TH];
#pragma unroll
    for (int t = 0; t < S::TH; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float* xs0f = (float*)xs0;
    float* xs1f = (float*)xs1;
    float* xs2f = (float*)xs2;
    float* vsf = (float*)vs;
    if constexpr (TS == 1) {
        fused_steps<MT, TS, CS, BW, VEC, 0, RF>(xr, xoff, step_b, U, g, ft, kb, wave, lane, kw, cs, bi, bj, xs0f, xs1f,
                                       xs2f, vsf, acc, xlo, cq0, cqn, nsteps);
    } else if (h == 0) {
        fused_steps<MT, TS, CS, BW, VEC, 0, RF>(xr, xoff, step_b, U, g, ft, kb, wave, lane, kw, cs, bi, bj, xs0f, xs1f,
                                       xs2f, vsf, acc, xlo, cq0, cqn, nsteps);
    } else {
        fused_steps<MT, TS, CS, BW, VEC, 1, RF>(xr, xoff, step_b, U, g, ft, kb, wave, lane, kw, cs, bi, bj, xs0f, xs1f,
                                       xs2f, vsf, acc, xlo, cq0, cqn, nsteps);
    }

    // ---- epilogue.  Every load has landed (fused_steps ends with a full
    // wait), so after a barrier the whole LDS allocation is free.  The four
    // objects are packed into one range; the epilogue addresses that range as
    // raw LDS, starting at the lowest object.
    constexpr int TH = S::TH, RN = S::RN, NF = S::NF, PH = S::PH, V1 = S::V1, VW1 = S::VW1;
    constexpr int G2 = S::G2, NR2 = S::NR2;
    typedef __attribute__((address_space(3))) float lds_f;
    auto lds_off = [](const float* p) { return (uint32_t)(uintptr_t)(const lds_f*)p; };
    const uint32_t ex_base =
        min(min(lds_off(xs0f), lds_off(xs1f)), min(lds_off(xs2f), lds_off(vsf)));
    lds_f* const ex = (lds_f*)(uintptr_t)ex_base;
    const int fset = cs / PH, ph = cs % PH;      // filter set and row half this wave ends up with
    float msum[CS > 1 ? V1 : 1];
#define WINO_ACC(f) acc[(f) % TH][(f) / TH]
    if constexpr (CS > 1) {
        // Channel sum: run dst of part src goes to block (dst, src) of this
        // (filter block, row group) -- src != dst only, with OWN1 -- and wave
        // dst adds the CS runs in part order (its own from its registers).
        constexpr int NB1 = S::NB1;
        lds_f* const e1 = ex + (kw * TS + h) * (CS * NB1 * V1 * 64) + lane * VW1;
        auto blk1 = [&](int dst, int src) {
            return e1 + (dst * NB1 + (S::OWN1 && src > dst ? src - 1 : src)) * (V1 * 64);
        };
        __syncthreads();
#pragma unroll
        for (int dst = 0; dst < CS; ++dst) {
            if (S::OWN1 && dst == cs) continue;
            lds_f* blk = blk1(dst, cs);
#pragma unroll
            for (int q = 0; q < V1 / VW1; ++q) {
                const int f0 = dst * V1 + q * VW1;
                if constexpr (VW1 == 4) {
                    *(__attribute__((address_space(3))) f32x4*)(blk + q * 64 * 4) =
                        f32x4{WINO_ACC(f0), WINO_ACC(f0 + 1), WINO_ACC(f0 + 2), WINO_ACC(f0 + 3)};
                } else {
                    typedef float f32x2 __attribute__((ext_vector_type(2)));
                    *(__attribute__((address_space(3))) f32x2*)(blk + q * 64 * 2) =
                        f32x2{WINO_ACC(f0), WINO_ACC(f0 + 1)};
                }
            }
        }
        __syncthreads();
        auto sum1 = [&](auto csc) {
            constexpr int OWN = decltype(csc)::value;         // -1: own run from LDS too
            const int me = OWN >= 0 ? OWN : cs;
#pragma unroll
            for (int src = 0; src < CS; ++src) {
                const lds_f* blk = src == OWN ? e1 : blk1(me, src);
#pragma unroll
                for (int q = 0; q < V1 / VW1; ++q) {
                    float w[VW1];
                    if (src == OWN) {
#pragma unroll
                        for (int i = 0; i < VW1; ++i) w[i] = WINO_ACC((OWN >= 0 ? OWN : 0) * V1 + q * VW1 + i);
                    } else if constexpr (VW1 == 4) {
                        const f32x4 a4 = *(const __attribute__((address_space(3))) f32x4*)(blk + q * 64 * 4);
                        w[0] = a4[0]; w[1] = a4[1]; w[2] = a4[2]; w[3] = a4[3];
                    } else {
                        typedef float f32x2 __attribute__((ext_vector_type(2)));
                        const f32x2 a2 = *(const __attribute__((address_space(3))) f32x2*)(blk + q * 64 * 2);
                        w[0] = a2[0]; w[1] = a2[1];
                    }
#pragma unroll
                    for (int i = 0; i < VW1; ++i) msum[q * VW1 + i] = src == 0 ? w[i] : msum[q * VW1 + i] + w[i];
                }
            }
        };
        if constexpr (S::OWN1) with_ic(cs, sum1, std::make_integer_sequence<int, CS>{});
        else sum1(IC<-1>{});
    }

    // This wave's part of A^T M A for its NF filters: the rows of its row group
    // (and, for PH = 2, one half of them).
    float o[NF][MT][MT];
    auto part_tf = [&](auto hc) {
        constexpr int X0 = decltype(hc)::value * RN;
        constexpr int RH = RN / PH, TQ = RH * S::A;
#pragma unroll
        for (int j = 0; j < NF; ++j) {
            float m1[TQ];
#pragma unroll
            for (int t = 0; t < TQ; ++t) {
                if constexpr (CS == 1) m1[t] = acc[t][j];      // TQ = TH: the accumulators themselves
                else m1[t] = msum[j * TQ + t];
            }
            if constexpr (PH == 1) {
                output_tf_rows<MT, X0, RN, RF>(m1, o[j]);
            } else if (ph == 0) {
                output_tf_rows<MT, X0, RH, RF>(m1, o[j]);
            } else {
                output_tf_rows<MT, X0 + RH, RH, RF>(m1, o[j]);
            }
        }
    };
    if constexpr (TS == 1) part_tf(IC<0>{});
    else if (h == 0) part_tf(IC<0>{});
    else part_tf(IC<1>{});
#undef WINO_ACC

    // Output sum over the G2 waves of a filter set: wave q keeps rows
    // [q*NR2, (q+1)*NR2) of the set's NR rows (row rho = filter rho / MT,
    // output row rho % MT) and adds the G2 partials in order.
    const int q = h * PH + ph;
    float fin[NR2][MT];
#define WINO_O(rho, jj) o[(rho) / MT][(rho) % MT][jj]
    if constexpr (G2 == 1) {
#pragma unroll
        for (int rr = 0; rr < NR2; ++rr)
#pragma unroll
            for (int jj = 0; jj < MT; ++jj) fin[rr][jj] = WINO_O(rr, jj);
    } else {
        // after the channel sum's blocks (a disjoint range: no barrier between)
        lds_f* const e2 = ex + S::EX1 + (kw * S::NFG + fset) * (G2 * (G2 - 1) * NR2 * MT * 64) + lane * MT;
        auto blk2 = [&](int dst, int src) {
            return e2 + (dst * (G2 - 1) + (src < dst ? src : src - 1)) * (NR2 * MT * 64);
        };
        if constexpr (CS == 1) __syncthreads();  // the loop's LDS is free (CS > 1 synchronised above)
#pragma unroll
        for (int dst = 0; dst < G2; ++dst) {
            if (dst == q) continue;
            lds_f* blk = blk2(dst, q);
#pragma unroll
            for (int rr = 0; rr < NR2; ++rr) {
                const int rho = dst * NR2 + rr;
                if constexpr (MT == 4) {
                    *(__attribute__((address_space(3))) f32x4*)(blk + rr * 64 * 4) =
                        f32x4{WINO_O(rho, 0), WINO_O(rho, 1), WINO_O(rho, 2), WINO_O(rho, 3)};
                } else {
                    typedef float f32x2 __attribute__((ext_vector_type(2)));
                    *(__attribute__((address_space(3))) f32x2*)(blk + rr * 64 * 2) =
                        f32x2{WINO_O(rho, 0), WINO_O(rho, 1)};
                }
            }
        }
        __syncthreads();
        with_ic(q, [&](auto qc) {
            constexpr int OWN = decltype(qc)::value;
#pragma unroll
            for (int src = 0; src < G2; ++src) {
                const lds_f* blk = src == OWN ? e2 : blk2(OWN, src);
#pragma unroll
                for (int rr = 0; rr < NR2; ++rr) {
                    float w[MT];
                    if (src == OWN) {
#pragma unroll
                        for (int jj = 0; jj < MT; ++jj) w[jj] = WINO_O(OWN * NR2 + rr, jj);
                    } else if constexpr (MT == 4) {
                        const f32x4 a4 = *(const __attribute__((address_space(3))) f32x4*)(blk + rr * 64 * 4);
                        w[0] = a4[0]; w[1] = a4[1]; w[2] = a4[2]; w[3] = a4[3];
                    } else {
                        typedef float f32x2 __attribute__((ext_vector_type(2)));
                        const f32x2 a2 = *(const __attribute__((address_space(3))) f32x2*)(blk + rr * 64 * 2);
                        w[0] = a2[0]; w[1] = a2[1];
                    }
#pragma unroll
                    for (int jj = 0; jj < MT; ++jj) fin[rr][jj] = src == 0 ? w[jj] : fin[rr][jj] + w[jj];
                }
            }
        }, std::make_integer_sequence<int, G2>{});
    }
#undef WINO_O
    const int kset = (kgi * KGW + kw) * 16 + 4 * cl + fset * NF;   // first filter of this wave's set
    // A slice's partial output goes to its own plane of part, without ReLU.
    float* const yo = ft.nsl > 1 ? ypart + (size_t)sl * (size_t)ft.ysz : y;
    const bool rl = relu != 0 && ft.nsl == 1, vo = vec_ok != 0;
#pragma unroll
    for (int rr = 0; rr < NR2; ++rr) {
        const int rho = q * NR2 + rr;
        if (nts) store_row<MT, true>(yo, g, tc, kset + rho / MT, rho % MT, fin[rr], rl, vo);
        else store_row<MT, false>(yo, g, tc, kset + rho / MT, rho % MT, fin[rr], rl, vo);
    }
}

// ------------------------------------------------------------------ split
// The split path, for layers with many tiles: k_vblk writes the input
// transform to a tile-blocked workspace, then k_gemm_out runs the T GEMMs with
// the output transform in their epilogue.  The transform's adds then run once
// per (tile, channel) instead of once per filter group, and the GEMM loop is
// MFMAs and LDS reads only -- on gfx950 vector ALU work does not overlap the
// MFMAs of its SIMD, so it costs its full time inside a GEMM loop.
//
// Blocked V: Vb[tb][CQ4][T/4][64][4], tb = p / 16 a block of 16 consecutive
// tiles (in the order n, ti, tj, so only the batch's last block has slots past
// the last tile), CQ4 = CQ rounded up to a multiple of 4 (the padding quads
// hold zeros); element (t, c, tile p) at lane (c%4)*16 + p%16, slot t%4 of
// group t/4.  The input transform still works on rectangular patches of
// 16 tiles (BH x BW, sharing the halo in LDS); each lane stores its tile to
// that tile's block and slot, and a patch's columns or rows past the tile grid
// store nothing.

// Patch byte offsets of one image for load e = j*NT + tid of
// [4*NQ channels][PR rows][NE loads] (kInvalid outside the image or past the
// row); VEC loads are 16-byte chunks from a 4-aligned column xsh floats before
// the patch.
template <int MT, int NT, int NQ, int PR, int PC, int PCP, int VEC, int JX>
__device__ __forceinline__ void patch_offsets(uint32_t (&xoff)[JX], const Geom& g, int tid, int ti0, int tj0,
                                              int xsh) {
    constexpr int EW = VEC ? 4 : 1, NE = PCP / EW, XS = 4 * NQ * PR * PCP;
    const uint32_t plane_b = (uint32_t)g.H * g.W * 4;
    const int row0 = ti0 * MT - g.pad, col0 = tj0 * MT - g.pad - xsh;
#pragma unroll
    for (int j = 0; j < JX; ++j) {
        const int e = j * NT + tid;
        const int ch = e / (PR * NE), rem = e - ch * (PR * NE);
        const int r = rem / NE, c = (rem - r * NE) * EW;
        const int row = row0 + r, col = col0 + c;
        const bool ok = (e * EW < XS) & (VEC || c < PC) & ((unsigned)row < (unsigned)g.H) &
                        ((unsigned)col < (unsigned)g.W);
        const uint32_t off = (uint32_t)ch * plane_b + ((uint32_t)row * (uint32_t)g.W + (uint32_t)col) * 4u;
        xoff[j] = ok ? off : kInvalid;
    }
}

// One direct-to-LDS buffer load of BYTES per lane (a device function: the
// host pass rejects the 16-byte form written directly in a kernel body).
template <int BYTES>
__device__ __forceinline__ void lds_dma(__amdgpu_buffer_rsrc_t r, float* lds, uint32_t off, uint32_t soff = 0) {
    static_assert(BYTES == 4 || BYTES == 16, "dword or 16-byte loads");
    if constexpr (BYTES == 16) __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, off, soff, 0, 0);
    else __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 4, off, soff, 0, 0);
}

// ------------------------------------------------------------------ GEMM
// M_t[k][p] = sum_c U_t[c][k] V_t[c][p] for each transform position t.
// Workgroup: 4 positions (one t/4 group) x KT k-blocks x 4 p-blocks (64 x 64
// for KT = 4, 32 x 64 for KT = 2), four waves, each KT/2 x 2 blocks of 16 x 16
// for all 4 positions.  Channels advance 8 at a time (2 quads): a chunk is
// 2*KT U blocks and 8 V blocks of 1 KB (64 lanes x one 16-byte word of 4
// positions), copied straight into LDS by DMA into a ring of three stages,
// two chunks ahead of the products, so a chunk's load latency is hidden even
// when only one or two workgroups share a CU (the 1-D layers' T = 8 GEMMs).
// Each MFMA operand quadruple is then one ds_read_b128.  Blocks past K or P
// lie past the item's buffer ranges and quads past C get an out-of-range
// offset: both read as zero.  KT = 2 spreads layers that would give the CUs
// fewer than four 64 x 64 items each over more workgroups and pads K to 32.
template <int KT>
__global__ __launch_bounds__(256) void k_gemm(const float* __restrict__ U, const float* __restrict__ V,
                                              float* __restrict__ M, Geom g) {
    static_assert(KT == 2 || KT == 4, "k-blocks per tile");
    constexpr int KW = KT / 2, NS = 2 * KT + 8, NPW = NS / 4;   // k-blocks per wave, slots, DMA loads per wave
    // 12 or 16 KB a stage, at most 48 KB in all: three workgroups share a CU's 160 KB.
    __shared__ float4 st0[NS * 64], st1[NS * 64], st2[NS * 64];   // [A: quad, k-block | B: quad, p-block][lane]
    const int T = g.T, TG = g.T / 4;
    const int KB4 = (g.KB + KT - 1) / KT, PB4 = (g.PB + 3) >> 2;
    // Items (position group, p-tile, k-tile), k-tile fastest; each XCD runs one
    // contiguous range of items (workgroup b takes item (b % 8) * per + b / 8),
    // so the k-tiles that share a p-tile's V run together and V comes from HBM
    // into that XCD's L2 once.
    const long nitems = (long)TG * PB4 * KB4, per = (nitems + 7) / 8;
    const long item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nitems) return;
    const int kb0 = (int)(item % KB4) * KT;
    const long rest = item / KB4;
    const int pb0 = (int)(rest % PB4) * 4;
    const int tg = (int)(rest / PB4);     // positions 4*tg .. 4*tg+3
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wk = wave >> 1, wp = wave & 1;
    const int NC = (g.CQ + 1) >> 1;      // chunks of two quads

    // This item's U and V blocks as buffers: block j of the tile at
    // j * CQ * TG KB; a block past K or P lies past the range.
    const uint32_t bstride = (uint32_t)g.CQ * (uint32_t)TG * 1024u;
    const size_t ub = (size_t)min(g.KB - kb0, KT) * bstride, vb = (size_t)min(g.PB - pb0, 4) * bstride;
    const __amdgpu_buffer_rsrc_t ur = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(U + (size_t)kb0 * g.CQ * TG * 256), (short)0, (int)ub, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(V + (size_t)pb0 * g.CQ * TG * 256), (short)0, (int)vb, kRsrcWord3);
    auto stage = [&](auto sc) -> float4* {
        constexpr int S = decltype(sc)::value;
        if constexpr (S == 0) return st0;
        else if constexpr (S == 1) return st1;
        else return st2;
    };
    // DMA of chunk c into stage sc: wave w moves slots NPW*w .. NPW*w+NPW-1
    // of the NS (slot q < 2*KT: U block q % KT of quad q / KT; q >= 2*KT: V
    // block (q-2*KT) % 4 of quad (q-2*KT) / 4), NPW loads per wave per chunk.
    const uint32_t l16 = (uint32_t)lane * 16u;
    auto issue = [&](auto sc, int c) {
        float4* s = stage(sc);
#pragma unroll
        for (int i = 0; i < NPW; ++i) {
            const int q = wave * NPW + i;
            const bool a = q < 2 * KT;
            const int qq = a ? q : q - 2 * KT, w = a ? KT : 4, blk = qq % w;
            const int cq = 2 * c + qq / w;
            const uint32_t soff = cq < g.CQ ? (uint32_t)blk * bstride + ((uint32_t)cq * TG + tg) * 1024u
                                            : (a ? (uint32_t)ub : (uint32_t)vb);
            lds_dma<16>(a ? ur : vr, (float*)(s + q * 64), l16, __builtin_amdgcn_readfirstlane(soff));
        }
    };

    f32x4 acc[4][KW][2];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int i = 0; i < KW; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[q][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    issue(IC<0>{}, 0);
    if (NC > 1) issue(IC<1>{}, 1);
    // Chunk ch (stage ch % 3): at its start the NPW DMA loads of chunk ch+1
    // may still be in flight, not those of chunk ch; the barrier then tells
    // every wave that chunk ch is in LDS and chunk ch-1's stage is free for
    // chunk ch+2.
    auto chunk = [&](auto sc, int ch) {
        constexpr int S = decltype(sc)::value;
        if (ch + 1 < NC) wait_vm_lds<NPW>();
        else wait_vm_lds<0>();
        wg_barrier();
        if (ch + 2 < NC) issue(IC<(S + 2) % 3>{}, ch + 2);
        const float4* s = stage(sc);
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            float av[KW][4], bv[2][4];
#pragma unroll
            for (int i = 0; i < KW; ++i) {
                const float4 a = s[(q * KT + wk * KW + i) * 64 + lane];
                av[i][0] = a.x; av[i][1] = a.y; av[i][2] = a.z; av[i][3] = a.w;
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const float4 b = s[(2 * KT + q * 4 + wp * 2 + j) * 64 + lane];
                bv[j][0] = b.x; bv[j][1] = b.y; bv[j][2] = b.z; bv[j][3] = b.w;
            }
#pragma unroll
            for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
                for (int i = 0; i < KW; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) acc[t4][i][j] = mfma16x16x4(av[i][t4], bv[j][t4], acc[t4][i][j]);
        }
    };
    int ch = 0;
    for (; ch + 3 <= NC; ch += 3) {
        chunk(IC<0>{}, ch);
        chunk(IC<1>{}, ch + 1);
        chunk(IC<2>{}, ch + 2);
    }
    if (ch < NC) chunk(IC<0>{}, ch);
    if (ch + 1 < NC) chunk(IC<1>{}, ch + 1);
#pragma unroll
    for (int t4 = 0; t4 < 4; ++t4)
#pragma unroll
        for (int i = 0; i < KW; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int kb = kb0 + wk * KW + i, pb = pb0 + wp * 2 + j;
                if (kb < g.KB && pb < g.PB)
                    *(f32x4*)(M + (((size_t)pb * g.KB + kb) * T + 4 * tg + t4) * 256 + lane * 4) = acc[t4][i][j];
            }
}

template <int MT, int BW, int VEC>
struct VblkShape {
    static constexpr int A = MT + 2, T = A * A, BH = 16 / BW;
    static constexpr int NQ = 4;                          // channel quads per workgroup, one per wave
    static constexpr int PR = BH * MT + 2, PC = BW * MT + 2;
    static constexpr int EW = VEC ? 4 : 1;
    static constexpr int PCP = VEC ? (PC + 6) / 4 * 4 : (PC + 3) / 4 * 4;
    static constexpr int XS = 4 * NQ * PR * PCP;
    static constexpr int JX = (XS / EW + 255) / 256;
    static constexpr int XSP = JX * 256 * EW;
};

// One workgroup per (16-tile patch, 4 channel quads): the halo'd patch comes
// into LDS by DMA, each wave transforms one quad for the patch's 16 tiles and
// stores its 9 (m = 4) or 4 (m = 2) groups of 16 bytes per lane into the
// blocks of those tiles.  The workgroup of the batch's last patch also writes
// zeros to the last block's slots past the last tile.
template <int MT, int BW, int VEC>
__global__ __launch_bounds__(256) void k_vblk(const float* __restrict__ x, float* __restrict__ Vb, Geom g,
                                              int nbh, int nbw, int ncq4) {
    using S = VblkShape<MT, BW, VEC>;
    constexpr int A = S::A, T = S::T;
    __shared__ float4 xs[S::XSP / 4 + VEC];
    const int b = blockIdx.x;
    const int tb = b / ncq4, q4 = b - tb * ncq4;
    const int per_img = nbh * nbw;
    const int n = tb / per_img, r2 = tb - n * per_img;
    const int ti0 = (r2 / nbw) * S::BH, tj0 = (r2 % nbw) * BW;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, bi = l16 / BW, bj = l16 % BW, cl = lane >> 4;

    const size_t img = (size_t)g.C * g.H * g.W;
    const size_t img_b = img * 4;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + (size_t)n * img), (short)0, (int)(img_b < kInvalid ? img_b : kInvalid), kRsrcWord3);
    const int xsh = VEC ? (4 - g.pad % 4) % 4 : 0, xlo = (4 - xsh) % 4;
    uint32_t xoff[S::JX];
    patch_offsets<MT, 256, S::NQ, S::PR, S::PC, S::PCP, VEC, S::JX>(xoff, g, tid, ti0, tj0, xsh);
    const uint32_t cbase = (uint32_t)q4 * 16u * ((uint32_t)g.H * g.W * 4);
    float* xf = (float*)xs;
#pragma unroll
    for (int i = 0; i < S::JX; ++i) lds_dma<4 * S::EW>(xr, xf + xlo + (i * 256 + wave * 64) * S::EW, xoff[i] + cbase);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const int cq = q4 * 4 + wave;        // < CQ4; quads past CQ read zero patches and store zeros
    const float* wp = xf + ((wave * 4 + cl) * S::PR + bi * MT) * S::PCP + bj * MT + (xlo ? 4 : 0);
    float d[A][A];
#pragma unroll
    for (int u = 0; u < A; ++u) {
        const float* row = wp + u * S::PCP;
        if constexpr (MT == 4) {
            const float4 a4 = *(const float4*)row;
            const float2 b2 = *(const float2*)(row + 4);
            d[u][0] = a4.x; d[u][1] = a4.y; d[u][2] = a4.z; d[u][3] = a4.w; d[u][4] = b2.x; d[u][5] = b2.y;
        } else {
            const float2 a2 = *(const float2*)row;
            const float2 b2 = *(const float2*)(row + 2);
            d[u][0] = a2.x; d[u][1] = a2.y; d[u][2] = b2.x; d[u][3] = b2.y;
        }
    }
    float v[T];
    input_tf<MT>(d, v);
    // this lane's tile, and its block and slot in Vb
    const int ti = ti0 + bi, tj = tj0 + bj;
    const size_t qstride = (size_t)ncq4 * 4 * T * 64;              // floats of one block
    const int hi = lane & 0x30;                                     // (c % 4) * 16
    if (ti < g.th && tj < g.tw) {
        const int p = (n * g.th + ti) * g.tw + tj;
        float* dst = Vb + (size_t)(p >> 4) * qstride + (size_t)cq * T * 64 + (hi | (p & 15)) * 4;
#pragma unroll
        for (int g4 = 0; g4 < T / 4; ++g4)
            store_out<false>(dst + g4 * 256, v[4 * g4], v[4 * g4 + 1], v[4 * g4 + 2], v[4 * g4 + 3]);
    }
    const int tail = g.P & 15;
    if (tail && tb == g.N * nbh * nbw - 1 && l16 >= tail) {
        float* dst = Vb + (size_t)(g.P >> 4) * qstride + (size_t)cq * T * 64 + (hi | l16) * 4;
#pragma unroll
        for (int g4 = 0; g4 < T / 4; ++g4) store_out<false>(dst + g4 * 256, 0.f, 0.f, 0.f, 0.f);
    }
}

// fp16 (PREC 1) or bf16 (PREC 2) bits of v, to nearest with ties to even.
template <int PREC>
__device__ __forceinline__ uint32_t to16(float v) {
    if constexpr (PREC == 1) {
        return (uint32_t)__builtin_bit_cast(unsigned short, (_Float16)v);
    } else {
        const uint32_t u = __builtin_bit_cast(uint32_t, v);
        if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;        // NaN stays NaN
        return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;               // nearest, ties to even
    }
}

// Input transform by whole tile rows (the split path's Vb with nq = CQ
// rounded up to a multiple of 4, the staged path's V with nq = CQ): one
// workgroup per (R consecutive tile rows of the batch, channel quad).  The rows' halo'd
// patches (A image rows each, all columns) come into LDS by DMA; wave w then
// transforms tile blocks w, w+4, ... of the rows' tiles, lane = (channel,
// tile), and stores each block's 9 (m = 4) or 4 (m = 2) groups as whole 1 KiB
// runs.  The host picks R so that R*tw is a multiple of 16 where LDS allows:
// every block is then written by one workgroup (a block the row range only
// partly covers is completed by the neighbouring workgroup).  Loads are
// 16-byte column chunks starting xsh columns before the patch (the host takes
// this kernel only for widths that are a multiple of 4 and a 16-byte aligned
// x, so every chunk lies wholly inside or outside a row).
// LDS: [row r][channel][A rows][pitch] floats, shifted so that a tile's first
// column sits at a multiple of 4.  OUT = 1 / 2: the 16-bit paths' VH (fp16 /
// bf16, 16-channel groups, a lane's word holding four channels): the lane
// stores its channel's 16 bits, and a wave's store covers its quad's 128
// contiguous bytes of a group's position block; nq = 4 * C16.
template <int MT, int OUT = 0>
__global__ __launch_bounds__(256) void k_vrows(const float* __restrict__ x, float* __restrict__ Vb, Geom g,
                                               int R, int pitch, int nq) {
    constexpr int A = MT + 2, T = A * A, EW = 4;
    extern __shared__ float4 xs4[];
    float* xs = (float*)xs4;
    const int nrows = g.N * g.th;                        // tile rows of the batch
    const int ngr = (nrows + R - 1) / R;
    const int b = blockIdx.x;
    const int cq = b / ngr, gr0 = (b - cq * ngr) * R;    // quad, first tile row
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n0 = gr0 / g.th;
    const size_t img = (size_t)g.C * g.H * g.W;
    const size_t left = ((size_t)g.N - n0) * img * 4;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + (size_t)n0 * img), (short)0, (int)(left < kInvalid ? left : kInvalid), kRsrcWord3);
    const int xsh = (4 - g.pad % 4) % 4, xlo = (4 - xsh) % 4;
    const int cs = -g.pad - xsh;                         // image column of a patch row's first unit
    const int ne = pitch / EW;                           // units per patch row
    const int units = R * 4 * A * ne;
    const uint32_t plane_b = (uint32_t)g.H * g.W * 4;
    for (int e = tid; e < units; e += 256) {             // e = ((r*4 + c)*A + u)*ne + k
        const int k = e % ne, q1 = e / ne;
        const int u = q1 % A, q2 = q1 / A;
        const int c = q2 & 3, r = q2 >> 2;
        const int gr = gr0 + r, n = gr / g.th, ti = gr - n * g.th;
        const int row = ti * MT - g.pad + u, col = cs + k * EW, ch = cq * 4 + c;
        const bool ok = gr < nrows && ch < g.C && (unsigned)row < (unsigned)g.H && col >= 0 &&
                        col + EW <= g.W;
        const uint32_t off = ok ? (uint32_t)(n - n0) * (uint32_t)(img * 4) + (uint32_t)ch * plane_b +
                                      ((uint32_t)row * (uint32_t)g.W + (uint32_t)col) * 4u
                                : kInvalid;
        // the wave's 64 units are consecutive in LDS (lane order)
        lds_dma<4 * EW>(xr, xs + xlo + (e - lane) * EW, off);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    const int l16 = lane & 15, cl = lane >> 4;
    const int t0 = gr0 * g.tw, t1 = min(gr0 + R, nrows) * g.tw;   // this workgroup's tiles [t0, t1)
    const size_t qstride = (size_t)nq * T * 64;                   // floats of one block
    const int last_tail = (t1 == g.P && (g.P & 15)) ? 1 : 0;      // the batch's last block is partial
    // 16-bit VH: the half of (channel cq*4 + cl, tile l16) in block blk,
    // position t at [t * 256] (halves: [blk][C16][T][64 lanes][4])
    auto vh_dst = [&](int blk) {
        const int c16 = cq >> 2, q = cq & 3;
        return (unsigned short*)Vb + (((size_t)blk * (nq >> 2) + c16) * T * 64 + q * 16 + l16) * 4 + cl;
    };
    for (int blk = t0 / 16 + wave; blk <= (t1 - 1) / 16; blk += 4) {
        const int p = blk * 16 + l16;
        float* dst = Vb + (size_t)blk * qstride + (size_t)cq * T * 64 + lane * 4;
        if (p >= t0 && p < t1) {
            const int r = p / g.tw - gr0, tj = p % g.tw;
            const float* wp = xs + ((r * 4 + cl) * A) * pitch + tj * MT + (xlo ? 4 : 0);
            float d[A][A];
#pragma unroll
            for (int u = 0; u < A; ++u) {
                const float* rowp = wp + u * pitch;
                if constexpr (MT == 4) {
                    const float4 a4 = *(const float4*)rowp;
                    const float2 b2 = *(const float2*)(rowp + 4);
                    d[u][0] = a4.x; d[u][1] = a4.y; d[u][2] = a4.z; d[u][3] = a4.w; d[u][4] = b2.x; d[u][5] = b2.y;
                } else {
                    const float2 a2 = *(const float2*)rowp;
                    const float2 b2 = *(const float2*)(rowp + 2);
                    d[u][0] = a2.x; d[u][1] = a2.y; d[u][2] = b2.x; d[u][3] = b2.y;
                }
            }
            float v[T];
            input_tf<MT>(d, v);
            if constexpr (OUT == 0) {
#pragma unroll
                for (int g4 = 0; g4 < T / 4; ++g4)
                    store_out<false>(dst + g4 * 256, v[4 * g4], v[4 * g4 + 1], v[4 * g4 + 2], v[4 * g4 + 3]);
            } else {
                unsigned short* h = vh_dst(blk);
#pragma unroll
                for (int t = 0; t < T; ++t) h[t * 256] = (unsigned short)to16<OUT>(v[t]);
            }
        } else if (last_tail && p >= g.P) {
            if constexpr (OUT == 0) {
#pragma unroll
                for (int g4 = 0; g4 < T / 4; ++g4) store_out<false>(dst + g4 * 256, 0.f, 0.f, 0.f, 0.f);
            } else {
                unsigned short* h = vh_dst(blk);
#pragma unroll
                for (int t = 0; t < T; ++t) h[t * 256] = 0;
            }
        }
    }
}

// GEMMs + output transform from Vb.  A workgroup of 8 waves computes two tile
// blocks for KGW = 8/TS filter blocks over all channels; wave (kw, h) owns
// filter block kw and transform rows [h*A/TS, (h+1)*A/TS) of both tile blocks
// (each filter operand it loads feeds two MFMAs).  Per step of NQ = 4 channel
// quads the two blocks' V (one contiguous run each) come into LDS by DMA one
// step ahead, in two stages; filters come one quad ahead into registers.  At
// the end each wave applies its share of A^T M A and, for TS = 2, the two row
// halves of a filter block are summed through LDS in a fixed order.
template <int MT>
struct GoShape {
    static constexpr int A = MT + 2, T = A * A, TG = T / 4;
    static constexpr int TS = MT == 4 ? 2 : 1, KGW = 8 / TS, RN = A / TS, TH = RN * A;
    static constexpr int TBW = 2, NQ = 4;                 // tile blocks, channel quads per step
    static constexpr int VST = TBW * NQ * T * 64;         // floats of one V stage
    static constexpr int JV = VST / 4 / 512;              // 16-byte DMA loads per thread per step
    static constexpr int NV = 4 * MT * MT;                // output values per lane per tile block
    static_assert(JV * 512 * 4 == VST, "whole DMA rounds");
};

template <int MT, int H>
__device__ __forceinline__ void go_steps(const __amdgpu_buffer_rsrc_t vr, uint32_t vbase0, uint32_t vbase1,
                                         const float* __restrict__ U, const Geom& g, int nsteps, int kb,
                                         int wave, int lane, float* vs0, float* vs1,
                                         f32x4 (&acc)[2][GoShape<MT>::TH]) {
    using S = GoShape<MT>;
    constexpr int A = S::A, RN = S::RN, X0 = H * RN, TH = S::TH, T = S::T, NQ = S::NQ;
    constexpr int G0 = X0 * A / 4, NG = (X0 * A + TH - 1) / 4 - G0 + 1;
    // V stage layout [block b][quad q][T/4][64][4]: the DMA of a step copies run
    // b (NQ quads of block b, contiguous in Vb) to [b]; load e = i*512 + tid.
    auto stage = [&](auto rc) -> float* {
        if constexpr (decltype(rc)::value == 0) return vs0;
        else return vs1;
    };
    // DMA loads i0 .. i1-1 (of JV) of step j's V into stage rc.  Unit e =
    // i*512 + tid of the stage is unit e of block 0's run or unit e - JV*256 of
    // block 1's; the padding quads of Vb are zeros, so no unit needs a mask.
    // The lane part of a unit's offset is tid16 (one register); the rest is
    // wave-uniform and goes into the scalar offset.  Only the load that
    // straddles the two runs needs a per-lane correction.
    const uint32_t tid16 = ((uint32_t)wave * 64 + lane) * 16u;
    auto issue_v = [&](auto rc, int j, auto i0c, auto i1c) {
        float* vs = stage(rc);
        const uint32_t qoff = (uint32_t)j * NQ * T * 256;       // bytes: NQ quads of T*64 floats
        static_for<decltype(i0c)::value, decltype(i1c)::value>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr uint32_t RUN = S::JV * 256 * 16;           // bytes of one block's run
            constexpr uint32_t E0 = (uint32_t)i * 8192u;         // the unit's stage offset is E0 + tid16
            float* dst = vs + (i * 512 + wave * 64) * 4;
            if constexpr (E0 + 8192u <= RUN) {
                lds_dma<16>(vr, dst, tid16, vbase0 + E0 + qoff);
            } else if constexpr (E0 >= RUN) {
                lds_dma<16>(vr, dst, tid16, vbase1 + (E0 - RUN) + qoff);
            } else {
                const uint32_t voff = tid16 < RUN - E0 ? tid16 : tid16 + (vbase1 - vbase0 - RUN);
                lds_dma<16>(vr, dst, voff, vbase0 + E0 + qoff);
            }
        });
    };
    const __amdgpu_buffer_rsrc_t ur = u_rsrc(U, g);
    const uint32_t ulane = (uint32_t)lane * 16u;
    auto load_u = [&](int cq, f32x4 (&ug)[NG]) {
        const int c = min(cq, g.CQ - 1);
        const uint32_t go = __builtin_amdgcn_readfirstlane((uint32_t)(((kb * g.CQ + c) * (T / 4) + G0) * 1024));
#pragma unroll
        for (int i = 0; i < NG; ++i) ug[i] = u_load(ur, ulane, go + i * 1024u);
    };
    // quad q of the stage: 2 blocks x TH MFMAs, V read group by group; after
    // group gi, between(gi) (the reload of that group's filter registers)
    auto quad = [&](const float* vs, int q, const f32x4 (&ug)[NG], auto&& between) {
#pragma unroll
        for (int gi = 0; gi < NG; ++gi) {
            f32x4 vv[2];
#pragma unroll
            for (int b = 0; b < 2; ++b) vv[b] = *(const f32x4*)(vs + (((b * NQ + q) * (T / 4) + G0 + gi) * 64 + lane) * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int t = (G0 + gi) * 4 + e - X0 * A;       // position within this wave's rows
                if (t >= 0 && t < TH) {
#pragma unroll
                    for (int b = 0; b < 2; ++b) acc[b][t] = mfma16x16x4(ug[gi][e], vv[b][e], acc[b][t]);
                }
            }
            between(gi);
        }
    };
    f32x4 ubuf[2][NG];                           // filter register sets of even and odd quads
    constexpr int JV = S::JV, JP = (JV + 2) / 3;
    // Filters come two quads ahead: after the MFMAs of position group gi of
    // quad q, group gi of quad q+2 is loaded into the registers they used (one
    // quad ahead, the loads that miss L2 -- the whole U does not fit one XCD's
    // L2 -- stalled the MFMAs: 680 against 649 us on the N=64 256-channel
    // layer).  Part q < 3 of the next step's V DMA (JP loads, spread so that
    // no wave stalls behind the whole burst) is issued at the start of quad q,
    // so at the start of step s+1 the 2*NG filter loads of quads 2 and 3 came
    // after the last part: all of its V has landed when at most those remain.
    constexpr int WAITN = 2 * NG;
    issue_v(IC<0>{}, 0, IC<0>{}, IC<JV>{});
    load_u(0, ubuf[0]);
    load_u(1, ubuf[1]);
    wait_vm_lds<WAITN>();             // V of step 0 has landed (for this wave)
    const uint32_t uq = (uint32_t)(kb * g.CQ) * (T / 4) + G0;
    auto step = [&](auto rc, int s) {  // s % 2 == R
        constexpr int R = decltype(rc)::value;
        wait_vm_lds<WAITN>();          // V of step s has landed (this wave)
        wg_barrier();                  // ... every wave's; stage R^1 (step s-1) is consumed
        const float* vs = stage(IC<R>{});
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            f32x4 (&cur)[NG] = ubuf[q & 1];
            auto part = [&](auto pc) {
                constexpr int P = decltype(pc)::value;
                constexpr int A0 = P * JP < JV ? P * JP : JV, A1 = (P + 1) * JP < JV ? (P + 1) * JP : JV;
                if (q == P) issue_v(IC<R ^ 1>{}, s + 1, IC<A0>{}, IC<A1>{});
            };
            part(IC<0>{});
            part(IC<1>{});
            part(IC<2>{});
            __builtin_amdgcn_sched_barrier(0);
            const uint32_t go2 = __builtin_amdgcn_readfirstlane(
                (uint32_t)((uq + (uint32_t)min(s * NQ + q + 2, g.CQ - 1) * (T / 4)) * 1024u));
            quad(vs, q, cur, [&](int gi) { cur[gi] = u_load(ur, ulane, go2 + (uint32_t)gi * 1024u); });
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    int s = 0;
    for (; s + 2 <= nsteps; s += 2) {      // straight-line body: exact wait analysis
        step(IC<0>{}, s);
        step(IC<1>{}, s + 1);
    }
    if (s < nsteps) step(IC<0>{}, s);
    __builtin_amdgcn_s_waitcnt(0);         // no load outlives the loop
}

// The same GEMMs on 16-bit operands (fp16 PREC 1, bf16 PREC 2) for the
// split path: v_mfma_f32_16x16x32_{f16,bf16} leaves its 16 x 16 result in the
// lane layout of v_mfma_f32_16x16x4_f32 (lane = tile, four consecutive
// filters), so the accumulators, and with them the epilogue, are the fp32
// kernel's.  A step is one 32-channel chunk: groups 2s and 2s+1 of the blocked
// VH ([block][C16][T][64][4 halves]), exactly the bytes of an fp32 step of 16
// channels, so the V DMA and its two LDS stages are go_steps's.  A position's
// B operand is the lane's 8-byte words of the two groups (two LDS reads); its
// A operand the lane's word of chunk s of UH ([KB][C32][T][64][8 halves], one
// 16-byte load).  The filters of position t come D positions ahead, into a
// ring of D operand registers: after t's products the ring slot takes
// position t + D (of this step, or of the next).  The V DMA of step s+1
// goes out in three parts at positions 0, TH/3 and 2*TH/3 of step s.
template <int MT, int H, int PREC>
__device__ __forceinline__ void go_steps16(const __amdgpu_buffer_rsrc_t vr, uint32_t vbase0, uint32_t vbase1,
                                           const __amdgpu_buffer_rsrc_t ur, uint32_t ubase, const Geom& g,
                                           int nsteps, int wave, int lane, float* vs0, float* vs1,
                                           f32x4 (&acc)[2][GoShape<MT>::TH]) {
    using S = GoShape<MT>;
    constexpr int A = S::A, X0 = H * S::RN, TH = S::TH, T = S::T;
    // filter lead: a third of a step for F(4x4) (TH = 18; the kernel's VGPRs
    // also hold the tail units' operands), half a step for F(2x2) (TH = 16)
    constexpr int D = MT == 4 ? TH / 3 : TH / 2;
    static_assert(TH % D == 0, "the ring wraps onto the next step's slots");
    auto stage = [&](auto rc) -> float* {
        if constexpr (decltype(rc)::value == 0) return vs0;
        else return vs1;
    };
    const uint32_t tid16 = ((uint32_t)wave * 64 + lane) * 16u;
    auto issue_v = [&](auto rc, int j, auto i0c, auto i1c) {
        float* vs = stage(rc);
        const uint32_t qoff = (uint32_t)j * T * 1024;             // bytes: two groups of T*512
        static_for<decltype(i0c)::value, decltype(i1c)::value>([&](auto ic) {
            constexpr int i = decltype(ic)::value;
            constexpr uint32_t RUN = S::JV * 256 * 16;           // bytes of one block's run
            constexpr uint32_t E0 = (uint32_t)i * 8192u;
            float* dst = vs + (i * 512 + wave * 64) * 4;
            if constexpr (E0 + 8192u <= RUN) {
                lds_dma<16>(vr, dst, tid16, vbase0 + E0 + qoff);
            } else if constexpr (E0 >= RUN) {
                lds_dma<16>(vr, dst, tid16, vbase1 + (E0 - RUN) + qoff);
            } else {
                const uint32_t voff = tid16 < RUN - E0 ? tid16 : tid16 + (vbase1 - vbase0 - RUN);
                lds_dma<16>(vr, dst, voff, vbase0 + E0 + qoff);
            }
        });
    };
    static_assert(T * 1024 == S::JV * 256 * 16, "a 16-bit step moves the bytes of an fp32 step");
    const uint32_t l16 = (uint32_t)lane * 16u;
    // A operand of (step s, position X0*A + t)
    auto load_u = [&](int s, int t, uint4& u) {
        const uint32_t go = __builtin_amdgcn_readfirstlane(ubase + (uint32_t)s * T * 1024u +
                                                           (uint32_t)(X0 * A + t) * 1024u);
        u = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ur, (int)l16, (int)go, 0));
    };
    // B operand of (block b, position X0*A + t) from a stage ([b][group][T][64][8 bytes])
    auto v_op = [&](const float* vs, int b, int t) {
        const uint2* w = (const uint2*)vs + (size_t)((b * 2) * T + X0 * A + t) * 64 + lane;
        const uint2 a = w[0], c = w[(size_t)T * 64];
        return make_uint4(a.x, a.y, c.x, c.y);
    };
    uint4 ur_[D];
    // Loads a step issues after its last V DMA part: the filter loads of
    // positions 2*PS .. TH-1, one each.  (The prologue issues D >= WAITN
    // filter loads after step 0's V.)
    constexpr int PS = TH / 3;
    constexpr int WAITN = TH - 2 * PS;
    static_assert(D >= WAITN, "the first wait covers step 0's V");
    issue_v(IC<0>{}, 0, IC<0>{}, IC<S::JV>{});
#pragma unroll
    for (int t = 0; t < D; ++t) load_u(0, t, ur_[t]);
    constexpr int JV = S::JV, JP = (JV + 2) / 3;
    auto step = [&](auto rc, int s) {  // s % 2 == R
        constexpr int R = decltype(rc)::value;
        wait_vm_lds<WAITN>();          // V of step s has landed (this wave)
        wg_barrier();                  // ... every wave's; stage R^1 (step s-1) is consumed
        const float* vs = stage(IC<R>{});
        const int sn = min(s + 1, nsteps - 1);
        static_for<0, TH>([&](auto tc) {
            constexpr int t = decltype(tc)::value;
            if constexpr (t % PS == 0 && t / PS < 3) {
                constexpr int P = t / PS;
                constexpr int A0 = P * JP < JV ? P * JP : JV, A1 = (P + 1) * JP < JV ? (P + 1) * JP : JV;
                issue_v(IC<R ^ 1>{}, s + 1, IC<A0>{}, IC<A1>{});
                __builtin_amdgcn_sched_barrier(0);
            }
            const uint4 v0 = v_op(vs, 0, t), v1 = v_op(vs, 1, t);
            acc[0][t] = mfma16x16x32<PREC>(ur_[t % D], v0, acc[0][t]);
            acc[1][t] = mfma16x16x32<PREC>(ur_[t % D], v1, acc[1][t]);
            if constexpr (t + D < TH) load_u(s, t + D, ur_[t % D]);
            else load_u(sn, t + D - TH, ur_[t % D]);
        });
    };
    int s = 0;
    for (; s + 2 <= nsteps; s += 2) {      // straight-line body: exact wait analysis
        step(IC<0>{}, s);
        step(IC<1>{}, s + 1);
    }
    if (s < nsteps) step(IC<0>{}, s);
    __builtin_amdgcn_s_waitcnt(0);         // no load outlives the loop
}

// The tile of lane l16 in block tb (16 consecutive tiles).
__device__ __forceinline__ TileCoord block_tile(int tb, int l16, const Geom& g) {
    return decode_tile(tb * 16 + l16, g);
}

// A GEMM + output-transform unit of a tail item: one tile block tb and one
// filter block kb over all channels.  The 8 waves are (row group h of TS) x
// (channel part cp of 8/TS); each multiplies its quads for its row group's
// positions, with U and V straight from memory to registers (no operand is
// shared between waves), one quad ahead.  Each wave then applies its row
// group's part of A^T M A to its accumulators, and the 8 partial outputs are
// summed through LDS in wave order: wave w adds and stores 1/8 of the values.
template <int MT, int H>
__device__ __forceinline__ void unit_steps(const __amdgpu_buffer_rsrc_t vr, const __amdgpu_buffer_rsrc_t ur,
                                           const Geom& g, int kb, int q0, int q1, int lane,
                                           f32x4 (&acc)[GoShape<MT>::TH]) {
    using S = GoShape<MT>;
    constexpr int A = S::A, X0 = H * S::RN, TH = S::TH, T = S::T;
    constexpr int G0 = X0 * A / 4, NG = (X0 * A + TH - 1) / 4 - G0 + 1;
    const uint32_t l16b = (uint32_t)lane * 16u;
    auto load = [&](int q, f32x4 (&ug)[NG], f32x4 (&vg)[NG]) {
        const int c = min(q, g.CQ - 1);    // quads past CQ: zero V, any filters
        const uint32_t go = __builtin_amdgcn_readfirstlane((uint32_t)(((kb * g.CQ + c) * (T / 4) + G0) * 1024));
        const uint32_t vo = __builtin_amdgcn_readfirstlane((uint32_t)((q * (T / 4) + G0) * 1024));
#pragma unroll
        for (int i = 0; i < NG; ++i) {
            ug[i] = u_load(ur, l16b, go + i * 1024u);
            vg[i] = u_load(vr, l16b, vo + i * 1024u);
        }
    };
    auto mma = [&](const f32x4 (&ug)[NG], const f32x4 (&vg)[NG]) {
#pragma unroll
        for (int t = 0; t < TH; ++t) {
            const int idx = X0 * A + t;
            acc[t] = mfma16x16x4(ug[idx / 4 - G0][idx % 4], vg[idx / 4 - G0][idx % 4], acc[t]);
        }
    };
    f32x4 ua[NG], va[NG], ub[NG], vb[NG];
    if (q0 < q1) load(q0, ua, va);
    for (int q = q0; q < q1; q += 2) {
        if (q + 1 < q1) load(q + 1, ub, vb);
        mma(ua, va);
        if (q + 2 < q1) load(q + 2, ua, va);
        if (q + 1 < q1) mma(ub, vb);
    }
}

// The 16-bit form of unit_steps: 32-channel chunks [c0, c1) of tile block
// (vr) and filter block (ubase into UH); per chunk and half of the wave's TH
// positions, the operands straight to registers (one 16-byte filter load, two
// 8-byte V loads per position), then their products.
template <int MT, int H, int PREC>
__device__ __forceinline__ void unit_steps16(const __amdgpu_buffer_rsrc_t vr, const __amdgpu_buffer_rsrc_t ur,
                                             uint32_t ubase, int c0, int c1, int lane,
                                             f32x4 (&acc)[GoShape<MT>::TH]) {
    using S = GoShape<MT>;
    constexpr int A = S::A, X0 = H * S::RN, TH = S::TH, T = S::T, HT = TH / 2;
    static_assert(TH % 2 == 0, "two halves");
    const uint32_t l16 = (uint32_t)lane * 16u, l8 = (uint32_t)lane * 8u;
    for (int c = c0; c < c1; ++c) {
        const uint32_t uo = __builtin_amdgcn_readfirstlane(ubase + (uint32_t)c * T * 1024u + (uint32_t)(X0 * A) * 1024u);
        const uint32_t vo = __builtin_amdgcn_readfirstlane((uint32_t)c * T * 1024u + (uint32_t)(X0 * A) * 512u);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            uint4 u[HT], v[HT];
#pragma unroll
            for (int i = 0; i < HT; ++i) {
                const uint32_t t = (uint32_t)(hh * HT + i);
                u[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ur, (int)l16, (int)(uo + t * 1024u), 0));
                const uint2 a = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(vr, (int)l8, (int)(vo + t * 512u), 0));
                const uint2 b = __builtin_bit_cast(
                    uint2, __builtin_amdgcn_raw_buffer_load_b64(vr, (int)l8, (int)(vo + (uint32_t)T * 512u + t * 512u), 0));
                v[i] = make_uint4(a.x, a.y, b.x, b.y);
            }
#pragma unroll
            for (int i = 0; i < HT; ++i) acc[hh * HT + i] = mfma16x16x32<PREC>(u[i], v[i], acc[hh * HT + i]);
        }
    }
}

// PREC 0: fp32 (nq = ncq4*4 channel quads per Vb block); 1 / 2: 16-bit (VH
// and UH, ncq4 = C32 chunks).
template <int MT, int PREC = 0>
__device__ __forceinline__ void gemm_out_unit(const float* __restrict__ Vb, const float* __restrict__ U,
                                              float* __restrict__ y, const Geom& g, int tb, int kb, int ncq4,
                                              bool relu, bool vec_ok, bool nts, float4* vs0, float4* vs1,
                                              int wave, int lane) {
    using S = GoShape<MT>;
    constexpr int TS = S::TS, TH = S::TH, T = S::T, CP = 8 / TS, NV = S::NV, VPW = NV / 8;
    static_assert(4 * NV * 64 <= S::VST, "four partial-output slots per LDS stage");
    static_assert(VPW % MT == 0, "whole output rows per wave");
    const int h = wave % TS, cp = wave / TS;
    const int nq = PREC ? ncq4 : ncq4 * 4;                  // quads, or 32-channel chunks
    const int qpp = (nq + CP - 1) / CP;
    const int q0 = min(cp * qpp, nq), q1 = min(nq, q0 + qpp);
    const size_t blk_b = PREC ? (size_t)nq * T * 1024 : (size_t)nq * T * 256;
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)((const char*)Vb + (size_t)tb * blk_b), (short)0, (int)(blk_b < kInvalid ? blk_b : kInvalid),
        kRsrcWord3);
    f32x4 acc[TH];
#pragma unroll
    for (int t = 0; t < TH; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float o[4][MT][MT];
    auto steps = [&](auto hc) {
        constexpr int HH = decltype(hc)::value;
        if constexpr (PREC == 0) {
            unit_steps<MT, HH>(vr, u_rsrc(U, g), g, kb, q0, q1, lane, acc);
        } else {
            const size_t uh_b = (size_t)g.KB * nq * T * 1024;
            const __amdgpu_buffer_rsrc_t ur = __builtin_amdgcn_make_buffer_rsrc(
                (void*)U, (short)0, (int)(uh_b < 0x7fffffffu ? uh_b : 0x7fffffffu), kRsrcWord3);
            unit_steps16<MT, HH, PREC>(vr, ur, (uint32_t)kb * (uint32_t)nq * T * 1024u, q0, q1, lane, acc);
        }
    };
    if constexpr (TS == 1) {
        steps(IC<0>{});
        fused_share<MT, 1, 1, 16, 0, 0>(acc, o);
    } else {
        if (h == 0) {
            steps(IC<0>{});
            fused_share<MT, 2, 1, 16, 0, 0>(acc, o);
        } else {
            steps(IC<1>{});
            fused_share<MT, 2, 1, 16, 0, 1>(acc, o);
        }
    }
    // Slot w of NV*64 floats: w < 4 in vs0, else vs1 (each branch names its
    // array, so the accesses stay LDS accesses).
    auto with_slot = [&](int w, auto&& f) {
        if (w < 4) f((float*)vs0 + (size_t)w * NV * 64 + lane);
        else f((float*)vs1 + (size_t)(w - 4) * NV * 64 + lane);
    };
    with_slot(wave, [&](float* slot) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j) slot[((r * MT + i) * MT + j) * 64] = o[r][i][j];
    });
    __syncthreads();
    float sum[VPW];
#pragma unroll
    for (int e = 0; e < VPW; ++e) sum[e] = 0.f;
#pragma unroll
    for (int w = 0; w < 8; ++w) {
        with_slot(w, [&](float* slot) {
#pragma unroll
            for (int e = 0; e < VPW; ++e) sum[e] += slot[(wave * VPW + e) * 64];
        });
    }
    const int f0 = wave * VPW, r = f0 / (MT * MT), i0 = (f0 % (MT * MT)) / MT;
    const TileCoord tc = block_tile(tb, lane & 15, g);
    const int k = kb * 16 + 4 * (lane >> 4) + r;
#pragma unroll
    for (int ii = 0; ii < VPW / MT; ++ii) {
        float row[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) row[j] = sum[ii * MT + j];
        if (g.nhwc) {                   // channel-last: one value per pixel
            const int oi = tc.ti * MT + i0 + ii;
            if (tc.valid && k < g.K && oi < g.Ho)
#pragma unroll
                for (int j = 0; j < MT; ++j) {
                    const int oj = tc.tj * MT + j;
                    if (oj < g.Wo)
                        y[(((size_t)tc.n * g.Ho + oi) * g.Wo + oj) * g.K + k] = relu ? fmaxf(row[j], 0.0f) : row[j];
                }
        } else {
            if (nts) store_row<MT, true>(y, g, tc, k, i0 + ii, row, relu, vec_ok);
            else store_row<MT, false>(y, g, tc, k, i0 + ii, row, relu, vec_ok);
        }
    }
}

// PREC 0: fp32 operands (Vb, U); 1 / 2: fp16 / bf16 (VH in 16-channel groups,
// UH in 32-channel chunks), through go_steps16 (and unit_steps16 for the tail).
template <int MT, int PREC = 0>
__global__ __launch_bounds__(512) void k_gemm_out(const float* __restrict__ Vb, const float* __restrict__ U,
                                                  float* __restrict__ y, Geom g, FusedTiling ft, int nb,
                                                  int relu, int vec_ok, int nts, int ntail) {
    using S = GoShape<MT>;
    constexpr int TS = S::TS, KGW = S::KGW, TH = S::TH, NV = S::NV;
    __shared__ float4 vs0[S::VST / 4], vs1[S::VST / 4];

    // item = (tile-block pair, filter group), XCD-aware as in k_fused; the
    // last ntail items run as 2*KGW units each after the others
    const int b = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int nmain = ft.nt * ft.nkg - ntail;
    auto decode = [&](int it, int& kgi, int& tp) {
        kgi = ft.kfast ? it % ft.nkg : it / ft.nt;
        tp = ft.kfast ? it / ft.nkg : it - kgi * ft.nt;
    };
    if (b >= 8 * ft.per) {
        const int u = b - 8 * ft.per;
        const int it = nmain + u / (2 * KGW), sub = u % (2 * KGW);
        int kgi, tp;
        decode(it, kgi, tp);
        const int tb = 2 * tp + sub / KGW, kb = kgi * KGW + sub % KGW;
        if (tb >= nb || kb >= g.KB) return;
        gemm_out_unit<MT, PREC>(Vb, U, y, g, tb, kb, PREC ? (g.C + 31) / 32 : (g.CQ + 3) / 4, relu != 0,
                                vec_ok != 0, nts != 0, vs0, vs1, wave, lane);
        return;
    }
    const int item = (b & 7) * ft.per + (b >> 3);
    if (item >= nmain) return;
    int kgi, tp;
    decode(item, kgi, tp);
    const int kw = wave / TS, h = wave % TS;
    const int kb = min(kgi * KGW + kw, g.KB - 1);
    const int cl = lane >> 4;

    // Vb as a buffer: a block past the last reads zeros
    const size_t blk_b = PREC ? (size_t)((g.C + 31) / 32) * g.T * 1024   // bytes of one tile block
                              : (size_t)((g.CQ + 3) / 4 * 4) * g.T * 256;
    const size_t tot_b = (size_t)nb * blk_b;
    const size_t first = (size_t)(2 * tp) * blk_b;
    const size_t left = tot_b - first;
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)((const char*)Vb + first), (short)0, (int)(left < kInvalid ? left : kInvalid), kRsrcWord3);

    f32x4 acc[2][TH];
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
        for (int t = 0; t < TH; ++t) acc[bb][t] = f32x4{0.f, 0.f, 0.f, 0.f};
    float* v0 = (float*)vs0;
    float* v1 = (float*)vs1;
    if constexpr (PREC != 0) {
        // UH as a buffer (the host keeps it below 2 GiB)
        const int c32 = (g.C + 31) / 32;
        const size_t uh_b = (size_t)g.KB * c32 * g.T * 1024;
        const __amdgpu_buffer_rsrc_t ur = __builtin_amdgcn_make_buffer_rsrc(
            (void*)U, (short)0, (int)(uh_b < 0x7fffffffu ? uh_b : 0x7fffffffu), kRsrcWord3);
        const uint32_t ubase = (uint32_t)kb * (uint32_t)c32 * (uint32_t)g.T * 1024u;
        if constexpr (TS == 1) {
            go_steps16<MT, 0, PREC>(vr, 0u, (uint32_t)blk_b, ur, ubase, g, ft.nsteps, wave, lane, v0, v1, acc);
        } else {
            if (h == 0) go_steps16<MT, 0, PREC>(vr, 0u, (uint32_t)blk_b, ur, ubase, g, ft.nsteps, wave, lane, v0, v1, acc);
            else go_steps16<MT, 1, PREC>(vr, 0u, (uint32_t)blk_b, ur, ubase, g, ft.nsteps, wave, lane, v0, v1, acc);
        }
    } else if constexpr (TS == 1) {
        go_steps<MT, 0>(vr, 0u, (uint32_t)blk_b, U, g, ft.nsteps, kb, wave, lane, v0, v1, acc);
    } else {
        if (h == 0) go_steps<MT, 0>(vr, 0u, (uint32_t)blk_b, U, g, ft.nsteps, kb, wave, lane, v0, v1, acc);
        else go_steps<MT, 1>(vr, 0u, (uint32_t)blk_b, U, g, ft.nsteps, kb, wave, lane, v0, v1, acc);
    }

    // This wave's share of A^T M A for both tile blocks.
    float o[2][4][MT][MT];
#pragma unroll
    for (int bb = 0; bb < 2; ++bb) {
        f32x4 a1[TH];
#pragma unroll
        for (int t = 0; t < TH; ++t) a1[t] = acc[bb][t];
        if constexpr (TS == 1) {
            fused_share<MT, 1, 8, 16, 0, 0>(a1, o[bb]);
        } else {
            if (h == 0) fused_share<MT, 2, 1, 16, 0, 0>(a1, o[bb]);
            else fused_share<MT, 2, 1, 16, 0, 1>(a1, o[bb]);
        }
    }
    const int kbase = (kgi * KGW + kw) * 16 + 4 * cl;
    auto tile_of = [&](int bb) { return block_tile(2 * tp + bb, lane & 15, g); };
    const bool rl = relu != 0, vo = vec_ok != 0;
    if constexpr (TS == 1) {
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            const TileCoord tc = tile_of(bb);
            if (g.nhwc) {
                if (nts) store_tile_nhwc<MT, true>(y, g, tc, kbase, o[bb], rl, vo);
                else store_tile_nhwc<MT, false>(y, g, tc, kbase, o[bb], rl, vo);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (nts) store_block<MT, true>(y, g, tc, kbase + r, o[bb][r], rl, vo);
                    else store_block<MT, false>(y, g, tc, kbase + r, o[bb][r], rl, vo);
                }
            }
        }
    } else {
        // Row half h of filter block kw sums tile block h (its own share plus
        // the other half's, written to LDS) and stores it.  Slot (kw, bb) of
        // NV*64 floats: kw < 2 in vs0, else vs1 (each branch names its array,
        // so the accesses stay LDS accesses).
        static_assert(4 * NV * 64 <= S::VST, "two exchange slots per filter block per stage");
        auto with_slot = [&](int bb, auto&& f) {
            const int k = (kw & 1) * 2 + bb;
            if (kw < 2) f((float*)vs0 + (size_t)k * NV * 64 + lane);
            else f((float*)vs1 + (size_t)k * NV * 64 + lane);
        };
        __syncthreads();                       // every wave is done with the V stages
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            if (bb == h) continue;
            with_slot(bb, [&](float* slot) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int i = 0; i < MT; ++i)
#pragma unroll
                        for (int j = 0; j < MT; ++j) slot[((r * MT + i) * MT + j) * 64] = o[bb][r][i][j];
            });
        }
        __syncthreads();
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            if (bb != h) continue;
            float sl[4][MT][MT];
            with_slot(bb, [&](float* slot) {
#pragma unroll
                for (int r = 0; r < 4; ++r)
#pragma unroll
                    for (int i = 0; i < MT; ++i)
#pragma unroll
                        for (int j = 0; j < MT; ++j) sl[r][i][j] = slot[((r * MT + i) * MT + j) * 64];
            });
            const TileCoord tc = tile_of(bb);
            float ob[4][MT][MT];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int i = 0; i < MT; ++i)
#pragma unroll
                    for (int j = 0; j < MT; ++j) ob[r][i][j] = o[bb][r][i][j] + sl[r][i][j];
            if (g.nhwc) {
                if (nts) store_tile_nhwc<MT, true>(y, g, tc, kbase, ob, rl, vo);
                else store_tile_nhwc<MT, false>(y, g, tc, kbase, ob, rl, vo);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (nts) store_block<MT, true>(y, g, tc, kbase + r, ob[r], rl, vo);
                    else store_block<MT, false>(y, g, tc, kbase + r, ob[r], rl, vo);
                }
            }
        }
    }
}

// ------------------------------------------------------------------ low C
// Layers with at most 4 input channels (a network's first layer).  The GEMMs
// contract over NC <= 4 channels, so the layer is bound by writing y; the
// fused kernels' per-workgroup phases (load, transform, MFMA, exchange,
// store) would run one after another on each CU.  Here a lane owns one tile:
// it keeps the transforms of its NC regions in registers and, filter by
// filter, forms M_t = sum_c U_t[c][k] V_t[c] with vector FMAs (U broadcast
// from LDS), applies A^T M A and stores the m x m block -- the stores of one
// filter drain while the next is computed.  A workgroup of 4 waves covers 256
// consecutive tiles and a range of KPW filters.
template <int MT, int NC, bool RELU>
__global__ __launch_bounds__(256) void k_lowc(const float* __restrict__ x, const float* __restrict__ U,
                                              float* __restrict__ y, Geom g, int ntg, int kpw, int vec_ok, int nts) {
    constexpr int A = MT + 2, T = A * A, TG = T / 4;
    extern __shared__ float4 us4[];                   // [kpw][NC][T]
    float* us = (float*)us4;
    const int tg = blockIdx.x % ntg, kf = blockIdx.x / ntg;
    const int k0 = kf * kpw, nk = min(kpw, g.K - k0);
    const int tid = threadIdx.x;
    // this workgroup's filters into LDS: element (t, c, k) of U is at lane
    // c*16 + k%16, slot t%4 of group ((k/16)*CQ*TG + t/4) (CQ = 1 here)
    for (int e = tid; e < nk * NC * T; e += 256) {
        const int kk = e / (NC * T), rem = e - kk * (NC * T), c = rem / T, t = rem - c * T;
        const int k = k0 + kk;
        us[e] = U[((size_t)(k / 16) * TG + t / 4) * 256 + (c * 16 + k % 16) * 4 + t % 4];
    }
    const int p = tg * 256 + tid;
    const TileCoord tc = decode_tile(p, g);
    float v[NC][T];
    {
        const int r0 = tc.ti * MT - g.pad, c0 = tc.tj * MT - g.pad;
        const float* xi = x + (size_t)tc.n * g.C * g.H * g.W;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float d[A][A];
#pragma unroll
            for (int u = 0; u < A; ++u)
#pragma unroll
                for (int w = 0; w < A; ++w) {
                    const int r = r0 + u, cc = c0 + w;
                    const bool ok = tc.valid && (unsigned)r < (unsigned)g.H && (unsigned)cc < (unsigned)g.W;
                    d[u][w] = ok ? xi[((size_t)c * g.H + r) * g.W + cc] : 0.0f;
                }
            input_tf<MT>(d, v[c]);
        }
    }
    __syncthreads();
    // A tile whose m x m block lies inside the image (all but the last tile row
    // and column) stores whole rows with vector stores, no per-row checks.
    const bool vo = vec_ok != 0;
    const bool inner = vo && tc.valid && tc.ti * MT + MT <= g.Ho && tc.tj * MT + MT <= g.Wo;
    const size_t plane = (size_t)g.Ho * g.Wo;
    float* yb = y + ((size_t)tc.n * g.K + k0) * plane + (size_t)(tc.ti * MT) * g.Wo + tc.tj * MT;
    for (int kk = 0; kk < nk; ++kk) {
        const float4* uk = (const float4*)(us + (size_t)kk * NC * T);
        float mv[T];
#pragma unroll
        for (int t4 = 0; t4 < TG; ++t4) {
            const float4 u0 = uk[t4];
            mv[4 * t4] = u0.x * v[0][4 * t4];
            mv[4 * t4 + 1] = u0.y * v[0][4 * t4 + 1];
            mv[4 * t4 + 2] = u0.z * v[0][4 * t4 + 2];
            mv[4 * t4 + 3] = u0.w * v[0][4 * t4 + 3];
#pragma unroll
            for (int c = 1; c < NC; ++c) {
                const float4 uc = uk[c * TG + t4];
                mv[4 * t4] = __builtin_fmaf(uc.x, v[c][4 * t4], mv[4 * t4]);
                mv[4 * t4 + 1] = __builtin_fmaf(uc.y, v[c][4 * t4 + 1], mv[4 * t4 + 1]);
                mv[4 * t4 + 2] = __builtin_fmaf(uc.z, v[c][4 * t4 + 2], mv[4 * t4 + 2]);
                mv[4 * t4 + 3] = __builtin_fmaf(uc.w, v[c][4 * t4 + 3], mv[4 * t4 + 3]);
            }
        }
        float o[MT][MT];
        output_tf<MT>(mv, o);
        if (RELU) {
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int j = 0; j < MT; ++j) o[i][j] = fmaxf(o[i][j], 0.0f);
        }
        if (inner) {
            float* r = yb + kk * plane;
#pragma unroll
            for (int i = 0; i < MT; ++i) {
                if constexpr (MT == 4) {
                    if (nts) store_out<true>(r + (size_t)i * g.Wo, o[i][0], o[i][1], o[i][2], o[i][3]);
                    else store_out<false>(r + (size_t)i * g.Wo, o[i][0], o[i][1], o[i][2], o[i][3]);
                } else {
                    if (nts) store_out<true>(r + (size_t)i * g.Wo, o[i][0], o[i][1]);
                    else store_out<false>(r + (size_t)i * g.Wo, o[i][0], o[i][1]);
                }
            }
        } else if (nts) {
            store_block<MT, true>(y, g, tc, k0 + kk, o, false, vo);
        } else {
            store_block<MT, false>(y, g, tc, k0 + kk, o, false, vo);
        }
    }
}

// ------------------------------------------------------------------ 16-bit operands
// Reduced-precision three-stage path: U and V are rounded to fp16 (PREC 1) or
// bf16 (PREC 2), to nearest with ties to even, and the T per-position GEMMs run
// on v_mfma_f32_16x16x32_{f16,bf16} with fp32 accumulation; M and the output
// transform stay fp32.  Filters come in 32-channel chunks, a lane carrying
// eight channels of its chunk -- four consecutive channels of each of its two
// 16-channel groups -- in one 16-byte word; inputs in 16-channel groups, a lane
// carrying four consecutive channels in one 8-byte word:
//   UH[KB][C32][T][64][8]: element (t, c, k) at lane ((c%16)/4)*16 + k%16,
//                          half ((c%32)/16)*4 + c%4
//   VH[PB][C16][T][64][4]: element (t, c, p) at lane ((c%16)/4)*16 + p%16, half c%4
// (C32 = ceil(C/32), C16 = 2*C32 groups, padding zero).  A UH word is exactly
// the lane's A operand of v_mfma_f32_16x16x32_{f16,bf16} (A[l%16] at eight
// reduction slots): one 16-byte load; the B operand is the lane's VH words of
// groups 2j and 2j+1 side by side.  The filter transform writes one 16-channel
// group at a time, the lane's 8-byte half (c%32)/16 of each word; the input
// transforms write whole 8-byte words (as 16-bit values of one channel per
// lane of a quad, 128 contiguous bytes per store, for k_vrows).


template <int PREC>
__device__ __forceinline__ uint2 pack16(float a, float b, float c, float d) {
    return make_uint2(to16<PREC>(a) | (to16<PREC>(b) << 16), to16<PREC>(c) | (to16<PREC>(d) << 16));
}


// One wave per (16-filter block, 16-channel group): lane = (k%16, channel
// quad); four channels' transforms per lane, one 8-byte store per position
// (positions 128 words apart: the other half of each 16-byte word is the
// chunk's other group).
template <int MT, int PREC, int... G>
__device__ __forceinline__ void filter16_groups(const float (&gg)[4][3][3], uint2* __restrict__ dst,
                                                std::integer_sequence<int, G...>) {
    auto one = [&](auto gc) {
        constexpr int GG = decltype(gc)::value;
        float4 f[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) f[e] = filter_tf4<MT, 4 * GG>(gg[e]);
        dst[(4 * GG + 0) * 128] = pack16<PREC>(f[0].x, f[1].x, f[2].x, f[3].x);
        dst[(4 * GG + 1) * 128] = pack16<PREC>(f[0].y, f[1].y, f[2].y, f[3].y);
        dst[(4 * GG + 2) * 128] = pack16<PREC>(f[0].z, f[1].z, f[2].z, f[3].z);
        dst[(4 * GG + 3) * 128] = pack16<PREC>(f[0].w, f[1].w, f[2].w, f[3].w);
    };
    (one(std::integral_constant<int, G>{}), ...);
}

// C16P = 2 * C32 groups per filter block (a padding group is written zero).
template <int MT, int PREC>
__global__ __launch_bounds__(256) void k_filter16(const float* __restrict__ gw, uint2* __restrict__ UH, int C,
                                                  int K, int C16P, long nw) {
    constexpr int T = (MT + 2) * (MT + 2), TG = T / 4;
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= nw) return;
    const int kb = (int)(w / C16P), c16 = (int)(w % C16P);
    const int k = kb * 16 + (lane & 15), c0 = c16 * 16 + (lane >> 4) * 4;
    float gg[4][3][3];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const bool ok = k < K && c0 + e < C;
        const float* src = gw + ((size_t)(ok ? k : 0) * C + (ok ? c0 + e : 0)) * 9;
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
            for (int s2 = 0; s2 < 3; ++s2) gg[e][r][s2] = ok ? src[r * 3 + s2] : 0.0f;
    }
    uint2* dst = UH + (((size_t)kb * (C16P >> 1) + (c16 >> 1)) * T * 64 + lane) * 2 + (c16 & 1);
    filter16_groups<MT, PREC>(gg, dst, std::make_integer_sequence<int, TG>{});
}

// One wave per (16-tile block, 16-channel group), XCD-contiguous runs; lane =
// (tile p%16, channel quad): four regions, their transforms packed four
// channels to an 8-byte word.  C16 = 2 * C32 groups (a padding group: zeros).
template <int MT, int PREC>
__global__ __launch_bounds__(256) void k_input16(const float* __restrict__ x, uint2* __restrict__ VH, Geom g,
                                                 int C16, long nwg) {
    constexpr int A = MT + 2, T = A * A;
    const int lane = threadIdx.x & 63;
    const long per = (nwg + 7) / 8, item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nwg) return;
    const long w = item * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * C16) return;
    const int pb = (int)(w / C16), c16 = (int)(w % C16);
    const int cq4 = lane >> 4;                                  // channel quad within the group
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const RegionPlan<MT> rp = make_region_plan<MT>(x, g, pb * 16, tc, cq4 * 4);
    uint32_t ph[T][2];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        // channel c16*16 + cq4*4 + e: the plan holds cq4*4, the wave-uniform
        // offset adds c16*16 + e planes
        const uint32_t chan = (c16 * 16 + cq4 * 4 + e < g.C) ? 0u : kInvalid;
        const int soff = __builtin_amdgcn_readfirstlane((c16 * 16 + e) * (int)rp.plane_bytes);
        float d[A][A];
#pragma unroll
        for (int u = 0; u < A; ++u) {
            const uint32_t rowq = rp.row[u] + chan;
#pragma unroll
            for (int v = 0; v < A; ++v)
                d[u][v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                              rp.rsrc, (int)(rowq + rp.col[v]), soff, 0));
        }
        float vv[T];
        input_tf<MT>(d, vv);
#pragma unroll
        for (int t = 0; t < T; ++t) {
            const uint32_t hbits = to16<PREC>(vv[t]);
            if (e & 1) ph[t][e >> 1] |= hbits << 16;
            else ph[t][e >> 1] = hbits;
        }
    }
    uint2* dst = VH + ((size_t)pb * C16 + c16) * T * 64 + lane;
#pragma unroll
    for (int t = 0; t < T; ++t) dst[t * 64] = make_uint2(ph[t][0], ph[t][1]);
}

// The T GEMMs on 16-bit operands, on v_mfma_f32_16x16x32_{f16,bf16}: one
// instruction takes a 32-channel chunk, the lane's 16-byte word of UH and of
// VH (A and B place the same channel in the same operand slot, so the
// instruction's reduction covers all 32).  Workgroup = NP positions x 8
// k-blocks x 8 p-blocks, 8 waves of NP x 4 k-blocks x 2 p-blocks each
// (XCD-contiguous item order).  A chunk is 16*NP 1 KB blocks (U of position x
// k-block: one UH block; then V of position x p-block: the two 512-byte group
// blocks of VH, lanes 0-31 the first, 32-63 the second) and comes into one of
// three LDS stages by DMA two chunks ahead, one 16-byte load per lane and
// block.  Blocks past the last read zero.
template <int PREC, int NP>
__global__ __launch_bounds__(512) void k_gemm16(const uint2* __restrict__ UH, const uint2* __restrict__ VH,
                                                float* __restrict__ M, Geom g, int C32) {
    constexpr int NPAIR = 16 * NP, PPW = NPAIR / 8;       // pairs per chunk, per wave
    __shared__ uint4 st0[NPAIR * 64], st1[NPAIR * 64], st2[NPAIR * 64];   // three stages of pairs x 1 KB
    const int T = g.T, TN = g.T / NP;
    const int KB8 = (g.KB + 7) >> 3, PB8 = (g.PB + 7) >> 3;
    const long nitems = (long)TN * PB8 * KB8, per = (nitems + 7) / 8;
    const long item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nitems) return;
    const int kb0 = (int)(item % KB8) * 8;
    const long rest = item / KB8;
    const int pb0 = (int)(rest % PB8) * 8;
    const int t0 = (int)(rest / PB8) * NP;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wk = wave >> 2, wp = wave & 3;              // k-blocks 4*wk .. +3, p-blocks 2*wp, +1
    const int NC = C32;
    const uint32_t gstride = (uint32_t)T * 1024;         // bytes between chunks of one block
    const uint32_t bstride = (uint32_t)C32 * gstride;    // bytes between blocks (UH and VH alike)
    // U and V of this item's blocks as buffers: a block past the last reads zeros
    const size_t ub = (size_t)min(g.KB - kb0, 8) * bstride, vb = (size_t)min(g.PB - pb0, 8) * bstride;
    const __amdgpu_buffer_rsrc_t ur = __builtin_amdgcn_make_buffer_rsrc(
        (void*)((const char*)UH + (size_t)kb0 * bstride), (short)0, (int)ub, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t vr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)((const char*)VH + (size_t)pb0 * bstride), (short)0, (int)vb, kRsrcWord3);
    auto stage = [&](auto sc) -> uint4* {
        constexpr int S = decltype(sc)::value;
        if constexpr (S == 0) return st0;
        else if constexpr (S == 1) return st1;
        else return st2;
    };
    // DMA of chunk c into stage sc: wave w moves blocks PPW*w .. PPW*w+PPW-1.
    const uint32_t u_off = (uint32_t)lane * 16u;
    const uint32_t v_off = (uint32_t)(lane >> 5) * (uint32_t)T * 512u + (uint32_t)(lane & 31) * 16u;
    auto issue = [&](auto sc, int c) {
        uint4* s = stage(sc);
#pragma unroll
        for (int i = 0; i < PPW; ++i) {
            const int q = wave * PPW + i, qq = q < 8 * NP ? q : q - 8 * NP, pos = qq >> 3, blk = qq & 7;
            if (q < 8 * NP) {
                const uint32_t soff = (uint32_t)blk * bstride + (uint32_t)c * gstride + (uint32_t)(t0 + pos) * 1024u;
                lds_dma<16>(ur, (float*)(s + q * 64), u_off, __builtin_amdgcn_readfirstlane(soff));
            } else {
                const uint32_t soff = (uint32_t)blk * bstride + (uint32_t)c * gstride + (uint32_t)(t0 + pos) * 512u;
                lds_dma<16>(vr, (float*)(s + q * 64), v_off, __builtin_amdgcn_readfirstlane(soff));
            }
        }
    };
    f32x4 acc[NP][4][2];
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[p][i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    // operand of lane l from pair q: its words of both groups
    // U: the lane's word; V: the lane's words of the two groups
    auto u_operand = [&](const uint4* s, int q) { return s[q * 64 + lane]; };
    auto v_operand = [&](const uint4* s, int q) {
        const uint2* w = (const uint2*)(s + q * 64);
        const uint2 a = w[lane], b = w[64 + lane];
        return make_uint4(a.x, a.y, b.x, b.y);
    };
    issue(IC<0>{}, 0);
    if (NC > 1) issue(IC<1>{}, 1);
    // Chunk ch (stage ch % 3): at its start the PPW DMA loads of chunk ch+1
    // may still be in flight, not those of chunk ch; the barrier then tells
    // every wave that chunk ch is in LDS and chunk ch-1's stage is free for
    // chunk ch+2.
    auto chunk = [&](auto sc, int ch) {
        constexpr int S = decltype(sc)::value;
        if (ch + 1 < NC) wait_vm_lds<PPW>();
        else wait_vm_lds<0>();
        wg_barrier();
        if (ch + 2 < NC) issue(IC<(S + 2) % 3>{}, ch + 2);
        const uint4* s = stage(sc);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            uint4 a[4], b[2];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = u_operand(s, p * 8 + wk * 4 + i);
#pragma unroll
            for (int j = 0; j < 2; ++j) b[j] = v_operand(s, 8 * NP + p * 8 + wp * 2 + j);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[p][i][j] = mfma16x16x32<PREC>(a[i], b[j], acc[p][i][j]);
        }
    };
    int ch = 0;
    for (; ch + 3 <= NC; ch += 3) {
        chunk(IC<0>{}, ch);
        chunk(IC<1>{}, ch + 1);
        chunk(IC<2>{}, ch + 2);
    }
    if (ch < NC) chunk(IC<0>{}, ch);
    if (ch + 1 < NC) chunk(IC<1>{}, ch + 1);
#pragma unroll
    for (int p = 0; p < NP; ++p)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int kb = kb0 + wk * 4 + i, pb = pb0 + wp * 2 + j;
                if (kb < g.KB && pb < g.PB)
                    *(f32x4*)(M + (((size_t)pb * g.KB + kb) * T + t0 + p) * 256 + lane * 4) = acc[p][i][j];
            }
}

static inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

hipError_t launch_filter_transform16(const float* gw, void* UH, int C, int K, int m, int prec, hipStream_t s) {
    // every group of C32 chunks (a padding group is written zero)
    const int C16P = (C + 31) / 32 * 2, KB = (K + 15) / 16;
    const long waves = (long)KB * C16P;
    if ((waves + 3) / 4 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    uint2* u = (uint2*)UH;
    if (m == 2 && prec == 1) hipLaunchKernelGGL((k_filter16<2, 1>), grid, block, 0, s, gw, u, C, K, C16P, waves);
    else if (m == 2) hipLaunchKernelGGL((k_filter16<2, 2>), grid, block, 0, s, gw, u, C, K, C16P, waves);
    else if (prec == 1) hipLaunchKernelGGL((k_filter16<4, 1>), grid, block, 0, s, gw, u, C, K, C16P, waves);
    else hipLaunchKernelGGL((k_filter16<4, 2>), grid, block, 0, s, gw, u, C, K, C16P, waves);
    return hipGetLastError();
}

hipError_t launch_staged16(const float* x, const void* UH, float* y, void* VH, float* M, const Geom& g, int prec,
                           bool relu, hipStream_t s) {
    const int C32 = (g.C + 31) / 32, C16 = 2 * C32;   // groups of the input transforms
    const long waves = (long)g.PB * C16, nwg = (waves + 3) / 4;
    if ((nwg + 7) / 8 * 8 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 gi((unsigned)((nwg + 7) / 8 * 8)), block(256);
    uint2* vh = (uint2*)VH;
    const int vec = g.W % 4 == 0 && aligned(x, 16);
    const VrowsPlan vp = vrows_plan(g, vec);
    if (vp.R > 0) {
        // by whole tile rows, the lanes of a quad storing their channels' 16 bits
        const long ngr = ((long)g.N * g.th + vp.R - 1) / vp.R;
        const dim3 gr((unsigned)(ngr * 4 * C16)), b256(256);
        float* vf = (float*)VH;
#define WINO_VROWS16(MT, P) \
    hipLaunchKernelGGL((k_vrows<MT, P>), gr, b256, vp.lds, s, x, vf, g, vp.R, vp.pitch, 4 * C16)
        if (g.m == 2 && prec == 1) WINO_VROWS16(2, 1);
        else if (g.m == 2) WINO_VROWS16(2, 2);
        else if (prec == 1) WINO_VROWS16(4, 1);
        else WINO_VROWS16(4, 2);
#undef WINO_VROWS16
    } else if (g.m == 2 && prec == 1) hipLaunchKernelGGL((k_input16<2, 1>), gi, block, 0, s, x, vh, g, C16, nwg);
    else if (g.m == 2) hipLaunchKernelGGL((k_input16<2, 2>), gi, block, 0, s, x, vh, g, C16, nwg);
    else if (prec == 1) hipLaunchKernelGGL((k_input16<4, 1>), gi, block, 0, s, x, vh, g, C16, nwg);
    else hipLaunchKernelGGL((k_input16<4, 2>), gi, block, 0, s, x, vh, g, C16, nwg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // one position per workgroup: 48 KB of LDS, so up to three workgroups share a CU
    constexpr int NP = 1;
    if ((size_t)8 * C32 * g.T * 1024 >= (size_t)kInvalid) return hipErrorInvalidConfiguration;   // 32-bit offsets
    const long nitems = (long)((g.PB + 7) / 8) * ((g.KB + 7) / 8) * (g.T / NP);
    const long wgs = (nitems + 7) / 8 * 8;
    if (wgs > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 b512(512);
    if (prec == 1)
        hipLaunchKernelGGL((k_gemm16<1, NP>), dim3((unsigned)wgs), b512, 0, s, (const uint2*)UH, vh, M, g, C32);
    else
        hipLaunchKernelGGL((k_gemm16<2, NP>), dim3((unsigned)wgs), b512, 0, s, (const uint2*)UH, vh, M, g, C32);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_output_transform(M, y, g, relu, s);
}

// ------------------------------------------------------------------ NHWC
// Channel-last tensors (x [N][H][W][C], y [N][Ho][Wo][K]) on the three-stage
// and split paths: only the input and output transforms see the layout; V, M
// and the GEMMs are the same.  Input: by tile rows through LDS (k_vrows_nhwc)
// where C % 4 == 0, x is 16-byte aligned and a tile row fits; else per 16-tile
// block: 16-byte channel-quad loads (k_input_nhwc4) or, for other C or
// alignments, one wave per (16-tile block, channel quad), quads of a block
// consecutive, each lane loading its region of one channel (the 4 lanes of a
// tile read 16 contiguous bytes per pixel).  Output (three stages): one wave
// per (16-tile block, 16-filter block); a lane holds its tile's four
// consecutive filters, so every output pixel is one 16-byte store.
template <int MT>
__global__ __launch_bounds__(256) void k_input_nhwc(const float* __restrict__ x, float* __restrict__ V, Geom g,
                                                    long nwg, int nq) {
    constexpr int A = MT + 2, T = A * A;
    const int lane = threadIdx.x & 63;
    const long per = (nwg + 7) / 8, item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nwg) return;
    const long w = item * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * nq) return;
    // channel quad fastest: the waves reading one pixel's C channels run together;
    // nq quads per block in V (quads past CQ are zeros)
    const int pb = (int)(w / nq), cq = (int)(w % nq);
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const int c = cq * 4 + (lane >> 4);
    const bool ok = tc.valid && c < g.C;
    const float* xn = x + (size_t)tc.n * g.H * g.W * g.C + (ok ? c : 0);
    const int r0 = tc.ti * MT - g.pad, c0 = tc.tj * MT - g.pad;
    float d[A][A];
#pragma unroll
    for (int u = 0; u < A; ++u)
#pragma unroll
        for (int v = 0; v < A; ++v) {
            const int row = r0 + u, col = c0 + v;
            const bool in = ok && (unsigned)row < (unsigned)g.H && (unsigned)col < (unsigned)g.W;
            d[u][v] = in ? xn[((size_t)row * g.W + col) * g.C] : 0.0f;
        }
    float vv[T];
    input_tf<MT>(d, vv);
    store_t4<T, true>(V + ((size_t)pb * nq + cq) * T * 64, lane, vv);
}

// With C % 4 == 0 a channel quad of a pixel is one aligned 16-byte word: one
// wave per (16-tile block, group of four channel quads); lane q*16 + t loads,
// for every region pixel of tile t, the four channels of quad 4*cg + q in one
// 16-byte load (the four lanes of a tile read 64 contiguous bytes), then
// transforms the four channels one after another into their lane slots
// c%4*16 + t of that quad's V block.  Offsets are 32-bit from the first image
// the block touches (the host checks that they fit below kInvalid); pixels
// outside the image and quads past CQ read as zero.
template <int MT>
__global__ __launch_bounds__(256) void k_input_nhwc4(const float* __restrict__ x, float* __restrict__ V, Geom g,
                                                     int CG, long nwg, int nq) {
    constexpr int A = MT + 2, T = A * A;
    const int lane = threadIdx.x & 63;
    const long per = (nwg + 7) / 8, item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nwg) return;
    const long w = item * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * CG) return;
    // quad groups of a block consecutive: the waves reading a pixel's C channels run together
    const int pb = (int)(w / CG), cg = (int)(w % CG);
    const int t = lane & 15, cq = cg * 4 + (lane >> 4);
    const TileCoord tc = decode_tile(pb * 16 + t, g);
    const int n0 = __builtin_amdgcn_readfirstlane(min(pb * 16, g.P - 1) / (g.th * g.tw));
    const size_t img = (size_t)g.H * g.W * g.C;
    const size_t left = ((size_t)g.N - n0) * img * 4;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + (size_t)n0 * img), (short)0, (int)(left < kInvalid ? left : kInvalid), kRsrcWord3);
    const bool ok = tc.valid && cq < g.CQ;
    const uint32_t base = (uint32_t)(tc.n - n0) * (uint32_t)(img * 4) + (uint32_t)cq * 16u;
    const int r0 = tc.ti * MT - g.pad, c0 = tc.tj * MT - g.pad;
    f32x4 d4[A][A];
#pragma unroll
    for (int u = 0; u < A; ++u)
#pragma unroll
        for (int v = 0; v < A; ++v) {
            const int row = r0 + u, col = c0 + v;
            const bool in = ok && (unsigned)row < (unsigned)g.H && (unsigned)col < (unsigned)g.W;
            const uint32_t off = in ? base + ((uint32_t)row * g.W + (uint32_t)col) * (uint32_t)g.C * 4u : kInvalid;
            d4[u][v] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (int)off, 0, 0));
        }
    // nq quads per block in V: CQ (three stages) or CQ rounded up to 4 (the
    // split path's blocked V, whose padding quads get the zeros read above)
    if (cq >= nq) return;
    float* blk = V + ((size_t)pb * nq + cq) * T * 64;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        float d[A][A];
#pragma unroll
        for (int u = 0; u < A; ++u)
#pragma unroll
            for (int v = 0; v < A; ++v) d[u][v] = d4[u][v][e];
        float vv[T];
        input_tf<MT>(d, vv);
        store_t4<T, true>(blk, e * 16 + t, vv);
    }
}

// With C % 4 == 0 and room in LDS, by whole tile rows as k_vrows does: one
// workgroup per (R consecutive tile rows of the batch, group of QG = 2^lqg <= 4
// channel quads), the groups of one row range consecutive in the XCD-aware
// item order (they share x's cache lines).  A thread loads, for columns
// (c / QG) and quads (c % QG) of the chunks c = tid, tid + 256, ..., the
// 16-byte channel quads of every region row (a pixel's QG quads are one
// contiguous run, so a wave reads whole runs and each x byte once per tile
// row), and writes them to LDS as [r][A rows][pitch][QGP] floats: the pixel
// pitch QGP = 4*QG + 1 (m = 4) or + 2 (m = 2) puts the 16 tiles x 4 channels
// that a wave reads on distinct banks.  Wave w then transforms (block, quad)
// tasks w, w+4, ..., lane = (channel, tile), and stores each block's
// position groups as whole 1 KiB runs; a block that two row ranges share is
// completed by the other workgroup, and the batch's last partial block gets
// zeros past the last tile.  Quads past CQ (the split path's padding) read as
// zeros.  Offsets are 32-bit from the first image the rows touch (the host
// checks that they fit below kInvalid).  Plain stores: the blocks two
// workgroups share meet in L2 (streaming stores measured 1.7x slower).
template <int MT>
__global__ __launch_bounds__(256) void k_vrows_nhwc(const float* __restrict__ x, float* __restrict__ V, Geom g,
                                                    int R, int lqg, int QGP, int pitch, int nq, int nitems) {
    constexpr int A = MT + 2, T = A * A;
    extern __shared__ float4 xs4[];
    float* xs = (float*)xs4;
    const int QG = 1 << lqg;
    const int nrows = g.N * g.th;
    const int nqg = (nq + QG - 1) >> lqg;
    const int per = (nitems + 7) / 8, item = (int)(blockIdx.x % 8) * per + (int)(blockIdx.x / 8);
    if (item >= nitems) return;
    const int qg = item % nqg, gr0 = item / nqg * R;
    const int q0 = qg * QG, nqw = min(QG, nq - q0);     // this workgroup's quads [q0, q0 + nqw)
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n0 = gr0 / g.th;
    const size_t img = (size_t)g.H * g.W * g.C;
    const size_t left = ((size_t)g.N - n0) * img * 4;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(x + (size_t)n0 * img), (short)0, (int)(left < kInvalid ? left : kInvalid), kRsrcWord3);
    const uint32_t img_b = (uint32_t)(img * 4), row_b = (uint32_t)g.W * (uint32_t)g.C * 4u;
    for (int c = tid; c < pitch * QG; c += 256) {
        const int lc = c >> lqg, q = c & (QG - 1);
        const int col = lc - g.pad, cq = q0 + q;
        const bool cok = (unsigned)col < (unsigned)g.W && q < nqw && cq < g.CQ;
        const uint32_t coff = (uint32_t)col * (uint32_t)g.C * 4u + (uint32_t)cq * 16u;
        float* const lp = xs + lc * QGP + 4 * q;
        for (int r = 0; r < R; ++r) {
            const int gr = gr0 + r, n = gr / g.th, ti = gr - n * g.th;
            const bool rok = cok && gr < nrows;
            f32x4 v[A];
#pragma unroll
            for (int u = 0; u < A; ++u) {
                const int row = ti * MT - g.pad + u;
                const bool ok = rok && (unsigned)row < (unsigned)g.H;
                const uint32_t off = ok ? (uint32_t)(n - n0) * img_b + (uint32_t)row * row_b + coff : kInvalid;
                v[u] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(xr, (int)off, 0, 0));
            }
#pragma unroll
            for (int u = 0; u < A; ++u) {
                float* d = lp + (r * A + u) * pitch * QGP;
                d[0] = v[u][0];
                d[1] = v[u][1];
                d[2] = v[u][2];
                d[3] = v[u][3];
            }
        }
    }
    __syncthreads();
    const int l16 = lane & 15, cl = lane >> 4;
    const int t0 = gr0 * g.tw, t1 = min(gr0 + R, nrows) * g.tw;   // this workgroup's tiles [t0, t1)
    const int b0 = t0 >> 4, nblk = ((t1 - 1) >> 4) - b0 + 1;
    const size_t qstride = (size_t)nq * T * 64;                   // floats of one block
    const bool last_tail = t1 == g.P && (g.P & 15);               // the batch's last block is partial
    for (int task = wave; task < nblk * nqw; task += 4) {
        const int bi = task / nqw, q = task - bi * nqw;
        const int blk = b0 + bi, p = blk * 16 + l16;
        float* dst = V + (size_t)blk * qstride + (size_t)(q0 + q) * T * 64 + lane * 4;
        if (p >= t0 && p < t1) {
            const int pr = p / g.tw, r = pr - gr0, tj = p - pr * g.tw;
            const float* wp = xs + (r * A * pitch + tj * MT) * QGP + 4 * q + cl;
            float d[A][A];
#pragma unroll
            for (int u = 0; u < A; ++u)
#pragma unroll
                for (int v = 0; v < A; ++v) d[u][v] = wp[(u * pitch + v) * QGP];
            float vv[T];
            input_tf<MT>(d, vv);
#pragma unroll
            for (int g4 = 0; g4 < T / 4; ++g4)
                store_out<false>(dst + g4 * 256, vv[4 * g4], vv[4 * g4 + 1], vv[4 * g4 + 2], vv[4 * g4 + 3]);
        } else if (last_tail && p >= g.P) {
#pragma unroll
            for (int g4 = 0; g4 < T / 4; ++g4) store_out<false>(dst + g4 * 256, 0.f, 0.f, 0.f, 0.f);
        }
    }
}

template <int MT>
__global__ __launch_bounds__(256) void k_output_nhwc(const float* __restrict__ M, float* __restrict__ y, Geom g,
                                                     int relu, int vec_ok) {
    constexpr int T = (MT + 2) * (MT + 2);
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (long)g.PB * g.KB) return;
    const int kb = (int)(w % g.KB);
    const TileCoord tc = decode_tile((int)(w / g.KB) * 16 + (lane & 15), g);
    const float* src = M + ((size_t)w * T) * 256 + lane * 4;
    f32x4 mv[T];
#pragma unroll
    for (int t = 0; t < T; ++t) mv[t] = *(const f32x4*)(src + t * 256);
    float o[4][MT][MT];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float m1[T];
#pragma unroll
        for (int t = 0; t < T; ++t) m1[t] = mv[t][r];
        output_tf<MT>(m1, o[r]);
    }
    store_tile_nhwc<MT>(y, g, tc, kb * 16 + 4 * (lane >> 4), o, relu != 0, vec_ok != 0);
}

// ------------------------------------------------------------------ 1-D
// 1 x r (axis 1, along W) and r x 1 (axis 2, along H) layers: regions of 8
// inputs along the axis give m = 9 - r outputs; T = 8 transform positions, so
// the blocked U, V and M layouts are those of the 2-D path with T = 8, and the
// GEMM stage is k_gemm unchanged.

// One wave per (16-filter block, 4-channel quad); lane = (c%4)*16 + k%16.
template <int R>
__global__ __launch_bounds__(256) void k_filter1d(const float* __restrict__ gw, float* __restrict__ U, int C,
                                                  int K, int CQ, long nw) {
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= nw) return;
    const int kb = (int)(w / CQ), cq = (int)(w % CQ);
    const int k = kb * 16 + (lane & 15), c = cq * 4 + (lane >> 4);
    const bool ok = k < K && c < C;
    const float* src = gw + ((size_t)(ok ? k : 0) * C + (ok ? c : 0)) * R;
    float g[R];
#pragma unroll
    for (int j = 0; j < R; ++j) g[j] = ok ? src[j] : 0.0f;
    float u[8];
    filter_tf8<R>(g, u);
    store_t4<8, false>(U + (size_t)w * 8 * 64, lane, u);
}

// One wave per (16-tile block, 4-channel quad), XCD-contiguous runs as in
// k_input; lane = (tile p%16, channel c%4) loads its 8 inputs along the axis
// (zero outside the image, past C and past P) and writes B^T d.
template <int MT, int AX>
__global__ __launch_bounds__(256) void k_input1d(const float* __restrict__ x, float* __restrict__ V, Geom g,
                                                 long nwg) {
    const int lane = threadIdx.x & 63;
    const long per = (nwg + 7) / 8, item = (long)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (item >= nwg) return;
    const long w = item * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (w >= (long)g.PB * g.CQ) return;
    const int cq = (int)(w / g.PB), pb = (int)(w % g.PB);
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const int c = cq * 4 + (lane >> 4);
    const bool ok = tc.valid && c < g.C;
    const float* xc = x + ((size_t)tc.n * g.C + (ok ? c : 0)) * g.H * g.W;
    float d[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        int row, col;
        if constexpr (AX == 1) {
            row = tc.ti;
            col = tc.tj * MT - g.pad + u;
        } else {
            row = tc.ti * MT - g.pad + u;
            col = tc.tj;
        }
        const bool in = ok && (unsigned)row < (unsigned)g.H && (unsigned)col < (unsigned)g.W;
        d[u] = in ? xc[(size_t)row * g.W + col] : 0.0f;
    }
    float v[8];
    bt8(d, v);
    store_t4<8, true>(V + ((size_t)pb * g.CQ + cq) * 8 * 64, lane, v);
}

// One wave per (16-tile block, 16-filter block): lane = (tile p%16, filter
// quad); gathers the 8 values of its four (tile, filter) pairs, applies A^T
// and writes m outputs per filter along the axis.
template <int MT, int AX>
__global__ __launch_bounds__(256) void k_output1d(const float* __restrict__ M, float* __restrict__ y, Geom g,
                                                  int relu) {
    const int lane = threadIdx.x & 63;
    const long w = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= (long)g.PB * g.KB) return;
    const int pb = (int)(w / g.KB), kb = (int)(w % g.KB);
    const TileCoord tc = decode_tile(pb * 16 + (lane & 15), g);
    const float* src = M + ((size_t)w * 8) * 256 + lane * 4;
    f32x4 mv[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) mv[t] = *(const f32x4*)(src + t * 256);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int k = kb * 16 + 4 * (lane >> 4) + r;
        if (!tc.valid || k >= g.K) continue;
        float a[8], o[MT];
#pragma unroll
        for (int t = 0; t < 8; ++t) a[t] = mv[t][r];
        at8<MT>(a, o);
        float* yk = y + ((size_t)tc.n * g.K + k) * g.Ho * g.Wo;
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const float v = relu ? fmaxf(o[i], 0.0f) : o[i];
            if constexpr (AX == 1) {
                const int col = tc.tj * MT + i;
                if (col < g.Wo) yk[(size_t)tc.ti * g.Wo + col] = v;
            } else {
                const int row = tc.ti * MT + i;
                if (row < g.Ho) yk[(size_t)row * g.Wo + tc.tj] = v;
            }
        }
    }
}

hipError_t launch_filter_transform_1d(const float* gw, float* U, int C, int K, int m, int r, hipStream_t s) {
    const int CQ = (C + 3) / 4, KB = (K + 15) / 16;
    const long waves = (long)KB * CQ;
    if ((waves + 3) / 4 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
    (void)m;
    if (r == 3) hipLaunchKernelGGL(k_filter1d<3>, grid, block, 0, s, gw, U, C, K, CQ, waves);
    else if (r == 5) hipLaunchKernelGGL(k_filter1d<5>, grid, block, 0, s, gw, U, C, K, CQ, waves);
    else hipLaunchKernelGGL(k_filter1d<7>, grid, block, 0, s, gw, U, C, K, CQ, waves);
    return hipGetLastError();
}

static hipError_t launch_input_1d(const float* x, float* V, const Geom& g, hipStream_t s) {
    const long waves = (long)g.PB * g.CQ, nwg = (waves + 3) / 4;
    if ((nwg + 7) / 8 * 8 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((nwg + 7) / 8 * 8)), block(256);
#define WINO_IN1D(MT, AX) \
    if (g.m == MT && g.axis == AX) { hipLaunchKernelGGL((k_input1d<MT, AX>), grid, block, 0, s, x, V, g, nwg); return hipGetLastError(); }
    WINO_IN1D(6, 1) WINO_IN1D(4, 1) WINO_IN1D(2, 1) WINO_IN1D(6, 2) WINO_IN1D(4, 2) WINO_IN1D(2, 2)
#undef WINO_IN1D
    return hipErrorInvalidValue;
}

static hipError_t launch_output_1d(const float* M, float* y, const Geom& g, bool relu, hipStream_t s) {
    const long waves = (long)g.PB * g.KB;
    if ((waves + 3) / 4 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
#define WINO_OUT1D(MT, AX) \
    if (g.m == MT && g.axis == AX) { hipLaunchKernelGGL((k_output1d<MT, AX>), grid, block, 0, s, M, y, g, (int)relu); return hipGetLastError(); }
    WINO_OUT1D(6, 1) WINO_OUT1D(4, 1) WINO_OUT1D(2, 1) WINO_OUT1D(6, 2) WINO_OUT1D(4, 2) WINO_OUT1D(2, 2)
#undef WINO_OUT1D
    return hipErrorInvalidValue;
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


// Streaming (non-temporal) stores of y pay off once y outgrows one XCD's 4 MB
// L2 (measured: plain stores 2-6% slower at 6-13 MB of output, 10% slower at
// 205 MB); below that plain stores complete sooner (3-6% faster at 0.4-3 MB).
constexpr size_t kStreamStoreBytes = 4u << 20;
static inline int stream_stores(const Geom& g) {
    return (size_t)g.N * g.K * g.Ho * g.Wo * sizeof(float) > kStreamStoreBytes ? 1 : 0;
}
// The split path's GEMM kernel streams y only past half of the 256 MB
// last-level cache: below that, plain stores leave y there for the next
// layer and also finish sooner themselves (VGG-16 at N = 32: layers with
// 51-103 MB of output 2-9% faster per call, the stack 3%); at 205 MB streaming
// stays ahead (the 112x112 layers 3-6%, the channel-last N = 64 256-channel
// layer 2%).
constexpr size_t kSplitStreamBytes = 128u << 20;
static inline int split_stream_stores(const Geom& g) {
    return (size_t)g.N * g.K * g.Ho * g.Wo * sizeof(float) > kSplitStreamBytes ? 1 : 0;
}

hipError_t launch_filter_transform(const float* gw, float* U, int C, int K, int m, int r, hipStream_t s) {
    const int CQ = (C + 3) / 4, KB = (K + 15) / 16, TG = (m + r - 1) * (m + r - 1) / 4;
    const long pairs = (long)KB * CQ;
    const bool all = pairs >= kFilterAllPairs;     // enough waves without splitting the positions
    const bool stage = all && CQ % 4 == 0;         // a workgroup's quads share their filters
    const long waves = all ? pairs : pairs * TG;
    if ((waves + 3) / 4 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
#define WINO_FILTER_LAUNCH(MT, R)                                                                         \
    if (stage) hipLaunchKernelGGL((k_filter<MT, true, true, R>), grid, block, 0, s, gw, U, C, K, CQ, waves);  \
    else if (all) hipLaunchKernelGGL((k_filter<MT, true, false, R>), grid, block, 0, s, gw, U, C, K, CQ, waves); \
    else hipLaunchKernelGGL((k_filter<MT, false, false, R>), grid, block, 0, s, gw, U, C, K, CQ, waves);
    if (r == 5) {
        WINO_FILTER_LAUNCH(2, 5)
    } else if (m == 2) {
        WINO_FILTER_LAUNCH(2, 3)
    } else {
        WINO_FILTER_LAUNCH(4, 3)
    }
#undef WINO_FILTER_LAUNCH
    return hipGetLastError();
}

// Row-wise channel-last input transform: tile rows per workgroup, log2 of the
// quads per workgroup, LDS pixel pitch and row pitch (floats), dynamic LDS
// bytes; R = 0 where one tile row of at least one quad does not fit, or the
// images a row range spans do not fit the 32-bit load offsets.
struct NhwcRowsPlan {
    int R, lqg, QGP, pitch;
    size_t lds;
};
// Three workgroups per CU; at most 4 quads per workgroup (measured on the
// N=64 256-channel 56x56 layer: 8 quads and one tile row 12 us slower, and
// every larger LDS share slower still).
constexpr size_t kNhwcRowsLds = 52 << 10;

static NhwcRowsPlan nhwc_rows_plan(const Geom& g, int nq) {
    NhwcRowsPlan p{0, 0, 0, 0, 0};
    p.pitch = g.tw * g.m + 2;
    int lqg = 0;
    while (lqg < 2 && (1 << lqg) < nq) ++lqg;           // the quads a workgroup needs, at most 4
    size_t row_b = 0;
    for (; lqg >= 0; --lqg) {
        p.QGP = 4 * (1 << lqg) + (g.m == 4 ? 1 : 2);
        row_b = (size_t)g.A * p.pitch * p.QGP * sizeof(float);
        if (row_b <= kNhwcRowsLds) break;
    }
    if (lqg < 0) return p;
    int gcd = 16, t = g.tw;
    while (t) {
        const int r = gcd % t;
        gcd = t;
        t = r;
    }
    int R = 16 / gcd;
    while (R > 1 && (size_t)R * row_b > kNhwcRowsLds) --R;
    const size_t img_b = (size_t)g.C * g.H * g.W * sizeof(float);
    while (R > 1 && (size_t)(R / g.th + 2) * img_b >= (size_t)kInvalid) --R;
    if ((size_t)(R / g.th + 2) * img_b >= (size_t)kInvalid) return p;
    const long items = ((long)g.N * g.th + R - 1) / R * (((long)nq + (1 << lqg) - 1) >> lqg);
    if ((items + 7) / 8 * 8 > 0x7fffffffL) return p;
    p.R = R;
    p.lqg = lqg;
    p.lds = R * row_b;
    return p;
}

// Channel-last input transform into V blocks of nq quads ([PB][nq][T/4][64][4]:
// nq = CQ for the three stages, CQ rounded up to 4 for the split path).
static hipError_t launch_input_nhwc(const float* x, float* V, const Geom& g, int nq, hipStream_t s) {
    const dim3 block(256);
    if (g.C % 4 == 0 && aligned(x, 16)) {
        const NhwcRowsPlan rp = nhwc_rows_plan(g, nq);
        if (rp.R > 0) {
            const int nitems = (int)(((long)g.N * g.th + rp.R - 1) / rp.R * ((nq + (1 << rp.lqg) - 1) >> rp.lqg));
            const dim3 grid((unsigned)((nitems + 7) / 8 * 8));
            if (g.m == 2)
                hipLaunchKernelGGL(k_vrows_nhwc<2>, grid, block, rp.lds, s, x, V, g, rp.R, rp.lqg, rp.QGP, rp.pitch,
                                   nq, nitems);
            else
                hipLaunchKernelGGL(k_vrows_nhwc<4>, grid, block, rp.lds, s, x, V, g, rp.R, rp.lqg, rp.QGP, rp.pitch,
                                   nq, nitems);
            return hipGetLastError();
        }
    }
    const long waves = (long)g.PB * nq, nwg = (waves + 3) / 4;
    if ((nwg + 7) / 8 * 8 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((nwg + 7) / 8 * 8));
    // 16-byte channel-quad loads when the quads are aligned and the 32-bit
    // offsets of the images one tile block spans (at most 16 / (th*tw) + 2)
    // stay below kInvalid
    const size_t img_b = (size_t)g.H * g.W * g.C * 4;
    const size_t span = (size_t)(16 / (g.th * g.tw) + 2);
    if (g.C % 4 == 0 && aligned(x, 16) && span * img_b < (size_t)kInvalid) {
        const int CG = (nq + 3) / 4;
        const long nwg4 = ((long)g.PB * CG + 3) / 4;
        const dim3 grid4((unsigned)((nwg4 + 7) / 8 * 8));
        if (g.m == 2) hipLaunchKernelGGL(k_input_nhwc4<2>, grid4, block, 0, s, x, V, g, CG, nwg4, nq);
        else hipLaunchKernelGGL(k_input_nhwc4<4>, grid4, block, 0, s, x, V, g, CG, nwg4, nq);
    } else if (g.m == 2) {
        hipLaunchKernelGGL(k_input_nhwc<2>, grid, block, 0, s, x, V, g, nwg, nq);
    } else {
        hipLaunchKernelGGL(k_input_nhwc<4>, grid, block, 0, s, x, V, g, nwg, nq);
    }
    return hipGetLastError();
}

hipError_t launch_input_transform(const float* x, float* V, const Geom& g, hipStream_t s) {
    if (g.axis != 0) return launch_input_1d(x, V, g, s);
    if (g.nhwc) return launch_input_nhwc(x, V, g, g.CQ, s);
    const long waves = (long)g.PB * g.CQ, nwg = (waves + 3) / 4;
    if ((nwg + 7) / 8 * 8 > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)((nwg + 7) / 8 * 8)), block(256);
    if (g.r == 3) {
        // by whole tile rows where the rows' patches fit LDS (the split path's kernel)
        const int vec = g.W % 4 == 0 && aligned(x, 16);
        const VrowsPlan vp = vrows_plan(g, vec);
        if (vp.R > 0) {
            const long ngr = ((long)g.N * g.th + vp.R - 1) / vp.R;
            const dim3 gr((unsigned)(ngr * g.CQ)), b256(256);
            if (g.m == 2) hipLaunchKernelGGL((k_vrows<2>), gr, b256, vp.lds, s, x, V, g, vp.R, vp.pitch, g.CQ);
            else hipLaunchKernelGGL((k_vrows<4>), gr, b256, vp.lds, s, x, V, g, vp.R, vp.pitch, g.CQ);
            return hipGetLastError();
        }
    }
    if (g.r == 5)
        hipLaunchKernelGGL((k_input<2, 5>), grid, block, 0, s, x, V, g, nwg);
    else if (g.m == 2)
        hipLaunchKernelGGL(k_input<2>, grid, block, 0, s, x, V, g, nwg);
    else
        hipLaunchKernelGGL(k_input<4>, grid, block, 0, s, x, V, g, nwg);
    return hipGetLastError();
}

hipError_t launch_batched_gemm(const float* U, const float* V, float* M, const Geom& g, hipStream_t s) {
    if ((size_t)4 * g.CQ * (g.T / 4) * 1024 >= (size_t)kInvalid) return hipErrorInvalidConfiguration;   // 32-bit offsets
    // 32 x 64 tiles when 64 x 64 ones would give the CUs fewer than four workgroups each
    const long items4 = (long)((g.PB + 3) / 4) * ((g.KB + 3) / 4) * (g.T / 4);
    const int kt = items4 < 4 * 256 ? 2 : 4;
    const long nitems = (long)((g.PB + 3) / 4) * ((g.KB + kt - 1) / kt) * (g.T / 4);
    const long wgs = (nitems + 7) / 8 * 8;
    if (wgs > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)wgs), block(256);
    if (kt == 2) hipLaunchKernelGGL(k_gemm<2>, grid, block, 0, s, U, V, M, g);
    else hipLaunchKernelGGL(k_gemm<4>, grid, block, 0, s, U, V, M, g);
    return hipGetLastError();
}

hipError_t launch_output_transform(const float* M, float* y, const Geom& g, bool relu, hipStream_t s) {
    if (g.axis != 0) return launch_output_1d(M, y, g, relu, s);
    if (g.nhwc) {
        const long waves = (long)g.PB * g.KB;
        if ((waves + 3) / 4 > 0x7fffffffL) return hipErrorInvalidConfiguration;
        const dim3 grid((unsigned)((waves + 3) / 4)), block(256);
        const int vk = (g.K % 4 == 0) && aligned(y, 16);
        if (g.m == 2) hipLaunchKernelGGL(k_output_nhwc<2>, grid, block, 0, s, M, y, g, (int)relu, vk);
        else hipLaunchKernelGGL(k_output_nhwc<4>, grid, block, 0, s, M, y, g, (int)relu, vk);
        return hipGetLastError();
    }
    const int vec_ok = (g.Wo % g.m == 0) && aligned(y, 4 * g.m);
    int R = 0, segs = 0, ipi;                      // items per image
    if (g.tw <= 64) {
        R = 64 / g.tw;
        ipi = (g.th + R - 1) / R;
    } else {
        segs = (g.tw + 63) / 64;
        ipi = g.th * segs;
    }
    const long nitems = (long)g.N * ipi, wgs = nitems * g.KB;
    if (wgs > 0x7fffffffL) return hipErrorInvalidConfiguration;
    const dim3 grid((unsigned)wgs), block(256);
    if (g.r == 5)
        hipLaunchKernelGGL((k_output<2, 5>), grid, block, 0, s, M, y, g, (int)relu, vec_ok, R, segs, ipi,
                           (int)nitems);
    else if (g.m == 2)
        hipLaunchKernelGGL(k_output<2>, grid, block, 0, s, M, y, g, (int)relu, vec_ok, R, segs, ipi, (int)nitems);
    else
        hipLaunchKernelGGL(k_output<4>, grid, block, 0, s, M, y, g, (int)relu, vec_ok, R, segs, ipi, (int)nitems);
    return hipGetLastError();
}

constexpr int kMaxLdsBytes = 160 * 1024;

static FastDiv make_fastdiv(uint32_t d) {
    FastDiv f;
    f.l = 0;
    while ((1ull << f.l) < d) ++f.l;
    f.m = (uint32_t)(((1ull << 32) * ((1ull << f.l) - d)) / d + 1);
    return f;
}

// The fused kernel's epilogue addresses its four LDS objects as one packed
// range: check once per instance that the compiled allocation is exactly their
// total (no padding between them) before its first launch outside a stream
// capture (the query is not made while a capture is being recorded).
template <int MT, int TS, int CS, int BW, int VEC, int R>
static hipError_t fused_lds_check(hipStream_t s) {
    static std::atomic<int> state{0};             // 0 unchecked, 1 checked, 2 mismatch
    const int st = state.load(std::memory_order_acquire);
    if (st) return st == 1 ? hipSuccess : hipErrorInvalidKernelFile;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone) return hipSuccess;
    hipFuncAttributes a;
    const hipError_t e = hipFuncGetAttributes(&a, reinterpret_cast<const void*>(&k_fused<MT, TS, CS, BW, VEC, R>));
    if (e != hipSuccess) return e;
    const bool ok = a.sharedSizeBytes == (size_t)FusedShape<MT, TS, CS, BW, VEC, R>::LDS_BYTES;
    state.store(ok ? 1 : 2, std::memory_order_release);
    return ok ? hipSuccess : hipErrorInvalidKernelFile;
}

// y[i] = max?(sum over slices s = 0, 1, ... of part[s][i]), in that order.
__global__ __launch_bounds__(256) void k_slice_sum(const float* __restrict__ part, float* __restrict__ y,
                                                   long long count, int nsl, int relu) {
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= count) return;
    float v = part[i];
    for (int k = 1; k < nsl; ++k) v += part[(size_t)k * (size_t)count + (size_t)i];
    y[i] = relu ? fmaxf(v, 0.0f) : v;
}

int slice_quads(const Geom& g, int nsl) { return (g.CQ + nsl - 1) / nsl; }
int slices_used(const Geom& g, int nsl) {
    const int q = slice_quads(g, nsl);
    return (g.CQ + q - 1) / q;
}

template <int MT, int TS, int CS, int BW, int R = 3>
static hipError_t fused_instance(const float* x, const float* U, float* y, const Geom& g, bool relu,
                                 hipStream_t s, int nsl_req, float* part) {
    using S = FusedShape<MT, TS, CS, BW, 0, R>;
    FusedTiling ft{};
    ft.nbh = (g.th + S::BH - 1) / S::BH;
    ft.nbw = (g.tw + BW - 1) / BW;
    ft.nt = g.N * ft.nbh * ft.nbw;
    ft.nkg = (g.KB + S::KGW - 1) / S::KGW;
    ft.nsl = part && nsl_req > 1 ? slices_used(g, nsl_req) : 1;
    ft.qsl = ft.nsl > 1 ? slice_quads(g, nsl_req) : g.CQ;
    ft.ysz = (long long)g.N * g.K * g.Ho * g.Wo;
    ft.d_sl = make_fastdiv((uint32_t)(ft.nt * ft.nkg));
    ft.per = (int)(((long)ft.nt * ft.nkg * ft.nsl + 7) / 8);
    ft.nsteps = (g.CQ + S::QS - 1) / S::QS;
    // Item order: estimate the bytes an XCD fetches past its L2 for each order,
    // with one workgroup per CU (32 per XCD) resident at a time.  Filter-group
    // major: every group re-reads the whole input; tile major: every resident
    // set of 32 items re-reads the filters of all its groups.
    {
        const double xb = 4.0 * g.N * g.C * g.H * g.W, ub = 4.0 * g.T * g.CQ * 4 * g.KB * 16;
        const double sets = (double)ft.nt * ft.nkg / 32.0;
        const double group_major = xb * ft.nkg + ub * sets / ft.nkg;
        const double tile_major = xb + ub * sets * (ft.nkg < 32 ? 1.0 : 32.0 / ft.nkg);
        ft.kfast = tile_major < group_major ? 1 : 0;
    }
    ft.d_item = make_fastdiv((uint32_t)(ft.kfast ? ft.nkg : ft.nt));
    ft.d_img = make_fastdiv((uint32_t)(ft.nbh * ft.nbw));
    ft.d_nbw = make_fastdiv((uint32_t)ft.nbw);
    const dim3 grid((unsigned)(8 * ft.per)), block(512);
    float* const pp = ft.nsl > 1 ? part : nullptr;
    const int vec_ok = (g.Wo % MT == 0) && aligned(y, 4 * MT) && (!pp || aligned(pp, 4 * MT));
    // Partial outputs are read back at once: plain stores keep them in L2.
    const int nts = pp ? 0 : stream_stores(g);
    auto finish = [&]() -> hipError_t {
        hipError_t e = hipGetLastError();
        if (e != hipSuccess || !pp) return e;
        const long long cnt = ft.ysz;
        hipLaunchKernelGGL(k_slice_sum, dim3((unsigned)((cnt + 255) / 256)), dim3(256), 0, s, pp, y, cnt, ft.nsl,
                           (int)relu);
        return hipGetLastError();
    };
    // 16-byte patch loads need rows of whole chunks and an aligned image base,
    // and the variant's larger stages must fit in LDS.
    if constexpr (FusedShape<MT, TS, CS, BW, 1, R>::LDS_BYTES <= kMaxLdsBytes) {
        if (g.W % 4 == 0 && aligned(x, 16)) {
            const hipError_t e = fused_lds_check<MT, TS, CS, BW, 1, R>(s);
            if (e != hipSuccess) return e;
            hipLaunchKernelGGL((k_fused<MT, TS, CS, BW, 1, R>), grid, block, 0, s, x, U, y, g, ft, (int)relu, vec_ok,
                               nts, pp);
            return finish();
        }
    }
    const hipError_t e = fused_lds_check<MT, TS, CS, BW, 0, R>(s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((k_fused<MT, TS, CS, BW, 0, R>), grid, block, 0, s, x, U, y, g, ft, (int)relu, vec_ok,
                       nts, pp);
    return finish();
}

hipError_t launch_fused(const float* x, const float* U, float* y, const Geom& g, FusedCfg c, bool relu,
                        hipStream_t s, float* part) {
    // 3x3, m = 2: all 16 positions per wave; m = 4 and 5x5 (alpha = 6): two
    // row groups of 18 positions.
    if (g.r == 5) {
#define WINO_FUSED_R5(CS, BW) \
    if (g.m == 2 && c.csplit == CS && c.bw == BW) return fused_instance<2, 2, CS, BW, 5>(x, U, y, g, relu, s, c.nsl, part);
        WINO_FUSED_R5(1, 16)
        WINO_FUSED_R5(2, 16)
        WINO_FUSED_R5(4, 16)
        WINO_FUSED_R5(1, 4)
        WINO_FUSED_R5(2, 4)
        WINO_FUSED_R5(4, 4)
#undef WINO_FUSED_R5
        return hipErrorInvalidValue;
    }
    if (g.r != 3) return hipErrorInvalidValue;
#define WINO_FUSED_CASE(MT, TS, CS, BW) \
    if (g.m == MT && c.csplit == CS && c.bw == BW) return fused_instance<MT, TS, CS, BW>(x, U, y, g, relu, s, c.nsl, part);
    WINO_FUSED_CASE(2, 1, 1, 16)
    WINO_FUSED_CASE(2, 1, 2, 16)
    WINO_FUSED_CASE(2, 1, 4, 16)
    WINO_FUSED_CASE(2, 1, 8, 16)
    WINO_FUSED_CASE(2, 1, 1, 4)
    WINO_FUSED_CASE(2, 1, 2, 4)
    WINO_FUSED_CASE(2, 1, 4, 4)
    WINO_FUSED_CASE(2, 1, 8, 4)
    WINO_FUSED_CASE(4, 2, 1, 16)
    WINO_FUSED_CASE(4, 2, 2, 16)
    WINO_FUSED_CASE(4, 2, 4, 16)
    WINO_FUSED_CASE(4, 2, 1, 4)
    WINO_FUSED_CASE(4, 2, 2, 4)
    WINO_FUSED_CASE(4, 2, 4, 4)
#undef WINO_FUSED_CASE
    return hipErrorInvalidValue;
}

// Tile blocks of the split path's workspace for block width bw.
long split_blocks(const Geom& g) { return ((long)g.P + 15) / 16; }
size_t vblk_elems(const Geom& g) { return (size_t)split_blocks(g) * ((g.CQ + 3) / 4 * 4) * g.T * 64; }

// Rows per workgroup of the row-wise input transform: R*tw a multiple of
// 16 (whole blocks) where that fits 64 KB of LDS, else fewer; R = 0 (the
// patch kernel) when one tile row's patch does not fit, or the images a row
// range spans do not fit the 32-bit load offsets.
VrowsPlan vrows_plan(const Geom& g, int vec) {
    VrowsPlan p{0, 0, 0};
    // Rows whose width is not a multiple of 4 floats (or an unaligned x) would
    // come in by 4-byte DMA, one float per lane: the per-block and per-region
    // kernels are faster there (VGG-16's 14x14 layers at N = 32: 20 -> 14 us;
    // 26-57 pixel wide layers: 7-12% of the split call, 4-13% of the staged one).
    if (!vec) return p;
    const int xsh = (4 - g.pad % 4) % 4;
    p.pitch = (xsh + g.tw * g.m + 2 + 3) / 4 * 4;
    const size_t row_b = (size_t)4 * g.A * p.pitch * sizeof(float);    // one tile row, 4 channels
    int gcd = 16, t = g.tw;
    while (t) {
        const int r = gcd % t;
        gcd = t;
        t = r;
    }
    int R = 16 / gcd;
    while (R > 1 && (size_t)R * row_b > kVrowsLds) --R;
    const size_t img_b = (size_t)g.C * g.H * g.W * sizeof(float);
    while (R > 1 && (size_t)(R / g.th + 2) * img_b >= (size_t)kInvalid) --R;
    if ((size_t)R * row_b > kVrowsLds || (size_t)(R / g.th + 2) * img_b >= (size_t)kInvalid) return p;
    p.R = R;
    p.lds = R * row_b + 16;
    return p;
}

SplitTail split_tail(const Geom& g) {
    const int kgw = g.m == 4 ? GoShape<4>::KGW : GoShape<2>::KGW;
    SplitTail t;
    t.items = (split_blocks(g) + 1) / 2 * ((g.KB + kgw - 1) / kgw);
    const long rem = t.items % kSplitCus;
    t.units = 2 * kgw;
    t.tail = (t.items > kSplitCus && rem > 0 && rem * t.units <= kSplitCus) ? rem : 0;
    return t;
}

template <int MT, int BW>
static hipError_t split_instance(const float* x, const float* U, float* y, float* Vb, const Geom& g, bool relu,
                                 hipStream_t s) {
    using GS = GoShape<MT>;
    FusedTiling ft{};
    ft.bw = BW;
    ft.nbh = (g.th + 16 / BW - 1) / (16 / BW);
    ft.nbw = (g.tw + BW - 1) / BW;
    const int ntb = g.N * ft.nbh * ft.nbw;      // 16-tile patches of the input transform
    const int nb = (int)split_blocks(g);        // 16-tile blocks of Vb and the GEMMs
    const int ncq4 = (g.CQ + 3) / 4;
    if (g.nhwc) {
        // channel-last x: the three stages' input transform, into blocks of CQ4 quads
        const hipError_t e = launch_input_nhwc(x, Vb, g, 4 * ncq4, s);
        if (e != hipSuccess) return e;
    } else {
        const int vec = g.W % 4 == 0 && aligned(x, 16);
        const VrowsPlan vp = vrows_plan(g, vec);
        if (vp.R > 0) {
            const long ngr = ((long)g.N * g.th + vp.R - 1) / vp.R;
            const dim3 grid((unsigned)(ngr * ncq4 * 4)), block(256);
            hipLaunchKernelGGL((k_vrows<MT>), grid, block, vp.lds, s, x, Vb, g, vp.R, vp.pitch, 4 * ncq4);
        } else {
            const dim3 grid((unsigned)((long)ntb * ncq4)), block(256);
            if (vec) hipLaunchKernelGGL((k_vblk<MT, BW, 1>), grid, block, 0, s, x, Vb, g, ft.nbh, ft.nbw, ncq4);
            else hipLaunchKernelGGL((k_vblk<MT, BW, 0>), grid, block, 0, s, x, Vb, g, ft.nbh, ft.nbw, ncq4);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const SplitTail st = split_tail(g);
    ft.nt = (nb + 1) / 2;
    ft.nkg = (g.KB + GS::KGW - 1) / GS::KGW;
    ft.per = (int)(((long)ft.nt * ft.nkg - st.tail + 7) / 8);
    ft.nsteps = (g.CQ + GS::NQ - 1) / GS::NQ;
    {   // item order: V of a tile pair is read by every filter group
        const double vb = 4.0 * vblk_elems(g), ub = 4.0 * g.T * g.CQ * 4 * g.KB * 16;
        const double sets = (double)ft.nt * ft.nkg / 32.0;
        const double group_major = vb * ft.nkg + ub * sets / ft.nkg;
        const double tile_major = vb + ub * sets * (ft.nkg < 32 ? 1.0 : 32.0 / ft.nkg);
        ft.kfast = tile_major < group_major ? 1 : 0;
    }
    const dim3 grid((unsigned)(8 * ft.per + st.tail * st.units)), block(512);
    // 16-byte output stores: whole m-wide rows (NCHW) or four channels of a pixel (NHWC)
    const int vec_ok = g.nhwc ? (g.K % 4 == 0 && aligned(y, 16)) : ((g.Wo % MT == 0) && aligned(y, 4 * MT));
    hipLaunchKernelGGL((k_gemm_out<MT>), grid, block, 0, s, Vb, U, y, g, ft, nb, (int)relu, vec_ok,
                       split_stream_stores(g), (int)st.tail);
    return hipGetLastError();
}

// The split path on 16-bit operands: the input transform into VH blocks of
// 2*C32 groups (by tile rows, or per 16-tile block for very wide images), then
// the GEMMs + output transform on 16-bit MFMAs (the last items as units, as
// for fp32).
template <int MT, int PREC>
static hipError_t split16_instance(const float* x, const void* UH, float* y, void* VH, const Geom& g, bool relu,
                                   hipStream_t s) {
    using GS = GoShape<MT>;
    const int c32 = (g.C + 31) / 32, c16p = 2 * c32;
    const int vec = g.W % 4 == 0 && aligned(x, 16);
    const VrowsPlan vp = vrows_plan(g, vec);
    if (vp.R > 0) {
        const long ngr = ((long)g.N * g.th + vp.R - 1) / vp.R;
        const dim3 gr((unsigned)(ngr * 4 * c16p)), b256(256);
        hipLaunchKernelGGL((k_vrows<MT, PREC>), gr, b256, vp.lds, s, x, (float*)VH, g, vp.R, vp.pitch, 4 * c16p);
    } else {
        const long waves = (long)g.PB * c16p, nwg = (waves + 3) / 4;
        if ((nwg + 7) / 8 * 8 > 0x7fffffffL) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL((k_input16<MT, PREC>), dim3((unsigned)((nwg + 7) / 8 * 8)), dim3(256), 0, s, x,
                           (uint2*)VH, g, c16p, nwg);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    FusedTiling ft{};
    const int nb = (int)split_blocks(g);
    const SplitTail st = split_tail(g);
    ft.nt = (nb + 1) / 2;
    ft.nkg = (g.KB + GS::KGW - 1) / GS::KGW;
    ft.per = (int)(((long)ft.nt * ft.nkg - st.tail + 7) / 8);
    ft.nsteps = c32;
    {   // item order: V of a tile pair is read by every filter group
        const double vb = 1024.0 * nb * c32 * g.T, ub = 1024.0 * g.T * c32 * g.KB;
        const double sets = (double)ft.nt * ft.nkg / 32.0;
        const double group_major = vb * ft.nkg + ub * sets / ft.nkg;
        const double tile_major = vb + ub * sets * (ft.nkg < 32 ? 1.0 : 32.0 / ft.nkg);
        ft.kfast = tile_major < group_major ? 1 : 0;
    }
    const dim3 grid((unsigned)(8 * ft.per + st.tail * st.units)), block(512);
    const int vec_ok = (g.Wo % MT == 0) && aligned(y, 4 * MT);
    hipLaunchKernelGGL((k_gemm_out<MT, PREC>), grid, block, 0, s, (const float*)VH, (const float*)UH, y, g, ft, nb,
                       (int)relu, vec_ok, split_stream_stores(g), (int)st.tail);
    return hipGetLastError();
}

hipError_t launch_split16(const float* x, const void* UH, float* y, void* VH, const Geom& g, int prec, bool relu,
                          hipStream_t s) {
    if (g.m == 2) return prec == 1 ? split16_instance<2, 1>(x, UH, y, VH, g, relu, s)
                                   : split16_instance<2, 2>(x, UH, y, VH, g, relu, s);
    return prec == 1 ? split16_instance<4, 1>(x, UH, y, VH, g, relu, s)
                     : split16_instance<4, 2>(x, UH, y, VH, g, relu, s);
}

hipError_t launch_split(const float* x, const float* U, float* y, float* Vb, const Geom& g, int bw, bool relu,
                        hipStream_t s) {
    if (g.m == 2) return bw == 16 ? split_instance<2, 16>(x, U, y, Vb, g, relu, s)
                                  : split_instance<2, 4>(x, U, y, Vb, g, relu, s);
    return bw == 16 ? split_instance<4, 16>(x, U, y, Vb, g, relu, s) : split_instance<4, 4>(x, U, y, Vb, g, relu, s);
}

// Low-C path: tile groups of 256 x filter ranges; the filters are split so the
// launch has at least ~512 workgroups when the layer has few tiles.
hipError_t launch_lowc(const float* x, const float* U, float* y, const Geom& g, bool relu, hipStream_t s) {
    const int ntg = (g.P + 255) / 256;
    int ks = 1;
    while (ks * 2 <= (g.K + 3) / 4 && (long)ntg * ks < 512) ks *= 2;
    int kpw = (g.K + ks - 1) / ks;
    if (kpw > 64) kpw = 64;                            // LDS: kpw*NC*T floats
    ks = (g.K + kpw - 1) / kpw;
    const dim3 grid((unsigned)((long)ntg * ks)), block(256);
    const int vec_ok = (g.Wo % g.m == 0) && aligned(y, 4 * g.m);
    const size_t lds = (size_t)kpw * g.C * g.T * sizeof(float);
    const int nts = stream_stores(g);
#define WINO_LOWC_CASE(MT, NC) \
    if (g.m == MT && g.C == NC) { \
        if (relu) hipLaunchKernelGGL((k_lowc<MT, NC, true>), grid, block, lds, s, x, U, y, g, ntg, kpw, vec_ok, nts); \
        else hipLaunchKernelGGL((k_lowc<MT, NC, false>), grid, block, lds, s, x, U, y, g, ntg, kpw, vec_ok, nts); \
        return hipGetLastError(); \
    }
    WINO_LOWC_CASE(2, 1) WINO_LOWC_CASE(2, 2) WINO_LOWC_CASE(2, 3) WINO_LOWC_CASE(2, 4)
    WINO_LOWC_CASE(4, 1) WINO_LOWC_CASE(4, 2) WINO_LOWC_CASE(4, 3) WINO_LOWC_CASE(4, 4)
#undef WINO_LOWC_CASE
    return hipErrorInvalidValue;
}

hipError_t launch_maxpool2x2(const float* x, float* y, int N, int C, int H, int W, hipStream_t s) {
    const int Ho = H / 2, Wo = W / 2;
    const long total = (long)N * C * Ho * Wo;
    const dim3 grid((unsigned)((total + 255) / 256)), block(256);
    hipLaunchKernelGGL(k_maxpool2x2, grid, block, 0, s, x, y, total, H, W, Ho, Wo);
    return hipGetLastError();
}

// ------------------------------------------------------------------ peak probe
// The fp32 matrix-core rate this chip sustains: every wave runs eight
// independent chains of v_mfma_f32_16x16x4_f32 (enough to cover the
// instruction's latency) on operands of 1.0, so each accumulator element ends
// at exactly 4 * iters.  Lane 0 of each wave writes the sum of its chains'
// first elements (32 * iters) to out[wave].
__global__ __launch_bounds__(256) void k_mfma_probe(int iters, float* __restrict__ out) {
    f32x4 acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float one = 1.0f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(one, one, acc[j], 0, 0, 0);
    }
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += acc[j][0];
    if ((threadIdx.x & 63) == 0) out[blockIdx.x * 4 + (threadIdx.x >> 6)] = sum;
}

hipError_t launch_mfma_probe(int iters, float* out, hipStream_t s) {
    hipLaunchKernelGGL(k_mfma_probe, dim3(kProbeWaves / 4), dim3(256), 0, s, iters, out);
    return hipGetLastError();
}

// ---- scratch of the allocation-free entry point ---------------------------
// One array per GPU the library runs on, resident until the process ends.  In
// host code `scratch` names a host-side stand-in, not device memory: its
// device address comes from hipGetSymbolAddress, once per device with that
// device current, and only that address is ever passed on.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;

hipError_t noalloc_scratch(void** out) {
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    static std::mutex mu;
    static void* addr[kMaxDevices];
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = addr[dev];
    return hipSuccess;
}

size_t filter_elems(int C, int K, int m, int r) {
    const size_t T = (size_t)(m + r - 1) * (m + r - 1);
    return T * (size_t)((C + 3) / 4) * 4 * (size_t)((K + 15) / 16) * 16;
}
size_t v_elems(const Geom& g) { return (size_t)g.PB * g.CQ * g.T * 64; }
size_t m_elems(const Geom& g) { return (size_t)g.PB * g.KB * g.T * 256; }

}  // namespace wino
