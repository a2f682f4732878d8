// C-ABI of libwino: argument validation, layer planning and dispatch.
// Every check runs before the first HIP call, so invalid calls enqueue nothing.
#include "../../include/wino.h"
#include "wino_internal.h"

#include <stdint.h>

using namespace wino;

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 40;      // per tensor, well inside size_t
constexpr int64_t kMaxTiles = ((int64_t)1 << 31) - 64;

constexpr unsigned kBlockMask = WINO_BLOCK_1x16 | WINO_BLOCK_4x4, kCsplitShift = 16, kSliceShift = 20;
constexpr unsigned kKnownFlags =
    WINO_FLAG_RELU | WINO_PREC_MASK | WINO_ALGO_MASK | kBlockMask | (0xFu << kCsplitShift) | (0xFu << kSliceShift);

// 16-bit GEMM operand format from the flags: 0 (fp32), 1 (fp16), 2 (bf16), -1 (invalid).
int prec_of(unsigned flags) {
    const unsigned p = flags & WINO_PREC_MASK;
    return p == 0 ? 0 : p == WINO_PREC_F16 ? 1 : p == WINO_PREC_BF16 ? 2 : -1;
}

// 16-bit operands: 32-channel chunks, 1 KB per (block, chunk, position).
size_t c32_elems(const Geom& g) { return (size_t)(g.C + 31) / 32; }
size_t vh_bytes(const Geom& g) { return (size_t)g.PB * c32_elems(g) * g.T * 1024; }

// Checked product of non-negative int64 values; false on overflow past kMaxElems.
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > kMaxElems / a) return false;
    *out = a * b;
    return *out <= kMaxElems;
}

// Supported (m, r): F(2x2,3x3), F(4x4,3x3), F(2x2,5x5).
bool supported(int m, int r) { return (r == 3 && (m == 2 || m == 4)) || (r == 5 && m == 2); }

int make_geom_r(int N, int C, int H, int W, int K, int pad, int m, int r, Geom* g) {
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || pad < 0) return WINO_ERR_INVALID_ARG;
    if (!supported(m, r)) return WINO_ERR_UNSUPPORTED;
    const int64_t Ho = (int64_t)H + 2 * (int64_t)pad - (r - 1);
    const int64_t Wo = (int64_t)W + 2 * (int64_t)pad - (r - 1);
    if (Ho < 1 || Wo < 1 || Ho > INT32_MAX / 2 || Wo > INT32_MAX / 2) return WINO_ERR_INVALID_ARG;
    const int64_t th = (Ho + m - 1) / m, tw = (Wo + m - 1) / m;
    int64_t t1, P, xin, xout;
    if (!mul_ok(th, tw, &t1) || !mul_ok(t1, N, &P) || P > kMaxTiles) return WINO_ERR_INVALID_ARG;
    if (!mul_ok((int64_t)N * C, (int64_t)H * W, &xin)) return WINO_ERR_INVALID_ARG;
    if (!mul_ok((int64_t)N * K, Ho * Wo, &xout)) return WINO_ERR_INVALID_ARG;
    const int64_t A = m + r - 1, T = A * A;
    const int64_t CQ = (C + 3) / 4, KB = (K + 15) / 16, PB = (P + 15) / 16;
    int64_t v, mm;
    if (!mul_ok(PB * CQ, T * 64, &v) || !mul_ok(PB * KB, T * 256, &mm)) return WINO_ERR_INVALID_ARG;
    g->N = N; g->C = C; g->H = H; g->W = W; g->K = K; g->pad = pad; g->m = m;
    g->Ho = (int)Ho; g->Wo = (int)Wo; g->th = (int)th; g->tw = (int)tw; g->P = (int)P;
    g->A = (int)A; g->T = (int)T; g->r = r; g->axis = 0; g->nhwc = 0;
    g->CQ = (int)CQ; g->KB = (int)KB; g->PB = (int)PB;
    return WINO_OK;
}

int make_geom(int N, int C, int H, int W, int K, int pad, int m, Geom* g) {
    return make_geom_r(N, C, H, W, K, pad, m, 3, g);
}

// 1-D layers: (m, r) in {(6,3), (4,5), (2,7)}, alpha = 8; padding along the
// filtered axis only; tiles 1 x m (along W) or m x 1 (along H).
bool supported_1d(int m, int r) { return (m == 6 && r == 3) || (m == 4 && r == 5) || (m == 2 && r == 7); }

int make_geom_1d(int N, int C, int H, int W, int K, int pad, int m, int r, int axis, Geom* g) {
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || pad < 0) return WINO_ERR_INVALID_ARG;
    if (!supported_1d(m, r) || (axis != WINO_AXIS_W && axis != WINO_AXIS_H)) return WINO_ERR_UNSUPPORTED;
    const bool aw = axis == WINO_AXIS_W;
    const int64_t L = (aw ? W : H) + 2 * (int64_t)pad - (r - 1);
    if (L < 1 || L > INT32_MAX / 2) return WINO_ERR_INVALID_ARG;
    const int64_t Ho = aw ? H : L, Wo = aw ? L : W;
    const int64_t th = aw ? Ho : (Ho + m - 1) / m, tw = aw ? (Wo + m - 1) / m : Wo;
    int64_t t1, P, xin, xout;
    if (!mul_ok(th, tw, &t1) || !mul_ok(t1, N, &P) || P > kMaxTiles) return WINO_ERR_INVALID_ARG;
    if (!mul_ok((int64_t)N * C, (int64_t)H * W, &xin)) return WINO_ERR_INVALID_ARG;
    if (!mul_ok((int64_t)N * K, Ho * Wo, &xout)) return WINO_ERR_INVALID_ARG;
    const int64_t CQ = (C + 3) / 4, KB = (K + 15) / 16, PB = (P + 15) / 16;
    int64_t v, mm;
    if (!mul_ok(PB * CQ, 8 * 64, &v) || !mul_ok(PB * KB, 8 * 256, &mm)) return WINO_ERR_INVALID_ARG;
    g->N = N; g->C = C; g->H = H; g->W = W; g->K = K; g->pad = pad; g->m = m;
    g->Ho = (int)Ho; g->Wo = (int)Wo; g->th = (int)th; g->tw = (int)tw; g->P = (int)P;
    g->A = 8; g->T = 8; g->r = r; g->axis = axis; g->nhwc = 0;
    g->CQ = (int)CQ; g->KB = (int)KB; g->PB = (int)PB;
    return WINO_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Plan: which algorithm, and which fused-kernel variant.
struct Plan {
    unsigned algo;        // WINO_ALGO_FUSED, WINO_ALGO_SPLIT or WINO_ALGO_STAGED
    bool automatic;       // chosen by the planner (split falls back to fused without workspace)
    FusedCfg cfg;
};

// Row groups per unit of the fused kernel: alpha = 4 (F(2x2,3x3)) keeps all
// 16 positions in one wave, alpha = 6 (F(4x4,3x3), F(2x2,5x5)) splits the 36
// positions over two waves.
int row_groups(const Geom& g) { return g.A == 4 ? 1 : 2; }

bool valid_cfg(const Geom& g, FusedCfg c) {
    if (c.csplit != 1 && c.csplit != 2 && c.csplit != 4 && c.csplit != 8) return false;
    if (row_groups(g) * c.csplit > 8) return false;
    return c.bw == 16 || c.bw == 4;
}

// Workgroups of the fused kernel for a variant: tile blocks x filter groups.
long fused_workgroups(const Geom& g, FusedCfg c) {
    const int bh = 16 / c.bw;
    const long nt = (long)g.N * ((g.th + bh - 1) / bh) * ((g.tw + c.bw - 1) / c.bw);
    const int kgw = 8 / (row_groups(g) * c.csplit);
    return nt * ((g.KB + kgw - 1) / kgw);
}

// Fraction of the tiles of a grid of bw-wide tile blocks that are real tiles.
double block_util(const Geom& g, int bw) {
    const int bh = 16 / bw;
    const double rows = (double)((g.th + bh - 1) / bh * bh), cols = (double)((g.tw + bw - 1) / bw * bw);
    return (double)g.th * g.tw / (rows * cols);
}

// Estimated time (ns) of the fused and split algorithms: both kernels run one
// workgroup per CU, so a launch takes ceil(items/256) rounds of one
// workgroup's MFMA work at an efficiency measured for each kernel family on
// MI355X (fused: by filter blocks per workgroup), plus, for split, the
// HBM-bound input transform (patches read with halo, tile-blocked V written).
constexpr double kCus = 256.0, kFlopPerClk = 256.0, kClkGHz = 2.2, kHbmBytesPerNs = 7000.0;

double rounds(long items) { return (double)((items + (long)kCus - 1) / (long)kCus); }

double fused_ns(const Geom& g, FusedCfg c) {
    const int kgw = 8 / (row_groups(g) * c.csplit);
    const double eff = kgw >= 4 ? 0.58 : kgw == 2 ? 0.42 : 0.33;
    const double work = 2.0 * 16 * kgw * 16 * (4.0 * g.CQ) * g.T;      // FLOP per workgroup
    return rounds(fused_workgroups(g, c)) * work / (kFlopPerClk * eff) / kClkGHz;
}

double split_ns(const Geom& g) {
    const int kgw = g.m == 4 ? 4 : 8;
    const double cq4 = (g.CQ + 3) / 4 * 4;
    const double work = 2.0 * 2 * 16 * kgw * 16 * (4.0 * cq4) * g.T;    // FLOP per item
    // the tail's units run in one round of about a quarter of an item's time
    const SplitTail t = split_tail(g);
    const double item_rounds = rounds(t.items - t.tail) + (t.tail ? 0.25 : 0.0);
    const double gemm = item_rounds * work / (kFlopPerClk * 0.74) / kClkGHz;
    const double bytes = 1.5 * 4.0 * g.N * g.C * g.H * g.W + 4.0 * (double)split_blocks(g) * cq4 * g.T * 64;
    return gemm + bytes / kHbmBytesPerNs;
}

size_t split_workspace(const Geom& g) { return vblk_elems(g) * sizeof(float); }

// The 16-bit split path's VH: tile blocks x C32 chunks x T x 1 KB.
size_t split16_workspace(const Geom& g) { return (size_t)split_blocks(g) * c32_elems(g) * g.T * 1024; }

// Partial outputs of the channel slices: [slices used][N][K][Ho][Wo].
size_t slice_workspace(const Geom& g, int nsl) {
    return (size_t)slices_used(g, nsl) * g.N * g.K * g.Ho * g.Wo * sizeof(float);
}

// Offsets into x that the NCHW input kernels form (see kInvalidOffset): one
// image for the fused and split kernels; for the staged input transforms the
// images one 16-tile block spans, at most 16 / (th*tw) + 2.
bool image_fits(const Geom& g) { return (int64_t)g.C * g.H * g.W * 4 < (int64_t)kInvalidOffset; }
bool block_images_fit(const Geom& g) {
    const int64_t span = 16 / ((int64_t)g.th * g.tw) + 2;
    return span * ((int64_t)g.C * g.H * g.W * 4) < (int64_t)kInvalidOffset;
}

// The fused and split kernels read channels past the slice (or past C) as
// zeros: such a load's offset lies past the buffer's record count.  That holds
// only while no 32-bit offset wraps round: the largest one a kernel forms must
// stay below 2^32.
constexpr int64_t kOffsetLimit = (int64_t)1 << 32;

// Fused kernel: a step loads 4*QS channel planes (QS = 8 / row groups quads),
// the prefetch runs up to three steps past a slice's last, and a load outside
// the image adds its step's offset to kInvalidOffset.
bool fused_offsets_fit(const Geom& g, const FusedCfg& c) {
    const int64_t plane_b = (int64_t)g.H * g.W * 4, qs = 8 / row_groups(g);
    const int64_t qsl = c.nsl > 1 ? (g.CQ + c.nsl - 1) / c.nsl : g.CQ;
    const int64_t steps = (qsl + qs - 1) / qs;
    return (int64_t)kInvalidOffset + (steps + 3) * 4 * qs * plane_b < kOffsetLimit;
}

// Split path's input transform: a workgroup loads 16 channel planes from the
// offset of its group of 4 quads, over CQ rounded up to whole groups.
bool split_offsets_fit(const Geom& g) {
    const int64_t plane_b = (int64_t)g.H * g.W * 4, ncq4 = (g.CQ + 3) / 4;
    return (int64_t)kInvalidOffset + ncq4 * 16 * plane_b < kOffsetLimit;
}

// 16-bit input transforms: per 16-tile block (k_input16) a channel past C adds
// its plane offset (up to C rounded up to 32) to kInvalidOffset; by tile rows
// the images a row range spans must fit.
bool prec_offsets_fit(const Geom& g) {
    const int64_t plane_b = (int64_t)g.H * g.W * 4;
    return block_images_fit(g) && (int64_t)kInvalidOffset + (int64_t)c32_elems(g) * 32 * plane_b < kOffsetLimit;
}

bool plan_fits(const Geom& g, const Plan& p) {
    if (p.algo == WINO_ALGO_STAGED) return block_images_fit(g);
    if (p.algo == WINO_ALGO_FUSED) return image_fits(g) && fused_offsets_fit(g, p.cfg);
    if (p.algo == WINO_ALGO_SPLIT) return image_fits(g) && split_offsets_fit(g);
    return true;
}

int make_plan_unchecked(const Geom& g, unsigned flags, Plan* p);

// The plan, or WINO_ERR_UNSUPPORTED where its input kernels' offsets would not
// fit.  AUTO moves on to the next algorithm that fits: an unsliced fused plan
// to split, then to the three stages.
int make_plan(const Geom& g, unsigned flags, Plan* p) {
    const int st = make_plan_unchecked(g, flags, p);
    if (st != WINO_OK || g.axis != 0 || g.nhwc) return st;
    if (prec_of(flags)) return prec_offsets_fit(g) ? WINO_OK : WINO_ERR_UNSUPPORTED;
    if (plan_fits(g, *p)) return WINO_OK;
    if (!p->automatic) return WINO_ERR_UNSUPPORTED;
    if (p->algo == WINO_ALGO_FUSED && g.r == 3) {
        Plan q = *p;
        q.algo = WINO_ALGO_SPLIT;
        q.cfg.nsl = 1;
        if (plan_fits(g, q)) {
            *p = q;
            return WINO_OK;
        }
    }
    p->algo = WINO_ALGO_STAGED;
    p->cfg.nsl = 1;
    return plan_fits(g, *p) ? WINO_OK : WINO_ERR_UNSUPPORTED;
}

int make_plan_unchecked(const Geom& g, unsigned flags, Plan* p) {
    if (flags & ~kKnownFlags) return WINO_ERR_UNSUPPORTED;
    const unsigned algo = flags & WINO_ALGO_MASK;
    if (algo != WINO_ALGO_AUTO && algo != WINO_ALGO_FUSED && algo != WINO_ALGO_STAGED && algo != WINO_ALGO_SPLIT &&
        algo != WINO_ALGO_LOWC)
        return WINO_ERR_UNSUPPORTED;
    if (algo == WINO_ALGO_LOWC && g.C > 4) return WINO_ERR_UNSUPPORTED;
    const unsigned blk = flags & kBlockMask;
    // 1-D filters, channel-last tensors and 16-bit operands run the three
    // stages (input transform, GEMMs, output transform); channel-last 3x3
    // layers and 16-bit operands also the split path (its GEMM kernel stores y
    // channel-last, or runs on 16-bit MFMAs).  Of the other one-kernel
    // variants, the fused kernel also takes 5x5 filters of NCHW tensors, the
    // split and low-channel ones only 3x3.
    const int prec = prec_of(flags);
    if (prec < 0) return WINO_ERR_UNSUPPORTED;
    if (prec && (g.r != 3 || g.axis != 0 || g.nhwc)) return WINO_ERR_UNSUPPORTED;
    if (g.axis != 0 || g.nhwc || prec) {
        // the split GEMM kernel addresses U through a 32-bit buffer range
        const bool can_split = g.axis == 0 && g.r == 3 &&
                               (prec ? (int64_t)g.KB * (int64_t)c32_elems(g) * g.T * 1024 <= 0x7fffffffLL
                                     : g.nhwc && (int64_t)g.KB * g.CQ * g.T * 256 <= 0x7fffffffLL);
        if ((algo != WINO_ALGO_AUTO && algo != WINO_ALGO_STAGED && !(algo == WINO_ALGO_SPLIT && can_split)) ||
            blk || (flags >> kCsplitShift) & 0xF || (flags >> kSliceShift) & 0xF)
            return WINO_ERR_UNSUPPORTED;
        p->automatic = algo == WINO_ALGO_AUTO;
        p->cfg = FusedCfg{1, 16, 1};
        // AUTO: split on layers with at least two full rounds of its items
        // (tile-block pair x filter group) on the CUs, where the saved M round
        // trip outweighs its per-item prologue and epilogue.
        p->algo = algo == WINO_ALGO_SPLIT || (p->automatic && can_split && split_tail(g).items >= 2 * kSplitCus)
                      ? WINO_ALGO_SPLIT
                      : WINO_ALGO_STAGED;
        return WINO_OK;
    }
    if (blk == kBlockMask) return WINO_ERR_UNSUPPORTED;
    const int sl_req = (int)((flags >> kSliceShift) & 0xF);
    if (sl_req > 8 || (sl_req > 1 && (algo != WINO_ALGO_FUSED || sl_req > g.CQ))) return WINO_ERR_UNSUPPORTED;
    if (g.r != 3 && (algo == WINO_ALGO_SPLIT || algo == WINO_ALGO_LOWC)) return WINO_ERR_UNSUPPORTED;
    const int cs_req = (int)((flags >> kCsplitShift) & 0xF);
    p->algo = algo == WINO_ALGO_AUTO ? WINO_ALGO_FUSED : algo;
    p->automatic = algo == WINO_ALGO_AUTO;
    // Fused variant.  Tile blocks: a row of 16 tiles when the tile grid is at
    // least 12 wide and those blocks waste not much more of their tiles than
    // 4 x 4 ones (row blocks run faster per tile: measured about 15% with
    // equal waste), else 4 x 4.  Channel split: the smallest that gives the
    // 256 CUs a workgroup each (more filter blocks per workgroup share the
    // staged input patch) and leaves no wave without a filter block of its
    // own, else the largest available.
    FusedCfg c;
    c.nsl = 1;
    c.bw = blk == WINO_BLOCK_1x16 ? 16
         : blk == WINO_BLOCK_4x4  ? 4
         : (g.tw >= 12 && block_util(g, 16) >= 0.75 * block_util(g, 4) ? 16 : 4);
    if (cs_req) {
        c.csplit = cs_req;
    } else {
        const int max_cs = 8 / row_groups(g);
        c.csplit = 1;
        while (c.csplit < max_cs &&
               (fused_workgroups(g, c) < 240 || 8 / (row_groups(g) * c.csplit) > g.KB))
            c.csplit *= 2;
    }
    if (p->algo == WINO_ALGO_FUSED && !valid_cfg(g, c)) return WINO_ERR_UNSUPPORTED;
    // The fused and split kernels address U through a 32-bit buffer range.
    if (p->algo != WINO_ALGO_STAGED && (int64_t)g.KB * g.CQ * g.T * 256 > 0x7fffffffLL) return WINO_ERR_UNSUPPORTED;
    p->cfg = c;
    // Layers with at most 4 channels: the low-C kernel.
    if (p->automatic && g.r == 3 && g.C <= 4 && !cs_req && !blk) {
        p->algo = WINO_ALGO_LOWC;
        return WINO_OK;
    }
    // Split path where the estimates favour it.
    if (p->automatic && g.r == 3 && !cs_req && split_ns(g) < fused_ns(g, c))
        p->algo = WINO_ALGO_SPLIT;
    // Channel slices over workgroups for fused layers that leave CUs idle with
    // a long channel loop each (deep layers at small batch): double the slices
    // while the workgroups still fit one round on the 256 CUs and every slice
    // keeps at least 4 channel steps.  Partial outputs go to the workspace and
    // one more launch sums them in slice order.
    if (p->algo == WINO_ALGO_FUSED && sl_req > 1) {
        p->cfg.nsl = sl_req;
    } else if (p->algo == WINO_ALGO_FUSED && p->automatic && !sl_req) {
        const long wgs = fused_workgroups(g, c);
        const int qs = 8 / row_groups(g);                   // quads per channel step
        const int steps = (g.CQ + qs - 1) / qs;
        int nsl = 1;
        while (nsl < 8 && wgs * nsl * 2 <= (long)kCus && steps / (nsl * 2) >= 4) nsl *= 2;
        p->cfg.nsl = nsl;
    }
    return WINO_OK;
}

int hip_status(hipError_t e) { return e == hipSuccess ? WINO_OK : WINO_ERR_HIP; }

}  // namespace

extern "C" {

const char* wino_status_string(int status) {
    switch (status) {
        case WINO_OK: return "ok";
        case WINO_ERR_INVALID_ARG: return "invalid argument";
        case WINO_ERR_UNSUPPORTED: return "unsupported configuration";
        case WINO_ERR_WORKSPACE: return "workspace missing or too small";
        case WINO_ERR_HIP: return "HIP launch error";
        default: return "unknown status";
    }
}

int wino_version(void) { return 100; }

size_t wino_filter_bytes_r(int C, int K, int m, int r) {
    if (C <= 0 || K <= 0 || !supported(m, r)) return 0;
    int64_t e;
    const int a = m + r - 1;
    if (!mul_ok((int64_t)(C + 3) / 4 * 4, (int64_t)(K + 15) / 16 * 16, &e) || !mul_ok(e, a * a, &e))
        return 0;
    return (size_t)e * sizeof(float);
}

size_t wino_filter_bytes(int C, int K, int m) { return wino_filter_bytes_r(C, K, m, 3); }

size_t wino_filter_bytes_p(int C, int K, int m, unsigned prec) {
    if (prec == 0) return wino_filter_bytes(C, K, m);
    if (C <= 0 || K <= 0 || (m != 2 && m != 4) || prec_of(prec) <= 0 || (prec & ~WINO_PREC_MASK)) return 0;
    int64_t e;
    if (!mul_ok((int64_t)(C + 31) / 32 * 32, (int64_t)(K + 15) / 16 * 16, &e) || !mul_ok(e, (m + 2) * (m + 2), &e))
        return 0;
    return (size_t)e * 2;
}

size_t wino_input_tf_bytes_r(int N, int C, int H, int W, int pad, int m, int r) {
    Geom g;
    if (make_geom_r(N, C, H, W, 1, pad, m, r, &g) != WINO_OK) return 0;
    return v_elems(g) * sizeof(float);
}

size_t wino_gemm_out_bytes_r(int N, int K, int H, int W, int pad, int m, int r) {
    Geom g;
    if (make_geom_r(N, 1, H, W, K, pad, m, r, &g) != WINO_OK) return 0;
    return m_elems(g) * sizeof(float);
}

size_t wino_input_tf_bytes(int N, int C, int H, int W, int pad, int m) {
    return wino_input_tf_bytes_r(N, C, H, W, pad, m, 3);
}

size_t wino_gemm_out_bytes(int N, int K, int H, int W, int pad, int m) {
    return wino_gemm_out_bytes_r(N, K, H, W, pad, m, 3);
}

size_t wino_workspace_bytes_r(int N, int C, int H, int W, int K, int pad, int m, int r, unsigned flags) {
    Geom g;
    Plan p;
    if (make_geom_r(N, C, H, W, K, pad, m, r, &g) != WINO_OK || make_plan(g, flags, &p) != WINO_OK)
        return (size_t)-1;
    if (prec_of(flags) && p.algo == WINO_ALGO_SPLIT) return split16_workspace(g);
    if (prec_of(flags)) return round_up(vh_bytes(g), 256) + m_elems(g) * sizeof(float);
    if (p.algo == WINO_ALGO_FUSED && p.cfg.nsl > 1) return slice_workspace(g, p.cfg.nsl);
    if (p.algo == WINO_ALGO_FUSED || p.algo == WINO_ALGO_LOWC) return 0;
    if (p.algo == WINO_ALGO_SPLIT) return split_workspace(g);
    return round_up(v_elems(g) * sizeof(float), 256) + m_elems(g) * sizeof(float);
}

int wino_plan_r(int N, int C, int H, int W, int K, int pad, int m, int r, unsigned flags, unsigned* algo,
                int* slices) {
    if (!algo || !slices) return WINO_ERR_INVALID_ARG;
    Geom g;
    int st = make_geom_r(N, C, H, W, K, pad, m, r, &g);
    if (st != WINO_OK) return st;
    Plan p;
    st = make_plan(g, flags, &p);
    if (st != WINO_OK) return st;
    *algo = p.algo;
    *slices = p.algo == WINO_ALGO_FUSED && p.cfg.nsl > 1 ? slices_used(g, p.cfg.nsl) : 1;
    return WINO_OK;
}

size_t wino_workspace_bytes(int N, int C, int H, int W, int K, int pad, int m, unsigned flags) {
    return wino_workspace_bytes_r(N, C, H, W, K, pad, m, 3, flags);
}

int wino_filter_transform_r(const float* gw, float* U, int C, int K, int m, int r, void* stream) {
    if (!gw || !U || C <= 0 || K <= 0) return WINO_ERR_INVALID_ARG;
    if (!supported(m, r)) return WINO_ERR_UNSUPPORTED;
    const size_t ub = wino_filter_bytes_r(C, K, m, r);
    if (ub == 0) return WINO_ERR_INVALID_ARG;
    if (overlap(gw, (size_t)K * C * r * r * sizeof(float), U, ub)) return WINO_ERR_INVALID_ARG;
    return hip_status(launch_filter_transform(gw, U, C, K, m, r, (hipStream_t)stream));
}

int wino_filter_transform(const float* gw, float* U, int C, int K, int m, void* stream) {
    return wino_filter_transform_r(gw, U, C, K, m, 3, stream);
}

int wino_filter_transform_p(const float* gw, void* U, int C, int K, int m, unsigned prec, void* stream) {
    if (prec == 0) return wino_filter_transform(gw, (float*)U, C, K, m, stream);
    if (!gw || !U || C <= 0 || K <= 0) return WINO_ERR_INVALID_ARG;
    if ((m != 2 && m != 4) || prec_of(prec) <= 0 || (prec & ~WINO_PREC_MASK)) return WINO_ERR_UNSUPPORTED;
    const size_t ub = wino_filter_bytes_p(C, K, m, prec);
    if (ub == 0) return WINO_ERR_INVALID_ARG;
    if (overlap(gw, (size_t)K * C * 9 * sizeof(float), U, ub)) return WINO_ERR_INVALID_ARG;
    return hip_status(launch_filter_transform16(gw, U, C, K, m, prec_of(prec), (hipStream_t)stream));
}

int wino_conv2d_r(const float* x, const float* U, float* y, int N, int C, int H, int W, int K, int pad, int m,
                  int r, unsigned flags, void* workspace, size_t workspace_bytes, void* stream) {
    if (!x || !U || !y) return WINO_ERR_INVALID_ARG;
    Geom g;
    int st = make_geom_r(N, C, H, W, K, pad, m, r, &g);
    if (st != WINO_OK) return st;
    Plan p;
    st = make_plan(g, flags, &p);
    if (st != WINO_OK) return st;
    const size_t xb = (size_t)N * C * H * W * sizeof(float);
    const size_t yb = (size_t)N * K * g.Ho * g.Wo * sizeof(float);
    const int prec = prec_of(flags);
    const size_t ub = prec ? wino_filter_bytes_p(C, K, m, flags & WINO_PREC_MASK) : wino_filter_bytes_r(C, K, m, r);
    if (overlap(x, xb, y, yb) || overlap(U, ub, y, yb)) return WINO_ERR_INVALID_ARG;
    const bool relu = (flags & WINO_FLAG_RELU) != 0;
    hipStream_t s = (hipStream_t)stream;
    if (prec && p.algo == WINO_ALGO_SPLIT) {
        const size_t need = split16_workspace(g);
        if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
        if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
            return WINO_ERR_INVALID_ARG;
        return hip_status(launch_split16(x, U, y, workspace, g, prec, relu, s));
    }
    if (prec) {
        const size_t vb = round_up(vh_bytes(g), 256);
        const size_t need = vb + m_elems(g) * sizeof(float);
        if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
        if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
            return WINO_ERR_INVALID_ARG;
        return hip_status(launch_staged16(x, U, y, workspace, (float*)((char*)workspace + vb), g, prec, relu, s));
    }
    if (p.algo == WINO_ALGO_SPLIT) {
        const size_t need = split_workspace(g);
        if (!workspace || workspace_bytes < need) {
            if (!p.automatic) return WINO_ERR_WORKSPACE;
            p.algo = WINO_ALGO_FUSED;          // no room for V: the fused kernel, where its offsets fit
            if (!plan_fits(g, p)) return WINO_ERR_WORKSPACE;
        } else {
            if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
                return WINO_ERR_INVALID_ARG;
            return hip_status(launch_split(x, U, y, (float*)workspace, g, p.cfg.bw, relu, s));
        }
    }
    if (p.algo == WINO_ALGO_FUSED && p.cfg.nsl > 1) {
        const size_t need = slice_workspace(g, p.cfg.nsl);
        if (!workspace || workspace_bytes < need) {
            if (!p.automatic) return WINO_ERR_WORKSPACE;
            p.cfg.nsl = 1;                      // no room for the partial outputs: unsliced
            if (!plan_fits(g, p)) return WINO_ERR_WORKSPACE;
        } else {
            if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
                return WINO_ERR_INVALID_ARG;
            return hip_status(launch_fused(x, U, y, g, p.cfg, relu, s, (float*)workspace));
        }
    }
    if (p.algo == WINO_ALGO_FUSED) return hip_status(launch_fused(x, U, y, g, p.cfg, relu, s));
    if (p.algo == WINO_ALGO_LOWC) return hip_status(launch_lowc(x, U, y, g, relu, s));

    const size_t vb = round_up(v_elems(g) * sizeof(float), 256);
    const size_t need = vb + m_elems(g) * sizeof(float);
    if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
    if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
        return WINO_ERR_INVALID_ARG;
    float* V = (float*)workspace;
    float* M = (float*)((char*)workspace + vb);
    st = hip_status(launch_input_transform(x, V, g, s));
    if (st != WINO_OK) return st;
    st = hip_status(launch_batched_gemm(U, V, M, g, s));
    if (st != WINO_OK) return st;
    return hip_status(launch_output_transform(M, y, g, relu, s));
}

int wino_conv2d(const float* x, const float* U, float* y, int N, int C, int H, int W, int K, int pad, int m,
                unsigned flags, void* workspace, size_t workspace_bytes, void* stream) {
    return wino_conv2d_r(x, U, y, N, C, H, W, K, pad, m, 3, flags, workspace, workspace_bytes, stream);
}

int wino_conv2d_noalloc(const float* x, const float* U, float* y, int N, int C, int H, int W, int K, int pad,
                        int m, unsigned flags, void* stream) {
    if (!x || !U || !y) return WINO_ERR_INVALID_ARG;
    Geom g;
    int st = make_geom(N, C, H, W, K, pad, m, &g);
    if (st != WINO_OK) return st;
    Plan p;
    st = make_plan(g, flags, &p);
    if (st != WINO_OK) return st;
    const size_t need = wino_workspace_bytes(N, C, H, W, K, pad, m, flags);
    if (need == (size_t)-1) return WINO_ERR_UNSUPPORTED;
    // AUTO falls back to a plan whose workspace fits (wino_conv2d_r decides,
    // given the array's size); explicit choices must fit as asked.
    if (need > kNoAllocScratchBytes && !p.automatic) return WINO_ERR_WORKSPACE;
    // the aliasing checks of wino_conv2d, before the scratch lookup (a HIP call)
    const size_t xb = (size_t)N * C * H * W * sizeof(float);
    const size_t yb = (size_t)N * K * g.Ho * g.Wo * sizeof(float);
    const size_t ub = prec_of(flags) ? wino_filter_bytes_p(C, K, m, flags & WINO_PREC_MASK) : wino_filter_bytes(C, K, m);
    if (overlap(x, xb, y, yb) || overlap(U, ub, y, yb)) return WINO_ERR_INVALID_ARG;
    void* ws = nullptr;
    if (need > 0) {
        st = hip_status(noalloc_scratch(&ws));
        if (st != WINO_OK) return st;
    }
    return wino_conv2d_r(x, U, y, N, C, H, W, K, pad, m, 3, flags, ws, ws ? kNoAllocScratchBytes : 0, stream);
}

int wino_input_transform_r(const float* x, float* V, int N, int C, int H, int W, int pad, int m, int r,
                           void* stream) {
    if (!x || !V) return WINO_ERR_INVALID_ARG;
    Geom g;
    const int st = make_geom_r(N, C, H, W, 1, pad, m, r, &g);
    if (st != WINO_OK) return st;
    if (overlap(x, (size_t)N * C * H * W * sizeof(float), V, v_elems(g) * sizeof(float)))
        return WINO_ERR_INVALID_ARG;
    if (!block_images_fit(g)) return WINO_ERR_UNSUPPORTED;
    return hip_status(launch_input_transform(x, V, g, (hipStream_t)stream));
}

int wino_input_transform(const float* x, float* V, int N, int C, int H, int W, int pad, int m, void* stream) {
    return wino_input_transform_r(x, V, N, C, H, W, pad, m, 3, stream);
}

int wino_batched_gemm_r(const float* U, const float* V, float* M, int N, int C, int H, int W, int K, int pad,
                        int m, int r, void* stream) {
    if (!U || !V || !M) return WINO_ERR_INVALID_ARG;
    Geom g;
    const int st = make_geom_r(N, C, H, W, K, pad, m, r, &g);
    if (st != WINO_OK) return st;
    const size_t mb = m_elems(g) * sizeof(float);
    if (overlap(M, mb, U, wino_filter_bytes_r(C, K, m, r)) || overlap(M, mb, V, v_elems(g) * sizeof(float)))
        return WINO_ERR_INVALID_ARG;
    return hip_status(launch_batched_gemm(U, V, M, g, (hipStream_t)stream));
}

int wino_batched_gemm(const float* U, const float* V, float* M, int N, int C, int H, int W, int K, int pad, int m,
                      void* stream) {
    return wino_batched_gemm_r(U, V, M, N, C, H, W, K, pad, m, 3, stream);
}

int wino_output_transform_r(const float* M, float* y, int N, int K, int H, int W, int pad, int m, int r,
                            unsigned flags, void* stream) {
    if (!M || !y) return WINO_ERR_INVALID_ARG;
    if (flags & ~WINO_FLAG_RELU) return WINO_ERR_UNSUPPORTED;
    Geom g;
    const int st = make_geom_r(N, 1, H, W, K, pad, m, r, &g);
    if (st != WINO_OK) return st;
    if (overlap(M, m_elems(g) * sizeof(float), y, (size_t)N * K * g.Ho * g.Wo * sizeof(float)))
        return WINO_ERR_INVALID_ARG;
    return hip_status(launch_output_transform(M, y, g, (flags & WINO_FLAG_RELU) != 0, (hipStream_t)stream));
}

int wino_output_transform(const float* M, float* y, int N, int K, int H, int W, int pad, int m, unsigned flags,
                          void* stream) {
    return wino_output_transform_r(M, y, N, K, H, W, pad, m, 3, flags, stream);
}

size_t wino_filter_bytes_1d(int C, int K, int m, int r) {
    if (C <= 0 || K <= 0 || !supported_1d(m, r)) return 0;
    int64_t e;
    if (!mul_ok((int64_t)(C + 3) / 4 * 4, (int64_t)(K + 15) / 16 * 16, &e) || !mul_ok(e, 8, &e)) return 0;
    return (size_t)e * sizeof(float);
}

int wino_filter_transform_1d(const float* gw, float* U, int C, int K, int m, int r, void* stream) {
    if (!gw || !U || C <= 0 || K <= 0) return WINO_ERR_INVALID_ARG;
    if (!supported_1d(m, r)) return WINO_ERR_UNSUPPORTED;
    const size_t ub = wino_filter_bytes_1d(C, K, m, r);
    if (ub == 0) return WINO_ERR_INVALID_ARG;
    if (overlap(gw, (size_t)K * C * r * sizeof(float), U, ub)) return WINO_ERR_INVALID_ARG;
    return hip_status(launch_filter_transform_1d(gw, U, C, K, m, r, (hipStream_t)stream));
}

size_t wino_workspace_bytes_1d(int N, int C, int H, int W, int K, int pad, int m, int r, int axis,
                               unsigned flags) {
    Geom g;
    Plan p;
    if (make_geom_1d(N, C, H, W, K, pad, m, r, axis, &g) != WINO_OK || make_plan(g, flags, &p) != WINO_OK)
        return (size_t)-1;
    return round_up(v_elems(g) * sizeof(float), 256) + m_elems(g) * sizeof(float);
}

int wino_conv2d_1d(const float* x, const float* U, float* y, int N, int C, int H, int W, int K, int pad, int m,
                   int r, int axis, unsigned flags, void* workspace, size_t workspace_bytes, void* stream) {
    if (!x || !U || !y) return WINO_ERR_INVALID_ARG;
    Geom g;
    int st = make_geom_1d(N, C, H, W, K, pad, m, r, axis, &g);
    if (st != WINO_OK) return st;
    Plan p;
    st = make_plan(g, flags, &p);
    if (st != WINO_OK) return st;
    const size_t xb = (size_t)N * C * H * W * sizeof(float);
    const size_t yb = (size_t)N * K * g.Ho * g.Wo * sizeof(float);
    const size_t ub = wino_filter_bytes_1d(C, K, m, r);
    if (overlap(x, xb, y, yb) || overlap(U, ub, y, yb)) return WINO_ERR_INVALID_ARG;
    const size_t vb = round_up(v_elems(g) * sizeof(float), 256);
    const size_t need = vb + m_elems(g) * sizeof(float);
    if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
    if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
        return WINO_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)stream;
    float* V = (float*)workspace;
    float* M = (float*)((char*)workspace + vb);
    st = hip_status(launch_input_transform(x, V, g, s));
    if (st != WINO_OK) return st;
    st = hip_status(launch_batched_gemm(U, V, M, g, s));
    if (st != WINO_OK) return st;
    return hip_status(launch_output_transform(M, y, g, (flags & WINO_FLAG_RELU) != 0, s));
}

size_t wino_workspace_bytes_nhwc(int N, int C, int H, int W, int K, int pad, int m, unsigned flags) {
    Geom g;
    Plan p;
    if (make_geom(N, C, H, W, K, pad, m, &g) != WINO_OK) return (size_t)-1;
    g.nhwc = 1;
    if (make_plan(g, flags, &p) != WINO_OK) return (size_t)-1;
    if (p.algo == WINO_ALGO_SPLIT) return split_workspace(g);
    return round_up(v_elems(g) * sizeof(float), 256) + m_elems(g) * sizeof(float);
}

int wino_conv2d_nhwc(const float* x, const float* U, float* y, int N, int C, int H, int W, int K, int pad, int m,
                     unsigned flags, void* workspace, size_t workspace_bytes, void* stream) {
    if (!x || !U || !y) return WINO_ERR_INVALID_ARG;
    Geom g;
    int st = make_geom(N, C, H, W, K, pad, m, &g);
    if (st != WINO_OK) return st;
    g.nhwc = 1;
    Plan p;
    st = make_plan(g, flags, &p);
    if (st != WINO_OK) return st;
    const size_t xb = (size_t)N * C * H * W * sizeof(float);
    const size_t yb = (size_t)N * K * g.Ho * g.Wo * sizeof(float);
    const size_t ub = wino_filter_bytes(C, K, m);
    if (overlap(x, xb, y, yb) || overlap(U, ub, y, yb)) return WINO_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)stream;
    if (p.algo == WINO_ALGO_SPLIT) {
        const size_t need = split_workspace(g);
        if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
        if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
            return WINO_ERR_INVALID_ARG;
        return hip_status(launch_split(x, U, y, (float*)workspace, g, 16, (flags & WINO_FLAG_RELU) != 0, s));
    }
    const size_t vb = round_up(v_elems(g) * sizeof(float), 256);
    const size_t need = vb + m_elems(g) * sizeof(float);
    if (!workspace || workspace_bytes < need) return WINO_ERR_WORKSPACE;
    if (overlap(workspace, need, x, xb) || overlap(workspace, need, y, yb) || overlap(workspace, need, U, ub))
        return WINO_ERR_INVALID_ARG;
    float* V = (float*)workspace;
    float* M = (float*)((char*)workspace + vb);
    st = hip_status(launch_input_transform(x, V, g, s));
    if (st != WINO_OK) return st;
    st = hip_status(launch_batched_gemm(U, V, M, g, s));
    if (st != WINO_OK) return st;
    return hip_status(launch_output_transform(M, y, g, (flags & WINO_FLAG_RELU) != 0, s));
}

int wino_maxpool2x2(const float* x, float* y, int N, int C, int H, int W, void* stream) {
    if (!x || !y || N <= 0 || C <= 0 || H < 2 || W < 2) return WINO_ERR_INVALID_ARG;
    int64_t e;
    if (!mul_ok((int64_t)N * C, (int64_t)H * W, &e)) return WINO_ERR_INVALID_ARG;
    if (overlap(x, (size_t)e * sizeof(float), y, (size_t)N * C * (H / 2) * (W / 2) * sizeof(float)))
        return WINO_ERR_INVALID_ARG;
    return hip_status(launch_maxpool2x2(x, y, N, C, H, W, (hipStream_t)stream));
}

int wino_probe_mfma_f32(int iters, float* out, void* stream) {
    if (!out || iters < 1 || iters > kProbeMaxIters) return WINO_ERR_INVALID_ARG;
    return hip_status(launch_mfma_probe(iters, out, (hipStream_t)stream));
}

size_t wino_probe_mfma_f32_flops(int iters) {
    if (iters < 1 || iters > kProbeMaxIters) return 0;
    return (size_t)kProbeWaves * (size_t)iters * 8 * (2 * 16 * 16 * 4);
}

}  // extern "C"
