// Tile bookkeeping shared by the fp32 and bf16 convolution kernels.
// Internal to libim2win.
#pragma once

#include "common.h"

#include <algorithm>

namespace im2win {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBf16ChunkChannels = 16;   // bf16: input channels per chunk (MFMA reduction width)

constexpr int kConvThreads = 256;            // 4 waves of 64 lanes
constexpr int kConvLdsBudgetBytes = 64 * 1024;    // preferred LDS per workgroup
constexpr int kConvLdsMaxBytes = 160 * 1024;      // gfx950 LDS per workgroup
constexpr int kConvLdsPipelinedBytes = 80 * 1024; // two double-buffered workgroups per CU

struct ConvArgs {
    const void* src;   // window tensor (unfused) or input x (fused)
    const void* w;     // K x C x Fh x Fw
    float* y;          // N x K x Ho x Wo
    int c, h, w_in, k, fh, fw, sh, sw, ph, pw;
    int ho, wo, wp, row_len, used_len, taps;
    int npix, howo;
    int rc;            // input channels per chunk
    int strip_cap;     // LDS strip positions reserved per channel
    int sc;            // fp32: LDS stride between channel strips (floats)
    int fp;            // fp32: LDS stride between filter rows (floats)
    int bm;            // output channels per workgroup
    int ksplit;        // fp32: 0 = k-slots split by channel halves, 1 = by filter rows
    int kpad;          // fp32: filter-tile rows, rc*taps rounded up to even
    int tc;            // bf16: filter taps staged per pass
    int num_jtiles;
    FastDiv div_wo, div_ho, div_kpad, div_taps, div_fw, div_row, div_fh, div_tc2;
    int d_row, d_k, d_u;   // kConvThreads = d_row*L + d_k*Fh + d_u (fused walk)
    int e_row, e_k, e_u;   // 64 (one wave) = e_row*L + e_k*Fh + e_u (fused DMA walk)
    int stage;             // LDS elements per pipeline stage
    int svec;              // unfused: strips staged by 16-byte copies (plane % vchunk == 0)
    int vchunk;            // elements per 16 bytes (4 fp32, 8 bf16)
    int fvec;              // filter rows staged by 16-byte copies
    FastDiv div_fp, div_ckmid;
    FastDiv div_lenmid;    // by len_mid, the run length of a whole image (plain layout)
    // fused fp32: the tile's input rows are copied to LDS (raw rows), then
    // expanded on chip into the strip layout
    int xvec;              // rows of x are whole 16-byte vectors (W % 4 == 0)
    int raw_pitch;         // LDS floats per channel of the raw rows
    int raw_off;           // LDS float offset of the raw rows
    int rmid;              // input rows that the windows of a whole image use
    int ylo_mid;           // first of them
    FastDiv div_w, div_sh, div_rmid;   // by W, sh, max(rmid, 1)
    // bf16: channel-inner LDS layout (positions of 16 bytes = 8 channels)
    int cl_pitch;          // LDS positions per window-tensor row (>= row_len)
    int cl_pb;             // positions per strip plane (one plane per 8-channel half)
    int cl_fpb;            // positions per filter plane
    int ilv;               // fp32 unfused: copies issued from inside the MFMA loop
    int fpack;             // fp32: w is the filter repacked into chunk blocks (pack_filter_f32_kernel)
};


// Geometry of the window-tensor runs that one pixel tile reads (per channel).
struct TileRuns {
    int p0, plast;
    int i0, m0, n0;     // first pixel
    int i1, m1, n1;     // last pixel
    int nseg;           // images touched
    int qa0;            // first run starts at this column of row m0
    int len0, len_mid, len_last, strip_len;
    // LDS placement of the runs.  Plain layout: run s starts at seg_off(s),
    // runs back to back.  16-byte layout (a.svec): every run starts on a
    // 16-byte boundary and run 0 is shifted by its global misalignment
    // shift0, so that 16-byte copies land aligned; ck* count 16-byte chunks.
    int shift0, ck0, ck_mid, ck_last, ck_total;
    int d_first, d_second, d_stride, extent;   // data start of run 0, of run 1, run pitch, LDS floats used

    __host__ __device__ void init(int ptile, int bn, const ConvArgs& a) {
        p0 = ptile * bn;
        plast = (p0 + bn < a.npix ? p0 + bn : a.npix) - 1;
        const int g0 = (int)fast_div((uint32_t)p0, a.div_wo);
        const int g1 = (int)fast_div((uint32_t)plast, a.div_wo);
        n0 = p0 - g0 * a.wo;
        n1 = plast - g1 * a.wo;
        i0 = (int)fast_div((uint32_t)g0, a.div_ho);
        i1 = (int)fast_div((uint32_t)g1, a.div_ho);
        m0 = g0 - i0 * a.ho;
        m1 = g1 - i1 * a.ho;
        nseg = i1 - i0 + 1;
        qa0 = n0 * a.sw * a.fh;
        const int qb_last = (n1 * a.sw + a.fw) * a.fh;
        len_mid = (a.ho - 1) * a.row_len + a.used_len;
        if (nseg == 1) {
            len0 = (m1 - m0) * a.row_len + qb_last - qa0;
            len_last = 0;
            strip_len = len0;
        } else {
            len0 = (a.ho - 1 - m0) * a.row_len + a.used_len - qa0;
            len_last = m1 * a.row_len + qb_last;
            strip_len = len0 + (nseg - 2) * len_mid + len_last;
        }
        if (a.svec) {
            const int vc = a.vchunk;   // elements per 16-byte chunk (4 fp32, 8 bf16)
            shift0 = (m0 * a.row_len + qa0) & (vc - 1);
            ck0 = (shift0 + len0 + vc - 1) / vc;
            ck_mid = (len_mid + vc - 1) / vc;
            ck_last = (len_last + vc - 1) / vc;
            ck_total = nseg == 1 ? ck0 : ck0 + (nseg - 2) * ck_mid + ck_last;
            d_first = shift0;
            d_second = vc * ck0;
            d_stride = vc * ck_mid;
            extent = vc * ck_total;
        } else {
            shift0 = 0;
            ck0 = ck_mid = ck_last = ck_total = 0;
            d_first = 0;
            d_second = len0;
            d_stride = len_mid;
            extent = strip_len;
        }
    }
    // LDS offset of the first element of run s
    __host__ __device__ int seg_off(int s) const {
        return s == 0 ? d_first : d_second + (s - 1) * d_stride;
    }
    __host__ __device__ int seg_len(int s) const {
        return s == 0 ? len0 : (s == nseg - 1 ? len_last : len_mid);
    }
    __host__ __device__ int seg_m(int s) const { return s == 0 ? m0 : 0; }
    __host__ __device__ int seg_q(int s) const { return s == 0 ? qa0 : 0; }
};

// One run (image segment) of a tile, computed from values held in registers
// (a select between struct fields would otherwise be turned into a load).
struct SegRun {
    int off, len, m, q;
};

__host__ __device__ inline SegRun seg_run(int s, int nseg, int len0, int len_mid, int len_last,
                                          int m0, int qa0, int d_first, int d_second,
                                          int d_stride) {
    SegRun r;
    r.off = s == 0 ? d_first : d_second + (s - 1) * d_stride;
    r.len = s == 0 ? len0 : (s == nseg - 1 ? len_last : len_mid);
    r.m = s == 0 ? m0 : 0;
    r.q = s == 0 ? qa0 : 0;
    return r;
}

// Strip offset of the window of pixel p (its column in the implicit GEMM) and
// the output offset of its channel-0 element.  Pixels past the end of the
// tile are clamped to the first pixel of the tile (computed, never stored).
__host__ __device__ inline int pixel_base(const TileRuns& tr, const ConvArgs& a, int p,
                                          int64_t* yoff) {
    const int g = (int)fast_div((uint32_t)p, a.div_wo);
    const int n = p - g * a.wo;
    const int i = (int)fast_div((uint32_t)g, a.div_ho);
    const int m = g - i * a.ho;
    const int s = i - tr.i0;
    *yoff = (int64_t)i * a.k * a.howo + m * a.wo + n;
    return tr.seg_off(s) + (m - tr.seg_m(s)) * a.row_len + n * a.sw * a.fh - tr.seg_q(s);
}

// Input rows of x that one pixel tile uses, per image segment of its runs:
// segment 0 reads rows [ylo0, ylo0 + r0), the middle segments (whole images)
// [ylo_mid, ylo_mid + rmid) and the last [ylo_mid, ylo_mid + rlast).  In LDS
// they are stored back to back, segment after segment (rtot rows).
struct RawRows {
    int ylo0, r0, rlast, rtot;
};

__host__ __device__ inline int clamp_rows(int lo, int hi) { return hi > lo ? hi - lo : 0; }

__host__ __device__ inline RawRows raw_rows(const TileRuns& tr, const ConvArgs& a) {
    RawRows r;
    const int m_end0 = tr.nseg == 1 ? tr.m1 : a.ho - 1;
    const int lo0 = tr.m0 * a.sh - a.ph;
    r.ylo0 = lo0 > 0 ? lo0 : 0;
    const int hi0 = m_end0 * a.sh - a.ph + a.fh;
    r.r0 = clamp_rows(r.ylo0, hi0 < a.h ? hi0 : a.h);
    const int hil = tr.m1 * a.sh - a.ph + a.fh;
    r.rlast = tr.nseg == 1 ? 0 : clamp_rows(a.ylo_mid, hil < a.h ? hil : a.h);
    r.rtot = tr.nseg == 1 ? r.r0 : r.r0 + (tr.nseg - 2) * a.rmid + r.rlast;
    return r;
}

__host__ __device__ inline int mod16(int v) { return ((v % 16) + 16) % 16; }
__host__ __device__ inline int round_up4(int v) { return (v + 3) & ~3; }

// bf16 channel-inner LDS layout of one tile's strips: positions of 16 bytes
// (8 channels), one plane per 8-channel half.  Row m of image segment s
// starts at seg_base(s) + (m - seg_m(s))*cl_pitch - seg_q(s).  The row pitch
// is congruent to sw*Fh*Wo and the segment bases to sw*Fh times the number
// of tile pixels before them (mod 16 positions), so the windows of the
// tile's flattened pixels P start at positions congruent to sw*Fh*P + sb0:
// for odd sw*Fh, 16 consecutive pixels fall in 16 different 16-byte bank
// groups.  sb0 is the 4-position alignment shift of the first run.
struct ClLayout {
    int sb0, sb1, sp, extent;
    __host__ __device__ int seg_base(int s) const { return s == 0 ? sb0 : sb1 + (s - 1) * sp; }
};

__host__ __device__ inline ClLayout cl_layout(const TileRuns& tr, const ConvArgs& a) {
    ClLayout c;
    const int lp = a.cl_pitch, spx = a.sw * a.fh, hw = a.ho * a.wo;
    const int last_col = (tr.n1 * a.sw + a.fw) * a.fh;   // end of the tile's last row
    c.sb0 = tr.shift0;
    const int m_end0 = tr.nseg == 1 ? tr.m1 : a.ho - 1;
    const int end0 = c.sb0 + (m_end0 - tr.m0) * lp + round_up4(tr.nseg == 1 ? last_col : a.used_len) - tr.qa0;
    if (tr.nseg == 1) {
        c.sb1 = 0;
        c.sp = 0;
        c.extent = end0;
        return c;
    }
    c.sb1 = end0 + mod16(spx * (hw - tr.m0 * a.wo - tr.n0) + c.sb0 - end0);
    const int full = (a.ho - 1) * lp + round_up4(a.used_len);
    c.sp = full + mod16(spx * hw - full);
    c.extent = c.sb1 + (tr.nseg - 2) * c.sp + tr.m1 * lp + round_up4(last_col);
    return c;
}

// LDS position of in-plane element e of segment s's window-tensor plane.
__host__ __device__ inline int cl_pos(const ClLayout& c, const TileRuns& tr, const ConvArgs& a, int s, int e) {
    const int row = (int)fast_div((uint32_t)e, a.div_row);
    return c.seg_base(s) + (row - tr.seg_m(s)) * a.cl_pitch + (e - row * a.row_len) - tr.seg_q(s);
}

// LDS position of the window of pixel p, and the output offset of its
// channel-0 element (pixels past the tile are clamped to its first pixel).
__host__ __device__ inline int cl_pixel_base(const ClLayout& c, const TileRuns& tr, const ConvArgs& a, int p,
                                             int64_t* yoff) {
    const int g = (int)fast_div((uint32_t)p, a.div_wo);
    const int n = p - g * a.wo;
    const int i = (int)fast_div((uint32_t)g, a.div_ho);
    const int m = g - i * a.ho;
    const int s = i - tr.i0;
    *yoff = (int64_t)i * a.k * a.howo + m * a.wo + n;
    return c.seg_base(s) + (m - tr.seg_m(s)) * a.cl_pitch + n * a.sw * a.fh - tr.seg_q(s);
}

// Packed bf16 filter of the fast kernels (whole 16-channel chunks, whole
// tiles of BM output channels).  One block per (output-channel tile jt,
// chunk ch), blocks in order jt*nchunks + ch, each 2*T*BM pieces of 16 bytes
// laid out as the filter planes of an LDS stage: piece P = g*T*BM + t*BM + jj
// holds channels 16ch + 8g .. 16ch + 8g + 7 of tap t (window order
// t = v*Fh + u) of output channel jt*BM + jj.  A chunk's block is therefore
// one contiguous range that 16-byte DMA copies into LDS unchanged.
struct PackedPiece {
    int j, c0, nat, lds_pos;   // output channel, first input channel, tap (u*Fw + v), LDS position
};

__host__ __device__ inline PackedPiece packed_piece(int64_t gid, int t_taps, int fh, int fw, int bm,
                                                    int nchunks, int cl_fpb) {
    const int pieces = 2 * t_taps * bm, plane = t_taps * bm;
    const int64_t blk = gid / pieces;
    const int pc = (int)(gid - blk * pieces);
    const int jt = (int)(blk / nchunks), ch = (int)(blk - (int64_t)jt * nchunks);
    const int g = pc / plane, q = pc - g * plane;
    const int t = q / bm, jj = q - t * bm;
    const int v = t / fh, u = t - v * fh;
    PackedPiece r;
    r.j = jt * bm + jj;
    r.c0 = kBf16ChunkChannels * ch + 8 * g;
    r.nat = u * fw + v;
    r.lds_pos = g * cl_fpb + q;
    return r;
}

// Inverse of packed_piece: the piece holding channels 16ch + 8g .. + 7 of tap
// t of output channel j.
__host__ __device__ inline int64_t packed_index(int j, int ch, int g, int t, int t_taps, int bm,
                                                int nchunks) {
    const int jt = j / bm, jj = j - jt * bm;
    return (((int64_t)jt * nchunks + ch) * 2 + g) * (int64_t)(t_taps * bm) + (int64_t)t * bm + jj;
}

// Filter packing: a workgroup repacks kPackRows output channels x one chunk
// of 16 input channels through LDS (reads of whole filter rows, writes of
// kPackRows consecutive pieces).
constexpr int kPackRows = 8;

// Host bound of ClLayout::extent over the tiles of `bn` pixels.
inline int64_t cl_extent_bound(const Geometry& g, int bn, int64_t pitch) {
    const int64_t dmax = (g.wo - 1 + bn - 1) / g.wo;
    const int64_t nseg = std::min<int64_t>(dmax + 1, (bn - 1) / (g.ho * g.wo) + 2);
    return 4 + (dmax + 1) * pitch + 20 * nseg;
}

// Launch plan of a convolution kernel (chosen on the host).
struct ConvPlan {
    enum Kind { kNone, kF32Lds, kBf16Lds };
    Kind kind = kNone;     // fp32 strips (fp32, or bf16 widened) / channel-inner bf16 strips
    int bm = 0, bn = 0;    // output channels x pixels per workgroup
    int rc = 0;            // input channels per LDS chunk
    int tc = 0;            // bf16: taps per filter pass
    int split = 0;         // fp32: k-slot split (0 channel halves, 1 filter rows)
    int64_t strip_cap = 0; // LDS strip positions per channel
    int64_t sc = 0, fp = 0;  // fp32: LDS strides of strips and filter rows
    int64_t stage = 0;       // LDS elements per pipeline stage
    int64_t raw_pitch = 0;   // fused fp32: LDS floats per channel of the raw input rows
    int64_t cl_pitch = 0;    // bf16: LDS positions per window-tensor row
    int64_t cl_fpb = 0;      // bf16: positions per filter plane (strip planes: strip_cap)
    int64_t strip_items = 0; // bf16, 16-byte strip loads: bound of the staging items per tile
    int fused_fast = 0;      // bf16: the fused kernel builds strips from raw row items
    int fast = 0;            // bf16 unfused: the fast kernel (16-byte strip loads, packed filter)
    int fused_ipt = 1;       // bf16 fused kernel: raw items per thread
    int svec = 0;            // unfused: 16-byte strip copies
    int fvec = 0;            // 16-byte filter-row copies
    int64_t lds_bytes = 0;
};

ConvPlan plan_conv_f32(const Geometry& g);
ConvPlan plan_conv_bf16(const Geometry& g, bool fused);
ConvArgs conv_args_f32(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                       float* y, bool fused);
ConvArgs conv_args_bf16(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                        float* y, bool fused);

// bf16 kernel: channels per chunk and per-thread staging registers (items)
constexpr int kBf16Chunk = kBf16ChunkChannels;
constexpr int kBf16StripVecItems = 2;
constexpr int kBf16StripScalarItems = 8;
constexpr int kBf16FilterScalarItems = 16;
constexpr int kF32ExpandGroups = 10;  // fused fp32 expansion map: raw floats per channel / 64
constexpr int kBf16Spare = 64;        // spare positions at the end of every strip plane
constexpr int kBf16FusedItems = 2;    // fused kernel: at most this many raw items per thread (2 elements x 8 channels)
constexpr int kIlvSlots = 8;          // fp32 copies issued inside the MFMA loop: per lane and channel / chunk
int launch_conv_f32_plan(const Geometry& g, const ConvPlan& p, bool fused, const void* src,
                         const void* w, void* scratch, float* y, hipStream_t stream, char* err,
                         size_t errlen);
// Bytes of the repacked filter an fp32-strip plan reads (0: w as given).
int64_t filter_scratch_f32(const Geometry& g, const ConvPlan& p);

struct TileCfg {
    int bm, bn;
};

// ---------------------------------------------------------------------------
// bf16 convolution with one image per workgroup (conv_bf16_image.hip)
// ---------------------------------------------------------------------------
constexpr int kImgThreads = 512;     // 8 waves: 4 groups of 32 output channels x 2 halves of the pixels
constexpr int kImgChunk = 32;        // input channels per chunk (one MFMA per tap)
constexpr int kImgNPB = 7;           // 16-pixel blocks per wave (193 to 224 output pixels per image)
constexpr int kImgStripItems = 2;    // unfused staging items per thread (4 positions x 8 channels)
constexpr int kImgBRing = 4;         // B fragments in flight + 1 (LDS reads issued ahead of their MFMAs)
constexpr int kImgFusedItems = 2;    // fused staging items per thread (2 input elements x 8 channels)

struct ImgArgs {
    const uint16_t* src;   // window tensor (unfused) or x (fused)
    const uint16_t* wf;    // filter in fragment order
    float* y;
    int c, h, w, k, sh, sw, ph, pw, ho, wo;
    int wr;                // window-tensor row width in input columns
    int row_len;           // wr * Fh
    int npix;              // Ho * Wo
    int pitch;             // LDS positions per window-tensor row
    int plane_pos;         // LDS positions per 8-channel plane
    int stage_pos;         // LDS positions per stage (4 planes)
    int plane_src;         // elements per channel plane of src (Ho*row_len, or H*W)
    int ngroups;           // staging groups per channel plane (4 positions, or 2 elements)
    int nkt;               // K / 128
    int nchunks;           // C / 32
    int grid;              // workgroups (N * nkt)
    int xcd_remap;         // place the workgroups of one image on one XCD
};

struct ImgPlan {
    bool ok = false;
    int64_t pitch = 0, plane_pos = 0, stage_pos = 0, lds_bytes = 0, plane_src = 0, ngroups = 0, grid = 0;
};

// The plan of the one-image-per-workgroup kernel, or !ok when the shape is
// not one it takes (bf16, 3x3 filter, C a multiple of 32, K of 128, 193 to
// 224 output pixels per image, odd sw*Fh, strips of both stages in LDS, the
// staging items of both variants within the per-thread registers).  Both
// variants take a shape or neither, so that they stage the same strips and
// run the same matrix-core sequence.
ImgPlan plan_image_bf16(const Geometry& g, bool fused);
ImgArgs image_args(const Geometry& g, const ImgPlan& p, const void* src, const void* wf, float* y);
// Repacks w into `scratch` (K*C*Fh*Fw*2 bytes) and launches the convolution.
int launch_conv_bf16_image(const Geometry& g, const ImgPlan& p, bool fused, const void* src,
                           const void* w, void* scratch, float* y, hipStream_t stream);

// ---------------------------------------------------------------------------
// fp32 convolution by bands of output rows (conv_f32_band.hip)
// ---------------------------------------------------------------------------
constexpr int kBandThreads = 256;      // 4 waves
constexpr int kBandChunk = 8;          // input channels per chunk: 4 pairs, one channel per k-slot
constexpr int kBandMaxSeg = 24;        // 64-element parts per channel slot (1536 strip elements)
// LDS floats per channel slot: the longest strip plus 32 banks, so that the
// two k-slots of a pair (adjacent slots) start in different banks
constexpr int kBandSlot = 64 * kBandMaxSeg + 32;
constexpr int kBandStageBytes = kBandChunk * kBandSlot * 4;   // one chunk of strips

// How a workgroup copies strips into LDS.
constexpr int kBandWide = 0;     // window-tensor rows, 16-byte copies (16-byte aligned planes)
constexpr int kBandNarrow = 1;   // window-tensor rows, 4-byte copies
constexpr int kBandGather = 2;   // fused: each strip position gathered from x
constexpr int kBandRaw = 3;      // fused: the band's input rows, zero-padded, 16-byte copies
constexpr int kBandRawGroups = 6;   // raw mode: copies (groups of rows) per channel slot, at most

// Offset that no staging buffer reaches (image slabs are below 2^30 bytes):
// a buffer load from it reads zero.
constexpr uint32_t kBandOutside = 0x40000000u;

struct F32BandArgs {
    const float* src;      // window tensor (unfused) or x (fused)
    const float* wt;       // filter, K x C x Fh x Fw
    float* y;
    int n, c, h, w, k, sh, sw, ph, pw, ho, wo;
    int row_len;           // window-tensor row length L
    int plane_src;         // elements per channel plane of src (Ho*L, or H*W)
    int rows;              // output rows per band
    int nbands;            // bands per image, ceil(Ho / rows)
    int ks;                // waves that split the reduction of one output (4 or 2)
    int nkt;               // groups of (4 / ks) * 32 output channels
    int nchunks;           // C / 8
    int grid;              // workgroups (N * nbands * nkt)
    int xcd_remap;         // place consecutive workgroups on one XCD
    int mode;              // kBandWide, kBandNarrow, kBandGather or kBandRaw
    int slotf;             // small-C kernel: LDS floats per channel slot
    int total;             // small-C kernel: bands (x channel groups) of the layer
    int per_wg;            // small-C kernel: consecutive bands per workgroup
    int rrows, rpitch;     // small-C fused: raw input rows per band, LDS floats per raw row
    int rlpad;             // small-C fused: LDS floats before column 0 of a raw row (zero, >= pw)
    int rawwide, rparts;   // small-C fused: raw rows by 16-byte copies; copies per row
    int rlanes, rrpi;      // band raw mode: 16-byte lanes per raw row (rpitch / 4), rows per copy
    int rgroups;           // band raw mode: copies per channel slot
    int ipb;               // whole images per band (bands of several images), else 1
    FastDiv div_row, div_wo, div_ho;   // by L, by Wo, by Ho
};

// The band of output rows, image and output-channel group of one workgroup.
// A band of several whole images (ipb > 1) is a run of rows [0, nrows) that
// goes on from one image's last row to the next image's first: the images'
// strips sit back to back in a channel slot exactly as consecutive rows do,
// so window reads need no change; copies and stores skip the other channels
// of each image (band_image_skip).
struct BandTile {
    int img, band, kt;     // first image, band of that image (0 for several images)
    int m0, nrows, npix;   // output rows [m0, m0 + nrows), npix = nrows * Wo
    int shift;             // wide copies: strip element 0 sits at slot position shift
    int nimg;              // images the band covers (1, or up to ipb)
};

__host__ __device__ inline BandTile band_tile(const F32BandArgs& a, int bid) {
    BandTile t;
    t.kt = bid % a.nkt;
    const int ib = bid / a.nkt;
    if (a.ipb > 1) {
        t.band = 0;
        t.img = ib * a.ipb;
        t.nimg = a.n - t.img < a.ipb ? a.n - t.img : a.ipb;
        t.m0 = 0;
        t.nrows = t.nimg * a.ho;
    } else {
        t.band = ib % a.nbands;
        t.img = ib / a.nbands;
        t.nimg = 1;
        t.m0 = t.band * a.rows;
        t.nrows = a.ho - t.m0 < a.rows ? a.ho - t.m0 : a.rows;
    }
    t.npix = t.nrows * a.wo;
    t.shift = a.mode == kBandWide ? (t.m0 * a.row_len) & 3 : 0;
    return t;
}

// Image (from the band's first) of band row m (0 for bands of one image).
__host__ __device__ inline int band_row_image(const F32BandArgs& a, int m) {
    return a.ipb > 1 ? (int)fast_div((uint32_t)m, a.div_ho) : 0;
}

// LDS byte address, in stage 0, of the window start of the pixel of `lane`
// in pixel block b, in channel slot `slot`; pixels past the band are
// clamped to its last pixel (computed, never stored).
// Raw mode: the window starts at raw row ml*sh, column n*sw - pw of the
// slot; tap (u, v) adds u*rpitch + v.
__host__ __device__ inline uint32_t band_window(const F32BandArgs& a, const BandTile& t, int fh, int slot, int lane,
                                                int b) {
    int p = b * 32 + (lane & 31);
    if (p > t.npix - 1) p = t.npix - 1;
    const int ml = (int)fast_div((uint32_t)p, a.div_wo), n = p - ml * a.wo;
    if (a.mode == kBandRaw)
        return (uint32_t)(slot * kBandSlot + ml * a.sh * a.rpitch + a.rlpad - a.pw + n * a.sw) * 4u;
    return (uint32_t)(slot * kBandSlot + t.shift + ml * a.row_len + n * a.sw * fh) * 4u;
}

// Source byte offset, within one channel plane of the staging source, of
// part s of a slot copy for `lane`, or kBandOutside (reads zero).  The band's
// strip is the run of window-tensor rows [m0, m0 + nrows) of the plane.
// Wide: elements s*256 + 4*lane .. + 3 of the run, counted from `shift`
// elements before its start (a 16-byte boundary).  Narrow: element
// s*64 + lane of the run.  Gather: run position s*64 + lane, i.e.
// window-tensor element (m, k, u), read from x[m*sh + u - ph][k - pw]
// (zero in the padding).
__host__ __device__ inline uint32_t band_source(const F32BandArgs& a, const BandTile& t, int mode, int fh, int s,
                                                int lane) {
    if (mode == kBandRaw) {
        // copy s: raw rows s*rrpi .. of the band (input rows m0*sh - ph + r),
        // rlanes lanes of 4 floats per row, columns 4*li - rlpad; the pad
        // columns, rows outside the image and rows past rrows read zero
        const int r = s * a.rrpi + lane / a.rlanes, li = lane - (lane / a.rlanes) * a.rlanes;
        const int yy = t.m0 * a.sh - a.ph + r, xx = 4 * li - a.rlpad;
        const bool inside = r < a.rrows && yy >= 0 && yy < a.h && xx >= 0 && xx + 4 <= a.w;
        return inside ? (uint32_t)(yy * a.w + xx) * 4u : kBandOutside;
    }
    // (several images: run element e of image q lies q images of C planes
    // further in the source, i.e. e + q*(C-1)*plane elements)
    const int len = t.nrows * a.row_len;
    const uint32_t skip = (uint32_t)(a.c - 1) * (uint32_t)a.plane_src;
    if (mode == kBandWide) {
        const int e = s * 256 + lane * 4;
        if (e >= t.shift + len) return kBandOutside;
        const int el = t.m0 * a.row_len - t.shift + e;
        const int q = band_row_image(a, (int)fast_div((uint32_t)el, a.div_row));
        return ((uint32_t)el + (uint32_t)q * skip) * 4u;
    }
    const int pos = s * 64 + lane;
    if (mode == kBandNarrow) {
        if (pos >= len) return kBandOutside;
        const int el = t.m0 * a.row_len + pos;
        const int q = band_row_image(a, (int)fast_div((uint32_t)el, a.div_row));
        return ((uint32_t)el + (uint32_t)q * skip) * 4u;
    }
    const int ml = (int)fast_div((uint32_t)pos, a.div_row), rem = pos - ml * a.row_len;
    const int k = rem / fh, u = rem - k * fh;
    const int q = band_row_image(a, t.m0 + ml), mi = t.m0 + ml - q * a.ho;
    const int yy = mi * a.sh + u - a.ph, xx = k - a.pw;
    const bool inside = pos < len && yy >= 0 && yy < a.h && xx >= 0 && xx < a.w;
    return inside ? ((uint32_t)(yy * a.w + xx) + (uint32_t)q * (uint32_t)a.c * (uint32_t)a.plane_src) * 4u
                  : kBandOutside;
}

// Elements of y between pixel p of a band's output-channel plane and where
// it is stored, beyond p itself: the other channels of the images before
// p's (0 for bands of one image).
__host__ __device__ inline uint32_t band_image_skip(const F32BandArgs& a, int p) {
    if (a.ipb == 1) return 0;
    const int q = (int)fast_div(fast_div((uint32_t)p, a.div_wo), a.div_ho);
    return (uint32_t)q * (uint32_t)(a.k - 1) * (uint32_t)(a.ho * a.wo);
}

// LDS byte offset, within a stage, of part `part` of channel slot `slot`
// (256 elements wide, 64 otherwise, rrpi raw rows in raw mode).
__host__ __device__ inline uint32_t band_dest_slot(const F32BandArgs& a, int mode, int slot, int part) {
    const int bytes = mode == kBandWide ? 1024 : mode == kBandRaw ? a.rrpi * a.rpitch * 4 : 256;
    return (uint32_t)(slot * kBandSlot * 4 + part * bytes);
}

// Copy j of wave wv (one wave per SIMD): channel slot 2*wv + (j & 1), part
// j / 2.  (Two waves per SIMD: copy j of wave wv is slot wv, part j.)
__host__ __device__ inline uint32_t band_dest(const F32BandArgs& a, int mode, int wv, int j) {
    return band_dest_slot(a, mode, 2 * wv + (j & 1), j >> 1);
}


// Copies per wave and chunk (two channel slots).
__host__ __device__ constexpr int band_copies(int mode) {
    return mode == kBandWide ? 2 * (kBandMaxSeg / 4) : mode == kBandRaw ? 2 * kBandRawGroups : 2 * kBandMaxSeg;
}

// Raw mode for a fused band convolution of this shape and input, or not:
// rows of x whole 16-byte vectors (W a multiple of 4, x 16-byte aligned),
// a raw row of rlanes 16-byte lanes holding rlpad >= pw zero columns, the
// row and the columns a window reaches, and the band's rows in at most
// kBandRawGroups copies of 64 / rlanes rows each, inside one slot.  Fills
// rrows, rpitch, rlpad, rlanes, rrpi and rgroups.
bool band_raw_mode(const Geometry& g, int rows, const void* x, F32BandArgs* a);

struct F32BandPlan {
    bool ok = false;
    int ks = 0;            // reduction split (4: 32 output channels per workgroup; 2: 64)
    int rows = 0;          // output rows per band
    int nb = 0;            // 32-pixel blocks per band
    int ipb = 1;           // whole images per band (rows = Ho), or 1
    int64_t lds_bytes = 0, grid = 0;
    double eff = 0;        // useful share of the matrix-core work the launch occupies
};

// The plan of the band kernel, or !ok when the shape is not one it takes
// (fp32; 3x3 or 3x5 filter; C a multiple of 16, K of 32 (of 64 with the
// two-way split, 3x3 only); a band of rows, or of several whole images,
// whose strips fit a slot and whose pixels fill 4-7 blocks of 32 (9 or 11-14
// with the two-way split); at most 4 rounds of 256 workgroups unless each
// workgroup has at least 12M multiply-adds to do, and at least 85% of the
// occupied matrix-core work useful after rounding the grid to whole rounds).
// The plan does not depend on fusion, so both variants take a shape or
// neither.
F32BandPlan plan_band_f32(const Geometry& g);
// Whether the band kernels are built for nb pixel blocks with the ks-way split.
bool band_nb_compiled(int ks, int nb);
F32BandArgs band_args_f32(const Geometry& g, const F32BandPlan& p, bool fused, const void* src, const void* w,
                          float* y);
int launch_conv_f32_band(const Geometry& g, const F32BandPlan& p, bool fused, const void* src, const void* w,
                         float* y, hipStream_t stream);

// The band kernel for layers with few input channels (conv_f32_band.hip):
// all C channels' strips of a band in LDS at once (one slot of slotf floats
// per channel, two buffers), 64 output channels per workgroup, the two
// k-slots of an MFMA holding the top and the bottom half of the filter rows,
// two waves per block of 32 output channels splitting the k-steps; one
// persistent workgroup per CU walks through per_wg consecutive bands.
constexpr int kSmallCChannels = 3;          // C the kernels are built for
constexpr int kSmallCWavesPerSimd = 2;      // 8 waves, each half of the band's pixel blocks

// Band bid of the small-C kernel: output-channel group slowest, so that a
// workgroup's run of consecutive bands shares one filter.
__host__ __device__ inline BandTile smallc_tile(const F32BandArgs& a, int bid) {
    BandTile t;
    const int per_kt = a.n * a.nbands;
    t.kt = bid / per_kt;
    const int ib = bid - t.kt * per_kt;
    t.img = ib / a.nbands;
    t.band = ib - t.img * a.nbands;
    t.m0 = t.band * a.rows;
    t.nrows = a.ho - t.m0 < a.rows ? a.ho - t.m0 : a.rows;
    t.npix = t.nrows * a.wo;
    t.shift = a.mode == kBandWide ? (t.m0 * a.row_len) & 3 : 0;
    t.nimg = 1;
    return t;
}

// The reduction of the small-C kernel in k-steps of two elements, one per
// k-slot of the MFMA: first the channel pairs (2p, 2p + 1), slot 0 taking
// channel 2p and slot 1 channel 2p + 1 at the same filter tap (u, v); then,
// for odd C, the last channel with filter rows u and u + Fh - ceil(Fh/2) in
// the two slots, u < ceil(Fh/2), where for odd Fh the middle row comes up in
// both and slot 1's copy has zero weight.  Within a group the slots differ
// by a fixed offset (one channel; Fh - ceil(Fh/2) rows), so one LDS read per
// step serves both.
struct SmallCStep {
    int c, u, v;   // channel, filter row and column this k-slot multiplies
    bool zero;     // zero weight (the repeated middle row)
    bool pair;     // in the channel-pair group
};
__host__ __device__ constexpr int smallc_steps(int c, int fh, int fw) {
    return (c / 2) * fh * fw + (c % 2) * ((fh + 1) / 2) * fw;
}
__host__ __device__ constexpr SmallCStep smallc_step(int c, int fh, int fw, int q, int slot) {
    const int ga = (c / 2) * fh * fw;
    if (q < ga) {
        const int pr = q / (fh * fw), r = q - pr * (fh * fw);
        return SmallCStep{2 * pr + slot, r / fw, r % fw, false, true};
    }
    const int hu = (fh + 1) / 2, r = q - ga, u = r / fw + slot * (fh - hu);
    return SmallCStep{c - 1, u, r % fw, slot == 1 && u < hu, false};
}

// LDS byte offset, within a channel slot, of the window start of the pixel of
// `lane` in pixel block b (the same for both k-slots; the step adds the
// slots' offsets).  Pixels past the band are clamped to its last pixel.
__host__ __device__ inline uint32_t smallc_window(const F32BandArgs& a, const BandTile& t, int fh, int lane, int b) {
    int p = b * 32 + (lane & 31);
    if (p > t.npix - 1) p = t.npix - 1;
    const int ml = (int)fast_div((uint32_t)p, a.div_wo), n = p - ml * a.wo;
    return (uint32_t)(t.shift + ml * a.row_len + n * a.sw * fh) * 4u;
}

// Fused: byte offset, in a raw-row buffer, of the window that lane `lane`
// of pixel block b reads (the zero-padded input row ml*sh, column
// n*sw - pw); filter tap (c, u, v) adds ((c*rrows + u)*rpitch + v) floats.
// Pixels past the band repeat the last.
__host__ __device__ inline uint32_t smallc_raw_window(const F32BandArgs& a, const BandTile& t, int fh, int lane, int b) {
    int p = b * 32 + (lane & 31);
    if (p > t.npix - 1) p = t.npix - 1;
    const int ml = (int)fast_div((uint32_t)p, a.div_wo), n = p - ml * a.wo;
    return (uint32_t)(ml * a.sh * a.rpitch + a.rlpad - a.pw + n * a.sw) * 4u;
}

// Parts (copies of 256 elements wide, 64 otherwise) of one channel slot.
__host__ __device__ inline int smallc_parts(const F32BandArgs& a, const BandTile& t) {
    const int len = t.nrows * a.row_len;
    return a.mode == kBandWide ? (t.shift + len + 255) / 256 : (len + 63) / 64;
}

// The plan of the small-C band kernel, or !ok (fp32; C = 3; 3x3, 7x7 or
// 11x11 filter; K a multiple of 32, in groups of 64; a band of rows whose
// pixels fill 4-7 blocks of 32 and whose three strips (or raw input rows),
// twice, fit with the partial sums in LDS; at least 55% of the occupied
// matrix-core work useful, counting ceil(bands / 256) bands per workgroup
// and the idle half of a last group of 32 channels).  Independent of fusion.
F32BandPlan plan_band_small_c_f32(const Geometry& g);
F32BandArgs band_args_small_c_f32(const Geometry& g, const F32BandPlan& p, bool fused, const void* src,
                                  const void* w, float* y);
int launch_conv_f32_band_small_c(const Geometry& g, const F32BandPlan& p, bool fused, const void* src,
                                 const void* w, float* y, hipStream_t stream);

// Upper bound of the per-channel strip length over all pixel tiles of `bn`
// pixels: a tile spanning D row boundaries reads D*L + (n1-n0)*sw*Fh + Fw*Fh
// elements with n1 - n0 = (pixels - 1) - D*Wo; the bound is linear in D.
inline int64_t strip_bound(const Geometry& g, int bn) {
    const int64_t dmax = (g.wo - 1 + bn - 1) / g.wo;
    auto at = [&](int64_t d) {
        return d * (g.row_len - g.wo * g.sw * g.fh) + (int64_t)(bn - 1) * g.sw * g.fh + g.fw * g.fh;
    };
    return std::max<int64_t>(1, std::max(at(0), at(dmax))) + 1;
}

// Strip capacity: the plain bound plus, for runs of 16-byte chunks of `vc`
// elements (vc = 0: plain layout), the shift of run 0 and the rounding of
// every run to whole chunks.
inline int64_t strip_capacity(const Geometry& g, int bn, int vc) {
    const int64_t cap = strip_bound(g, bn);
    if (vc == 0) return cap;
    const int64_t dmax = (g.wo - 1 + bn - 1) / g.wo;
    const int64_t nseg = std::min<int64_t>(dmax + 1, (bn - 1) / (g.ho * g.wo) + 2);
    return cap + (vc - 1) * (1 + nseg);
}

// Fused fp32 with the per-element expansion (filters of more than three
// rows, or long raw rows): where raw row r of a tile goes in the strips.
// Element xx of the row lands at base + (xx + pw)*fh + i*(row_len - sh) for
// i < cnt (window rows m_lo + i, filter row yy + ph - m*sh), each position
// kept only inside [lo, hi), the run of the row's segment.  The kernel
// computes the entries once per tile; the plan checker replays them.
struct RawRowEntry {
    int base, cnt, lo, hi;
};

__host__ __device__ inline RawRowEntry raw_row_entry(const ConvArgs& a, const TileRuns& tr,
                                                     const RawRows& rr, int r) {
    int sg, yy;
    if (r < rr.r0) {
        sg = 0;
        yy = rr.ylo0 + r;
    } else {
        sg = 1 + (int)fast_div((uint32_t)(r - rr.r0), a.div_rmid);
        if (sg > tr.nseg - 1) sg = tr.nseg - 1;
        yy = a.ylo_mid + (r - rr.r0 - (sg - 1) * a.rmid);
    }
    const SegRun sr = seg_run(sg, tr.nseg, tr.len0, tr.len_mid, tr.len_last, tr.m0, tr.qa0, 0,
                              tr.d_second, tr.d_stride);
    const int m_end = sg == tr.nseg - 1 ? tr.m1 : a.ho - 1;
    const int t = yy + a.ph - a.fh + 1;   // m*sh >= t
    int m_lo = t <= 0 ? 0 : (int)fast_div((uint32_t)(t + a.sh - 1), a.div_sh);
    if (m_lo < sr.m) m_lo = sr.m;
    int m_hi = (int)fast_div((uint32_t)(yy + a.ph), a.div_sh);
    if (m_hi > m_end) m_hi = m_end;
    RawRowEntry e;
    e.base = sr.off + (m_lo - sr.m) * a.row_len + (yy + a.ph - m_lo * a.sh) - sr.q;
    e.cnt = m_hi - m_lo + 1;
    e.lo = sr.off;
    e.hi = sr.off + sr.len;
    return e;
}

// Upper bound of RawRows::rtot over all tiles of `bn` pixels: the window
// rows a tile spans, each segment adding the filter height.
// Upper bound of RawRows::rtot over all tiles of `bn` pixels.  A segment of
// q window rows uses (q - 1)*sh + Fh input rows, and at most H; a tile spans
// at most dmax + 1 window rows in ns segments, so at most
// min(ns*H, (dmax + 1 - ns)*sh + ns*Fh) input rows.
inline int64_t raw_rows_bound(const Geometry& g, int bn) {
    const int64_t dmax = (g.wo - 1 + bn - 1) / g.wo;   // row boundaries crossed
    const int64_t nseg = std::min<int64_t>(dmax + 1, (bn - 1) / (g.ho * g.wo) + 2);
    int64_t best = 0;
    for (int64_t ns = 1; ns <= nseg; ++ns)
        best = std::max(best, std::min<int64_t>(ns * g.h, (dmax + 1 - ns) * g.sh + ns * g.fh));
    return best;
}

// Common launch arguments (everything except the per-dtype chunking).
inline ConvArgs make_conv_args(const Geometry& g, const void* src, const void* w, float* y,
                               int bm) {
    ConvArgs a;
    a.src = src;
    a.w = w;
    a.y = y;
    a.c = (int)g.c; a.h = (int)g.h; a.w_in = (int)g.w; a.k = (int)g.k;
    a.fh = (int)g.fh; a.fw = (int)g.fw; a.sh = (int)g.sh; a.sw = (int)g.sw;
    a.ph = (int)g.ph; a.pw = (int)g.pw;
    a.ho = (int)g.ho; a.wo = (int)g.wo; a.wp = (int)g.wp;
    a.row_len = (int)g.row_len; a.used_len = (int)g.used_len; a.taps = (int)g.taps;
    a.npix = (int)g.npix; a.howo = (int)(g.ho * g.wo);
    a.rc = 1; a.strip_cap = 1; a.kpad = 2; a.tc = 1;
    a.sc = 1; a.fp = 1; a.bm = bm; a.ksplit = 0;
    a.num_jtiles = (int)((g.k + bm - 1) / bm);
    a.div_wo = make_fastdiv((uint32_t)a.wo);
    a.div_ho = make_fastdiv((uint32_t)a.ho);
    a.div_taps = make_fastdiv((uint32_t)a.taps);
    a.div_fw = make_fastdiv((uint32_t)a.fw);
    a.div_row = make_fastdiv((uint32_t)a.row_len);
    a.div_fh = make_fastdiv((uint32_t)a.fh);
    a.div_kpad = make_fastdiv(2);
    a.div_tc2 = make_fastdiv(2);
    a.d_row = kConvThreads / a.row_len;
    const int rem = kConvThreads % a.row_len;
    a.d_k = rem / a.fh;
    a.d_u = rem % a.fh;
    a.e_row = 64 / a.row_len;
    a.e_k = (64 % a.row_len) / a.fh;
    a.e_u = (64 % a.row_len) % a.fh;
    a.stage = 0;
    a.svec = 0;
    a.vchunk = 16 / g.elem;
    a.fvec = 0;
    a.div_fp = make_fastdiv(1);
    a.div_ckmid = make_fastdiv(1);
    a.div_lenmid = make_fastdiv((uint32_t)((g.ho - 1) * g.row_len + g.used_len));
    a.xvec = (g.w & 3) == 0 ? 1 : 0;
    a.raw_pitch = 0;
    a.raw_off = 0;
    a.ylo_mid = (int)std::max<int64_t>(0, -g.ph);
    a.rmid = (int)std::max<int64_t>(0, std::min<int64_t>(g.h, (g.ho - 1) * g.sh - g.ph + g.fh) - a.ylo_mid);
    a.div_w = make_fastdiv((uint32_t)g.w);
    a.div_sh = make_fastdiv((uint32_t)g.sh);
    a.div_rmid = make_fastdiv((uint32_t)std::max(a.rmid, 1));
    a.cl_pitch = a.row_len;
    a.cl_pb = 0;
    a.cl_fpb = 0;
    a.ilv = 0;
    a.fpack = 0;
    return a;
}

}  // namespace im2win
