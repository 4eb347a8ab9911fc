// fp32 im2win convolution on gfx950 matrix cores (Alg. 2 semantics).
//
// The convolution is an implicit GEMM  Y[j][p] = sum_kk F[j][kk] * Win[kk][p]
// over output channels j, output pixels p = (i, m, n) and reduction index
// kk = (r, u, v).  The window tensor stores the window of pixel p, channel r
// as the contiguous run [base(p), base(p) + Fw*Fh) of row (i, r, m), tap
// (u, v) at offset v*Fh + u; horizontally adjacent windows overlap inside
// one strip and are read from the same on-chip copy (the reuse the paper's
// loop order is built around, Sec. III-B).
//
// Workgroup = 4 waves (8 for the generic kernels in the cases launch_cfg
// names) computing a BM (channels) x BN (pixels) tile of Y.
// Pixels are tiled in flattened (i, m, n) order, so a tile reads a few
// window-tensor rows, which for one channel are contiguous in memory (one run
// per image).  Per chunk of input channels:
//   - unfused: the runs and the filter rows are copied straight from global
//     memory into LDS by the global_load_lds DMA path (no register round
//     trip; a wave issues every copy of the chunk, then waits once);
//   - fused: the strips are built in LDS from x, zero padding included
//     (gathers batched eight per thread), the window tensor is never written;
//   - v_mfma_f32_32x32x2f32 runs with A = filter rows (32 channels) and
//     B = window columns (32 pixels); each accumulator register then holds 32
//     consecutive pixels of one output channel, so NCHW stores coalesce.
// The matrix core's two k-slots (lanes 0-31 / 32-63) take either the two
// halves of the channel chunk or the top and bottom filter rows, whichever
// pads the reduction less; either way the second half is the first shifted
// by a constant, so with the filter size known at compile time every tap
// offset is an immediate of the LDS read.
#include "conv_common.h"

#include <cstdio>

namespace im2win {
namespace {

// Input elements are fp32, or bf16 bit patterns widened to fp32 (exact) for
// bf16 problems whose channel-inner tiles do not fit in LDS.
__device__ inline float to_f32(float v) { return v; }
__device__ inline float to_f32(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

typedef __attribute__((address_space(3))) void lds_void;

// Barrier that also publishes the copies this wave issued to LDS by DMA
// (global_load_lds): they complete through the vector-memory counter, which
// the workgroup barrier's own fence does not wait for.
__device__ inline void dma_barrier() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
}

// One wave copies `len` consecutive floats from global memory to LDS (DMA).
__device__ inline void dma_run(const float* g, float* l, int len, int lane) {
    for (int e0 = 0; e0 < len; e0 += 64) {
        if (e0 + lane < len)
            __builtin_amdgcn_global_load_lds(g + e0 + lane, (lds_void*)(l + e0), 4, 0, 0);
    }
}

// Zero the strips of channel slots [c0, c1) over the tile's extent.
__device__ inline void zero_channels(float* S, const ConvArgs& a, const TileRuns& tr, int c0, int c1) {
    for (int c = c0; c < c1; ++c)
        for (int e = threadIdx.x; e < tr.extent; e += (int)blockDim.x) S[c * a.sc + e] = 0.0f;
}

// Stage one channel chunk [r0, r0 + rc_act) of one tile into S (strips,
// stride sc per channel) and F (filter rows, stride fp), issuing copies only:
// fp32 data moves by DMA (global_load_lds) and lands while the previous chunk
// is being multiplied; the caller's next barrier waits for it.
//   F[jj][0 .. rc_act*T)   filter rows in natural (r, u, v) order
//   S[rc][0 .. strip_len)  window-tensor runs (unfused), or the same strip
//                          positions gathered from x, zero where they fall in
//                          the padding (fused)
template <typename TIn, bool FUSED, bool FILTER_ONLY = false>
__device__ inline void stage(float* S, float* F, const ConvArgs& a, const TileRuns& tr, int j0,
                             int r0, int rc_act, int rc_stage) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nw = (int)(blockDim.x >> 6);   // waves (a power of two)
    const int kreal = rc_act * a.taps;
    const int nrows_f = min(a.k - j0, a.bm);
    constexpr bool kDma = sizeof(TIn) == 4;
    if (kDma && a.fpack) {
        // the repacked filter holds this tile's chunk as one block laid out
        // like the LDS rows (zeros past the chunk's taps and past K): 16-byte
        // copies of a contiguous range
        const int nchunks = (a.c + a.rc - 1) / a.rc;
        const float* blk = static_cast<const float*>(a.w) +
                           ((int64_t)(j0 / a.bm) * nchunks + r0 / a.rc) * a.bm * a.fp;
        const int units = (a.bm * a.fp) >> 2;
        for (int c0 = wave * 64; c0 < units; c0 += (int)blockDim.x) {
            const int c = c0 + lane;
            if (c < units) __builtin_amdgcn_global_load_lds(blk + 4 * c, (lds_void*)(F + 4 * c0), 16, 0, 0);
        }
    } else if (kDma && a.fvec) {
        // filter rows are whole 16-byte chunks (C*T and the chunk's rc*T are
        // multiples of 4): one DMA instruction fills 64 consecutive 16-byte
        // chunks of the row-major tile (rows of stride fp, a multiple of 4)
        const float* w = static_cast<const float*>(a.w) + ((int64_t)j0 * a.c + r0) * a.taps;
        const int64_t wrow = (int64_t)a.c * a.taps;
        const int cpr = a.fp >> 2, creal = kreal >> 2;
        const int total = nrows_f * cpr;
        for (int c0 = wave * 64; c0 < total; c0 += (int)blockDim.x) {
            const int c = c0 + lane;
            const int jj = (int)fast_div((uint32_t)c, a.div_fp);
            const int col = c - jj * cpr;
            if (c < total && col < creal)
                __builtin_amdgcn_global_load_lds(w + jj * wrow + 4 * col, (lds_void*)(F + 4 * c0), 16, 0, 0);
        }
    } else if (kDma) {
        // one DMA instruction fills 64 consecutive LDS floats of the row-major
        // tile (rows of stride fp), lane by lane from the matching filter row
        const float* w = static_cast<const float*>(a.w) + ((int64_t)j0 * a.c + r0) * a.taps;
        const int64_t wrow = (int64_t)a.c * a.taps;
        const int total = nrows_f * a.fp;
        for (int e0 = wave * 64; e0 < total; e0 += (int)blockDim.x) {
            const int e = e0 + lane;
            const int jj = (int)fast_div((uint32_t)e, a.div_fp);
            const int col = e - jj * a.fp;
            if (e < total && col < kreal)
                __builtin_amdgcn_global_load_lds(w + jj * wrow + col, (lds_void*)(F + e0), 4, 0, 0);
        }
    } else {
        const TIn* w = static_cast<const TIn*>(a.w);
        for (int jj = wave; jj < nrows_f; jj += nw) {
            const TIn* g = w + ((int64_t)(j0 + jj) * a.c + r0) * a.taps;
            for (int e = lane; e < kreal; e += 64) F[jj * a.fp + e] = to_f32(g[e]);
        }
    }
    // a short last chunk under the channel split is padded with zero channels
    // up to a whole chunk, so that every chunk runs the same MFMA sequence
    if (rc_stage > rc_act) {
        if (!FILTER_ONLY) zero_channels(S, a, tr, rc_act, rc_stage);
        const int nz = (rc_stage - rc_act) * a.taps;
        if (!(kDma && a.fpack))   // (the repacked blocks hold these zeros)
            for (int jj = wave; jj < a.bm; jj += nw)
                for (int e = lane; e < nz; e += 64) F[jj * a.fp + kreal + e] = 0.0f;
    }
    if (FILTER_ONLY) return;
    const TIn* src = static_cast<const TIn*>(a.src);
    const int nseg = tr.nseg, i0 = tr.i0, len0 = tr.len0, len_mid = tr.len_mid,
              len_last = tr.len_last, m0 = tr.m0, qa0 = tr.qa0, d_first = tr.d_first,
              d_second = tr.d_second, d_stride = tr.d_stride;
    if (!FUSED && kDma && a.svec) {
        // 16-byte copies: channel rc's runs fill ck_total consecutive 16-byte
        // chunks of its strip; chunk c belongs to run s and reads from that
        // run's 16-byte-aligned start.  Window-tensor planes are multiples of
        // four elements, so no chunk leaves its plane.
        const float* srcf = reinterpret_cast<const float*>(src);
        const int64_t plane_len = (int64_t)a.ho * a.row_len;
        const int ck0 = tr.ck0, ck_mid = tr.ck_mid, ck_total = tr.ck_total;
        const int start0 = m0 * a.row_len + qa0 - tr.shift0;
        // blocks of 64 chunks of all the chunk's channels, to the waves
        // round-robin (chunks of fewer than four channels keep every wave busy)
        const int nb = (ck_total + 63) >> 6;
        for (int rc = 0; rc < rc_act; ++rc) {
            float* l = S + rc * a.sc;
            // block rc*nb + b goes to wave (rc*nb + b) % nw
            for (int b = (wave - rc * nb) & (nw - 1); b < nb; b += nw) {
                const int c0 = b * 64;
                const int c = c0 + lane;
                int sgi = 0, cs = c;
                if (c >= ck0) {
                    sgi = 1 + (int)fast_div((uint32_t)(c - ck0), a.div_ckmid);
                    if (sgi > nseg - 1) sgi = nseg - 1;
                    cs = c - ck0 - (sgi - 1) * ck_mid;
                }
                const float* g = srcf + ((int64_t)(i0 + sgi) * a.c + r0 + rc) * plane_len +
                                 (sgi == 0 ? start0 : 0) + 4 * cs;
                if (c < ck_total)
                    __builtin_amdgcn_global_load_lds(g, (lds_void*)(l + 4 * c0), 16, 0, 0);
            }
        }
        return;
    }
    const int nruns = rc_act * nseg;
    if (!FUSED && kDma && nruns < nw) {
        // fewer runs than waves (one or two channels): blocks of 64 floats of
        // the runs, counted run after run, to the waves round-robin (block gb
        // goes to wave gb % 4); otherwise whole runs, below
        const float* srcf = reinterpret_cast<const float*>(src);
        int gstart = 0;   // blocks before the current run
        for (int rc = 0; rc < rc_act; ++rc)
            for (int s = 0; s < nseg; ++s) {
                const SegRun sr = seg_run(s, nseg, len0, len_mid, len_last, m0, qa0, d_first, d_second, d_stride);
                const int nbq = (sr.len + 63) >> 6;
                const float* g = srcf + (((int64_t)(i0 + s) * a.c + r0 + rc) * a.ho + sr.m) * a.row_len + sr.q;
                float* l = S + rc * a.sc + sr.off;
                for (int b = (wave - gstart) & (nw - 1); b < nbq; b += nw)
                    if (64 * b + lane < sr.len)
                        __builtin_amdgcn_global_load_lds(g + 64 * b + lane, (lds_void*)(l + 64 * b), 4, 0, 0);
                gstart += nbq;
            }
        return;
    }
    for (int q = wave; q < nruns; q += nw) {
        const int rc = q / nseg, s = q - rc * nseg;
        const SegRun sr = seg_run(s, nseg, len0, len_mid, len_last, m0, qa0, d_first, d_second, d_stride);
        float* l = S + rc * a.sc + sr.off;
        const int len = sr.len;
        if (!FUSED) {
            const TIn* g = src + (((int64_t)(i0 + s) * a.c + r0 + rc) * a.ho + sr.m) * a.row_len + sr.q;
            if (kDma)
                dma_run(reinterpret_cast<const float*>(g), l, len, lane);
            else
                for (int e = lane; e < len; e += 64) l[e] = to_f32(g[e]);
        } else {
            // strip position qa + e of this run is x[(ma + row)*sh + u - ph][k - pw]
            // with (row, k, u) the mixed-radix digits of qa + e over (L, Fh);
            // each lane walks its position in steps of one wave (64)
            const TIn* plane = src + ((int64_t)(i0 + s) * a.c + r0 + rc) * a.h * a.w_in;
            const int pos = sr.q + lane;
            int row = (int)fast_div((uint32_t)pos, a.div_row);
            const int qq = pos - row * a.row_len;
            int kcol = (int)fast_div((uint32_t)qq, a.div_fh);
            int u = qq - kcol * a.fh;
            for (int e0 = 0; e0 < len; e0 += 64) {
                const int e = e0 + lane;
                const int yy = (sr.m + row) * a.sh + u - a.ph;
                const int xx = kcol - a.pw;
                const bool inb = (unsigned)yy < (unsigned)a.h && (unsigned)xx < (unsigned)a.w_in;
                if (e < len) {
                    if (!inb)
                        l[e] = 0.0f;
                    else if (kDma)
                        __builtin_amdgcn_global_load_lds(
                            reinterpret_cast<const float*>(plane) + (int64_t)yy * a.w_in + xx,
                            (lds_void*)(l + e0), 4, 0, 0);
                    else
                        l[e] = to_f32(plane[(int64_t)yy * a.w_in + xx]);
                }
                u += a.e_u;
                if (u >= a.fh) { u -= a.fh; ++kcol; }
                kcol += a.e_k;
                if (kcol >= a.wp) { kcol -= a.wp; ++row; }
                row += a.e_row;
            }
        }
    }
}

// Segment of raw row r of a tile and the input row y it holds.
__device__ inline int raw_segment(int r, const RawRows& rr, int nseg, const ConvArgs& a, int* yy) {
    if (r < rr.r0) {
        *yy = rr.ylo0 + r;
        return 0;
    }
    int s = 1 + (int)fast_div((uint32_t)(r - rr.r0), a.div_rmid);
    if (s > nseg - 1) s = nseg - 1;
    *yy = a.ylo_mid + (r - rr.r0 - (s - 1) * a.rmid);
    return s;
}

// Fused fp32: copy the input rows that channels [r0, r0 + rc_act) of the
// tile use into X[rc][0 .. rtot*W), segment after segment (DMA; the rows of
// one segment are contiguous in x).  16-byte copies when rows are whole
// vectors, else one float per lane.  BLOCKS: the copy units (vectors or
// floats) of all the chunk's channels, in blocks of 64, go to the waves
// round-robin (raw_blocks); expand_raw uses the same assignment, so a wave
// expands what it copied, and chunks of fewer than four channels keep every
// wave busy.  Otherwise wave w copies channels w, w + 4, ... (the expansion
// map reads raw rows only after a barrier).
__device__ inline int raw_blocks(const ConvArgs& a, const RawRows& rr, int* units) {
    *units = a.xvec ? (rr.rtot * a.w_in) >> 2 : rr.rtot * a.w_in;
    return (*units + 63) >> 6;
}

template <bool BLOCKS>
__device__ inline void stage_raw(float* X, const ConvArgs& a, const TileRuns& tr, const RawRows& rr,
                                 int r0, int rc_act) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nw = (int)(blockDim.x >> 6);   // waves (a power of two)
    const float* x = static_cast<const float*>(a.src);
    const int64_t plane = (int64_t)a.h * a.w_in;
    const int nseg = tr.nseg, i0 = tr.i0;
    int units;
    const int nb = raw_blocks(a, rr, &units);
    // units c0 .. c0 + 63 of channel rc
    auto copy_block = [&](int rc, int c0) {
        const float* xp = x + ((int64_t)i0 * a.c + r0 + rc) * plane;
        float* l = X + rc * a.raw_pitch;
        const int c = c0 + lane;
        const int e = a.xvec ? 4 * c : c;
        const int r = (int)fast_div((uint32_t)e, a.div_w);
        int yy;
        const int sg = raw_segment(r, rr, nseg, a, &yy);
        const float* src = xp + (int64_t)sg * a.c * plane + (int64_t)yy * a.w_in + (e - r * a.w_in);
        if (c < units) {
            if (a.xvec)
                __builtin_amdgcn_global_load_lds(src, (lds_void*)(l + 4 * c0), 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds(src, (lds_void*)(l + c0), 4, 0, 0);
        }
    };
    if constexpr (BLOCKS) {
        // block rc*nb + b goes to wave (rc*nb + b) % 4
        for (int rc = 0; rc < rc_act; ++rc)
            for (int b = (wave - rc * nb) & (nw - 1); b < nb; b += nw) copy_block(rc, b * 64);
    } else {
        for (int rc = wave; rc < rc_act; rc += nw)
            for (int c0 = 0; c0 < units; c0 += 64) copy_block(rc, c0);
    }
}

// stage_raw<true> with the source row offsets of the tile read from RS
// (RS[r] = segment * C*H*W + yy*W of raw row r, from the channel's plane in
// the tile's first image; written once per kernel): the same copies, without
// the per-unit segment arithmetic.
__device__ inline void stage_raw_rows(float* X, const int64_t* RS, const ConvArgs& a, const TileRuns& tr,
                                      const RawRows& rr, int r0, int rc_act) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nw = (int)(blockDim.x >> 6);   // waves (a power of two)
    const float* x = static_cast<const float*>(a.src);
    const int64_t plane = (int64_t)a.h * a.w_in;
    int units;
    const int nb = raw_blocks(a, rr, &units);
    for (int rc = 0; rc < rc_act; ++rc) {
        const float* xp = x + ((int64_t)tr.i0 * a.c + r0 + rc) * plane;
        float* l = X + rc * a.raw_pitch;
        // block rc*nb + b goes to wave (rc*nb + b) % nw, as in stage_raw
        for (int b = (wave - rc * nb) & (nw - 1); b < nb; b += nw) {
            const int c0 = b * 64, c = c0 + lane;
            if (c >= units) continue;
            const int e = a.xvec ? 4 * c : c;
            const int r = (int)fast_div((uint32_t)e, a.div_w);
            const float* src = xp + RS[r] + (e - r * a.w_in);
            if (a.xvec)
                __builtin_amdgcn_global_load_lds(src, (lds_void*)(l + 4 * c0), 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds(src, (lds_void*)(l + c0), 4, 0, 0);
        }
    }
}

// Fused fp32: write every raw element x[yy][xx] of channel rc to the strip
// positions that hold it, one per window row m with filter row
// u = yy + ph - m*sh in [0, Fh): position (m, k = xx + pw, u) of the run
// (the on-chip form of the transformation's scatter).  Positions in the
// padding are never written; they were zeroed once.  An odd last chunk under
// the channel split gets one zero channel.
// TRIM: rows end before the input does (trimmed layout), so input columns
// from wp - pw on are skipped.  RT holds the tile's raw-row entries
// (raw_row_entry), written once per kernel.
template <bool TRIM>
__device__ inline void expand_raw_cols(float* S, const float* X, const int4* RT, const ConvArgs& a,
                                       const TileRuns& tr, const RawRows& rr, int rc_act, int rc_stage) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nw = (int)(blockDim.x >> 6);   // waves (a power of two)
    const int vw = a.xvec ? 4 : 1;
    const int dstep = a.row_len - a.sh;   // next window row: one row on, sh filter rows up
    int n;
    const int nb = raw_blocks(a, rr, &n);
    for (int rc = 0; rc < rc_act; ++rc) {
        const float* xl = X + rc * a.raw_pitch;
        float* sl = S + rc * a.sc;
        // block rc*nb + b goes to wave (rc*nb + b) % nw, as in stage_raw
        for (int b = (wave - rc * nb) & (nw - 1); b < nb; b += nw) {
            const int q = b * 64 + lane;
            if (q >= n) continue;
            const int e = q * vw;
            const int r = (int)fast_div((uint32_t)e, a.div_w);
            const int xx = e - r * a.w_in;
            const int4 en = RT[r];   // base, cnt, lo, hi
            // elements of the vector that land in a row
            const int nv = TRIM ? min(vw, a.wp - a.pw - xx) : vw;
            float v[4];
            if (vw == 4) {
                const float4 f = *reinterpret_cast<const float4*>(xl + e);
                v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
            } else {
                v[0] = xl[e];
            }
            int d = en.x + (xx + a.pw) * a.fh;
            const unsigned span = (unsigned)(en.w - en.z);
            for (int i = 0; i < en.y; ++i, d += dstep) {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (j < nv && (unsigned)(d + j * a.fh - en.z) < span) sl[d + j * a.fh] = v[j];
            }
        }
    }
    if (rc_stage > rc_act) zero_channels(S, a, tr, rc_act, rc_stage);
}

__device__ inline void expand_raw(float* S, const float* X, const int4* RT, const ConvArgs& a,
                                  const TileRuns& tr, const RawRows& rr, int rc_act, int rc_stage) {
    if (a.wp - a.pw < a.w_in) expand_raw_cols<true>(S, X, RT, a, tr, rr, rc_act, rc_stage);
    else expand_raw_cols<false>(S, X, RT, a, tr, rr, rc_act, rc_stage);
}

// Fused fp32, small tiles: the destinations of every raw element that a lane
// expands are the same for every chunk and channel, so they are computed once
// per kernel.  Lane l expands raw elements e = l + 64k (k < kExpandK) of each
// of its channels; dst[k][i] is the strip offset (within a channel) of window
// row m_lo + i, or, when that row does not exist or holds no such position,
// the lane's own spare slot among the kExpandSpare positions that end every
// channel's strip (past any window; one slot for many lanes of a store would
// serialise it).  Entries are plain offsets, so a store needs no select.
constexpr int kExpandK = kF32ExpandGroups;
constexpr int kExpandMaxRaw = 64 * kExpandK;   // raw floats per channel
constexpr int kExpandSpare = 64;               // spare strip positions per channel

template <int FH>
struct ExpandMap {
    int dst[kExpandK][FH];
};

template <int FH>
__device__ inline void expand_map_build(ExpandMap<FH>& mp, const ConvArgs& a, const TileRuns& tr,
                                        const RawRows& rr) {
    const int lane = threadIdx.x & 63;
    const int n = rr.rtot * a.w_in;
    const int nseg = tr.nseg;
#pragma unroll
    for (int k = 0; k < kExpandK; ++k) {
        const int e = lane + 64 * k;
#pragma unroll
        for (int i = 0; i < FH; ++i) mp.dst[k][i] = a.sc - kExpandSpare + lane;
        if (e < n) {
            const int r = (int)fast_div((uint32_t)e, a.div_w);
            const int xx = e - r * a.w_in;
            int yy;
            const int sg = raw_segment(r, rr, nseg, a, &yy);
            const SegRun sr = seg_run(sg, nseg, tr.len0, tr.len_mid, tr.len_last, tr.m0, tr.qa0, 0,
                                      tr.d_second, tr.d_stride);
            const int m_end = sg == nseg - 1 ? tr.m1 : a.ho - 1;
            const int t = yy + a.ph - a.fh + 1;
            int m_lo = t <= 0 ? 0 : (int)fast_div((uint32_t)(t + a.sh - 1), a.div_sh);
            if (m_lo < sr.m) m_lo = sr.m;
            int m_hi = (int)fast_div((uint32_t)(yy + a.ph), a.div_sh);
            if (m_hi > m_end) m_hi = m_end;
#pragma unroll
            for (int i = 0; i < FH; ++i) {
                const int m = m_lo + i;
                const int u = yy + a.ph - m * a.sh;
                const int rel = (m - sr.m) * a.row_len + (xx + a.pw) * a.fh + u - sr.q;
                if (m <= m_hi && (unsigned)rel < (unsigned)sr.len && xx + a.pw < a.wp) mp.dst[k][i] = sr.off + rel;
            }
        }
    }
}

template <int FH>
__device__ inline void expand_map_apply(float* S, const float* X, const ExpandMap<FH>& mp,
                                        const ConvArgs& a, const TileRuns& tr, int rc_act, int rc_stage) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nw = (int)(blockDim.x >> 6);   // waves (a power of two)
    const int ngroups = a.raw_pitch >> 6;   // raw pitch is a multiple of 64
    for (int rc = wave; rc < rc_act; rc += nw) {
        const float* xl = X + rc * a.raw_pitch + lane;
        float* sl = S + rc * a.sc;
        float v[kExpandK];   // all reads in flight before the first write (the
                             // buffer ends with kExpandMaxRaw floats of slack)
#pragma unroll
        for (int k = 0; k < kExpandK; ++k) v[k] = xl[64 * k];
#pragma unroll
        for (int k = 0; k < kExpandK; ++k) {
            if (k < ngroups) {
#pragma unroll
                for (int i = 0; i < FH; ++i) sl[mp.dst[k][i]] = v[k];
            }
        }
    }
    if (rc_stage > rc_act) zero_channels(S, a, tr, rc_act, rc_stage);
}

template <int NJ, int NP>
__device__ inline void mfma_step(f32x16 (&acc)[NJ][NP], const float* F, const float* S,
                                 const int (&fl)[NJ], const int (&sl)[NP], int fo, int so,
                                 bool dead) {
    float av[NJ], bv[NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) av[jb] = F[fl[jb] + fo];
#pragma unroll
    for (int pb = 0; pb < NP; ++pb) bv[pb] = S[sl[pb] + so];
    if (dead) {
#pragma unroll
        for (int jb = 0; jb < NJ; ++jb) av[jb] = 0.0f;
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) bv[pb] = 0.0f;
    }
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
            acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
}

// Operands of one filter row u of one channel iteration (FW taps) in registers.
template <int FW, int NJ, int NP>
struct RowRegs {
    float a[NJ][FW];
    float b[NP][FW];
};

// MFMA over one staged chunk: `iters` channels per k-slot.  FH, FW > 0 fix
// the filter size at compile time (tap offsets become immediates).  The
// reduction is walked in groups of one filter row (FW taps); the operands of
// the next group are read from LDS into a second register set before the
// matrix-core instructions of the current group are issued, so LDS latency is
// hidden behind the MFMAs of the same wave.  ROWS: the k-slots are split by
// filter rows (the second k-slot has no row left when Fh is odd: zeroed).
struct NoHook {
    __device__ void operator()(int) const {}
};

// `hook(g)` runs after the matrix-core instructions of group g have been
// issued (the copies of the next chunk are issued there, so they overlap
// the MFMAs).
template <int FH, int FW, bool ROWS, int NJ, int NP, typename Hook = NoHook>
__device__ inline void compute_chunk(f32x16 (&acc)[NJ][NP], const float* F, const float* S,
                                     const ConvArgs& a, const int (&fl)[NJ], const int (&sl)[NP],
                                     int kl, int iters, Hook&& hook = Hook()) {
    if constexpr (FH > 0 && FW > 0) {
        constexpr int T = FH * FW, U0 = (FH + 1) / 2;
        constexpr int UEND = ROWS ? U0 : FH;
        const int ng = iters * UEND;
        const int sc = a.sc;
        RowRegs<FW, NJ, NP> r0, r1;
        auto load = [&](RowRegs<FW, NJ, NP>& r, int g) {
            const int it = g / UEND, u = g - it * UEND;
            const int fo = it * T + u * FW, so = it * sc + u;
#pragma unroll
            for (int v = 0; v < FW; ++v) {
#pragma unroll
                for (int jb = 0; jb < NJ; ++jb) r.a[jb][v] = F[fl[jb] + fo + v];
#pragma unroll
                for (int pb = 0; pb < NP; ++pb) r.b[pb][v] = S[sl[pb] + so + v * FH];
            }
        };
        auto mma = [&](RowRegs<FW, NJ, NP>& r, int g) {
            bool dead = false;
            if constexpr (ROWS && (FH & 1)) dead = kl && (g % UEND == UEND - 1);
#pragma unroll
            for (int v = 0; v < FW; ++v) {
                float av[NJ], bv[NP];
#pragma unroll
                for (int jb = 0; jb < NJ; ++jb) av[jb] = dead ? 0.0f : r.a[jb][v];
#pragma unroll
                for (int pb = 0; pb < NP; ++pb) bv[pb] = dead ? 0.0f : r.b[pb][v];
#pragma unroll
                for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
                    for (int pb = 0; pb < NP; ++pb)
                        acc[jb][pb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[jb], bv[pb], acc[jb][pb], 0, 0, 0);
            }
        };
        if (ng <= 0) return;
        load(r0, 0);
        int g = 0;
        for (; g + 2 <= ng; g += 2) {
            load(r1, g + 1);
            mma(r0, g);
            hook(g);
            if (g + 2 < ng) load(r0, g + 2);
            mma(r1, g + 1);
            hook(g + 1);
        }
        if (g < ng) {
            mma(r0, g);
            hook(g);
        }
    } else {
        const int fh = a.fh, fw = a.fw, T = fh * fw, u0 = (fh + 1) >> 1;
        const int uend = ROWS ? u0 : fh;
        for (int it = 0; it < iters; ++it) {
            const int fo = it * T, so = it * a.sc;
            for (int u = 0; u < uend; ++u) {
                const bool dead = ROWS && kl && (u + u0 >= fh);
                for (int v = 0; v < fw; ++v)
                    mfma_step<NJ, NP>(acc, F, S, fl, sl, fo + u * fw + v, so + v * fh + u, dead);
                hook(it * uend + u);
            }
        }
    }
}

// MODE: 0 unfused; 1 fused (the strips of the chunk are gathered or
// expanded after the MFMAs); 2 fused fp32 with the expansion map and
// double-buffered raw rows (filters of up to 3 rows, small tiles);
// 3 unfused with 16-byte strips and filter rows whose copies are issued from
// inside the MFMA loop, from per-lane offsets computed once; 4 as 2, with the
// filter-row and raw-row copies from per-lane offsets computed once (whole
// chunks, 16-byte filter rows).

// MODE 3 copies of one tile: the 16-byte strip copies of one channel and the
// filter-row copies of one whole chunk, as in stage(), from per-lane byte
// offsets that hold for every chunk and channel but for the channel offset
// (kIlvNone: the lane has no copy in that slot).  Bases are wave-uniform and
// offsets 32-bit, so each copy is one scalar-base load with a vector offset.
constexpr uint32_t kIlvNone = 0xffffffffu;

struct IlvCopies {
    const char* s_base = nullptr;  // channel 0 of the tile's first image
    const char* f_base = nullptr;  // channel 0 of the tile's first filter
    uint32_t s_off[kIlvSlots];
    uint32_t f_off[kIlvSlots];
    int ck_total = 0, f_total = 0;

    __device__ void init(const ConvArgs& a, const TileRuns& tr, int j0) {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int64_t plane = (int64_t)a.ho * a.row_len;
        ck_total = tr.ck_total;
        s_base = static_cast<const char*>(a.src) + 4 * (int64_t)tr.i0 * a.c * plane;
        const int start0 = tr.m0 * a.row_len + tr.qa0 - tr.shift0;
#pragma unroll
        for (int i = 0; i < kIlvSlots; ++i) {
            const int c = 64 * i + lane;
            int sgi = 0, cs = c;
            if (c >= tr.ck0) {
                sgi = 1 + (int)fast_div((uint32_t)(c - tr.ck0), a.div_ckmid);
                if (sgi > tr.nseg - 1) sgi = tr.nseg - 1;
                cs = c - tr.ck0 - (sgi - 1) * tr.ck_mid;
            }
            const uint32_t e = (uint32_t)(sgi * a.c * (int)plane + (sgi == 0 ? start0 : 0) + 4 * cs);
            s_off[i] = c < ck_total ? 4 * e : kIlvNone;
        }
        f_base = static_cast<const char*>(a.w) + 4 * (int64_t)j0 * a.c * a.taps;
        const int cpr = a.fp >> 2, creal = (a.rc * a.taps) >> 2;
        f_total = min(a.k - j0, a.bm) * cpr;
#pragma unroll
        for (int i = 0; i < kIlvSlots; ++i) {
            const int c = wave * 64 + kConvThreads * i + lane;
            const int jj = (int)fast_div((uint32_t)c, a.div_fp);
            const int col = c - jj * cpr;
            f_off[i] = c < f_total && col < creal ? (uint32_t)(4 * (jj * a.c * a.taps + 4 * col)) : kIlvNone;
        }
    }
    // the filter part of init() alone (the fused kernel stages no strips)
    __device__ void init_filter(const ConvArgs& a, int j0) {
        const int lane = threadIdx.x & 63;
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        f_base = static_cast<const char*>(a.w) + 4 * (int64_t)j0 * a.c * a.taps;
        const int cpr = a.fp >> 2, creal = (a.rc * a.taps) >> 2;
        f_total = min(a.k - j0, a.bm) * cpr;
#pragma unroll
        for (int i = 0; i < kIlvSlots; ++i) {
            const int c = wave * 64 + kConvThreads * i + lane;
            const int jj = (int)fast_div((uint32_t)c, a.div_fp);
            const int col = c - jj * cpr;
            f_off[i] = c < f_total && col < creal ? (uint32_t)(4 * (jj * a.c * a.taps + 4 * col)) : kIlvNone;
        }
    }
    // filter rows of the whole chunk starting at channel r0 into F
    __device__ void filter(float* F, const ConvArgs& a, int r0) const {
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const char* b = f_base + 4 * (int64_t)r0 * a.taps;
#pragma unroll
        for (int i = 0; i < kIlvSlots; ++i) {
            uint32_t o = f_off[i];
            asm volatile("" : "+v"(o));  // widened here, not held widened across the loop
            if (kConvThreads * i < f_total && o != kIlvNone)
                __builtin_amdgcn_global_load_lds(reinterpret_cast<const float*>(b + o),
                                                 (lds_void*)(F + 4 * (wave * 64 + kConvThreads * i)), 16, 0, 0);
        }
    }
    // strip of channel r0 + rc into its LDS slot in S
    __device__ void strips(float* S, const ConvArgs& a, int rc, int r0) const {
        const char* b = s_base + 4 * (int64_t)(r0 + rc) * a.ho * a.row_len;
        float* l = S + rc * a.sc;
#pragma unroll
        for (int i = 0; i < kIlvSlots; ++i) {
            uint32_t o = s_off[i];
            asm volatile("" : "+v"(o));
            if (64 * i < ck_total && o != kIlvNone)
                __builtin_amdgcn_global_load_lds(reinterpret_cast<const float*>(b + o),
                                                 (lds_void*)(l + 4 * 64 * i), 16, 0, 0);
        }
    }
};

// MODE 4 raw-row copies: the byte offsets of this lane's copy units of one
// channel's raw rows from that channel's plane in the tile's first image
// (the same for every channel), computed once per kernel.  stage_raw<false>
// issues the same copies with the offsets worked out per chunk.
struct RawCopies {
    uint32_t off[kExpandK];
    int units = 0;
    __device__ void init(const ConvArgs& a, const TileRuns& tr, const RawRows& rr) {
        const int lane = threadIdx.x & 63;
        const int64_t plane = (int64_t)a.h * a.w_in;
        raw_blocks(a, rr, &units);
#pragma unroll
        for (int k = 0; k < kExpandK; ++k) {
            const int c = 64 * k + lane;
            const int e = a.xvec ? 4 * c : c;
            const int r = (int)fast_div((uint32_t)e, a.div_w);
            int yy;
            const int sg = raw_segment(r, rr, tr.nseg, a, &yy);
            const int64_t o = (int64_t)sg * a.c * plane + (int64_t)yy * a.w_in + (e - r * a.w_in);
            off[k] = c < units ? (uint32_t)(4 * o) : kIlvNone;
        }
    }
    // channels r0 + wave, r0 + wave + 4, ... of the chunk into X
    __device__ void copy(float* X, const ConvArgs& a, int i0, int r0, int rc_act) const {
        const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        const int64_t plane = (int64_t)a.h * a.w_in;
        for (int rc = wave; rc < rc_act; rc += 4) {
            const char* b = reinterpret_cast<const char*>(static_cast<const float*>(a.src) +
                                                          ((int64_t)i0 * a.c + r0 + rc) * plane);
            float* l = X + rc * a.raw_pitch;
#pragma unroll
            for (int k = 0; k < kExpandK; ++k) {
                uint32_t o = off[k];
                asm volatile("" : "+v"(o));   // widened here, not held widened across the loop
                if (64 * k < units && o != kIlvNone) {
                    if (a.xvec)
                        __builtin_amdgcn_global_load_lds(reinterpret_cast<const float*>(b + o),
                                                         (lds_void*)(l + 4 * 64 * k), 16, 0, 0);
                    else
                        __builtin_amdgcn_global_load_lds(reinterpret_cast<const float*>(b + o),
                                                         (lds_void*)(l + 64 * k), 4, 0, 0);
                }
            }
        }
    }
};

// NT threads: 256 (4 waves), or 512 (8 waves, two per SIMD) for the generic
// modes 0 and 1 when the tile's LDS leaves room for one workgroup per CU.
template <typename TIn, int FH, int FW, bool ROWS, int BM, int BN, int TJ, int TP, int MODE, int NT = kConvThreads>
__global__ __launch_bounds__(NT) void conv_f32_kernel(ConvArgs a) {
    constexpr bool FUSED = MODE == 1 || MODE == 2 || MODE == 4;
    constexpr bool ILV = MODE == 3;
    // MODE 4: MODE 2 with the filter-row and raw-row copies from per-lane
    // offsets computed once
    constexpr bool FASTCP = MODE == 4;
    static_assert((BM / TJ) * (BN / TP) == NT / 64, "one wave per TJ x TP block");
    static_assert(NT == kConvThreads || MODE == 0 || MODE == 1, "8 waves only for the generic modes");
    constexpr int NJ = TJ / 32, NP = TP / 32;
    constexpr int WAVES_P = BN / TP;

    extern __shared__ __align__(16) unsigned char smem[];
    float* S = reinterpret_cast<float*>(smem);   // stage s: S + s*stage, F + s*stage
    float* F = S + a.rc * a.sc;

    const int jtile = blockIdx.x % a.num_jtiles;
    const int ptile = blockIdx.x / a.num_jtiles;
    const int j0 = jtile * BM;

    TileRuns tr;
    tr.init(ptile, BN, a);

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wj = wave / WAVES_P, wp_ = wave % WAVES_P;
    const int l32 = lane & 31, kl = lane >> 5;

    // Per-lane LDS bases.  The second k-slot (kl = 1) is the first shifted by
    // half a channel chunk, or by the top half of the filter rows.
    const int fh = FH > 0 ? FH : a.fh, fw = FW > 0 ? FW : a.fw;
    const int u0 = (fh + 1) >> 1;
    const int half_full = a.rc >> 1;
    const int df = ROWS ? u0 * fw : half_full * fh * fw;
    const int ds = ROWS ? u0 : half_full * a.sc;
    int sl[NP];
    int64_t yoff[NP];
    bool pvalid[NP];
#pragma unroll
    for (int pb = 0; pb < NP; ++pb) {
        int p = tr.p0 + wp_ * TP + pb * 32 + l32;
        pvalid[pb] = p <= tr.plast;
        if (!pvalid[pb]) p = tr.p0;
        sl[pb] = pixel_base(tr, a, p, &yoff[pb]) + kl * ds;
    }
    int fl[NJ];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb) fl[jb] = (wj * TJ + jb * 32 + l32) * a.fp + kl * df;

    f32x16 acc[NJ][NP];
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[jb][pb][v] = 0.0f;

    // Two LDS stages: while chunk c is multiplied out of one, the copies of
    // chunk c+1 land in the other.  One barrier per chunk: it waits for the
    // copies of chunk c (vmcnt 0 in every wave) and for every wave to be done
    // with chunk c-1, whose stage the copies of chunk c+1 then overwrite.
    //
    // Fused fp32 (RAW): the chunk's input rows are copied to LDS (X) instead
    // and expanded into the strips after a second barrier; the copies of
    // chunk c+1 land while chunk c is multiplied.  The strips' padding
    // positions are zeroed once and never written again.
    constexpr bool RAW = FUSED && sizeof(TIn) == 4;
    const int nchunks = (a.c + a.rc - 1) / a.rc;
    float* X = S + a.raw_off;
    RawRows rr{};
    // the map holds FH destinations per element: kept for filters of up to
    // three rows (larger ones expand with the per-element decode)
    constexpr bool use_map = RAW && (MODE == 2 || MODE == 4);
    static_assert(!use_map || (FH > 0 && FH <= 3), "expansion map for filters of up to 3 rows");
    constexpr int FHM = use_map ? FH : 1;
    ExpandMap<FHM> emap;
    // With the map the raw rows are double-buffered (chunk k in
    // X + (k % 2) * rc * raw_pitch): the copies of chunk c+2 land while chunk
    // c+1 is expanded, so the expansion needs no wait of its own and runs
    // ahead of the MFMAs of chunk c, all within one barrier interval.
    // (selected by arithmetic on the LDS base: a pointer picked from an array
    // loses its address space, and reads through it become flat loads that
    // wait for every copy in flight)
    // without the map: the raw-row entries of the tile after the raw rows
    int4* RT = reinterpret_cast<int4*>(X + a.rc * a.raw_pitch);
    // and their source row offsets (at most raw_pitch / W rows each)
    int64_t* RS = reinterpret_cast<int64_t*>(RT + a.raw_pitch / a.w_in);
    const int xstride = a.rc * a.raw_pitch + kExpandMaxRaw;
    auto Xb = [&](int k) { return X + (k & 1) * xstride; };
    IlvCopies ilv;
    RawCopies rcp;
    {
        const int rc_act = min(a.rc, a.c);
        const int rc_stage = ROWS ? rc_act : a.rc;
        if constexpr (RAW) {
            rr = raw_rows(tr, a);
            for (int sg = 0; sg < 2; ++sg)
                for (int e = threadIdx.x; e < a.rc * a.sc; e += (int)blockDim.x) S[sg * a.stage + e] = 0.0f;
            if constexpr (FASTCP) {
                // whole chunks only: rc_act = rc_stage = rc
                ilv.init_filter(a, j0);
                rcp.init(a, tr, rr);
                rcp.copy(X, a, tr.i0, 0, a.rc);
                if (nchunks > 1) rcp.copy(Xb(1), a, tr.i0, a.rc, a.rc);
                ilv.filter(F, a, 0);
            } else {
                stage_raw<!use_map>(X, a, tr, rr, 0, rc_act);
                if (use_map && nchunks > 1) stage_raw<false>(Xb(1), a, tr, rr, a.rc, min(a.rc, a.c - a.rc));
                stage<TIn, FUSED, true>(S, F, a, tr, j0, 0, rc_act, rc_stage);
            }
            if (use_map) expand_map_build<FHM>(emap, a, tr, rr);
            else
                for (int r = threadIdx.x; r < rr.rtot; r += (int)blockDim.x) {
                    const RawRowEntry en = raw_row_entry(a, tr, rr, r);
                    RT[r] = make_int4(en.base, en.cnt, en.lo, en.hi);
                    int yy;
                    const int sg = raw_segment(r, rr, tr.nseg, a, &yy);
                    RS[r] = (int64_t)sg * a.c * ((int64_t)a.h * a.w_in) + (int64_t)yy * a.w_in;
                }
            dma_barrier();   // zeros and row entries written, raw rows of chunk 0 (and 1) landed
            if (use_map) expand_map_apply<FHM>(S, X, emap, a, tr, rc_act, rc_stage);
            else expand_raw(S, X, RT, a, tr, rr, rc_act, rc_stage);
        } else {
            stage<TIn, FUSED>(S, F, a, tr, j0, 0, rc_act, rc_stage);
        }
    }
    if constexpr (ILV) ilv.init(a, tr, j0);

    for (int ch = 0; ch < nchunks; ++ch) {
        const int r0 = ch * a.rc;
        const int rc_act = min(a.rc, a.c - r0);
        const float* Sc = S + (ch & 1) * a.stage;
        const float* Fc = F + (ch & 1) * a.stage;
        const int r1 = r0 + a.rc;
        const int rc1 = min(a.rc, a.c - r1);
        const int rc_stage1 = ROWS ? rc1 : a.rc;
        const int off = ((ch + 1) & 1) * a.stage;
        dma_barrier();
        // MODE 3: a whole next chunk is copied from inside the MFMA loop (its
        // plans have whole chunks only, so no chunk is staged here)
        const bool ilv_next = ILV && ch + 1 < nchunks;
        if (!ILV && ch + 1 < nchunks) {
            if constexpr (FASTCP) {
                // whole chunks only (the plan asks C % rc == 0)
                ilv.filter(F + off, a, r1);
                if (ch + 2 < nchunks) rcp.copy(Xb(ch), a, tr.i0, r1 + a.rc, a.rc);
                expand_map_apply<FHM>(S + off, Xb(ch + 1), emap, a, tr, rc1, rc_stage1);
            } else if constexpr (RAW) {
                stage<TIn, FUSED, true>(S + off, F + off, a, tr, j0, r1, rc1, rc_stage1);
                if (use_map) {
                    // copies of chunk c+2; expansion of chunk c+1, whose copies the barrier published
                    if (ch + 2 < nchunks) stage_raw<false>(Xb(ch), a, tr, rr, r1 + a.rc, min(a.rc, a.c - r1 - a.rc));
                    expand_map_apply<FHM>(S + off, Xb(ch + 1), emap, a, tr, rc1, rc_stage1);
                } else {
                    stage_raw_rows(X, RS, a, tr, rr, r1, rc1);
                }
            } else {
                stage<TIn, FUSED>(S + off, F + off, a, tr, j0, r1, rc1, rc_stage1);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        // wave w copies channels w, w + 4, ...: one channel per row group
        auto hook = [&](int g) {
            if constexpr (ILV) {
                if (ilv_next) {
                    const int rc = 4 * g + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
                    if (g == 0) ilv.filter(F + off, a, r1);
                    if (rc < rc1) ilv.strips(S + off, a, rc, r1);
                }
            }
        };
        if (ROWS) compute_chunk<FH, FW, true, NJ, NP>(acc, Fc, Sc, a, fl, sl, kl, rc_act, hook);
        else compute_chunk<FH, FW, false, NJ, NP>(acc, Fc, Sc, a, fl, sl, kl, half_full, hook);
        if constexpr (ILV) {
            if (ilv_next) {
                const int ng = ROWS ? rc_act * ((FH + 1) / 2) : half_full * FH;
                for (int rc = 4 * ng + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); rc < rc1; rc += 4) ilv.strips(S + off, a, rc, r1);
            }
        }
        if constexpr (RAW) {
            // Without the map: a wave expands the raw-row blocks it copied
            // itself (the same round-robin assignment), so waiting for its
            // own copies is enough; the next barrier publishes the strips.
            if (!use_map && ch + 1 < nchunks) {
                __builtin_amdgcn_sched_barrier(0);
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                expand_raw(S + off, X, RT, a, tr, rr, rc1, rc_stage1);
            }
        }
    }

    // D[row][col]: col = lane%32 (pixel), row = 8*(v/4) + 4*(lane/32) + v%4 (channel)
#pragma unroll
    for (int jb = 0; jb < NJ; ++jb)
#pragma unroll
        for (int pb = 0; pb < NP; ++pb) {
            if (!pvalid[pb]) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int j = j0 + wj * TJ + jb * 32 + 8 * (v >> 2) + 4 * kl + (v & 3);
                if (j < a.k) a.y[yoff[pb] + (int64_t)j * a.howo] = acc[jb][pb][v];
            }
        }
}

// fp32 filters whose chunk rows are not whole 16-byte vectors (rc*Fh*Fw not
// a multiple of 4): w (K x C x Fh x Fw) rewritten into one block per (tile of
// bm output channels, chunk of rc input channels), each laid out exactly like
// the tile's LDS filter rows: row jj holds the chunk's rc*Fh*Fw taps of output
// channel j0 + jj, then zeros up to the row stride fp; rows past K are zero.
// The convolution then stages a chunk with 16-byte copies of one block.
__global__ __launch_bounds__(256) void pack_filter_f32_kernel(const float* __restrict__ w, float* __restrict__ wp,
                                                              int k, int c, int taps, int bm, int rc, int fp,
                                                              int nchunks, int64_t total) {
    const int64_t per_blk = (int64_t)bm * fp;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        const int64_t blk = i / per_blk;
        const int e = (int)(i - blk * per_blk);
        const int jj = e / fp, col = e - jj * fp;
        const int jt = (int)(blk / nchunks), ch = (int)(blk - (int64_t)jt * nchunks);
        const int j = jt * bm + jj, r0 = ch * rc;
        const int kreal = min(rc, c - r0) * taps;
        wp[i] = (j < k && col < kreal) ? w[((int64_t)j * c + r0) * taps + col] : 0.0f;
    }
}

// LDS floats of the raw rows of the fused fp32 kernel: with the expansion
// map (filters of up to 3 rows, raw rows of up to kExpandMaxRaw floats) two
// buffers, each with kExpandMaxRaw floats of slack for the map's reads;
// without it one buffer and, per raw row of the tile (at most raw_pitch / W),
// its expansion entry (4 ints) and its source offset (one int64).
int64_t raw_floats(int fh, int rc, int64_t raw_pitch, int64_t w) {
    if (fh <= 3 && raw_pitch <= kExpandMaxRaw) return 2 * (rc * raw_pitch + kExpandMaxRaw);
    return rc * raw_pitch + 6 * (raw_pitch / w);
}

template <typename TIn, int FH, int FW, bool ROWS, int BM, int BN, int TJ, int TP>
void launch_cfg(const ConvArgs& a, int64_t blocks, int64_t lds, bool fused, hipStream_t stream) {
    auto kern = conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ, TP, 0>;
    constexpr int kIlvMode = sizeof(TIn) == 4 && FH > 0 ? 3 : 0;
    bool generic = true;   // mode 0 or 1
    if (!fused && a.svec && a.fvec && a.ilv) {
        kern = conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ, TP, kIlvMode>;
        generic = kIlvMode == 0;
    }
    if (fused) kern = conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ, TP, 1>;
    if constexpr (sizeof(TIn) == 4 && FH > 0 && FH <= 3)
        if (fused && a.raw_pitch <= kExpandMaxRaw) {
            kern = a.ilv ? conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ, TP, 4>
                         : conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ, TP, 2>;
            generic = false;
        }
    if (fused && sizeof(TIn) == 4) lds += raw_floats(a.fh, a.rc, a.raw_pitch, a.w_in) * 4;
    // 8 waves of half the wave tile: for one workgroup per CU (two waves per
    // SIMD instead of one), and for the generic fused kernel, whose staging
    // and expansion the extra waves hide (measured faster on every layer it
    // runs; the unfused generic kernel gained nothing at two workgroups per CU)
    constexpr int TJ8 = TJ >= 64 ? TJ / 2 : TJ, TP8 = TJ >= 64 ? TP : TP / 2;
    int threads = kConvThreads;
    if constexpr (TJ8 >= 32 && TP8 >= 32 && (BM / TJ8) * (BN / TP8) == 8)
        if (generic && (fused || lds > kConvLdsPipelinedBytes)) {
            kern = fused ? conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ8, TP8, 1, 512>
                         : conv_f32_kernel<TIn, FH, FW, ROWS, BM, BN, TJ8, TP8, 0, 512>;
            threads = 512;
        }
    if (lds > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(threads), (size_t)lds, stream, a);
}

template <typename TIn, int FH, int FW, bool ROWS>
void launch_tile_split(const ConvPlan& p, const ConvArgs& a, int64_t blocks, bool fused,
                       hipStream_t stream) {
    if (p.bm == 64 && p.bn == 256) launch_cfg<TIn, FH, FW, ROWS, 64, 256, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bm == 128) launch_cfg<TIn, FH, FW, ROWS, 128, 128, 64, 64>(a, blocks, p.lds_bytes, fused, stream);
    else if (p.bn == 128) launch_cfg<TIn, FH, FW, ROWS, 64, 128, 32, 64>(a, blocks, p.lds_bytes, fused, stream);
    else launch_cfg<TIn, FH, FW, ROWS, 64, 64, 32, 32>(a, blocks, p.lds_bytes, fused, stream);
}

template <typename TIn, int FH, int FW>
void launch_tile(const ConvPlan& p, const ConvArgs& a, int64_t blocks, bool fused,
                 hipStream_t stream) {
    if (p.split) launch_tile_split<TIn, FH, FW, true>(p, a, blocks, fused, stream);
    else launch_tile_split<TIn, FH, FW, false>(p, a, blocks, fused, stream);
}

// LDS of one workgroup: two pipeline stages, each holding the strips of rc
// channels (stride sc) and bm filter rows (stride fp, odd so that 32
// consecutive rows fall in different banks), with slack for the reads past
// the last tap that a dead k-slot makes.
int64_t f32_layout(const Geometry& g, int bm, int rc, int64_t cap, bool fvec, int split,
                   int64_t* sc, int64_t* fp, int64_t* stage) {
    *sc = (cap + g.fh + 3) & ~int64_t(3);
    // fused fp32 with filters of up to 3 rows: spare expansion slots per strip
    if (g.elem == 4 && g.fh <= 3) *sc += kExpandSpare;
    // channel split: the second k-slot reads (rc/2)*sc floats after the first;
    // (rc/2)*sc = 32 mod 64 puts the two half-waves' window reads on
    // disjoint banks (all 64 lanes conflict-free for an odd pixel stride)
    if (!split) {
        const int64_t half = rc / 2;
        for (int i = 0; i < 16; ++i) {
            if ((half * (*sc + 4 * i)) % 64 == 32) {
                *sc += 4 * i;
                break;
            }
        }
    }
    *fp = (int64_t)rc * g.taps + g.fw + 1;
    if (fvec) {
        // 16-byte rows: a multiple of 4 floats, and not of 8, so that 32
        // consecutive rows spread over 8 banks (4-way, not 8-way, conflicts)
        *fp = (*fp + 3) & ~int64_t(3);
        if ((*fp & 7) == 0) *fp += 4;
    } else if ((*fp & 1) == 0) {
        ++*fp;   // odd stride: 32 consecutive rows fall in 32 banks
    }
    *stage = ((int64_t)rc * *sc + (int64_t)bm * *fp + g.fw + 4 + 3) & ~int64_t(3);
    return 2 * *stage * 4;
}

// Filter rows can be staged by 16-byte copies when every row of every
// channel chunk starts on a 16-byte boundary.
bool filter_vec(const Geometry& g, int rc) {
    return g.elem == 4 && ((g.c * g.taps) & 3) == 0 && ((rc * g.taps) & 3) == 0;
}

// Strips can be staged by 16-byte copies when a window-tensor plane is a
// whole number of 16-byte chunks (fp32: Ho*Wp*Fh divisible by 4).
bool strips_vec(const Geometry& g) { return g.elem == 4 && ((g.ho * g.row_len) & 3) == 0; }

// LDS floats per channel for the raw input rows of a fused fp32 tile.
// (a multiple of 64: the expansion map reads whole groups of 64)
int64_t raw_pitch_f32(const Geometry& g, int bn) {
    return (raw_rows_bound(g, bn) * g.w + 63) & ~int64_t(63);
}

// Zero reduction slots each way of splitting the two k-slots adds: one zero
// channel in total (odd C, channel halves) or one zero filter row per channel
// (odd Fh, row halves).
int choose_split(const Geometry& g) {
    const int64_t chan = (g.c & 1) ? g.taps : 0;
    const int64_t rows = (g.fh & 1) ? g.c * g.fw : 0;
    return rows < chan ? 1 : 0;
}

}  // namespace

// compute units of the MI355X (gfx950), for the tile-count cost below
constexpr int64_t kCUs = 256;

ConvPlan plan_conv_f32(const Geometry& g) {
    // Every tile shape that fits is costed and the cheapest is taken.  The
    // cost of a shape is the work of one tile (bm x bn outputs over the whole
    // reduction, padding included) times the number of tiles the busiest CU
    // runs, ceil(tiles / 256), divided by the shape's relative matrix-core
    // efficiency (measured on the 3x3 to 11x11 layers: a 64x256 tile keeps
    // four 32x32 accumulators per wave and stages the filter least often; the
    // 64x64 tile has one accumulator per wave).  A CU that runs only one tile
    // has one wave per SIMD and reaches about half the rate, so a busiest-CU
    // count of one costs double.  Both pipeline stages together are sized for
    // 80 KB of LDS (two workgroups per CU); only shapes that fit nothing there
    // use up to the full 160 KB.
    struct Cand { TileCfg t; double eff; };
    const Cand cands[] = {{{64, 256}, 1.0}, {{128, 128}, 0.85}, {{64, 128}, 0.87}, {{64, 64}, 0.7}};
    const int split = choose_split(g);
    const int step = split ? 1 : 2;
    const int64_t rc_max = std::min<int64_t>(split ? g.c : ((g.c + 1) & ~int64_t(1)), 32);
    for (const int64_t budget : {int64_t(kConvLdsPipelinedBytes), int64_t(kConvLdsMaxBytes)}) {
        ConvPlan best;
        double best_cost = 0.0;
        for (const Cand& cd : cands) {
            const TileCfg t = cd.t;
            const bool vec = strips_vec(g);
            const int64_t cap = strip_capacity(g, t.bn, vec ? 4 : 0);
            // largest chunk that fits; among those that keep the filter rows
            // 16-byte aligned, the largest of those if one fits
            ConvPlan p, pv;
            for (int rc = step; rc <= rc_max; rc += step) {
                int64_t sc, fp, st;
                const bool fv = filter_vec(g, rc);
                const int64_t lds = f32_layout(g, t.bm, rc, cap, fv, split, &sc, &fp, &st);
                const int64_t raw = g.elem == 4 ? raw_pitch_f32(g, t.bn) : 0;
                if (lds + (raw ? raw_floats((int)g.fh, rc, raw, g.w) : 0) * 4 > budget) continue;
                ConvPlan q;
                q.kind = ConvPlan::kF32Lds;
                q.bm = t.bm; q.bn = t.bn; q.rc = rc; q.tc = (int)g.taps; q.split = split;
                q.strip_cap = cap; q.sc = sc; q.fp = fp; q.stage = st; q.lds_bytes = lds;
                q.svec = vec ? 1 : 0;
                q.fvec = fv ? 1 : 0;
                q.raw_pitch = raw;
                p = q;
                if (fv) pv = q;
            }
            if (pv.kind != ConvPlan::kNone) p = pv;
            if (p.kind == ConvPlan::kNone) continue;
            const int64_t tiles = ((g.npix + t.bn - 1) / t.bn) * ((g.k + t.bm - 1) / t.bm);
            const int64_t per_cu = (tiles + kCUs - 1) / kCUs;
            const double cost = double(per_cu) * (per_cu == 1 ? 2.0 : 1.0) * t.bm * t.bn / cd.eff;
            if (best.kind == ConvPlan::kNone || cost < best_cost) { best = p; best_cost = cost; }
        }
        if (best.kind != ConvPlan::kNone) return best;
    }
    return ConvPlan();
}

ConvArgs conv_args_f32(const Geometry& g, const ConvPlan& p, const void* src, const void* w,
                       float* y, bool fused) {
    ConvArgs a = make_conv_args(g, src, w, y, p.bm);
    a.svec = (!fused && p.svec) ? 1 : 0;
    a.rc = p.rc;
    a.strip_cap = (int)p.strip_cap;
    a.sc = (int)p.sc;
    a.fp = (int)p.fp;
    a.stage = (int)p.stage;
    a.ksplit = p.split;
    a.fvec = p.fvec;
    a.div_fp = make_fastdiv((uint32_t)(p.fvec ? p.fp / 4 : p.fp));
    a.div_ckmid = make_fastdiv((uint32_t)((((g.ho - 1) * g.row_len + g.used_len) + 3) >> 2));
    a.raw_pitch = (int)p.raw_pitch;
    a.raw_off = 2 * (int)p.stage;
    // MODE 3 copies a channel's strip (at most sc / 4 chunks of 16 bytes,
    // since it fits its LDS slot) and a chunk's filter rows with kIlvSlots
    // copies per lane, at 32-bit offsets from the tile's first image
    const int64_t plane = (int64_t)g.ho * g.row_len;
    const int64_t segs = p.bn / ((int64_t)g.ho * g.wo) + 2;
    // (byte offsets below 2^32); the filter-row split keeps the copies
    // before the MFMAs (its MODE 3 build holds too many registers)
    a.ilv = (!fused && p.svec && p.fvec && p.split == 0 && g.c % p.rc == 0 && p.sc / 4 <= 64 * kIlvSlots &&
             (int64_t)p.bm * (p.fp / 4) <= (int64_t)kConvThreads * kIlvSlots &&
             segs * g.c * plane < (1ll << 30) && (int64_t)p.bm * g.c * g.fh * g.fw < (1ll << 30)) ? 1 : 0;
    // fp32 filter rows that are not whole vectors: copied from a repacked filter
    a.fpack = (g.elem == 4 && !p.fvec) ? 1 : 0;
    // fused fp32 with the expansion map (MODE 4): filter-row and raw-row
    // copies from offsets computed once per lane (byte offsets below 2^32:
    // the input planes of the tile's images, the filter rows of the tile)
    if (fused && g.elem == 4 && g.fh <= 3 && p.raw_pitch <= kExpandMaxRaw)
        a.ilv = (p.fvec && g.c % p.rc == 0 && (int64_t)p.bm * (p.fp / 4) <= (int64_t)kConvThreads * kIlvSlots &&
                 segs * g.c * g.h * g.w < (1ll << 30) && g.k * g.c * g.fh * g.fw < (1ll << 30)) ? 1 : 0;
    return a;
}

int64_t filter_scratch_f32(const Geometry& g, const ConvPlan& p) {
    if (g.elem != 4 || p.fvec) return 0;
    const int64_t nchunks = (g.c + p.rc - 1) / p.rc;
    const int64_t jtiles = (g.k + p.bm - 1) / p.bm;
    return jtiles * nchunks * p.bm * p.fp * 4;
}

int launch_conv_f32_plan(const Geometry& g, const ConvPlan& p, bool fused, const void* src,
                         const void* w, void* scratch, float* y, hipStream_t stream, char* err,
                         size_t errlen) {
    ConvArgs a = conv_args_f32(g, p, src, w, y, fused);
    const int64_t blocks = ((g.npix + p.bn - 1) / p.bn) * a.num_jtiles;
    if (blocks > 0x7fffffff) {
        snprintf(err, errlen, "conv: grid of %lld workgroups is too large", (long long)blocks);
        return -5;
    }
    if (a.fpack) {
        // the filter, repacked into the caller's scratch (filter_scratch_f32 bytes)
        const int64_t nchunks = (g.c + p.rc - 1) / p.rc;
        const int64_t total = (int64_t)a.num_jtiles * nchunks * p.bm * p.fp;
        const int64_t pblocks = std::min<int64_t>((total + 255) / 256, 65536);
        hipLaunchKernelGGL(pack_filter_f32_kernel, dim3((unsigned)pblocks), dim3(256), 0, stream,
                           static_cast<const float*>(w), static_cast<float*>(scratch), (int)g.k, (int)g.c,
                           (int)g.taps, p.bm, p.rc, (int)p.fp, (int)nchunks, total);
        a.w = scratch;
    }
    if (g.elem == 2) launch_tile<uint16_t, 0, 0>(p, a, blocks, fused, stream);
    else if (g.fh == 3 && g.fw == 3) launch_tile<float, 3, 3>(p, a, blocks, fused, stream);
    else if (g.fh == 3 && g.fw == 5) launch_tile<float, 3, 5>(p, a, blocks, fused, stream);
    else if (g.fh == 7 && g.fw == 7) launch_tile<float, 7, 7>(p, a, blocks, fused, stream);
    else if (g.fh == 5 && g.fw == 5) launch_tile<float, 5, 5>(p, a, blocks, fused, stream);
    else if (g.fh == 11 && g.fw == 11) launch_tile<float, 11, 11>(p, a, blocks, fused, stream);
    else if (g.fh == 1 && g.fw == 1) launch_tile<float, 1, 1>(p, a, blocks, fused, stream);
    else launch_tile<float, 0, 0>(p, a, blocks, fused, stream);
    return 0;
}

int launch_conv_f32(const Geometry& g, bool fused, const void* src, const void* w, void* scratch,
                    float* y, hipStream_t stream, char* err, size_t errlen) {
    const F32BandPlan bp = plan_band_f32(g);
    if (bp.ok) return launch_conv_f32_band(g, bp, fused, src, w, y, stream);
    const F32BandPlan sp = plan_band_small_c_f32(g);
    if (sp.ok) return launch_conv_f32_band_small_c(g, sp, fused, src, w, y, stream);
    const ConvPlan p = plan_conv_f32(g);
    if (p.kind == ConvPlan::kNone) return launch_conv_plain(g, fused, src, w, y, stream, err, errlen);
    return launch_conv_f32_plan(g, p, fused, src, w, scratch, y, stream, err, errlen);
}

}  // namespace im2win
