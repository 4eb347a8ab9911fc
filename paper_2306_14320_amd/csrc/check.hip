// Host-side bounds check of the launch plans.  It replays, with the very
// functions the kernels call (XformBlock, TileRuns,
// pixel_base), every workgroup of the transformation and of the convolution
// for a descriptor and verifies that each LDS and device-memory index the
// kernels form stays inside its buffer.  No HIP calls.
#include <cstdarg>
#include <cstdio>
#include <vector>

#include "common.h"
#include "conv_common.h"

namespace im2win {
namespace {

struct Report {
    int64_t violations = 0;
    char* msg;
    size_t msglen;
    void fail(const char* fmt, ...) {
        if (violations++ == 0) {
            va_list ap;
            va_start(ap, fmt);
            vsnprintf(msg, msglen, fmt, ap);
            va_end(ap);
        }
    }
};

void check_transform(const Geometry& g, Report& r) {
    const XformPlan p = plan_transform(g);
    if (!p.use_lds) return;   // the direct kernel indexes rows only through bounds-checked x
    const XformArgs a = transform_args(g, p, nullptr, nullptr);
    const int64_t x_elems = g.n * g.c * g.h * g.w;
    const int64_t ws_elems = g.n * g.c * g.ho * g.row_len;
    const int64_t lds_elems = p.lds_bytes / g.elem;
    std::vector<uint8_t> hits;
    int64_t next_out = 0;
    for (int64_t b = 0; b < p.blocks && r.violations < 16; ++b) {
        XformBlock blk;
        blk.init(b, a);
        if (blk.nplanes < 1 || blk.nrows < 1)
            r.fail("transform block %lld: empty run", (long long)b);
        if (blk.shift + blk.olen + a.vec > lds_elems || (blk.obase - blk.shift) % a.vec != 0)
            r.fail("transform block %lld: run of %d (+%d) elements, LDS holds %lld", (long long)b,
                   blk.olen, blk.shift, (long long)lds_elems);
        if (blk.obase != next_out)
            r.fail("transform block %lld: output run starts at %lld, expected %lld", (long long)b,
                   (long long)blk.obase, (long long)next_out);
        next_out = blk.obase + blk.olen;
        if (next_out > ws_elems)
            r.fail("transform block %lld: writes up to %lld of %lld", (long long)b,
                   (long long)next_out, (long long)ws_elems);
        // (an empty footprint, rows of padding only, divides nothing)
        if (a.g > 1 && blk.nrin > 0 && (int64_t)blk.nrin * g.w != (int64_t)a.div_plane.d)
            r.fail("transform block %lld: footprint per plane %lld, divisor %u", (long long)b,
                   (long long)blk.nrin * g.w, a.div_plane.d);
        // replay the scatter: every LDS write inside the run, each element of
        // the run written once if it has a source in x and never if padding
        hits.assign(blk.olen, 0);
        const int per_plane = blk.nrin * a.w;
        const int total = blk.nplanes * per_plane;
        for (int f = 0; f < total && r.violations < 16; ++f) {
            const int pj = a.g > 1 ? (int)fast_div((uint32_t)f, a.div_plane) : 0;
            const int rem = f - pj * per_plane;
            const int rr = (int)fast_div((uint32_t)rem, a.div_w);
            const int yy = blk.y_lo + rr, xx = rem - rr * a.w;
            const int64_t src = (blk.plane0 + pj) * (int64_t)g.h * g.w + (int64_t)yy * g.w + xx;
            if (pj >= blk.nplanes || yy < 0 || yy >= g.h || src < 0 || src >= x_elems) {
                r.fail("transform block %lld: footprint element %d reads x[%lld]", (long long)b, f,
                       (long long)src);
                break;
            }
            int mf, ml;
            blk.rows_of(yy, a, &mf, &ml);
            for (int m = mf; m <= ml; ++m) {
                if (xx + a.pw >= a.wp) break;   // past the row's end (trimmed rows): skipped
                const int u = yy + a.ph - m * a.sh;
                const int li = blk.lds_index(pj, m, xx + a.pw, u, a) - blk.shift;
                if (u < 0 || u >= a.fh || li < 0 || li >= blk.olen) {
                    r.fail("transform block %lld: scatter to %d outside the run", (long long)b, li);
                    break;
                }
                ++hits[li];
            }
        }
        for (int e = 0; e < blk.olen && r.violations < 16; ++e) {
            const int q = e % a.row_len, row = e / a.row_len;
            const int k = q / a.fh, u = q % a.fh;
            const int m = blk.m0 + row % blk.nrows;
            const int yy = m * a.sh + u - a.ph, xx = k - a.pw;
            const bool has_src = yy >= 0 && yy < g.h && xx >= 0 && xx < g.w;
            if (hits[e] != (has_src ? 1 : 0)) {
                r.fail("transform block %lld: element %d written %d times (source %d)", (long long)b,
                       e, hits[e], (int)has_src);
                break;
            }
        }
    }
    if (r.violations == 0 && next_out != ws_elems)
        r.fail("transform: workgroups write %lld of %lld elements", (long long)next_out,
               (long long)ws_elems);
}

void check_conv_variant(const Geometry& g, const ConvPlan& p, bool fused, Report& r) {
    const bool bf16 = p.kind == ConvPlan::kBf16Lds;
    const ConvArgs a = bf16 ? conv_args_bf16(g, p, nullptr, nullptr, nullptr, fused)
                            : conv_args_f32(g, p, nullptr, nullptr, nullptr, fused);
    const char* what = fused ? "fused conv" : "conv";
    const int64_t ws_elems = g.n * g.c * g.ho * g.row_len;
    const int64_t plane = g.ho * g.row_len;
    const int64_t y_elems = g.n * g.k * g.ho * g.wo;
    const int64_t ptiles = (g.npix + p.bn - 1) / p.bn;
    int64_t covered = 0;
    for (int64_t t = 0; t < ptiles && r.violations < 16; ++t) {
        TileRuns tr;
        tr.init((int)t, p.bn, a);
        if (tr.extent > p.strip_cap || tr.strip_len < 1)
            r.fail("%s tile %lld: strip of %d positions, LDS holds %lld", what, (long long)t,
                   tr.extent, (long long)p.strip_cap);
        int prev_end = 0;
        for (int s = 0; s < tr.nseg; ++s) {
            const int len = tr.seg_len(s);
            const int off = tr.seg_off(s);
            if (len < 1 || off < prev_end || off + len > tr.extent)
                r.fail("%s tile %lld: run %d [%d, %d) overlaps or leaves the strip of %d", what,
                       (long long)t, s, off, off + len, tr.extent);
            prev_end = off + len;
            // window-tensor source of the run, for the first and the last channel
            const int64_t first = (((int64_t)(tr.i0 + s) * g.c + 0) * g.ho + tr.seg_m(s)) * g.row_len + tr.seg_q(s);
            const int64_t last = (((int64_t)(tr.i0 + s) * g.c + g.c - 1) * g.ho + tr.seg_m(s)) * g.row_len + tr.seg_q(s) + len;
            if (first < 0 || last > ws_elems)
                r.fail("%s tile %lld: run %d reads window tensor [%lld, %lld) of %lld", what,
                       (long long)t, s, (long long)first, (long long)last, (long long)ws_elems);
            if ((int64_t)tr.seg_m(s) * g.row_len + tr.seg_q(s) + len > plane)
                r.fail("%s tile %lld: run %d runs past its plane", what, (long long)t, s);
            if (a.svec) {
                // 16-byte copies of vc elements: aligned start and rounded end
                // stay in the plane, and the chunks of run s are the LDS
                // chunks [(off - shift)/vc, ...)
                const int vc = a.vchunk;
                const int64_t in_plane = (int64_t)tr.seg_m(s) * g.row_len + tr.seg_q(s);
                const int shift = s == 0 ? tr.shift0 : 0;
                if (vc * g.elem != 16 || (in_plane % vc) != shift || (plane % vc) != 0 ||
                    ((in_plane - shift + vc * (int64_t)((shift + len + vc - 1) / vc)) > plane) ||
                    ((off - shift) % vc) != 0)
                    r.fail("%s tile %lld: 16-byte run %d misplaced (shift %d)", what, (long long)t, s, shift);
            }
        }
        if (!fused && a.ilv && (tr.ck_total > 64 * kIlvSlots || 4 * (int64_t)tr.ck_total > p.sc))
            r.fail("conv tile %lld: %d 16-byte strip copies, in-loop issue covers %d (slot %lld)", (long long)t,
                   tr.ck_total, 64 * kIlvSlots, (long long)p.sc);
        if (fused && !bf16 && g.elem == 4) {
            // raw input rows: inside x and inside their LDS area; their
            // expansion writes each strip position once if it has a source
            // in x, never if it lies in the padding
            const RawRows rw = raw_rows(tr, a);
            if ((int64_t)rw.rtot * g.w > a.raw_pitch || (a.raw_pitch & 3) || (a.raw_off & 3))
                r.fail("fused conv tile %lld: %d raw rows of %lld, LDS pitch %d", (long long)t, rw.rtot,
                       (long long)g.w, a.raw_pitch);
            // copies from per-lane offsets computed once: every copy unit of
            // a channel has a slot, and the byte offsets of the units (from
            // the channel's plane in the tile's first image) stay below 2^32
            if (a.ilv) {
                const int units = a.xvec ? rw.rtot * (int)g.w / 4 : rw.rtot * (int)g.w;
                const int64_t span = (int64_t)tr.nseg * g.c * g.h * g.w;
                if (units > 64 * kF32ExpandGroups || 4 * span >= (int64_t(1) << 32) || g.c % p.rc != 0 ||
                    !p.fvec || p.bm * (p.fp / 4) > (int64_t)kConvThreads * kIlvSlots)
                    r.fail("fused conv tile %lld: %d raw copy units (slots %d), offsets up to %lld bytes",
                           (long long)t, units, 64 * kF32ExpandGroups, (long long)(4 * span));
            }
            std::vector<uint8_t> hit(tr.extent > 0 ? tr.extent : 1, 0);
            for (int rr = 0; rr < rw.rtot && r.violations < 16; ++rr) {
                int yy, sg;
                if (rr < rw.r0) { sg = 0; yy = rw.ylo0 + rr; }
                else {
                    sg = 1 + (rr - rw.r0) / std::max(a.rmid, 1);
                    if (sg > tr.nseg - 1) sg = tr.nseg - 1;
                    yy = a.ylo_mid + (rr - rw.r0 - (sg - 1) * a.rmid);
                }
                if (yy < 0 || yy >= g.h || tr.i0 + sg >= g.n) {
                    r.fail("fused conv tile %lld: raw row %d reads x row %d of image %d", (long long)t, rr, yy, tr.i0 + sg);
                    break;
                }
                const int m_st = tr.seg_m(sg), q_st = tr.seg_q(sg), len = tr.seg_len(sg), off = tr.seg_off(sg);
                const int m_end = sg == tr.nseg - 1 ? tr.m1 : (int)g.ho - 1;
                for (int xx = 0; xx < g.w && xx + g.pw < g.wp; ++xx)   // (trimmed rows end early)
                    for (int m = m_st; m <= m_end; ++m) {
                        const int u = yy + (int)g.ph - m * (int)g.sh;
                        if (u < 0 || u >= g.fh) continue;
                        const int rel = (m - m_st) * (int)g.row_len + (xx + (int)g.pw) * (int)g.fh + u - q_st;
                        if (rel >= 0 && rel < len) ++hit[off + rel];
                    }
            }
            // without the expansion map the kernel places raw elements through
            // per-row entries (raw_row_entry): they must write exactly the
            // positions of the model above, inside the strips, and fit the
            // LDS the plan reserves for them
            const bool map = g.fh <= 3 && a.raw_pitch <= 64 * kF32ExpandGroups;
            if (!map) {
                if (rw.rtot > a.raw_pitch / (int)g.w)
                    r.fail("fused conv tile %lld: %d raw-row entries, LDS holds %lld", (long long)t, rw.rtot,
                           (long long)(a.raw_pitch / g.w));
                std::vector<uint8_t> hit2(hit.size(), 0);
                for (int rr = 0; rr < rw.rtot && r.violations < 16; ++rr) {
                    const RawRowEntry en = raw_row_entry(a, tr, rw, rr);
                    if (en.lo < 0 || en.hi > tr.extent || en.lo > en.hi)
                        r.fail("fused conv tile %lld: raw row %d run [%d, %d) outside the strips", (long long)t, rr,
                               en.lo, en.hi);
                    for (int xx = 0; xx < g.w && xx + g.pw < g.wp; ++xx)
                        for (int i = 0; i < en.cnt; ++i) {
                            const int d = en.base + (xx + (int)g.pw) * (int)g.fh + i * ((int)g.row_len - (int)g.sh);
                            if (d >= en.lo && d < en.hi) ++hit2[d];
                        }
                }
                if (hit2 != hit) r.fail("fused conv tile %lld: raw-row entries place elements elsewhere", (long long)t);
            }
            for (int sg = 0; sg < tr.nseg && r.violations < 16; ++sg) {
                const int m_st = tr.seg_m(sg), q_st = tr.seg_q(sg), len = tr.seg_len(sg), off = tr.seg_off(sg);
                for (int e = 0; e < len; ++e) {
                    const int pos = m_st * (int)g.row_len + q_st + e;
                    const int m = pos / (int)g.row_len, qq = pos % (int)g.row_len;
                    const int yy = m * (int)g.sh + qq % (int)g.fh - (int)g.ph, xx = qq / (int)g.fh - (int)g.pw;
                    const bool src = yy >= 0 && yy < g.h && xx >= 0 && xx < g.w;
                    if (hit[off + e] != (src ? 1 : 0)) {
                        r.fail("fused conv tile %lld: strip position %d written %d times (source %d)",
                               (long long)t, off + e, hit[off + e], (int)src);
                        break;
                    }
                }
            }
        }
        for (int q = 0; q < p.bn; ++q) {
            int px = tr.p0 + q;
            const bool valid = px <= tr.plast;
            if (!valid) px = tr.p0;
            int64_t yoff;
            const int base = pixel_base(tr, a, px, &yoff);
            // the window must lie inside its own run of the strip
            const int gi = px / (int)g.wo, ii = gi / (int)g.ho;
            const int s = ii - tr.i0;
            if (s < 0 || s >= tr.nseg || base < tr.seg_off(s) ||
                base + (int)g.taps > tr.seg_off(s) + tr.seg_len(s)) {
                r.fail("%s tile %lld: pixel %d window [%d, %d) outside run %d", what, (long long)t,
                       px, base, base + (int)g.taps, s);
                break;
            }
            if (valid) {
                ++covered;
                const int mm = gi - ii * (int)g.ho, nn = px - gi * (int)g.wo;
                if (yoff != (int64_t)ii * g.k * g.ho * g.wo + (int64_t)mm * g.wo + nn ||
                    yoff + (g.k - 1) * g.ho * g.wo >= y_elems)
                    r.fail("%s tile %lld: pixel %d output offset %lld", what, (long long)t, px,
                           (long long)yoff);
            }
        }
    }
    if (r.violations == 0 && covered != g.npix)
        r.fail("%s: tiles cover %lld of %lld pixels", what, (long long)covered, (long long)g.npix);
}

// bf16 channel-inner kernel: replay every staging item of every tile with
// the kernel's own decode (segment, in-plane element, LDS position) and check
// that loads stay inside the source planes, stores inside the strip plane,
// and that every tap of every pixel's window reads the LDS position holding
// exactly the window-tensor element that the tap needs.
void check_conv_bf16_variant(const Geometry& g, const ConvPlan& p, bool fused, Report& r) {
    const ConvArgs a = conv_args_bf16(g, p, nullptr, nullptr, nullptr, fused);
    const char* what = fused ? "fused bf16 conv" : "bf16 conv";
    const int64_t plane = g.ho * g.row_len;
    const int64_t y_elems = g.n * g.k * g.ho * g.wo;
    const int64_t ptiles = (g.npix + p.bn - 1) / p.bn;
    const int64_t pb = p.strip_cap;
    int64_t covered = 0;
    std::vector<int64_t> src;   // window-tensor element (segment * plane + e) held by each LDS position
    for (int64_t t = 0; t < ptiles && r.violations < 16; ++t) {
        TileRuns tr;
        tr.init((int)t, p.bn, a);
        const ClLayout cl = cl_layout(tr, a);
        if (cl.extent > pb || cl.sb0 < 0 || cl.sb1 < 0 || cl.sp < 0)
            r.fail("%s tile %lld: LDS extent %d, plane holds %lld", what, (long long)t, cl.extent, (long long)pb);
        src.assign(pb, -1);
        auto put = [&](int s, int64_t e, int pos) {
            if (tr.i0 + s >= g.n || e < 0 || e >= plane || pos < 0 || pos >= pb) {
                r.fail("%s tile %lld: element %lld of segment %d to LDS %d", what, (long long)t, (long long)e, s, pos);
                return;
            }
            src[pos] = (int64_t)s * plane + e;
        };
        // (capacities of the 4-wave kernels; the 8-wave 128 x 256 kernels hold
        // at least as many items per workgroup)
        const int64_t items = a.svec ? 2 * (int64_t)tr.ck_total : 2 * (int64_t)tr.strip_len;
        const int64_t cap_items = (int64_t)kConvThreads *
                                  (a.svec ? (p.strip_items > kConvThreads ? 2 : 1) : kBf16StripScalarItems);
        if (items > cap_items)
            r.fail("%s tile %lld: %lld strip items, registers hold %lld", what, (long long)t,
                   (long long)items, (long long)cap_items);
        const bool raw_items = fused && p.fused_fast;
        if (raw_items) {
            // fused kernel from raw row items: every item's source inside x,
            // its destinations the strip positions of the window-tensor
            // elements it holds (spare slots aside)
            const RawRows rw = raw_rows(tr, a);
            const int nitems = rw.rtot * (int)g.w;
            if (nitems > kConvThreads * p.fused_ipt || p.fused_ipt > kBf16FusedItems || (g.w & 1))
                r.fail("%s tile %lld: %d raw items, registers hold %d", what, (long long)t, nitems,
                       kConvThreads * p.fused_ipt);
            for (int q = 0; q < nitems && r.violations < 16; ++q) {
                const int e0 = 2 * (q >> 1);
                const int rr2 = e0 / (int)g.w, xx = e0 - rr2 * (int)g.w;
                int sg = rr2 < rw.r0 ? 0 : 1 + (rr2 - rw.r0) / std::max(a.rmid, 1);
                if (sg > tr.nseg - 1) sg = tr.nseg - 1;
                const int yy = sg == 0 ? rw.ylo0 + rr2 : a.ylo_mid + (rr2 - rw.r0 - (sg - 1) * a.rmid);
                if (yy < 0 || yy >= g.h || xx + 1 >= g.w + 1 || tr.i0 + sg >= g.n) {
                    r.fail("%s tile %lld: item %d reads x row %d col %d of image %d", what, (long long)t, q, yy,
                           xx, tr.i0 + sg);
                    break;
                }
                const int m_st = tr.seg_m(sg), q_st = tr.seg_q(sg), len = tr.seg_len(sg);
                const int m_end = sg == tr.nseg - 1 ? tr.m1 : (int)g.ho - 1;
                for (int m = m_st; m <= m_end; ++m) {
                    const int u = yy + (int)g.ph - m * (int)g.sh;
                    if (u < 0 || u >= g.fh) continue;
                    for (int h = 0; h < 2; ++h) {
                        if (xx + h + g.pw >= g.wp) continue;   // past a trimmed row's end
                        const int e_in = m * (int)g.row_len + (xx + h + (int)g.pw) * (int)g.fh + u;
                        const int rel = e_in - (m_st * (int)g.row_len + q_st);
                        if (rel >= 0 && rel < len) put(sg, e_in, cl_pos(cl, tr, a, sg, e_in));
                    }
                }
            }
        } else if (a.svec) {
            const int start0 = tr.m0 * a.row_len + tr.qa0 - tr.shift0;
            for (int c = 0; c < tr.ck_total && r.violations < 16; ++c) {
                int s = 0, cs = c;
                if (c >= tr.ck0) {
                    s = 1 + (int)fast_div((uint32_t)(c - tr.ck0), a.div_ckmid);
                    if (s > tr.nseg - 1) s = tr.nseg - 1;
                    cs = c - tr.ck0 - (s - 1) * tr.ck_mid;
                }
                const int e = (s == 0 ? start0 : 0) + 4 * cs;
                const int pos = cl_pos(cl, tr, a, s, e);
                if ((e & 3) || e + 4 > plane) {
                    r.fail("%s tile %lld: 8-byte group at element %d of a plane of %lld", what, (long long)t, e, (long long)plane);
                    break;
                }
                for (int w = 0; w < 4; ++w) {
                    if (cl_pos(cl, tr, a, s, e + w) != pos + w) {
                        r.fail("%s tile %lld: group at element %d crosses a row", what, (long long)t, e);
                        break;
                    }
                    put(s, e + w, pos + w);
                }
            }
        } else {
            for (int q = 0; q < tr.strip_len && r.violations < 16; ++q) {
                int s = 0, base = 0;
                if (q >= tr.len0) {
                    s = 1 + (int)fast_div((uint32_t)(q - tr.len0), a.div_lenmid);
                    if (s > tr.nseg - 1) s = tr.nseg - 1;
                    base = tr.len0 + (s - 1) * tr.len_mid;
                }
                const int e = (s == 0 ? tr.m0 * a.row_len + tr.qa0 : 0) + q - base;
                put(s, e, cl_pos(cl, tr, a, s, e));
            }
        }
        for (int q = 0; q < p.bn && r.violations < 16; ++q) {
            int px = tr.p0 + q;
            const bool valid = px <= tr.plast;
            if (!valid) px = tr.p0;
            int64_t yoff;
            const int base = cl_pixel_base(cl, tr, a, px, &yoff);
            const int gi = px / (int)g.wo, ii = gi / (int)g.ho;
            const int mm = gi - ii * (int)g.ho, nn = px - gi * (int)g.wo;
            const int s = ii - tr.i0;
            for (int tp = 0; tp < g.taps; ++tp) {
                const int64_t e = (int64_t)mm * g.row_len + (int64_t)nn * g.sw * g.fh + tp;
                int64_t want = (int64_t)s * plane + e;
                if (raw_items) {
                    // padding elements are never written (zero since the start)
                    const int64_t qq = e % g.row_len;
                    const int64_t yy = mm * g.sh + qq % g.fh - g.ph, xx = qq / g.fh - g.pw;
                    if (yy < 0 || yy >= g.h || xx < 0 || xx >= g.w) want = -1;
                }
                if (base + tp < 0 || base + tp >= pb - kBf16Spare || src[base + tp] != want) {
                    r.fail("%s tile %lld: pixel %d tap %d reads LDS %d", what, (long long)t, px, tp, base + tp);
                    break;
                }
            }
            if (valid) {
                ++covered;
                if (yoff != (int64_t)ii * g.k * g.ho * g.wo + (int64_t)mm * g.wo + nn ||
                    yoff + (g.k - 1) * g.ho * g.wo >= y_elems)
                    r.fail("%s tile %lld: pixel %d output offset %lld", what, (long long)t, px, (long long)yoff);
            }
        }
    }
    if (r.violations == 0 && covered != g.npix)
        r.fail("%s: tiles cover %lld of %lld pixels", what, (long long)covered, (long long)g.npix);
}

// Packed bf16 filter: every piece reads 8 channels inside w, the blocks tile
// the packed buffer, and within a block the DMA destination of piece P (the
// kernels' dma_filter: plane P / (T*BM), position P mod T*BM) is the LDS
// position packed_piece() assigns, where the matrix-core reads expect
// channels c0 .. c0+7 of tap t of output channel j: each filter position of
// both planes filled exactly once.
void check_packed_filter(const Geometry& g, const ConvPlan& p, Report& r) {
    const int T = (int)g.taps, bm = p.bm, plane = T * bm, pieces = 2 * plane;
    const int nchunks = (int)(g.c / kBf16Chunk);
    if (g.c % kBf16Chunk || g.k % bm || plane % 64) {
        r.fail("conv: packed bf16 filter with C %% 16 = %lld, K %% BM = %lld, T*BM = %d", (long long)(g.c % 16),
               (long long)(g.k % bm), plane);
        return;
    }
    const int64_t npieces = g.k * g.c * T / 8;
    if (npieces * 16 > conv_scratch_bytes(g, false) && npieces * 16 > conv_scratch_bytes(g, true)) {
        r.fail("conv: filter scratch of %lld bytes, the packed filter needs %lld",
               (long long)std::max(conv_scratch_bytes(g, false), conv_scratch_bytes(g, true)),
               (long long)(npieces * 16));
        return;
    }
    if (npieces != (g.k / bm) * (int64_t)nchunks * pieces) {
        r.fail("conv: %lld packed pieces, blocks hold %lld", (long long)npieces,
               (long long)((g.k / bm) * nchunks * pieces));
        return;
    }
    std::vector<int> seen(2 * (size_t)p.cl_fpb, 0);
    for (int64_t gid = 0; gid < npieces && r.violations < 16; ++gid) {
        const PackedPiece pc = packed_piece(gid, T, (int)g.fh, (int)g.fw, bm, nchunks, (int)p.cl_fpb);
        const int64_t blk = gid / pieces;
        const int P = (int)(gid - blk * pieces);
        const int jt = (int)(blk / nchunks), ch = (int)(blk % nchunks);
        const int gg = P / plane, q = P % plane, t = q / bm, jj = q % bm;
        const int v = t / (int)g.fh, u = t % (int)g.fh;
        const int dma_pos = gg * (int)p.cl_fpb + P - gg * plane;
        if (pc.j != jt * bm + jj || pc.j >= g.k || pc.c0 != 16 * ch + 8 * gg || pc.c0 + 8 > g.c ||
            packed_index(pc.j, ch, gg, t, T, bm, nchunks) != gid || g.k % kPackRows ||
            pc.nat != u * g.fw + v || pc.nat >= T || pc.lds_pos != dma_pos || dma_pos < 0 ||
            dma_pos >= 2 * p.cl_fpb || (gg == 0 && dma_pos >= p.cl_fpb))
            r.fail("conv: packed filter piece %lld -> j %d c0 %d tap %d LDS %d (DMA %d)", (long long)gid, pc.j,
                   pc.c0, pc.nat, pc.lds_pos, dma_pos);
        else if (blk == 0)
            ++seen[dma_pos];
    }
    for (int gg = 0; gg < 2 && r.violations < 16; ++gg)
        for (int q = 0; q < plane; ++q)
            if (seen[gg * p.cl_fpb + q] != 1) {
                r.fail("conv: packed filter LDS position %d of plane %d written %d times", q, gg,
                       seen[gg * p.cl_fpb + q]);
                break;
            }
}

// One-image-per-workgroup bf16 kernel: replays the kernel's own index
// arithmetic for every lane of every wave (window reads of each tap, staging
// loads and LDS writes, filter-fragment loads, output stores) and checks
// that every index stays inside its buffer, that the LDS positions the
// windows read hold exactly the window-tensor elements Alg. 2 sums (written
// once per chunk, or padding that is never written), and that every output
// is stored exactly once.
void check_conv_image(const Geometry& g, bool fused, const ImgPlan& p, Report& r) {
    const ImgArgs a = image_args(g, p, nullptr, nullptr, nullptr);
    const int T = (int)g.taps, FH = (int)g.fh;
    if (p.lds_bytes != 2 * p.stage_pos * 16 || p.lds_bytes > kConvLdsMaxBytes || p.stage_pos != 4 * p.plane_pos ||
        p.pitch < g.row_len || (p.pitch - g.sw * g.fh * g.wo) % 16 != 0)
        r.fail("image conv: LDS layout (pitch %lld, plane %lld, %lld bytes)", (long long)p.pitch,
               (long long)p.plane_pos, (long long)p.lds_bytes);
    // workgroup -> (image, K tile) is a bijection
    std::vector<uint8_t> seen_wg(a.grid, 0);
    for (int b = 0; b < a.grid; ++b) {
        const int bid = a.xcd_remap ? (b & 7) * (a.grid >> 3) + (b >> 3) : b;
        if (bid < 0 || bid >= a.grid || seen_wg[bid]++) {
            r.fail("image conv: workgroup %d maps to %d (repeated or out of range)", b, bid);
            return;
        }
    }
    // What each LDS position of one stage holds after the staging of a
    // chunk: -1 never written, else (channel group, window-tensor element
    // m*row_len + k*Fh + u) encoded as g*2^28 + element.
    const int64_t plane_elems = (int64_t)g.ho * g.row_len;
    std::vector<int64_t> holds(p.stage_pos, -1);
    const int SI = fused ? kImgFusedItems : kImgStripItems;
    const int64_t src_chan = (int64_t)g.c * p.plane_src;   // elements per image
    for (int tid = 0; tid < kImgThreads; ++tid)
        for (int k = 0; k < SI; ++k) {
            const int item = tid + k * kImgThreads;
            if (item >= 4 * a.ngroups) continue;
            const int gg = item / a.ngroups, e = item - gg * a.ngroups;
            if (!fused) {
                const int64_t off = (int64_t)gg * 8 * a.plane_src + 4 * e;
                // loads: 4 elements of channels 8gg .. 8gg+7 of the last chunk's planes
                const int64_t last = (int64_t)(a.nchunks - 1) * kImgChunk * a.plane_src + off + 7 * (int64_t)a.plane_src + 3;
                if (last >= src_chan || off % 4) r.fail("image conv: strip load of item %d reads %lld of %lld", item,
                                                        (long long)last, (long long)src_chan);
                const int m = (4 * e) / a.row_len, q = 4 * e - m * a.row_len;
                for (int pq = 0; pq < 4; ++pq) {
                    const int64_t pos = (int64_t)gg * a.plane_pos + (int64_t)m * a.pitch + q + pq;
                    if (q + pq >= a.row_len || pos < 0 || pos >= (gg + 1) * (int64_t)a.plane_pos || holds[pos] != -1) {
                        r.fail("image conv: item %d writes LDS position %lld twice or out of its plane", item, (long long)pos);
                        return;
                    }
                    holds[pos] = ((int64_t)gg << 28) + (int64_t)m * g.row_len + q + pq;
                }
            } else {
                const int64_t off = (int64_t)gg * 8 * a.plane_src + 2 * e;
                const int64_t last = (int64_t)(a.nchunks - 1) * kImgChunk * a.plane_src + off + 7 * (int64_t)a.plane_src + 1;
                if (last >= src_chan || off % 2) r.fail("image conv: x load of item %d reads %lld of %lld", item,
                                                        (long long)last, (long long)src_chan);
                const int yy = (2 * e) / a.w, xx = 2 * e - yy * a.w;
                for (int u = 0; u < FH; ++u) {
                    const int t = yy + a.ph - u;
                    const int m = t >= 0 ? t / a.sh : -1;
                    if (!(t >= 0 && m * a.sh == t && m < a.ho && xx + a.pw < a.wr)) continue;
                    for (int d = 0; d < 2; ++d) {
                        if (d == 1 && !(xx + 1 + a.pw < a.wr)) continue;
                        const int kk = xx + d + a.pw;
                        const int64_t pos = (int64_t)gg * a.plane_pos + (int64_t)m * a.pitch + (int64_t)kk * FH + u;
                        if (pos < 0 || pos >= (gg + 1) * (int64_t)a.plane_pos || holds[pos] != -1) {
                            r.fail("image conv: x item %d writes LDS position %lld twice or out of its plane", item,
                                   (long long)pos);
                            return;
                        }
                        holds[pos] = ((int64_t)gg << 28) + (int64_t)m * g.row_len + (int64_t)kk * FH + u;
                    }
                }
            }
        }
    // window reads: every tap of every lane's window is the element Alg. 2
    // sums (or, fused, padding that reads zero)
    const int64_t frags = g.k * g.c * T * 2 / 16;   // scratch in 16-byte units
    for (int wv = 0; wv < kImgThreads / 64 && r.violations < 16; ++wv) {
        const int kp = wv & 3, half = wv >> 2;
        for (int lane = 0; lane < 64; ++lane) {
            const int gl = lane >> 4;
            for (int q = 0; q < kImgNPB; ++q) {
                int pix = (half * kImgNPB + q) * 16 + (lane & 15);
                if (pix > a.npix - 1) pix = a.npix - 1;
                const int m = pix / a.wo, n = pix - m * a.wo;
                const int64_t base = (int64_t)gl * a.plane_pos + (int64_t)m * a.pitch + (int64_t)n * a.sw * FH;
                for (int t = 0; t < T; ++t) {
                    const int64_t pos = base + t;
                    const int v = t / FH, u = t - v * FH;
                    const int64_t want = ((int64_t)gl << 28) + (int64_t)m * g.row_len + ((int64_t)n * a.sw + v) * FH + u;
                    const bool pad_ok = fused && holds[pos] == -1 &&
                                        ((int64_t)m * a.sh + u - a.ph < 0 || (int64_t)m * a.sh + u - a.ph >= a.h ||
                                         (int64_t)n * a.sw + v - a.pw < 0 || (int64_t)n * a.sw + v - a.pw >= a.w);
                    if (pos < 0 || pos >= p.stage_pos || (holds[pos] != want && !pad_ok)) {
                        r.fail("image conv: wave %d lane %d block %d tap %d reads LDS %lld holding %lld, wants %lld", wv,
                               lane, q, t, (long long)pos, (long long)(pos >= 0 && pos < p.stage_pos ? holds[pos] : -2),
                               (long long)want);
                        break;
                    }
                }
            }
            // filter fragments (16-byte units) of the last chunk of the last K tile
            const int64_t idx = ((((int64_t)(a.nkt - 1) * 4 + kp) * a.nchunks + a.nchunks - 1) * T + T - 1) * 2 * 64 +
                                64 + lane;
            if (idx >= frags) r.fail("image conv: filter fragment %lld of %lld", (long long)idx, (long long)frags);
        }
    }
    // outputs: each (image, channel, pixel) stored once
    std::vector<uint8_t> out((size_t)g.k * a.npix, 0);
    for (int kt = 0; kt < a.nkt; ++kt)
        for (int wv = 0; wv < kImgThreads / 64; ++wv)
            for (int lane = 0; lane < 64; ++lane)
                for (int q = 0; q < kImgNPB; ++q) {
                    const int pix = ((wv >> 2) * kImgNPB + q) * 16 + (lane & 15);
                    if (pix >= a.npix) continue;
                    for (int i = 0; i < 2; ++i)
                        for (int v = 0; v < 4; ++v) {
                            const int j = kt * 128 + (wv & 3) * 32 + i * 16 + 4 * (lane >> 4) + v;
                            if (j >= g.k) { r.fail("image conv: output channel %d", j); return; }
                            ++out[(size_t)j * a.npix + pix];
                        }
                }
    for (size_t i = 0; i < out.size(); ++i)
        if (out[i] != 1) {
            r.fail("image conv: output %zu of an image stored %d times", i, (int)out[i]);
            return;
        }
    if (conv_scratch_bytes(g, fused) < g.k * g.c * T * 2)
        r.fail("image conv: filter scratch of %lld bytes", (long long)conv_scratch_bytes(g, fused));
    (void)plane_elems;
}

// fp32 band kernel: replays the workgroup map (each (image, band, channel
// group) once), and for every band: every staging copy of every wave (source
// inside the image slab or the zero-reading offset, LDS destination inside the
// copy's channel slot, each strip position written once with the
// window-tensor element it must hold), every window read of every wave, lane,
// pair, tap and pixel block, the filter rows, the partial-sum area and the
// output stores (each output of the layer exactly once).
// (With the two-way split the kernel runs two waves per SIMD: each of its
// 8 waves copies every part of one channel slot, where the 4 waves replayed
// here copy every part of two slots each, so both issue the same copies;
// waves w and w + 4 read the windows of wave w below for the first
// ceil(NB/2) pixel blocks and the rest: the same reads and outputs.)
void check_conv_band_f32(const Geometry& g, bool fused, const F32BandPlan& p, Report& r) {
    const F32BandArgs a = band_args_f32(g, p, fused, nullptr, nullptr, nullptr);
    const int T = (int)g.taps, FH = (int)g.fh, FW = (int)g.fw;
    const int KS = p.ks, PP = 4 / KS, CB = 4 / KS, nb = p.nb;
    const int64_t stage_f = kBandStageBytes / 4;
    // several whole images per band: a run of ipb*Ho rows
    const bool multi = a.ipb > 1;
    const int64_t brows = multi ? (int64_t)a.ipb * g.ho : a.rows;
    const int64_t groups = multi ? (g.n + a.ipb - 1) / a.ipb : g.n * a.nbands;
    if (2 * (int64_t)kBandStageBytes > p.lds_bytes ||
        (int64_t)(KS == 4 ? 4 : 2) * 32 * nb * 32 * 4 > p.lds_bytes || p.lds_bytes > kConvLdsMaxBytes ||
        (KS != 4 && KS != 2) || a.rows < 1 || nb * 32 < brows * a.wo || (nb - 1) * 32 >= brows * a.wo ||
        brows * g.row_len + 3 > 64 * kBandMaxSeg || g.c % (2 * kBandChunk) || g.k % (32 * CB) ||
        (int64_t)a.nbands * a.rows < g.ho || (int64_t)(a.nbands - 1) * a.rows >= g.ho ||
        (multi && (a.rows != g.ho || a.nbands != 1 || a.ipb > g.n || a.mode == kBandRaw)) || !band_nb_compiled(KS, nb) ||
        groups * a.nkt != a.grid) {
        r.fail("fp32 band conv: plan (ks %d, %d rows, %d images, nb %d, %lld bytes of LDS)", KS, a.rows, a.ipb, nb,
               (long long)p.lds_bytes);
        return;
    }
    F32BandArgs raw_probe = a;
    const bool raw = fused && !multi && band_raw_mode(g, a.rows, nullptr, &raw_probe);
    if (a.mode != (fused ? (raw ? kBandRaw : kBandGather) : (g.ho * g.row_len) % 4 == 0 ? kBandWide : kBandNarrow))
        r.fail("fp32 band conv: copy mode %d", a.mode);
    if (raw && (a.rlpad < g.pw || a.rlpad % 4 || a.rpitch != 4 * a.rlanes || a.rlanes > 64 || a.rrpi != 64 / a.rlanes ||
                a.rpitch < a.rlpad + std::max(g.w, (g.wo - 1) * g.sw + g.fw - g.pw) ||
                a.rrows != (a.rows - 1) * g.sh + g.fh || a.rgroups * a.rrpi < a.rrows ||
                a.rgroups > kBandRawGroups || (int64_t)a.rgroups * a.rrpi * a.rpitch > kBandSlot || g.w % 4)) {
        r.fail("fp32 band conv: raw rows (pitch %d, pad %d, %d rows per copy, %d copies)", a.rpitch, a.rlpad, a.rrpi,
               a.rgroups);
        return;
    }
    std::vector<uint8_t> seen_wg(a.grid, 0);
    for (int b = 0; b < a.grid; ++b) {
        const int bid = a.xcd_remap ? (b & 7) * (a.grid >> 3) + (b >> 3) : b;
        if (bid < 0 || bid >= a.grid || seen_wg[bid]++) {
            r.fail("fp32 band conv: workgroup %d maps to %d (repeated or out of range)", b, bid);
            return;
        }
    }
    const int nj = band_copies(a.mode);
    const int per = a.mode == kBandWide || a.mode == kBandRaw ? 4 : 1;   // floats per lane and copy
    const uint64_t slab = (uint64_t)g.c * a.plane_src * 4;
    const uint64_t plane_bytes = (uint64_t)a.plane_src * 4;
    if ((uint64_t)a.ipb * slab >= kBandOutside)
        r.fail("fp32 band conv: source of %d image slabs of %llu bytes", a.ipb, (unsigned long long)slab);
    const int64_t kZero = -2;
    const int64_t hw = g.ho * g.wo;
    std::vector<int64_t> holds(stage_f);
    // outputs: of image 0 (bands of one image: every band of it), or of the
    // band's images (several images: each band checked on its own)
    std::vector<uint8_t> out((size_t)g.k * hw * (multi ? a.ipb : 1), 0);
    // bands checked: every band of image 0, or (several images) the first
    // band and the last, which may hold fewer images
    std::vector<int> checked;
    if (multi) {
        checked.push_back(0);
        if (groups > 1) checked.push_back((int)groups - 1);
    } else {
        for (int band = 0; band < a.nbands; ++band) checked.push_back(band);
    }
    for (int band : checked) {
        if (r.violations) break;
        // (channel group 0 of the band: the staging and the reads do not
        // depend on it)
        const BandTile t = band_tile(a, band * a.nkt);
        const int want_img = multi ? band * a.ipb : 0;
        const int want_nimg = multi ? (int)std::min<int64_t>(a.ipb, g.n - want_img) : 1;
        if (t.band != (multi ? 0 : band) || t.img != want_img || t.nimg != want_nimg || t.kt != 0 ||
            t.m0 != (multi ? 0 : band * a.rows) || t.nrows < 1 || (multi && t.nrows != want_nimg * g.ho) ||
            t.npix > nb * 32 || (a.mode == kBandWide && t.shift + (int64_t)t.nrows * g.row_len > 64 * kBandMaxSeg)) {
            r.fail("fp32 band conv: band %d (rows %d + %d, image %d + %d, shift %d)", band, t.m0, t.nrows, t.img,
                   t.nimg, t.shift);
            return;
        }
        if (multi) std::fill(out.begin(), out.end(), 0);
        const uint64_t src_bytes = (uint64_t)t.nimg * slab;   // the copies' buffer: the band's image slabs
        // staging: holds[float of a stage] = slot << 24 | window-tensor
        // element of the plane, or kZero (a copy wrote zero), or -1
        std::fill(holds.begin(), holds.end(), -1);
        for (int wv = 0; wv < kBandThreads / 64; ++wv)
            for (int j = 0; j < nj; ++j)
                for (int lane = 0; lane < 64; ++lane) {
                    // raw mode: copies past rgroups and lanes past rrpi whole rows are skipped
                    if (a.mode == kBandRaw && ((j >> 1) >= a.rgroups || lane >= a.rrpi * a.rlanes)) continue;
                    const int cc = 2 * wv + (j & 1);
                    const uint32_t off = band_source(a, t, a.mode, FH, j >> 1, lane);
                    const int64_t dst = band_dest(a, a.mode, wv, j) + (int64_t)lane * per * 4;
                    if (dst < (int64_t)cc * kBandSlot * 4 || dst + per * 4 > (int64_t)(cc + 1) * kBandSlot * 4) {
                        r.fail("fp32 band conv: copy %d of wave %d lane %d writes LDS byte %lld outside slot %d", j,
                               wv, lane, (long long)dst, cc);
                        return;
                    }
                    // the last real chunk reads inside the slab; the one past
                    // it (issued, never used) reads only zeros (several
                    // images: or the next image's first planes, inside the
                    // source); no offset wraps.  (Several images: off lies
                    // in the channel-0 plane of one of the band's images.)
                    const uint64_t last = ((uint64_t)(a.nchunks - 1) * kBandChunk + cc) * plane_bytes + off;
                    const uint64_t past = ((uint64_t)a.nchunks * kBandChunk + cc) * plane_bytes + off;
                    if (past >= (uint64_t(1) << 32) || (!multi && past < src_bytes) ||
                        (off != kBandOutside &&
                         ((off % slab) + per * 4 > plane_bytes || off / slab >= (uint64_t)t.nimg ||
                          last + per * 4 > src_bytes))) {
                        r.fail("fp32 band conv: copy %d of wave %d lane %d reads byte %llu of %llu source bytes", j,
                               wv, lane, (unsigned long long)last, (unsigned long long)src_bytes);
                        return;
                    }
                    if (a.mode == kBandRaw) {
                        // raw row r, column xx .. xx+3 of the band (x row
                        // m0*sh - ph + r), or zeros outside the image and the row
                        const int r2 = (j >> 1) * a.rrpi + lane / a.rlanes, li = lane % a.rlanes;
                        const int64_t yy = (int64_t)t.m0 * g.sh - g.ph + r2, xx = 4 * li - a.rlpad;
                        const bool in = r2 < a.rrows && yy >= 0 && yy < g.h && xx >= 0 && xx + 4 <= g.w;
                        if ((off != kBandOutside) != in || (in && off != (uint32_t)(yy * g.w + xx) * 4u) ||
                            dst / 4 != (int64_t)cc * kBandSlot + (int64_t)r2 * a.rpitch + 4 * li) {
                            r.fail("fp32 band conv: raw copy %d of wave %d lane %d: source %u, LDS float %lld", j, wv,
                                   lane, off, (long long)(dst / 4));
                            return;
                        }
                        for (int e = 0; e < 4; ++e) {
                            const int64_t f = dst / 4 + e;
                            if (holds[f] != -1) {
                                r.fail("fp32 band conv: LDS float %lld written twice", (long long)f);
                                return;
                            }
                            holds[f] = in ? ((int64_t)cc << 24) + yy * g.w + xx + e : kZero;
                        }
                        continue;
                    }
                    for (int e = 0; e < per; ++e) {
                        const int64_t f = dst / 4 + e;
                        // strip position of this float: band-run element pos
                        const int64_t pos = per == 1 ? (int64_t)(j >> 1) * 64 + lane
                                                     : (int64_t)(j >> 1) * 256 + lane * 4 + e - t.shift;
                        int64_t v = kZero;
                        if (off != kBandOutside) {
                            // element of the band's run of rows (several
                            // images: row m of the run is row m % Ho of image
                            // m / Ho of the band, C planes further per image)
                            const int64_t elem = (int64_t)t.m0 * g.row_len + pos;
                            const int64_t q = multi ? elem / g.row_len / g.ho : 0;
                            if (!fused && (int64_t)off / 4 + e != elem + q * (g.c - 1) * a.plane_src) {
                                r.fail("fp32 band conv: strip position %lld copied from element %u", (long long)pos,
                                       off / 4 + e);
                                return;
                            }
                            if (fused) {   // the x element of window-tensor element elem (transform's definition)
                                const int64_t m = elem / g.row_len - q * g.ho, k = (elem % g.row_len) / FH,
                                              u = elem % FH;
                                const int64_t yy = m * g.sh + u - g.ph, xx = k - g.pw;
                                if (pos < 0 || pos >= (int64_t)t.nrows * g.row_len || yy < 0 || yy >= g.h ||
                                    xx < 0 || xx >= g.w || (int64_t)off / 4 != q * g.c * a.plane_src + yy * g.w + xx) {
                                    r.fail("fp32 band conv: strip position %lld gathered from x element %u",
                                           (long long)pos, off / 4);
                                    return;
                                }
                            }
                            v = ((int64_t)cc << 24) + elem;
                        }
                        if (holds[f] != -1) {
                            r.fail("fp32 band conv: LDS float %lld written twice", (long long)f);
                            return;
                        }
                        holds[f] = v;
                    }
                }
        // window reads: every tap of every lane's window is the element
        // Alg. 2 sums (the padding of the fused variant reads a zero copy)
        for (int wv = 0; wv < kBandThreads / 64 && r.violations == 0; ++wv) {
            const int ks = wv % KS;
            for (int lane = 0; lane < 64; ++lane)
                for (int b = 0; b < nb; ++b) {
                    int pix = b * 32 + (lane & 31);
                    if (pix > t.npix - 1) pix = t.npix - 1;
                    const int64_t m = t.m0 + pix / g.wo, n = pix % g.wo;   // row of the band's run
                    const int64_t mi = multi ? m % g.ho : m;                   // row of its image
                    for (int pp = 0; pp < PP; ++pp) {
                        const int cc = 2 * (ks * PP + pp) + (lane >> 5);
                        for (int tap = 0; tap < T; ++tap) {
                            const int u = tap / FW, v = tap % FW;
                            const int64_t f = band_window(a, t, FH, 2 * ks * PP + (lane >> 5), lane, b) / 4 +
                                              (int64_t)pp * 2 * kBandSlot +
                                              (a.mode == kBandRaw ? (int64_t)u * a.rpitch + v : (int64_t)v * FH + u);
                            const int64_t yy = mi * g.sh + u - g.ph, xx = n * g.sw + v - g.pw;
                            const bool pad = yy < 0 || yy >= g.h || xx < 0 || xx >= g.w;
                            // window-tensor element (raw mode: the x element)
                            const int64_t elem =
                                a.mode == kBandRaw ? yy * g.w + xx : m * g.row_len + (n * g.sw + v) * FH + u;
                            const bool ok = f >= 0 && f < stage_f &&
                                            (a.mode == kBandRaw ? holds[f] == (pad ? kZero : ((int64_t)cc << 24) + elem)
                                                                : (holds[f] == ((int64_t)cc << 24) + elem ||
                                                                   (fused && pad && holds[f] == kZero)));
                            if (!ok) {
                                r.fail("fp32 band conv: band %d wave %d lane %d block %d pair %d tap %d reads LDS float "
                                       "%lld holding %lld, wants element %lld of slot %d", band, wv, lane, b, pp, tap,
                                       (long long)f, (long long)(f >= 0 && f < stage_f ? holds[f] : -3),
                                       (long long)elem, cc);
                                return;
                            }
                        }
                    }
                }
        }
        // outputs of this band (image 0): every channel group, block, pixel
        // (the four-way split stores pixels tid, tid + 256, ... below npix;
        // the two-way split the pixels of its blocks below npix)
        for (int kt = 0; kt < a.nkt; ++kt)
            for (int cb = 0; cb < CB; ++cb)
                for (int p2 = 0; p2 < (KS == 4 ? t.npix : nb * 32); ++p2) {
                    if (p2 >= t.npix) continue;
                    for (int ch = 0; ch < 32; ++ch) {
                        const int64_t j = (int64_t)(kt * CB + cb) * 32 + ch;
                        if (j >= g.k) { r.fail("fp32 band conv: output channel %lld", (long long)j); return; }
                        // the kernel's store offset from the band's first
                        // pixel of channel j
                        const int64_t at = (int64_t)t.m0 * g.wo + p2 + band_image_skip(a, p2);
                        const int64_t q = multi ? p2 / hw : 0;
                        if (at != q * g.k * hw + p2 - q * hw + (int64_t)t.m0 * g.wo) {
                            r.fail("fp32 band conv: pixel %d of band %d stored at %lld", p2, band, (long long)at);
                            return;
                        }
                        ++out[(size_t)(j * hw + at)];
                    }
                }
        if (multi)
            for (size_t i = 0; i < (size_t)t.nimg * g.k * hw; ++i)
                if (out[i] != 1) {
                    r.fail("fp32 band conv: output %zu of band %d stored %d times", i, band, (int)out[i]);
                    return;
                }
    }
    if (r.violations) return;
    if (!multi)
        for (size_t i = 0; i < out.size(); ++i)
            if (out[i] != 1) {
                r.fail("fp32 band conv: output %zu of an image stored %d times", i, (int)out[i]);
                return;
            }
    // filter rows: the last chunk's pair of the last channel group
    const int64_t wmax = (((int64_t)(a.nkt - 1) * CB * 32 + CB * 32 - 1) * g.c + (a.nchunks - 1) * kBandChunk + 7) * T + T - 1;
    if (wmax >= g.k * g.c * T)
        r.fail("fp32 band conv: filter element %lld of %lld", (long long)wmax, (long long)(g.k * g.c * T));
    // stage 1, the farthest pair and tap stay inside one LDS read's reach
    const int64_t tap_reach = a.mode == kBandRaw ? (int64_t)(FH - 1) * a.rpitch + FW : T;
    if (kBandStageBytes + (PP - 1) * 2 * kBandSlot * 4 + tap_reach * 4 >= 65536)
        r.fail("fp32 band conv: LDS read offsets exceed 16 bits");
    if (conv_scratch_bytes(g, fused) != 0)
        r.fail("fp32 band conv: scratch of %lld bytes requested", (long long)conv_scratch_bytes(g, fused));
}

// fp32 small-C band kernel: the workgroup map, and for every band every
// staging copy (source inside the image slab or the zero-reading offset, LDS
// destination inside its channel slot or raw row, each LDS float written
// once; fused, the expansion of the raw rows into the strips), every window
// read of every wave, lane, k-step and pixel block (the element Alg. 2
// multiplies with the weight that step carries; the zero-weight duplicate
// row reads an element of the same window), the filter reads and each
// output stored once.
void check_conv_band_small_c_f32(const Geometry& g, bool fused, const F32BandPlan& p, Report& r) {
    const F32BandArgs a = band_args_small_c_f32(g, p, fused, nullptr, nullptr, nullptr);
    const int C = (int)g.c, FH = (int)g.fh, FW = (int)g.fw, T = FH * FW;
    const int HU = (FH + 1) / 2, S = smallc_steps(C, FH, FW), SW = (S + 1) / 2, nb = p.nb;
    const int64_t slot_bytes = (int64_t)a.slotf * 4;
    const int64_t rb_f = (int64_t)C * a.rrows * a.rpitch;   // floats of one raw-row buffer (fused)
    if (C != kSmallCChannels || p.ks != 2 || p.lds_bytes > kConvLdsMaxBytes ||
        p.lds_bytes != std::max(2 * C * slot_bytes, 2 * rb_f * 4) + (int64_t)2 * 32 * nb * 32 * 4 ||
        a.rrows != (a.rows - 1) * g.sh + g.fh || a.rlpad < g.pw || a.rlpad % 4 || a.rpitch < a.rlpad + g.w ||
        a.rpitch % 4 || (a.rawwide && g.w % 4) || a.rparts * 64 * (a.rawwide ? 4 : 1) < g.w || nb * 32 < a.rows * a.wo ||
        (nb - 1) * 32 >= a.rows * a.wo || g.k % 32 || a.nkt != (g.k + 63) / 64 || (int64_t)g.n * a.nbands * a.nkt != a.total ||
        (int64_t)a.nbands * a.rows < g.ho || (int64_t)(a.nbands - 1) * a.rows >= g.ho || a.per_wg < 1 ||
        (int64_t)a.grid * a.per_wg < a.total || (int64_t)(a.grid - 1) * a.per_wg >= a.total) {
        r.fail("fp32 small-C band conv: plan (%d rows, nb %d, slot %d floats, %lld bytes of LDS, %d x %d bands)", a.rows,
               nb, a.slotf, (long long)p.lds_bytes, a.grid, a.per_wg);
        return;
    }
    if (fused ? a.mode != kBandGather : (a.mode != kBandWide && a.mode != kBandNarrow)) {
        r.fail("fp32 small-C band conv: copy mode %d", a.mode);
        return;
    }
    // workgroup w walks bands [w*per_wg, min((w+1)*per_wg, total)): every
    // band once, alternating between the two strip buffers
    std::vector<uint8_t> seen_band(a.total, 0);
    for (int wg = 0; wg < a.grid; ++wg)
        for (int b = wg * a.per_wg; b < std::min((wg + 1) * a.per_wg, a.total); ++b)
            if (seen_band[b]++) {
                r.fail("fp32 small-C band conv: band %d walked twice", b);
                return;
            }
    for (int b = 0; b < a.total; ++b)
        if (!seen_band[b]) {
            r.fail("fp32 small-C band conv: band %d never walked", b);
            return;
        }
    const int per = a.mode == kBandWide ? 4 : 1;
    const int part = a.mode == kBandWide ? 256 : 64;
    const uint64_t slab = (uint64_t)C * a.plane_src * 4;
    const int64_t kZero = -2;
    std::vector<int64_t> holds((size_t)C * a.slotf);
    std::vector<int64_t> raw((size_t)rb_f);
    std::vector<uint8_t> out((size_t)g.k * g.ho * g.wo, 0);
    // Unfused: the strip copies of band t, each strip position written once
    // with (channel << 24) + its window-tensor element, or zero past the strip.
    auto stage_strips = [&](const BandTile& t) {
        const int np = smallc_parts(a, t);
        if ((int64_t)np * part > a.slotf) {
            r.fail("fp32 small-C band conv: %d parts of %d floats in a slot of %d", np, part, a.slotf);
            return false;
        }
        for (int j = 0; j < C * np; ++j)
            for (int lane = 0; lane < 64; ++lane) {
                const int c = j / np, sp = j % np;
                const uint32_t off = band_source(a, t, a.mode, FH, sp, lane);
                const int64_t dst = (int64_t)c * a.slotf + (int64_t)sp * part + (int64_t)lane * per;   // float index
                if (dst < (int64_t)c * a.slotf || dst + per > (int64_t)(c + 1) * a.slotf) {
                    r.fail("fp32 small-C band conv: copy %d lane %d writes LDS float %lld outside slot %d", j, lane,
                           (long long)dst, c);
                    return false;
                }
                if (off != kBandOutside && ((uint64_t)c * a.plane_src * 4 + off + per * 4 > slab ||
                                            off + per * 4 > (uint64_t)a.plane_src * 4)) {
                    r.fail("fp32 small-C band conv: copy %d lane %d reads byte %u of a plane", j, lane, off);
                    return false;
                }
                for (int e = 0; e < per; ++e) {
                    const int64_t pos = per == 1 ? (int64_t)sp * 64 + lane : (int64_t)sp * 256 + lane * 4 + e - t.shift;
                    int64_t v = kZero;
                    if (off != kBandOutside) {
                        const int64_t elem = (int64_t)t.m0 * g.row_len + pos;
                        if ((int64_t)off / 4 + e != elem) {
                            r.fail("fp32 small-C band conv: strip position %lld copied from element %u", (long long)pos,
                                   off / 4 + e);
                            return false;
                        }
                        v = ((int64_t)c << 24) + elem;
                    }
                    if (holds[dst + e] != -1) {
                        r.fail("fp32 small-C band conv: LDS float %lld written twice", (long long)(dst + e));
                        return false;
                    }
                    holds[dst + e] = v;
                }
            }
        return true;
    };
    // Fused: the pad columns the kernel zeroes once (both buffers' rows: the
    // map must reach exactly the columns outside 0..W-1), then the raw-row
    // copies of band t, each data float written once with (channel << 24) +
    // its x element, or zero for rows outside the image.
    std::vector<int64_t> pads((size_t)2 * rb_f, -1);
    {
        const int padc = a.rpitch - g.w;
        for (int i = 0; i < 2 * C * a.rrows * padc; ++i) {
            const int row = i / padc, k = i % padc;
            const int64_t col = k < a.rlpad ? k : g.w + k;
            if (col >= a.rpitch || (col >= a.rlpad && col < a.rlpad + g.w) || pads[(size_t)row * a.rpitch + col] != -1) {
                r.fail("fp32 small-C band conv: pad zero %d lands on raw column %lld", i, (long long)col);
                return;
            }
            pads[(size_t)row * a.rpitch + col] = kZero;
        }
    }
    auto stage_raw = [&](const BandTile& t) {
        std::copy(pads.begin(), pads.begin() + rb_f, raw.begin());   // buffer 0's pads (buffer 1's are alike)
        if (!std::equal(pads.begin(), pads.begin() + rb_f, pads.begin() + rb_f)) {
            r.fail("fp32 small-C band conv: the two raw buffers' pad columns differ");
            return false;
        }
        const int rper = a.rawwide ? 4 : 1;
        const int64_t y0 = (int64_t)t.m0 * g.sh - g.ph;
        for (int j = 0; j < C * a.rrows * a.rparts; ++j)
            for (int lane = 0; lane < 64; ++lane) {
                const int row = j / a.rparts, pr = j % a.rparts, c = row / a.rrows, rr = row % a.rrows;
                const int64_t yy = y0 + rr, xx = (int64_t)pr * 64 * rper + lane * rper;
                if (xx >= g.w) continue;   // lane masked off
                const int64_t dst = (int64_t)row * a.rpitch + a.rlpad + xx;
                if (xx + rper > g.w || dst + rper > rb_f || (rper == 4 && dst % 4)) {
                    r.fail("fp32 small-C band conv: raw copy %d lane %d writes float %lld past its row", j, lane,
                           (long long)dst);
                    return false;
                }
                const bool in = yy >= 0 && yy < g.h;
                if (in && ((uint64_t)((c * g.h + yy) * g.w + xx) * 4 + rper * 4 > slab)) {
                    r.fail("fp32 small-C band conv: raw copy %d lane %d reads past the image", j, lane);
                    return false;
                }
                for (int e = 0; e < rper; ++e) {
                    if (raw[dst + e] != -1) {
                        r.fail("fp32 small-C band conv: raw float %lld written twice", (long long)(dst + e));
                        return false;
                    }
                    raw[dst + e] = in ? ((int64_t)c << 24) + yy * g.w + xx + e : kZero;
                }
            }
        return true;
    };
    for (int band = 0; band < a.nbands && r.violations == 0; ++band) {
        const BandTile t = smallc_tile(a, band);   // image 0, output-channel group 0
        if (t.band != band || t.img != 0 || t.kt != 0 || t.nrows < 1 || t.npix > nb * 32) {
            r.fail("fp32 small-C band conv: band %d", band);
            return;
        }
        std::fill(holds.begin(), holds.end(), -1);
        if (!fused && !stage_strips(t)) return;
        if (fused && !stage_raw(t)) return;
        for (int wv = 0; wv < kBandThreads / 64 && r.violations == 0; ++wv) {
            const int ks = wv & 1, nq = ks == 0 ? SW : S - SW;
            for (int lane = 0; lane < 64; ++lane)
                for (int b = 0; b < nb; ++b) {
                    int pix = b * 32 + (lane & 31);
                    if (pix > t.npix - 1) pix = t.npix - 1;
                    const int64_t m = t.m0 + pix / g.wo, n = pix % g.wo;
                    const int sl = lane >> 5;
                    for (int i = 0; i < nq; ++i) {
                        const int q = ks * SW + i;
                        // the element this slot multiplies, and the kernel's read:
                        // the slot's base (one channel further in the pair
                        // steps, Fh - HU rows in the last channel's) plus
                        // slot 0's element offset
                        const SmallCStep st = smallc_step(C, FH, FW, q, sl), s0 = smallc_step(C, FH, FW, q, 0);
                        const int c = st.c, uu = st.u, v = st.v;
                        const int64_t f =
                            fused ? smallc_raw_window(a, t, FH, lane, b) / 4 +
                                        (st.pair ? (int64_t)sl * a.rrows : (int64_t)(C - 1) * a.rrows + sl * (FH - HU)) *
                                            a.rpitch +
                                        ((st.pair ? (int64_t)s0.c * a.rrows : 0) + s0.u) * a.rpitch + s0.v
                                  : smallc_window(a, t, FH, lane, b) / 4 +
                                        (st.pair ? (int64_t)sl * a.slotf : (int64_t)(C - 1) * a.slotf + sl * (FH - HU)) +
                                        (st.pair ? (int64_t)s0.c * a.slotf : 0) + (int64_t)s0.v * FH + s0.u;
                        const std::vector<int64_t>& src = fused ? raw : holds;
                        const int64_t yy = m * g.sh + uu - g.ph, xx = n * g.sw + v - g.pw;
                        const bool pad = yy < 0 || yy >= g.h || xx < 0 || xx >= g.w;
                        // unfused: the window-tensor element; fused: the x element, zero in the padding
                        const int64_t elem = fused ? yy * g.w + xx : m * g.row_len + (n * g.sw + v) * FH + uu;
                        const int64_t want = fused && pad ? kZero : ((int64_t)c << 24) + elem;
                        const bool in = f >= 0 && f < (int64_t)src.size();
                        const bool ok = in && uu < FH && src[f] == want;
                        if (!ok) {
                            r.fail("fp32 small-C band conv: band %d wave %d lane %d block %d step %d reads LDS float "
                                   "%lld holding %lld, wants element %lld of channel %d", band, wv, lane, b, q,
                                   (long long)f, (long long)(in ? src[f] : -3), (long long)elem, c);
                            return;
                        }
                    }
                }
        }
        // blocks of output channels past K store nothing; their filter
        // offsets lie past the filter, so they read zeros
        for (int kt = 0; kt < a.nkt; ++kt)
            for (int cb = 0; cb < 2; ++cb) {
                if ((kt * 2 + cb) * 32 >= g.k) {
                    if ((uint64_t)(kt * 2 + cb) * 32 * C * T * 4 < (uint64_t)g.k * C * T * 4) {
                        r.fail("fp32 small-C band conv: idle channel block %d reads the filter", kt * 2 + cb);
                        return;
                    }
                    continue;
                }
                for (int p2 = 0; p2 < t.npix; ++p2)
                    for (int ch = 0; ch < 32; ++ch)
                        ++out[(size_t)((kt * 2 + cb) * 32 + ch) * g.ho * g.wo + (size_t)t.m0 * g.wo + p2];
            }
    }
    if (r.violations) return;
    for (size_t i = 0; i < out.size(); ++i)
        if (out[i] != 1) {
            r.fail("fp32 small-C band conv: output %zu of an image stored %d times", i, (int)out[i]);
            return;
        }
    // outputs go through a buffer resource over one image of y: valid
    // offsets inside it, the dropped-store offset (plus any channel) past its
    // end, no wrap
    const uint64_t y_bytes = (uint64_t)g.k * g.ho * g.wo * 4;
    if (y_bytes > kBandOutside || (uint64_t)kBandOutside + 31ull * g.ho * g.wo * 4 >= (uint64_t(1) << 32))
        r.fail("fp32 small-C band conv: y image of %llu bytes against the dropped-store offset",
               (unsigned long long)y_bytes);
    // every (filter row, column) of every channel is multiplied exactly once
    // per output (the repeated middle row's second copy has zero weight)
    std::vector<int> used((size_t)C * T, 0);
    for (int q = 0; q < S; ++q)
        for (int sl = 0; sl < 2; ++sl) {
            const SmallCStep st = smallc_step(C, FH, FW, q, sl);
            if (st.c < 0 || st.c >= C || st.u < 0 || st.u >= FH || st.v < 0 || st.v >= FW) {
                r.fail("fp32 small-C band conv: step %d slot %d multiplies channel %d row %d column %d", q, sl, st.c,
                       st.u, st.v);
                return;
            }
            if (!st.zero) ++used[(size_t)(st.c * FH + st.u) * FW + st.v];
        }
    for (size_t i = 0; i < used.size(); ++i)
        if (used[i] != 1) {
            r.fail("fp32 small-C band conv: filter element %zu multiplied %d times", i, used[i]);
            return;
        }
    if (conv_scratch_bytes(g, fused) != 0)
        r.fail("fp32 small-C band conv: scratch of %lld bytes requested", (long long)conv_scratch_bytes(g, fused));
}

void check_conv(const Geometry& g, bool fused_plan, Report& r) {
    const F32BandPlan sp = plan_band_small_c_f32(g);
    if (sp.ok && !plan_band_f32(g).ok) {
        check_conv_band_small_c_f32(g, fused_plan, sp, r);
        return;
    }
    const F32BandPlan fp = plan_band_f32(g);
    if (fp.ok) {
        check_conv_band_f32(g, fused_plan, fp, r);
        return;
    }
    const ImgPlan ip = plan_image_bf16(g, fused_plan);
    if (ip.ok) {
        check_conv_image(g, fused_plan, ip, r);
        return;
    }
    const ConvPlan p = g.elem == 2 ? plan_conv_bf16(g, fused_plan) : plan_conv_f32(g);
    // no tile fits in LDS: the per-output kernel runs instead, which indexes
    // every operand directly (no LDS, no plan)
    if (p.kind == ConvPlan::kNone) return;
    const bool bf16 = p.kind == ConvPlan::kBf16Lds;
    if (p.lds_bytes > kConvLdsMaxBytes)
        r.fail("conv: plan uses %lld bytes of LDS", (long long)p.lds_bytes);
    if (!bf16) {
        // fp32 layout: two stages of S[rc][sc] then F[bm][fp]; a k-slot reads
        // at most T + fw past a channel's first tap of a filter row (dead
        // row-split slot) and fh past the last strip position
        if (p.sc < p.strip_cap + g.fh || p.fp < p.rc * g.taps + g.fw + 1 ||
            p.stage < p.rc * p.sc + p.bm * p.fp + g.fw || p.lds_bytes < 4 * 2 * p.stage ||
            (p.sc & 3) != 0 || (p.stage & 3) != 0)
            r.fail("conv: fp32 LDS layout too small (sc %lld, fp %lld, %lld bytes)", (long long)p.sc,
                   (long long)p.fp, (long long)p.lds_bytes);
        if (p.split == 0 && (p.rc & 1))
            r.fail("conv: channel split with an odd chunk of %d", p.rc);
        if (p.fvec && (((g.c * g.taps) & 3) || ((p.rc * g.taps) & 3) || (p.fp & 3)))
            r.fail("conv: 16-byte filter rows with misaligned rows (fp %lld)", (long long)p.fp);
        // repacked filter (rows not whole vectors): blocks of bm*fp floats,
        // copied in 16-byte units to the 16-byte aligned LDS filter rows of a
        // stage; the buffer holds every (tile of output channels, chunk) block
        const ConvArgs af = conv_args_f32(g, p, nullptr, nullptr, nullptr, false);
        if (af.fpack) {
            const int64_t nch = (g.c + p.rc - 1) / p.rc;
            const int64_t jt_last = (g.k - 1) / p.bm, blk_last = jt_last * nch + (nch - 1);
            if (((int64_t)p.bm * p.fp) % 4 || (p.rc * p.sc) % 4 || p.stage % 4 ||
                (blk_last + 1) * p.bm * p.fp != (int64_t)af.num_jtiles * nch * p.bm * p.fp ||
                (int64_t)p.bm * p.fp > p.stage - p.rc * p.sc)
                r.fail("conv: repacked filter blocks of %lld floats do not fit the stage (fp %lld)",
                       (long long)(p.bm * p.fp), (long long)p.fp);
            // the caller's scratch (conv_scratch_bytes) holds every block
            const int64_t need = (blk_last + 1) * p.bm * p.fp * 4;
            if (conv_scratch_bytes(g, false) < need || conv_scratch_bytes(g, true) < need)
                r.fail("conv: filter scratch of %lld bytes, the repacked filter needs %lld",
                       (long long)conv_scratch_bytes(g, false), (long long)need);
        }
        if (conv_args_f32(g, p, nullptr, nullptr, nullptr, false).ilv &&
            (!p.fvec || p.bm * (p.fp / 4) > (int64_t)kConvThreads * kIlvSlots))
            r.fail("conv: %lld 16-byte filter copies per chunk, in-loop issue covers %d", (long long)(p.bm * (p.fp / 4)),
                   kConvThreads * kIlvSlots);
        // raw rows: two buffers with 768 floats of slack each when the map is used
        const int64_t mx = 64 * kF32ExpandGroups;
        const int64_t rawf = (g.fh <= 3 && p.raw_pitch <= mx) ? 2 * (p.rc * p.raw_pitch + mx)
                                                              : p.rc * p.raw_pitch + 6 * (p.raw_pitch / g.w);
        if (g.elem == 4 && p.lds_bytes + 4 * rawf > kConvLdsMaxBytes)
            r.fail("conv: fused plan uses %lld bytes of LDS", (long long)(p.lds_bytes + 4 * rawf));
        if (g.elem == 4 && g.fh <= 3 && p.sc < p.strip_cap + g.fh + 64)
            r.fail("conv: strip stride %lld leaves no spare expansion slots", (long long)p.sc);
        if (g.elem == 4 && (p.raw_pitch & 63))
            r.fail("conv: raw row pitch %lld is not a multiple of 64", (long long)p.raw_pitch);
    }
    if (bf16) {
        // two stages of two strip planes [strip_cap] and two filter planes
        // [cl_fpb >= taps*bm] of 8-element positions
        if (p.rc != kBf16Chunk || p.tc != g.taps || p.cl_fpb < g.taps * p.bm ||
            p.stage < 16 * (p.strip_cap + p.cl_fpb) || p.lds_bytes < 2 * 2 * p.stage ||
            (p.bm & (p.bm - 1)) != 0 || p.cl_pitch < g.row_len)
            r.fail("conv: bf16 LDS layout too small (stage %lld, %lld bytes)", (long long)p.stage,
                   (long long)p.lds_bytes);
        if (p.fvec && ((g.c * g.taps) & 7))
            r.fail("conv: 16-byte bf16 filter rows with C*T = %lld", (long long)(g.c * g.taps));
        if (!p.fvec && 2 * g.taps * p.bm > (int64_t)kConvThreads * kBf16FilterScalarItems)
            r.fail("conv: %lld bf16 filter items exceed the staging registers",
                   (long long)(2 * g.taps * p.bm));
        if (p.fast || p.fused_fast) check_packed_filter(g, p, r);
    }
    if (bf16) {
        // unfused and fused plans may differ (the unfused fast kernel has a
        // larger tile); each is checked for the variant that uses it
        check_conv_bf16_variant(g, p, fused_plan, r);
        return;
    }
    if (fused_plan) return;   // fp32: one plan for both variants
    check_conv_variant(g, p, false, r);
    if (p.svec) check_conv_variant(g, p, true, r);
}

}  // namespace

int64_t check_plans(const Geometry& g, char* msg, size_t msglen) {
    Report r;
    r.msg = msg;
    r.msglen = msglen;
    if (msglen) msg[0] = '\0';
    check_transform(g, r);
    check_conv(g, false, r);
    check_conv(g, true, r);
    return r.violations;
}

}  // namespace im2win
