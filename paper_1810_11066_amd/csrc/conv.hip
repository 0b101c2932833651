// Bitserial conv2d / dense kernels for gfx950 (wave64).
//
// Both kernels evaluate, for every output, Eq. 2 over packed bit-planes:
//   out = sum_{i<A} sum_{j<W} 2^(i+j) sum_t f(a_i[t], w_j[t])
// with f = popcount(a AND w) for unipolar weights and
// f = popcount(a AND w) - popcount(a AND NOT w) for bipolar weights (Sec. 2.2).
// Accumulation is in uint32 and wraps; the host rejects any problem whose
// exact result could leave int32, so the wrapped sum equals the exact result.
//
// Three kernel families; the host picks one per call (launch_conv):
//
// conv_pix_kernel      "pixels on lanes" (conv_pix.h): lane l owns one output
//                      pixel and keeps its packed input patch in VGPRs; the
//                      filter words of each output channel are uniform across
//                      the wave and arrive by scalar loads as the SGPR operand
//                      of v_and_b32.  The fastest family for the 3x3 and 1x1
//                      ResNet layers; used first where it applies.
// conv_ocl_kernel      "output channels on lanes" (conv_fast.h): lane l owns
//                      output channel oc0 + l, the wave walks groups of P
//                      output pixels of one row; activation words are uniform
//                      across the wave (scalar loads), filter words of the
//                      block's 64 channels are staged once in LDS.  Serves
//                      the shapes the pixel kernel does not (wide channels,
//                      oc not a multiple of 4).
// conv_generic_kernel  one output per thread, runtime everything; serves
//                      every remaining shape.
//
// In both fast families the inner loop is one v_and_b32 (SGPR x VGPR) and one
// accumulating v_bcnt_u32_b32 per word pair, into A+W-1 per-shift
// accumulators per output; the shift-add (and bipolar correction) runs once
// per output.
#include <cstdio>

#include "conv_fast.h"
#include "conv_pix.h"

namespace bs {
namespace {

using fast::kBlock;
using fast::kWavesPerBlock;
using fast::FastArgs;
using fast::KernelFn;

// ---------------------------------------------------------------------------
struct GenericArgs {
    const uint32_t* act;
    const uint32_t* wts;
    int32_t* out;
    ConvShape s;
    int32_t cw;
    uint32_t total;   // n*oh*ow*oc, < 2^31
    FastDiv div_oc, div_ow, div_oh;
};

__global__ __launch_bounds__(kBlock) void conv_generic_kernel(GenericArgs g) {
    const ConvShape& s = g.s;
    const int cw = g.cw;
    for (uint32_t f = blockIdx.x * kBlock + threadIdx.x; f < g.total;
         f += gridDim.x * kBlock) {
        const uint32_t pix = g.div_oc.div(f), o = f - pix * (uint32_t)s.oc;
        const uint32_t rowi = g.div_ow.div(pix), ox = pix - rowi * (uint32_t)s.ow;
        const uint32_t img = g.div_oh.div(rowi), oy = rowi - img * (uint32_t)s.oh;
        uint32_t sum = 0;
        for (int r = 0; r < s.kh; ++r) {
            const int iy = (int)oy * s.sh - s.ph + r;
            if (iy < 0 || iy >= s.h) continue;          // zero padding
            for (int c = 0; c < s.kw; ++c) {
                const int ix = (int)ox * s.sw - s.pw + c;
                if (ix < 0 || ix >= s.w) continue;      // zero padding
                const uint32_t* ap =
                    g.act + (((int64_t)img * s.h + iy) * s.w + ix) *
                                (int64_t)s.abits * cw;
                const uint32_t* wp =
                    g.wts + (((int64_t)o * s.kh + r) * s.kw + c) *
                                (int64_t)s.wbits * cw;
                for (int t = 0; t < cw; ++t) {
                    for (int i = 0; i < s.abits; ++i) {
                        const uint32_t a = ap[i * cw + t];
                        for (int j = 0; j < s.wbits; ++j) {
                            const uint32_t w = wp[j * cw + t];
                            uint32_t term = __builtin_popcount(a & w);
                            if (s.bipolar_w) term -= __builtin_popcount(a & ~w);
                            sum += term << (i + j);
                        }
                    }
                }
            }
        }
        g.out[f] = (int32_t)sum;
    }
}

KernelFn pick_fast(int a, int w, bool b, int k, int s, int p, int cw) {
    switch (a) {
        case 1: return fast::pick_w<1>(w, b, k, s, p, cw);
        case 2: return fast::pick_w<2>(w, b, k, s, p, cw);
        case 3: return fast::pick_w<3>(w, b, k, s, p, cw);
        default: return fast::pick_w<4>(w, b, k, s, p, cw);
    }
}

constexpr int64_t kMaxLdsBytes = 64 * 1024;

#ifndef BS_PIX_WAVES_PER_SIMD
#define BS_PIX_WAVES_PER_SIMD 8
#endif

#ifndef BS_CONV_WAVES_PER_SIMD
#define BS_CONV_WAVES_PER_SIMD 4
#endif

int64_t fast_lds_bytes(const ConvShape& s) {
    const int64_t cw = (s.c + 31) / 32;
    return 64 * (int64_t)s.kh * s.kw * s.wbits * cw * 4;
}

int pick_group_pixels(int ow) { return ow % 7 == 0 ? 7 : 8; }

}  // namespace

bool conv_has_fast_path(const ConvShape& s) {
    const int64_t cw = (s.c + 31) / 32;
    const int p = pick_group_pixels(s.ow);
    if (s.abits > 4 || s.wbits > 4) return false;
    if (s.kh != s.kw || (s.kh != 1 && s.kh != 3)) return false;
    if (s.sh != s.sw || (s.sh != 1 && s.sh != 2)) return false;
    if (cw % 2 != 0) return false;
    if (fast_lds_bytes(s) > kMaxLdsBytes) return false;
    // padded input pixels of a group row are read from the zero buffer
    const int64_t ni = (int64_t)(p - 1) * s.sw + s.kw;
    if (ni * s.abits * cw * 4 > fast::kZeroBytes) return false;
    const int64_t gpr = (s.ow + p - 1) / p;
    const int64_t groups = (int64_t)s.n * s.oh * gpr;
    if (groups >= INT32_MAX / 2) return false;
    // scalar-load addressing uses 32-bit byte offsets into the activations
    const int64_t act_bytes = (int64_t)s.n * s.h * s.w * s.abits * cw * 4;
    if (act_bytes >= INT32_MAX) return false;
    return true;
}

namespace {

// Pixels-on-lanes kernel for this shape, or nullptr.
pix::PixKernelFn pix_kernel_for(const ConvShape& s, int* ocb) {
    const int64_t cw = (s.c + 31) / 32;
    if (s.abits > 4 || s.wbits > 4) return nullptr;
    if (s.kh != s.kw || s.sh != s.sw) return nullptr;
    if ((int64_t)s.n * s.oh * s.ow >= INT32_MAX) return nullptr;
    pix::PixKernelFn fn = pix::pick(s.abits, s.wbits, s.bipolar_w, s.kh, s.sh,
                                    (int)cw, ocb);
    // output tiles are written in 16-byte quads of channels
    if (!fn || s.oc % 4 != 0) return nullptr;
    return fn;
}

// Launch configuration of a pixels-on-lanes call.
void plan_pix(const ConvShape& s, pix::PixArgs* g, dim3* grid, size_t* lds) {
    g->h = s.h; g->w = s.w; g->oc = s.oc; g->oh = s.oh; g->ow = s.ow;
    g->sh = s.sh; g->sw = s.sw; g->ph = s.ph; g->pw = s.pw;
    g->npix = s.n * s.oh * s.ow;
    g->div_ow.init((uint32_t)s.ow);
    g->div_oh.init((uint32_t)s.oh);
    const int64_t bx = ((int64_t)g->npix + pix::kBlock - 1) / pix::kBlock;
    // split the output channels so that the chip holds several rounds of
    // waves (256 CUs x 4 SIMDs x BS_PIX_WAVES_PER_SIMD)
    const int64_t waves_x = bx * (pix::kBlock / 64);
    int64_t ysplit = (256 * 4 * (int64_t)BS_PIX_WAVES_PER_SIMD + waves_x - 1) /
                     waves_x;
    const int64_t max_split = (s.oc + pix::kChunk - 1) / pix::kChunk;
    if (ysplit > max_split) ysplit = max_split;
    if (ysplit < 1) ysplit = 1;
    int64_t per = (s.oc + ysplit - 1) / ysplit;
    per = (per + pix::kChunk - 1) / pix::kChunk * pix::kChunk;
    if (per > s.oc) per = s.oc;
    g->oc_per_block = (int32_t)per;
    const int64_t by = (s.oc + per - 1) / per;
    *grid = dim3((uint32_t)bx, (uint32_t)by);
    *lds = (size_t)(pix::kBlock / 64) * pix::kTileWords * 4;
}

// Launch configuration of a channels-on-lanes call.
void plan_fast(const ConvShape& s, FastArgs* g, dim3* grid, size_t* lds) {
    const int32_t cw = (s.c + 31) / 32;
    const int p = pick_group_pixels(s.ow);
    g->h = s.h; g->w = s.w; g->cw = cw; g->oc = s.oc; g->oh = s.oh;
    g->ow = s.ow; g->ph = s.ph; g->pw = s.pw;
    g->plane_bytes = cw * 4;
    g->pix_bytes = s.abits * cw * 4;
    g->gpr = (s.ow + p - 1) / p;
    g->total_groups = s.n * s.oh * g->gpr;
    g->div_gpr.init((uint32_t)g->gpr);
    g->div_oh.init((uint32_t)s.oh);
    const int oc_blocks = (s.oc + 63) / 64;
    // persistent grid: about BS_CONV_WAVES_PER_SIMD resident waves on each
    // SIMD (256 CUs x 4 SIMDs), no more blocks than groups need
    const int64_t want_blocks =
        (256 * 4 * (int64_t)BS_CONV_WAVES_PER_SIMD / kWavesPerBlock +
         oc_blocks - 1) / oc_blocks;
    const int64_t need_blocks =
        ((int64_t)g->total_groups + kWavesPerBlock - 1) / kWavesPerBlock;
    const int64_t bx = want_blocks < need_blocks ? want_blocks : need_blocks;
    *grid = dim3((uint32_t)bx, oc_blocks);
    *lds = (size_t)fast_lds_bytes(s);
}

void plan_generic(const ConvShape& s, const uint32_t* act, const uint32_t* wts,
                  int32_t* out, GenericArgs* g, dim3* grid) {
    g->act = act;
    g->wts = wts;
    g->out = out;
    g->s = s;
    g->cw = (s.c + 31) / 32;
    g->total = (uint32_t)((int64_t)s.n * s.oh * s.ow * s.oc);
    g->div_oc.init((uint32_t)s.oc);
    g->div_ow.init((uint32_t)s.ow);
    g->div_oh.init((uint32_t)s.oh);
    int64_t blocks = ((int64_t)g->total + kBlock - 1) / kBlock;
    if (blocks > 65535) blocks = 65535;
    if (blocks < 1) blocks = 1;
    *grid = dim3((uint32_t)blocks);
}

enum class Family { kPixels, kChannels, kGeneric };

// The kernel family a call takes: mode 0 tries pixels-on-lanes, then
// channels-on-lanes, then generic; 3 and 2 try only their own family before
// generic; 1 is generic only.
Family choose(const ConvShape& s, int mode, pix::PixKernelFn* pfn, int* ocb) {
    if (mode == 0 || mode == 3) {
        if ((*pfn = pix_kernel_for(s, ocb)) != nullptr) return Family::kPixels;
    }
    if ((mode == 0 || mode == 2) && conv_has_fast_path(s))
        return Family::kChannels;
    return Family::kGeneric;
}

}  // namespace

hipError_t launch_conv(const ConvShape& s, const uint32_t* act,
                       const uint32_t* wts, int32_t* out, int mode,
                       hipStream_t st) {
    pix::PixKernelFn pfn = nullptr;
    int ocb = 1;
    dim3 grid;
    size_t lds = 0;
    switch (choose(s, mode, &pfn, &ocb)) {
        case Family::kPixels: {
            pix::PixArgs g;
            plan_pix(s, &g, &grid, &lds);
            void* args[] = {&act, &wts, &out, &g};
            return hipLaunchKernel((const void*)pfn, grid, dim3(pix::kBlock),
                                   args, lds, st);
        }
        case Family::kChannels: {
            FastArgs g;
            plan_fast(s, &g, &grid, &lds);
            const KernelFn fn = pick_fast(s.abits, s.wbits, s.bipolar_w, s.kh,
                                          s.sh, pick_group_pixels(s.ow),
                                          g.cw);
            void* args[] = {&act, &wts, &out, &g};
            return hipLaunchKernel((const void*)fn, grid, dim3(kBlock), args,
                                   lds, st);
        }
        case Family::kGeneric:
        default: {
            GenericArgs g;
            plan_generic(s, act, wts, out, &g, &grid);
            conv_generic_kernel<<<grid, kBlock, 0, st>>>(g);
            return hipGetLastError();
        }
    }
}

int describe_conv(const ConvShape& s, int mode, char* buf, size_t len) {
    pix::PixKernelFn pfn = nullptr;
    int ocb = 1;
    dim3 grid;
    size_t lds = 0;
    const int cw = (s.c + 31) / 32;
    const char* enc = s.bipolar_w ? "bipolar" : "unipolar";
    switch (choose(s, mode, &pfn, &ocb)) {
        case Family::kPixels: {
            pix::PixArgs g;
            plan_pix(s, &g, &grid, &lds);
            return snprintf(buf, len,
                            "conv_pix_kernel<A=%d,W=%d,%s,K=%d,S=%d,CW=%d,"
                            "OCB=%d> grid=%ux%u block=%d lds=%zu "
                            "oc_per_block=%d",
                            s.abits, s.wbits, enc, s.kh, s.sh, cw, ocb, grid.x,
                            grid.y, pix::kBlock, lds, g.oc_per_block);
        }
        case Family::kChannels: {
            FastArgs g;
            plan_fast(s, &g, &grid, &lds);
            return snprintf(buf, len,
                            "conv_ocl_kernel<A=%d,W=%d,%s,K=%d,S=%d,P=%d,"
                            "CW=%d> grid=%ux%u block=%d lds=%zu",
                            s.abits, s.wbits, enc, s.kh, s.sh,
                            pick_group_pixels(s.ow), cw, grid.x, grid.y,
                            kBlock, lds);
        }
        case Family::kGeneric:
        default: {
            GenericArgs g;
            plan_generic(s, nullptr, nullptr, nullptr, &g, &grid);
            return snprintf(buf, len,
                            "conv_generic_kernel A=%d W=%d %s grid=%u "
                            "block=%d",
                            s.abits, s.wbits, enc, grid.x, kBlock);
        }
    }
}

}  // namespace bs
