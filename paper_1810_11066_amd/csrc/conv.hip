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
#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

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

// One output of the convolution, plain loops over in-range taps and words.
// With u the plain binary value sum_j +-2^j b_j of a code (the top plane of
// signed data negative) every encoding is affine in u: value = alpha u + beta
// with (alpha, beta) = (1, 0) for unipolar and signed codes and
// (2, -(2^B - 1)) for bipolar ones.  Over the in-range taps
//   sum value(a) value(w) = aa aw S + aa bw SA + ba aw SW + ba bw N
// where S = sum_{i,j} +-2^(i+j) popcount(a_i AND w_j) (Eq. 2 with the sign of
// each plane pair), SA and SW the plane-weighted popcounts of the activation
// and weight words, and N the number of in-range channel values.  All sums
// wrap in uint32; the host's overflow bound makes the result exact.
__device__ __forceinline__ uint32_t generic_output(
    const ConvShape& s, const uint32_t* __restrict__ act,
    const uint32_t* __restrict__ wts, int cw, uint32_t img, uint32_t oy,
    uint32_t ox, uint32_t o) {
    const bool sa_neg = s.aenc == kSigned, sw_neg = s.wenc == kSigned;
    uint32_t sum = 0, sa = 0, sw = 0, nval = 0;
    for (int r = 0; r < s.kh; ++r) {
        const int iy = (int)oy * s.sh - s.ph + r;
        if (iy < 0 || iy >= s.h) continue;          // zero padding
        for (int c = 0; c < s.kw; ++c) {
            const int ix = (int)ox * s.sw - s.pw + c;
            if (ix < 0 || ix >= s.w) continue;      // zero padding
            const uint32_t* ap =
                act + (((int64_t)img * s.h + iy) * s.w + ix) *
                          (int64_t)s.abits * cw;
            const uint32_t* wp =
                wts + (((int64_t)o * s.kh + r) * s.kw + c) *
                          (int64_t)s.wbits * cw;
            nval += (uint32_t)s.c;
            for (int t = 0; t < cw; ++t) {
                for (int i = 0; i < s.abits; ++i) {
                    const uint32_t a = ap[i * cw + t];
                    const bool ni = sa_neg && i == s.abits - 1;
                    const uint32_t pa = (uint32_t)__builtin_popcount(a) << i;
                    sa += ni ? 0u - pa : pa;
                    for (int j = 0; j < s.wbits; ++j) {
                        const uint32_t w = wp[j * cw + t];
                        const bool nj = sw_neg && j == s.wbits - 1;
                        const uint32_t term =
                            (uint32_t)__builtin_popcount(a & w) << (i + j);
                        sum += ni != nj ? 0u - term : term;
                    }
                }
                for (int j = 0; j < s.wbits; ++j) {
                    const bool nj = sw_neg && j == s.wbits - 1;
                    const uint32_t pw =
                        (uint32_t)__builtin_popcount(wp[j * cw + t]) << j;
                    sw += nj ? 0u - pw : pw;
                }
            }
        }
    }
    const uint32_t aa = s.aenc == kBipolar ? 2u : 1u;
    const uint32_t ba = s.aenc == kBipolar ? 0u - ((1u << s.abits) - 1) : 0u;
    const uint32_t aw = s.wenc == kBipolar ? 2u : 1u;
    const uint32_t bw = s.wenc == kBipolar ? 0u - ((1u << s.wbits) - 1) : 0u;
    return aa * aw * sum + aa * bw * sa + ba * aw * sw + ba * bw * nval;
}

__global__ __launch_bounds__(kBlock) void conv_generic_kernel(GenericArgs g) {
    const ConvShape& s = g.s;
    for (uint32_t f = blockIdx.x * kBlock + threadIdx.x; f < g.total;
         f += gridDim.x * kBlock) {
        const uint32_t pix = g.div_oc.div(f), o = f - pix * (uint32_t)s.oc;
        const uint32_t rowi = g.div_ow.div(pix), ox = pix - rowi * (uint32_t)s.ow;
        const uint32_t img = g.div_oh.div(rowi), oy = rowi - img * (uint32_t)s.oh;
        g.out[f] = (int32_t)generic_output(s, g.act, g.wts, g.cw, img, oy, ox,
                                           o);
    }
}

// Requantized, bit-packed output, plain loops: one thread per (pixel, word
// of 32 output channels).
struct GenericRequantArgs {
    const uint32_t* act;
    const uint32_t* wts;
    uint32_t* out;
    ConvShape s;
    int32_t cw;
    int32_t words;        // ceil(oc / 32)
    uint32_t total;       // npix * words, < 2^31
    float scale, qmax;
    int32_t bits;
    FastDiv div_words, div_ow, div_oh;
};

__global__ __launch_bounds__(kBlock) void conv_generic_requant_kernel(
    GenericRequantArgs g) {
    const ConvShape& s = g.s;
    for (uint32_t f = blockIdx.x * kBlock + threadIdx.x; f < g.total;
         f += gridDim.x * kBlock) {
        const uint32_t pix = g.div_words.div(f), w = f - pix * (uint32_t)g.words;
        const uint32_t rowi = g.div_ow.div(pix), ox = pix - rowi * (uint32_t)s.ow;
        const uint32_t img = g.div_oh.div(rowi), oy = rowi - img * (uint32_t)s.oh;
        uint32_t word[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        const int c1 = min(32, s.oc - 32 * (int)w);
        for (int c = 0; c < c1; ++c) {
            const uint32_t v = generic_output(s, g.act, g.wts, g.cw, img, oy,
                                              ox, 32 * w + c);
            const uint32_t code =
                quant_code<false>((float)(int32_t)v, g.scale, g.qmax);
            // constant indices keep word[] in registers
#pragma unroll
            for (int b = 0; b < 8; ++b)
                if (b < g.bits) word[b] |= ((code >> b) & 1u) << c;
        }
        uint32_t* dst = g.out + (size_t)pix * (uint32_t)(g.bits * g.words) + w;
#pragma unroll
        for (int b = 0; b < 8; ++b)
            if (b < g.bits) dst[(size_t)b * g.words] = word[b];
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
    // unipolar activations with unipolar or bipolar filters only
    if (s.aenc != kUnipolar || s.wenc == kSigned) return false;
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

// Images per launch of the pixels-on-lanes kernel: all of them, or as many
// as keep the packed activations and the int32 output (not the packed
// output of a requantizing call) within the kernel's 32-bit buffer offsets
// and its unit counts within int32; 0 when one image is already too large.
// Bytes of one image's activations as a pixels-on-lanes kernel with
// activation source src reads them: bit-packed words, uint8 codes or
// float32 values.
int64_t pix_act_image_bytes(const ConvShape& s, int src) {
    const int64_t hw = (int64_t)s.h * s.w;
    if (src == pix::kSrcCodes) return hw * s.c;
    if (src == pix::kSrcFloat) return hw * s.c * 4;
    return hw * s.abits * ((s.c + 31) / 32) * 4;
}

int64_t pix_images_per_launch(const ConvShape& s, bool req,
                              int src = pix::kSrcPacked) {
    const int64_t act_img = pix_act_image_bytes(s, src);
    const int64_t pix_img = (int64_t)s.oh * s.ow;
    const int64_t out_img = req ? 0 : pix_img * s.oc * 4;
    const int64_t lim = pix::kMaxBufferBytes;
    int64_t n = s.n;
    if (act_img > 0) n = n < lim / act_img ? n : lim / act_img;
    if (out_img > 0) n = n < lim / out_img ? n : lim / out_img;
    // npix < 2^31 and units = ceil(npix / 64) * (oc / 4) < 2^30
    const int64_t by_pix = (INT32_MAX - 64) / pix_img;
    n = n < by_pix ? n : by_pix;
    while (n > 0 && ((n * pix_img + 63) / 64) * (s.oc / 4) >= INT32_MAX / 2)
        n = n / 2;
    return n;
}

// Pixels-on-lanes kernel for this shape, or nullptr.  src: where the
// activations come from (pix::kSrcPacked, kSrcCodes, kSrcFloat); the staged
// forms read whole 32-code words of each pixel, so they need c % 32 == 0.
pix::PixKernelFn pix_kernel_for(const ConvShape& s, bool req, int src,
                                pix::PlanInfo* info, bool dual = false) {
    const int64_t cw = (s.c + 31) / 32;
    if (s.abits > 4 || s.wbits > 4) return nullptr;
    if (s.kh != s.kw || s.sh != s.sw) return nullptr;
    // output tiles are written in 16-byte quads of channels
    if (s.oc % 4 != 0) return nullptr;
    if (src != pix::kSrcPacked && s.c % 32 != 0) return nullptr;
    if (pix_images_per_launch(s, req, src) < 1) return nullptr;
    return pix::pick(s.abits, s.wbits, s.aenc, s.wenc, s.kh, s.sh, (int)cw,
                     req, src, dual, info);
}

// Compute units of the current device (cached per device).
int device_cus() {
    static std::atomic<int> cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount,
                              dev) != hipSuccess || v < 1)
        v = 256;
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

// Resident blocks of fn per CU (register, LDS and wave-slot limits), cached
// per kernel and device.  The runtime counts SGPRs the way the compiler does,
// which overstates residency above 80 SGPRs; the pixel kernels use up to 96,
// where the hardware holds pix::kWavesPerSimd waves per SIMD.
int resident_blocks(pix::PixKernelFn fn, size_t lds) {
    struct Entry { pix::PixKernelFn fn; int dev; size_t lds; int blocks; };
    static std::mutex mu;
    static std::vector<Entry> cache;
    int dev = 0;
    (void)hipGetDevice(&dev);
    {
        std::lock_guard<std::mutex> lock(mu);
        for (const Entry& e : cache)
            if (e.fn == fn && e.dev == dev && e.lds == lds) return e.blocks;
    }
    int blocks = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &blocks, (const void*)fn, pix::kBlock, lds) != hipSuccess ||
        blocks < 1)
        return 1;
    // 4 SIMDs per CU
    const int cap = 4 * pix::kWavesPerSimd / pix::kWavesPerBlock;
    if (blocks > cap) blocks = cap;
    std::lock_guard<std::mutex> lock(mu);
    cache.push_back({fn, dev, lds, blocks});
    return blocks;
}

// Largest input region, in pixels, that a block of a staged launch packs
// into LDS (pix::block_region, or for strided 1x1 windows the block's output
// pixel count, for every block of the plan in g; blocks are only renumbered
// by the XCD-major order, so the set of regions is the same).  Exact, by a
// pass over the blocks, cached per shape and run length.
int64_t max_region_pixels(const ConvShape& s, const pix::PixArgs& g) {
    struct Entry {
        int32_t key[12];
        int64_t pixels;
    };
    static std::mutex mu;
    static std::vector<Entry> cache;
    const int32_t key[12] = {s.n, s.h, s.w, s.oh, s.ow, s.ph, s.kh, s.sh,
                             g.units, g.group_units, g.per_wave, g.npix};
    {
        std::lock_guard<std::mutex> lock(mu);
        for (const Entry& e : cache)
            if (memcmp(e.key, key, sizeof(key)) == 0) return e.pixels;
    }
    const int64_t per_block = (int64_t)pix::kWavesPerBlock * g.per_wave;
    int64_t best = 0;
    for (int64_t ub0 = 0; ub0 < g.units; ub0 += per_block) {
        const int64_t ub1 = ub0 + per_block < g.units ? ub0 + per_block
                                                      : g.units;
        const int64_t p0 = ub0 / g.group_units * 64;
        int64_t p1 = (ub1 - 1) / g.group_units * 64 + 63;
        if (p1 > g.npix - 1) p1 = g.npix - 1;
        if (s.kh == 1 && s.sh > 1) {
            // strided 1x1 windows gather one input pixel per output pixel
            // (pix::stage_gather)
            if (p1 + 1 - p0 > best) best = p1 + 1 - p0;
            continue;
        }
        const int64_t r0 = p0 / s.ow, n0 = r0 / s.oh, y0 = r0 % s.oh;
        const int64_t r1 = p1 / s.ow, n1 = r1 / s.oh, y1 = r1 % s.oh;
        const int64_t x0 = p0 - r0 * s.ow, x1 = p1 - r1 * s.ow;
        const int64_t a = y0 * s.sh - s.ph, b = y1 * s.sh - s.ph + s.kh - 1;
        const int64_t iy_lo = std::min<int64_t>(std::max<int64_t>(a, 0), s.h);
        const int64_t iy_hi =
            std::max<int64_t>(std::min<int64_t>(b, s.h - 1), -1);
        int64_t lo = (n0 * s.h + iy_lo) * s.w;
        int64_t hi = (n1 * s.h + iy_hi) * s.w + s.w;
        // the columns of the first and last tap rows that no tap reads
        // (pix::block_region)
        if (a >= 0 && a < s.h)
            lo += std::min<int64_t>(std::max<int64_t>(x0 * s.sw - s.pw, 0),
                                    s.w - 1);
        if (b >= 0 && b < s.h)
            hi -= s.w - 1 - std::max<int64_t>(
                                std::min<int64_t>(x1 * s.sw - s.pw + s.kw - 1,
                                                  s.w - 1),
                                0);
        if (hi < lo) hi = lo;
        if (hi - lo > best) best = hi - lo;
    }
    std::lock_guard<std::mutex> lock(mu);
    Entry e;
    memcpy(e.key, key, sizeof(key));
    e.pixels = best;
    if (cache.size() < 256) cache.push_back(e);
    return best;
}

// Launch configuration of a pixels-on-lanes call.  The work is units of
// (64-pixel group, 4 output channels); each wave takes a contiguous run of
// L units.  L is the smallest run that keeps the grid resident in one round
// (at most `resident` blocks per CU), adjusted upwards while that lowers the
// busiest CU's load (blocks per CU x L), so that CUs end together.
// `lds` is the dynamic LDS per block the plan assumes for residency.
void plan_pix_lds(const ConvShape& s, pix::PixKernelFn fn, int forced_run,
                  const Requant* rq, pix::PixArgs* g, dim3* grid,
                  size_t lds) {
    g->h = s.h; g->w = s.w; g->oh = s.oh; g->ow = s.ow;
    g->ph = s.ph; g->pw = s.pw;
    g->c = s.c;
    g->oc = s.oc;
    g->npix = s.n * s.oh * s.ow;
    g->quads = s.oc / 4;
    // requantizing kernels store packed bytes (8 channels = 2 quads of one
    // pixel), so their units are whole bytes
    g->unit_quads = rq ? 2 : 1;
    g->group_units = (g->quads + g->unit_quads - 1) / g->unit_quads;
    g->out_scale = rq ? rq->scale : 0.0f;
    g->out_bits = rq ? rq->bits : 0;
    g->out_qmax = rq ? (float)((1 << rq->bits) - 1) : 0.0f;
    g->out_words = (s.oc + 31) / 32;
    const int64_t groups = ((int64_t)g->npix + 63) / 64;
    const int64_t units = groups * g->group_units;
    g->units = (int32_t)units;
    g->div_ow.init((uint32_t)s.ow);
    g->div_oh.init((uint32_t)s.oh);
    g->div_units.init((uint32_t)g->group_units);
    // within kMaxBufferBytes (pix_images_per_launch)
    g->act_bytes = (int32_t)((int64_t)s.n * s.h * s.w * s.abits *
                             ((s.c + 31) / 32) * 4);
    g->out_bytes = rq ? 0 : (int32_t)((int64_t)g->npix * s.oc * 4);
    g->region_pixels = 0;
    g->in_scale = 0.0f;
    g->in_qmax = 0.0f;
    g->out1 = nullptr;
    g->out1_scale = 0.0f;
    g->out1_bytes = 0;
    const int64_t cus = device_cus();
    const int64_t slots = cus * resident_blocks(fn, lds);   // blocks
    const int64_t wpb = pix::kWavesPerBlock;
    int64_t lmin = (units + slots * wpb - 1) / (slots * wpb);
    if (lmin < 1) lmin = 1;
    auto load = [&](int64_t l) {   // busiest CU: blocks per CU x units
        const int64_t waves = (units + l - 1) / l;
        const int64_t blocks = (waves + wpb - 1) / wpb;
        return (blocks + cus - 1) / cus * l;
    };
    int64_t best = lmin;
    for (int64_t l = lmin + 1; l <= 2 * lmin; ++l)
        if (load(l) < load(best)) best = l;
    // 1x1 layers with few word pairs per result (A W words <= 16) are bound
    // by their int32 stores, not by the vector ALUs: runs of one tile chunk
    // of quads make every flush write whole 64-byte pieces of the pixel
    // rows (a run boundary inside a chunk leaves pieces of 16-48 bytes, which
    // the memory system handles at a fraction of the rate), however many
    // rounds of waves that takes.  Measured on the ResNet-18 1x1 layers:
    // 5-20 % faster than the balanced single-round plan.
    const int64_t cw = (s.c + 31) / 32;
    if (!rq && s.kh == 1 && s.abits * s.wbits * cw <= 16)
        best = pix::kChunk / 4;
    if (forced_run > 0) best = forced_run;
    if (best > units) best = units;
    g->per_wave = (int32_t)best;
    const int64_t waves = (units + best - 1) / best;
    *grid = dim3((uint32_t)((waves + wpb - 1) / wpb));
}

constexpr size_t kTileLds = (size_t)pix::kWavesPerBlock * pix::kTileWords * 4;
constexpr size_t kMaxBlockLds = 64 * 1024;

// Plan of a call with packed activations: the LDS holds the output tiles.
void plan_pix(const ConvShape& s, pix::PixKernelFn fn, int forced_run,
              const Requant* rq, pix::PixArgs* g, dim3* grid, size_t* lds) {
    *lds = kTileLds;
    plan_pix_lds(s, fn, forced_run, rq, g, grid, *lds);
}

// Plan of a staged call: the LDS also holds the block's packed input region
// plus one zero pixel, whose size depends on the run length, which depends
// on residency, which depends on the LDS: re-plan until the residency the
// plan assumed is the one its LDS allows.  False when the region does not
// fit a block's LDS.  src: kSrcCodes, or kSrcFloat with the quantizer's
// scale in_scale.
bool plan_pix_staged(const ConvShape& s, pix::PixKernelFn fn, int forced_run,
                     int src, float in_scale, pix::PixArgs* g, dim3* grid,
                     size_t* lds) {
    const size_t pwb = (size_t)s.abits * ((s.c + 31) / 32) * 4;
    size_t assumed = kTileLds;
    int run = forced_run;
    if (run == 0 && src == pix::kSrcFloat && s.kh == 1 && s.sh > 1) {
        // float32 pixels gathered for strided 1x1 windows: each workgroup
        // that takes part of a 64-pixel group loads and quantizes all of
        // the group's pixels, so runs are lengthened until at most two
        // workgroups share a group, as long as the grid keeps a workgroup
        // for at least every other CU (ResNet-18 layers 8 and 11 at batch
        // 128: 18.3 -> 15.5-16.8 and 13.7 -> 11.3-12.1 us per launch;
        // layer 5 already had two; at batch 16 layer 11's grid would fall
        // to 26 workgroups and its launch took 10.8 instead of 7.5 us)
        plan_pix_lds(s, fn, 0, nullptr, g, grid, assumed);
        const int two = 2 * pix::kWavesPerBlock;
        const int min_run = (g->group_units + two - 1) / two;
        const int64_t per_block = (int64_t)pix::kWavesPerBlock * min_run;
        const int64_t blocks = ((int64_t)g->units + per_block - 1) / per_block;
        if (g->per_wave < min_run && 2 * blocks >= device_cus())
            run = min_run;
    }
    for (int iter = 0; iter < 24; ++iter) {
        plan_pix_lds(s, fn, run, nullptr, g, grid, assumed);
        const int64_t region = max_region_pixels(s, *g);
        const size_t need = kTileLds + (size_t)(region + 1) * pwb;
        if (need > kMaxBlockLds) {
            // a block's rows do not fit: shorter runs (fewer pixels per
            // block), unless the caller fixed the run length
            if (forced_run > 0 || g->per_wave <= 1) return false;
            run = g->per_wave / 2;
            continue;
        }
        g->region_pixels = (int32_t)region;
        // the kernel reads the uint8 codes or float32 values (within
        // kMaxBufferBytes: pix_images_per_launch with src)
        g->act_bytes = (int32_t)(s.n * pix_act_image_bytes(s, src));
        g->in_scale = in_scale;
        g->in_qmax = (float)((1 << s.abits) - 1);
        *lds = need;
        if (need <= assumed ||
            resident_blocks(fn, need) >= resident_blocks(fn, assumed))
            return true;
        assumed = need;
    }
    return false;
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

// The second output of a paired kernel: the centre-tap 1x1 conv's packed
// filters, its output (shaped like the main one) and, for requantized
// output, its scale.
struct Pair {
    const uint32_t* wts1;
    int32_t* out1;
    float scale1;
};

// Launches the pixels-on-lanes kernel fn over the batch, in chunks of
// pix_images_per_launch images (a single launch unless the tensors pass
// 2 GB).  rq: requantized, bit-packed output (out holds uint32 words);
// pair: the second output of a paired kernel, or nullptr.
hipError_t launch_pix(const ConvShape& s, pix::PixKernelFn fn,
                      const uint32_t* act, const uint32_t* wts, int32_t* out,
                      int forced_run, const Requant* rq, hipStream_t st,
                      const Pair* pair = nullptr) {
    const int64_t per = pix_images_per_launch(s, rq != nullptr);
    const int64_t cw = (s.c + 31) / 32;
    const int64_t act_img = (int64_t)s.h * s.w * s.abits * cw;
    const int64_t out_img =
        rq ? (int64_t)s.oh * s.ow * rq->bits * ((s.oc + 31) / 32)
           : (int64_t)s.oh * s.ow * s.oc;
    // paired int32 output: runs of one tile chunk (4 quads), so that every
    // flush of either output writes whole, aligned 64-byte pieces of the
    // pixel rows.  Measured on ResNet-18 layers 4+5 at batch 128: 38.3 us
    // against 57.8 us with the balanced plan's runs of 7 (chunks straddling
    // 64-byte pieces, twice the bytes of a plain conv), and 46.5 us for the
    // two convolutions launched one after the other.
    if (pair && !rq && forced_run == 0 && s.oc % pix::kChunk == 0)
        forced_run = pix::kChunk / 4;
    for (int64_t n0 = 0; n0 < s.n; n0 += per) {
        ConvShape c = s;
        c.n = (int32_t)(s.n - n0 < per ? s.n - n0 : per);
        pix::PixArgs g;
        dim3 grid;
        size_t lds = 0;
        plan_pix(c, fn, forced_run, rq, &g, &grid, &lds);
        if (pair) {
            g.out1 = pair->out1 + n0 * out_img;
            g.out1_scale = pair->scale1;
            g.out1_bytes = g.out_bytes;
        }
        const uint32_t* a = act + n0 * act_img;
        int32_t* o = out + n0 * out_img;
        // kernels without a paired conv never read wts1
        const uint32_t* w1 = pair ? pair->wts1 : wts;
        const hipError_t e =
            launch(fn, grid, dim3(pix::kBlock), lds, st, a, wts, w1, o, g);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// Staged launch: uint8 activation codes (src kSrcCodes) or float32 values
// quantized with in_scale (kSrcFloat), NHWC [n][h][w][c], are bit-packed
// into each block's LDS by the conv kernel itself.  Every image chunk is
// planned before anything is enqueued; hipErrorNotSupported (nothing
// enqueued) when no staged kernel or no fitting plan exists.
hipError_t launch_pix_staged(const ConvShape& s, const void* act, int src,
                             float in_scale, const uint32_t* wts,
                             int32_t* out, int forced_run, hipStream_t st) {
    pix::PlanInfo info{};
    const pix::PixKernelFn fn = pix_kernel_for(s, false, src, &info);
    if (!fn) return hipErrorNotSupported;
    const int64_t per = pix_images_per_launch(s, false, src);
    struct Chunk {
        int64_t n0;
        pix::PixArgs g;
        dim3 grid;
        size_t lds;
    };
    std::vector<Chunk> chunks;
    for (int64_t n0 = 0; n0 < s.n; n0 += per) {
        ConvShape c = s;
        c.n = (int32_t)(s.n - n0 < per ? s.n - n0 : per);
        Chunk ch;
        ch.n0 = n0;
        if (!plan_pix_staged(c, fn, forced_run, src, in_scale, &ch.g,
                             &ch.grid, &ch.lds))
            return hipErrorNotSupported;
        chunks.push_back(ch);
    }
    const int64_t in_img = pix_act_image_bytes(s, src);
    const int64_t out_img = (int64_t)s.oh * s.ow * s.oc;
    for (const Chunk& ch : chunks) {
        const uint32_t* a = reinterpret_cast<const uint32_t*>(
            static_cast<const uint8_t*>(act) + ch.n0 * in_img);
        int32_t* o = out + ch.n0 * out_img;
        const hipError_t e = launch(fn, ch.grid, dim3(pix::kBlock), ch.lds, st,
                                    a, wts, wts, o, ch.g);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

enum class Family { kPixels, kChannels, kGeneric };

// The kernel family a call takes: mode 0 tries pixels-on-lanes, then
// channels-on-lanes, then generic; 3 and 2 try only their own family before
// generic; 1 is generic only.
Family choose(const ConvShape& s, int mode, pix::PixKernelFn* pfn,
              pix::PlanInfo* info) {
    if (mode == 0 || mode == 3) {
        if ((*pfn = pix_kernel_for(s, false, pix::kSrcPacked, info)) !=
            nullptr)
            return Family::kPixels;
    }
    if ((mode == 0 || mode == 2) && conv_has_fast_path(s))
        return Family::kChannels;
    return Family::kGeneric;
}

}  // namespace

hipError_t launch_conv(const ConvShape& s, const uint32_t* act,
                       const uint32_t* wts, int32_t* out,
                       const ConvOptions& opt, hipStream_t st) {
    const int mode = opt.mode;
    pix::PixKernelFn pfn = nullptr;
    pix::PlanInfo info{};
    dim3 grid;
    size_t lds = 0;
    switch (choose(s, mode, &pfn, &info)) {
        case Family::kPixels:
            return launch_pix(s, pfn, act, wts, out, opt.units_per_wave,
                              nullptr, st);
        case Family::kChannels: {
            FastArgs g;
            plan_fast(s, &g, &grid, &lds);
            const KernelFn fn = pick_fast(s.abits, s.wbits, s.bipolar_w, s.kh,
                                          s.sh, pick_group_pixels(s.ow),
                                          g.cw);
            return launch(fn, grid, dim3(kBlock), lds, st, act, wts, out, g);
        }
        case Family::kGeneric:
        default: {
            GenericArgs g;
            plan_generic(s, act, wts, out, &g, &grid);
            return launch(conv_generic_kernel, grid, dim3(kBlock), 0, st, g);
        }
    }
}

hipError_t launch_conv_requant(const ConvShape& s, const uint32_t* act,
                               const uint32_t* wts, uint32_t* out,
                               const Requant& rq, const ConvOptions& opt,
                               hipStream_t st) {
    // the pixels-on-lanes kernel (modes 0 and 3), else plain loops
    pix::PlanInfo info{};
    pix::PixKernelFn pfn = nullptr;
    if (opt.mode == 0 || opt.mode == 3)
        pfn = pix_kernel_for(s, true, pix::kSrcPacked, &info);
    if (pfn) {
        // the run-length override counts packed bytes (2 quads) here
        return launch_pix(s, pfn, act, wts, reinterpret_cast<int32_t*>(out),
                          opt.units_per_wave, &rq, st);
    }
    GenericRequantArgs g;
    g.act = act;
    g.wts = wts;
    g.out = out;
    g.s = s;
    g.cw = (s.c + 31) / 32;
    g.words = (s.oc + 31) / 32;
    g.total = (uint32_t)((int64_t)s.n * s.oh * s.ow * g.words);
    g.scale = rq.scale;
    g.qmax = (float)((1 << rq.bits) - 1);
    g.bits = rq.bits;
    g.div_words.init((uint32_t)g.words);
    g.div_ow.init((uint32_t)s.ow);
    g.div_oh.init((uint32_t)s.oh);
    int64_t blocks = ((int64_t)g.total + kBlock - 1) / kBlock;
    if (blocks > 65535) blocks = 65535;
    if (blocks < 1) blocks = 1;
    return launch(conv_generic_requant_kernel, dim3((uint32_t)blocks),
                  dim3(kBlock), 0, st, g);
}

// The centre-tap 1x1 conv paired with s: same input, stride and output
// grid, no padding.
static ConvShape pair_shape(const ConvShape& s) {
    ConvShape s1 = s;
    s1.kh = s1.kw = 1;
    s1.ph = s1.pw = 0;
    return s1;
}

hipError_t launch_conv_pair(const ConvShape& s, const uint32_t* act,
                            const uint32_t* wts, const uint32_t* wts1,
                            int32_t* out, int32_t* out1, const Requant* rq,
                            float scale1, const ConvOptions& opt,
                            hipStream_t st) {
    pix::PlanInfo info{};
    pix::PixKernelFn fn = nullptr;
    if (opt.mode == 0 || opt.mode == 3)
        fn = pix_kernel_for(s, rq != nullptr, pix::kSrcPacked, &info, true);
    if (fn) {
        const Pair pair{wts1, out1, scale1};
        return launch_pix(s, fn, act, wts, out, opt.units_per_wave, rq, st,
                          &pair);
    }
    // no paired kernel for this shape: the two convolutions one by one
    const ConvShape s1 = pair_shape(s);
    hipError_t e;
    if (rq) {
        e = launch_conv_requant(s, act, wts, reinterpret_cast<uint32_t*>(out),
                                *rq, opt, st);
        if (e != hipSuccess) return e;
        Requant rq1 = *rq;
        rq1.scale = scale1;
        return launch_conv_requant(s1, act, wts1,
                                   reinterpret_cast<uint32_t*>(out1), rq1, opt,
                                   st);
    }
    e = launch_conv(s, act, wts, out, opt, st);
    if (e != hipSuccess) return e;
    return launch_conv(s1, act, wts1, out1, opt, st);
}

hipError_t launch_conv_codes(const ConvShape& s, const uint8_t* act,
                             const uint32_t* wts, int32_t* out,
                             const ConvOptions& opt, hipStream_t st) {
    return launch_pix_staged(s, act, pix::kSrcCodes, 0.0f, wts, out,
                             opt.units_per_wave, st);
}

hipError_t launch_conv_quantized(const ConvShape& s, const float* act,
                                 float scale, const uint32_t* wts,
                                 int32_t* out, const ConvOptions& opt,
                                 hipStream_t st) {
    return launch_pix_staged(s, act, pix::kSrcFloat, scale, wts, out,
                             opt.units_per_wave, st);
}

namespace {

// The encodings a pixel-kernel specialisation was compiled for, as text.
void kernel_encodings(const pix::PlanInfo& info, char* out, size_t len) {
    static const char* const names[3] = {"unipolar", "bipolar", "signed"};
    if (info.enc / 3 == kUnipolar)
        snprintf(out, len, "%s", names[info.enc % 3]);
    else
        snprintf(out, len, "%s x %s", names[info.enc / 3],
                 names[info.enc % 3]);
}

}  // namespace

int describe_conv_staged(const ConvShape& s, bool from_float,
                         const ConvOptions& opt, char* buf, size_t len) {
    const int src = from_float ? pix::kSrcFloat : pix::kSrcCodes;
    pix::PlanInfo info{};
    const pix::PixKernelFn fn = pix_kernel_for(s, false, src, &info);
    if (!fn) return -1;
    // the plan of the first launch (of `launches` image chunks)
    const int64_t per = pix_images_per_launch(s, false, src);
    ConvShape c = s;
    c.n = (int32_t)(s.n < per ? s.n : per);
    pix::PixArgs g;
    dim3 grid;
    size_t lds = 0;
    if (!plan_pix_staged(c, fn, opt.units_per_wave, src, 1.0f, &g, &grid,
                         &lds))
        return -1;
    const int64_t launches = (s.n + per - 1) / per;
    char kenc[48];
    kernel_encodings(info, kenc, sizeof(kenc));
    return snprintf(buf, len,
                    "conv_pix_kernel<A=%d,W=%d,%s,K=%d,S=%d,CW=%d> "
                    "staged %s: patch=%dtaps x %dwords slice=%dch x "
                    "%dtaps grid=%u block=%d lds=%zu region=%dpx units=%d "
                    "units_per_wave=%d%s",
                    s.abits, s.wbits, kenc, s.kh, s.sh, (s.c + 31) / 32,
                    from_float ? "float32" : "codes",
                    info.tb, info.cb, info.ocb, info.ts, grid.x, pix::kBlock,
                    lds, g.region_pixels, g.units, g.per_wave,
                    launches > 1 ? " (per launch; batch split)" : "");
}

int describe_conv(const ConvShape& s, const ConvOptions& opt, char* buf,
                  size_t len) {
    const int mode = opt.mode;
    pix::PixKernelFn pfn = nullptr;
    pix::PlanInfo info{};
    dim3 grid;
    size_t lds = 0;
    const int cw = (s.c + 31) / 32;
    static const char* const names[3] = {"unipolar", "bipolar", "signed"};
    char enc[48];
    if (s.aenc == kUnipolar)
        snprintf(enc, sizeof(enc), "%s", names[s.wenc]);
    else
        snprintf(enc, sizeof(enc), "%s x %s", names[s.aenc], names[s.wenc]);
    switch (choose(s, mode, &pfn, &info)) {
        case Family::kPixels: {
            // the plan of the first launch (of `launches` image chunks)
            const int64_t per = pix_images_per_launch(s, false);
            ConvShape c = s;
            c.n = (int32_t)(s.n < per ? s.n : per);
            pix::PixArgs g;
            plan_pix(c, pfn, opt.units_per_wave, nullptr, &g, &grid, &lds);
            const int64_t launches = (s.n + per - 1) / per;
            char kenc[48];
            kernel_encodings(info, kenc, sizeof(kenc));
            return snprintf(buf, len,
                            "conv_pix_kernel<A=%d,W=%d,%s,K=%d,S=%d,CW=%d> "
                            "patch=%dtaps x %dwords slice=%dch x %dtaps "
                            "grid=%u block=%d lds=%zu units=%d "
                            "units_per_wave=%d%s",
                            s.abits, s.wbits, kenc, s.kh, s.sh, cw, info.tb,
                            info.cb, info.ocb, info.ts, grid.x, pix::kBlock,
                            lds, g.units, g.per_wave,
                            launches > 1 ? " (per launch; batch split)" : "");
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
