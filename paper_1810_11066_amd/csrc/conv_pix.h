// Pixels-on-lanes bitserial conv kernel template; instantiated in
// conv_pix.hip.
//
// Mapping.  Lane l of a block owns one output pixel (n, oy, ox); a block of
// 256 lanes covers 256 consecutive output pixels in NHWC order, and
// blockIdx.y selects a contiguous range of output channels.  Each lane loads
// the packed words of its K x K input patch once (vector loads; consecutive
// lanes read consecutive pixels), zeroes the taps that fall in the padding,
// and keeps the patch in VGPRs for all of its output channels.  The filter
// words of an output channel are the same for every lane, so they are read
// with scalar loads (the filters of a layer are small and stay in the scalar
// cache) and used as the SGPR operand of v_and_b32.
//
// Inner loop: per (tap, plane pair, word) one v_and_b32 (SGPR x VGPR) and one
// accumulating v_bcnt_u32_b32 into one of A+W-1 per-shift accumulators; the
// shift-add (and bipolar correction, whose popcount sum over the patch is
// computed once per lane) runs once per output.  Scalar work is one wait and
// a few offset adds per OCB output channels, so the vector unit stays fed.
//
// The filter loads of channel batch b+1 are issued before batch b is
// computed (two SGPR buffers); scalar loads return out of order, so the wait
// for batch b is placed explicitly before batch b+1 is issued.
#pragma once

#include "bs_internal.h"

namespace bs {
namespace pix {

constexpr int kBlock = 256;

struct PixArgs {
    int32_t h, w, oc, oh, ow, sh, sw, ph, pw;
    int32_t npix;          // n * oh * ow
    int32_t oc_per_block;  // output channels per blockIdx.y: a multiple of
                           // kChunk, or all of them (oc % 4 == 0)
    FastDiv div_ow, div_oh;
};

__device__ __forceinline__ void bcnt_acc(uint32_t& acc, uint32_t x) {
    asm("v_bcnt_u32_b32 %0, %1, %0" : "+v"(acc) : "v"(x));
}

// Order this wave's LDS writes before its following LDS reads (and the reads
// before later writes).  The tile is private to the wave, so no block-wide
// barrier is needed.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ void wait_scalar_loads() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt untouched
}

typedef const uint32_t __attribute__((address_space(1))) gu32;

// Filter words of OCB consecutive output channels: OHWI packing puts each
// filter's K*K*W*CW words contiguously and consecutive filters next to each
// other, so a batch is one contiguous run (merged into wide scalar loads).
template <int K, int W, int CW, int OCB>
struct FilterBatch {
    uint32_t w[OCB][K * K][W][CW];
};

template <int K, int W, int CW, int OCB>
__device__ __forceinline__ void load_filters(FilterBatch<K, W, CW, OCB>& fb,
                                             gu32* __restrict__ wts,
                                             int oc) {
    constexpr int FW = K * K * W * CW;   // words per filter
    gu32* src = wts + (size_t)oc * FW;
#pragma unroll
    for (int o = 0; o < OCB; ++o)
#pragma unroll
        for (int t = 0; t < K * K; ++t)
#pragma unroll
            for (int j = 0; j < W; ++j)
#pragma unroll
                for (int c = 0; c < CW; ++c)
                    fb.w[o][t][j][c] = src[((o * K * K + t) * W + j) * CW + c];
}

// The OCB channels of a batch are interleaved and each accumulator is split
// in two (even / odd taps), so consecutive popcounts go to 2 * OCB * (A+W-1)
// independent accumulators instead of one dependency chain per channel.
template <int A, int W, bool BIP, int K, int CW, int OCB>
__device__ __forceinline__ void compute_batch(
    const uint32_t (&patch)[K * K][A][CW],
    const FilterBatch<K, W, CW, OCB>& fb, uint32_t sa, uint32_t (&val)[OCB]) {
    constexpr int NS = A + W - 1;
    uint32_t acc[2][OCB][NS];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int o = 0; o < OCB; ++o)
#pragma unroll
            for (int s = 0; s < NS; ++s) acc[h][o][s] = 0;
#pragma unroll
    for (int t = 0; t < K * K; ++t)
#pragma unroll
        for (int c = 0; c < CW; ++c)
#pragma unroll
            for (int j = 0; j < W; ++j)
#pragma unroll
                for (int i = 0; i < A; ++i)
#pragma unroll
                    for (int o = 0; o < OCB; ++o)
                        bcnt_acc(acc[(t * CW + c) & 1][o][i + j],
                                 patch[t][i][c] & fb.w[o][t][j][c]);
#pragma unroll
    for (int o = 0; o < OCB; ++o) {
        uint32_t v = 0;
#pragma unroll
        for (int s = 0; s < NS; ++s) v += (acc[0][o][s] + acc[1][o][s]) << s;
        // bipolar weight value 2w - (2^W - 1): 2*sum - (2^W - 1)*sum(a)
        if (BIP) v = 2u * v - (uint32_t)((1 << W) - 1) * sa;
        val[o] = v;
    }
}

// Output tile staging.  With pixels on lanes, the NHWC output of one output
// channel is 4 bytes per lane at a stride of oc * 4 bytes -- one memory
// request per lane.  Results are therefore collected per wave in LDS as a
// 64-pixel x kChunk-channel tile and written back with each lane storing 16
// contiguous bytes (4 lanes per pixel row of the chunk).
constexpr int kChunk = 16;                 // output channels per LDS tile
constexpr int kTileStride = kChunk + 1;    // words per pixel row (padded)
constexpr int kTileWords = 64 * kTileStride;

__device__ __forceinline__ void flush_tile(
    const uint32_t* __restrict__ tile, int32_t* __restrict__ out,
    int pix0, int npix, int oc_total, int oc_base, int nch, int lane) {
    // nch (a multiple of 4, at most kChunk) channels of 64 pixels:
    // nch / 4 lanes per pixel row
    const int lanes_per_pix = nch >> 2;
    const int pix_per_round = 64 / lanes_per_pix;
    const bool active = lane < pix_per_round * lanes_per_pix;
    for (int r = 0; r < 64; r += pix_per_round) {
        const int px = r + lane / lanes_per_pix;
        const int q = lane % lanes_per_pix;
        if (active && px < 64 && pix0 + px < npix) {
            const uint32_t* t = tile + px * kTileStride + 4 * q;
            *reinterpret_cast<uint4*>(
                out + (int64_t)(pix0 + px) * oc_total + oc_base + 4 * q) =
                make_uint4(t[0], t[1], t[2], t[3]);
        }
    }
}

// A, W: bit-widths; BIP: bipolar weights; K: square kernel size; S: stride;
// CW: words per bit-plane; OCB: output channels per filter batch.
template <int A, int W, bool BIP, int K, int S, int CW, int OCB>
__global__ __launch_bounds__(kBlock) void conv_pix_kernel(
    const uint32_t* __restrict__ act, const uint32_t* __restrict__ wts,
    int32_t* __restrict__ out, PixArgs g) {
    constexpr int PW = A * CW;           // words per packed input pixel
    const int p = blockIdx.x * kBlock + threadIdx.x;
    const bool valid = p < g.npix;
    const uint32_t pc = (uint32_t)(valid ? p : g.npix - 1);
    const uint32_t rowi = g.div_ow.div(pc);
    const int ox = (int)(pc - rowi * (uint32_t)g.ow);
    const uint32_t img = g.div_oh.div(rowi);
    const int oy = (int)(rowi - img * (uint32_t)g.oh);

    // the lane's input patch; taps in the zero padding are zero
    uint32_t patch[K * K][A][CW];
#pragma unroll
    for (int r = 0; r < K; ++r) {
        const int iy = oy * S - g.ph + r;
#pragma unroll
        for (int s = 0; s < K; ++s) {
            const int ix = ox * S - g.pw + s;
            const bool in = (unsigned)iy < (unsigned)g.h &&
                            (unsigned)ix < (unsigned)g.w;
            const int64_t pix = in ? ((int64_t)img * g.h + iy) * g.w + ix : 0;
            const uint32_t* src = act + pix * PW;
            uint32_t wv[PW];
            if constexpr (PW % 4 == 0) {
#pragma unroll
                for (int k = 0; k < PW; k += 4) {
                    const uint4 x = *reinterpret_cast<const uint4*>(src + k);
                    wv[k] = x.x; wv[k + 1] = x.y; wv[k + 2] = x.z; wv[k + 3] = x.w;
                }
            } else if constexpr (PW % 2 == 0) {
#pragma unroll
                for (int k = 0; k < PW; k += 2) {
                    const uint2 x = *reinterpret_cast<const uint2*>(src + k);
                    wv[k] = x.x; wv[k + 1] = x.y;
                }
            } else {
#pragma unroll
                for (int k = 0; k < PW; ++k) wv[k] = src[k];
            }
#pragma unroll
            for (int i = 0; i < A; ++i)
#pragma unroll
                for (int c = 0; c < CW; ++c)
                    patch[r * K + s][i][c] = in ? wv[i * CW + c] : 0u;
        }
    }
    uint32_t sa = 0;   // bipolar: sum_i 2^i popcount(a_i) over the patch
    if (BIP) {
#pragma unroll
        for (int t = 0; t < K * K; ++t)
#pragma unroll
            for (int i = 0; i < A; ++i)
#pragma unroll
                for (int c = 0; c < CW; ++c)
                    sa += (uint32_t)__builtin_popcount(patch[t][i][c]) << i;
    }

    gu32* gw = (gu32*)(wts);
    const int oc0 = blockIdx.y * g.oc_per_block;
    const int oc1 = min(oc0 + g.oc_per_block, g.oc);

    // per-wave output tile in LDS
    extern __shared__ uint32_t lds[];
    const int lane = threadIdx.x & 63;
    uint32_t* tile = lds + (threadIdx.x >> 6) * kTileWords;
    const int pix0 = p - lane;   // first pixel of this wave

    FilterBatch<K, W, CW, OCB> f0, f1;
    uint32_t val[OCB];
    load_filters<K, W, CW, OCB>(f0, gw, oc0);
    for (int oc = oc0; oc < oc1; oc += 2 * OCB) {
        wait_scalar_loads();
        const bool more = oc + OCB < oc1;
        if (more) load_filters<K, W, CW, OCB>(f1, gw, oc + OCB);
        __builtin_amdgcn_sched_barrier(0);
        compute_batch<A, W, BIP, K, CW, OCB>(patch, f0, sa, val);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int o = 0; o < OCB; ++o)
            tile[lane * kTileStride + (oc - oc0) % kChunk + o] = val[o];
        if (more) {
            wait_scalar_loads();
            if (oc + 2 * OCB < oc1)
                load_filters<K, W, CW, OCB>(f0, gw, oc + 2 * OCB);
            __builtin_amdgcn_sched_barrier(0);
            compute_batch<A, W, BIP, K, CW, OCB>(patch, f1, sa, val);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int o = 0; o < OCB; ++o)
                tile[lane * kTileStride + (oc + OCB - oc0) % kChunk + o] =
                    val[o];
        }
        // a full chunk of channels (or the last, shorter one) is ready
        const int done = oc + 2 * OCB - oc0;
        if (done % kChunk == 0 || oc + 2 * OCB >= oc1) {
            const int base = oc0 + ((done - 1) / kChunk) * kChunk;
            wave_lds_sync();
            flush_tile(tile, out, pix0, g.npix, g.oc, base,
                       min(kChunk, oc1 - base), lane);
            wave_lds_sync();
        }
    }
}

using PixKernelFn = void (*)(const uint32_t*, const uint32_t*, int32_t*,
                             PixArgs);

// Kernel for a supported (A, W, bipolar, K, S, CW) or nullptr; also reports
// the filter batch size the kernel uses.
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb);

}  // namespace pix
}  // namespace bs
