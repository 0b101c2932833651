// Output-channels-on-lanes bitserial conv kernel template; instantiated per
// activation bit-width in conv_fast_a{1,2,3,4}.hip so the specialisations
// compile in parallel.
//
// Mapping.  Lane l of a wave owns output channel oc_base + l; a wave walks
// groups of P consecutive output pixels of one output row.  For a group and a
// filter row r, the input pixels under the group form one contiguous run of
// NI = (P-1) S + K pixels in NHWC memory.  Their packed words are identical
// for all 64 lanes, so they are fetched with scalar loads into SGPRs; the
// filter words are per lane (per output channel) and come from LDS, where the
// block's 64 filters are staged once, laid out [tap][plane][word pair][lane]
// so that the 64 lanes read 64 consecutive 8-byte slots (no bank conflicts).
//
// Inner loop: per (pixel, tap, plane pair, word) one v_and_b32 (SGPR x VGPR)
// and one accumulating v_bcnt_u32_b32 into one of A+W-1 per-shift int32
// accumulators of the P x 64 register tile.  The shift-add over shift levels
// (and the bipolar correction 2 sum - (2^W - 1) sum_i 2^i popcount(a_i)) runs
// once per output; stores are 64 consecutive int32 per pixel.
//
// Scalar-issue budget.  A SIMD issues at most one scalar and one vector
// instruction per cycle slot, so the address arithmetic of the scalar loads
// must stay well below the AND/popcount count.  Addresses are therefore 32-bit
// byte offsets from the activation base (the host limits the packed tensor to
// 2^31 bytes), advanced incrementally, and groups that lie fully inside the
// image take a path without per-pixel border selects.
#pragma once

#include "bs_internal.h"

namespace bs {
namespace fast {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;

struct FastArgs {
    int32_t h, w, cw, oc, oh, ow, ph, pw;
    int32_t pix_bytes;     // A * cw * 4: one packed input pixel
    int32_t plane_bytes;   // cw * 4: one bit-plane of one pixel
    int32_t gpr;           // pixel groups per output row, ceil(ow / P)
    int32_t total_groups;  // n * oh * gpr
    int32_t gpw;           // groups per wave
    FastDiv div_gpr, div_oh;
};

// Accumulate one filter row for one group: NI input pixels starting at byte
// offset `off` (pixel q at off + q * pix_bytes), word pair t2 already folded
// into `off`.  EDGE: some pixels may lie in the zero padding; those are read
// from the row's first pixel (always valid) and replaced by zeros.
// acc += popcount(x), pinned to the accumulating form of v_bcnt_u32_b32.
// Written as plain C the compiler regroups chains of such sums into
// v_bcnt(x, 0) + v_add3, one extra VALU op per two words.
__device__ __forceinline__ void bcnt_acc(uint32_t& acc, uint32_t x) {
    asm("v_bcnt_u32_b32 %0, %1, %0" : "+v"(acc) : "v"(x));
}

// Accumulate one filter row for one group: NI input pixels starting at byte
// offset `off` (pixel q at off + q * pix_bytes), word pair t2 already folded
// into `off`.  Offsets are unsigned 32-bit so that each scalar load takes its
// offset straight from an SGPR.  EDGE: some pixels may lie in the zero
// padding; those are read from the row's first pixel (always valid) and
// replaced by zeros.
template <int A, int W, bool BIP, int K, int S, int P, bool EDGE>
__device__ __forceinline__ void accumulate_row(
    const char* __restrict__ act, uint32_t off, uint32_t valid_off, int ix0,
    int width, uint32_t pix_bytes, uint32_t plane_bytes,
    const uint2 (&wr)[K][W], uint32_t (&acc)[P][A + W - 1],
    uint32_t (&sa)[P]) {
    constexpr int NI = (P - 1) * S + K;
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        bool v = true;
        uint32_t o = off;
        if (EDGE) {
            v = (unsigned)(ix0 + q) < (unsigned)width;
            o = v ? off : valid_off;
        }
        uint32_t a[A][2];
#pragma unroll
        for (int i = 0; i < A; ++i) {
            const uint2 x = *reinterpret_cast<const uint2*>(
                act + (size_t)(o + (uint32_t)i * plane_bytes));
            a[i][0] = (EDGE && !v) ? 0u : x.x;
            a[i][1] = (EDGE && !v) ? 0u : x.y;
        }
        uint32_t pc = 0;
        if (BIP) {
#pragma unroll
            for (int i = 0; i < A; ++i)
                pc += (uint32_t)(__builtin_popcount(a[i][0]) +
                                 __builtin_popcount(a[i][1]))
                      << i;
        }
#pragma unroll
        for (int s = 0; s < K; ++s) {
            const int d = q - s;
            if (d < 0 || d % S != 0 || d / S >= P) continue;  // compile time
            const int p = d / S;
#pragma unroll
            for (int j = 0; j < W; ++j)
#pragma unroll
                for (int i = 0; i < A; ++i) {
                    bcnt_acc(acc[p][i + j], a[i][0] & wr[s][j].x);
                    bcnt_acc(acc[p][i + j], a[i][1] & wr[s][j].y);
                }
            if (BIP) sa[p] += pc;
        }
        off += pix_bytes;
    }
}

// A, W: bit-widths; BIP: bipolar weights; K: square kernel size; S: stride
// (both directions); P: output pixels per group (register tile P x 64).
template <int A, int W, bool BIP, int K, int S, int P>
__global__ __launch_bounds__(kBlock) void conv_ocl_kernel(
    const uint32_t* __restrict__ act, const uint32_t* __restrict__ wts,
    int32_t* __restrict__ out, FastArgs g) {
    extern __shared__ uint32_t lds[];
    constexpr int NI = (P - 1) * S + K;  // input pixels under one group row
    constexpr int NS = A + W - 1;        // shift levels i + j
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cw = g.cw;                 // even
    const int half = cw >> 1;
    const int oc_base = blockIdx.y * 64;
    const int noc = min(64, g.oc - oc_base);
    const int wwords = K * K * W * cw;   // packed words per filter

    // Stage the 64 filters: word widx of filter o goes to
    // lds[((widx / 2) * 64 + o) * 2 + widx % 2]; missing filters are zero.
    {
        const uint32_t* src = wts + (int64_t)oc_base * wwords;
        const int total = 64 * wwords;
        for (int e = threadIdx.x; e < total; e += kBlock) {
            const int widx = e >> 6, o = e & 63;
            const uint32_t v = o < noc ? src[(int64_t)o * wwords + widx] : 0u;
            lds[((widx >> 1) * 64 + o) * 2 + (widx & 1)] = v;
        }
    }
    __syncthreads();

    const uint2* lw = reinterpret_cast<const uint2*>(lds) + lane;
    const char* abytes = reinterpret_cast<const char*>(act);
    const uint32_t pix_bytes = (uint32_t)g.pix_bytes;
    const uint32_t plane_bytes = (uint32_t)g.plane_bytes;
    const bool oc_ok = lane < noc;
    const int64_t g0 = ((int64_t)blockIdx.x * kWavesPerBlock + wave) * g.gpw;

    for (int gi = 0; gi < g.gpw; ++gi) {
        const int64_t grp64 = g0 + gi;
        if (grp64 >= g.total_groups) break;
        const uint32_t grp = (uint32_t)grp64;
        const uint32_t rowi = g.div_gpr.div(grp);
        const int gx = (int)(grp - rowi * (uint32_t)g.gpr);
        const uint32_t img = g.div_oh.div(rowi);
        const int oy = (int)(rowi - img * (uint32_t)g.oh);
        const int ox0 = gx * P;
        const int ix0 = ox0 * S - g.pw;
        const bool interior = ix0 >= 0 && ix0 + NI <= g.w;

        uint32_t acc[P][NS];
        uint32_t sa[P];   // bipolar: sum_i 2^i popcount(a_i) over the window
#pragma unroll
        for (int p = 0; p < P; ++p) {
            sa[p] = 0;
#pragma unroll
            for (int s = 0; s < NS; ++s) acc[p][s] = 0;
        }

#pragma unroll
        for (int r = 0; r < K; ++r) {
            const int iy = oy * S - g.ph + r;
            if (iy < 0 || iy >= g.h) continue;           // zero padding row
            const int row_pix = ((int)img * g.h + iy) * g.w;
            // (may wrap below zero for ix0 < 0; such pixels are never read)
            const uint32_t row_off = (uint32_t)(row_pix + ix0) * pix_bytes;
            const uint32_t valid_off = (uint32_t)row_pix * pix_bytes;
            for (int t2 = 0; t2 < half; ++t2) {
                uint2 wr[K][W];
#pragma unroll
                for (int s = 0; s < K; ++s)
#pragma unroll
                    for (int j = 0; j < W; ++j)
                        wr[s][j] = lw[(((r * K + s) * W + j) * half + t2) * 64];
                if (interior)
                    accumulate_row<A, W, BIP, K, S, P, false>(
                        abytes, row_off + 8u * t2, 0u, ix0, g.w, pix_bytes,
                        plane_bytes, wr, acc, sa);
                else
                    accumulate_row<A, W, BIP, K, S, P, true>(
                        abytes, row_off + 8u * t2, valid_off + 8u * t2, ix0,
                        g.w, pix_bytes, plane_bytes, wr, acc, sa);
            }
        }

        const int64_t orow = ((int64_t)img * g.oh + oy) * g.ow;
#pragma unroll
        for (int p = 0; p < P; ++p) {
            const int ox = ox0 + p;
            if (ox < g.ow && oc_ok) {
                uint32_t val = 0;
#pragma unroll
                for (int s = 0; s < NS; ++s) val += acc[p][s] << s;
                // bipolar weight value 2w - (2^W - 1): 2*sum - (2^W - 1)*sum(a)
                if (BIP) val = 2u * val - (uint32_t)((1 << W) - 1) * sa[p];
                out[(orow + ox) * g.oc + oc_base + lane] = (int32_t)val;
            }
        }
    }
}

using KernelFn = void (*)(const uint32_t*, const uint32_t*, int32_t*,
                         FastArgs);

// Kernel for (A, wbits, bipolar, kernel size, stride, group pixels); defined
// for A = 1..4 in conv_fast_a<A>.hip.
template <int A>
KernelFn pick_w(int w, bool b, int k, int s, int p);
template <> KernelFn pick_w<1>(int w, bool b, int k, int s, int p);
template <> KernelFn pick_w<2>(int w, bool b, int k, int s, int p);
template <> KernelFn pick_w<3>(int w, bool b, int k, int s, int p);
template <> KernelFn pick_w<4>(int w, bool b, int k, int s, int p);

}  // namespace fast
}  // namespace bs
