// Output-channels-on-lanes bitserial conv kernel template; instantiated in
// conv_fast_*.hip so the specialisations compile in parallel.
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
// instruction per slot, and scalar loads return out of order (a wave can only
// wait for all of them), so the kernel keeps scalar work per AND/popcount
// pair small:
//  * CW (words per bit-plane) is a template parameter where a specialisation
//    exists, so every load offset inside a group row is an immediate and
//    adjacent loads merge into wide s_load_dwordxN; CW = 0 is the runtime
//    fallback, whose offsets are 32-bit SGPR adds;
//  * taps in the zero padding (rows and pixels) read a static zero buffer
//    instead of branching, so a group body is straight-line code; a group
//    fully inside the image skips even the per-pixel pointer select.
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
    FastDiv div_gpr, div_oh;
};

// acc += popcount(x), pinned to the accumulating form of v_bcnt_u32_b32.
// Written as plain C the compiler regroups chains of such sums into
// v_bcnt(x, 0) + v_add3, one extra VALU op per two words.
__device__ __forceinline__ void bcnt_acc(uint32_t& acc, uint32_t x) {
    asm("v_bcnt_u32_b32 %0, %1, %0" : "+v"(acc) : "v"(x));
}

// Zero-filled memory standing in for input pixels in the zero padding.  A
// padded pixel q of a group row is read at zero + q * pix_bytes + (plane and
// word offsets), so the buffer covers a whole row segment; the host checks
// NI * pix_bytes against its size.
constexpr int kZeroBytes = 16384;
__device__ const uint32_t kZeroPixels[kZeroBytes / 4] = {};

// Bytes in the global address space: selecting between two such pointers
// keeps the result a global (not generic) pointer, so uniform loads through
// it still become scalar loads.
typedef const char __attribute__((address_space(1))) gchar;
typedef const uint64_t __attribute__((address_space(1))) gu64;

__device__ __forceinline__ uint64_t load_pair(gchar* base, uint32_t off,
                                              uint32_t imm) {
    return *(gu64*)(base + (size_t)off + imm);
}

// Operands of one pipeline stage: one filter row r and one word pair t2 of
// every bit-plane -- the activation words of the NI input pixels under the
// group (SGPRs) and this lane's filter words for the K taps of the row
// (VGPRs).
template <int A, int W, int K, int NI>
struct Stage {
    uint32_t a[NI][A][2];
    uint2 wr[K][W];
};

// Wait until every outstanding scalar-memory and LDS load has returned.
__device__ __forceinline__ void wait_loads() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), vmcnt/expcnt untouched
}

// Issue the loads of stage (r, t2).  Taps in the zero padding read the zero
// buffer: a padded row (interior groups) or padded pixel (EDGE groups) keeps
// the same immediate offsets, only its base and SGPR offset change.
template <int A, int W, bool BIP, int K, int S, int P, int CW, bool EDGE>
__device__ __forceinline__ void load_stage(
    Stage<A, W, K, (P - 1) * S + K>& st, gchar* __restrict__ act,
    const uint2* __restrict__ lw, const FastArgs& g, uint32_t img, int oy,
    int ix0, int r, int t2, int half, uint32_t pixb, uint32_t planeb) {
    constexpr int NI = (P - 1) * S + K;
    gchar* zero = (gchar*)(kZeroPixels);
    const int iy = oy * S - g.ph + r;
    const bool row_ok = (unsigned)iy < (unsigned)g.h;
    const int row_pix = ((int)img * g.h + iy) * g.w;
    const uint32_t t2b = 8u * (uint32_t)t2;
    if (EDGE) {
        // exact (non-negative) offset of each in-image pixel
#pragma unroll
        for (int q = 0; q < NI; ++q) {
            const bool v = row_ok && (unsigned)(ix0 + q) < (unsigned)g.w;
            gchar* b = v ? act : zero;
            const uint32_t o = (v ? (uint32_t)(row_pix + ix0 + q) * pixb
                                  : (uint32_t)q * pixb) + t2b;
#pragma unroll
            for (int i = 0; i < A; ++i) {
                const uint64_t x = load_pair(b, o, (uint32_t)i * planeb);
                st.a[q][i][0] = (uint32_t)x;
                st.a[q][i][1] = (uint32_t)(x >> 32);
            }
        }
    } else {
        // one row offset (ix0 >= 0); the pixel index goes to the immediate
        gchar* b = row_ok ? act : zero;
        const uint32_t o =
            (row_ok ? (uint32_t)(row_pix + ix0) * pixb : 0u) + t2b;
#pragma unroll
        for (int q = 0; q < NI; ++q)
#pragma unroll
            for (int i = 0; i < A; ++i) {
                const uint64_t x = load_pair(
                    b, o, (uint32_t)q * pixb + (uint32_t)i * planeb);
                st.a[q][i][0] = (uint32_t)x;
                st.a[q][i][1] = (uint32_t)(x >> 32);
            }
    }
#pragma unroll
    for (int s = 0; s < K; ++s)
#pragma unroll
        for (int j = 0; j < W; ++j)
            st.wr[s][j] = lw[(((r * K + s) * W + j) * half + t2) * 64];
}

// AND + popcount of one stage into the P x (A+W-1) accumulators.
template <int A, int W, bool BIP, int K, int S, int P>
__device__ __forceinline__ void compute_stage(
    const Stage<A, W, K, (P - 1) * S + K>& st, uint32_t (&acc)[P][A + W - 1],
    uint32_t (&sa)[P]) {
    constexpr int NI = (P - 1) * S + K;
#pragma unroll
    for (int q = 0; q < NI; ++q) {
        uint32_t pc = 0;
        if (BIP) {
#pragma unroll
            for (int i = 0; i < A; ++i)
                pc += (uint32_t)(__builtin_popcount(st.a[q][i][0]) +
                                 __builtin_popcount(st.a[q][i][1]))
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
                    bcnt_acc(acc[p][i + j], st.a[q][i][0] & st.wr[s][j].x);
                    bcnt_acc(acc[p][i + j], st.a[q][i][1] & st.wr[s][j].y);
                }
            if (BIP) sa[p] += pc;
        }
    }
}

// One group: P output pixels (ox0 .. ox0+P-1 of output row oy of image img)
// times the wave's 64 output channels.  EDGE: some input pixels of the group
// lie left or right of the image; decided once per group so that each
// variant keeps its accumulators in fixed registers.
//
// The K * cw/2 stages run as a two-deep software pipeline: after waiting for
// stage n the loads of stage n+1 are issued, then stage n is computed, so the
// latency of the scalar loads hides behind a stage of AND/popcount work.
// (Scalar loads return out of order, so the wait for stage n must come before
// stage n+1 is issued, which is why the wait is explicit.)  Stages too large
// for two SGPR buffers run one at a time.
template <int A, int W, bool BIP, int K, int S, int P, int CW, bool EDGE>
__device__ __forceinline__ void group_body(
    gchar* __restrict__ act, int32_t* __restrict__ out,
    const uint2* __restrict__ lw, const FastArgs& g, uint32_t img, int oy,
    int ox0, int oc_base, int lane, bool oc_ok, bool full) {
    constexpr int NI = (P - 1) * S + K;  // input pixels under one group row
    constexpr int NS = A + W - 1;        // shift levels i + j
    constexpr bool kTwoDeep = NI * A * 2 <= 40;
    const int ix0 = ox0 * S - g.pw;
    const int half = (CW > 0 ? CW : g.cw) >> 1;
    const int nst = K * half;
    const uint32_t pixb = CW > 0 ? (uint32_t)(A * CW * 4) : (uint32_t)g.pix_bytes;
    const uint32_t planeb = CW > 0 ? (uint32_t)(CW * 4) : (uint32_t)g.plane_bytes;

    uint32_t acc[P][NS];
    uint32_t sa[P];   // bipolar: sum_i 2^i popcount(a_i) over the window
#pragma unroll
    for (int p = 0; p < P; ++p) {
        sa[p] = 0;
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[p][s] = 0;
    }

    Stage<A, W, K, NI> s0, s1;
    int r = 0, t2 = 0;   // stage being loaded next
    auto advance = [&]() {
        if (++t2 == half) { t2 = 0; ++r; }
    };
    if (kTwoDeep) {
        load_stage<A, W, BIP, K, S, P, CW, EDGE>(s0, act, lw, g, img, oy, ix0,
                                                 r, t2, half, pixb, planeb);
        advance();
        for (int n = 0; n < nst; n += 2) {
            wait_loads();
            if (n + 1 < nst) {
                load_stage<A, W, BIP, K, S, P, CW, EDGE>(
                    s1, act, lw, g, img, oy, ix0, r, t2, half, pixb, planeb);
                advance();
            }
            __builtin_amdgcn_sched_barrier(0);
            compute_stage<A, W, BIP, K, S, P>(s0, acc, sa);
            __builtin_amdgcn_sched_barrier(0);
            if (n + 1 < nst) {
                wait_loads();
                if (n + 2 < nst) {
                    load_stage<A, W, BIP, K, S, P, CW, EDGE>(
                        s0, act, lw, g, img, oy, ix0, r, t2, half, pixb,
                        planeb);
                    advance();
                }
                __builtin_amdgcn_sched_barrier(0);
                compute_stage<A, W, BIP, K, S, P>(s1, acc, sa);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    } else {
        for (int n = 0; n < nst; ++n) {
            load_stage<A, W, BIP, K, S, P, CW, EDGE>(s0, act, lw, g, img, oy,
                                                     ix0, r, t2, half, pixb,
                                                     planeb);
            advance();
            wait_loads();
            compute_stage<A, W, BIP, K, S, P>(s0, acc, sa);
        }
    }

    // Epilogue: shift-add the shift levels (and apply the bipolar correction)
    // and store.  Groups with all P pixels inside the output row and all 64
    // channels present (the common case) store without per-pixel branches.
    uint32_t val[P];
#pragma unroll
    for (int p = 0; p < P; ++p) {
        uint32_t v = 0;
#pragma unroll
        for (int s = 0; s < NS; ++s) v += acc[p][s] << s;
        // bipolar weight value 2w - (2^W - 1): 2*sum - (2^W - 1)*sum(a)
        if (BIP) v = 2u * v - (uint32_t)((1 << W) - 1) * sa[p];
        val[p] = v;
    }
    int32_t* o = out + (((int64_t)img * g.oh + oy) * g.ow + ox0) * g.oc +
                 oc_base + lane;
    if (full) {
#pragma unroll
        for (int p = 0; p < P; ++p) o[(int64_t)p * g.oc] = (int32_t)val[p];
    } else {
#pragma unroll
        for (int p = 0; p < P; ++p)
            if (ox0 + p < g.ow && oc_ok) o[(int64_t)p * g.oc] = (int32_t)val[p];
    }
}

// A, W: bit-widths; BIP: bipolar weights; K: square kernel size; S: stride
// (both directions); P: output pixels per group (register tile P x 64);
// CW: words per bit-plane (0: taken from the arguments at run time).
template <int A, int W, bool BIP, int K, int S, int P, int CW>
__global__ __launch_bounds__(kBlock) void conv_ocl_kernel(
    const uint32_t* __restrict__ act, const uint32_t* __restrict__ wts,
    int32_t* __restrict__ out, FastArgs g) {
    extern __shared__ uint32_t lds[];
    constexpr int NI = (P - 1) * S + K;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int cw = CW > 0 ? CW : g.cw;   // even
    const int oc_base = blockIdx.y * 64;
    const int noc = min(64, g.oc - oc_base);
    const int wwords = K * K * W * cw;   // packed words per filter

    // Stage the 64 filters: word widx of filter o goes to
    // lds[((widx / 2) * 64 + o) * 2 + widx % 2]; missing filters are zero.
    // The block's filters are one contiguous run of 64 * wwords words, read
    // with consecutive threads on consecutive words.
    {
        const uint32_t* src = wts + (int64_t)oc_base * wwords;
        const int total = noc * wwords;
        for (int e = threadIdx.x; e < 64 * wwords; e += kBlock) {
            const int o = e / wwords, widx = e - o * wwords;
            const uint32_t v = e < total ? src[e] : 0u;
            lds[((widx >> 1) * 64 + o) * 2 + (widx & 1)] = v;
        }
    }
    __syncthreads();

    const uint2* lw = reinterpret_cast<const uint2*>(lds) + lane;
    gchar* abytes = (gchar*)(act);
    const bool oc_ok = lane < noc;
    // Persistent waves: wave w of the grid takes groups w, w + nw, w + 2 nw..
    // (neighbouring groups, which share input rows, run at the same time).
    const uint32_t nw = gridDim.x * kWavesPerBlock;
    for (uint32_t grp = blockIdx.x * kWavesPerBlock + wave;
         grp < (uint32_t)g.total_groups; grp += nw) {
        const uint32_t rowi = g.div_gpr.div(grp);
        const int gx = (int)(grp - rowi * (uint32_t)g.gpr);
        const uint32_t img = g.div_oh.div(rowi);
        const int oy = (int)(rowi - img * (uint32_t)g.oh);
        const int ox0 = gx * P;
        const int ix0 = ox0 * S - g.pw;
        const bool full = noc == 64 && ox0 + P <= g.ow;
        if (ix0 >= 0 && ix0 + NI <= g.w)
            group_body<A, W, BIP, K, S, P, CW, false>(
                abytes, out, lw, g, img, oy, ox0, oc_base, lane, oc_ok, full);
        else
            group_body<A, W, BIP, K, S, P, CW, true>(
                abytes, out, lw, g, img, oy, ox0, oc_base, lane, oc_ok, full);
    }
}

using KernelFn = void (*)(const uint32_t*, const uint32_t*, int32_t*,
                         FastArgs);

// Kernel for (A, wbits, bipolar, kernel size, stride, group pixels, words
// per plane); the word count is a compile-time constant when a
// specialisation for it exists and a run-time argument otherwise.  Defined
// for A = 1..4 by the compile units of conv_fast_inst.hip.
template <int A>
KernelFn pick_w(int w, bool b, int k, int s, int p, int cw);
template <> KernelFn pick_w<1>(int w, bool b, int k, int s, int p, int cw);
template <> KernelFn pick_w<2>(int w, bool b, int k, int s, int p, int cw);
template <> KernelFn pick_w<3>(int w, bool b, int k, int s, int p, int cw);
template <> KernelFn pick_w<4>(int w, bool b, int k, int s, int p, int cw);

}  // namespace fast
}  // namespace bs
