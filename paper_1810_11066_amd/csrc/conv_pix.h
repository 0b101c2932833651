// Pixels-on-lanes bitserial conv kernel template; instantiated in
// conv_pix.hip.
//
// Mapping.  Lane l of a wave owns one output pixel of a 64-pixel group
// (consecutive output pixels in NHWC order).  The work of a layer is the
// sequence of units (group, quad of 4 output channels), group-major; each
// wave takes one contiguous run of units, so a wave visits at most a few
// groups and, inside a group, a contiguous range of output channels.  The
// host sizes the runs so that the whole grid is resident at once and every
// CU holds the same number of waves (no second round, no straggler CUs).
//
// Per group, each lane loads the packed words of its K x K input patch
// (vector loads; consecutive lanes read consecutive pixels), zeroes the taps
// in the padding, and keeps the patch in VGPRs for all the channels of its
// run.  When the whole patch does not fit (wide layers), it is taken one tap
// block at a time -- a filter row, or a single tap -- with tap blocks as the
// outer loop and partial sums added into the LDS output tile.  Filter words
// are the same for every lane, so they are read with scalar loads (a layer's
// filters are small and stay in the scalar cache) and used as the SGPR
// operand of v_and_b32.
//
// Inner loop: per (tap, plane pair, word) one v_and_b32 (SGPR x VGPR) and one
// accumulating v_bcnt_u32_b32 into one of 2 (A+W-1) per-shift accumulators
// (split by tap parity so consecutive popcounts are independent); the
// shift-add (and bipolar correction, whose patch popcount sum is computed
// once per group) runs once per output.
//
// Filter words stream through two SGPR slices of at most kSliceWords words
// each: the slice for step s+1 is requested before step s computes, and the
// wait for it sits explicitly before step s+1 (scalar loads return out of
// order, so only a full lgkmcnt(0) wait is exact).
//
// Occupancy.  The hardware reserves more SGPRs per wave than the compiler's
// count: measured on gfx950, 8 waves fit on a SIMD up to 80 SGPRs, 7 up to
// 96 and 6 above.  The kernel is therefore compiled for at most 80 SGPRs
// (the slice bound keeps the channel loop within that; what does not fit is
// spilled to VGPR lanes in the per-group code), and the host's occupancy
// query, which counts the way the compiler does, is then exact.
#pragma once

#include "bs_internal.h"

namespace bs {
namespace pix {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;
constexpr int kSliceWords = 24;     // filter words per SGPR slice

struct PixArgs {
    int32_t h, w, oh, ow, ph, pw;
    int32_t oc;            // output channels, a multiple of 4
    int32_t npix;          // n * oh * ow
    int32_t quads;         // oc / 4
    int32_t units;         // ceil(npix / 64) * quads, < 2^31
    int32_t per_wave;      // units per wave (the last waves may get fewer)
    FastDiv div_ow, div_oh, div_quads;
};

__device__ __forceinline__ void bcnt_acc(uint32_t& acc, uint32_t x) {
    asm("v_bcnt_u32_b32 %0, %1, %0" : "+v"(acc) : "v"(x));
}
__device__ __forceinline__ void bcnt_first(uint32_t& acc, uint32_t x) {
    asm("v_bcnt_u32_b32 %0, %1, 0" : "=v"(acc) : "v"(x));
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

// Static plan of a specialisation.
//
// Patch: TB taps of the K x K window are held in VGPRs at a time -- all of
// them when they fit in kMaxPatchWords, else one filter row, else one tap --
// so there are NTB = K*K / TB tap blocks.
//
// Filter stream: a filter (OHWI) is K*K*W*CW contiguous words and
// consecutive filters are adjacent.  Within a tap block a channel's words are
// TB*W*CW contiguous words.  They are consumed in SGPR slices of at most
// kSliceWords: OCB = 2 whole filters when two fit (single tap block only),
// else one channel and TS taps per slice (NP = TB / TS slices).
template <int A, int W, int K, int CW>
struct Plan {
    static constexpr int kMaxPatchWords = 72;
    static constexpr int KK = K * K;
    static constexpr int TB = KK * A * CW <= kMaxPatchWords ? KK
                            : K * A * CW <= kMaxPatchWords ? K : 1;
    static constexpr int NTB = KK / TB;
    static constexpr int FW = KK * W * CW;              // words per filter
    static constexpr int BW = TB * W * CW;              // per tap block
    static constexpr int OCB = NTB == 1 && BW * 2 <= kSliceWords ? 2 : 1;
    static constexpr int TS =                           // taps per slice
        BW <= kSliceWords ? TB
        : (TB % 3 == 0 && 3 * W * CW <= kSliceWords) ? 3 : 1;
    static constexpr int NP = TB / TS;                  // slices per block
    static constexpr int SW = OCB * TS * W * CW;        // words per slice
    static constexpr int STEPS = 4 / OCB * NP;          // slices per quad
    static constexpr bool kFits = TS * W * CW <= kSliceWords &&
                                  TB * A * CW <= kMaxPatchWords;
    static_assert(OCB == 1 || NP == 1, "a slice is whole filters or part of one");
    static_assert(STEPS % 2 == 0, "slice buffers alternate within a quad");
};

template <int SW>
struct Slice {
    uint32_t w[SW];
};

template <int SW>
__device__ __forceinline__ void load_slice(Slice<SW>& s, gu32* src) {
#pragma unroll
    for (int k = 0; k < SW; ++k) s.w[k] = src[k];
}

// Output tile staging.  With pixels on lanes, the NHWC output of one output
// channel is 4 bytes per lane at a stride of oc * 4 bytes -- one memory
// request per lane.  Results are therefore collected per wave in LDS as a
// 64-pixel x kChunk-channel tile and written back with each lane storing 16
// contiguous bytes (nch / 4 lanes per pixel).
constexpr int kChunk = 16;                 // output channels per LDS tile
constexpr int kTileStride = kChunk + 1;    // words per pixel row (padded)
constexpr int kTileWords = 64 * kTileStride;

__device__ __forceinline__ void flush_tile(
    const uint32_t* __restrict__ tile, int32_t* __restrict__ out,
    int pix0, int npix, int oc_total, int oc_base, int nch, int lane) {
    // nch in {4, 8, 12, 16}: lpp = nch / 4 lanes per pixel, lpp rounds of
    // 64 (pixel, quad) entries.  e / lpp for e < 256 is (e * m) >> 16 with
    // m = ceil(2^16 / lpp): the error e (m lpp - 2^16) / (lpp 2^16) stays
    // below 1/lpp - frac(e / lpp) for every such e.
    const int lpp = nch >> 2;
    const uint32_t m = lpp == 1 ? 65536u : lpp == 2 ? 32768u
                     : lpp == 3 ? 21846u : 16384u;
    for (int r = 0; r < lpp; ++r) {
        const uint32_t e = (uint32_t)(r * 64 + lane);
        const int px = (int)((e * m) >> 16);
        const int q = (int)e - px * lpp;
        if (pix0 + px < npix) {
            const uint32_t* t = tile + px * kTileStride + 4 * q;
            *reinterpret_cast<uint4*>(
                out + (int64_t)(pix0 + px) * oc_total + oc_base + 4 * q) =
                make_uint4(t[0], t[1], t[2], t[3]);
        }
    }
}

// One quad of output channels over tap block tb: 4 / OCB batches of OCB
// channels, NP slices each.  `src` points at the quad's first channel's words
// of this tap block; batch b, slice p reads src + b*OCB*FW + p*TS*W*CW.
// Slice buffer f[s & 1] holds step s; on entry f[0] holds (or is receiving)
// step 0, and on exit f[0] is receiving the next quad's first slice (at
// src + 4*FW) when `prefetch` is set.  `patch` holds the block's TB taps.
template <int A, int W, bool BIP, int K, int CW>
__device__ __forceinline__ void compute_quad(
    const uint32_t (&patch)[Plan<A, W, K, CW>::TB][A][CW], uint32_t sa,
    gu32* src, bool prefetch, Slice<Plan<A, W, K, CW>::SW> (&f)[2],
    uint32_t (&val)[4]) {
    using Pl = Plan<A, W, K, CW>;
    constexpr int NS = A + W - 1;
    constexpr int OCB = Pl::OCB, TS = Pl::TS, NP = Pl::NP, SW = Pl::SW;
    constexpr int FW = Pl::FW, TSW = TS * W * CW;
#pragma unroll
    for (int b = 0; b < 4 / OCB; ++b) {
        uint32_t acc[2][OCB][NS];
        bool fresh[2][OCB][NS];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int o = 0; o < OCB; ++o)
#pragma unroll
                for (int s = 0; s < NS; ++s) fresh[h][o][s] = true;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int st = b * NP + p;
            wait_scalar_loads();
            if (st + 1 < Pl::STEPS) {
                const int nb = (st + 1) / NP, np = (st + 1) % NP;
                load_slice<SW>(f[(st + 1) & 1],
                               src + nb * OCB * FW + np * TSW);
            } else if (prefetch) {
                load_slice<SW>(f[0], src + 4 * FW);
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int tt = 0; tt < TS; ++tt)
#pragma unroll
                for (int c = 0; c < CW; ++c)
#pragma unroll
                    for (int j = 0; j < W; ++j)
#pragma unroll
                        for (int i = 0; i < A; ++i)
#pragma unroll
                            for (int o = 0; o < OCB; ++o) {
                                const int t = p * TS + tt;
                                const int h = (t * CW + c) & 1;
                                const uint32_t x =
                                    patch[t][i][c] &
                                    f[st & 1].w[((o * TS + tt) * W + j) * CW + c];
                                if (fresh[h][o][i + j]) {
                                    bcnt_first(acc[h][o][i + j], x);
                                    fresh[h][o][i + j] = false;
                                } else {
                                    bcnt_acc(acc[h][o][i + j], x);
                                }
                            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int o = 0; o < OCB; ++o) {
            uint32_t v = 0;
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const uint32_t a0 = fresh[0][o][s] ? 0u : acc[0][o][s];
                const uint32_t a1 = fresh[1][o][s] ? 0u : acc[1][o][s];
                v += (a0 + a1) << s;
            }
            // bipolar weight value 2w - (2^W - 1): 2*sum - (2^W - 1)*sum(a)
            if (BIP) v = 2u * v - (uint32_t)((1 << W) - 1) * sa;
            val[b * OCB + o] = v;
        }
    }
}

// Loads the lane's input words for taps [t0, t0 + TB) of the window (zero
// for taps in the padding) and, for bipolar weights, their popcount sum
// sum_i 2^i popcount(a_i).
template <int A, bool BIP, int K, int S, int CW, int TB>
__device__ __forceinline__ uint32_t load_patch(
    uint32_t (&patch)[TB][A][CW], const uint32_t* __restrict__ act,
    const PixArgs& g, uint32_t img, int oy, int ox, int t0) {
    constexpr int PW = A * CW;           // words per packed input pixel
#pragma unroll
    for (int tt = 0; tt < TB; ++tt) {
        const int t = t0 + tt;
        const int r = t / K, s = t - r * K;
        const int iy = oy * S - g.ph + r;
        const int ix = ox * S - g.pw + s;
        const bool in = (unsigned)iy < (unsigned)g.h &&
                        (unsigned)ix < (unsigned)g.w;
        // 32-bit word offsets: the host keeps the activations below 2^31
        // words; a padded tap reads pixel 0 and is masked below
        const uint32_t pix =
            in ? ((uint32_t)img * (uint32_t)g.h + (uint32_t)iy) *
                         (uint32_t)g.w + (uint32_t)ix
               : 0u;
        const uint32_t* src = act + (size_t)(pix * (uint32_t)PW);
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
        // the load is unconditional (a padded tap reads pixel 0) and its
        // value masked, so the loads stay straight-line code
        const uint32_t keep = in ? 0xFFFFFFFFu : 0u;
#pragma unroll
        for (int i = 0; i < A; ++i)
#pragma unroll
            for (int c = 0; c < CW; ++c)
                patch[tt][i][c] = wv[i * CW + c] & keep;
    }
    uint32_t sa = 0;
    if (BIP) {
#pragma unroll
        for (int tt = 0; tt < TB; ++tt)
#pragma unroll
            for (int i = 0; i < A; ++i)
#pragma unroll
                for (int c = 0; c < CW; ++c)
                    sa += (uint32_t)__builtin_popcount(patch[tt][i][c]) << i;
    }
    return sa;
}

// A, W: bit-widths; BIP: bipolar weights; K: square kernel size; S: stride;
// CW: words per bit-plane.
template <int A, int W, bool BIP, int K, int S, int CW>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_num_sgpr(80)))
void conv_pix_kernel(
    const uint32_t* __restrict__ act, const uint32_t* __restrict__ wts,
    int32_t* __restrict__ out, PixArgs g) {
    using Pl = Plan<A, W, K, CW>;
    constexpr int FW = Pl::FW, TB = Pl::TB, NTB = Pl::NTB;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6)));
    // units [u, u_end) of this wave; per_wave * waves < 2^31 (host)
    int u = wave * g.per_wave;
    const int u_end = min(u + g.per_wave, g.units);

    extern __shared__ uint32_t lds[];
    uint32_t* tile = lds + (threadIdx.x >> 6) * kTileWords;
    gu32* gw = (gu32*)(wts);

    while (u < u_end) {
        const int grp = (int)g.div_quads.div((uint32_t)u);
        const int q0 = u - grp * g.quads;
        const int q1 = min(g.quads, q0 + (u_end - u));
        const int pix0 = grp * 64;

        // this lane's output pixel (the last pixel stands in past the end)
        const int p = pix0 + lane;
        const uint32_t pc = (uint32_t)(p < g.npix ? p : g.npix - 1);
        const uint32_t rowi = g.div_ow.div(pc);
        const int ox = (int)(pc - rowi * (uint32_t)g.ow);
        const uint32_t img = g.div_oh.div(rowi);
        const int oy = (int)(rowi - img * (uint32_t)g.oh);

        uint32_t patch[TB][A][CW];
        if constexpr (NTB == 1) {
            // whole patch: one pass over the segment's quads, the slice
            // pipeline running across tile flushes
            const uint32_t sa =
                load_patch<A, BIP, K, S, CW, TB>(patch, act, g, img, oy, ox, 0);
            gu32* src = gw + (size_t)(4 * q0) * FW;
            Slice<Pl::SW> f[2];
            load_slice<Pl::SW>(f[0], src);
            const int nq = q1 - q0;
            int chunk_base = 4 * q0;   // first channel held in the tile
            int held = 0;              // quads held in the tile
            for (int qi = 0; qi < nq; ++qi) {
                uint32_t val[4];
                compute_quad<A, W, BIP, K, CW>(patch, sa,
                                               src + (size_t)qi * 4 * FW,
                                               qi + 1 < nq, f, val);
#pragma unroll
                for (int o = 0; o < 4; ++o)
                    tile[lane * kTileStride + held * 4 + o] = val[o];
                ++held;
                if (held == kChunk / 4 || qi + 1 == nq) {
                    wave_lds_sync();
                    flush_tile(tile, out, pix0, g.npix, g.oc, chunk_base,
                               held * 4, lane);
                    wave_lds_sync();
                    chunk_base += held * 4;
                    held = 0;
                }
            }
        } else {
            // tap blocks outermost, per tile chunk of up to kChunk channels;
            // partial sums of later blocks are added in the tile
            for (int sub = q0; sub < q1; sub += kChunk / 4) {
                const int nq = min(kChunk / 4, q1 - sub);
                for (int tb = 0; tb < NTB; ++tb) {
                    const uint32_t sa = load_patch<A, BIP, K, S, CW, TB>(
                        patch, act, g, img, oy, ox, tb * TB);
                    gu32* src = gw + (size_t)(4 * sub) * FW + tb * Pl::BW;
                    Slice<Pl::SW> f[2];
                    load_slice<Pl::SW>(f[0], src);
                    for (int qi = 0; qi < nq; ++qi) {
                        uint32_t val[4];
                        compute_quad<A, W, BIP, K, CW>(
                            patch, sa, src + (size_t)qi * 4 * FW, qi + 1 < nq,
                            f, val);
                        // only this lane touches its tile row until the flush
                        uint32_t* t = tile + lane * kTileStride + qi * 4;
                        if (tb == 0) {
#pragma unroll
                            for (int o = 0; o < 4; ++o) t[o] = val[o];
                        } else {
#pragma unroll
                            for (int o = 0; o < 4; ++o) t[o] += val[o];
                        }
                    }
                }
                wave_lds_sync();
                flush_tile(tile, out, pix0, g.npix, g.oc, 4 * sub, nq * 4,
                           lane);
                wave_lds_sync();
            }
        }
        u += q1 - q0;
    }
}

using PixKernelFn = void (*)(const uint32_t*, const uint32_t*, int32_t*,
                             PixArgs);

// Kernel for a supported (A, W, bipolar, K, S, CW) or nullptr; also reports
// the output channels per filter slice (ocb), taps per slice (ts) and taps
// per tap block (tb).
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb,
                 int* ts, int* tb);

}  // namespace pix
}  // namespace bs
