// int8 matrix-core convolution: a labelled comparison baseline, not the
// bitserial method (declared in include/int8_mfma.h; built as its own
// library, libint8mfma.so).
//
// Implicit GEMM on the MFMA units: M = output pixels, N = output channels,
// K = taps x input channels.  One unit of work is 32 output pixels x 64
// output channels; a wave computes it as 2 x 4 tiles of 16 x 16 with
// v_mfma_i32_16x16x64_i8, one 64-channel slice of one tap per instruction.
//
// Operands.  For a 16 x 16 x 64 product lane l supplies, for row (or column)
// l % 16, the 16 bytes of lane group l / 16.  The filters are the A operand
// (rows: output channels) and the pixels the B operand (columns): a filter
// fragment is the 16 bytes of an output channel's OHWI row at channels
// 16 (l / 16) .. + 16 of the slice, a pixel fragment one 16-byte load of the
// pixel's NHWC input row at the same channels (a tap in the padding loads
// at an offset past the buffer and reads zeros).  A and B take the same
// (lane group, byte) -> k assignment, so the product sums matching channels
// whatever order the instruction gives k.  The 16 x 16 result leaves lane l
// holding rows 4 (l / 16) .. + 3 of column l % 16: four consecutive output
// channels of one pixel, stored as one 16-byte piece of its NHWC row.
//
// Filters are staged once per persistent workgroup in LDS as B fragments,
// [tap][slice][16-channel tile][lane][16 bytes]: each lane reads its 16
// bytes of a fragment at consecutive addresses (one ds_read_b128, no bank
// conflicts), and every wave of the workgroup reuses them for all its units.
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdio.h>

#include "int8_mfma.h"

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int64_t kMaxBytes = (int64_t)kOutOfRange - 65536;
constexpr int kMaxLds = 64 * 1024;

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

thread_local char g_err[256];

int fail(int st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

// Division by a fixed divisor d >= 1 for dividends below 2^31, by one
// multiply-high, an add and a shift (the round-up method of Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994):
// l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1,
// n / d = (mulhi(n, m) + n) >> l.
struct Div {
    uint32_t m;
    int32_t l;
};

Div make_div(int32_t d) {
    int l = 0;
    while ((1ll << l) < d) ++l;
    const uint64_t m =
        ((uint64_t)1 << 32) * (((uint64_t)1 << l) - (uint64_t)d) / (uint64_t)d + 1;
    return Div{(uint32_t)m, l};
}

__host__ __device__ inline int32_t div(int32_t n, Div d) {
    const uint32_t t =
        (uint32_t)(((uint64_t)(uint32_t)n * (uint64_t)d.m) >> 32);
    return (int32_t)((t + (uint32_t)n) >> d.l);
}

struct Args {
    int32_t h, w, c, oc, stride, pad, oh, ow;
    int32_t npix;     // n * oh * ow
    int32_t units;    // ceil(npix / 32) * (oc / 64)
    int32_t kc;       // c / 64
    int32_t act_bytes, out_bytes;
    int32_t tiles;    // staged kernel: ceil(npix / kTilePx)
    int32_t fbytes;   // filter bytes (oc * kh * kw * c)
    Div by_ow, by_oh;
};

// Staged kernel: a workgroup takes tiles of kTilePx consecutive output
// pixels (32 per wave); the whole input rows their windows touch are copied
// into LDS once per tile, and every tap's pixel fragments are read from
// there.
constexpr int kTilePx = 32 * kWaves;
constexpr int kMaxPieces = 8;   // 16-byte pieces per thread: 32 KiB rows

// The flat NHWC input pixels [lo, hi) of the whole input rows that tile
// `tile` reads: from the first output pixel's top window row to the last
// one's bottom window row, both clamped into the image.  Every in-range tap
// of every pixel of the tile lies inside.
__host__ __device__ inline void tile_rows(const Args& g, int k, int tile,
                                          int32_t* lo, int32_t* hi) {
    const int p0 = tile * kTilePx;
    const int p1 = (p0 + kTilePx < g.npix ? p0 + kTilePx : g.npix) - 1;
    const int r0 = div(p0, g.by_ow), r1 = div(p1, g.by_ow);
    const int img0 = div(r0, g.by_oh), img1 = div(r1, g.by_oh);
    int ylo = (r0 - img0 * g.oh) * g.stride - g.pad;
    int yhi = (r1 - img1 * g.oh) * g.stride - g.pad + k - 1;
    ylo = ylo < 0 ? 0 : (ylo > g.h - 1 ? g.h - 1 : ylo);
    yhi = yhi < 0 ? 0 : (yhi > g.h - 1 ? g.h - 1 : yhi);
    *lo = (img0 * g.h + ylo) * g.w;
    *hi = (img1 * g.h + yhi + 1) * g.w;
}

__device__ __forceinline__ Rsrc make_rsrc(const void* p, int32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0,
                                             bytes, 0x00020000);
}

// Filters into LDS as B fragments: element e = (fragment, lane), fragment
// (tap, slice, tile) -> 16 bytes of filter row (o, tap) at channel
// slice * 64 + 16 (lane / 16), o = tile * 16 + lane % 16.
template <int KK>
__device__ __forceinline__ void stage_filters(uint4* frag, const int8_t* wts,
                                              const Args& g) {
    const int nt_all = g.oc / 16;
    const int nfrag = KK * g.kc * nt_all;
    for (int e = threadIdx.x; e < nfrag * 64; e += kBlock) {
        const int f = e >> 6, l = e & 63;
        const int t = f % nt_all, ts = f / nt_all;
        const int sl = ts % g.kc, tap = ts / g.kc;
        const int o = t * 16 + (l & 15);
        frag[e] = *reinterpret_cast<const uint4*>(
            wts + ((size_t)o * KK + tap) * g.c + sl * 64 + 16 * (l >> 4));
    }
    __syncthreads();
}

// Where this lane's two pixels (one per 16-pixel half of a unit's tile) read
// their windows.  The last pixel stands in for pixels past the end: its
// loads stay in the tensor and its stores are dropped.
struct Pix {
    int iy0[2], ix0[2];
    uint32_t base[2];
};

__device__ __forceinline__ Pix pixel_geometry(const Args& g, int tile,
                                              int lane) {
    Pix q;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        int p = tile * 32 + 16 * m + (lane & 15);
        p = p < g.npix ? p : g.npix - 1;
        const int row = div(p, g.by_ow), ox = p - row * g.ow;
        const int img = div(row, g.by_oh), oy = row - img * g.oh;
        q.iy0[m] = oy * g.stride - g.pad;
        q.ix0[m] = ox * g.stride - g.pad;
        q.base[m] = ((uint32_t)(img * g.h + q.iy0[m]) * (uint32_t)g.w +
                     (uint32_t)q.ix0[m]) * (uint32_t)g.c +
                    16u * (uint32_t)(lane >> 4);
    }
    return q;
}

// The A fragments (pixels) of one tap and one 64-channel slice; a tap in the
// padding loads at an offset past the buffer, which reads zeros.
template <int K>
__device__ __forceinline__ void load_pixels(const Args& g, Rsrc ra,
                                            const Pix& q, int tap, int sl,
                                            v4i (&dst)[2]) {
    const int r = tap / K, s = tap - r * K;
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const bool in = (unsigned)(q.iy0[m] + r) < (unsigned)g.h &&
                        (unsigned)(q.ix0[m] + s) < (unsigned)g.w;
        const uint32_t off =
            in ? q.base[m] + (uint32_t)r * (uint32_t)g.w * (uint32_t)g.c +
                     (uint32_t)s * (uint32_t)g.c + 64u * (uint32_t)sl
               : kOutOfRange;
        dst[m] = __builtin_bit_cast(
            v4i, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0, 0));
    }
}

// 2 x 4 tiles of 16 x 16: the pixels of one tap against the four
// 16-channel filter tiles of the unit's 64-channel block.
template <int KK>
__device__ __forceinline__ void mfma_tap(const uint4* frag, const Args& g,
                                         int tap, int sl, int cb, int lane,
                                         const v4i (&a)[2], v4i (&acc)[2][4]) {
    const int nt_all = g.oc / 16;
    const uint4* fb =
        frag + ((size_t)((tap * g.kc + sl) * nt_all + cb * 4)) * 64 + lane;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const v4i b = __builtin_bit_cast(v4i, fb[t * 64]);
        acc[0][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, a[0], acc[0][t],
                                                         0, 0, 0);
        acc[1][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(b, a[1], acc[1][t],
                                                         0, 0, 0);
    }
}

// lane l holds channels 4 (l / 16) .. + 3 of each 16-channel tile for pixel
// l % 16 of each half: one 16-byte piece of the pixel's NHWC row
__device__ __forceinline__ void store_unit(const Args& g, Rsrc ro, int tile,
                                           int cb, int lane,
                                           const v4i (&acc)[2][4]) {
#pragma unroll
    for (int m = 0; m < 2; ++m) {
        const int p = tile * 32 + 16 * m + (lane & 15);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int o = cb * 64 + t * 16 + 4 * (lane >> 4);
            const uint32_t off =
                p < g.npix ? ((uint32_t)p * (uint32_t)g.oc + (uint32_t)o) * 4u
                           : kOutOfRange;
            __builtin_amdgcn_raw_buffer_store_b128(
                __builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned,
                                   acc[m][t]),
                ro, off, 0, 0);
        }
    }
}

// 1x1 windows: one tap per slice, loads then products per slice.
__global__ __launch_bounds__(kBlock) void conv_i8_mfma_1x1_kernel(
    const int8_t* __restrict__ act, const int8_t* __restrict__ wts,
    int32_t* __restrict__ out, Args g) {
    extern __shared__ uint4 frag[];
    stage_filters<1>(frag, wts, g);
    const Rsrc ra = make_rsrc(act, g.act_bytes);
    const Rsrc ro = make_rsrc(out, g.out_bytes);
    const int lane = threadIdx.x & 63, ncb = g.oc / 64;
    const int wave = __builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kWaves + (threadIdx.x >> 6)));
    const int nwaves = gridDim.x * kWaves;
    for (int u = wave; u < g.units; u += nwaves) {
        const int tile = u / ncb, cb = u - tile * ncb;
        const Pix q = pixel_geometry(g, tile, lane);
        v4i acc[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = v4i{0, 0, 0, 0};
        for (int sl = 0; sl < g.kc; ++sl) {
            v4i a[2];
            load_pixels<1>(g, ra, q, 0, sl, a);
            mfma_tap<1>(frag, g, 0, sl, cb, lane, a, acc);
        }
        store_unit(g, ro, tile, cb, lane, acc);
    }
}

// 3x3 windows, software-pipelined: the pixel fragments of the step two
// taps ahead load while the current tap's products run, from a ring of
// three slots.  Nine taps fill the ring a whole number of times, so every
// step's slot is a compile-time index; the lookahead runs across slices and
// into the wave's next unit, whose loads are then in flight while this
// unit's results are stored.
__global__ __launch_bounds__(kBlock) void conv_i8_mfma_3x3_kernel(
    const int8_t* __restrict__ act, const int8_t* __restrict__ wts,
    int32_t* __restrict__ out, Args g) {
    constexpr int K = 3, KK = 9, kAhead = 2, kRing = 3;
    static_assert(KK % kRing == 0 && kAhead < kRing, "ring");
    extern __shared__ uint4 frag[];
    stage_filters<KK>(frag, wts, g);
    const Rsrc ra = make_rsrc(act, g.act_bytes);
    const Rsrc ro = make_rsrc(out, g.out_bytes);
    const int lane = threadIdx.x & 63, ncb = g.oc / 64;
    const int wave = __builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kWaves + (threadIdx.x >> 6)));
    const int nwaves = gridDim.x * kWaves;
    int u = wave;
    if (u >= g.units) return;   // wave-uniform, after the last barrier
    int tile = u / ncb, cb = u - tile * ncb;
    Pix cur = pixel_geometry(g, tile, lane);
    v4i ring[kRing][2];
#pragma unroll
    for (int j = 0; j < kAhead; ++j) load_pixels<K>(g, ra, cur, j, 0, ring[j]);
    for (;;) {
        const int un = u + nwaves;
        const bool has_next = un < g.units;
        const int tile_n = un / ncb, cb_n = un - tile_n * ncb;
        const Pix nxt = pixel_geometry(g, has_next ? tile_n : tile, lane);
        v4i acc[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = v4i{0, 0, 0, 0};
        for (int sl = 0; sl < g.kc; ++sl) {
#pragma unroll
            for (int tap = 0; tap < KK; ++tap) {
                // keep each step's loads where they are issued: the
                // scheduler would otherwise sink them next to their use
                __builtin_amdgcn_sched_barrier(0);
                const int ta = tap + kAhead;
                if (ta < KK)
                    load_pixels<K>(g, ra, cur, ta, sl, ring[ta % kRing]);
                else if (sl + 1 < g.kc)
                    load_pixels<K>(g, ra, cur, ta - KK, sl + 1,
                                   ring[ta % kRing]);
                else if (has_next)
                    load_pixels<K>(g, ra, nxt, ta - KK, 0, ring[ta % kRing]);
                mfma_tap<KK>(frag, g, tap, sl, cb, lane, ring[tap % kRing],
                             acc);
            }
        }
        store_unit(g, ro, tile, cb, lane, acc);
        if (!has_next) break;
        u = un;
        tile = tile_n;
        cb = cb_n;
        cur = nxt;
    }
}

// Input rows through LDS.  Per tile: the rows are fetched into registers
// (kPieces 16-byte pieces per thread) while the previous tile computes, then
// written to LDS between two barriers; a tap's pixel fragment is one
// ds_read_b128 from the rows (or from a 64-byte zero block for a tap in the
// padding).  A wave computes its 32 pixels against every 64-channel filter
// block in turn.
template <int K, int kPieces, int KC>
__global__ __launch_bounds__(kBlock) void conv_i8_staged_kernel(
    const int8_t* __restrict__ act, const int8_t* __restrict__ wts,
    int32_t* __restrict__ out, Args g) {
    constexpr int KK = K * K;
    extern __shared__ uint4 frag[];
    uint4* const zero = frag + g.fbytes / 16;
    uint4* const rows = zero + 4;
    if (threadIdx.x < 4) zero[threadIdx.x] = uint4{0u, 0u, 0u, 0u};
    stage_filters<KK>(frag, wts, g);
    const Rsrc ra = make_rsrc(act, g.act_bytes);
    const Rsrc ro = make_rsrc(out, g.out_bytes);
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int ncb = g.oc / 64, cw = g.c / 16;
    uint4 piece[kPieces];
    auto fetch = [&](int32_t lo, int32_t hi) {
        const int n = (hi - lo) * cw;
        const uint32_t base = (uint32_t)lo * (uint32_t)g.c;
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            const int j = tid + k * kBlock;
            if (j < n)
                piece[k] = __builtin_bit_cast(
                    uint4, __builtin_amdgcn_raw_buffer_load_b128(
                               ra, base + 16u * (uint32_t)j, 0, 0));
        }
    };
    auto put = [&](int32_t lo, int32_t hi) {
        const int n = (hi - lo) * cw;
#pragma unroll
        for (int k = 0; k < kPieces; ++k) {
            const int j = tid + k * kBlock;
            if (j < n) rows[j] = piece[k];
        }
    };
    int tile = blockIdx.x;   // the grid has at most g.tiles workgroups
    int32_t lo, hi;
    tile_rows(g, K, tile, &lo, &hi);
    fetch(lo, hi);
    put(lo, hi);
    __syncthreads();
    for (;;) {
        const int next = tile + (int)gridDim.x;   // block-uniform
        int32_t nlo = 0, nhi = 0;
        if (next < g.tiles) {
            tile_rows(g, K, next, &nlo, &nhi);
            fetch(nlo, nhi);
        }
        int q0[2], iy0[2], ix0[2], pix[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            pix[m] = tile * kTilePx + wv * 32 + 16 * m + (lane & 15);
            // a pixel past the end reads the last pixel's window; its
            // results are not stored
            const int p = pix[m] < g.npix ? pix[m] : g.npix - 1;
            const int row = div(p, g.by_ow), ox = p - row * g.ow;
            const int img = div(row, g.by_oh), oy = row - img * g.oh;
            iy0[m] = oy * g.stride - g.pad;
            ix0[m] = ox * g.stride - g.pad;
            q0[m] = (img * g.h + iy0[m]) * g.w + ix0[m] - lo;
        }
        // the pixel fragments (A) and filter fragments (B) of one step
        auto fragments = [&](int tap, int sl, int cb, v4i (&a)[2],
                             v4i (&b)[4]) {
            const int r = tap / K, s = tap - r * K;
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const bool in = (unsigned)(iy0[m] + r) < (unsigned)g.h &&
                                (unsigned)(ix0[m] + s) < (unsigned)g.w;
                const uint4* src = in ? rows + (q0[m] + r * g.w + s) * cw +
                                            sl * 4 + (lane >> 4)
                                      : zero + (lane >> 4);
                a[m] = __builtin_bit_cast(v4i, *src);
            }
            const uint4* fb =
                frag + ((size_t)((tap * g.kc + sl) * (g.oc / 16) + cb * 4)) *
                           64 + lane;
#pragma unroll
            for (int t = 0; t < 4; ++t) b[t] = __builtin_bit_cast(v4i, fb[t * 64]);
        };
        auto products = [&](const v4i (&a)[2], const v4i (&b)[4],
                            v4i (&acc)[2][4]) {
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int m = 0; m < 2; ++m)
                    acc[m][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                        b[t], a[m], acc[m][t], 0, 0, 0);
        };
        auto compute = [&](int cb, v4i (&acc)[2][4]) {
#pragma unroll
            for (int m = 0; m < 2; ++m)
#pragma unroll
                for (int t = 0; t < 4; ++t) acc[m][t] = v4i{0, 0, 0, 0};
            if constexpr (KC > 0) {
                // every step unrolled, the next step's fragments read from
                // LDS while this step's products run
                constexpr int kSteps = KC * KK;
                v4i a[2][2], b[2][4];
                fragments(0, 0, cb, a[0], b[0]);
#pragma unroll
                for (int j = 0; j < kSteps; ++j) {
                    if (j + 1 < kSteps)
                        fragments((j + 1) % KK, (j + 1) / KK, cb,
                                  a[(j + 1) & 1], b[(j + 1) & 1]);
                    products(a[j & 1], b[j & 1], acc);
                    // keep the reads a step ahead of their products
                    __builtin_amdgcn_sched_barrier(0);
                }
            } else {
                for (int sl = 0; sl < g.kc; ++sl) {
#pragma unroll
                    for (int tap = 0; tap < KK; ++tap) {
                        v4i a[2], b[4];
                        fragments(tap, sl, cb, a, b);
                        products(a, b, acc);
                    }
                }
            }
        };
        auto store = [&](int cb, const v4i (&acc)[2][4]) {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int o = cb * 64 + t * 16 + 4 * (lane >> 4);
                    const uint32_t off =
                        pix[m] < g.npix
                            ? ((uint32_t)pix[m] * (uint32_t)g.oc +
                               (uint32_t)o) * 4u
                            : kOutOfRange;
                    __builtin_amdgcn_raw_buffer_store_b128(
                        __builtin_bit_cast(
                            __attribute__((ext_vector_type(4))) unsigned,
                            acc[m][t]),
                        ro, off, 0, 0);
                }
            }
        };
        v4i acc[2][4];
        for (int cb = 0; cb + 1 < ncb; ++cb) {
            compute(cb, acc);
            store(cb, acc);
        }
        compute(ncb - 1, acc);
        if (next >= g.tiles) {
            store(ncb - 1, acc);
            break;
        }
        // The last results are stored after the next rows are in LDS:
        // loads and stores retire in issue order, so waiting for the
        // prefetched rows would otherwise wait for those stores too.
        __syncthreads();   // every wave is done reading this tile's rows
        put(nlo, nhi);
        __syncthreads();
        store(ncb - 1, acc);
        tile = next;
        lo = nlo;
    }
}

// pieces rounded up to an even count; KC slices unrolled (0: a loop)
template <int K, int KC>
const void* staged_for_kc(int pieces) {
    switch ((pieces + 1) / 2) {
        case 1: return (const void*)conv_i8_staged_kernel<K, 2, KC>;
        case 2: return (const void*)conv_i8_staged_kernel<K, 4, KC>;
        case 3: return (const void*)conv_i8_staged_kernel<K, 6, KC>;
        default: return (const void*)conv_i8_staged_kernel<K, 8, KC>;
    }
}

// (3x3 filters within 64 KiB have c = oc = 64: one slice)
const void* staged_for(int k, int pieces, int kc) {
    if (k == 3) return kc == 1 ? staged_for_kc<3, 1>(pieces)
                               : staged_for_kc<3, 0>(pieces);
    return kc == 1 ? staged_for_kc<1, 1>(pieces)
         : kc == 2 ? staged_for_kc<1, 2>(pieces)
                   : staged_for_kc<1, 0>(pieces);
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

extern "C" {

const char* i8mfma_last_error(void) { return g_err; }

int i8mfma_conv2d(const i8mfma_conv_params* p, const int8_t* act,
                  const int8_t* wts, int32_t* out, void* stream) {
    if (!p || !act || !wts || !out)
        return fail(I8MFMA_ERR_INVALID_ARG, "NULL argument");
    if (!aligned16(act) || !aligned16(wts) || !aligned16(out))
        return fail(I8MFMA_ERR_INVALID_ARG, "pointers must be 16-byte aligned");
    if (p->n < 1 || p->h < 1 || p->w < 1 || p->c < 1 || p->oc < 1 ||
        p->kh < 1 || p->kw < 1 || p->stride < 1 || p->pad < 0)
        return fail(I8MFMA_ERR_INVALID_ARG, "bad sizes");
    const int64_t eh = (int64_t)p->h + 2 * p->pad - p->kh;
    const int64_t ew = (int64_t)p->w + 2 * p->pad - p->kw;
    if (eh < 0 || ew < 0)
        return fail(I8MFMA_ERR_INVALID_ARG, "kernel larger than padded input");
    const int64_t oh = eh / p->stride + 1, ow = ew / p->stride + 1;
    if (p->kh != p->kw || (p->kh != 1 && p->kh != 3))
        return fail(I8MFMA_ERR_UNSUPPORTED, "kernels 1x1 or 3x3 only");
    if (p->c % 64 != 0 || p->oc % 64 != 0)
        return fail(I8MFMA_ERR_UNSUPPORTED, "c and oc must be multiples of 64");
    const int64_t wbytes = (int64_t)p->oc * p->kh * p->kw * p->c;
    if (wbytes > kMaxLds)
        return fail(I8MFMA_ERR_UNSUPPORTED, "filters exceed 64 KiB of LDS");
    const int64_t act_bytes = (int64_t)p->n * p->h * p->w * p->c;
    const int64_t npix = (int64_t)p->n * oh * ow;
    const int64_t out_bytes = npix * p->oc * 4;
    if (act_bytes > kMaxBytes || out_bytes > kMaxBytes)
        return fail(I8MFMA_ERR_UNSUPPORTED, "tensors of 2 GiB or more");
    Args g;
    g.h = p->h; g.w = p->w; g.c = p->c; g.oc = p->oc;
    g.stride = p->stride; g.pad = p->pad;
    g.oh = (int32_t)oh; g.ow = (int32_t)ow;
    g.npix = (int32_t)npix;
    g.units = (int32_t)(((npix + 31) / 32) * (p->oc / 64));
    g.kc = p->c / 64;
    g.act_bytes = (int32_t)act_bytes;
    g.out_bytes = (int32_t)out_bytes;
    g.tiles = (int32_t)((npix + kTilePx - 1) / kTilePx);
    g.by_ow = make_div(g.ow);
    g.by_oh = make_div(g.oh);
    g.fbytes = (int32_t)wbytes;
    int dev = 0, cus = 256, max_lds = 160 * 1024;
    if (hipGetDevice(&dev) == hipSuccess) {
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                    dev);
        (void)hipDeviceGetAttribute(
            &max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    }
    // the staged kernel when the largest tile's input rows fit its pieces
    // and LDS; else the direct kernel, which reads every tap from memory
    int64_t rows_bytes = 0;
    for (int t = 0; t < g.tiles; ++t) {
        int32_t lo, hi;
        tile_rows(g, p->kh, t, &lo, &hi);
        const int64_t b = (int64_t)(hi - lo) * p->c;
        if (b > rows_bytes) rows_bytes = b;
    }
    const int pieces = (int)((rows_bytes + 16 * kBlock - 1) / (16 * kBlock));
    const int64_t staged_lds = wbytes + 64 + rows_bytes;
    const bool staged = pieces <= kMaxPieces && staged_lds <= max_lds;
    const void* fn;
    size_t lds;
    int64_t need;
    if (staged) {
        fn = staged_for(p->kh, pieces, g.kc);
        lds = (size_t)staged_lds;
        need = g.tiles;
    } else {
        fn = p->kh == 3 ? (const void*)conv_i8_mfma_3x3_kernel
                        : (const void*)conv_i8_mfma_1x1_kernel;
        lds = (size_t)wbytes;
        need = (g.units + kWaves - 1) / kWaves;
    }
    int per_cu = 1;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock,
                                                     lds) != hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    // persistent workgroups: one round on every CU, no more than the work
    int64_t blocks = (int64_t)cus * per_cu;
    if (blocks > need) blocks = need;
    void* args[] = {&act, &wts, &out, &g};
    const hipError_t e = hipLaunchKernel(fn, dim3((uint32_t)blocks),
                                         dim3(kBlock), args, lds,
                                         (hipStream_t)stream);
    if (e != hipSuccess)
        return fail(I8MFMA_ERR_HIP, "launch: %s", hipGetErrorString(e));
    g_err[0] = '\0';
    return I8MFMA_OK;
}

}  // extern "C"
