// Pixels-on-lanes bitserial conv kernel template; instantiated in
// conv_pix.hip.
//
// Mapping.  Lane l of a wave owns one output pixel of a 64-pixel group
// (consecutive output pixels in NHWC order).  The work of a layer is the
// sequence of units (group, quad of 4 output channels), group-major; each
// wave takes one contiguous run of units, so a wave visits at most a few
// groups and, inside a group, a contiguous range of output channels.  The
// host sizes the runs so that the whole grid is resident at once and every
// CU holds the same number of waves (no second round, no straggler CUs);
// store-bound 1x1 layers instead run one 16-channel tile chunk per wave.
// Blocks take their work in XCD-major order.
//
// Per group, each lane loads the packed words of its K x K input patch
// (raw buffer loads, consecutive lanes reading consecutive pixels; a tap in
// the padding reads past the buffer and gets zeros) and keeps the patch in
// VGPRs for all the channels of its run.  When the whole patch does not
// fit (wide layers), it is taken one tap block at a time -- a filter row, or
// a single tap -- with tap blocks as the outer loop and partial sums added
// into the LDS output tile.  Filter words are the same for every lane, so
// they are read with scalar loads and used as the SGPR operand of
// v_and_b32 (the scalar cache holds a small layer's filters; for the large
// ones, up to the 4 MB of a 4096 x 4096 dense layer, the kernel time was
// measured not to depend on it).
//
// Inner loop: per (tap, plane pair, word) one v_and_b32 (SGPR x VGPR) and one
// accumulating v_bcnt_u32_b32 into one of A+W-1 per-shift accumulators (5-7
// resident waves hide the dependence of consecutive popcounts on one
// accumulator; a second set split by tap parity cost registers and
// epilogue adds); the shift-add (and bipolar correction, whose patch
// popcount sum is computed once per group) runs once per output.
//
// Filter words stream through two SGPR slices of at most kSliceWords words
// each: the slice for step s+1 is requested before step s computes, and the
// wait for it sits explicitly before step s+1 (scalar loads return out of
// order, so only a full lgkmcnt(0) wait is exact).
//
// Occupancy.  The hardware reserves more SGPRs per wave than the compiler's
// count: measured on gfx950, 8 waves fit on a SIMD up to 80 SGPRs, 7 up to
// 96 and 6 above.  VGPRs come from 512 per lane in granules of 8 (64 -> 8
// waves, 72 -> 7, 80 -> 6, 88-96 -> 5, up to 128 -> 4), as the occupancy
// query counts them.  The kernel is compiled for at most 96 SGPRs
// (the slice bound keeps the channel loop within that; what does not fit is
// spilled to VGPR lanes in the per-group code), and the host caps the
// occupancy query, which counts the way the compiler does, at
// kWavesPerSimd = 7 waves per SIMD.  At 80 SGPRs (8 waves) the spills of the
// per-group code cost more than the eighth wave gains.
#pragma once

#include "bs_internal.h"

namespace bs {
namespace pix {

constexpr int kBlock = 256;
constexpr int kWavesPerBlock = kBlock / 64;
constexpr int kWavesPerSimd = 7;    // resident at up to 96 SGPRs per wave
constexpr int kSliceWords = 24;     // filter words per SGPR slice

// Operand encodings of a specialisation: E = 3 * (activation encoding) +
// (weight encoding), each kUnipolar, kBipolar or kSigned.
//
// Every encoding is affine in the plain binary value u of a code (the sum of
// its planes' +-2^j, the top plane of signed data negative): value =
// alpha u + beta, (alpha, beta) = (1, 0) unipolar or signed, (2, -(2^B - 1))
// bipolar.  Over the in-range taps of a window
//   sum value(a) value(w) = aa aw S + aa bw SA + ba aw SW + ba bw N,
// S = sum_{i,j} +-2^(i+j) popcount(a_i AND w_j) (the inner loop, plane pairs
// of opposite sign in separate accumulators), SA and SW the plane-weighted
// popcounts of the window's activation and (in-range) filter words, N the
// number of in-range channel values.  SA and N are per lane; SW depends on
// the lane's in-range taps and the channel: the scalar unit counts the bits
// of each tap's filter words from the SGPR slice, and one v_dot2_u32_u16 per
// pair of taps weighs them by the lane's in-range flags.
//
// +-1 data on both sides (the XNOR case) takes the paper's form instead:
// per in-range tap the product is c - 2 popcount(a XOR w), so the inner loop
// counts the bits of (a XOR w) AND keep, keep being the lane's all-ones /
// all-zeros in-range mask of the tap -- one v_bitop3_b32 and one v_bcnt per
// word, the cost of the unipolar loop -- and the epilogue is N - 2 D.
template <int E>
struct Enc {
    static constexpr int AE = E / 3, WE = E % 3;
    static constexpr bool kSignedPairs = AE == kSigned || WE == kSigned;
    static constexpr bool kXnor = AE == kBipolar && WE == kBipolar;
    // the sign of plane pair (i, j) of an A x W product
    static constexpr bool neg(int i, int j, int A, int W) {
        return (AE == kSigned && i == A - 1) != (WE == kSigned && j == W - 1);
    }
};

struct PixArgs {
    int32_t h, w, oh, ow, ph, pw;
    int32_t oc;            // output channels, a multiple of 4
    int32_t npix;          // n * oh * ow
    int32_t quads;         // oc / 4
    int32_t unit_quads;    // quads per unit: 1 (int32 out), 2 (packed out)
    int32_t group_units;   // units per 64-pixel group: ceil(quads / unit_quads)
    int32_t units;         // ceil(npix / 64) * group_units, < 2^31
    int32_t per_wave;      // units per wave (the last waves may get fewer)
    // requantized output (packed kernels only)
    float out_scale, out_qmax;
    int32_t out_bits;      // 1..8
    int32_t out_words;     // ceil(oc / 32): words per plane of a pixel
    FastDiv div_ow, div_oh, div_units;
    int32_t c;             // input channels (+-1 activations only)
    int32_t act_bytes;     // size of the activations, bytes: the packed
                           // words, the uint8 codes (kSrcCodes) or the
                           // float32 values (kSrcFloat)
    int32_t out_bytes;     // size of the int32 output, bytes (0: packed out)
    // activations staged in LDS (SRC != kSrcPacked): the most input pixels
    // any block's region holds (its LDS size)
    int32_t region_pixels;
    // float32 activations (kSrcFloat): the quantizer's scale and top code
    float in_scale, in_qmax;
    // paired 1x1 conv (DUAL kernels; its packed filters [oc][W][CW] are the
    // kernel's wts1 argument): its output (int32 [npix][oc], or packed codes
    // with out1_scale), and the int32 output's size in bytes (0 for packed
    // output)
    int32_t* out1;
    float out1_scale;
    int32_t out1_bytes;
};

// Where a specialisation's activations come from:
//   kSrcPacked  bit-packed words [n][h][w][A][CW] in HBM (bs_pack output);
//   kSrcCodes   uint8 codes [n][h][w][C], C = 32 CW: each block bit-packs the
//               input rows its outputs read into LDS first.  The packed
//               activations never reach HBM: the separate pack launch and
//               its round trip are gone, at the price of packing each
//               block's halo rows again.
//   kSrcFloat   float32 activations [n][h][w][C] (1x1 windows): as
//               kSrcCodes, each value quantized on the way (unipolar, scale
//               and qmax in PixArgs) before it is packed.
constexpr int kSrcPacked = 0, kSrcCodes = 1, kSrcFloat = 2;

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
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Static plan of a specialisation.
//
// Reduction blocks: the K*K taps x CW words per plane of a window are split
// into NB = (K*K / TB) * (CW / CB) blocks of TB taps x CB words.  A block's
// patch (TB*A*CB words per lane) is what sits in VGPRs: the whole window when
// it fits in kMaxPatchWords, else one filter row, else one tap, else (very
// wide 1x1 layers, dense) one tap and CB words of each plane.  With NB > 1
// blocks are the outer loop and their partial sums are added in the LDS
// tile; small block patches are double-buffered (the next block's words load
// while the current block computes).
//
// Filter stream: a filter (OHWI) is FW = K*K*W*CW contiguous words and
// consecutive filters are adjacent.  Within a block, a channel's words are
// TB taps x W planes x CB words (contiguous when CB == CW).  They are consumed
// in SGPR slices of at most kSliceWords: OCB = 2 whole filters when two fit
// (NB == 1 only), else one channel and TS taps per slice (NP = TB / TS
// slices per block).
template <int A, int W, int K, int CW>
struct Plan {
    static constexpr int kMaxPatchWords = 72;
    static constexpr int KK = K * K;
    // one tap's filter words must fit a slice, else taps go one at a time
    // and the words of each plane are split as well
    static constexpr bool kWideTap = W * CW > kSliceWords;
    static constexpr int TB = kWideTap ? 1
                            : KK * A * CW <= kMaxPatchWords ? KK
                            : K * A * CW <= kMaxPatchWords ? K : 1;
    // words per plane in a block: all of them, or the largest power of two
    // whose patch and one-tap slice stay small
    static constexpr int cb_split() {
        int cb = CW;
        while (cb > 1 && (A * cb > 32 || W * cb > kSliceWords)) cb >>= 1;
        return cb;
    }
    static constexpr int CB =
        !kWideTap && TB * A * CW <= kMaxPatchWords ? CW : cb_split();
    static constexpr int NCB = CW / CB;                 // word chunks
    static constexpr int NB = KK / TB * NCB;            // reduction blocks
    static constexpr int PB = TB * A * CB;              // patch words / block
    static constexpr bool DBUF = NB > 1 && 2 * PB <= 48;
    static constexpr int FW = KK * W * CW;              // words per filter
    static constexpr int BW = TB * W * CB;              // per block, channel
    static constexpr int OCB = NB == 1 && BW * 2 <= kSliceWords ? 2 : 1;
    static constexpr int TS =                           // taps per slice
        BW <= kSliceWords ? TB
        : (TB % 3 == 0 && 3 * W * CB <= kSliceWords) ? 3 : 1;
    static constexpr int NP = TB / TS;                  // slices per block
    static constexpr int NPAIR = (TS + 1) / 2;          // tap pairs / slice
    static constexpr int SW = OCB * TS * W * CB;        // words per slice
    static constexpr int STEPS = 4 / OCB * NP;          // slices per quad
    static constexpr bool kFits = TS * W * CB <= kSliceWords &&
                                  PB <= kMaxPatchWords && CW % CB == 0;
    static_assert(OCB == 1 || NP == 1, "a slice is whole filters or part of one");
    static_assert(STEPS % 2 == 0, "slice buffers alternate within a quad");
    static_assert(CB == CW || TB == 1, "word chunks only with one tap");
};

// Per-lane tap data of a reduction block (+-1 activations only): the
// in-range mask of each tap (XNOR) or the in-range flags of tap pairs of
// each slice as u16 pairs (unipolar filters).
template <int A, int W, int K, int CW>
struct TapInfo {
    using Pl = Plan<A, W, K, CW>;
    uint32_t keep[Pl::TB];
    uint32_t pairs[Pl::NP][Pl::NPAIR];
};

// (a XOR w) AND keep in one v_bitop3_b32.  The function is symmetric in a
// and w, so with the mask as the middle operand its truth table (bits 3 and
// 6: a != w with keep set) reads the same whichever of the outer operands
// supplies the high index bit.
__device__ __forceinline__ uint32_t xor_keep(uint32_t a, uint32_t keep,
                                             uint32_t w) {
    return __builtin_amdgcn_bitop3_b32(a, keep, w, 0x48);
}

// Bits set in two consecutive filter words of an SGPR slice (uniform: one
// s_bcnt1_i32_b64 on the aligned register pair).
__device__ __forceinline__ uint32_t popcount2(uint32_t lo, uint32_t hi) {
    return (uint32_t)__builtin_popcountll((uint64_t)hi << 32 | lo);
}

template <int SW>
struct Slice {
    uint32_t w[SW];
};

// One slice: OCB channels x TS taps x W planes x CB words, gathered from the
// OHWI filters at channel stride FW, tap stride W*CW and plane stride CW
// (compile-time offsets, so contiguous runs merge into wide scalar loads).
template <int A, int W, int K, int CW>
__device__ __forceinline__ void load_slice(
    Slice<Plan<A, W, K, CW>::SW>& s, gu32* src) {
    using Pl = Plan<A, W, K, CW>;
#pragma unroll
    for (int o = 0; o < Pl::OCB; ++o)
#pragma unroll
        for (int tt = 0; tt < Pl::TS; ++tt)
#pragma unroll
            for (int j = 0; j < W; ++j)
#pragma unroll
                for (int c = 0; c < Pl::CB; ++c)
                    s.w[((o * Pl::TS + tt) * W + j) * Pl::CB + c] =
                        src[o * Pl::FW + (tt * W + j) * CW + c];
}

// Requantized, bit-packed output of one pixel: the codes of 8 consecutive
// output channels (2 quads) gathered bit by bit into one byte per plane
// (channel c of the byte -> bit c, LSB first; bytes of a word are
// little-endian, so byte k of word w holds channels 32 w + 8 k ..), stored
// as bytes -- 8-channel pieces let a wave's run end on any second quad
// without sharing a store with its neighbour.
struct PackedOut {
    uint32_t codes[2];   // the codes of each quad, one byte per channel

    __device__ __forceinline__ void clear() { codes[0] = codes[1] = 0; }
    // codes of the 4 channels of quad `half` (0 or 1) of the byte: the int32
    // results are exact in float32 (far below 2^24) and never NaN, so the
    // clamp of the quantizer is one v_med3
    __device__ __forceinline__ void add4(const uint32_t (&val)[4],
                                         const PixArgs& g, int half) {
        add4(val, g.out_scale, g, half);
    }
    __device__ __forceinline__ void add4(const uint32_t (&val)[4],
                                         float scale, const PixArgs& g,
                                         int half) {
        uint32_t bytes = 0;
#pragma unroll
        for (int o = 0; o < 4; ++o) {
            const float r =
                __builtin_rintf((float)(int32_t)val[o] * scale);
            bytes |= (uint32_t)__builtin_amdgcn_fmed3f(r, 0.0f, g.out_qmax)
                     << (8 * o);
        }
        // (selects, not an indexed store: a runtime index into a register
        // array would go through scratch memory)
        codes[0] = half ? codes[0] : bytes;
        codes[1] = half ? bytes : codes[1];
    }
    // the byte of channels [8 k8, 8 k8 + 8) of pixel pix, every plane; the
    // byte of the last channels also zeroes the rest of its word (the tail
    // bits of the packed layout)
    __device__ __forceinline__ void store(int32_t* __restrict__ out,
                                          const PixArgs& g, int pix, int k8) {
        uint8_t* dst = reinterpret_cast<uint8_t*>(out) +
                       (size_t)pix * (uint32_t)(4 * g.out_bits * g.out_words) +
                       (uint32_t)k8;
        const int last = (g.oc + 7) / 8 - 1;
        const int pad = k8 == last ? 3 - (k8 & 3) : 0;
#pragma unroll
        for (int b = 0; b < 8; ++b)
            if (b < g.out_bits) {
                uint8_t* d = dst + (size_t)b * (uint32_t)(4 * g.out_words);
                d[0] = (uint8_t)(nibble_of(codes[0], b) |
                                 nibble_of(codes[1], b) << 4);
                for (int z = 1; z <= pad; ++z) d[z] = 0;
            }
    }
};

// Output tile staging.  With pixels on lanes, the NHWC output of one output
// channel is 4 bytes per lane at a stride of oc * 4 bytes -- one memory
// request per lane.  Results are therefore collected per wave in LDS as a
// 64-pixel x kChunk-channel tile and written back with each lane storing 16
// contiguous bytes (nch / 4 lanes per pixel).
constexpr int kChunk = 16;                 // output channels per LDS tile
constexpr int kTileStride = kChunk + 1;    // words per pixel row (padded)
constexpr int kTileWords = 64 * kTileStride;

// Buffer resources.  Activations are read and int32 results written
// through raw buffer instructions: an access at an offset past the buffer's
// size reads zeros or is dropped.  A tap in the padding therefore only needs
// the offset kOutOfRange -- no address arithmetic per tap, no masking of the
// loaded words -- and so does a store for a pixel past the end, which keeps
// the stores of a flush unconditional (a fixed number of memory operations
// after a prefetch, which the compiler's wait counts rely on).  The host
// keeps both tensors below kMaxBufferBytes, so that kOutOfRange plus any
// instruction offset stays out of range.  The scalar offset of every store
// is the constant 0: a wide buffer store whose scalar offset is a register
// has been seen to lose its data when the next instruction overwrote the
// data registers, a wait the compiler only inserts for the constant form.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int64_t kMaxBufferBytes = (int64_t)kOutOfRange - 65536;
constexpr int kRsrcWord3 = 0x00020000;   // 32-bit data format (gfx9 family)

__device__ __forceinline__ Rsrc make_rsrc(const void* p, int32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0,
                                             bytes, kRsrcWord3);
}

// Cache policy of the int32 result stores (the buffer instruction's aux
// bits): 0, the default write-back through the XCD's L2, or kStoreAgent
// (sc1), agent scope, which writes through that L2.  Measured per launch on
// ResNet-18 layers 6-12 and the 128- and 256-channel layers of the encodings
// workloads (at least 4 words per plane, A >= 2), agent-scope stores are
// 1-2.7 us shorter: less is left dirty for the write-back that ends each
// launch.  For the 64-channel layers (2 words per plane) and the one-bit
// activation kernels they are neutral or up to 4.7 us longer, and there the
// default stays.
constexpr int kStoreAgent = 16;
template <int A, int CW>
constexpr int out_store_policy() {
    return CW >= 4 && A >= 2 ? kStoreAgent : 0;
}

// Where a lane's 16-byte pieces of a tile flush go.  A flush moves the
// tile's 64 pixels x kChunk channels in kFlushRounds rounds: in round r lane
// l stores quad l % kFlushRounds of pixel r * 64 / kFlushRounds +
// l / kFlushRounds (kChunk / 4 lanes per pixel, so a round writes runs of
// 4 kChunk contiguous bytes).  Round r's byte offset is that of round 0 plus
// (64 / kFlushRounds) r oc 4; the lane's part is recomputed per flush rather
// than held across the channel loop, where registers are scarce.  Only the
// group holding the last pixel needs per-round checks.
constexpr int kFlushRounds = kChunk / 4;
constexpr int kFlushPixels = 64 / kFlushRounds;    // pixels per round

struct FlushMap {
    int pix0, npix, oc;    // uniform

    __device__ __forceinline__ void init(int pix0_, int npix_, int oc_) {
        pix0 = pix0_;
        npix = npix_;
        oc = oc_;
    }
};

// Writes channels [oc_base, oc_base + nch) of the group's 64 pixels from the
// wave's tile (nch a multiple of 4 up to kChunk: the lanes of quads below
// nch / 4 take part, the others store out of range).  SERIAL: one round's
// data in registers at a time, for flushes that run while a large input
// patch is held.  CPOL: the stores' cache policy (out_store_policy).
template <bool SERIAL, int CPOL>
__device__ __forceinline__ void flush_tile(const uint32_t* __restrict__ tile,
                                           Rsrc out, const FlushMap& fm,
                                           int oc_base, int nch, int lane) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const uint32_t rstep = 4u * kFlushPixels * (uint32_t)fm.oc;  // per round
    const int q = lane % kFlushRounds, pr = lane / kFlushRounds;
    const bool qin = q < (nch >> 2);
    const uint32_t o0 = ((uint32_t)(fm.pix0 + pr) * (uint32_t)fm.oc +
                         (uint32_t)(oc_base + 4 * q)) * 4u;
    const uint32_t* t = tile + pr * kTileStride + 4 * q;
#pragma unroll
    for (int r = 0; r < kFlushRounds; ++r) {
        const uint32_t* e = t + kFlushPixels * r * kTileStride;
        const u32x4 v = {e[0], e[1], e[2], e[3]};
        const bool in = qin && fm.pix0 + kFlushPixels * r + pr < fm.npix;
        __builtin_amdgcn_raw_buffer_store_b128(
            v, out, in ? o0 + (uint32_t)r * rstep : kOutOfRange, 0, CPOL);
        if constexpr (SERIAL) __builtin_amdgcn_sched_barrier(0);
    }
}

// One output channel of the paired 1x1 conv: Eq. 2 over the centre tap's
// words pc (A planes x CW words) and the channel's filter words f (W planes
// x CW words, uniform), plus the bipolar-filter correction with lc1, the
// plane-weighted popcount of pc.
template <int A, int W, int E, int CW>
__device__ __forceinline__ uint32_t centre_1x1(const uint32_t (&pc)[A][CW],
                                               const uint32_t* f,
                                               uint32_t lc1) {
    constexpr int NS = A + W - 1;
    uint32_t acc[NS];
    bool fresh[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) fresh[s] = true;
#pragma unroll
    for (int c = 0; c < CW; ++c)
#pragma unroll
        for (int j = 0; j < W; ++j)
#pragma unroll
            for (int i = 0; i < A; ++i) {
                const uint32_t x = pc[i][c] & f[j * CW + c];
                if (fresh[i + j]) {
                    bcnt_first(acc[i + j], x);
                    fresh[i + j] = false;
                } else {
                    bcnt_acc(acc[i + j], x);
                }
            }
    uint32_t v = 0;
#pragma unroll
    for (int s = 0; s < NS; ++s) v += (fresh[s] ? 0u : acc[s]) << s;
    if constexpr (E % 3 == kBipolar) v = 2u * v - (uint32_t)((1 << W) - 1) * lc1;
    return v;
}

// One quad of output channels over one reduction block: 4 / OCB batches of
// OCB channels, NP slices each.  `src` points at the quad's first channel's
// words of this block; batch b, slice p starts at src + b*OCB*FW + p*TS*W*CW.
// Slice buffer f[s & 1] holds step s; on entry f[0] holds (or is receiving)
// step 0, and on exit f[0] is receiving the slice at `next` (the next quad's
// or block's first slice; callers with nothing left pass any valid slice
// address, so the load never needs a branch or a null check).  `patch` holds
// the block's TB taps x A planes x CB words.
template <int A, int W, int E, int K, int CW>
__device__ __forceinline__ void compute_quad(
    const uint32_t (&patch)[Plan<A, W, K, CW>::TB][A][Plan<A, W, K, CW>::CB],
    uint32_t lc, const TapInfo<A, W, K, CW>& tv, gu32* src, gu32* next,
    Slice<Plan<A, W, K, CW>::SW> (&f)[2], uint32_t (&val)[4]) {
    using Pl = Plan<A, W, K, CW>;
    using En = Enc<E>;
    static_assert(En::AE != kBipolar || (A == 1 && W == 1),
                  "+-1 activations are specialised for A == W == 1");
    constexpr int NS = A + W - 1;
    constexpr int NA = En::kSignedPairs ? 2 * NS : NS;   // accumulators
    constexpr int OCB = Pl::OCB, TS = Pl::TS, NP = Pl::NP, CB = Pl::CB;
    constexpr int FW = Pl::FW, TSW = TS * W * CW;
#pragma unroll
    for (int b = 0; b < 4 / OCB; ++b) {
        uint32_t acc[OCB][NA];
        bool fresh[OCB][NA];
        uint32_t corr[OCB];   // SW: in-range filter popcounts (bipolar acts)
#pragma unroll
        for (int o = 0; o < OCB; ++o) corr[o] = 0;
#pragma unroll
        for (int o = 0; o < OCB; ++o)
#pragma unroll
            for (int s = 0; s < NA; ++s) fresh[o][s] = true;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
            const int st = b * NP + p;
            wait_scalar_loads();
            if (st + 1 < Pl::STEPS) {
                const int nb = (st + 1) / NP, np = (st + 1) % NP;
                load_slice<A, W, K, CW>(f[(st + 1) & 1],
                                        src + nb * OCB * FW + np * TSW);
            } else {
                load_slice<A, W, K, CW>(f[0], next);
            }
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (En::AE == kBipolar && !En::kXnor) {
                // W == 1: per tap, the bits of its CB filter words (uniform,
                // on the scalar unit, two words per count); taps 2m and
                // 2m+1 of the slice share one dot2 with the lane's flags
#pragma unroll
                for (int o = 0; o < OCB; ++o)
#pragma unroll
                    for (int m = 0; m < Pl::NPAIR; ++m) {
                        uint32_t cnt[2] = {0, 0};
#pragma unroll
                        for (int e = 0; e < 2; ++e) {
                            if (2 * m + e >= TS) continue;
                            const uint32_t* wt =
                                &f[st & 1].w[(o * TS + 2 * m + e) * CB];
#pragma unroll
                            for (int c = 0; c + 1 < CB; c += 2)
                                cnt[e] += popcount2(wt[c], wt[c + 1]);
                            if (CB & 1)
                                cnt[e] += __builtin_popcount(wt[CB - 1]);
                        }
                        corr[o] = __builtin_amdgcn_udot2(
                            __builtin_bit_cast(u16x2, tv.pairs[p][m]),
                            __builtin_bit_cast(u16x2, cnt[0] | cnt[1] << 16),
                            corr[o], false);
                    }
            }
#pragma unroll
            for (int tt = 0; tt < TS; ++tt)
#pragma unroll
                for (int c = 0; c < CB; ++c)
#pragma unroll
                    for (int j = 0; j < W; ++j)
#pragma unroll
                        for (int i = 0; i < A; ++i)
#pragma unroll
                            for (int o = 0; o < OCB; ++o) {
                                const int t = p * TS + tt;
                                const int s =
                                    i + j + (En::neg(i, j, A, W) ? NS : 0);
                                const uint32_t wv =
                                    f[st & 1].w[((o * TS + tt) * W + j) * CB + c];
                                const uint32_t x =
                                    En::kXnor
                                        ? xor_keep(patch[t][i][c], tv.keep[t], wv)
                                        : patch[t][i][c] & wv;
                                if (fresh[o][s]) {
                                    bcnt_first(acc[o][s], x);
                                    fresh[o][s] = false;
                                } else {
                                    bcnt_acc(acc[o][s], x);
                                }
                            }
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int o = 0; o < OCB; ++o) {
            uint32_t v = 0;
#pragma unroll
            for (int s = 0; s < NA; ++s) {
                const uint32_t a = fresh[o][s] ? 0u : acc[o][s];
                if (s < NS) v += a << s;
                else v -= a << (s - NS);
            }
            if constexpr (En::kXnor) {
                // v counts the in-range disagreements D: N - 2 D
                v = lc - 2u * v;
            } else if constexpr (En::AE == kBipolar) {
                // +-1 activations, unipolar 1-bit filters: 2 S - SW
                v = 2u * v - corr[o];
            } else if constexpr (En::WE == kBipolar) {
                // bipolar weight value 2w - (2^W - 1): 2 S - (2^W - 1) SA
                v = 2u * v - (uint32_t)((1 << W) - 1) * lc;
            }
            val[b * OCB + o] = v;
        }
    }
}

// The lane's input window: byte offset of its top-left input pixel
// (iy0, ix0) -- wrapped modulo 2^32 when that pixel lies in the padding; only
// in-range taps use it, and for those the sum is the true offset -- and the
// window's origin.
struct Window {
    uint32_t base;
    int iy0, ix0;
};

// ---- staged activations ---------------------------------------------------

// Bit-planes 0..A-1 of 32 codes held as bytes in d[0..7] (code 4 m + k in
// byte k of d[m]): bit u of plane word b is bit b of code u.  Per plane and
// dword, the plane's bits are masked (bit b of each byte) and one
// v_dot4_u32_u8 against the byte weights 2^k (or 2^(4+k) for the second
// dword of a pair) adds them, shifted by b, into one byte of 8 codes; four
// such bytes make the word.
template <int A>
__device__ __forceinline__ void pack32_planes(const uint32_t (&d)[8],
                                              uint32_t (&w)[A]) {
#pragma unroll
    for (int b = 0; b < A; ++b) {
        const uint32_t m = 0x01010101u << b;
        uint32_t byte[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            byte[j] = __builtin_amdgcn_udot4(d[2 * j] & m, 0x08040201u, 0u,
                                             false);
            byte[j] = __builtin_amdgcn_udot4(d[2 * j + 1] & m, 0x80402010u,
                                             byte[j], false);
        }
        // byte[j] holds codes 8 j .. 8 j + 7 at bits b .. b + 7
        const uint32_t lo24 = byte[0] | byte[1] << 8 | byte[2] << 16;
        w[b] = (lo24 >> b) | (byte[3] >> b) << 24;
    }
}

// The 32 codes of one staged item (channels 32 t .. 32 t + 31 of one input
// pixel, starting at element e of the NHWC activations) as bytes in d[0..7]
// (code 4 m + k in byte k of d[m]).  Codes: two 16-byte loads.  Float32:
// eight, each value quantized as bs_quantize does (quant_code).  in false
// (a pixel in the padding): the loads fall past the buffer and read zeros,
// which are code 0 either way.
template <int SRC>
__device__ __forceinline__ void load_item(uint32_t (&d)[8], Rsrc src,
                                          uint32_t e, bool in,
                                          const PixArgs& g) {
    if constexpr (SRC == kSrcFloat) {
        const uint32_t off = in ? 4u * e : kOutOfRange;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const float4 f = __builtin_bit_cast(
                float4, __builtin_amdgcn_raw_buffer_load_b128(
                            src, off + 16u * (uint32_t)m, 0, 0));
            d[m] = quant_code<false>(f.x, g.in_scale, g.in_qmax) |
                   quant_code<false>(f.y, g.in_scale, g.in_qmax) << 8 |
                   quant_code<false>(f.z, g.in_scale, g.in_qmax) << 16 |
                   quant_code<false>(f.w, g.in_scale, g.in_qmax) << 24;
        }
    } else {
        const uint32_t off = in ? e : kOutOfRange;
        const uint4 a = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(src, off, 0, 0));
        const uint4 b = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(src, off + 16u, 0, 0));
        d[0] = a.x; d[1] = a.y; d[2] = a.z; d[3] = a.w;
        d[4] = b.x; d[5] = b.y; d[6] = b.z; d[7] = b.w;
    }
}

// Items of one staging pass a thread has in flight before it packs any:
// four 32-byte code loads, or one item's eight float32 loads (32 values, as
// many registers as the four code items).
template <int SRC>
constexpr int stage_items_in_flight() {
    return SRC == kSrcFloat ? 1 : 4;
}

// Input region of a block: the flat NHWC input pixels [lo, hi) that hold
// every in-range tap of the block's output pixels, from the first tap of
// its first output pixel to the last tap of its last one.  The first tap row
// a of the first output row y0 is read by no other output row (the next
// one's taps start S rows lower), and only by the block's pixels at x >= x0,
// so its columns left of x0 S - pw stay out; likewise the last tap row of the
// last output row right of x1 S - pw + K - 1.  The host sizes the LDS with
// the same rule.
struct Region {
    int32_t lo, hi;
};

template <int K, int S>
__device__ __forceinline__ Region block_region(const PixArgs& g, int p_first,
                                               int p_last) {
    const uint32_t r0 = g.div_ow.div((uint32_t)p_first);
    const uint32_t n0 = g.div_oh.div(r0), y0 = r0 - n0 * (uint32_t)g.oh;
    const int x0 = p_first - (int)(r0 * (uint32_t)g.ow);
    const uint32_t r1 = g.div_ow.div((uint32_t)p_last);
    const uint32_t n1 = g.div_oh.div(r1), y1 = r1 - n1 * (uint32_t)g.oh;
    const int x1 = p_last - (int)(r1 * (uint32_t)g.ow);
    // first and last input row of the block's taps, clamped to [0, h] and
    // [-1, h - 1]: with padding above K - 1 an output row can lie wholly in
    // the padding, and its image then contributes no row (row h of image
    // n0 is row 0 of image n0 + 1; row -1 of image n1 ends image n1 - 1)
    const int a = (int)y0 * S - g.ph, b = (int)y1 * S - g.ph + K - 1;
    const int iy_lo = min(max(a, 0), g.h);
    const int iy_hi = max(min(b, g.h - 1), -1);
    Region rg;
    rg.lo = ((int)n0 * g.h + iy_lo) * g.w;
    rg.hi = ((int)n1 * g.h + iy_hi) * g.w + g.w;
    if (a >= 0 && a < g.h) rg.lo += min(max(x0 * S - g.pw, 0), g.w - 1);
    if (b >= 0 && b < g.h)
        rg.hi -= g.w - 1 - max(min(x1 * S - g.pw + K - 1, g.w - 1), 0);
    // an all-padding block (no in-range tap) holds nothing; the host sized
    // the LDS for the largest region, which bounds every block's
    rg.hi = min(max(rg.hi, rg.lo), rg.lo + g.region_pixels);
    return rg;
}

// Fills the block's region in LDS: packed words [pixel - lo][A][CW] of the
// input pixels [lo, hi), then one pixel of zeros (what the taps in the
// padding read).  Each thread packs (pixel, word) items of 32 codes; the
// loads of consecutive threads are consecutive 32-byte pieces of the NHWC
// rows.  A thread issues the loads of U items before it packs any of them,
// so that the fill waits for memory about once rather than once per item.
template <int A, int CW, int SRC>
__device__ __forceinline__ void stage_region(uint32_t* __restrict__ region,
                                             Rsrc src, Region rg,
                                             const PixArgs& g) {
    constexpr int PW = A * CW;                 // words per packed pixel
    constexpr int U = stage_items_in_flight<SRC>();
    // item = 32 codes (one word of every plane of one pixel); items are
    // numbered in memory order, so item i starts at element 32 i of the
    // region
    const int items = (rg.hi - rg.lo) * CW;
    const uint32_t base = (uint32_t)rg.lo * (uint32_t)(32 * CW);
    for (int it0 = threadIdx.x; it0 < items; it0 += U * kBlock) {
        uint32_t d[U][8];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = it0 + u * kBlock;
            if (it < items)
                load_item<SRC>(d[u], src, base + 32u * (uint32_t)it, true, g);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = it0 + u * kBlock;
            if (it < items) {
                const int pl = it / CW, t = it - pl * CW;
                uint32_t w[A];
                pack32_planes<A>(d[u], w);
#pragma unroll
                for (int b = 0; b < A; ++b)
                    region[pl * PW + b * CW + t] = w[b];
            }
        }
    }
    const int zero = (rg.hi - rg.lo) * PW;
    for (int i = threadIdx.x; i < PW; i += kBlock) region[zero + i] = 0;
}

// Strided 1x1 windows read one input pixel per output pixel, S rows and S
// columns apart.  Their region is gathered instead: the input pixels of the
// block's output pixels [q_lo, q_hi), in output order ([q - q_lo][A][CW]
// words), so that the rows and columns no tap reads are neither loaded nor
// packed; an output pixel whose input pixel lies in the padding gets zeros
// (its loads fall past the buffer).  Then the zero pixel, as stage_region.
template <int A, int CW, int S, int SRC>
__device__ __forceinline__ void stage_gather(uint32_t* __restrict__ region,
                                             Rsrc src, const PixArgs& g,
                                             int q_lo, int q_hi) {
    constexpr int PW = A * CW;
    constexpr int U = stage_items_in_flight<SRC>();
    const int items = (q_hi - q_lo) * CW;
    for (int it0 = threadIdx.x; it0 < items; it0 += U * kBlock) {
        uint32_t d[U][8];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = it0 + u * kBlock;
            if (it < items) {
                const int q = q_lo + it / CW, t = it % CW;
                const uint32_t row = g.div_ow.div((uint32_t)q);
                const int x = q - (int)(row * (uint32_t)g.ow);
                const uint32_t img = g.div_oh.div(row);
                const int y = (int)(row - img * (uint32_t)g.oh);
                const int iy = y * S - g.ph, ix = x * S - g.pw;
                const bool in = (unsigned)iy < (unsigned)g.h &&
                                (unsigned)ix < (unsigned)g.w;
                const uint32_t e =
                    ((img * (uint32_t)g.h + (uint32_t)iy) * (uint32_t)g.w +
                     (uint32_t)ix) * (uint32_t)(32 * CW) + 32u * (uint32_t)t;
                load_item<SRC>(d[u], src, e, in, g);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int it = it0 + u * kBlock;
            if (it < items) {
                const int pl = it / CW, t = it % CW;
                uint32_t w[A];
                pack32_planes<A>(d[u], w);
#pragma unroll
                for (int b = 0; b < A; ++b)
                    region[pl * PW + b * CW + t] = w[b];
            }
        }
    }
    const int zero = (q_hi - q_lo) * PW;
    for (int i = threadIdx.x; i < PW; i += kBlock) region[zero + i] = 0;
}

// Loads the lane's words of one reduction block from the staged region: the
// same taps [t0, t0 + TB) and words [c0, c0 + CB) of each plane as
// load_patch, at byte offsets relative to the region (win.base is relative
// to its first pixel; a tap in the padding reads the zero pixel at byte
// offset zero_off).  With TB = K*K and CB = CW: the whole patch.
template <int A, int K, int CW, int TB, int CB>
__device__ __forceinline__ void load_patch_lds(
    uint32_t (&patch)[TB][A][CB], const uint32_t* __restrict__ region,
    const PixArgs& g, const Window& win, uint32_t zero_off, int t0, int c0) {
    constexpr uint32_t PWB = 4 * A * CW;
    const uint32_t rowb = (uint32_t)g.w * PWB;
    const char* base = reinterpret_cast<const char*>(region);
#pragma unroll
    for (int tt = 0; tt < TB; ++tt) {
        const int t = t0 + tt;
        const int r = t / K, s = t - r * K;
        const bool in = (unsigned)(win.iy0 + r) < (unsigned)g.h &&
                        (unsigned)(win.ix0 + s) < (unsigned)g.w;
        const uint32_t off =
            (in ? win.base + (uint32_t)r * rowb + (uint32_t)s * PWB
                : zero_off) + 4u * (uint32_t)c0;
#pragma unroll
        for (int i = 0; i < A; ++i) {
            const char* p = base + off + 4u * (uint32_t)(i * CW);
            if constexpr (CB % 4 == 0) {
#pragma unroll
                for (int k = 0; k < CB; k += 4) {
                    const uint4 x = *reinterpret_cast<const uint4*>(p + 4 * k);
                    patch[tt][i][k] = x.x; patch[tt][i][k + 1] = x.y;
                    patch[tt][i][k + 2] = x.z; patch[tt][i][k + 3] = x.w;
                }
            } else if constexpr (CB % 2 == 0) {
#pragma unroll
                for (int k = 0; k < CB; k += 2) {
                    const uint2 x = *reinterpret_cast<const uint2*>(p + 4 * k);
                    patch[tt][i][k] = x.x; patch[tt][i][k + 1] = x.y;
                }
            } else {
#pragma unroll
                for (int k = 0; k < CB; ++k)
                    patch[tt][i][k] =
                        *reinterpret_cast<const uint32_t*>(p + 4 * k);
            }
        }
    }
}

// Loads the lane's input words of one reduction block: taps [t0, t0 + TB)
// of the window and words [c0, c0 + CB) of each of the A planes (zero for
// taps in the padding: their offset is out of the buffer's range).
template <int A, int K, int CW, int TB, int CB>
__device__ __forceinline__ void load_patch(uint32_t (&patch)[TB][A][CB],
                                           Rsrc act, const PixArgs& g,
                                           const Window& win, int t0, int c0) {
    constexpr uint32_t PWB = 4 * A * CW;     // bytes per packed input pixel
    const uint32_t rowb = (uint32_t)g.w * PWB;
#pragma unroll
    for (int tt = 0; tt < TB; ++tt) {
        const int t = t0 + tt;
        const int r = t / K, s = t - r * K;
        const bool in = (unsigned)(win.iy0 + r) < (unsigned)g.h &&
                        (unsigned)(win.ix0 + s) < (unsigned)g.w;
        const uint32_t off =
            (in ? win.base + (uint32_t)r * rowb + (uint32_t)s * PWB
                : kOutOfRange) + 4u * (uint32_t)c0;
#pragma unroll
        for (int i = 0; i < A; ++i) {
            const uint32_t o = off + 4u * (uint32_t)(i * CW);
            if constexpr (CB % 4 == 0) {
#pragma unroll
                for (int k = 0; k < CB; k += 4) {
                    const auto x = __builtin_amdgcn_raw_buffer_load_b128(
                        act, o + 4u * k, 0, 0);
                    patch[tt][i][k] = x[0]; patch[tt][i][k + 1] = x[1];
                    patch[tt][i][k + 2] = x[2]; patch[tt][i][k + 3] = x[3];
                }
            } else if constexpr (CB % 2 == 0) {
#pragma unroll
                for (int k = 0; k < CB; k += 2) {
                    const auto x = __builtin_amdgcn_raw_buffer_load_b64(
                        act, o + 4u * k, 0, 0);
                    patch[tt][i][k] = x[0]; patch[tt][i][k + 1] = x[1];
                }
            } else {
#pragma unroll
                for (int k = 0; k < CB; ++k)
                    patch[tt][i][k] =
                        __builtin_amdgcn_raw_buffer_load_b32(act, o + 4u * k,
                                                             0, 0);
            }
        }
    }
}

// SA of a block: sum_i +-2^i popcount(a_i) over its words (the top plane of
// signed activations negative).
template <int A, int TB, int CB, bool SGN>
__device__ __forceinline__ uint32_t patch_sum(
    const uint32_t (&patch)[TB][A][CB]) {
    uint32_t sa = 0;
#pragma unroll
    for (int tt = 0; tt < TB; ++tt)
#pragma unroll
        for (int i = 0; i < A; ++i)
#pragma unroll
            for (int c = 0; c < CB; ++c) {
                const uint32_t x = (uint32_t)__builtin_popcount(patch[tt][i][c])
                                   << i;
                sa += SGN && i == A - 1 ? 0u - x : x;
            }
    return sa;
}

// Per-lane constants of reduction block nb (taps t0 = (nb / NCB) TB ..): the
// tap data of +-1 activations (TapInfo), and the lane constant lc the
// epilogue adds: SA for bipolar filters of unipolar or signed activations,
// N (in-range channel values of the block) for +-1 data, 0 otherwise.
template <int A, int W, int E, int K, int S, int CW>
__device__ __forceinline__ uint32_t block_consts(
    const uint32_t (&patch)[Plan<A, W, K, CW>::TB][A][Plan<A, W, K, CW>::CB],
    TapInfo<A, W, K, CW>& tv, const PixArgs& g, int oy, int ox, int nb) {
    using Pl = Plan<A, W, K, CW>;
    using En = Enc<E>;
    if constexpr (En::AE == kBipolar) {
        const int tb = nb / Pl::NCB, cb = nb - tb * Pl::NCB;
        const int t0 = tb * Pl::TB;
        uint32_t nv = 0;
#pragma unroll
        for (int p = 0; p < Pl::NP; ++p)
#pragma unroll
            for (int m = 0; m < Pl::NPAIR; ++m) {
                uint32_t flag[2] = {0, 0};
#pragma unroll
                for (int e = 0; e < 2; ++e) {
                    const int tt = p * Pl::TS + 2 * m + e;
                    if (2 * m + e >= Pl::TS) continue;
                    const int t = t0 + tt;
                    const int r = t / K, q = t - r * K;
                    const int iy = oy * S - g.ph + r, ix = ox * S - g.pw + q;
                    flag[e] = (unsigned)iy < (unsigned)g.h &&
                              (unsigned)ix < (unsigned)g.w;
                    tv.keep[tt] = 0u - flag[e];
                }
                tv.pairs[p][m] = flag[0] | flag[1] << 16;
                nv += flag[0] + flag[1];
            }
        if constexpr (En::kXnor) {
            // channels of the block's words
            const int ch = min(32 * Pl::CB, g.c - 32 * Pl::CB * cb);
            return nv * (uint32_t)ch;
        }
        return 0u;
    } else if constexpr (En::WE == kBipolar) {
        return patch_sum<A, Pl::TB, Pl::CB, En::AE == kSigned>(patch);
    } else {
        return 0u;
    }
}

// Offset of reduction block nb's words inside a filter.
template <int A, int W, int K, int CW>
__device__ __forceinline__ int block_offset(int nb) {
    using Pl = Plan<A, W, K, CW>;
    const int tb = nb / Pl::NCB, cb = nb - tb * Pl::NCB;
    return tb * Pl::TB * W * CW + cb * Pl::CB;
}

// Quads [0, nq) of a tile chunk over reduction block nb: results written to
// (nb == 0) or added to (nb > 0) the lane's tile row.  On exit f[0] is
// receiving `next_block` (the next block's first slice, or any valid slice
// address when there is none).
template <int A, int W, int E, int K, int S, int CW>
__device__ __forceinline__ void run_block(
    const uint32_t (&patch)[Plan<A, W, K, CW>::TB][A][Plan<A, W, K, CW>::CB],
    gu32* src, int nq, int nb, gu32* next_block,
    Slice<Plan<A, W, K, CW>::SW> (&f)[2], uint32_t* row, const PixArgs& g,
    int oy, int ox) {
    using Pl = Plan<A, W, K, CW>;
    TapInfo<A, W, K, CW> tv;
    const uint32_t lc =
        block_consts<A, W, E, K, S, CW>(patch, tv, g, oy, ox, nb);
#pragma unroll 1
    for (int qi = 0; qi < nq; ++qi) {
        uint32_t val[4];
        gu32* q = src + (size_t)qi * 4 * Pl::FW;
        compute_quad<A, W, E, K, CW>(
            patch, lc, tv, q, qi + 1 < nq ? q + 4 * Pl::FW : next_block, f,
            val);
        // only this lane touches its tile row until the flush
        uint32_t* t = row + qi * 4;
        if (nb == 0) {
#pragma unroll
            for (int o = 0; o < 4; ++o) t[o] = val[o];
        } else {
#pragma unroll
            for (int o = 0; o < 4; ++o) t[o] += val[o];
        }
    }
}

// Block index in the order of the work, XCD-major.  The dispatcher deals
// blocks to the 8 XCDs round-robin (block b to XCD b % 8), and each XCD
// has its own L2; numbering the blocks of XCD x consecutively (x * q +
// min(x, r) + b / 8 for q = blocks / 8, r = blocks % 8, a bijection) gives
// each XCD a contiguous range of pixel groups, so the input rows that
// neighbouring groups share (the window's halo) are fetched into one L2.
constexpr int kXcds = 8;

__device__ __forceinline__ int xcd_block() {
    const int b = blockIdx.x, n = gridDim.x;
    const int q = n / kXcds, r = n % kXcds, x = b % kXcds;
    return x * q + min(x, r) + b / kXcds;
}

// One group visit of a wave: units [w0, w1) of a 64-pixel group, i.e.
// quads [q0, q1) of its output channels, and the lane's pixel p = pix0 +
// lane at (oy, ox) with its input window and flush offsets.
struct Visit {
    int w0, w1, q0, q1, pix0, p, ox, oy;
    Window win;
    FlushMap fm;
};

// Patches of at most this many words are requested a visit ahead.
constexpr int kAheadWords = 16;

// Waves per SIMD the compiler must leave room for: kWavesPerSimd (72 VGPRs)
// for the kernels that fit there without spilling -- at most 2 plane pairs
// of unipolar activations (unipolar or bipolar filters), int32 output, and a
// block patch of at most 48 words with its double buffer -- where a register
// or two over 72 would cost a wave and change the launch plan (ResNet-18
// layer 10: 73 VGPRs, 6 waves, 40.1 us; 72 VGPRs, 7 waves, 38.2 us); for the
// others whatever their patch needs.
// Paired kernels (DUAL) follow the same rule (at 96 VGPRs the 72-word-patch
// ones would spill to scratch; they take 4 waves).
template <int A, int W, int E, int K, int CW, bool REQ, bool DUAL>
constexpr int min_waves_per_simd() {
    using Pl = Plan<A, W, K, CW>;
    return !REQ && A * W <= 2 && E / 3 == kUnipolar && E % 3 != kSigned &&
                   Pl::PB * (Pl::DBUF ? 2 : 1) <= 48
               ? kWavesPerSimd
               : 1;
}

// A, W: bit-widths; E: operand encodings (Enc); K: square kernel size;
// S: stride; CW: words per bit-plane; REQ: requantize and bit-pack the output
// (out then holds [npix][out_bits][out_words] uint32 words) instead of
// storing int32; SRC: where the activations come from (kSrcPacked, or
// kSrcCodes / kSrcFloat staged in LDS); DUAL: also the 1x1 conv of
// the same stride whose input pixel is the window's centre tap (pad
// (K-1)/2), over the same output grid and channels, with filters wts1 and
// output g.out1 (whole patches only).  wts1 is a kernel argument, read-only
// and unaliased like wts, so that its uniform loads may be scalar loads.
template <int A, int W, int E, int K, int S, int CW, bool REQ, int SRC,
          bool DUAL>
__global__ __launch_bounds__(kBlock) __attribute__((
    amdgpu_num_sgpr(96),
    amdgpu_waves_per_eu(min_waves_per_simd<A, W, E, K, CW, REQ, DUAL>())))
void conv_pix_kernel(
    const uint32_t* __restrict__ act, const uint32_t* __restrict__ wts,
    const uint32_t* __restrict__ wts1, int32_t* __restrict__ out,
    PixArgs g) {
    using Pl = Plan<A, W, K, CW>;
    constexpr int FW = Pl::FW, NB = Pl::NB;
    constexpr int kCpol = out_store_policy<A, CW>();
    static_assert(SRC == kSrcPacked || !REQ,
                  "staged activations: int32 output");
    static_assert(SRC != kSrcFloat || K == 1,
                  "float32 activations: 1x1 windows");
    static_assert(!DUAL || (NB == 1 && K % 2 == 1 && SRC == kSrcPacked &&
                            (E == 3 * kUnipolar + kUnipolar ||
                             E == 3 * kUnipolar + kBipolar)),
                  "paired 1x1 conv: whole patches, unipolar activations");
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(
        (int)(xcd_block() * kWavesPerBlock + (threadIdx.x >> 6)));
    // units [u, u_end) of this wave; per_wave * waves < 2^31 (host)
    int u = wave * g.per_wave;
    const int u_end = min(u + g.per_wave, g.units);

    extern __shared__ uint32_t lds[];
    uint32_t* tile = lds + (threadIdx.x >> 6) * kTileWords;
    gu32* gw = (gu32*)(wts);
    const Rsrc ract = make_rsrc(act, g.act_bytes);
    const Rsrc rout = make_rsrc(out, g.out_bytes);
    [[maybe_unused]] const Rsrc rout1 = make_rsrc(g.out1, g.out1_bytes);

    // staged activations: the block packs its input region into LDS (after
    // the waves' output tiles) before any wave computes; every wave of the
    // block takes part, also one whose own run is empty.  Strided 1x1
    // windows gather one input pixel per output pixel (stage_gather).
    constexpr bool kGather = SRC != kSrcPacked && K == 1 && S > 1;
    [[maybe_unused]] const uint32_t* region = lds + kWavesPerBlock * kTileWords;
    [[maybe_unused]] int32_t region_lo = 0;
    [[maybe_unused]] uint32_t zero_off = 0;
    if constexpr (SRC != kSrcPacked) {
        const int per_block = kWavesPerBlock * g.per_wave;
        const int ub0 = xcd_block() * per_block;
        if (ub0 >= g.units) return;            // the whole block is idle
        const int ub1 = min(ub0 + per_block, g.units);
        const int p_first = (int)g.div_units.div((uint32_t)ub0) * 64;
        const int p_last = min(
            (int)g.div_units.div((uint32_t)(ub1 - 1)) * 64 + 63, g.npix - 1);
        if constexpr (kGather) {
            // the host sized the LDS for the largest block's pixel count
            const int q_hi = min(p_last + 1, p_first + g.region_pixels);
            stage_gather<A, CW, S, SRC>(lds + kWavesPerBlock * kTileWords,
                                        ract, g, p_first, q_hi);
            region_lo = p_first;
            zero_off = (uint32_t)(q_hi - p_first) * (uint32_t)(4 * A * CW);
        } else {
            const Region rg = block_region<K, S>(g, p_first, p_last);
            stage_region<A, CW, SRC>(lds + kWavesPerBlock * kTileWords, ract,
                                     rg, g);
            region_lo = rg.lo;
            zero_off = (uint32_t)(rg.hi - rg.lo) * (uint32_t)(4 * A * CW);
        }
        __syncthreads();
    }

    // one group visit: the run's units in the current 64-pixel group
    auto visit_at = [&](int u0) {
        Visit v;
        const int grp = (int)g.div_units.div((uint32_t)u0);
        v.w0 = u0 - grp * g.group_units;                     // first unit
        v.w1 = min(g.group_units, v.w0 + (u_end - u0));
        v.q0 = v.w0 * g.unit_quads;
        v.q1 = min(g.quads, v.w1 * g.unit_quads);
        v.pix0 = grp * 64;
        // this lane's output pixel (the last pixel stands in past the end)
        v.p = v.pix0 + lane;
        const uint32_t pc = (uint32_t)(v.p < g.npix ? v.p : g.npix - 1);
        const uint32_t rowi = g.div_ow.div(pc);
        v.ox = (int)(pc - rowi * (uint32_t)g.ow);
        const uint32_t img = g.div_oh.div(rowi);
        v.oy = (int)(rowi - img * (uint32_t)g.oh);
        v.win.iy0 = v.oy * S - g.ph;
        v.win.ix0 = v.ox * S - g.pw;
        if constexpr (kGather)
            v.win.base = (pc - (uint32_t)region_lo) * (uint32_t)(4 * A * CW);
        else
            v.win.base = ((img * (uint32_t)g.h + (uint32_t)v.win.iy0) *
                              (uint32_t)g.w + (uint32_t)v.win.ix0 -
                          (uint32_t)region_lo) *
                         (uint32_t)(4 * A * CW);
        if constexpr (!REQ) v.fm.init(v.pix0, g.npix, g.oc);
        return v;
    };

    if constexpr (NB == 1) {
        // whole patch: one pass over each visit's quads, the slice pipeline
        // running across tile flushes.  With a small patch the next visit's
        // words are requested before this visit's last stores: vmcnt counts
        // loads and stores in order, so a load issued after them would wait
        // for their completion (and the HBM-bound 1x1 layers would stall).
        constexpr bool kAhead = Pl::PB <= kAheadWords && SRC == kSrcPacked;
        // the paired 1x1 conv's filter words of one quad, and the centre tap
        [[maybe_unused]] constexpr int F1 = 4 * W * CW;
        [[maybe_unused]] constexpr int kCentre = K * K / 2;
        [[maybe_unused]] gu32* gw1 = (gu32*)(wts1);
        // flushes run while the patch is held: keep their registers few
        // when the patch is large (all four rounds hoisted cost 4-9 VGPRs)
        constexpr bool kSerialFlush = Pl::PB > 32;
        if (u >= u_end) return;
        Visit v = visit_at(u);
        uint32_t patch[Pl::TB][A][CW];
        if constexpr (SRC != kSrcPacked)
            load_patch_lds<A, K, CW, K * K, CW>(patch, region, g, v.win,
                                                zero_off, 0, 0);
        else
            load_patch<A, K, CW, Pl::TB, CW>(patch, ract, g, v.win, 0, 0);
        if constexpr (kAhead && !REQ) {
            // an empty flush (every store out of range): the loop is then
            // entered, as it is re-entered, with the patch load followed by
            // one flush's stores, so the wait for the patch can leave those
            // in flight
            flush_tile<kSerialFlush, kCpol>(tile, rout, v.fm, 0, 0, lane);
            if constexpr (DUAL)
                flush_tile<kSerialFlush, kCpol>(tile, rout1, v.fm, 0, 0,
                                                lane);
        }
        while (true) {
            if constexpr (kAhead) {
                // take the patch words here, outside the channel loop: the
                // wait for them is then placed here and counts past the
                // stores that followed their load (a first use inside the
                // loop gets a full wait in front of it instead)
#pragma unroll
                for (int t = 0; t < Pl::TB; ++t)
#pragma unroll
                    for (int i = 0; i < A; ++i)
#pragma unroll
                        for (int c = 0; c < CW; ++c)
                            asm volatile("" ::"v"(patch[t][i][c]));
            }
            TapInfo<A, W, K, CW> tv;
            const uint32_t lc =
                block_consts<A, W, E, K, S, CW>(patch, tv, g, v.oy, v.ox, 0);
            // bipolar filters of the paired 1x1 conv: SA of the centre tap
            [[maybe_unused]] uint32_t lc1 = 0;
            if constexpr (DUAL && E % 3 == kBipolar) {
#pragma unroll
                for (int i = 0; i < A; ++i)
#pragma unroll
                    for (int c = 0; c < CW; ++c)
                        lc1 += (uint32_t)__builtin_popcount(
                                   patch[kCentre][i][c]) << i;
            }
            gu32* src = gw + (size_t)(4 * v.q0) * FW;
            Slice<Pl::SW> f[2];
            load_slice<A, W, K, CW>(f[0], src);
            const int nq = v.q1 - v.q0;
            int chunk_base = 4 * v.q0;   // first channel held in the tile
            int held = 0;                // quads held in the tile
            PackedOut po, po1;
            po.clear();
            po1.clear();
            // the paired 1x1 conv's 4 channels of quad qg (its filters by one
            // scalar load), computed after the main conv's results of the
            // tile chunk have been flushed, so only the centre tap and one
            // accumulator set are live
            // channel by channel, each result handed to `put` before the
            // next channel starts (a scheduling barrier keeps the compiler
            // from interleaving the channels' accumulators)
            [[maybe_unused]] auto quad1 = [&](int qg, auto&& put)
                __attribute__((always_inline)) {
                uint32_t f1[F1];
                // scalar loads (uniform index, read-only unaliased filters):
                // a vector load here would wait, through vmcnt, for the tile
                // stores issued just before
                gu32* q1 =
                    gw1 + (size_t)__builtin_amdgcn_readfirstlane(qg) * F1;
#pragma unroll
                for (int k = 0; k < F1; ++k) f1[k] = q1[k];
#pragma unroll
                for (int o = 0; o < 4; ++o) {
                    put(o, centre_1x1<A, W, E, CW>(patch[kCentre],
                                                   f1 + o * W * CW, lc1));
                    __builtin_amdgcn_sched_barrier(0);
                }
            };
            // the tile chunk's stores: the main conv's channels
            // [chunk_base, chunk_base + 4 held), then, for paired kernels,
            // the same channels of the 1x1 conv through the same tile (every
            // flush writes 64-byte pieces of the pixel rows)
            auto flush_chunk = [&]() __attribute__((always_inline)) {
                wave_lds_sync();
                flush_tile<kSerialFlush, kCpol>(tile, rout, v.fm,
                                                chunk_base, held * 4, lane);
                if constexpr (DUAL) {
                    wave_lds_sync();
                    uint32_t* row = tile + lane * kTileStride;
#pragma unroll 1
                    for (int h = 0; h < held; ++h)
                        quad1(chunk_base / 4 + h,
                              [&](int o, uint32_t x)
                                  __attribute__((always_inline)) {
                                      row[h * 4 + o] = x;
                                  });
                    wave_lds_sync();
                    flush_tile<kSerialFlush, kCpol>(tile, rout1, v.fm,
                                                    chunk_base, held * 4,
                                                    lane);
                }
                wave_lds_sync();
                chunk_base += held * 4;
                held = 0;
            };
            auto quad = [&](int qi) __attribute__((always_inline)) {
                uint32_t val[4];
                gu32* q = src + (size_t)qi * 4 * FW;
                compute_quad<A, W, E, K, CW>(
                    patch, lc, tv, q, qi + 1 < nq ? q + 4 * FW : src, f, val);
                if constexpr (REQ) {
                    // a packed byte holds 2 quads; runs start on a byte
                    const int qg = v.q0 + qi;
                    po.add4(val, g, qg & 1);
                    if constexpr (DUAL) {
                        uint32_t val1[4];
                        quad1(qg, [&](int o, uint32_t x)
                                      __attribute__((always_inline)) {
                                          val1[o] = x;
                                      });
                        po1.add4(val1, g.out1_scale, g, qg & 1);
                    }
                    if ((qg & 1) == 1 && qi + 1 < nq) {
                        if (v.p < g.npix) {
                            po.store(out, g, v.p, qg >> 1);
                            if constexpr (DUAL)
                                po1.store(g.out1, g, v.p, qg >> 1);
                        }
                        po.clear();
                        po1.clear();
                    }
                } else {
#pragma unroll
                    for (int o = 0; o < 4; ++o)
                        tile[lane * kTileStride + held * 4 + o] = val[o];
                    ++held;
                    if (held == kChunk / 4 && qi + 1 < nq) flush_chunk();
                }
            };
            // the visit's first quad outside the loop: its taps are used in
            // load order, so each waits only for its own load, and the
            // arithmetic starts while the later taps are still arriving (a
            // first use inside the loop waits for the whole patch)
            quad(0);
            for (int qi = 1; qi < nq; ++qi) quad(qi);
            u += v.w1 - v.w0;
            const bool more = u < u_end;
            Visit nv;
            uint32_t pn[Pl::TB][A][CW];
            if constexpr (kAhead) {
                if (more) {
                    nv = visit_at(u);
                    load_patch<A, K, CW, Pl::TB, CW>(pn, ract, g, nv.win, 0,
                                                     0);
                }
            }
            // the visit's last byte or tile chunk
            if constexpr (REQ) {
                if (v.p < g.npix) {
                    po.store(out, g, v.p, (v.q1 - 1) >> 1);
                    if constexpr (DUAL)
                        po1.store(g.out1, g, v.p, (v.q1 - 1) >> 1);
                }
            } else {
                flush_chunk();
            }
            if (!more) break;
            if constexpr (kAhead) {
                v = nv;
#pragma unroll
                for (int t = 0; t < Pl::TB; ++t)
#pragma unroll
                    for (int i = 0; i < A; ++i)
#pragma unroll
                        for (int c = 0; c < CW; ++c) patch[t][i][c] = pn[t][i][c];
            } else {
                v = visit_at(u);
                if constexpr (SRC != kSrcPacked)
                    load_patch_lds<A, K, CW, K * K, CW>(patch, region, g,
                                                        v.win, zero_off, 0, 0);
                else
                    load_patch<A, K, CW, Pl::TB, CW>(patch, ract, g, v.win, 0,
                                                     0);
            }
        }
    } else {
        // reduction blocks outermost, per tile chunk of up to kChunk
        // channels; partial sums of later blocks are added in the tile
        using Patch = uint32_t[Pl::TB][A][Pl::CB];
        uint32_t* row = tile + lane * kTileStride;
        while (u < u_end) {
            const Visit v = visit_at(u);
            const int q0 = v.q0, q1 = v.q1, p = v.p;
            PackedOut po;
            po.clear();
            for (int sub = q0; sub < q1; sub += kChunk / 4) {
                const int nq = min(kChunk / 4, q1 - sub);
                gu32* qsrc = gw + (size_t)(4 * sub) * FW;
                Slice<Pl::SW> f[2];
                load_slice<A, W, K, CW>(f[0], qsrc);
                auto blk = [&](int nb) {
                    return qsrc + block_offset<A, W, K, CW>(nb);
                };
                auto load_block = [&](Patch& pt, int nb) {
                    const int tb = nb / Pl::NCB;
                    if constexpr (SRC != kSrcPacked)
                        load_patch_lds<A, K, CW, Pl::TB, Pl::CB>(
                            pt, region, g, v.win, zero_off, tb * Pl::TB,
                            (nb - tb * Pl::NCB) * Pl::CB);
                    else
                        load_patch<A, K, CW, Pl::TB, Pl::CB>(
                            pt, ract, g, v.win, tb * Pl::TB,
                            (nb - tb * Pl::NCB) * Pl::CB);
                };
                if constexpr (Pl::DBUF) {
                    // block nb + 1 loads while block nb computes
                    Patch pa, pb;
                    load_block(pa, 0);
#pragma unroll 1
                    for (int nb = 0; nb < NB; nb += 2) {
                        if (nb + 1 < NB) load_block(pb, nb + 1);
                        run_block<A, W, E, K, S, CW>(
                            pa, blk(nb), nq, nb,
                            nb + 1 < NB ? blk(nb + 1) : qsrc, f, row, g, v.oy,
                            v.ox);
                        if (nb + 1 < NB) {
                            if (nb + 2 < NB) load_block(pa, nb + 2);
                            run_block<A, W, E, K, S, CW>(
                                pb, blk(nb + 1), nq, nb + 1,
                                nb + 2 < NB ? blk(nb + 2) : qsrc, f, row, g,
                                v.oy, v.ox);
                        }
                    }
                } else {
                    Patch pa;
#pragma unroll 1
                    for (int nb = 0; nb < NB; ++nb) {
                        load_block(pa, nb);
                        run_block<A, W, E, K, S, CW>(
                            pa, blk(nb), nq, nb,
                            nb + 1 < NB ? blk(nb + 1) : qsrc, f, row, g, v.oy,
                            v.ox);
                    }
                }
                if constexpr (REQ) {
                    // the lane's own tile row, 2 quads per packed byte
                    for (int qi = 0; qi < nq; ++qi) {
                        const int qg = sub + qi;
                        uint32_t val[4];
#pragma unroll
                        for (int o = 0; o < 4; ++o) val[o] = row[qi * 4 + o];
                        po.add4(val, g, qg & 1);
                        if ((qg & 1) == 1 || qg + 1 == q1) {
                            if (p < g.npix) po.store(out, g, p, qg >> 1);
                            po.clear();
                        }
                    }
                } else {
                    wave_lds_sync();
                    flush_tile<false, kCpol>(tile, rout, v.fm, 4 * sub,
                                             nq * 4, lane);
                    wave_lds_sync();
                }
            }
            u += v.w1 - v.w0;
        }
    }
}

using PixKernelFn = void (*)(const uint32_t*, const uint32_t*,
                             const uint32_t*, int32_t*, PixArgs);

// Plan of a kernel as the host reports it.
struct PlanInfo {
    int ocb, ts, tb, cb;
    int enc;    // E of the specialisation: 3 * activation + weight encoding
};

// Kernel for a supported (A, W, encodings, K, S, CW, requantized output) or
// nullptr, with its plan (output channels per filter slice, taps per slice,
// taps and words per plane of a reduction block).  ae / we are the operand
// encodings (kUnipolar, kBipolar, kSigned).  The specialisations are spread
// over several compile units of conv_pix_inst.hip so that they compile in
// parallel:
//   pick_a<A>          unipolar activations, unipolar or bipolar filters
//                      (W = 1..4 / W = 1), int32 or requantized output;
//   pick_signed<A>     signed filters W = 2..4 with unipolar activations,
//                      and signed activations with signed filters of the
//                      same width, int32 output;
//   pick_bipolar_act   +-1 activations with 1-bit filters, int32 output.
// dual: the paired kernel that also computes the centre-tap 1x1 conv.
PixKernelFn pick(int a, int w, int ae, int we, int k, int s, int cw, bool req,
                 int src, bool dual, PlanInfo* info);
template <int A>
PixKernelFn pick_a(int w, bool b, int k, int s, int cw, bool req, int src,
                   bool dual, PlanInfo* info);
template <> PixKernelFn pick_a<1>(int, bool, int, int, int, bool, int, bool,
                                  PlanInfo*);
template <> PixKernelFn pick_a<2>(int, bool, int, int, int, bool, int, bool,
                                  PlanInfo*);
template <> PixKernelFn pick_a<3>(int, bool, int, int, int, bool, int, bool,
                                  PlanInfo*);
template <> PixKernelFn pick_a<4>(int, bool, int, int, int, bool, int, bool,
                                  PlanInfo*);
template <int A>
PixKernelFn pick_signed(int w, int ae, int we, int k, int s, int cw,
                        PlanInfo* info);
template <> PixKernelFn pick_signed<1>(int, int, int, int, int, int, PlanInfo*);
template <> PixKernelFn pick_signed<2>(int, int, int, int, int, int, PlanInfo*);
template <> PixKernelFn pick_signed<3>(int, int, int, int, int, int, PlanInfo*);
template <> PixKernelFn pick_signed<4>(int, int, int, int, int, int, PlanInfo*);
PixKernelFn pick_bipolar_act(int we, int k, int s, int cw, PlanInfo* info);

// Specialisations (included by the sources above).  Requantizing variants
// exist for unipolar activations with unipolar or bipolar filters only;
// staged activations (src != kSrcPacked) for unipolar activations with
// unipolar or bipolar filters, int32 output; paired kernels (dual) for unipolar activations with
// unipolar or bipolar filters, 3x3 windows, whole patches, and at most 16
// filter words per quad of the 1x1 conv (W CW <= 4), int32 or requantized
// output.
template <int A, int W, int E, int K, int S, int CW>
PixKernelFn pick_kscw(bool req, int src, bool dual, PlanInfo* info) {
    using Pl = Plan<A, W, K, CW>;
    constexpr int UU = 3 * kUnipolar + kUnipolar, UB = 3 * kUnipolar + kBipolar;
    if constexpr (!Pl::kFits) {
        return nullptr;
    } else {
        info->ocb = Pl::OCB;
        info->ts = Pl::TS;
        info->tb = Pl::TB;
        info->cb = Pl::CB;
        info->enc = E;
        if (dual) {
            if constexpr (Pl::NB == 1 && K == 3 && W * CW <= 4 &&
                          (E == UU || E == UB)) {
                if (src != kSrcPacked) return nullptr;
                return req ? conv_pix_kernel<A, W, E, K, S, CW, true,
                                             kSrcPacked, true>
                           : conv_pix_kernel<A, W, E, K, S, CW, false,
                                             kSrcPacked, true>;
            } else {
                return nullptr;
            }
        }
        if (src != kSrcPacked) {
            if constexpr (E == UU || E == UB) {
                if (req) return nullptr;
                if (src == kSrcCodes)
                    return conv_pix_kernel<A, W, E, K, S, CW, false,
                                           kSrcCodes, false>;
                // float32 activations: 1x1 windows only (a 3x3 window's
                // staging would read its float rows in one burst before
                // any arithmetic, as long as a separate quantize + pack)
                if constexpr (K == 1) {
                    if (src == kSrcFloat)
                        return conv_pix_kernel<A, W, E, K, S, CW, false,
                                               kSrcFloat, false>;
                }
                return nullptr;
            } else {
                return nullptr;
            }
        }
        if constexpr (E == UU || E == UB)
            return req ? conv_pix_kernel<A, W, E, K, S, CW, true, kSrcPacked,
                                         false>
                       : conv_pix_kernel<A, W, E, K, S, CW, false, kSrcPacked,
                                         false>;
        else
            return req ? nullptr
                       : conv_pix_kernel<A, W, E, K, S, CW, false, kSrcPacked,
                                         false>;
    }
}

// Words per plane: 1..16 for 3x3 windows; 1x1 windows (and dense, a 1x1
// conv) up to 128 words = 4096 input channels.
template <int A, int W, int E, int K, int S>
PixKernelFn pick_cw(int cw, bool req, int src, bool dual, PlanInfo* info) {
    switch (cw) {
        case 1: return pick_kscw<A, W, E, K, S, 1>(req, src, dual, info);
        case 2: return pick_kscw<A, W, E, K, S, 2>(req, src, dual, info);
        case 4: return pick_kscw<A, W, E, K, S, 4>(req, src, dual, info);
        case 8: return pick_kscw<A, W, E, K, S, 8>(req, src, dual, info);
        case 16: return pick_kscw<A, W, E, K, S, 16>(req, src, dual, info);
        default: break;
    }
    if constexpr (K == 1) {
        switch (cw) {
            case 32: return pick_kscw<A, W, E, K, S, 32>(req, src, dual, info);
            case 64: return pick_kscw<A, W, E, K, S, 64>(req, src, dual, info);
            case 128:
                return pick_kscw<A, W, E, K, S, 128>(req, src, dual, info);
            default: break;
        }
    }
    return nullptr;
}

template <int A, int W, int E>
PixKernelFn pick_ks(int k, int s, int cw, bool req, int src, bool dual,
                    PlanInfo* info) {
    if (k == 1)
        return s == 1 ? pick_cw<A, W, E, 1, 1>(cw, req, src, dual, info)
                      : pick_cw<A, W, E, 1, 2>(cw, req, src, dual, info);
    if (k == 3)
        return s == 1 ? pick_cw<A, W, E, 3, 1>(cw, req, src, dual, info)
                      : pick_cw<A, W, E, 3, 2>(cw, req, src, dual, info);
    return nullptr;
}

// Unipolar activations: every weight width 1..4 with unipolar weights;
// bipolar weights at W = 1.
template <int A>
PixKernelFn pick_for_a(int w, bool b, int k, int s, int cw, bool req, int src,
                       bool dual, PlanInfo* info) {
    constexpr int UU = 3 * kUnipolar + kUnipolar, UB = 3 * kUnipolar + kBipolar;
    if (b) return w == 1 ? pick_ks<A, 1, UB>(k, s, cw, req, src, dual, info)
                         : nullptr;
    switch (w) {
        case 1: return pick_ks<A, 1, UU>(k, s, cw, req, src, dual, info);
        case 2: return pick_ks<A, 2, UU>(k, s, cw, req, src, dual, info);
        case 3: return pick_ks<A, 3, UU>(k, s, cw, req, src, dual, info);
        case 4: return pick_ks<A, 4, UU>(k, s, cw, req, src, dual, info);
        default: return nullptr;
    }
}

// Signed filters of width 2..4 with unipolar activations; signed
// activations with signed filters of the same width.
template <int A>
PixKernelFn pick_signed_for_a(int w, int ae, int we, int k, int s, int cw,
                              PlanInfo* info) {
    constexpr int US = 3 * kUnipolar + kSigned, SS = 3 * kSigned + kSigned;
    if (we != kSigned) return nullptr;
    if (ae == kSigned) {
        if constexpr (A >= 2)
            return w == A ? pick_ks<A, A, SS>(k, s, cw, false, kSrcPacked,
                                              false, info)
                          : nullptr;
        else
            return nullptr;
    }
    if (ae != kUnipolar) return nullptr;
    switch (w) {
        case 2:
            return pick_ks<A, 2, US>(k, s, cw, false, kSrcPacked, false,
                                      info);
        case 3:
            return pick_ks<A, 3, US>(k, s, cw, false, kSrcPacked, false,
                                      info);
        case 4:
            return pick_ks<A, 4, US>(k, s, cw, false, kSrcPacked, false,
                                      info);
        default: return nullptr;
    }
}

}  // namespace pix
}  // namespace bs
