// Quantize and bit-pack kernels for gfx950 (wave64).
//
// quantize       float32 -> uint8 codes (Sec. 3.1 quantization operator)
// pack           uint8 codes -> bit-planes packed into uint32 words along the
//                reduction axis, layout [rows][bits][ceil(k/32)] (Sec. 2.2,
//                Sec. 3.1, MBK')
// quantize_pack  both in one pass over the float32 data
//
// All three stream HBM once and do a few integer ops per element, so they
// are bound by memory bandwidth; the kernels are shaped for coalesced
// 16-byte (or 256-byte-per-wave) accesses.
#include "bs_internal.h"

namespace bs {
namespace {

constexpr int kBlock = 256;
constexpr int kMaxBlocks = 8192;

// One quantizer code: round-half-to-even of a single binary32 product,
// clamped to [0, qmax] with NaN sent to 0.  Bipolar: 1 iff x >= 0.
// (A lone multiply followed by rint leaves nothing to contract into an FMA.)
template <bool BIP>
__device__ __forceinline__ uint32_t code_of(float x, float scale, float qmax) {
    if (BIP) return x >= 0.0f ? 1u : 0u;
    float r = __builtin_rintf(x * scale);
    r = r > 0.0f ? r : 0.0f;   // negative, -0 and NaN -> 0
    r = r < qmax ? r : qmax;   // saturate (+inf included)
    return (uint32_t)r;
}

template <bool BIP>
__device__ __forceinline__ uint32_t codes4(float4 f, float scale, float qmax) {
    return code_of<BIP>(f.x, scale, qmax) |
           (code_of<BIP>(f.y, scale, qmax) << 8) |
           (code_of<BIP>(f.z, scale, qmax) << 16) |
           (code_of<BIP>(f.w, scale, qmax) << 24);
}

// ---------------------------------------------------------------------------
// quantize: 16 elements per thread per step (four 16-byte loads, one 16-byte
// store); the n % 16 tail is done one element per thread.
template <bool BIP>
__global__ __launch_bounds__(kBlock) void quantize_kernel(
    const float* __restrict__ x, uint8_t* __restrict__ q, int64_t n,
    float scale, float qmax) {
    const int64_t nvec = n >> 4;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t nthr = (int64_t)gridDim.x * kBlock;
    const float4* xv = reinterpret_cast<const float4*>(x);
    uint4* qv = reinterpret_cast<uint4*>(q);
    for (int64_t v = tid; v < nvec; v += nthr) {
        float4 f0 = xv[4 * v + 0], f1 = xv[4 * v + 1];
        float4 f2 = xv[4 * v + 2], f3 = xv[4 * v + 3];
        qv[v] = make_uint4(codes4<BIP>(f0, scale, qmax),
                           codes4<BIP>(f1, scale, qmax),
                           codes4<BIP>(f2, scale, qmax),
                           codes4<BIP>(f3, scale, qmax));
    }
    const int64_t tail = nvec << 4;
    if (tid < n - tail)
        q[tail + tid] = (uint8_t)code_of<BIP>(x[tail + tid], scale, qmax);
}

// ---------------------------------------------------------------------------
// pack, k % 32 == 0: one thread per 32-element group (= one output word per
// plane).  The group's 32 bytes are two 16-byte loads; consecutive threads
// read consecutive 32-byte chunks.  Plane b of four bytes v is gathered in
// registers: the bits sit at 0, 8, 16, 24 after (v >> b) & 0x01010101 and two
// shift-or steps fold them into the low nibble.
__device__ __forceinline__ uint32_t nibble_of(uint32_t v, int b) {
    uint32_t x = (v >> b) & 0x01010101u;
    x = (x | (x >> 7)) & 0x00030003u;   // bits 0,1 and 16,17
    return (x | (x >> 14)) & 0xFu;      // bits 0..3
}

template <int A>
__global__ __launch_bounds__(kBlock) void pack32_kernel(
    const uint8_t* __restrict__ q, uint32_t* __restrict__ packed,
    uint32_t groups, FastDiv kwdiv) {
    const uint32_t kw = kwdiv.d;
    const uint4* src = reinterpret_cast<const uint4*>(q);
    for (uint32_t g = blockIdx.x * kBlock + threadIdx.x; g < groups;
         g += gridDim.x * kBlock) {
        const uint4 lo = src[2 * (size_t)g], hi = src[2 * (size_t)g + 1];
        const uint32_t v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
        const uint32_t row = kwdiv.div(g), t = g - row * kw;
        uint32_t* dst = packed + (size_t)row * A * kw + t;
#pragma unroll
        for (int b = 0; b < A; ++b) {
            uint32_t word = 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) word |= nibble_of(v[i], b) << (4 * i);
            dst[(size_t)b * kw] = word;
        }
    }
}

// ---------------------------------------------------------------------------
// Wave-ballot packing, any k and any alignment: one wave handles a 64-element
// chunk of one row.  Lane l holds element 64c + l; the wave ballot of bit b
// is then exactly the two packed words 2c, 2c+1 of plane b (bit l <- lane l),
// so no per-lane bit shuffling is needed.  Used for the uint8 input when k is
// not a multiple of 32 and for the float input whenever k is not.
template <bool FROM_FLOAT, bool BIP>
__global__ __launch_bounds__(kBlock) void pack_ballot_kernel(
    const void* __restrict__ src, uint32_t* __restrict__ packed, int64_t rows,
    int64_t k, int bits, float scale, float qmax) {
    const int lane = threadIdx.x & 63;
    const int64_t nchunks = (k + 63) >> 6;
    const int64_t kw = (k + 31) >> 5;
    const int64_t total = rows * nchunks;
    const int64_t nwaves = ((int64_t)gridDim.x * kBlock) >> 6;
    for (int64_t wid = ((int64_t)blockIdx.x * kBlock + threadIdx.x) >> 6;
         wid < total; wid += nwaves) {
        const int64_t row = wid / nchunks, c = wid - row * nchunks;
        const int64_t e = c * 64 + lane;
        uint32_t code = 0;
        if (e < k) {
            if (FROM_FLOAT)
                code = code_of<BIP>(
                    static_cast<const float*>(src)[row * k + e], scale, qmax);
            else
                code = static_cast<const uint8_t*>(src)[row * k + e];
        }
        uint32_t* dst = packed + row * bits * kw;
        for (int b = 0; b < bits; ++b) {
            const uint64_t m = __ballot((code >> b) & 1u);
            const int64_t t = 2 * c + lane;
            if (lane < 2 && t < kw)
                dst[b * kw + t] = lane == 0 ? (uint32_t)m : (uint32_t)(m >> 32);
        }
    }
}

// ---------------------------------------------------------------------------
// quantize_pack, k % 32 == 0: one wave produces 64 consecutive output words
// (2048 consecutive elements of the flat [rows][k] array, which never splits
// a word across rows).  Each step loads 64 consecutive floats (256 coalesced
// bytes per wave), quantizes them and takes one ballot per plane; the ballot
// is words 2c, 2c+1 of the block and is parked in lanes 2c, 2c+1.  After 32
// steps lane l holds word l of every plane and stores it.
template <int A, bool BIP>
__global__ __launch_bounds__(kBlock) void quantize_pack_ballot_kernel(
    const float* __restrict__ x, uint32_t* __restrict__ packed,
    uint32_t nwords, FastDiv kwdiv, float scale, float qmax) {
    const int lane = threadIdx.x & 63;
    const uint32_t kw = kwdiv.d;
    const uint32_t wave0 = (blockIdx.x * kBlock + threadIdx.x) >> 6;
    const uint32_t nwaves = (gridDim.x * kBlock) >> 6;
    for (uint32_t base = wave0 * 64u; base < nwords; base += nwaves * 64u) {
        uint32_t words[A];
#pragma unroll
        for (int b = 0; b < A; ++b) words[b] = 0;
        const float* xb = x + (size_t)base * 32 + lane;
        const uint32_t left = nwords - base;   // words still to produce
#pragma unroll 8
        for (int c = 0; c < 32; ++c) {
            uint32_t code = 0;
            // lanes 0-31 feed word 2c, lanes 32-63 word 2c+1
            if ((uint32_t)(2 * c + (lane >> 5)) < left)
                code = code_of<BIP>(xb[(size_t)c * 64], scale, qmax);
#pragma unroll
            for (int b = 0; b < A; ++b) {
                const uint64_t m = __ballot((code >> b) & 1u);
                words[b] = lane == 2 * c ? (uint32_t)m : words[b];
                words[b] = lane == 2 * c + 1 ? (uint32_t)(m >> 32) : words[b];
            }
        }
        const uint32_t wi = base + lane;
        if (wi < nwords) {
            const uint32_t row = kwdiv.div(wi), t = wi - row * kw;
            uint32_t* dst = packed + (size_t)row * A * kw + t;
#pragma unroll
            for (int b = 0; b < A; ++b) dst[(size_t)b * kw] = words[b];
        }
    }
}

int grid_for(int64_t work_items, int per_block) {
    int64_t b = (work_items + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > kMaxBlocks) b = kMaxBlocks;
    return (int)b;
}

template <int A>
hipError_t launch_pack32(const uint8_t* q, uint32_t* packed, uint32_t groups,
                         const FastDiv& d, hipStream_t st) {
    pack32_kernel<A><<<grid_for(groups, kBlock), kBlock, 0, st>>>(q, packed,
                                                                  groups, d);
    return hipGetLastError();
}

template <int A, bool BIP>
hipError_t launch_qpack(const float* x, uint32_t* packed, uint32_t nwords,
                        const FastDiv& d, float scale, float qmax,
                        hipStream_t st) {
    // 64 words per wave, 4 waves per block
    quantize_pack_ballot_kernel<A, BIP>
        <<<grid_for(nwords, 256), kBlock, 0, st>>>(x, packed, nwords, d,
                                                    scale, qmax);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const float* x, uint8_t* q, int64_t n, float scale,
                           int bits, bool bipolar, hipStream_t st) {
    const float qmax = (float)((1 << bits) - 1);
    const int grid = grid_for((n >> 4) + 1, kBlock);
    if (bipolar)
        quantize_kernel<true><<<grid, kBlock, 0, st>>>(x, q, n, scale, qmax);
    else
        quantize_kernel<false><<<grid, kBlock, 0, st>>>(x, q, n, scale, qmax);
    return hipGetLastError();
}

hipError_t launch_pack(const uint8_t* q, uint32_t* packed, int64_t rows,
                       int64_t k, int bits, hipStream_t st) {
    const int64_t kw = (k + 31) / 32;
    const int64_t groups = rows * kw;
    if (k % 32 == 0 && groups < (int64_t)INT32_MAX) {
        FastDiv d;
        d.init((uint32_t)kw);
        switch (bits) {
            case 1: return launch_pack32<1>(q, packed, (uint32_t)groups, d, st);
            case 2: return launch_pack32<2>(q, packed, (uint32_t)groups, d, st);
            case 3: return launch_pack32<3>(q, packed, (uint32_t)groups, d, st);
            case 4: return launch_pack32<4>(q, packed, (uint32_t)groups, d, st);
            case 5: return launch_pack32<5>(q, packed, (uint32_t)groups, d, st);
            case 6: return launch_pack32<6>(q, packed, (uint32_t)groups, d, st);
            case 7: return launch_pack32<7>(q, packed, (uint32_t)groups, d, st);
            default: return launch_pack32<8>(q, packed, (uint32_t)groups, d, st);
        }
    }
    const int64_t waves = rows * ((k + 63) / 64);
    pack_ballot_kernel<false, false><<<grid_for(waves, 4), kBlock, 0, st>>>(
        q, packed, rows, k, bits, 0.0f, 0.0f);
    return hipGetLastError();
}

hipError_t launch_quantize_pack(const float* x, uint32_t* packed,
                                int64_t rows, int64_t k, float scale, int bits,
                                bool bipolar, hipStream_t st) {
    const float qmax = (float)((1 << bits) - 1);
    const int64_t nwords = rows * ((k + 31) / 32);
    if (k % 32 == 0 && nwords < (int64_t)INT32_MAX - 64) {
        FastDiv d;
        d.init((uint32_t)(k / 32));
        if (bipolar) return launch_qpack<1, true>(x, packed, (uint32_t)nwords,
                                                  d, scale, qmax, st);
        switch (bits) {
            case 1: return launch_qpack<1, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 2: return launch_qpack<2, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 3: return launch_qpack<3, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 4: return launch_qpack<4, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 5: return launch_qpack<5, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 6: return launch_qpack<6, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            case 7: return launch_qpack<7, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
            default: return launch_qpack<8, false>(x, packed, (uint32_t)nwords, d, scale, qmax, st);
        }
    }
    const int64_t waves = rows * ((k + 63) / 64);
    if (bipolar)
        pack_ballot_kernel<true, true><<<grid_for(waves, 4), kBlock, 0, st>>>(
            x, packed, rows, k, bits, scale, qmax);
    else
        pack_ballot_kernel<true, false><<<grid_for(waves, 4), kBlock, 0, st>>>(
            x, packed, rows, k, bits, scale, qmax);
    return hipGetLastError();
}

}  // namespace bs
