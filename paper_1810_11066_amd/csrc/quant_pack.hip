// Quantize and bit-pack kernels for gfx950 (wave64).
//
// quantize       float32 -> uint8 codes (Sec. 3.1 quantization operator)
// pack           uint8 codes -> bit-planes packed into uint32 words along the
//                reduction axis, layout [rows][bits][ceil(k/32)] (Sec. 2.2,
//                Sec. 3.1, MBK')
// quantize_pack  both in one pass over the float32 data
//
// All three stream HBM once and do a few integer ops per element, so they
// are bound by memory bandwidth.  Every load is a 16-byte vector load with
// consecutive lanes reading consecutive addresses; the bits of one packed
// word are gathered in registers and joined across lanes with DPP ORs (or
// wave ballots in the any-k fallback).
//
// Inputs are read once, with non-temporal loads: they do not push out of the
// caches what the surrounding kernels leave there -- in particular the int32
// output of a preceding convolution, whose write-back to HBM then overlaps
// the next convolution (bound by the vector ALUs) instead of this kernel.
// Measured on the ResNet-18 layers at batch 128: quantize+pack+conv steps
// 4-17 % shorter.
#include "bs_internal.h"

namespace bs {
namespace {

__device__ __forceinline__ uint4 stream_load(const uint4* p) {
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 t =
        __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(t[0], t[1], t[2], t[3]);
}
__device__ __forceinline__ float4 stream_load(const float4* p) {
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    const f32x4 t =
        __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    return make_float4(t[0], t[1], t[2], t[3]);
}

constexpr int kBlock = 256;
constexpr int kMaxBlocks = 8192;

// ENC: kUnipolar, kBipolar or kSigned (qmax as for quant_code_enc)
template <int ENC>
__device__ __forceinline__ uint32_t code_of(float x, float scale, float qmax) {
    return quant_code_enc<ENC>(x, scale, qmax);
}

template <int ENC>
__device__ __forceinline__ uint32_t codes4(float4 f, float scale, float qmax) {
    return code_of<ENC>(f.x, scale, qmax) |
           (code_of<ENC>(f.y, scale, qmax) << 8) |
           (code_of<ENC>(f.z, scale, qmax) << 16) |
           (code_of<ENC>(f.w, scale, qmax) << 24);
}

// ---------------------------------------------------------------------------
// quantize: 16 elements per thread per step (four 16-byte loads, one 16-byte
// store); the n % 16 tail is done one element per thread.
template <int ENC>
__global__ __launch_bounds__(kBlock) void quantize_kernel(
    const float* __restrict__ x, uint8_t* __restrict__ q, int64_t n,
    float scale, float qmax) {
    const int64_t nvec = n >> 4;
    const int64_t tid = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t nthr = (int64_t)gridDim.x * kBlock;
    const float4* xv = reinterpret_cast<const float4*>(x);
    uint4* qv = reinterpret_cast<uint4*>(q);
    for (int64_t v = tid; v < nvec; v += nthr) {
        float4 f0 = stream_load(xv + 4 * v + 0);
        float4 f1 = stream_load(xv + 4 * v + 1);
        float4 f2 = stream_load(xv + 4 * v + 2);
        float4 f3 = stream_load(xv + 4 * v + 3);
        qv[v] = make_uint4(codes4<ENC>(f0, scale, qmax),
                           codes4<ENC>(f1, scale, qmax),
                           codes4<ENC>(f2, scale, qmax),
                           codes4<ENC>(f3, scale, qmax));
    }
    const int64_t tail = nvec << 4;
    if (tid < n - tail)
        q[tail + tid] = (uint8_t)code_of<ENC>(x[tail + tid], scale, qmax);
}

// ---------------------------------------------------------------------------
// Cross-lane OR with a DPP lane permutation (all source lanes are inside the
// 8-lane group, so every lane reads a defined value).
constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]: lane ^ 1
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]: lane ^ 2
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror: lane i <-> 7 - i

template <int CTRL>
__device__ __forceinline__ uint32_t or_dpp(uint32_t v) {
    return v | (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF,
                                                     false);
}

// pack, k % 32 == 0: a wave packs 128 consecutive words of the flat
// [rows][k / 32] word array (4096 codes, which never split a word across
// rows).  Load j (0..3) reads 16 codes per lane, lanes consecutive, so every
// load is one coalesced 1 KiB.  Lanes 2p, 2p+1 of load j hold the two halves
// of word 32 j + p: each gathers its 16 bits of plane b in registers and one
// DPP OR joins the halves.  Lane 2p + i keeps word 32 j + p when j % 2 == i
// (slot j / 2); one ds_bpermute per plane and slot then moves word w to lane
// w % 64, so the stores write 64 consecutive words.
template <int A>
__global__ __launch_bounds__(kBlock) void pack_dpp_kernel(
    const uint8_t* __restrict__ q, uint32_t* __restrict__ packed,
    uint32_t nwords, FastDiv kwdiv) {
    const int lane = threadIdx.x & 63;
    const uint32_t kw = kwdiv.d;
    const uint4* src = reinterpret_cast<const uint4*>(q);
    const uint32_t wave0 = (blockIdx.x * kBlock + threadIdx.x) >> 6;
    const uint32_t nwaves = (gridDim.x * kBlock) >> 6;
    // lane l's words (l and 64 + l of the chunk) come from lane 2 (l % 32) +
    // l / 32, which holds them in slots 0 and 1
    const int from = (2 * (lane & 31) + (lane >> 5)) * 4;
    for (uint32_t base = wave0 * 128u; base < nwords; base += nwaves * 128u) {
        const uint32_t left = nwords - base;
        uint4 v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            // this lane's 16 codes belong to word 32 j + lane / 2
            const bool ok = (uint32_t)(32 * j + (lane >> 1)) < left;
            v[j] = ok ? stream_load(src + (size_t)base * 2 + 64 * j + lane)
                      : make_uint4(0, 0, 0, 0);
        }
        uint32_t keep[A][2];
#pragma unroll
        for (int b = 0; b < A; ++b) keep[b][0] = keep[b][1] = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int b = 0; b < A; ++b) {
                uint32_t h = nibble_of(v[j].x, b) | nibble_of(v[j].y, b) << 4 |
                             nibble_of(v[j].z, b) << 8 |
                             nibble_of(v[j].w, b) << 12;
                h <<= 16 * (lane & 1);
                h = or_dpp<kDppQuadXor1>(h);
                if ((lane & 1) == (j & 1)) keep[b][j >> 1] = h;
            }
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const uint32_t wi = base + 64 * s + lane;
            uint32_t word[A];
#pragma unroll
            for (int b = 0; b < A; ++b)
                word[b] = (uint32_t)__builtin_amdgcn_ds_bpermute(
                    from, (int)keep[b][s]);
            if (wi < nwords) {
                const uint32_t row = kwdiv.div(wi), t = wi - row * kw;
                uint32_t* dst = packed + (size_t)row * A * kw + t;
#pragma unroll
                for (int b = 0; b < A; ++b) dst[(size_t)b * kw] = word[b];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Wave-ballot packing, any k and any alignment: one wave handles a 64-element
// chunk of one row.  Lane l holds element 64c + l; the wave ballot of bit b
// is then exactly the two packed words 2c, 2c+1 of plane b (bit l <- lane l),
// so no per-lane bit shuffling is needed.  Used for the uint8 input when k is
// not a multiple of 32 and for the float input whenever k is not.
template <bool FROM_FLOAT, int ENC>
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
                code = code_of<ENC>(
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
// quantize_pack, k % 32 == 0: a wave produces 64 consecutive words of the
// flat [rows][k / 32] word array (2048 floats).  Load j (0..7) reads one
// float4 per lane, lanes consecutive (coalesced 1 KiB).  The 8 lanes
// 8m .. 8m+7 of load j hold word 8 j + m, 4 elements each: every lane
// quantizes its 4 values, places their plane-b bits at 4 (lane % 8), and
// three DPP ORs combine the group.  Lane 8m + i keeps word 8 j + m when
// j == i; a ds_bpermute per plane then moves word w to lane w.
template <int A, int ENC>
__global__ __launch_bounds__(kBlock) void quantize_pack_dpp_kernel(
    const float* __restrict__ x, uint32_t* __restrict__ packed,
    uint32_t nwords, FastDiv kwdiv, float scale, float qmax) {
    const int lane = threadIdx.x & 63;
    const uint32_t kw = kwdiv.d;
    const float4* xv = reinterpret_cast<const float4*>(x);
    const uint32_t wave0 = (blockIdx.x * kBlock + threadIdx.x) >> 6;
    const uint32_t nwaves = (gridDim.x * kBlock) >> 6;
    // word l is held by lane 8 (l % 8) + l / 8
    const int from = (8 * (lane & 7) + (lane >> 3)) * 4;
    for (uint32_t base = wave0 * 64u; base < nwords; base += nwaves * 64u) {
        const uint32_t left = nwords - base;
        float4 f[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const bool ok = (uint32_t)(8 * j + (lane >> 3)) < left;
            f[j] = ok ? stream_load(xv + (size_t)base * 8 + 64 * j + lane)
                      : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        uint32_t keep[A];
#pragma unroll
        for (int b = 0; b < A; ++b) keep[b] = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t c4 = codes4<ENC>(f[j], scale, qmax);
#pragma unroll
            for (int b = 0; b < A; ++b) {
                uint32_t h = nibble_of(c4, b) << (4 * (lane & 7));
                h = or_dpp<kDppQuadXor1>(h);
                h = or_dpp<kDppQuadXor2>(h);
                h = or_dpp<kDppHalfMirror>(h);
                if ((lane & 7) == j) keep[b] = h;
            }
        }
        uint32_t word[A];
#pragma unroll
        for (int b = 0; b < A; ++b)
            word[b] = (uint32_t)__builtin_amdgcn_ds_bpermute(from, (int)keep[b]);
        const uint32_t wi = base + lane;
        if (wi < nwords) {
            const uint32_t row = kwdiv.div(wi), t = wi - row * kw;
            uint32_t* dst = packed + (size_t)row * A * kw + t;
#pragma unroll
            for (int b = 0; b < A; ++b) dst[(size_t)b * kw] = word[b];
        }
    }
}

// ---------------------------------------------------------------------------
// pack_ex: the codes viewed as [outer][k][inner], the reduction axis k at
// stride `inner` (NCHW activations, OIHW filters).  A thread builds word t of
// every plane for V consecutive rows i0 .. i0+V-1 of one outer index: for
// each of the word's 32 elements it makes one V-byte load (neighbouring
// threads take neighbouring rows, so a load instruction reads one contiguous
// span), then moves every bit into place with an extract and a shift-or.
// The words are stored where the layout puts them.
template <int V>
__global__ __launch_bounds__(kBlock) void pack_strided_kernel(
    const uint8_t* __restrict__ q, uint32_t* __restrict__ packed,
    int64_t outer, int64_t k, int64_t inner, int bits, int layout) {
    const int64_t kw = (k + 31) >> 5;
    const int64_t iv = inner / V;            // V divides inner (host)
    const int64_t total = outer * kw * iv;
    const int64_t rows = outer * inner;
    for (int64_t f = (int64_t)blockIdx.x * kBlock + threadIdx.x; f < total;
         f += (int64_t)gridDim.x * kBlock) {
        const int64_t ig = f % iv, rest = f / iv;
        const int64_t t = rest % kw, o = rest / kw;
        const int64_t i0 = ig * V;
        const int64_t left = k - 32 * t;
        const int u_end = left < 32 ? (int)left : 32;
        const uint8_t* src = q + (o * k + 32 * t) * inner + i0;
        uint32_t word[V][8];
#pragma unroll
        for (int v = 0; v < V; ++v)
#pragma unroll
            for (int b = 0; b < 8; ++b) word[v][b] = 0;
        for (int u = 0; u < u_end; ++u) {
            uint32_t x;
            if constexpr (V == 4)
                x = *reinterpret_cast<const uint32_t*>(src + (int64_t)u * inner);
            else
                x = src[(int64_t)u * inner];
#pragma unroll
            for (int v = 0; v < V; ++v)
#pragma unroll
                for (int b = 0; b < 8; ++b)
                    if (b < bits) word[v][b] |= ((x >> (8 * v + b)) & 1u) << u;
        }
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int64_t r = o * inner + i0 + v;
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                if (b >= bits) continue;
                int64_t at;
                if (layout == kLayoutMBK) at = (r * bits + b) * kw + t;
                else if (layout == kLayoutMKB) at = (r * kw + t) * bits + b;
                else at = ((int64_t)b * rows + r) * kw + t;
                packed[at] = word[v][b];
            }
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
hipError_t launch_pack32(const uint8_t* q, uint32_t* packed, uint32_t nwords,
                         const FastDiv& d, hipStream_t st) {
    // 128 words per wave, 4 waves per block
    return launch(pack_dpp_kernel<A>, dim3(grid_for(nwords, 512)),
                  dim3(kBlock), 0, st, q, packed, nwords, d);
}

template <int A, int ENC>
hipError_t launch_qpack(const float* x, uint32_t* packed, uint32_t nwords,
                        const FastDiv& d, float scale, float qmax,
                        hipStream_t st) {
    // 64 words per wave, 4 waves per block
    return launch(quantize_pack_dpp_kernel<A, ENC>,
                  dim3(grid_for(nwords, 256)), dim3(kBlock), 0, st, x, packed,
                  nwords, d, scale, qmax);
}

}  // namespace

// qmax of an encoding: the top unipolar code, the top signed value
static float enc_qmax(int bits, int enc) {
    return enc == kSigned ? (float)((1 << (bits - 1)) - 1)
                          : (float)((1 << bits) - 1);
}

hipError_t launch_quantize(const float* x, uint8_t* q, int64_t n, float scale,
                           int bits, int enc, hipStream_t st) {
    const float qmax = enc_qmax(bits, enc);
    const dim3 grid(grid_for((n >> 4) + 1, kBlock));
    if (enc == kBipolar)
        return launch(quantize_kernel<kBipolar>, grid, dim3(kBlock), 0, st, x,
                      q, n, scale, qmax);
    if (enc == kSigned)
        return launch(quantize_kernel<kSigned>, grid, dim3(kBlock), 0, st, x,
                      q, n, scale, qmax);
    return launch(quantize_kernel<kUnipolar>, grid, dim3(kBlock), 0, st, x, q,
                  n, scale, qmax);
}

hipError_t launch_pack(const uint8_t* q, uint32_t* packed, int64_t rows,
                       int64_t k, int bits, hipStream_t st) {
    const int64_t kw = (k + 31) / 32;
    const int64_t groups = rows * kw;
    if (k % 32 == 0 && groups < (int64_t)INT32_MAX - 128) {
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
    return launch(pack_ballot_kernel<false, kUnipolar>,
                  dim3(grid_for(waves, 4)), dim3(kBlock), 0, st, q, packed,
                  rows, k, bits, 0.0f, 0.0f);
}

hipError_t launch_pack_ex(const uint8_t* q, uint32_t* packed, int64_t outer,
                          int64_t k, int64_t inner, int bits, int layout,
                          hipStream_t st) {
    if (inner == 1 && layout == kLayoutMBK)
        return launch_pack(q, packed, outer, k, bits, st);
    const int64_t kw = (k + 31) / 32;
    if (inner % 4 == 0)
        return launch(pack_strided_kernel<4>,
                      dim3(grid_for(outer * kw * (inner / 4), kBlock)),
                      dim3(kBlock), 0, st, q, packed, outer, k, inner, bits,
                      layout);
    return launch(pack_strided_kernel<1>,
                  dim3(grid_for(outer * kw * inner, kBlock)), dim3(kBlock), 0,
                  st, q, packed, outer, k, inner, bits, layout);
}

namespace {

template <int ENC>
hipError_t quantize_pack_enc(const float* x, uint32_t* packed, int64_t rows,
                             int64_t k, float scale, int bits, float qmax,
                             hipStream_t st) {
    const int64_t nwords = rows * ((k + 31) / 32);
    if (k % 32 == 0 && nwords < (int64_t)INT32_MAX - 64) {
        FastDiv d;
        d.init((uint32_t)(k / 32));
        const uint32_t nw = (uint32_t)nwords;
        switch (bits) {
            case 1: return launch_qpack<1, ENC>(x, packed, nw, d, scale, qmax, st);
            case 2: return launch_qpack<2, ENC>(x, packed, nw, d, scale, qmax, st);
            case 3: return launch_qpack<3, ENC>(x, packed, nw, d, scale, qmax, st);
            case 4: return launch_qpack<4, ENC>(x, packed, nw, d, scale, qmax, st);
            case 5: return launch_qpack<5, ENC>(x, packed, nw, d, scale, qmax, st);
            case 6: return launch_qpack<6, ENC>(x, packed, nw, d, scale, qmax, st);
            case 7: return launch_qpack<7, ENC>(x, packed, nw, d, scale, qmax, st);
            default: return launch_qpack<8, ENC>(x, packed, nw, d, scale, qmax, st);
        }
    }
    const int64_t waves = rows * ((k + 63) / 64);
    return launch(pack_ballot_kernel<true, ENC>, dim3(grid_for(waves, 4)),
                  dim3(kBlock), 0, st, x, packed, rows, k, bits, scale, qmax);
}

}  // namespace

hipError_t launch_quantize_pack(const float* x, uint32_t* packed,
                                int64_t rows, int64_t k, float scale, int bits,
                                int enc, hipStream_t st) {
    const float qmax = enc_qmax(bits, enc);
    if (enc == kBipolar)
        return quantize_pack_enc<kBipolar>(x, packed, rows, k, scale, 1, qmax,
                                           st);
    if (enc == kSigned)
        return quantize_pack_enc<kSigned>(x, packed, rows, k, scale, bits,
                                          qmax, st);
    return quantize_pack_enc<kUnipolar>(x, packed, rows, k, scale, bits, qmax,
                                        st);
}

}  // namespace bs
