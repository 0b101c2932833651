// Internal declarations shared by the HIP sources of libbitserial.so.
// Not installed; the public interface is include/bitserial.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bs {

// Division of a non-negative int32 by a fixed positive divisor with one
// 64-bit multiply and a shift: q = (n * m) >> s, m = ceil(2^s / d),
// s = 32 + ceil(log2 d).  Exact for every n < 2^31 (the rounding error
// n (m d - 2^s) / (d 2^s) stays below 1/d because m d - 2^s < d <= 2^(s-32)).
struct FastDiv {
    uint64_t m;
    uint32_t s;
    uint32_t d;

    __host__ void init(uint32_t divisor) {
        d = divisor;
        uint32_t sh = 0;
        while ((1ull << sh) < divisor) ++sh;
        s = 32 + sh;
        m = ((1ull << s) + divisor - 1) / divisor;
    }
    __host__ __device__ __forceinline__ uint32_t div(uint32_t n) const {
        return (uint32_t)(((uint64_t)n * m) >> s);
    }
};

// One quantizer code (the reading of the quantization operator used
// throughout): round-half-to-even of a single binary32 product, clamped to
// [0, qmax] with NaN sent to 0.  Bipolar: 1 iff x >= 0.  (A lone multiply
// followed by rint leaves nothing to contract into an FMA.)
template <bool BIP>
__device__ __forceinline__ uint32_t quant_code(float x, float scale,
                                               float qmax) {
    if (BIP) return x >= 0.0f ? 1u : 0u;
    float r = __builtin_rintf(x * scale);
    r = r > 0.0f ? r : 0.0f;   // negative, -0 and NaN -> 0
    r = r < qmax ? r : qmax;   // saturate (+inf included)
    return (uint32_t)r;
}

// Signed (two's complement) code: round-half-to-even of the binary32
// product clamped to [-(hmax + 1), hmax] with NaN sent to 0, returned as its
// low bits (hmax = 2^(bits-1) - 1).
__device__ __forceinline__ uint32_t quant_code_signed(float x, float scale,
                                                      float hmax) {
    float r = __builtin_rintf(x * scale);
    r = r == r ? r : 0.0f;                 // NaN -> 0
    r = r > -hmax - 1.0f ? r : -hmax - 1.0f;
    r = r < hmax ? r : hmax;               // saturate (+-inf included)
    return (uint32_t)(int32_t)r & (uint32_t)(2.0f * hmax + 1.0f);
}

// Operand encodings (the values of bs_encoding).
constexpr int kUnipolar = 0, kBipolar = 1, kSigned = 2;

// Code of one value under encoding ENC; qmax is 2^bits - 1 for unipolar
// codes and 2^(bits-1) - 1 for signed ones (bipolar ignores it).
template <int ENC>
__device__ __forceinline__ uint32_t quant_code_enc(float x, float scale,
                                                   float qmax) {
    if constexpr (ENC == kSigned) return quant_code_signed(x, scale, qmax);
    else return quant_code<ENC == kBipolar>(x, scale, qmax);
}

// Bits b of the four bytes of v (bit b of byte k -> bit k of the result).
__device__ __forceinline__ uint32_t nibble_of(uint32_t v, int b) {
    uint32_t x = (v >> b) & 0x01010101u;
    x = (x | (x >> 7)) & 0x00030003u;   // bits 0,1 and 16,17
    return (x | (x >> 14)) & 0xFu;      // bits 0..3
}

// ---- kernel launch -------------------------------------------------------

// The calling host thread's timing events (bs_set_timing_events); both
// null unless a benchmark set them.
struct TimingEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
TimingEvents& timing_events();

// Launches fn.  With the thread's timing events set, the launch goes
// through hipExtLaunchKernel, which has the runtime stamp the events with
// this dispatch's own start and end.
hipError_t launch_kernel(const void* fn, dim3 grid, dim3 block, void** args,
                         size_t lds, hipStream_t st);

template <typename T>
struct Ident {
    using type = T;
};

// Typed form: the arguments convert to the kernel's parameter types.
template <typename... P>
hipError_t launch(void (*fn)(P...), dim3 grid, dim3 block, size_t lds,
                  hipStream_t st, typename Ident<P>::type... args) {
    void* argv[] = {(void*)&args...};
    return launch_kernel((const void*)fn, grid, block, argv, lds, st);
}

// ---- launchers (each returns hipSuccess or the launch error) -------------

// enc: kUnipolar, kBipolar or kSigned
hipError_t launch_quantize(const float* x, uint8_t* q, int64_t n, float scale,
                           int bits, int enc, hipStream_t st);

hipError_t launch_pack(const uint8_t* q, uint32_t* packed, int64_t rows,
                       int64_t k, int bits, hipStream_t st);

// Packed layouts (the values of bs_layout).
constexpr int kLayoutMBK = 0, kLayoutMKB = 1, kLayoutBMK = 2;

// q viewed as [outer][k][inner], packed along k into the given layout with
// rows o * inner + i.
hipError_t launch_pack_ex(const uint8_t* q, uint32_t* packed, int64_t outer,
                          int64_t k, int64_t inner, int bits, int layout,
                          hipStream_t st);

hipError_t launch_quantize_pack(const float* x, uint32_t* packed,
                                int64_t rows, int64_t k, float scale, int bits,
                                int enc, hipStream_t st);

// Geometry of a convolution as the kernels see it; dense is the 1x1 case
// with n = 1, h = 1, w = m.
struct ConvShape {
    int32_t n, h, w, c, oc, kh, kw, sh, sw, ph, pw, oh, ow;
    int32_t abits, wbits;
    int32_t aenc, wenc;   // kUnipolar, kBipolar, kSigned
    bool bipolar_w;       // wenc == kBipolar
};

// Kernel selection for a conv call.  mode 0: the fastest applicable kernel;
// 1: generic only; 2: the channels-on-lanes kernel where it applies; 3: the
// pixels-on-lanes kernel where it applies (2 and 3 fall back to the generic
// kernel).  units_per_wave > 0 overrides the run length the host would pick
// for the pixels-on-lanes kernel (units of 64 pixels x 4 output channels).
struct ConvOptions {
    int mode = 0;
    int units_per_wave = 0;
};

hipError_t launch_conv(const ConvShape& s, const uint32_t* act,
                       const uint32_t* wts, int32_t* out,
                       const ConvOptions& opt, hipStream_t st);

// Requantized output of a conv: codes of out_bits bits (quant_code of the
// int32 result converted to float32, times out_scale), bit-packed along the
// output channels as [n][oh][ow][out_bits][ceil(oc / 32)] uint32 words.
struct Requant {
    float scale;
    int bits;       // 1..8
};

hipError_t launch_conv_requant(const ConvShape& s, const uint32_t* act,
                               const uint32_t* wts, uint32_t* out,
                               const Requant& rq, const ConvOptions& opt,
                               hipStream_t st);

// A KxK conv s (odd K, pad (K-1)/2) and the 1x1 conv of the same stride
// over the same input, whose input pixel is the window's centre tap, so that
// both share the output grid: wts1 [oc][1][1][wbits][cw] filters, out1
// shaped like out.  rq: both outputs requantized and packed (scale1 for
// out1) instead of int32.  One paired launch where a kernel covers the
// shape, otherwise the two convolutions one after the other.
hipError_t launch_conv_pair(const ConvShape& s, const uint32_t* act,
                            const uint32_t* wts, const uint32_t* wts1,
                            int32_t* out, int32_t* out1, const Requant* rq,
                            float scale1, const ConvOptions& opt,
                            hipStream_t st);

// Conv of unpacked uint8 activation codes, NHWC [n][h][w][c]: the conv
// kernel bit-packs each block's input rows into LDS.  hipErrorNotSupported,
// with nothing enqueued, when no such kernel covers the shape.
hipError_t launch_conv_codes(const ConvShape& s, const uint8_t* act,
                             const uint32_t* wts, int32_t* out,
                             const ConvOptions& opt, hipStream_t st);

// Conv of float32 activations, NHWC [n][h][w][c], quantized (unipolar,
// scale) and bit-packed into each block's LDS by the conv kernel (1x1
// windows).  hipErrorNotSupported, with nothing enqueued, when no such
// kernel covers the shape.
hipError_t launch_conv_quantized(const ConvShape& s, const float* act,
                                 float scale, const uint32_t* wts,
                                 int32_t* out, const ConvOptions& opt,
                                 hipStream_t st);

// Writes the kernel and launch configuration launch_conv would use for this
// shape and mode into buf (snprintf semantics); returns the snprintf result.
int describe_conv(const ConvShape& s, const ConvOptions& opt, char* buf,
                  size_t len);

// The same for launch_conv_codes (from_float false) or
// launch_conv_quantized (true): the staged plan; -1, with buf untouched,
// where the launch would return hipErrorNotSupported.
int describe_conv_staged(const ConvShape& s, bool from_float,
                         const ConvOptions& opt, char* buf, size_t len);

// True when launch_conv with mode 0 would use a specialised kernel.
bool conv_has_fast_path(const ConvShape& s);

}  // namespace bs
