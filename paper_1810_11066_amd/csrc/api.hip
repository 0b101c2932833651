// extern "C" entry points of libbitserial.so (declared in include/bitserial.h):
// argument validation, the int32 overflow guard, and dispatch to the kernels.
// Every check runs on the host before anything is enqueued, so an invalid
// call never touches device memory.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "bitserial.h"
#include "bs_internal.h"

namespace {

thread_local char g_err[512];
thread_local bs::ConvOptions g_conv_opt;
thread_local bs::TimingEvents g_timing;

bs_status fail(bs_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return st;
}

bs_status ok() {
    g_err[0] = '\0';
    return BS_OK;
}

bs_status from_hip(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(BS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bs_status check_ptr(const void* p, const char* name) {
    if (!p) return fail(BS_ERR_INVALID_ARG, "%s is NULL", name);
    if (!aligned16(p))
        return fail(BS_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
    return BS_OK;
}

// An output must not share a byte with an input: the kernels read inputs
// while other waves write outputs, in no fixed order.  Inputs may alias each
// other (a product of a matrix with itself).  Sizes in bytes; empty ranges
// never overlap.
bs_status check_disjoint(const void* out, uint64_t out_bytes, const char* oname,
                         const void* in, uint64_t in_bytes, const char* iname) {
    const uintptr_t o = (uintptr_t)out, i = (uintptr_t)in;
    if (out_bytes > 0 && in_bytes > 0 && o < i + in_bytes &&
        i < o + out_bytes)
        return fail(BS_ERR_INVALID_ARG, "%s overlaps %s", oname, iname);
    return BS_OK;
}

uint64_t packed_bytes(int64_t rows, int bits, int64_t k) {
    return (uint64_t)rows * (uint64_t)bits * (uint64_t)((k + 31) / 32) * 4u;
}

// The operands of a conv call must not overlap its output.
bs_status check_conv_buffers(const bs::ConvShape& s, const void* act,
                             const void* wts, const void* out,
                             uint64_t out_bytes) {
    const uint64_t cw = (uint64_t)((s.c + 31) / 32);
    const uint64_t act_bytes =
        (uint64_t)s.n * s.h * s.w * (uint64_t)s.abits * cw * 4u;
    const uint64_t w_bytes =
        (uint64_t)s.oc * s.kh * s.kw * (uint64_t)s.wbits * cw * 4u;
    bs_status st;
    if ((st = check_disjoint(out, out_bytes, "out", act, act_bytes,
                             "act_packed")) != BS_OK)
        return st;
    return check_disjoint(out, out_bytes, "out", wts, w_bytes, "w_packed");
}

bs_status check_bits(int bits, const char* name) {
    if (bits < 1 || bits > 8)
        return fail(BS_ERR_INVALID_ARG, "%s = %d is outside 1..8", name, bits);
    return BS_OK;
}

// An encoding of conv/dense operands: signed (two's complement) data needs a
// sign plane and at least one magnitude plane.
bs_status check_enc(int enc, int bits, const char* name) {
    if (enc != BS_UNIPOLAR && enc != BS_BIPOLAR && enc != BS_SIGNED)
        return fail(BS_ERR_INVALID_ARG, "unknown %s encoding %d", name, enc);
    if (enc == BS_SIGNED && bits < 2)
        return fail(BS_ERR_INVALID_ARG, "signed %s need >= 2 bits", name);
    return BS_OK;
}

bs_status check_scale_enc(float scale, int bits, bs_encoding enc) {
    if (!isfinite(scale) || !(scale > 0.0f))
        return fail(BS_ERR_INVALID_ARG, "scale must be finite and > 0");
    bs_status st;
    if ((st = check_enc((int)enc, bits, "quantization")) != BS_OK) return st;
    if (enc == BS_BIPOLAR && bits != 1)
        return fail(BS_ERR_INVALID_ARG,
                    "bipolar quantization is 1-bit (bits = %d)", bits);
    return BS_OK;
}

// Largest magnitude a value of `bits` bits takes under an encoding:
// unipolar 2^bits - 1, bipolar |2u - (2^bits - 1)| <= 2^bits - 1, signed
// 2^(bits-1) (the most negative value).
uint64_t max_abs(int enc, int bits) {
    return enc == BS_SIGNED ? (1ull << (bits - 1)) : (1ull << bits) - 1;
}

// max|a| * max|w| * taps * c must fit int32 for the exact result to.
bs_status check_overflow(int abits, int aenc, int wbits, int wenc,
                         int64_t taps, int64_t c) {
    unsigned __int128 bound = (unsigned __int128)max_abs(aenc, abits) *
                              max_abs(wenc, wbits) * (uint64_t)taps *
                              (uint64_t)c;
    if (bound > (unsigned __int128)INT32_MAX)
        return fail(BS_ERR_OVERFLOW,
                    "%llu*%llu*%lld*%lld exceeds int32",
                    (unsigned long long)max_abs(aenc, abits),
                    (unsigned long long)max_abs(wenc, wbits),
                    (long long)taps, (long long)c);
    return BS_OK;
}

// Shape checks shared by bs_conv2d and bs_dense; fills the kernel geometry.
bs_status check_conv(const bs_conv2d_params* p, bs::ConvShape* s) {
    if (!p) return fail(BS_ERR_INVALID_ARG, "params is NULL");
    if (p->n < 1 || p->h < 1 || p->w < 1 || p->c < 1 || p->oc < 1 ||
        p->kh < 1 || p->kw < 1)
        return fail(BS_ERR_INVALID_ARG, "sizes must be >= 1");
    if (p->stride_h < 1 || p->stride_w < 1)
        return fail(BS_ERR_INVALID_ARG, "stride must be >= 1");
    if (p->pad_h < 0 || p->pad_w < 0)
        return fail(BS_ERR_INVALID_ARG, "padding must be >= 0");
    bs_status st;
    if ((st = check_bits(p->abits, "abits")) != BS_OK) return st;
    if ((st = check_bits(p->wbits, "wbits")) != BS_OK) return st;
    if ((st = check_enc(p->aenc, p->abits, "activation")) != BS_OK) return st;
    if ((st = check_enc(p->wenc, p->wbits, "weight")) != BS_OK) return st;
    const int64_t eh = (int64_t)p->h + 2 * (int64_t)p->pad_h - p->kh;
    const int64_t ew = (int64_t)p->w + 2 * (int64_t)p->pad_w - p->kw;
    if (eh < 0 || ew < 0)
        return fail(BS_ERR_INVALID_ARG, "kernel larger than padded input");
    if ((st = check_overflow(p->abits, p->aenc, p->wbits, p->wenc,
                             (int64_t)p->kh * p->kw, p->c)) != BS_OK)
        return st;
    const int64_t oh = eh / p->stride_h + 1, ow = ew / p->stride_w + 1;
    const int64_t pixels = (int64_t)p->n * oh * ow;
    const int64_t cw = ((int64_t)p->c + 31) / 32;
    if (pixels * p->oc > INT32_MAX)
        return fail(BS_ERR_UNSUPPORTED, "output has more than 2^31-1 elements");
    if ((int64_t)p->n * p->h * p->w * p->abits * cw > ((int64_t)1 << 40) ||
        (int64_t)p->oc * p->kh * p->kw * p->wbits * cw > INT32_MAX)
        return fail(BS_ERR_UNSUPPORTED, "packed operand too large");
    s->n = p->n; s->h = p->h; s->w = p->w; s->c = p->c; s->oc = p->oc;
    s->kh = p->kh; s->kw = p->kw; s->sh = p->stride_h; s->sw = p->stride_w;
    s->ph = p->pad_h; s->pw = p->pad_w;
    s->oh = (int32_t)oh; s->ow = (int32_t)ow;
    s->abits = p->abits; s->wbits = p->wbits;
    s->aenc = p->aenc; s->wenc = p->wenc;
    s->bipolar_w = p->wenc == BS_BIPOLAR;
    return BS_OK;
}

}  // namespace

namespace bs {

TimingEvents& timing_events() { return g_timing; }

hipError_t launch_kernel(const void* fn, dim3 grid, dim3 block, void** args,
                         size_t lds, hipStream_t st) {
    TimingEvents& t = g_timing;
    if (t.start || t.stop) {
        const hipError_t e = hipExtLaunchKernel(fn, grid, block, args, lds, st,
                                                t.start, t.stop, 0);
        // the start event belongs to the first dispatch only; the stop
        // event to every one, so the last stamps it
        t.start = nullptr;
        return e;
    }
    return hipLaunchKernel(fn, grid, block, args, lds, st);
}

}  // namespace bs

extern "C" {

int bs_abi_version(void) { return 109; }

int64_t bs_packed_words(int64_t k) { return k <= 0 ? 0 : (k + 31) / 32; }

const char* bs_status_string(bs_status s) {
    switch (s) {
        case BS_OK: return "ok";
        case BS_ERR_INVALID_ARG: return "invalid argument";
        case BS_ERR_UNSUPPORTED: return "unsupported";
        case BS_ERR_OVERFLOW: return "int32 overflow possible";
        case BS_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

const char* bs_last_error(void) { return g_err; }

bs_status bs_set_kernel_mode(int mode) {
    if (mode < 0 || mode > 3)
        return fail(BS_ERR_INVALID_ARG, "kernel mode must be 0..3");
    g_conv_opt.mode = mode;
    return ok();
}

bs_status bs_set_units_per_wave(int units) {
    if (units < 0) return fail(BS_ERR_INVALID_ARG, "units per wave must be >= 0");
    g_conv_opt.units_per_wave = units;
    return ok();
}

bs_status bs_set_timing_events(void* start, void* stop) {
    g_timing.start = (hipEvent_t)start;
    g_timing.stop = (hipEvent_t)stop;
    return ok();
}

bs_status bs_quantize(const float* x, uint8_t* q, int64_t n, float scale,
                      int bits, bs_encoding enc, bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(x, "x")) != BS_OK) return st;
    if ((st = check_ptr(q, "q")) != BS_OK) return st;
    if (n < 0) return fail(BS_ERR_INVALID_ARG, "n < 0");
    if ((st = check_bits(bits, "bits")) != BS_OK) return st;
    if ((st = check_scale_enc(scale, bits, enc)) != BS_OK) return st;
    if (n == 0) return ok();
    if ((st = check_disjoint(q, (uint64_t)n, "q", x, (uint64_t)n * 4u,
                             "x")) != BS_OK)
        return st;
    return from_hip(bs::launch_quantize(x, q, n, scale, bits, (int)enc,
                                        (hipStream_t)stream),
                    "bs_quantize launch");
}

bs_status bs_pack(const uint8_t* q, uint32_t* packed, int64_t rows, int64_t k,
                  int bits, bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(q, "q")) != BS_OK) return st;
    if ((st = check_ptr(packed, "packed")) != BS_OK) return st;
    if (rows < 0) return fail(BS_ERR_INVALID_ARG, "rows < 0");
    if (k < 1) return fail(BS_ERR_INVALID_ARG, "k < 1");
    if ((st = check_bits(bits, "bits")) != BS_OK) return st;
    if (rows > ((int64_t)1 << 40) / k)
        return fail(BS_ERR_UNSUPPORTED, "tensor too large");
    if (rows == 0) return ok();
    if ((st = check_disjoint(packed, packed_bytes(rows, bits, k), "packed", q,
                             (uint64_t)rows * (uint64_t)k, "q")) != BS_OK)
        return st;
    return from_hip(bs::launch_pack(q, packed, rows, k, bits,
                                    (hipStream_t)stream),
                    "bs_pack launch");
}

bs_status bs_pack_ex(const uint8_t* q, uint32_t* packed, int64_t outer,
                     int64_t k, int64_t inner, int bits, bs_layout layout,
                     bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(q, "q")) != BS_OK) return st;
    if ((st = check_ptr(packed, "packed")) != BS_OK) return st;
    if (outer < 0) return fail(BS_ERR_INVALID_ARG, "outer < 0");
    if (k < 1) return fail(BS_ERR_INVALID_ARG, "k < 1");
    if (inner < 1) return fail(BS_ERR_INVALID_ARG, "inner < 1");
    if ((st = check_bits(bits, "bits")) != BS_OK) return st;
    if (layout != BS_LAYOUT_MBK && layout != BS_LAYOUT_MKB &&
        layout != BS_LAYOUT_BMK)
        return fail(BS_ERR_INVALID_ARG, "unknown layout %d", (int)layout);
    if (k > ((int64_t)1 << 40) || inner > ((int64_t)1 << 40) / k ||
        outer > ((int64_t)1 << 40) / (k * inner))
        return fail(BS_ERR_UNSUPPORTED, "tensor too large");
    if (outer == 0) return ok();
    if ((st = check_disjoint(packed, packed_bytes(outer * inner, bits, k),
                             "packed", q,
                             (uint64_t)outer * (uint64_t)k * (uint64_t)inner,
                             "q")) != BS_OK)
        return st;
    return from_hip(bs::launch_pack_ex(q, packed, outer, k, inner, bits,
                                       (int)layout, (hipStream_t)stream),
                    "bs_pack_ex launch");
}

bs_status bs_quantize_pack(const float* x, uint32_t* packed, int64_t rows,
                           int64_t k, float scale, int bits, bs_encoding enc,
                           bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(x, "x")) != BS_OK) return st;
    if ((st = check_ptr(packed, "packed")) != BS_OK) return st;
    if (rows < 0) return fail(BS_ERR_INVALID_ARG, "rows < 0");
    if (k < 1) return fail(BS_ERR_INVALID_ARG, "k < 1");
    if ((st = check_bits(bits, "bits")) != BS_OK) return st;
    if ((st = check_scale_enc(scale, bits, enc)) != BS_OK) return st;
    if (rows > ((int64_t)1 << 40) / k)
        return fail(BS_ERR_UNSUPPORTED, "tensor too large");
    if (rows == 0) return ok();
    if ((st = check_disjoint(packed, packed_bytes(rows, bits, k), "packed", x,
                             (uint64_t)rows * (uint64_t)k * 4u, "x")) != BS_OK)
        return st;
    return from_hip(bs::launch_quantize_pack(x, packed, rows, k, scale, bits,
                                             (int)enc, (hipStream_t)stream),
                    "bs_quantize_pack launch");
}

bs_status bs_conv2d_out_shape(const bs_conv2d_params* p, int32_t* oh,
                              int32_t* ow) {
    if (!p || !oh || !ow) return fail(BS_ERR_INVALID_ARG, "NULL argument");
    if (p->kh < 1 || p->kw < 1 || p->stride_h < 1 || p->stride_w < 1 ||
        p->pad_h < 0 || p->pad_w < 0 || p->h < 1 || p->w < 1)
        return fail(BS_ERR_INVALID_ARG, "invalid geometry");
    const int64_t eh = (int64_t)p->h + 2 * (int64_t)p->pad_h - p->kh;
    const int64_t ew = (int64_t)p->w + 2 * (int64_t)p->pad_w - p->kw;
    if (eh < 0 || ew < 0)
        return fail(BS_ERR_INVALID_ARG, "kernel larger than padded input");
    *oh = (int32_t)(eh / p->stride_h + 1);
    *ow = (int32_t)(ew / p->stride_w + 1);
    return ok();
}

bs_status bs_conv2d(const bs_conv2d_params* p, const uint32_t* act_packed,
                    const uint32_t* w_packed, int32_t* out,
                    bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act_packed, "act_packed")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(out, "out")) != BS_OK) return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if ((st = check_conv_buffers(
             s, act_packed, w_packed, out,
             (uint64_t)s.n * s.oh * s.ow * (uint64_t)s.oc * 4u)) != BS_OK)
        return st;
    return from_hip(bs::launch_conv(s, act_packed, w_packed, out,
                                    g_conv_opt, (hipStream_t)stream),
                    "bs_conv2d launch");
}

// The checks of a paired call beyond bs_conv2d's: the 1x1 conv's input pixel
// must be the window's centre tap (square odd window, pad (K-1)/2, equal
// strides), and no output may overlap an input or the other output.
static bs_status check_pair(const bs_conv2d_params* p,
                            const bs::ConvShape& s, const void* act,
                            const void* wts, const void* wts1,
                            const void* out, const void* out1,
                            uint64_t out_bytes) {
    if (p->kh != p->kw || p->kh % 2 == 0 || p->pad_h != (p->kh - 1) / 2 ||
        p->pad_w != (p->kw - 1) / 2 || p->stride_h != p->stride_w)
        return fail(BS_ERR_INVALID_ARG,
                    "the paired 1x1 conv reads the window's centre tap: it "
                    "needs kh == kw odd, pad (kh - 1) / 2 on both axes and "
                    "equal strides");
    bs_status st;
    if ((st = check_conv_buffers(s, act, wts, out, out_bytes)) != BS_OK)
        return st;
    if ((st = check_conv_buffers(s, act, wts, out1, out_bytes)) != BS_OK)
        return st;
    const uint64_t w1_bytes = packed_bytes(s.oc, s.wbits, s.c);
    if ((st = check_disjoint(out, out_bytes, "out", wts1, w1_bytes,
                             "w1_packed")) != BS_OK)
        return st;
    if ((st = check_disjoint(out1, out_bytes, "out1", wts1, w1_bytes,
                             "w1_packed")) != BS_OK)
        return st;
    return check_disjoint(out1, out_bytes, "out1", out, out_bytes, "out");
}

bs_status bs_conv2d_pair(const bs_conv2d_params* p, const uint32_t* act_packed,
                         const uint32_t* w_packed, const uint32_t* w1_packed,
                         int32_t* out, int32_t* out1, bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act_packed, "act_packed")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(w1_packed, "w1_packed")) != BS_OK) return st;
    if ((st = check_ptr(out, "out")) != BS_OK) return st;
    if ((st = check_ptr(out1, "out1")) != BS_OK) return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if ((st = check_pair(p, s, act_packed, w_packed, w1_packed, out, out1,
                         (uint64_t)s.n * s.oh * s.ow * (uint64_t)s.oc * 4u)) !=
        BS_OK)
        return st;
    return from_hip(bs::launch_conv_pair(s, act_packed, w_packed, w1_packed,
                                         out, out1, nullptr, 0.0f, g_conv_opt,
                                         (hipStream_t)stream),
                    "bs_conv2d_pair launch");
}

bs_status bs_conv2d_pair_requant(const bs_conv2d_params* p,
                                 const uint32_t* act_packed,
                                 const uint32_t* w_packed,
                                 const uint32_t* w1_packed, float out_scale,
                                 float out1_scale, int out_bits,
                                 uint32_t* out_packed, uint32_t* out1_packed,
                                 bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act_packed, "act_packed")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(w1_packed, "w1_packed")) != BS_OK) return st;
    if ((st = check_ptr(out_packed, "out_packed")) != BS_OK) return st;
    if ((st = check_ptr(out1_packed, "out1_packed")) != BS_OK) return st;
    if ((st = check_bits(out_bits, "out_bits")) != BS_OK) return st;
    if ((st = check_scale_enc(out_scale, out_bits, BS_UNIPOLAR)) != BS_OK)
        return st;
    if ((st = check_scale_enc(out1_scale, out_bits, BS_UNIPOLAR)) != BS_OK)
        return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if ((int64_t)s.n * s.oh * s.ow * ((s.oc + 31) / 32) >= INT32_MAX)
        return fail(BS_ERR_UNSUPPORTED, "output too large");
    if ((st = check_pair(p, s, act_packed, w_packed, w1_packed, out_packed,
                         out1_packed,
                         packed_bytes((int64_t)s.n * s.oh * s.ow, out_bits,
                                      s.oc))) != BS_OK)
        return st;
    bs::Requant rq;
    rq.scale = out_scale;
    rq.bits = out_bits;
    return from_hip(bs::launch_conv_pair(
                        s, act_packed, w_packed, w1_packed,
                        reinterpret_cast<int32_t*>(out_packed),
                        reinterpret_cast<int32_t*>(out1_packed), &rq,
                        out1_scale, g_conv_opt, (hipStream_t)stream),
                    "bs_conv2d_pair_requant launch");
}

// Why bs_conv2d_codes refuses a shape.
const char* const kNoFusedKernel =
    "no fused kernel covers this shape (it needs c = 32 times a power of "
    "two (at most 512 for 3x3 windows, 4096 for 1x1 ones), oc a multiple of "
    "4, square kernels of size 1 or 3, stride 1 or 2, unipolar activations "
    "of 1-4 bits with unipolar filters of 1-4 bits or bipolar 1-bit "
    "filters, and the input rows of one workgroup's outputs within its "
    "LDS); bit-pack the activations and call bs_conv2d";

// bs_pack of the codes fused into bs_conv2d: validation as bs_conv2d, with
// the codes' bytes in the overlap check.
bs_status bs_conv2d_codes(const bs_conv2d_params* p, const uint8_t* act_codes,
                          const uint32_t* w_packed, int32_t* out,
                          bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act_codes, "act_codes")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(out, "out")) != BS_OK) return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    const uint64_t out_bytes = (uint64_t)s.n * s.oh * s.ow * (uint64_t)s.oc * 4u;
    const uint64_t act_bytes = (uint64_t)s.n * s.h * s.w * (uint64_t)s.c;
    const uint64_t w_bytes = packed_bytes((int64_t)s.oc * s.kh * s.kw,
                                          s.wbits, s.c);
    if ((st = check_disjoint(out, out_bytes, "out", act_codes, act_bytes,
                             "act_codes")) != BS_OK)
        return st;
    if ((st = check_disjoint(out, out_bytes, "out", w_packed, w_bytes,
                             "w_packed")) != BS_OK)
        return st;
    const hipError_t e = bs::launch_conv_codes(s, act_codes, w_packed, out,
                                               g_conv_opt, (hipStream_t)stream);
    if (e == hipErrorNotSupported)
        return fail(BS_ERR_UNSUPPORTED, "bs_conv2d_codes: %s", kNoFusedKernel);
    return from_hip(e, "bs_conv2d_codes launch");
}

// Why bs_conv2d_quantized refuses a shape.
const char* const kNoQuantizedKernel =
    "no fused kernel covers this shape (it needs a 1x1 window, stride 1 or "
    "2, c = 32 times a power of two up to 4096, oc a multiple of 4, "
    "unipolar activations of 1-4 bits with unipolar filters of 1-4 bits or "
    "bipolar 1-bit filters, and one workgroup's input pixels within its "
    "LDS); quantize and bit-pack the activations (bs_quantize_pack) and call "
    "bs_conv2d";

// bs_quantize_pack of float32 activations fused into bs_conv2d: validation
// as bs_conv2d and bs_quantize_pack (unipolar), with the float32 bytes in
// the overlap check.
bs_status bs_conv2d_quantized(const bs_conv2d_params* p, const float* act,
                              float act_scale, const uint32_t* w_packed,
                              int32_t* out, bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act, "act")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(out, "out")) != BS_OK) return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if (p->aenc != BS_UNIPOLAR)
        return fail(BS_ERR_UNSUPPORTED,
                    "bs_conv2d_quantized: unipolar activations only");
    if ((st = check_scale_enc(act_scale, p->abits, BS_UNIPOLAR)) != BS_OK)
        return st;
    const uint64_t out_bytes = (uint64_t)s.n * s.oh * s.ow * (uint64_t)s.oc * 4u;
    const uint64_t act_bytes =
        (uint64_t)s.n * s.h * s.w * (uint64_t)s.c * 4u;
    const uint64_t w_bytes = packed_bytes((int64_t)s.oc * s.kh * s.kw,
                                          s.wbits, s.c);
    if ((st = check_disjoint(out, out_bytes, "out", act, act_bytes, "act")) !=
        BS_OK)
        return st;
    if ((st = check_disjoint(out, out_bytes, "out", w_packed, w_bytes,
                             "w_packed")) != BS_OK)
        return st;
    const hipError_t e = bs::launch_conv_quantized(
        s, act, act_scale, w_packed, out, g_conv_opt, (hipStream_t)stream);
    if (e == hipErrorNotSupported)
        return fail(BS_ERR_UNSUPPORTED, "bs_conv2d_quantized: %s",
                    kNoQuantizedKernel);
    return from_hip(e, "bs_conv2d_quantized launch");
}

bs_status bs_conv2d_requant(const bs_conv2d_params* p,
                            const uint32_t* act_packed,
                            const uint32_t* w_packed, float out_scale,
                            int out_bits, uint32_t* out_packed,
                            bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(act_packed, "act_packed")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(out_packed, "out_packed")) != BS_OK) return st;
    if ((st = check_bits(out_bits, "out_bits")) != BS_OK) return st;
    if ((st = check_scale_enc(out_scale, out_bits, BS_UNIPOLAR)) != BS_OK)
        return st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if ((int64_t)s.n * s.oh * s.ow * ((s.oc + 31) / 32) >= INT32_MAX)
        return fail(BS_ERR_UNSUPPORTED, "output too large");
    if ((st = check_conv_buffers(
             s, act_packed, w_packed, out_packed,
             packed_bytes((int64_t)s.n * s.oh * s.ow, out_bits, s.oc))) !=
        BS_OK)
        return st;
    bs::Requant rq;
    rq.scale = out_scale;
    rq.bits = out_bits;
    return from_hip(bs::launch_conv_requant(s, act_packed, w_packed,
                                            out_packed, rq, g_conv_opt,
                                            (hipStream_t)stream),
                    "bs_conv2d_requant launch");
}

bs_status bs_conv2d_describe(const bs_conv2d_params* p, char* buf,
                             int32_t len) {
    if (!buf || len < 1) return fail(BS_ERR_INVALID_ARG, "buf/len");
    buf[0] = '\0';
    bs_status st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    bs::describe_conv(s, g_conv_opt, buf, (size_t)len);
    return ok();
}

bs_status bs_conv2d_codes_describe(const bs_conv2d_params* p, char* buf,
                                   int32_t len) {
    if (!buf || len < 1) return fail(BS_ERR_INVALID_ARG, "buf/len");
    buf[0] = '\0';
    bs_status st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if (bs::describe_conv_staged(s, false, g_conv_opt, buf, (size_t)len) <
        0) {
        buf[0] = '\0';
        return fail(BS_ERR_UNSUPPORTED, "bs_conv2d_codes: %s",
                    kNoFusedKernel);
    }
    return ok();
}

bs_status bs_conv2d_quantized_describe(const bs_conv2d_params* p, char* buf,
                                       int32_t len) {
    if (!buf || len < 1) return fail(BS_ERR_INVALID_ARG, "buf/len");
    buf[0] = '\0';
    bs_status st;
    bs::ConvShape s;
    if ((st = check_conv(p, &s)) != BS_OK) return st;
    if (p->aenc != BS_UNIPOLAR)
        return fail(BS_ERR_UNSUPPORTED,
                    "bs_conv2d_quantized: unipolar activations only");
    if (bs::describe_conv_staged(s, true, g_conv_opt, buf, (size_t)len) < 0) {
        buf[0] = '\0';
        return fail(BS_ERR_UNSUPPORTED, "bs_conv2d_quantized: %s",
                    kNoQuantizedKernel);
    }
    return ok();
}

bs_status bs_dense_ex(int64_t m, int64_t n, int64_t k, int abits,
                      bs_encoding aenc, int wbits, bs_encoding wenc,
                      const uint32_t* a_packed, const uint32_t* w_packed,
                      int32_t* out, bs_stream_t stream) {
    bs_status st;
    if ((st = check_ptr(a_packed, "a_packed")) != BS_OK) return st;
    if ((st = check_ptr(w_packed, "w_packed")) != BS_OK) return st;
    if ((st = check_ptr(out, "out")) != BS_OK) return st;
    if (m < 1 || n < 1 || k < 1)
        return fail(BS_ERR_INVALID_ARG, "m, n, k must be >= 1");
    if (m > INT32_MAX || n > INT32_MAX || k > INT32_MAX)
        return fail(BS_ERR_UNSUPPORTED, "dimension beyond int32");
    // dense == 1x1 convolution over an m-pixel image
    bs_conv2d_params p;
    p.n = 1; p.h = 1; p.w = (int32_t)m; p.c = (int32_t)k; p.oc = (int32_t)n;
    p.kh = 1; p.kw = 1; p.stride_h = 1; p.stride_w = 1; p.pad_h = 0;
    p.pad_w = 0; p.abits = abits; p.wbits = wbits; p.aenc = aenc;
    p.wenc = wenc;
    bs::ConvShape s;
    if ((st = check_conv(&p, &s)) != BS_OK) return st;
    if ((st = check_conv_buffers(s, a_packed, w_packed, out,
                                 (uint64_t)m * (uint64_t)n * 4u)) != BS_OK)
        return st;
    return from_hip(bs::launch_conv(s, a_packed, w_packed, out, g_conv_opt,
                                    (hipStream_t)stream),
                    "bs_dense launch");
}

bs_status bs_dense(int64_t m, int64_t n, int64_t k, int abits, int wbits,
                   bs_encoding wenc, const uint32_t* a_packed,
                   const uint32_t* w_packed, int32_t* out, bs_stream_t stream) {
    return bs_dense_ex(m, n, k, abits, BS_UNIPOLAR, wbits, wenc, a_packed,
                       w_packed, out, stream);
}

}  // extern "C"
