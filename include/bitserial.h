/*
 * bitserial.h -- C ABI of libbitserial.so: low-precision bitserial operators
 * (quantize, bit-pack, bitserial conv2d and dense) for AMD MI355X (gfx950).
 *
 * Method: "Automating Generation of Low Precision Deep Learning Operators"
 * (Cowan, Moreau, Chen, Ceze).  A B-bit tensor is split into B bit-planes,
 * each plane packed into uint32 words along the reduction axis (Sec. 2.2,
 * Sec. 3.1); a dot product of an A-bit and a W-bit vector is then
 *   sum_{i<A} sum_{j<W} 2^(i+j) popcount(a_i AND w_j)            (Eq. 1, Eq. 2)
 * and, for weights in the bipolar (+1/-1) format, each AND term becomes
 *   popcount(a_i AND w_j) - popcount(a_i AND NOT w_j).
 *
 * Conventions shared by every entry point:
 *  - Data pointers are DEVICE pointers (HBM) owned by the caller; the library
 *    never allocates, frees or keeps them.  Every base pointer must be
 *    16-byte aligned (all torch / hipMalloc allocations are).
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = null stream).
 *    A returned BS_OK means the work was enqueued.  Faults inside a kernel
 *    surface at the caller's next synchronisation of that stream.
 *  - Arguments are validated on the host before anything is enqueued; an
 *    invalid call returns its status and enqueues nothing, so no output byte
 *    is written.  bs_last_error() then describes the problem.
 *  - An empty problem (n == 0 or rows == 0) is valid and enqueues nothing.
 *  - An output must not share a byte with an input (inputs may alias each
 *    other, e.g. one packed matrix as both operands of bs_dense): a call
 *    whose output range, as its sizes define it, overlaps an input's returns
 *    BS_ERR_INVALID_ARG.
 *  - Results are exact integers and do not depend on launch configuration;
 *    no kernel uses atomics, so repeated calls are bit-identical.
 *  - Thread safety: calls from several host threads are safe; the only
 *    library state is per thread (the error string, the kernel mode, the
 *    run-length override and the timing events).
 *  - Concurrency: calls on different streams may run on the GPU at the same
 *    time.  A call touches device memory only through its own inputs and
 *    outputs, so concurrent calls are independent unless one writes what
 *    another reads or writes; order those on one stream or with events.
 *    Independent batches spread over two streams let one call's kernel fill
 *    the GPU while the previous one drains.
 */
#ifndef BITSERIAL_H
#define BITSERIAL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BS_OK = 0,
    BS_ERR_INVALID_ARG = 1, /* NULL/misaligned pointer, bad size or bit-width */
    BS_ERR_UNSUPPORTED = 2, /* valid request this library does not implement */
    BS_ERR_OVERFLOW = 3,    /* the exact result could exceed int32 */
    BS_ERR_HIP = 4          /* the HIP runtime refused the launch */
} bs_status;

/* Encoding of the codes (Sec. 2.2), with b_j the bit of plane j of a B-bit code:
 *   BS_UNIPOLAR  value sum_j 2^j b_j;
 *   BS_BIPOLAR   value sum_j 2^j (2 b_j - 1): a 1-bit plane stands for +1
 *                (bit 1) or -1 (bit 0), the form whose products the paper
 *                computes with XNOR;
 *   BS_SIGNED    two's complement (B >= 2): the top plane weighs -2^(B-1),
 *                i.e. every binary dot product is weighted by the sign of its
 *                planes. */
typedef enum { BS_UNIPOLAR = 0, BS_BIPOLAR = 1, BS_SIGNED = 2 } bs_encoding;

/* Position of the bit axis B in a packed tensor of rows M and packed
 * reduction axis K' (Sec. 3.1, bitpacking operator): */
typedef enum {
    BS_LAYOUT_MBK = 0,   /* [rows][bits][words]  (what conv and dense read) */
    BS_LAYOUT_MKB = 1,   /* [rows][words][bits]  (bits innermost) */
    BS_LAYOUT_BMK = 2    /* [bits][rows][words]  (bits outermost) */
} bs_layout;

/* A hipStream_t, kept opaque so this header does not need HIP headers. */
typedef void *bs_stream_t;

/* Number of uint32 words one bit-plane of k elements packs into: ceil(k/32). */
int64_t bs_packed_words(int64_t k);

/* Quantization of float data to `bits`-bit codes (Sec. 3.1; Sec. 1 lists the
 * quantization operator).  The paper gives no formula; this library fixes:
 *   unipolar: q = clamp(round_half_to_even(fl32(x * scale)), 0, 2^bits - 1),
 *             NaN -> 0, +inf -> 2^bits - 1, subnormals not flushed;
 *   bipolar (bits must be 1): q = 1 if x >= 0 (including -0.0) else 0, NaN -> 0.
 * x: [n] float32 (device), q: [n] uint8 (device).  scale: finite, > 0.
 * Errors: BS_ERR_INVALID_ARG for NULL/misaligned pointers, n < 0, bits outside
 * 1..8, bipolar with bits != 1, non-finite or non-positive scale. */
bs_status bs_quantize(const float *x, uint8_t *q, int64_t n, float scale,
                      int bits, bs_encoding enc, bs_stream_t stream);

/* Bit packing (Sec. 2.2 packing into a storage word; Sec. 3.1 bitpacking
 * operator with the bit axis placed between rows and the packed reduction
 * axis, layout MBK').
 * q: [rows][k] uint8 codes, row-major (device).
 * packed: [rows][bits][ceil(k/32)] uint32 (device), fully overwritten:
 *   bit u of word t of plane b of row r = bit b of q[r][32 t + u];
 *   bits for elements past k are 0; bits of q at or above `bits` are ignored.
 * Conv activations pack with rows = N*H*W, k = C; OHWI conv filters with
 * rows = OC*KH*KW, k = C; dense operands with rows = M (or N_out), k = K.
 * Errors: BS_ERR_INVALID_ARG for NULL/misaligned pointers, rows < 0, k < 1,
 * bits outside 1..8. */
bs_status bs_pack(const uint8_t *q, uint32_t *packed, int64_t rows, int64_t k,
                  int bits, bs_stream_t stream);

/* General bit packing (Sec. 3.1: the caller chooses the reduction axis and
 * where the bit axis goes).  q is viewed as [outer][k][inner] uint8 codes
 * (device): the reduction axis k has stride `inner`.  Packed row
 * r = o * inner + i holds the k codes q[o][.][i]; words and bits as in bs_pack,
 * in the given layout:
 *   BS_LAYOUT_MBK  packed[r][b][t]        (inner = 1: exactly bs_pack)
 *   BS_LAYOUT_MKB  packed[r][t][b]
 *   BS_LAYOUT_BMK  packed[b][r][t]        with t < ceil(k/32), b < bits.
 * NCHW activations packed with outer = n, k = c, inner = h*w give the packed
 * NHWC tensor bs_conv2d reads; OIHW filters (outer = oc, k = c,
 * inner = kh*kw) give the packed OHWI filters.  packed (device) is fully
 * overwritten, tail bits 0.
 * Errors: BS_ERR_INVALID_ARG for NULL/misaligned pointers, outer < 0, k < 1,
 * inner < 1, bits outside 1..8, an unknown layout; BS_ERR_UNSUPPORTED beyond
 * 2^40 codes. */
bs_status bs_pack_ex(const uint8_t *q, uint32_t *packed, int64_t outer,
                     int64_t k, int64_t inner, int bits, bs_layout layout,
                     bs_stream_t stream);

/* Fused quantize + pack: identical output to bs_quantize followed by bs_pack
 * on the same [rows][k] float32 tensor, without the uint8 intermediate.
 * Errors: as bs_quantize and bs_pack. */
bs_status bs_quantize_pack(const float *x, uint32_t *packed, int64_t rows,
                           int64_t k, float scale, int bits, bs_encoding enc,
                           bs_stream_t stream);

/* Bitserial 2-D convolution (Sec. 3.2; NHWC data, direct convolution without
 * an im2col copy).  Activations and filters each take any bs_encoding.
 *   act_packed: [n][h][w][abits][ceil(c/32)] uint32 (bs_pack of NHWC codes)
 *   w_packed:   [oc][kh][kw][wbits][ceil(c/32)] uint32 (bs_pack of OHWI codes)
 *   out:        [n][oh][ow][oc] int32, oh = (h + 2 pad_h - kh) / stride_h + 1,
 *               ow likewise; every element is written.
 *   out[n][y][x][o] = sum over in-range taps (r,s) and channels c of
 *     value(a) * value(w), the values of the codes under aenc and wenc:
 *     the integer convolution of the decoded tensors with zero padding (a
 *     padded position is 0, also for bipolar activations, so it contributes
 *     nothing).  Unipolar data is Eq. 2,
 *     sum_{i,j} 2^(i+j) sum_t popcount(a_i[t] AND w_j[t]); bipolar operands
 *     add popcount corrections (for +-1 data the sum over a tap's c channels
 *     is c - 2 popcount(a XOR w), the XNOR form); signed operands weight
 *     each plane pair by the sign of its planes.
 * Errors: BS_ERR_INVALID_ARG (NULL/misaligned pointers, non-positive sizes,
 * bit-widths outside 1..8, an unknown encoding, signed data with fewer than
 * 2 bits, stride < 1, pad < 0, oh or ow < 1); BS_ERR_UNSUPPORTED (sizes
 * beyond the 2^31 pixel / 2^31 word-index range); BS_ERR_OVERFLOW when
 * max|a| max|w| kh kw c > 2^31 - 1, with max|v| = 2^bits - 1 for unipolar
 * and bipolar codes and 2^(bits-1) for signed ones. */
typedef struct {
    int32_t n, h, w, c;       /* NHWC activations */
    int32_t oc, kh, kw;       /* OHWI filters: oc filters of kh x kw x c */
    int32_t stride_h, stride_w;
    int32_t pad_h, pad_w;
    int32_t abits, wbits;     /* 1..8 */
    int32_t aenc, wenc;       /* bs_encoding of activations and filters */
} bs_conv2d_params;

/* Output height/width of a conv; BS_ERR_INVALID_ARG if either would be < 1. */
bs_status bs_conv2d_out_shape(const bs_conv2d_params *p, int32_t *oh,
                              int32_t *ow);

bs_status bs_conv2d(const bs_conv2d_params *p, const uint32_t *act_packed,
                    const uint32_t *w_packed, int32_t *out,
                    bs_stream_t stream);

/* Bitserial conv2d of unpacked activation codes: the activation pack of
 * Sec. 3.1 fused into the conv.  Exactly bs_pack of act_codes followed by
 * bs_conv2d (the paper times the activation pack with the conv; here it is
 * part of the conv kernel): every workgroup bit-packs the input rows its
 * outputs read into LDS and convolves from there, so the packed activations
 * never reach HBM.
 *   act_codes: [n][h][w][c] uint8 NHWC codes (device); bits of a code at or
 *              above abits are ignored, as in bs_pack;
 *   w_packed, out and the result: as bs_conv2d.
 * p->aenc is the encoding of the codes.
 * Errors: as bs_conv2d; BS_ERR_UNSUPPORTED when no fused kernel covers the
 * shape (c must be 32 times a power of two, at most 512 for 3x3 windows
 * and 4096 for 1x1 ones, oc a multiple of 4, kernels square of size 1 or 3,
 * stride 1 or 2, unipolar activations of 1-4 bits with unipolar filters of
 * 1-4 bits or bipolar 1-bit filters, and the packed input rows that the
 * windows of 256 consecutive output pixels span, plus 17 KB, within 64 KB
 * of LDS -- only very wide rows or very many channels miss this): pack
 * with bs_pack and call bs_conv2d instead.
 * Nothing is enqueued on any error. */
bs_status bs_conv2d_codes(const bs_conv2d_params *p, const uint8_t *act_codes,
                          const uint32_t *w_packed, int32_t *out,
                          bs_stream_t stream);

/* Bitserial conv2d of float32 activations: the quantization and bit-pack
 * of Sec. 3.1 fused into the conv, for 1x1 windows.  Exactly
 * bs_quantize_pack of act (unipolar, act_scale, p->abits bits) followed by
 * bs_conv2d: every workgroup quantizes and bit-packs, into LDS, the input
 * pixels its outputs read -- at stride 2 only those, a quarter of the
 * input -- and convolves from there; neither codes nor packed words reach
 * HBM.
 *   act: [n][h][w][c] float32 NHWC (device), quantized as bs_quantize
 *        does (round half to even of act * act_scale, clamped to
 *        [0, 2^abits - 1], NaN to 0);
 *   w_packed, out and the result: as bs_conv2d.
 * Errors: as bs_conv2d; BS_ERR_INVALID_ARG for a scale bs_quantize
 * refuses; BS_ERR_UNSUPPORTED for activations that are not unipolar and
 * when no fused kernel covers the shape (a 1x1 window at stride 1 or 2,
 * c 32 times a power of two up to 4096, oc a multiple of 4, activations
 * of 1-4 bits with unipolar filters of 1-4 bits or bipolar 1-bit filters,
 * and the packed input pixels of 256 consecutive output pixels, plus
 * 17 KB, within 64 KB of LDS): quantize and pack with bs_quantize_pack
 * and call bs_conv2d instead.  Nothing is enqueued on any error. */
bs_status bs_conv2d_quantized(const bs_conv2d_params *p, const float *act,
                              float act_scale, const uint32_t *w_packed,
                              int32_t *out, bs_stream_t stream);

/* Bitserial conv2d whose result is requantized and bit-packed as the next
 * layer's activations (layer chaining, toward the end-to-end low-precision
 * inference of Sec. 7): the int32 result v of bs_conv2d for each output is
 * converted to float32, quantized as bs_quantize does (unipolar,
 * q = clamp(round_half_even(fl32(v * out_scale)), 0, 2^out_bits - 1)) and
 * packed as bs_pack does, along the output channels:
 *   out_packed: [n][oh][ow][out_bits][ceil(oc/32)] uint32, tail bits zero.
 * Equals bs_conv2d followed by bs_quantize_pack of its output converted to
 * float32 (round to nearest even; exact while |v| <= 2^24), without ever
 * writing the int32 result.  Device pointers as in bs_conv2d; out_packed
 * must not overlap the inputs.
 * Errors: as bs_conv2d; BS_ERR_INVALID_ARG for out_bits outside 1..8 or a
 * non-finite or non-positive out_scale. */
bs_status bs_conv2d_requant(const bs_conv2d_params *p,
                            const uint32_t *act_packed,
                            const uint32_t *w_packed, float out_scale,
                            int out_bits, uint32_t *out_packed,
                            bs_stream_t stream);

/* A ResNet downsampling block's two convolutions of one input in one pass
 * (Table 1 layers 4 and 5, 7 and 8, 10 and 11): the KxK conv p, and the 1x1
 * conv with the same stride, no padding and oc filters w1_packed, whose
 * input pixel for every output position is the centre tap of the KxK
 * window; p must have kh == kw odd, pad (kh - 1) / 2 on both axes and equal
 * strides, so that both convolutions have the same output grid.  Exactly
 * bs_conv2d(p, act_packed, w_packed, out) and bs_conv2d of the 1x1 conv
 * (w1_packed, out1), with the packed activations read once and the 1x1
 * conv's products taken from the KxK window's centre-tap words already in
 * registers: its added work is 1/(kh kw) of the KxK conv's.
 *   w1_packed: [oc][1][1][wbits][ceil(c/32)] uint32 (bs_pack of [oc][c]);
 *   out, out1: [n][oh][ow][oc] int32 each; every element is written.
 * Shapes no paired kernel covers run as the two convolutions one after the
 * other, with the same results.
 * Errors: as bs_conv2d; BS_ERR_INVALID_ARG for a window that is not square
 * and odd, other padding, unequal strides, or outputs that overlap each
 * other or an input. */
bs_status bs_conv2d_pair(const bs_conv2d_params *p, const uint32_t *act_packed,
                         const uint32_t *w_packed, const uint32_t *w1_packed,
                         int32_t *out, int32_t *out1, bs_stream_t stream);

/* bs_conv2d_pair with both outputs requantized and bit-packed as
 * bs_conv2d_requant does (out_bits-bit unipolar codes; out_scale for the
 * KxK conv, out1_scale for the 1x1 conv):
 *   out_packed, out1_packed: [n][oh][ow][out_bits][ceil(oc/32)] uint32.
 * Errors: as bs_conv2d_pair and bs_conv2d_requant. */
bs_status bs_conv2d_pair_requant(const bs_conv2d_params *p,
                                 const uint32_t *act_packed,
                                 const uint32_t *w_packed,
                                 const uint32_t *w1_packed, float out_scale,
                                 float out1_scale, int out_bits,
                                 uint32_t *out_packed, uint32_t *out1_packed,
                                 bs_stream_t stream);

/* Describes, as text, the kernel and launch configuration that bs_conv2d
 * would use for p under the calling thread's kernel mode (template
 * parameters, grid, block, LDS bytes).  Writes at most len bytes including
 * the terminating NUL into the caller's buffer buf (truncating); host only,
 * nothing is enqueued.  A dense call of shape (m, n, k) is described by the
 * 1x1 conv n = 1, h = 1, w = m, c = k, oc = n.
 * Errors: as bs_conv2d's parameter checks; BS_ERR_INVALID_ARG for a NULL
 * buf or len < 1. */
bs_status bs_conv2d_describe(const bs_conv2d_params *p, char *buf,
                             int32_t len);

/* As bs_conv2d_describe, for bs_conv2d_codes (the activation pack fused
 * into the conv, Sec. 3.1 bitpack with Eq. 2): the staged kernel and its
 * launch plan -- grid, block, LDS bytes (output tiles plus the largest
 * input region a workgroup packs), that region in pixels, run length.
 * Host only, nothing is enqueued.
 * Errors: as bs_conv2d_describe; BS_ERR_UNSUPPORTED (buf empty) where
 * bs_conv2d_codes would return it. */
bs_status bs_conv2d_codes_describe(const bs_conv2d_params *p, char *buf,
                                   int32_t len);

/* As bs_conv2d_codes_describe, for bs_conv2d_quantized.
 * Errors: as bs_conv2d_describe; BS_ERR_UNSUPPORTED (buf empty) where
 * bs_conv2d_quantized would return it. */
bs_status bs_conv2d_quantized_describe(const bs_conv2d_params *p, char *buf,
                                       int32_t len);

/* Bitserial dense / matrix multiply (Sec. 3.2; evaluated in Sec. 6.2.1):
 *   a_packed: [m][abits][ceil(k/32)], w_packed: [n][wbits][ceil(k/32)] uint32
 *   (each output neuron's weights contiguous along the reduction axis),
 *   out: [m][n] int32, out[r][o] = sum_k value(a[r][k]) * value(w[o][k]),
 *   unipolar activations, weights under wenc (as bs_conv2d).
 * Errors: as bs_conv2d, with the overflow bound max|a| max|w| k. */
bs_status bs_dense(int64_t m, int64_t n, int64_t k, int abits, int wbits,
                   bs_encoding wenc, const uint32_t *a_packed,
                   const uint32_t *w_packed, int32_t *out, bs_stream_t stream);

/* bs_dense with an activation encoding as well (bipolar +-1 activations,
 * signed activations).  Layouts, results and errors as bs_dense. */
bs_status bs_dense_ex(int64_t m, int64_t n, int64_t k, int abits,
                      bs_encoding aenc, int wbits, bs_encoding wenc,
                      const uint32_t *a_packed, const uint32_t *w_packed,
                      int32_t *out, bs_stream_t stream);

/* Static description of a status code. */
const char *bs_status_string(bs_status s);

/* Detail of the last non-OK status returned on the calling thread ("" if
 * none).  The string stays valid until the next call on that thread. */
const char *bs_last_error(void);

/* Selects which conv/dense kernels serve later calls made on the calling
 * host thread:
 *   0 = the fastest kernel that applies to the shape (default),
 *   1 = the plain generic kernel for every shape,
 *   2 = the output-channels-on-lanes kernel where it applies,
 *   3 = the pixels-on-lanes kernel where it applies
 * (2 and 3 use the generic kernel for shapes they do not cover).  All give
 * identical results; the switch exists so tests can check each kernel
 * against the others and against the reference.
 * Errors: BS_ERR_INVALID_ARG for a mode outside 0..3. */
bs_status bs_set_kernel_mode(int mode);

/* Overrides, for later conv/dense calls on the calling host thread, how much
 * work each wave of the pixels-on-lanes kernel takes: a contiguous run of
 * `units` units of (64 output pixels x 4 output channels).  0 (the default)
 * lets the library choose the run that fills the GPU in one balanced round
 * (for bs_conv2d_quantized with strided 1x1 windows, lengthened until at
 * most two workgroups share a group of 64 output pixels, while the grid
 * keeps a workgroup for at least every other compute unit).
 * Results do not depend on it; it exists for tests of the run boundaries and
 * for tuning.  Errors: BS_ERR_INVALID_ARG for units < 0. */
bs_status bs_set_units_per_wave(int units);

/* Timing of the library's own kernels, for benchmarks.  The next kernel the
 * library launches for a call made on the calling host thread is launched
 * with `start` as its dispatch's start event, and every kernel until the
 * events are cleared with `stop` as its stop event (hipExtLaunchKernel; the
 * handles are hipEvent_t the caller created, e.g. with hipEventCreate).  The
 * runtime stamps them with the dispatches' own start and end on the GPU, so
 * after one call hipEventElapsedTime(start, stop) is the time from its first
 * kernel's start to its last kernel's end -- for a one-kernel call, the
 * duration a kernel trace reports -- without the gaps that events recorded
 * between launches add.  Set the pair again before each call to be timed.
 * Either handle may be NULL; NULL, NULL clears.  The library neither creates
 * nor destroys the events.  Returns BS_OK. */
bs_status bs_set_timing_events(void *start, void *stop);

/* ABI version of this header (major * 100 + minor). */
int bs_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif /* BITSERIAL_H */
