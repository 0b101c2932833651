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

struct Args {
    int32_t h, w, c, oc, stride, pad, oh, ow;
    int32_t npix;     // n * oh * ow
    int32_t units;    // ceil(npix / 32) * (oc / 64)
    int32_t kc;       // c / 64
    int32_t act_bytes, out_bytes;
};

__device__ __forceinline__ Rsrc make_rsrc(const void* p, int32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0,
                                             bytes, 0x00020000);
}

template <int K>
__global__ __launch_bounds__(kBlock) void conv_i8_mfma_kernel(
    const int8_t* __restrict__ act, const int8_t* __restrict__ wts,
    int32_t* __restrict__ out, Args g) {
    extern __shared__ uint4 frag[];
    constexpr int KK = K * K;
    const int tid = threadIdx.x, lane = tid & 63;
    const int nt_all = g.oc / 16;
    // stage the B fragments: element e = (fragment, lane), fragment
    // (tap, slice, tile) -> 16 bytes of filter row (o, tap) at channel
    // slice * 64 + 16 (lane / 16), o = tile * 16 + lane % 16
    const int nfrag = KK * g.kc * nt_all;
    for (int e = tid; e < nfrag * 64; e += kBlock) {
        const int f = e >> 6, l = e & 63;
        const int t = f % nt_all, ts = f / nt_all;
        const int sl = ts % g.kc, tap = ts / g.kc;
        const int o = t * 16 + (l & 15);
        frag[e] = *reinterpret_cast<const uint4*>(
            wts + ((size_t)o * KK + tap) * g.c + sl * 64 + 16 * (l >> 4));
    }
    __syncthreads();

    const Rsrc ra = make_rsrc(act, g.act_bytes);
    const Rsrc ro = make_rsrc(out, g.out_bytes);
    const int ncb = g.oc / 64;
    const int wave = __builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kWaves + (tid >> 6)));
    const int nwaves = gridDim.x * kWaves;
    const uint32_t rowb = (uint32_t)g.w * (uint32_t)g.c;
    for (int u = wave; u < g.units; u += nwaves) {
        const int tile = u / ncb, cb = u - tile * ncb;
        // this lane's pixel in each 16-pixel half (the last pixel stands in
        // past the end: loads stay in the tensor, stores are dropped)
        int iy0[2], ix0[2];
        uint32_t base[2];
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            int p = tile * 32 + 16 * m + (lane & 15);
            p = p < g.npix ? p : g.npix - 1;
            const int row = p / g.ow, ox = p - row * g.ow;
            const int img = row / g.oh, oy = row - img * g.oh;
            iy0[m] = oy * g.stride - g.pad;
            ix0[m] = ox * g.stride - g.pad;
            base[m] = ((uint32_t)(img * g.h + iy0[m]) * (uint32_t)g.w +
                       (uint32_t)ix0[m]) * (uint32_t)g.c +
                      16u * (uint32_t)(lane >> 4);
        }
        v4i acc[2][4];
#pragma unroll
        for (int m = 0; m < 2; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = v4i{0, 0, 0, 0};
        for (int sl = 0; sl < g.kc; ++sl) {
            // every tap's A fragments first, then the products: the loads
            // of a slice are in flight together
            v4i a[KK][2];
#pragma unroll
            for (int tap = 0; tap < KK; ++tap) {
                const int r = tap / K, s = tap - r * K;
#pragma unroll
                for (int m = 0; m < 2; ++m) {
                    const bool in = (unsigned)(iy0[m] + r) < (unsigned)g.h &&
                                    (unsigned)(ix0[m] + s) < (unsigned)g.w;
                    const uint32_t off =
                        in ? base[m] + (uint32_t)r * rowb +
                                 (uint32_t)s * (uint32_t)g.c +
                                 64u * (uint32_t)sl
                           : kOutOfRange;
                    a[tap][m] = __builtin_bit_cast(
                        v4i, __builtin_amdgcn_raw_buffer_load_b128(ra, off, 0,
                                                                   0));
                }
            }
#pragma unroll
            for (int tap = 0; tap < KK; ++tap) {
                const uint4* fb =
                    frag + ((size_t)((tap * g.kc + sl) * nt_all + cb * 4)) * 64 +
                    lane;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const v4i b = __builtin_bit_cast(v4i, fb[t * 64]);
                    acc[0][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                        b, a[tap][0], acc[0][t], 0, 0, 0);
                    acc[1][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                        b, a[tap][1], acc[1][t], 0, 0, 0);
                }
            }
        }
        // lane l holds channels 4 (l / 16) .. + 3 of the 16-channel tile
        // for pixel l % 16 of each half
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int p = tile * 32 + 16 * m + (lane & 15);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int o = cb * 64 + t * 16 + 4 * (lane >> 4);
                const uint32_t off =
                    p < g.npix
                        ? ((uint32_t)p * (uint32_t)g.oc + (uint32_t)o) * 4u
                        : kOutOfRange;
                __builtin_amdgcn_raw_buffer_store_b128(
                    __builtin_bit_cast(
                        __attribute__((ext_vector_type(4))) unsigned,
                        acc[m][t]),
                    ro, off, 0, 0);
            }
        }
    }
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
    const void* fn = p->kh == 3 ? (const void*)conv_i8_mfma_kernel<3>
                                : (const void*)conv_i8_mfma_kernel<1>;
    int dev = 0, cus = 256, per_cu = 1;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount,
                                    dev);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kBlock,
                                                     (size_t)wbytes) !=
            hipSuccess ||
        per_cu < 1)
        per_cu = 1;
    // persistent workgroups: one round on every CU, no more than the units
    int64_t blocks = (int64_t)cus * per_cu;
    const int64_t need = (g.units + kWaves - 1) / kWaves;
    if (blocks > need) blocks = need;
    void* args[] = {&act, &wts, &out, &g};
    const hipError_t e = hipLaunchKernel(fn, dim3((uint32_t)blocks),
                                         dim3(kBlock), args, (size_t)wbytes,
                                         (hipStream_t)stream);
    if (e != hipSuccess)
        return fail(I8MFMA_ERR_HIP, "launch: %s", hipGetErrorString(e));
    g_err[0] = '\0';
    return I8MFMA_OK;
}

}  // extern "C"
