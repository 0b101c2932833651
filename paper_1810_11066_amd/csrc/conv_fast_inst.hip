// Specialisations of the channels-on-lanes conv kernel for BS_A-bit
// activations (BS_A = 1..4).  The build compiles this source once per
// activation width, each with its own -DBS_A, so that the widths compile in
// parallel.
#include "conv_fast.h"

#ifndef BS_A
#error "BS_A (activation bits, 1..4) must be defined"
#endif
#if BS_A < 1 || BS_A > 4
#error "BS_A must be 1..4"
#endif

namespace bs {
namespace fast {
namespace {

// Bit-width/encoding combinations that also get compile-time word counts
// (the ResNet-18 workloads at A1W1, A2W1, A2W2, A3W3 and bipolar weights);
// every other combination runs with the word count as an argument.
template <int A_, int W_, bool B_>
constexpr bool kSpecialiseWords =
    (A_ == 1 && W_ == 1) || (A_ == 2 && W_ == 1) ||
    (A_ == 2 && W_ == 2 && !B_) || (A_ == 3 && W_ == 3 && !B_);

template <int A_, int W_, bool B_, int K, int S, int P>
KernelFn pick_cw(int cw) {
    if constexpr (kSpecialiseWords<A_, W_, B_>) {
        switch (cw) {
            case 2: return conv_ocl_kernel<A_, W_, B_, K, S, P, 2>;
            case 4: return conv_ocl_kernel<A_, W_, B_, K, S, P, 4>;
            case 8: return conv_ocl_kernel<A_, W_, B_, K, S, P, 8>;
            case 16: return conv_ocl_kernel<A_, W_, B_, K, S, P, 16>;
            default: break;
        }
    }
    return conv_ocl_kernel<A_, W_, B_, K, S, P, 0>;
}
template <int A_, int W_, bool B_, int K, int S>
KernelFn pick_p(int p, int cw) {
    return p == 7 ? pick_cw<A_, W_, B_, K, S, 7>(cw)
                  : pick_cw<A_, W_, B_, K, S, 8>(cw);
}
template <int A_, int W_, bool B_>
KernelFn pick_ks(int k, int s, int p, int cw) {
    if (k == 1) return s == 1 ? pick_p<A_, W_, B_, 1, 1>(p, cw)
                              : pick_p<A_, W_, B_, 1, 2>(p, cw);
    return s == 1 ? pick_p<A_, W_, B_, 3, 1>(p, cw)
                  : pick_p<A_, W_, B_, 3, 2>(p, cw);
}
template <int A_, int W_>
KernelFn pick_b(bool b, int k, int s, int p, int cw) {
    return b ? pick_ks<A_, W_, true>(k, s, p, cw)
             : pick_ks<A_, W_, false>(k, s, p, cw);
}

}  // namespace

template <>
KernelFn pick_w<BS_A>(int w, bool b, int k, int s, int p, int cw) {
    switch (w) {
        case 1: return pick_b<BS_A, 1>(b, k, s, p, cw);
        case 2: return pick_b<BS_A, 2>(b, k, s, p, cw);
        case 3: return pick_b<BS_A, 3>(b, k, s, p, cw);
        default: return pick_b<BS_A, 4>(b, k, s, p, cw);
    }
}

}  // namespace fast
}  // namespace bs
