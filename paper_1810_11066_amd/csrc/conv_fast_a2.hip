// Specialisations of the fast bitserial conv kernel for 2-bit activations.
#include "conv_fast.h"

namespace bs {
namespace fast {
namespace {

template <int A, int W, bool B, int K, int S>
KernelFn pick_p(int p) {
    return p == 7 ? conv_ocl_kernel<A, W, B, K, S, 7>
                  : conv_ocl_kernel<A, W, B, K, S, 8>;
}
template <int A, int W, bool B>
KernelFn pick_ks(int k, int s, int p) {
    if (k == 1) return s == 1 ? pick_p<A, W, B, 1, 1>(p) : pick_p<A, W, B, 1, 2>(p);
    return s == 1 ? pick_p<A, W, B, 3, 1>(p) : pick_p<A, W, B, 3, 2>(p);
}
template <int A, int W>
KernelFn pick_b(bool b, int k, int s, int p) {
    return b ? pick_ks<A, W, true>(k, s, p) : pick_ks<A, W, false>(k, s, p);
}
}  // namespace

template <>
KernelFn pick_w<2>(int w, bool b, int k, int s, int p) {
    constexpr int A = 2;
    switch (w) {
        case 1: return pick_b<A, 1>(b, k, s, p);
        case 2: return pick_b<A, 2>(b, k, s, p);
        case 3: return pick_b<A, 3>(b, k, s, p);
        default: return pick_b<A, 4>(b, k, s, p);
    }
}

}  // namespace fast
}  // namespace bs
