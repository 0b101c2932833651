// Specialisations of the pixels-on-lanes bitserial conv kernel.
#include "conv_pix.h"

namespace bs {
namespace pix {
namespace {

// Register budgets: the lane's patch (K*K*A*CW VGPRs) and two filter batches
// (2 * OCB*K*K*W*CW SGPRs) must fit next to the accumulators and addresses.
constexpr int kMaxPatchWords = 72;
constexpr int kMaxBatchWords = 40;

template <int K, int W, int CW>
constexpr int batch_size() {
    constexpr int fw = K * K * W * CW;
    return fw * 4 <= kMaxBatchWords ? 4 : fw * 2 <= kMaxBatchWords ? 2 : 1;
}

template <int A, int W, bool B, int K, int S, int CW>
PixKernelFn pick_kscw(int* ocb) {
    constexpr int fw = K * K * W * CW;
    if constexpr (K * K * A * CW > kMaxPatchWords || fw > kMaxBatchWords) {
        return nullptr;
    } else {
        constexpr int OCB = batch_size<K, W, CW>();
        *ocb = OCB;
        return conv_pix_kernel<A, W, B, K, S, CW, OCB>;
    }
}

template <int A, int W, bool B, int K, int S>
PixKernelFn pick_cw(int cw, int* ocb) {
    switch (cw) {
        case 1: return pick_kscw<A, W, B, K, S, 1>(ocb);
        case 2: return pick_kscw<A, W, B, K, S, 2>(ocb);
        case 4: return pick_kscw<A, W, B, K, S, 4>(ocb);
        default: return nullptr;
    }
}

template <int A, int W, bool B>
PixKernelFn pick_ks(int k, int s, int cw, int* ocb) {
    if (k == 1) return s == 1 ? pick_cw<A, W, B, 1, 1>(cw, ocb)
                              : pick_cw<A, W, B, 1, 2>(cw, ocb);
    if (k == 3) return s == 1 ? pick_cw<A, W, B, 3, 1>(cw, ocb)
                              : pick_cw<A, W, B, 3, 2>(cw, ocb);
    return nullptr;
}

}  // namespace

// The bit-width/encoding combinations of the ResNet-18 workloads.
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb) {
    if (s != 1 && s != 2) return nullptr;
    if (a == 1 && w == 1) return b ? pick_ks<1, 1, true>(k, s, cw, ocb)
                                   : pick_ks<1, 1, false>(k, s, cw, ocb);
    if (a == 2 && w == 1) return b ? pick_ks<2, 1, true>(k, s, cw, ocb)
                                   : pick_ks<2, 1, false>(k, s, cw, ocb);
    if (a == 2 && w == 2 && !b) return pick_ks<2, 2, false>(k, s, cw, ocb);
    if (a == 3 && w == 3 && !b) return pick_ks<3, 3, false>(k, s, cw, ocb);
    return nullptr;
}

}  // namespace pix
}  // namespace bs
