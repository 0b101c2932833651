// Specialisations of the pixels-on-lanes bitserial conv kernel.
#include "conv_pix.h"

namespace bs {
namespace pix {
namespace {

// The lane's patch (K*K*A*CW words) lives in VGPRs next to the accumulators
// and addresses; beyond this many words occupancy falls too far.
constexpr int kMaxPatchWords = 72;

template <int A, int W, bool B, int K, int S, int CW>
PixKernelFn pick_kscw(int* ocb, int* ts) {
    using St = Stream<K, W, CW>;
    if constexpr (K * K * A * CW > kMaxPatchWords || !St::kFits) {
        return nullptr;
    } else {
        *ocb = St::OCB;
        *ts = St::TS;
        return conv_pix_kernel<A, W, B, K, S, CW>;
    }
}

template <int A, int W, bool B, int K, int S>
PixKernelFn pick_cw(int cw, int* ocb, int* ts) {
    switch (cw) {
        case 1: return pick_kscw<A, W, B, K, S, 1>(ocb, ts);
        case 2: return pick_kscw<A, W, B, K, S, 2>(ocb, ts);
        case 4: return pick_kscw<A, W, B, K, S, 4>(ocb, ts);
        case 8:
            if constexpr (K == 1) return pick_kscw<A, W, B, K, S, 8>(ocb, ts);
            return nullptr;
        case 16:
            if constexpr (K == 1) return pick_kscw<A, W, B, K, S, 16>(ocb, ts);
            return nullptr;
        default: return nullptr;
    }
}

template <int A, int W, bool B>
PixKernelFn pick_ks(int k, int s, int cw, int* ocb, int* ts) {
    if (k == 1) return s == 1 ? pick_cw<A, W, B, 1, 1>(cw, ocb, ts)
                              : pick_cw<A, W, B, 1, 2>(cw, ocb, ts);
    if (k == 3) return s == 1 ? pick_cw<A, W, B, 3, 1>(cw, ocb, ts)
                              : pick_cw<A, W, B, 3, 2>(cw, ocb, ts);
    return nullptr;
}

}  // namespace

// The bit-width/encoding combinations of the ResNet-18 workloads.
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb,
                 int* ts) {
    if (s != 1 && s != 2) return nullptr;
    if (a == 1 && w == 1) return b ? pick_ks<1, 1, true>(k, s, cw, ocb, ts)
                                   : pick_ks<1, 1, false>(k, s, cw, ocb, ts);
    if (a == 2 && w == 1) return b ? pick_ks<2, 1, true>(k, s, cw, ocb, ts)
                                   : pick_ks<2, 1, false>(k, s, cw, ocb, ts);
    if (a == 2 && w == 2 && !b) return pick_ks<2, 2, false>(k, s, cw, ocb, ts);
    if (a == 3 && w == 3 && !b) return pick_ks<3, 3, false>(k, s, cw, ocb, ts);
    return nullptr;
}

}  // namespace pix
}  // namespace bs
