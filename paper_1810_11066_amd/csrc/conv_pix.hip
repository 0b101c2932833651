// Specialisations of the pixels-on-lanes bitserial conv kernel.
#include "conv_pix.h"

namespace bs {
namespace pix {
namespace {

template <int A, int W, bool B, int K, int S, int CW>
PixKernelFn pick_kscw(int* ocb, int* ts, int* tb) {
    using Pl = Plan<A, W, K, CW>;
    if constexpr (!Pl::kFits) {
        return nullptr;
    } else {
        *ocb = Pl::OCB;
        *ts = Pl::TS;
        *tb = Pl::TB;
        return conv_pix_kernel<A, W, B, K, S, CW>;
    }
}

template <int A, int W, bool B, int K, int S>
PixKernelFn pick_cw(int cw, int* ocb, int* ts, int* tb) {
    switch (cw) {
        case 1: return pick_kscw<A, W, B, K, S, 1>(ocb, ts, tb);
        case 2: return pick_kscw<A, W, B, K, S, 2>(ocb, ts, tb);
        case 4: return pick_kscw<A, W, B, K, S, 4>(ocb, ts, tb);
        case 8: return pick_kscw<A, W, B, K, S, 8>(ocb, ts, tb);
        case 16: return pick_kscw<A, W, B, K, S, 16>(ocb, ts, tb);
        default: return nullptr;
    }
}

template <int A, int W, bool B>
PixKernelFn pick_ks(int k, int s, int cw, int* ocb, int* ts, int* tb) {
    if (k == 1) return s == 1 ? pick_cw<A, W, B, 1, 1>(cw, ocb, ts, tb)
                              : pick_cw<A, W, B, 1, 2>(cw, ocb, ts, tb);
    if (k == 3) return s == 1 ? pick_cw<A, W, B, 3, 1>(cw, ocb, ts, tb)
                              : pick_cw<A, W, B, 3, 2>(cw, ocb, ts, tb);
    return nullptr;
}

}  // namespace

// The bit-width/encoding combinations of the ResNet-18 workloads.
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb,
                 int* ts, int* tb) {
    if (s != 1 && s != 2) return nullptr;
    if (a == 1 && w == 1)
        return b ? pick_ks<1, 1, true>(k, s, cw, ocb, ts, tb)
                 : pick_ks<1, 1, false>(k, s, cw, ocb, ts, tb);
    if (a == 2 && w == 1)
        return b ? pick_ks<2, 1, true>(k, s, cw, ocb, ts, tb)
                 : pick_ks<2, 1, false>(k, s, cw, ocb, ts, tb);
    if (a == 2 && w == 2 && !b)
        return pick_ks<2, 2, false>(k, s, cw, ocb, ts, tb);
    if (a == 3 && w == 3 && !b)
        return pick_ks<3, 3, false>(k, s, cw, ocb, ts, tb);
    return nullptr;
}

}  // namespace pix
}  // namespace bs
