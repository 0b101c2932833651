// Specialisations of the pixels-on-lanes bitserial conv kernel.
#include "conv_pix.h"

namespace bs {
namespace pix {
namespace {

struct PlanOut {
    int *ocb, *ts, *tb, *cb;
};

template <int A, int W, bool B, int K, int S, int CW>
PixKernelFn pick_kscw(const PlanOut& o) {
    using Pl = Plan<A, W, K, CW>;
    if constexpr (!Pl::kFits) {
        return nullptr;
    } else {
        *o.ocb = Pl::OCB;
        *o.ts = Pl::TS;
        *o.tb = Pl::TB;
        *o.cb = Pl::CB;
        return conv_pix_kernel<A, W, B, K, S, CW>;
    }
}

// Words per plane: 1..16 for 3x3 windows; 1x1 windows (and dense, a 1x1
// conv) up to 128 words = 4096 input channels.
template <int A, int W, bool B, int K, int S>
PixKernelFn pick_cw(int cw, const PlanOut& o) {
    switch (cw) {
        case 1: return pick_kscw<A, W, B, K, S, 1>(o);
        case 2: return pick_kscw<A, W, B, K, S, 2>(o);
        case 4: return pick_kscw<A, W, B, K, S, 4>(o);
        case 8: return pick_kscw<A, W, B, K, S, 8>(o);
        case 16: return pick_kscw<A, W, B, K, S, 16>(o);
        default: break;
    }
    if constexpr (K == 1) {
        switch (cw) {
            case 32: return pick_kscw<A, W, B, K, S, 32>(o);
            case 64: return pick_kscw<A, W, B, K, S, 64>(o);
            case 128: return pick_kscw<A, W, B, K, S, 128>(o);
            default: break;
        }
    }
    return nullptr;
}

template <int A, int W, bool B>
PixKernelFn pick_ks(int k, int s, int cw, const PlanOut& o) {
    if (k == 1) return s == 1 ? pick_cw<A, W, B, 1, 1>(cw, o)
                              : pick_cw<A, W, B, 1, 2>(cw, o);
    if (k == 3) return s == 1 ? pick_cw<A, W, B, 3, 1>(cw, o)
                              : pick_cw<A, W, B, 3, 2>(cw, o);
    return nullptr;
}

}  // namespace

// The bit-width/encoding combinations of the ResNet-18 workloads.
PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, int* ocb,
                 int* ts, int* tb, int* cb) {
    if (s != 1 && s != 2) return nullptr;
    const PlanOut o{ocb, ts, tb, cb};
    if (a == 1 && w == 1)
        return b ? pick_ks<1, 1, true>(k, s, cw, o)
                 : pick_ks<1, 1, false>(k, s, cw, o);
    if (a == 2 && w == 1)
        return b ? pick_ks<2, 1, true>(k, s, cw, o)
                 : pick_ks<2, 1, false>(k, s, cw, o);
    if (a == 2 && w == 2 && !b) return pick_ks<2, 2, false>(k, s, cw, o);
    if (a == 3 && w == 3 && !b) return pick_ks<3, 3, false>(k, s, cw, o);
    return nullptr;
}

}  // namespace pix
}  // namespace bs
