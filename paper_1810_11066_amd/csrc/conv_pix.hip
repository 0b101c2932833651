// Dispatch to the pixels-on-lanes conv specialisations (the compile units of
// conv_pix_inst.hip).
#include "conv_pix.h"

namespace bs {
namespace pix {

PixKernelFn pick(int a, int w, int ae, int we, int k, int s, int cw, bool req,
                 int src, bool dual, PlanInfo* info) {
    if (s != 1 && s != 2) return nullptr;
    if (ae == kBipolar) {
        if (a != 1 || w != 1 || we == kSigned || req || src != kSrcPacked ||
            dual)
            return nullptr;
        return pick_bipolar_act(we, k, s, cw, info);
    }
    if (we == kSigned || ae == kSigned) {
        if (req || src != kSrcPacked || dual) return nullptr;
        switch (a) {
            case 1: return pick_signed<1>(w, ae, we, k, s, cw, info);
            case 2: return pick_signed<2>(w, ae, we, k, s, cw, info);
            case 3: return pick_signed<3>(w, ae, we, k, s, cw, info);
            case 4: return pick_signed<4>(w, ae, we, k, s, cw, info);
            default: return nullptr;
        }
    }
    const bool b = we == kBipolar;
    switch (a) {
        case 1: return pick_a<1>(w, b, k, s, cw, req, src, dual, info);
        case 2: return pick_a<2>(w, b, k, s, cw, req, src, dual, info);
        case 3: return pick_a<3>(w, b, k, s, cw, req, src, dual, info);
        case 4: return pick_a<4>(w, b, k, s, cw, req, src, dual, info);
        default: return nullptr;
    }
}

}  // namespace pix
}  // namespace bs
