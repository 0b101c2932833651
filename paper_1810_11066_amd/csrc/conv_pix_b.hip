// Pixels-on-lanes conv specialisations for +-1 activations (1-bit bipolar
// codes) with 1-bit filters: bipolar filters (the XNOR case) or unipolar ones.
#include "conv_pix.h"

namespace bs {
namespace pix {

PixKernelFn pick_bipolar_act(int we, int k, int s, int cw, PlanInfo* info) {
    constexpr int BB = 3 * kBipolar + kBipolar, BU = 3 * kBipolar + kUnipolar;
    if (we == kBipolar) return pick_ks<1, 1, BB>(k, s, cw, false, info);
    if (we == kUnipolar) return pick_ks<1, 1, BU>(k, s, cw, false, info);
    return nullptr;
}

}  // namespace pix
}  // namespace bs
