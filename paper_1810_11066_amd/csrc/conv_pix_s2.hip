// Pixels-on-lanes conv specialisations with signed (two's complement)
// operands, 2-bit activations.
#include "conv_pix.h"

namespace bs {
namespace pix {

template <>
PixKernelFn pick_signed<2>(int w, int ae, int we, int k, int s, int cw,
                           PlanInfo* info) {
    return pick_signed_for_a<2>(w, ae, we, k, s, cw, info);
}

}  // namespace pix
}  // namespace bs
