// Pixels-on-lanes conv specialisations for 1-bit activations.
#include "conv_pix.h"

namespace bs {
namespace pix {

template <>
PixKernelFn pick_a<1>(int w, bool b, int k, int s, int cw, bool req,
                      PlanInfo* info) {
    return pick_for_a<1>(w, b, k, s, cw, req, info);
}

}  // namespace pix
}  // namespace bs
