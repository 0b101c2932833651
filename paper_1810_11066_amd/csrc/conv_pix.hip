// Dispatch to the pixels-on-lanes conv specialisations (conv_pix_a<A>.hip).
#include "conv_pix.h"

namespace bs {
namespace pix {

PixKernelFn pick(int a, int w, bool b, int k, int s, int cw, bool req,
                 PlanInfo* info) {
    if (s != 1 && s != 2) return nullptr;
    switch (a) {
        case 1: return pick_a<1>(w, b, k, s, cw, req, info);
        case 2: return pick_a<2>(w, b, k, s, cw, req, info);
        case 3: return pick_a<3>(w, b, k, s, cw, req, info);
        case 4: return pick_a<4>(w, b, k, s, cw, req, info);
        default: return nullptr;
    }
}

}  // namespace pix
}  // namespace bs
