// One unit of the pixels-on-lanes conv specialisations.  The build compiles
// this source once per unit, so that the ~1500 kernels compile in parallel:
//   -DBS_PIX_FAMILY=0 -DBS_A=<1..4>  unipolar activations of BS_A bits with
//                                    unipolar (W = 1..4) or bipolar (W = 1)
//                                    filters, int32 or requantized output;
//   -DBS_PIX_FAMILY=1 -DBS_A=<1..4>  signed filters (W = 2..4) with unipolar
//                                    activations, and signed activations with
//                                    signed filters of the same width;
//   -DBS_PIX_FAMILY=2                +-1 activations with 1-bit filters.
#include "conv_pix.h"

#ifndef BS_PIX_FAMILY
#error "BS_PIX_FAMILY (0, 1 or 2) must be defined"
#endif
#if BS_PIX_FAMILY != 2 && (!defined(BS_A) || BS_A < 1 || BS_A > 4)
#error "BS_A (activation bits, 1..4) must be defined for families 0 and 1"
#endif

namespace bs {
namespace pix {

#if BS_PIX_FAMILY == 0
template <>
PixKernelFn pick_a<BS_A>(int w, bool b, int k, int s, int cw, bool req,
                         int src, bool dual, PlanInfo* info) {
    return pick_for_a<BS_A>(w, b, k, s, cw, req, src, dual, info);
}
#elif BS_PIX_FAMILY == 1
template <>
PixKernelFn pick_signed<BS_A>(int w, int ae, int we, int k, int s, int cw,
                              PlanInfo* info) {
    return pick_signed_for_a<BS_A>(w, ae, we, k, s, cw, info);
}
#else
PixKernelFn pick_bipolar_act(int we, int k, int s, int cw, PlanInfo* info) {
    constexpr int BB = 3 * kBipolar + kBipolar, BU = 3 * kBipolar + kUnipolar;
    if (we == kBipolar)
        return pick_ks<1, 1, BB>(k, s, cw, false, kSrcPacked, false, info);
    if (we == kUnipolar)
        return pick_ks<1, 1, BU>(k, s, cw, false, kSrcPacked, false, info);
    return nullptr;
}
#endif

}  // namespace pix
}  // namespace bs
