// Instantiations of the fused decode + matrix-core kernel for convolutions.
#include "aq_fused_kernel.h"

namespace aq {

template <int KIND, int CM, int DEC, int MC>
static hipError_t conv_tiles(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
#define AQ_TILE(TBM, TBN, TUPL) \
    if (p.bm == TBM && p.bn == TBN && p.upl == TUPL) return fused_launch_cfg<KIND, CM, AQ_F16, DEC, MC, TBM, TBN, TUPL>(geo, p, fl);
    if constexpr (KIND == 1) {
        AQ_TILE(64, 96, 3)
        AQ_TILE(64, 64, 3)
        AQ_TILE(128, 64, 3)
        AQ_TILE(128, 64, 6)
        AQ_TILE(64, 64, 6)
    } else {
        AQ_TILE(64, 96, 4)
        AQ_TILE(64, 64, 4)
    }
#undef AQ_TILE
    return hipErrorInvalidConfiguration;
}

template <int KIND, int CM>
static hipError_t conv_dec(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    if (p.dec == FUSED_DEC_PK16 && p.mc == 2) return conv_tiles<KIND, CM, FUSED_DEC_PK16, 2>(geo, p, fl);
    if (p.dec == FUSED_DEC_PK16 && p.mc == 4) return conv_tiles<KIND, CM, FUSED_DEC_PK16, 4>(geo, p, fl);
    if (p.dec == FUSED_DEC_T16G) return conv_tiles<KIND, CM, FUSED_DEC_T16G, 1>(geo, p, fl);
    if (p.dec == FUSED_DEC_REC) return conv_tiles<KIND, CM, FUSED_DEC_REC, 1>(geo, p, fl);
    return hipErrorInvalidConfiguration;
}

hipError_t launch_fused_conv3(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    return conv_dec<1, 1>(geo, p, fl);
}

hipError_t launch_fused_conv1(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    return conv_dec<2, 4>(geo, p, fl);
}

}  // namespace aq
