// Instantiations of the fused decode + matrix-core kernel for linear layers.
#include "aq_fused_kernel.h"

namespace aq {

template <int XT, int DEC, int MC>
static hipError_t lin_tiles(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
#define AQ_TILE(TBM, TBN, TUPL) \
    if (p.bm == TBM && p.bn == TBN && p.upl == TUPL) return fused_launch_cfg<0, 4, XT, DEC, MC, TBM, TBN, TUPL>(geo, p, fl);
    AQ_TILE(64, 96, 8)
    if (p.bm == 64 && p.bn == 64 && p.upl == 8) {
        // pre-decoded operands: two workgroups per compute unit (the tile fits 256
        // registers per lane); with the in-loop decode they would share the LDS
        // gather throughput, which measured slower
        constexpr int occ = DEC == FUSED_DEC_REC ? 2 : 1;
        return fused_launch_cfg<0, 4, XT, DEC, MC, 64, 64, 8, occ>(geo, p, fl);
    }
    AQ_TILE(32, 128, 4)
    AQ_TILE(32, 64, 4)
#undef AQ_TILE
    return hipErrorInvalidConfiguration;
}

template <int XT>
static hipError_t lin_dec(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    if (p.dec == FUSED_DEC_PK16 && p.mc == 2) return lin_tiles<XT, FUSED_DEC_PK16, 2>(geo, p, fl);
    if (p.dec == FUSED_DEC_PK16 && p.mc == 4) return lin_tiles<XT, FUSED_DEC_PK16, 4>(geo, p, fl);
    if (p.dec == FUSED_DEC_T16G) return lin_tiles<XT, FUSED_DEC_T16G, 1>(geo, p, fl);
    if (p.dec == FUSED_DEC_REC) return lin_tiles<XT, FUSED_DEC_REC, 1>(geo, p, fl);
    return hipErrorInvalidConfiguration;
}

hipError_t launch_fused_linear(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    if (fl.x_dtype == AQ_I8) return lin_dec<AQ_I8>(geo, p, fl);
    return lin_dec<AQ_F16>(geo, p, fl);
}

hipError_t launch_fused_forward(const Geom& geo, const FusedPlan& p, const FusedLaunch& fl) {
    if (p.kind == 1) return launch_fused_conv3(geo, p, fl);
    if (p.kind == 2) return launch_fused_conv1(geo, p, fl);
    return launch_fused_linear(geo, p, fl);
}

}  // namespace aq
