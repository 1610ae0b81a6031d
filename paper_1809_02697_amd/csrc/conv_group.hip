// Blocked convolution on fp32 MFMA (gfx950): the group kernels, several
// independent NCHW16c convolutions in one launch (conv_kernel.h).
#include "conv_kernel.h"

namespace neo {
namespace conv_detail {

hipError_t dispatch_group(const ConvConfig& c, int g, const ConvGroupArgs& ga, int wgs,
                          hipStream_t st) {
    switch (c.fk * 8 + c.fp) {
        case 1 * 8 + 1: return group_by_g<1, 1>(g, c.waves, ga, wgs, st);
        case 1 * 8 + 2: return group_by_g<1, 2>(g, c.waves, ga, wgs, st);
        case 1 * 8 + 4: return group_by_g<1, 4>(g, c.waves, ga, wgs, st);
        case 2 * 8 + 1: return group_by_g<2, 1>(g, c.waves, ga, wgs, st);
        case 2 * 8 + 2: return group_by_g<2, 2>(g, c.waves, ga, wgs, st);
        case 2 * 8 + 4: return group_by_g<2, 4>(g, c.waves, ga, wgs, st);
        case 4 * 8 + 1: return group_by_g<4, 1>(g, c.waves, ga, wgs, st);
        case 4 * 8 + 2: return group_by_g<4, 2>(g, c.waves, ga, wgs, st);
        case 4 * 8 + 4: return group_by_g<4, 4>(g, c.waves, ga, wgs, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace conv_detail
}  // namespace neo
