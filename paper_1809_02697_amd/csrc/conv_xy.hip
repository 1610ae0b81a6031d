// Blocked convolution on fp32 MFMA (gfx950): the kernel family for every pair
// of input / output blocks other than NCHW16c -> NCHW16c (conv_kernel.h).
#include "conv_kernel.h"

namespace neo {
namespace conv_detail {

template hipError_t dispatch_all<true>(const ConvConfig&, int, bool, bool, const ConvArgs&,
                                       hipStream_t);

}  // namespace conv_detail
}  // namespace neo
