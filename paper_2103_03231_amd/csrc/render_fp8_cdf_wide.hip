// render_fp8_cdf_wide.hip - render kernels with mixed fp8 networks (bf16
// first and head layers, fp8 hidden layers) and inverse-CDF placement
// (Sec. 5.1) over 192 or 256 classes (two head sweeps), both depth-network
// inputs.
#include "render_kernel.h"

namespace donerf {

hipError_t launch_render_fp8_cdf_wide(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream) {
    return launch_placement<kFP8, kBf16CB, kBf16NW, kBf16Occ, kPlaceCdfWide>(ncap, din, a, grid, stream);
}

}  // namespace donerf
