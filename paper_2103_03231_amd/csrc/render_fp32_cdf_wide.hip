// render_fp32_cdf_wide.hip - render kernels with fp32 networks and inverse-CDF
// placement (Sec. 5.1) over 192 or 256 classes (two head sweeps), both
// depth-network inputs.  One translation unit per precision and placement so
// that the variants compile in parallel.
#include "render_kernel.h"

namespace donerf {

hipError_t launch_render_fp32_cdf_wide(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream) {
    return launch_placement<kF32, 1, 4, 1, kPlaceCdfWide>(ncap, din, a, grid, stream);
}

}  // namespace donerf
