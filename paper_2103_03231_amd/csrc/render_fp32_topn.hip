// render_fp32_topn.hip - render kernels with fp32 networks and top-N placement,
// both depth-network inputs.  One translation unit per precision and
// placement so that the variants compile in parallel.
#include "render_kernel.h"

namespace donerf {

hipError_t launch_render_fp32_topn(int ncap, int din, const RenderArgs& a, dim3 grid, hipStream_t stream) {
    return launch_placement<kF32, 1, 4, 1, kPlaceTopN>(ncap, din, a, grid, stream);
}

}  // namespace donerf
