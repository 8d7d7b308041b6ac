// Chunkwise quasi-Newton form (App. D) on the matrix cores: the mode-1
// instantiations of the pipelined kernel in scan_pipe_kernel.hpp.
#include "scan_pipe_kernel.hpp"

namespace swila {

size_t newton_workspace_bytes(int B, int H, int T, int Dv, int J) {
    const size_t tpad = (size_t)((T + kC - 1) / kC) * kC;
    return (size_t)B * H * J * Dv * tpad * sizeof(float);
}

hipError_t launch_newton(const LayerArgs &a, const NewtonArgs &na, hipStream_t stream) {
    if (!na.pred || na.max_iters < 1) return hipErrorInvalidValue;
    if (a.gk) return hipErrorInvalidValue;   // App. D linearises the plain recurrence
    if (na.iters) {
        hipLaunchKernelGGL(int_fill_kernel, dim3(1), dim3(64), 0, stream, na.iters, 2, 0);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return launch_mode<1>(a, na, stream);
}

}  // namespace swila
