// Exact chunk scan on the matrix cores, Temporal SwiLA (Sec. 3.3, App. B.3):
// the mode-2 instantiations of the pipelined kernel in scan_pipe_kernel.hpp.
#include "scan_pipe_kernel.hpp"

namespace swila {

hipError_t launch_scan_pipe_temporal(const LayerArgs &a, hipStream_t stream) {
    if (!a.gk || !a.gq) return hipErrorInvalidValue;
    return launch_mode<2>(a, NewtonArgs{}, stream);
}

}  // namespace swila
