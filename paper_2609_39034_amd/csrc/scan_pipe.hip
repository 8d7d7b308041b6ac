// Exact chunk scan on the matrix cores, plain SwiLA (Sec. 3.2): the mode-0
// instantiations of the pipelined kernel in scan_pipe_kernel.hpp.
#include "scan_pipe_kernel.hpp"

namespace swila {

hipError_t launch_scan_pipe(const LayerArgs &a, hipStream_t stream) {
    if (a.gk) return launch_scan_pipe_temporal(a, stream);
    return launch_mode<0>(a, NewtonArgs{}, stream);
}

}  // namespace swila
