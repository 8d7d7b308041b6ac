// Token-by-token scan instantiated for Dk = 64 (see scan_direct_kernel.hpp).
#include "scan_direct_kernel.hpp"

namespace swila {

hipError_t launch_scan_direct_dk64(const LayerArgs &a, hipStream_t stream) {
    return launch_dk<64>(a, stream);
}

hipError_t launch_scan_direct_aux_dk64(const LayerArgs &a, hipStream_t stream) {
    return launch_aux_dk<64>(a, stream);
}

}  // namespace swila
