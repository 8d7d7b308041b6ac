// Token-by-token scan instantiated for Dk = 16 (see scan_direct_kernel.hpp).
#include "scan_direct_kernel.hpp"

namespace swila {

hipError_t launch_scan_direct_dk16(const LayerArgs &a, hipStream_t stream) {
    return launch_dk<16>(a, stream);
}

hipError_t launch_scan_direct_aux_dk16(const LayerArgs &a, hipStream_t stream) {
    return launch_aux_dk<16>(a, stream);
}

}  // namespace swila
