// Token-by-token SwiLA scan (Sec. 3.2: eq. recurrence, eq. responsibility,
// eq. retrieval): dispatch on the key size Dk.  The kernel and its launch rules
// are in scan_direct_kernel.hpp; each Dk is compiled in scan_direct_dk*.hip.
#include "launch.hpp"

namespace swila {

hipError_t launch_scan_direct_dk16(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_dk32(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_dk64(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_dk128(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_aux_dk16(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_aux_dk32(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_aux_dk64(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_direct_aux_dk128(const LayerArgs &a, hipStream_t stream);

hipError_t launch_scan_direct(const LayerArgs &a, hipStream_t stream) {
    switch (a.Dk) {
        case 16: return launch_scan_direct_dk16(a, stream);
        case 32: return launch_scan_direct_dk32(a, stream);
        case 64: return launch_scan_direct_dk64(a, stream);
        case 128: return launch_scan_direct_dk128(a, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_scan_direct_aux(const LayerArgs &a, hipStream_t stream) {
    if (!a.delta_out || !a.ckpt || a.gk || a.decay) return hipErrorInvalidValue;
    switch (a.Dk) {
        case 16: return launch_scan_direct_aux_dk16(a, stream);
        case 32: return launch_scan_direct_aux_dk32(a, stream);
        case 64: return launch_scan_direct_aux_dk64(a, stream);
        case 128: return launch_scan_direct_aux_dk128(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace swila
