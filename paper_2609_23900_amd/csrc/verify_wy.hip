// Tree WY verification on MFMA (placeholder until the kernel lands).
#include "launch.h"

namespace lumo {

hipError_t launch_wy(const lumo_gdn_dims&, const lumo_tree_desc&, const GdnArgs&, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace lumo
