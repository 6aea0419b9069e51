// Two deferred WY verifications in one launch (verify_wy.hip).
#pragma once
#include "launch.h"

namespace lumo {

// Calls a and b, each as launch_wy with its pending path (the 32-column form for both,
// which gives the same bits as the 64-column one): blocks of a first, then those of b.
// Both must take the same operand preparation of queries and keys, and trees of at most
// kStack + 1 levels (hipErrorNotSupported otherwise).
hipError_t launch_wy_pair(const lumo_gdn_dims& da, const lumo_tree_desc& desca, const GdnArgs& aa, const PendArgs& pa,
                          const lumo_gdn_dims& db, const lumo_tree_desc& descb, const GdnArgs& ab, const PendArgs& pb,
                          hipStream_t s);

}  // namespace lumo
