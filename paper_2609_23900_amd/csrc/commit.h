// Commit entry points beyond launch_commit (launch.h).
#pragma once
#include "launch.h"

namespace lumo {

// Path derivation and conv-history publication with each layer's history and x in a
// buffer of its own (pointer tables passed by value, at most kMaxLayerTable layers).
constexpr int kMaxLayerTable = 128;
hipError_t launch_commit_hist_layers(const lumo_gdn_dims& d, const lumo_tree_desc& desc, const CommitArgs& a,
                                     const void* const* x_layers, void* const* hist_layers, hipStream_t s);

}  // namespace lumo
