// Internal helpers shared by the host-side translation units of the library.
#pragma once

#include <stdint.h>

#include "lumo_tree.h"

namespace lumo {

// Record a printf-style message for lumo_last_error() and return `st`.
lumo_status fail(lumo_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// Seg record and seg_nodes entry widths of the plan blob.
constexpr int kSegWords = 4;      // {request, source cut, first entry, length}
constexpr int kSegNodeWords = 3;  // {absolute row, writes output, cut to export}
constexpr int kPreChunk = 32;     // preorder positions per chunk
constexpr int kPreStack = 16;     // path-stack candidate slots per chunk
constexpr int kPreCiWords = 4;    // candidate-slot words per preorder position (16 bytes)

}  // namespace lumo
