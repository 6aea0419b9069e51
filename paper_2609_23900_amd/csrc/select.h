// Host launcher of the draft-selection kernels (arguments already validated by the
// C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lumo {

// Fused draft selection: rows x n_split blocks of four wavefronts; with n_split > 1 each
// wavefront's words go to `parts` ([rows][n_split][4][k + 1] words) and a merge kernel
// writes the outputs.
struct SelectArgs {
    const void* logits;
    int32_t rows;
    int32_t vocab;
    long ld;
    int32_t dtype;
    int32_t k;
    int32_t ties;
    int32_t n_split;
    int32_t* spine;
    int32_t* cand;
    uint64_t* parts;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t s);

}  // namespace lumo
