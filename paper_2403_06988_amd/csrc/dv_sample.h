// Internal declarations of the masked sampling kernels (dv_sample.hip).
#pragma once

#include "dv_internal.h"

namespace dv {

// Workspace: the meeting words of rows split over blocks (row_meet_bytes
// for the launch's chunks per row; zero before the first call, left zero
// by every call).
size_t sample_workspace_bytes(int B, int V);

hipError_t launch_masked_sample(const int32_t *next_state, const uint32_t *allow, int S, int V,
                                const int32_t *states, const void *logits, int dtype, int B, int64_t ld,
                                float inv_temperature, uint64_t seed, uint64_t offset, int32_t *token,
                                int32_t *new_state, void *workspace, hipStream_t stream);

}  // namespace dv
