// Internal entry between the C-ABI sources of librksc (not part of the public ABI).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/rksc.h"

namespace rksc {

// The verify pass of rksc_verify_forward (same validation and launches) on a
// workspace of workspace_bytes at `workspace` (256-byte aligned).
rksc_status verify_call(const rksc_weights* w, const rksc_prefix_kv* kv, const int32_t* branch_tokens,
                        int32_t n_branches, int32_t branch_len, float tau, int32_t patience, float* entropy,
                        int32_t* exit_layer, float* hidden_last, void* workspace, size_t workspace_bytes,
                        void* stream);

// Workspace bytes of that pass for this shape (the status of its shape checks).
rksc_status verify_workspace(const rksc_model_config* cfg, int32_t n_branches, int32_t branch_len, int32_t n_prefix,
                             size_t* bytes);

}  // namespace rksc
