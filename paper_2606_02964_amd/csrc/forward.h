// forward.h -- msa_forward's body, shared by the entry points that run it.
#pragma once

#include <cstddef>
#include <cstdint>

#include "msa.h"

namespace msa {

// Checks, then the attention launch and (for split tiles) the merge launch,
// with the given workspace.  `who` names the entry point in error messages.
msa_status forward_impl(const char* who, msa_plan_t plan, const void* q, const void* k_cache,
                        const void* v_cache, const int32_t* block_table, void* o, float* lse,
                        void* workspace, size_t workspace_bytes, void* hip_stream);

// Workspace bytes a plan's msa_forward needs (plan non-null).
int64_t plan_workspace_bytes(msa_plan_t plan);

}  // namespace msa
