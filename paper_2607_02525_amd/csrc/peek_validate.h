// Opt-in device-side checks of the caller's device-resident inputs.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/peek.h"

namespace peek {

// Whether the environment variable PEEK_VALIDATE asks for the checks (set,
// and not "0").
bool validation_enabled();

// With the checks on and n > 0: offsets non-decreasing from >= 0 with every
// prompt shorter than 2^31 tokens (when d_offsets != NULL), last nodes in
// [0, num_nodes) (when d_last != NULL), match lengths inside their prompts
// (when d_mlen != NULL and d_offsets != NULL). Runs on `st` and waits for it.
// INVALID_ARGUMENT names the first failed check; PEEK_OK otherwise or when
// the checks are off.
peek_status validate_queue(int32_t n, const int64_t* d_offsets, const int32_t* d_last, const int32_t* d_mlen,
                           int32_t num_nodes, hipStream_t st);

}  // namespace peek
