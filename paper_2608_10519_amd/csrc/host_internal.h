// Host-side pieces of the C-ABI layer (host_api.cpp) that other translation
// units of the library call.  Not part of the public interface.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/sparstar.h"

namespace sparstar {

// The selector of sparstar_score_blocks (separate pool, score and select
// kernels), except that S may live in the caller's `scores` output: with
// scores != NULL the workspace only needs the pooled blocks (the first
// regions of the sparstar_score_workspace_bytes layout).  validate_only checks
// every argument, the workspace by its size alone, and launches nothing: no
// HIP call is made.  Returns a SPARSTAR_* code and sets the thread's message.
int score_blocks_internal(const void* q, const void* k, int B, int H, int64_t Lq, int64_t Lk, int D, int block_size,
                          const double* budget, int n_budget, const sparstar_range* keep, int n_keep,
                          int32_t* kv_num_blocks, int32_t* kv_indices, int kv_stride, float* scores, void* workspace,
                          size_t workspace_bytes, void* stream, bool validate_only);

// Bytes of the pooled-block regions (qbar, kbar) at the start of the selector
// workspace; 0 for invalid sizes.
size_t score_pooled_bytes(int B, int H, int64_t Lq, int64_t Lk, int D, int block_size);

// Sets the thread's last-error message and returns `code`.
int report_error(int code, const char* msg);

}  // namespace sparstar
