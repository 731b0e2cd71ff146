// Internal entry points of the host library used by other translation units
// (not part of the public interface in include/dbt.h).
#pragma once
#include <stddef.h>

#include "../../include/dbt.h"

namespace dbt {

// Sets the thread's dbt_last_error() message and returns s.
dbt_status set_error(dbt_status s, const char *msg);

// Bytes of the buffers a decode step of m writes and reads within the call
// (activations, split partials, logits and their statistics, MoE lists).
size_t step_bytes(const dbt_model *m);

// dbt_decode_step with those buffers at step_mem (at least step_bytes(m)
// device bytes, 256-byte aligned) instead of the model's workspace.
dbt_status decode_step_in(dbt_model *m, dbt_kv *kv, const dbt_step_in *in, int32_t branch_on, dbt_step_out *out,
                          dbt_stream stream, char *step_mem);

}  // namespace dbt
