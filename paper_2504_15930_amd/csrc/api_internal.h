// Host-side entry points shared between the C ABI (api.cpp) and the decode
// engine (engine.cpp).
#pragma once

#include "../../include/sl.h"
#include "sl_internal.h"

namespace sl {

// sl_decode_attn (fp8 false) or sl_decode_attn_fp8, with the decode engine's
// staged append for the following step (next; null for none) run in the same
// launch as the merge, after the step's attention has read the cache. The
// checks and errors are those of the public calls.
sl_status decode_attn_then_append(const sl_attn_desc *d, const uint16_t *q, const void *k_pages, const void *v_pages,
                                  const float *k_scales, const float *v_scales, const int32_t *block_table,
                                  const int32_t *seq_lens, float scale, uint16_t *out, bool fp8,
                                  const AppendParams *next);

}  // namespace sl
