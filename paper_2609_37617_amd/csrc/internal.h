// Library-internal calls between the translation units of libas2d.so
// (not part of the C ABI in include/as2d.h; hidden from the export table).
#pragma once
#include "../../include/as2d.h"

// Capture, if not yet captured, the verification graphs of one-request
// passes of 1..max_rows rows under the context's current execution mode
// and keep_logits setting (nothing is launched).  A caller that is about
// to run two contexts from two host threads calls it for both first, so
// that no graph is captured while another thread captures.
__attribute__((visibility("hidden"))) int as2d_prepare_graphs(as2d_ctx* ctx, int32_t max_rows);
