// Runtime entry points shared by the layer runtime and the whole-model
// driver (internal: not part of the C ABI).
#pragma once

#include "hb.h"

namespace hb {

// One iteration of a stack of layers that share configuration, pool size
// and stream, over one batch: the batch is validated, planned and its
// metadata uploaded once, and every layer's kernels read that upload.
// Layer l reads x_in[l] and writes x_out[l] (bf16 or fp32 per desc).
hb_status run_layer_stack(hb_layer* const* layers, int n, const hb_batch_desc* desc, const void* const* x_in,
                          void* const* x_out);

}  // namespace hb
