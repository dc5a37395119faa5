// Cross-attention variable aggregation: sequencing of its kernels and products.
#pragma once
#include "common.h"

namespace orbit {
size_t agg_saved_bytes(const orbit_agg_desc& a);
size_t agg_workspace_bytes(const orbit_agg_desc& a);
orbit_status agg_forward(const orbit_agg_desc& a, const void* tok, const orbit_agg_params& p, void* z,
                         void* saved, void* ws, size_t ws_bytes, hipStream_t s);
orbit_status agg_backward(const orbit_agg_desc& a, const void* tok, const orbit_agg_params& p, const void* saved,
                          const void* dz, void* dtok, const orbit_agg_grads& g, int accumulate, void* ws,
                          size_t ws_bytes, hipStream_t s);
}  // namespace orbit
