// Launch interface of the aggregation, routing and streaming-state kernels (internal).
#pragma once

#include "row_features.h"

namespace pr {

using AggParamsDev = pr_agg_params;

hipError_t launch_aggregate(const pr_token_features_t& feats, const int32_t* offsets, int32_t n_req,
                            const AggParamsDev& hp, const pr_request_agg_t& out, hipStream_t stream);
hipError_t launch_route(const float* scores, int32_t n_req, float thr, uint8_t* ship, int32_t* n_ship,
                        hipStream_t stream);
// slots == NULL clears every slot.
hipError_t launch_stream_clear(const StreamDev& s, const int32_t* slots, int32_t n, hipStream_t stream);
hipError_t launch_stream_finish(const StreamDev& s, const int32_t* slots, int32_t n, const AggParamsDev& hp,
                                float thr, const pr_request_agg_t& out, uint8_t* ship, hipStream_t stream);

}  // namespace pr
