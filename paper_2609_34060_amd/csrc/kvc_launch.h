// Internal interface between the host entry points (kvc_api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include "kvc.h"
#include "kvc_device.h"

namespace kvc {

struct ApplyArgs {
  PoolView pv;
  LayerPtrs layers;            // pools of layers [layer_begin, layer_begin + num_layers)
  const kvc_item* items;       // device
  const int32_t* src_tables;   // device or null
  const int32_t* dst_tables;   // device or null
  int32_t max_blocks;
  int32_t layer_begin;
  int32_t num_layers;
};

int apply_chunk_tokens();
hipError_t launch_apply(const ApplyArgs& a, kvc_dtype dtype, int max_rank, int max_tokens, int num_items,
                        hipStream_t stream);

}  // namespace kvc
