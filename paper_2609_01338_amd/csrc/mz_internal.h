// Layout sizes shared by the runtime and the eviction planner (host code).
#pragma once
#include <cstdint>

#include "../../include/mz.h"

namespace mzrt {

// Device bytes of one layer's weight unit: Q, KV, O, gate/up and down
// matrices in the GEMM layout, each 256-byte aligned, the unit 4 KiB aligned.
int64_t weight_unit_bytes(const mz_model_cfg& cfg);

// Device bytes of one KV chunk slot: chunk_tokens x (K and V) x dkv halves.
int64_t kv_slot_bytes(const mz_model_cfg& cfg);

// Message returned by mz_last_error(NULL) for calls that have no context.
void set_error(const char* msg);

}  // namespace mzrt
