// Host-side helpers shared by the runtime translation units.
#pragma once

#include <stdint.h>

#include <vector>

#include "dattri.h"

namespace dattri {

// The cost model in a calibration file (JSON, member "model"); values are
// not range-checked here.  INVALID_ARG with a message on any error.
dattri_status read_cost_calibration(const char* path, dattri_cost_model* out);

uint64_t derive_side_seed(uint64_t global_seed, int layer, int side);
uint64_t derive_mask_seed(uint64_t global_seed, int layer);
void mask_entries(uint64_t seed64, int d_in, int d_out, int m, int mask_id, int count,
                  std::vector<int32_t>& rows, std::vector<int32_t>& cols);
void philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
double gaussian_entry(uint64_t seed64, uint64_t e);
double rademacher_entry(uint64_t seed64, uint64_t e);  // +-1
uint16_t f32_to_bf16_rne(float f);
float bf16_to_f32(uint16_t h);
float round_to_compute(double x, int elt_bytes);
void seeded_map(uint64_t seed64, int d, int k, int elt_bytes, int kind, float* logical);
void pack_map(const float* logical, int d, int k, int elt_bytes, std::vector<uint8_t>& packed);

}  // namespace dattri
