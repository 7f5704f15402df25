#pragma once
#include <stdint.h>

namespace ebrl {
// count elements of tensor `tensor_id`, N(0, stdv^2), bf16 bit patterns or float32.
void generate_weight(uint64_t seed, uint32_t tensor_id, int64_t count, double stdv, bool bf16,
                     void* out);
}  // namespace ebrl
