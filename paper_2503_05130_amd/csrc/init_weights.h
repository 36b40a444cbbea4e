// Seeded random-init spec, library side (host code).
#pragma once

#include <cstdint>

namespace iefwd {

// key of tensor (layer, slot): mix(seed XOR mix(32 * layer + slot))
uint64_t tensor_key(uint64_t seed, uint32_t layer, uint32_t slot);

// Weight matrix with logical layout [in_dim, out_dim]; written output-major
// (dst is [out_dim, in_dim] bf16).  Output columns < qk_cols use sigma_qk when it
// is non-zero.  Multi-threaded.
void generate_matrix_transposed(uint64_t key, uint32_t in_dim, uint32_t out_dim, uint32_t qk_cols,
                                double sigma, double sigma_qk, uint16_t *dst);

// bf16 vector (biases): sigma * n
void generate_vector_bf16(uint64_t key, uint32_t n, double sigma, uint16_t *dst);

// fp32 vector (LN parameters): offset + sigma * n
void generate_vector_f32(uint64_t key, uint32_t n, double offset, double sigma, float *dst);

}  // namespace iefwd
