// Internal declarations shared by the library's own sources (host API and
// kernels).  Nothing here is part of the public ABI in include/rotor.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rotor.h"

namespace rotor {

// Row of the pair (s, t), d = t - s, in a chain's table: rows are stored by
// increasing d, then by s (1-based).
__host__ __device__ inline int64_t row_of(int L, int d, int s)
{
    return (int64_t)d * L - (int64_t)d * (d - 1) / 2 + (s - 1);
}

__host__ __device__ inline int64_t pitch_of(int64_t M) { return (M + 1 + 15) / 16 * 16; }

// Everything one fill launch needs to address a batch of tables.
struct Tables {
    const int64_t *params;  // [n_chains][6][L]
    int64_t *cost;          // [n_chains][rows][pitch]
    int16_t *dec;           // same indexing
    int L;
    int M;
    int n_chains;
    int64_t pitch;
    int64_t rows;           // L(L+1)/2
};

// Enqueue the whole table fill on `stream`.  Returns a HIP error code.
hipError_t launch_fill(const Tables &tb, hipStream_t stream);

// Enqueue the sequence walk (one workgroup per budget).
hipError_t launch_reconstruct(const int64_t *params, int L, int M, int64_t pitch, int64_t rows,
                              const int16_t *dec_chain, int n_budgets, const int64_t *budgets, int64_t cap,
                              rotor_op *ops, int64_t *count, int32_t *status, hipStream_t stream);

}  // namespace rotor
