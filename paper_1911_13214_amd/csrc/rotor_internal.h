// Internal declarations shared by the library's own sources (host API and
// kernels).  Nothing here is part of the public ABI in include/rotor.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rotor.h"

namespace rotor {

// Row of the pair (s, t), 1 <= s <= t <= L, in a chain's table: the upper
// triangle stored s-major, so the rows (s, s), (s, s+1), ..., (s, L) are
// consecutive and the row of (s, t+1) follows the row of (s, t).
__host__ __device__ inline int64_t row_of(int L, int s, int t)
{
    return (int64_t)(s - 1) * L - (int64_t)(s - 1) * (s - 2) / 2 + (t - s);
}

// Row pitch: M + 1 rounded up to 32 elements, so that every row of the int64
// table starts 256 bytes and every row of the 4-byte compact copy 128 bytes
// (one cache line) after an aligned table base.
__host__ __device__ inline int64_t pitch_of(int64_t M) { return (M + 1 + 31) / 32 * 32; }

// Row pitch of the 2-byte copy of the diagonal blocks: a multiple of 64
// elements (128 bytes).
__host__ __device__ inline int64_t half_pitch_of(int64_t pitch) { return (pitch + 63) / 64 * 64; }

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

// Device workspace of a fill: prefix sums of u_f, per block-diagonal value
// path and packed key width and the sums they are computed from, the gates
// m_none and m_all of every pair, a compact uint32 copy of the cost table
// (written and read by the pairs whose costs stay below 2^30), and a 2-byte
// copy of the cells of the diagonal blocks (chains whose costs there stay
// below 2^15).
struct Work {
    int64_t *pre;      // [n_chains][L + 1]
    int32_t *pbits;    // [n_chains][nb], nb = ceil(L / 16): packed key bits of block-diagonal D, -1: 64-bit path
    int64_t *bsum;     // [n_chains][2][nb + 1]: sums of prefix sums of u_f, and of u_b, to block ends
    int32_t *gnone;    // [n_chains][rows]
    int32_t *gall;     // [n_chains][rows]
    uint32_t *shadow;  // [n_chains][rows][pitch]
    int16_t *half;     // [n_chains][nb][16][16][half_pitch]: 2-byte copy of the diagonal blocks' cells
};

// Byte offsets of the workspace sections (each 256-byte aligned).
struct WorkLayout {
    uint64_t pre, pbits, bsum, gnone, gall, shadow, half, total;
};
WorkLayout work_layout(int n_chains, int L, int64_t pitch);
Work work_view(void *base, int n_chains, int L, int64_t pitch);

// Kernel classes of the fill, in the order of rotor_kernel_stats.
enum KernelClass { kLeaf = 0, kDiag = 1, kMiddle = 2, kEdge = 3, kPrep = 4 };

// Work of one launch, counted exactly from its grid: C_1 candidates (split
// points times budgets), C_2 candidates and final cells written.
struct LaunchWork {
    uint64_t split_candidates;
    uint64_t all_candidates;
    uint64_t cells;
};

// Optional hooks around every launch of the fill (timing, accounting).
struct LaunchObserver {
    virtual hipError_t before(KernelClass k, hipStream_t s) = 0;
    virtual hipError_t after(KernelClass k, const LaunchWork &w, hipStream_t s) = 0;
    virtual ~LaunchObserver() {}
};

// Enqueue the whole table fill on `stream` with one of the ROTOR_SCHEDULE_*
// orders.  Returns a HIP error code.
hipError_t launch_fill(const Tables &tb, const Work &w, int schedule, hipStream_t stream,
                       LaunchObserver *obs = nullptr);

// Enqueue the sequence walk (one workgroup per budget).
hipError_t launch_reconstruct(const int64_t *params, int L, int M, int64_t pitch, int64_t rows,
                              const int16_t *dec_chain, int n_budgets, const int64_t *budgets, int64_t cap,
                              rotor_op *ops, int64_t *count, int32_t *status, hipStream_t stream);

}  // namespace rotor
