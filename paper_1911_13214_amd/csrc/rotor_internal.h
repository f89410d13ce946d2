// Internal declarations shared by the library's own sources (host API and
// kernels).  Nothing here is part of the public ABI in include/rotor.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rotor_geometry.h"

namespace rotor {

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

// Device workspace of a fill: prefix sums of u_f and of u_f + u_b, per
// block-diagonal value path and packed key width and the sums they are
// computed from, the gates m_none and m_all of every pair and the budget
// G(s, t) from which C_2 reaches the least time (rotor_fill.hip), a domain
// status word per chain, the sizes
// by which operand budgets are shifted (clamped, see prep_kernel), a compact
// uint32 copy of the cost table (written and read by the pairs whose costs
// stay below 2^32 - 1), and a 2-byte copy of the cells of the diagonal blocks
// (chains whose costs there stay below 2^15).
struct Work {
    int64_t *pre;      // [n_chains][L + 1]
    int64_t *preall;   // [n_chains][L + 1]: prefix sums of u_f + u_b
    int32_t *pbits;    // [n_chains][nb], nb = ceil(L / 16): packed key bits of block-diagonal D, -1: 64-bit path
    int64_t *bsum;     // [n_chains][2][nb + 1]: sums of prefix sums of u_f, and of u_b, to block ends
    int32_t *gnone;    // [n_chains][rows]
    int32_t *gall;     // [n_chains][rows]
    int32_t *gsat;     // [n_chains][rows]: G(s, t), clamped like the gates
    int32_t *gblk;     // [n_chains][2][nb][nb]: per block (I, I + D), D >= 1, the least G of its
                       // cells, then the largest (INT32_MAX if some row has u_f = 0); per
                       // diagonal block (D = 0) its largest G plus its largest w_a, then its
                       // largest G
    int32_t *status;   // [n_chains]: ROTOR_OK, or ROTOR_EDOMAIN if the chain's parameters are outside the domain
    int32_t *shift;    // [n_chains][2][L]: w_a and w_abar of every stage, clamped into [0, M + 1]
    uint32_t *shadow;  // [n_chains][rows][pitch]
    int16_t *half;     // [n_chains][nb][16][16][half_pitch]: 2-byte copy of the diagonal blocks' cells
};

Work work_view(void *base, int n_chains, int L, int64_t pitch);

// Whether one chain's parameters [6][L] lie in the domain of the library
// (rotor_geometry.h), decided by the 64 lanes of one wave together; every
// lane returns the same answer.  The sums are checked term by term, so no
// value can wrap them.
__device__ inline bool chain_in_domain(const int64_t *p, int L, int lane)
{
    bool bad = false;
    uint64_t suf = 0, sub = 0;
    for (int l = lane; l < L; l += 64) {
        const int64_t uf = p[ROTOR_ROW_UF * L + l], ub = p[ROTOR_ROW_UB * L + l];
        bad |= uf < 0 || ub < 0 || (uint64_t)uf >= kCostBound || (uint64_t)ub >= kCostBound;
        for (int row = ROTOR_ROW_WA; row <= ROTOR_ROW_OB; ++row) {
            const int64_t v = p[row * L + l];
            bad |= v < 0 || v >= kMaxSize;
        }
        if (!bad) {  // each term below 2^44, at most 512 terms per lane: no wrap
            suf += (uint64_t)uf;
            sub += (uint64_t)ub;
        }
    }
    for (int off = 32; off >= 1; off /= 2) {
        suf += __shfl_xor(suf, off);
        sub += __shfl_xor(sub, off);
    }
    bad = __any(bad);
    // L * suf + sub < 2^44, without overflow
    return !bad && suf < kCostBound && sub < kCostBound && suf <= (kCostBound - sub) / (uint64_t)L;
}

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
    // no more launches on s before it joins the caller's stream
    virtual hipError_t end_stream(hipStream_t s) = 0;
    virtual ~LaunchObserver() {}
};

// Enqueue the whole table fill on `stream` with one of the ROTOR_SCHEDULE_*
// orders; with side_stream, the blocked orders run the inner middle ranges
// on the device's side stream beside the edges (joined back into `stream`),
// and the observer sees those launches on that stream.  Returns a HIP error
// code.
hipError_t launch_fill(const Tables &tb, const Work &w, int schedule, hipStream_t stream,
                       LaunchObserver *obs = nullptr, bool side_stream = true);

// Edges of the blocked fill by rows: whether a block-diagonal with `blocks`
// blocks over all chains takes them, and the launch of row 16(I + 1) - a of
// its `blocks` blocks (I, I + delta) per chain (finish: the middle kernels
// finished the corners).
bool row_edges(int64_t blocks);
void launch_edge_row(int a, int blocks, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w);

// Enqueue the sequence walk (one workgroup per budget).
hipError_t launch_reconstruct(const int64_t *params, int L, int M, int64_t pitch, int64_t rows,
                              const int16_t *dec_chain, int n_budgets, const int64_t *budgets, int64_t cap,
                              rotor_op *ops, int64_t *count, int32_t *status, hipStream_t stream);

}  // namespace rotor
