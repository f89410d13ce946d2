// Table fill of the optimal persistent checkpointing dynamic program
// (Theorem 1, Section 4.2 of Beaumont et al., arXiv 1911.13214) on gfx950.
//
// Wavefront over the sub-chain length d = t - s: every term of the
// recurrence for (s, t) lies on a strictly shorter sub-chain, so all cells
// of one diagonal are independent.  One launch fills one diagonal; within a
// launch a lane owns one budget m of one pair (s, t) of one chain, so the
// reads C(s, s'-1, m) and C(s', t, m - w_a^{s'-1}) of a wavefront are two
// contiguous 512-byte streams (m is the contiguous index of the table).
//
// Infinity.  The table stores INT64_MAX.  On load of a shifted operand the
// two top bits are cleared, which maps INT64_MAX to 2^62 - 1 and leaves every
// finite cost (< 2^60 in the domain) unchanged; the sum of a prefix of u_f,
// one such value and one unmasked value then cannot wrap in unsigned 64-bit
// arithmetic, and it is >= 2^62 - 1 exactly when an operand was infinite.
#include "rotor_internal.h"

namespace rotor {
namespace {

constexpr int64_t kInf = INT64_MAX;
constexpr uint64_t kInfLoaded = (1ull << 62) - 1;
constexpr uint64_t kLoadMask = (1ull << 62) - 1;
// Every finite sum of a u_f prefix and two finite costs is below 3 * 2^60;
// every sum with an infinite operand is at least 2^62 - 1.
constexpr uint64_t kFinite = 3ull << 60;
constexpr int kBlock = 256;

struct ChainRows {
    const int64_t *uf, *ub, *wa, *wabar, *of, *ob;  // stage l at index l-1
};

__device__ inline ChainRows chain_rows(const int64_t *__restrict__ params, int L, int c)
{
    const int64_t *p = params + (int64_t)c * ROTOR_N_ROWS * L;
    return {p + ROTOR_ROW_UF * L, p + ROTOR_ROW_UB * L, p + ROTOR_ROW_WA * L,
            p + ROTOR_ROW_WABAR * L, p + ROTOR_ROW_OF * L, p + ROTOR_ROW_OB * L};
}

// m_all(s, t): peak of F_all^s with delta^t stored, and of B^s with delta^s
// stored (Section 4.2; delta has the size of a).
__device__ inline int64_t gate_all(const ChainRows &r, int s, int t)
{
    int64_t fwd = r.wa[t - 1] + r.wabar[s - 1] + r.of[s - 1];
    int64_t bwd = r.wa[s - 1] + r.wabar[s - 1] + r.ob[s - 1];
    return fwd > bwd ? fwd : bwd;
}

// m_none(s, t), t > s: peak of F_ck^s and F_none^{s+1..t-1} with delta^t
// stored (Section 4.2).
__device__ inline int64_t gate_none(const ChainRows &r, int s, int t)
{
    int64_t g = r.wa[s - 1] + r.of[s - 1];
    for (int j = s + 1; j < t; ++j) {
        int64_t v = r.wa[j - 2] + r.wa[j - 1] + r.of[j - 1];
        g = v > g ? v : g;
    }
    return r.wa[t - 1] + g;
}

// Eq. (DP:Init): single-stage sub-chains (d = 0).
__global__ __launch_bounds__(kBlock) void leaf_kernel(const int64_t *__restrict__ params, int L, int M,
                                                      int64_t pitch, int64_t rows, int64_t *__restrict__ cost,
                                                      int16_t *__restrict__ dec)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int m = blockIdx.x * kBlock + threadIdx.x;
    if (m > M)
        return;
    const ChainRows r = chain_rows(params, L, c);
    const bool ok = m >= gate_all(r, s, s);
    const int64_t idx = ((int64_t)c * rows + row_of(L, 0, s)) * pitch + m;
    cost[idx] = ok ? r.uf[s - 1] + r.ub[s - 1] : kInf;
    dec[idx] = ok ? 0 : -1;
}

// Eq. (DP:mainrec) for every pair (s, s + d) of every chain.
__global__ __launch_bounds__(kBlock) void diag_kernel(const int64_t *__restrict__ params, int L, int M,
                                                      int64_t pitch, int64_t rows, int d,
                                                      int64_t *__restrict__ cost, int16_t *__restrict__ dec)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int t = s + d;
    const int m = blockIdx.x * kBlock + threadIdx.x;
    const ChainRows r = chain_rows(params, L, c);
    const int64_t g1 = gate_none(r, s, t);
    const int64_t g2 = gate_all(r, s, t);
    if (m > M)
        return;
    int64_t *tab = cost + (int64_t)c * rows * pitch;

    // C_1: min over s' = s+1..t of
    //   sum_{k=s}^{s'-1} u_f^k + C(s', t, m - w_a^{s'-1}) + C(s, s'-1, m),
    // visited in increasing s' with a strict <, so the smallest s' wins ties.
    // Step i = s' - s - 1 reads the rows (s, s+i) and (s+1+i, t); both row
    // indices move by a uniform amount per step.
    uint64_t best = kInfLoaded;
    int arg = -1;
    uint64_t prefix = 0;
    int64_t lrow = row_of(L, 0, s);          // (s, s)
    int64_t rrow = row_of(L, d - 1, s + 1);  // (s+1, t)
#pragma unroll 4
    for (int i = 0; i < d; ++i) {
        const int sp = s + 1 + i;
        prefix += (uint64_t)r.uf[sp - 2];
        const int64_t w = r.wa[sp - 2];
        const int64_t ri = (int64_t)m - w;
        const uint64_t a_raw = (uint64_t)tab[rrow * pitch + (ri >= 0 ? ri : 0)];
        const uint64_t b = (uint64_t)tab[lrow * pitch + m];
        // only the shifted operand is masked: prefix + a + b stays below 2^64
        // even when b is INT64_MAX, and is >= kFinite whenever an operand is
        // infinite or the shifted budget is negative
        const uint64_t a = ri >= 0 ? (a_raw & kLoadMask) : kInfLoaded;
        const uint64_t v = prefix + a + b;
        if (v < best) {
            best = v;
            arg = sp;
        }
        lrow += L - i;
        rrow -= L - (d - 1 - i);
    }
    if (m < g1) {
        best = kInfLoaded;
        arg = -1;
    }

    // C_2 = u_f^s + C(s+1, t, m - w_abar^s) + u_b^s, taken only if strictly
    // better (C_1 wins ties).
    const int64_t ri2 = (int64_t)m - r.wabar[s - 1];
    const uint64_t a2_raw = (uint64_t)tab[row_of(L, d - 1, s + 1) * pitch + (ri2 >= 0 ? ri2 : 0)];
    const uint64_t a2 = ri2 >= 0 ? (a2_raw & kLoadMask) : kInfLoaded;
    const uint64_t v2 = (uint64_t)(r.uf[s - 1] + r.ub[s - 1]) + a2;
    if (m >= g2 && v2 < best) {
        best = v2;
        arg = 0;
    }

    const bool finite = best < kFinite;
    const int64_t idx = row_of(L, d, s) * pitch + m;
    tab[idx] = finite ? (int64_t)best : kInf;
    dec[(int64_t)c * rows * pitch + idx] = finite ? (int16_t)arg : (int16_t)-1;
}

}  // namespace

hipError_t launch_fill(const Tables &tb, hipStream_t stream)
{
    const unsigned mblocks = (unsigned)((tb.M + 1 + kBlock - 1) / kBlock);
    leaf_kernel<<<dim3(mblocks, tb.L, tb.n_chains), kBlock, 0, stream>>>(tb.params, tb.L, tb.M, tb.pitch,
                                                                        tb.rows, tb.cost, tb.dec);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    for (int d = 1; d < tb.L; ++d) {
        diag_kernel<<<dim3(mblocks, tb.L - d, tb.n_chains), kBlock, 0, stream>>>(tb.params, tb.L, tb.M, tb.pitch,
                                                                                tb.rows, d, tb.cost, tb.dec);
        e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace rotor
