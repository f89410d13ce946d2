// Table fill of the optimal persistent checkpointing dynamic program
// (Theorem 1, Section 4.2 of Beaumont et al., arXiv 1911.13214) on gfx950.
//
// Recurrence.  For a pair (s, t), t > s, with k = s' - 1 ranging over
// [s, t-1], option C_1 is the min over k of
//     X(s, k) + Y(k, t),   X(s, k) = sum_{j=s}^{k} u_f^j + C(s, k, m),
//                          Y(k, t) = C(k+1, t, m - w_a^k),
// a min-plus product over k, batched over the budget m; option C_2 is
// u_f^s + u_b^s + C(s+1, t, m - w_abar^s).  Every term lies on a strictly
// shorter sub-chain.
//
// Keys.  A candidate is carried as one unsigned 64-bit key
//     (value << 16) | s'
// so one unsigned min keeps the smallest value and, among equal values, the
// smallest split s' -- the tie rule of the decision table.  C_2 is keyed with
// the low field 0xFFFF, above every split, so C_1 wins ties against it.
// Finite costs are below 2^44 (the domain), a value is a prefix sum plus two
// costs (< 2^46), so finite keys are below 2^62.  A loaded cost is shifted
// into place and the high word of the shifted value clamped to 2^30: finite
// costs are unchanged and INT64_MAX becomes just above 2^62, so any key with
// an infinite operand is at least 2^62 and a sum of two keys never wraps.
//
// Schedule.  The triangle of pairs is cut into 16 x 16 blocks (I, J) of stage
// ranges S_I x S_J.  Diagonal blocks (I, I) are filled diagonal by diagonal
// (diag_kernel).  Then, block-diagonal by block-diagonal (D = J - I = 1, 2,
// ...), the split points of a block fall in three ranges:
//   middle  k in [16(I+1), 16J]: X in blocks (I, K) and Y in blocks (K, J)
//           of smaller D -- all finished, the same range for every cell of
//           the block: a register-tiled min-plus product (middle_kernel);
//   low     k in [s, 16(I+1) - 1]: Y is a cell of the same block further down;
//   high    k in [16J + 1, t - 1]: X is a cell of the same block to the left.
// The low and high ranges hold at most 30 splits per cell and are taken by
// edge_kernel in 31 steps over the block's anti-diagonals a + b = q
// (a = 16(I+1) - s low splits, b = t - 16J - 1 high splits), each step
// reading only finished cells.
#include "rotor_internal.h"

namespace rotor {
namespace {

constexpr int64_t kInf = INT64_MAX;
constexpr int kT = 16;    // block side, in stages
constexpr int kSub = 8;   // per-wave register tile side
constexpr uint64_t kKeyInf = 1ull << 62;   // keys at or above this are infinite
constexpr uint64_t kShiftedOut = 1ull << 62;  // Y key of a budget shifted below 0
constexpr uint32_t kHiClamp = 1u << 30;
constexpr uint64_t kAllLow = 0xFFFF;       // low field of a C_2 key

struct ChainRows {
    const int64_t *uf, *ub, *wa, *wabar, *of, *ob;  // stage l at index l-1
};

__device__ inline ChainRows chain_rows(const int64_t *__restrict__ params, int L, int c)
{
    const int64_t *p = params + (int64_t)c * ROTOR_N_ROWS * L;
    return {p + ROTOR_ROW_UF * L, p + ROTOR_ROW_UB * L, p + ROTOR_ROW_WA * L,
            p + ROTOR_ROW_WABAR * L, p + ROTOR_ROW_OF * L, p + ROTOR_ROW_OB * L};
}

// A stored cost shifted into the value field of a key: finite costs (< 2^44)
// become cost << 16, INT64_MAX (whose shift fills the high word) has its high
// word clamped to 2^30, i.e. becomes at least 2^62.
__device__ inline uint64_t key_of(int64_t v)
{
    const uint64_t t = (uint64_t)v << 16;
    const uint32_t hi = min((uint32_t)(t >> 32), kHiClamp);
    return ((uint64_t)hi << 32) | (uint32_t)t;
}

typedef const __attribute__((address_space(1))) int64_t *global_cptr;

// Load budget m of a table row: global address space, 32-bit byte offset
// (M < 2^28).
__device__ inline int64_t load_at(const int64_t *row, int m)
{
    return *(global_cptr)((const char *)row + (uint32_t)m * 8u);
}

// m_all(s, t): peak of F_all^s with delta^t stored, and of B^s with delta^s
// stored (Section 4.2; delta has the size of a).
__device__ inline int64_t gate_all(const ChainRows &r, int s, int t)
{
    int64_t fwd = r.wa[t - 1] + r.wabar[s - 1] + r.of[s - 1];
    int64_t bwd = r.wa[s - 1] + r.wabar[s - 1] + r.ob[s - 1];
    return fwd > bwd ? fwd : bwd;
}

// The j-term of m_none(s, t) for one j in (s, t): F_none^j with a^{j-1} and
// delta^t stored.
__device__ inline int64_t none_term(const ChainRows &r, int j)
{
    return r.wa[j - 2] + r.wa[j - 1] + r.of[j - 1];
}

// m_none(s, t), t > s, given the max of the j-terms over s < j < t (0 when
// the range is empty): peak of F_ck^s and F_none^{s+1..t-1} with delta^t
// stored (Section 4.2).
__device__ inline int64_t gate_none(const ChainRows &r, int s, int t, int64_t jmax)
{
    const int64_t first = r.wa[s - 1] + r.of[s - 1];
    return r.wa[t - 1] + (first > jmax ? first : jmax);
}

__device__ inline uint64_t umin(uint64_t a, uint64_t b) { return b < a ? b : a; }

// Final value and decision of a cell from its best key.
__device__ inline void store_cell(int64_t *cost, int16_t *dec, int64_t idx, uint64_t best)
{
    if (best >= kKeyInf) {
        cost[idx] = kInf;
        dec[idx] = -1;
    } else {
        const uint32_t low = (uint32_t)(best & 0xFFFF);
        cost[idx] = (int64_t)(best >> 16);
        dec[idx] = low == kAllLow ? (int16_t)0 : (int16_t)low;
    }
}

// Eq. (DP:Init): single-stage sub-chains.
__global__ __launch_bounds__(256) void leaf_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int64_t *__restrict__ cost,
                                                   int16_t *__restrict__ dec)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int m = blockIdx.x * 256 + threadIdx.x;
    if (m > M)
        return;
    const ChainRows r = chain_rows(params, L, c);
    const bool ok = m >= gate_all(r, s, s);
    const int64_t idx = ((int64_t)c * rows + row_of(L, s, s)) * pitch + m;
    cost[idx] = ok ? r.uf[s - 1] + r.ub[s - 1] : kInf;
    dec[idx] = ok ? 0 : -1;
}

// Eq. (DP:mainrec) for the pairs (s, s + d) of one diagonal, all splits in
// one pass; with `in_block` only pairs inside one diagonal block are done.
__global__ __launch_bounds__(256) void diag_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int d, int in_block,
                                                   int64_t *__restrict__ cost, int16_t *__restrict__ dec)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int t = s + d;
    if (in_block && (s - 1) / kT != (t - 1) / kT)
        return;
    const int m = blockIdx.x * 256 + threadIdx.x;
    const ChainRows r = chain_rows(params, L, c);
    int64_t jmax = 0;
    for (int j = s + 1; j < t; ++j) {
        const int64_t v = none_term(r, j);
        jmax = v > jmax ? v : jmax;
    }
    const int64_t g1 = gate_none(r, s, t, jmax);
    const int64_t g2 = gate_all(r, s, t);
    if (m > M)
        return;
    const int64_t *tab = cost + (int64_t)c * rows * pitch;

    // C_1, splits in increasing s'; rows (s, s'-1) are consecutive, the row of
    // (s'+1, t) is L - s' rows after the row of (s', t).
    uint64_t best = ~0ull;
    uint64_t prefix = 0;
    const int64_t *left = tab + row_of(L, s, s) * pitch;
    const int64_t *right = tab + row_of(L, s + 1, t) * pitch;
#pragma unroll 4
    for (int sp = s + 1; sp <= t; ++sp) {
        prefix += (uint64_t)r.uf[sp - 2];
        const int64_t w = r.wa[sp - 2];
        const int ri = m - (int)w;
        const uint64_t x = key_of(load_at(left, m)) + (ri >= 0 ? ((prefix << 16) | (uint64_t)sp) : kShiftedOut);
        const uint64_t y = key_of(load_at(right, ri >= 0 ? ri : 0));
        best = umin(best, x + y);
        left += pitch;
        right += (int64_t)(L - sp) * pitch;
    }
    if (m < g1)
        best = ~0ull;
    if (m >= g2) {
        const int ri = m - (int)r.wabar[s - 1];
        if (ri >= 0) {
            const uint64_t v = key_of(load_at(tab + row_of(L, s + 1, t) * pitch, ri));
            best = umin(best, v + (((uint64_t)(r.uf[s - 1] + r.ub[s - 1]) << 16) | kAllLow));
        }
    }
    const int64_t idx = ((int64_t)c * rows + row_of(L, s, t)) * pitch + m;
    store_cell(cost, dec, idx, best);
}

// Middle splits of every block (I, I + D) of one block-diagonal.  A workgroup
// is one block at 64 budgets; its four waves hold the four 8 x 8 quarters of
// the block, one key per pair and lane.  For each middle split k the wave
// loads X for its 8 rows and Y for its 8 columns (the waves sharing rows or
// columns hit the same lines in L1/L2) and updates 64 keys; two register sets
// alternate so the loads of split k+1 are in flight during the updates of k.
// The prefix of u_f starts at the first middle split; edge_kernel adds the
// part from s.  Keys are stored in the cost table, where edge_kernel finishes
// the cells.
struct MiddleTile {
    const int64_t *xrow[kSub];  // row (s0 + i, k)
    const int64_t *yrow;        // row (k + 1, t0)
    int64_t ystep[kSub];        // row of (k + 1, t0 + j) relative to yrow
    int mc;
};

__device__ inline void middle_load(const MiddleTile &tl, int ri, int64_t (&rx)[kSub], int64_t (&ry)[kSub])
{
#pragma unroll
    for (int i = 0; i < kSub; ++i)
        rx[i] = load_at(tl.xrow[i], tl.mc);
#pragma unroll
    for (int j = 0; j < kSub; ++j)
        ry[j] = load_at(tl.yrow + tl.ystep[j], ri >= 0 ? ri : 0);
}

__device__ inline void middle_update(uint64_t (&key)[kSub][kSub], const int64_t (&rx)[kSub],
                                     const int64_t (&ry)[kSub], uint64_t pk)
{
    uint64_t x[kSub], y[kSub];
#pragma unroll
    for (int i = 0; i < kSub; ++i)
        x[i] = key_of(rx[i]) + pk;
#pragma unroll
    for (int j = 0; j < kSub; ++j)
        y[j] = key_of(ry[j]);
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j)
            key[i][j] = umin(key[i][j], x[i] + y[j]);
}

__global__ __launch_bounds__(256) void middle_kernel(const int64_t *__restrict__ params, int L, int M,
                                                     int64_t pitch, int64_t rows, int delta,
                                                     int64_t *__restrict__ cost)
{
    const int c = blockIdx.z;
    const int I = blockIdx.y;
    const int J = I + delta;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int m = blockIdx.x * 64 + lane;
    const int s0 = I * kT + (wave >> 1) * kSub + 1;
    const int t0 = J * kT + (wave & 1) * kSub + 1;
    if (t0 > L)
        return;
    const int nt = min(kSub, L - t0 + 1);
    const ChainRows r = chain_rows(params, L, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    const int k_lo = (I + 1) * kT;
    const int k_hi = J * kT;

    // X row of (s0 + i, k) advances one row per k; Y rows of (k+1, t0 + j) are
    // j rows after the row of (k+1, t0), which advances L - k - 1 rows per k.
    // Columns past L (last block) read the last valid column.
    MiddleTile tl;
#pragma unroll
    for (int i = 0; i < kSub; ++i)
        tl.xrow[i] = tab + row_of(L, s0 + i, k_lo) * pitch;
#pragma unroll
    for (int j = 0; j < kSub; ++j)
        tl.ystep[j] = (int64_t)(j < nt ? j : nt - 1) * pitch;
    tl.yrow = tab + row_of(L, k_lo + 1, t0) * pitch;
    tl.mc = m <= M ? m : M;
    auto advance = [&](int k) {  // from split k to k + 1
#pragma unroll
        for (int i = 0; i < kSub; ++i)
            tl.xrow[i] += pitch;
        tl.yrow += (int64_t)(L - k - 1) * pitch;
    };

    uint64_t key[kSub][kSub];
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j)
            key[i][j] = ~0ull;

    // a budget shifted below 0 makes every candidate of the split infinite:
    // it is folded into the constant added to X
    uint64_t prefix = 0;
    auto pk_of = [&](int k, int ri) {
        prefix += (uint64_t)r.uf[k - 1];
        return ri >= 0 ? ((prefix << 16) | (uint64_t)(k + 1)) : kShiftedOut;
    };
    int64_t ax[kSub], ay[kSub], bx[kSub], by[kSub];
    int k = k_lo;
    int ra = tl.mc - (int)r.wa[k - 1];
    middle_load(tl, ra, ax, ay);
    for (; k + 1 <= k_hi; k += 2) {
        advance(k);
        const int rb = tl.mc - (int)r.wa[k];
        middle_load(tl, rb, bx, by);
        middle_update(key, ax, ay, pk_of(k, ra));
        if (k + 2 <= k_hi) {
            advance(k + 1);
            ra = tl.mc - (int)r.wa[k + 1];
            middle_load(tl, ra, ax, ay);
        }
        middle_update(key, bx, by, pk_of(k + 1, rb));
    }
    if (k == k_hi)
        middle_update(key, ax, ay, pk_of(k, ra));

    if (m > M)
        return;
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j)
            if (j < nt)
                tab[row_of(L, s0 + i, t0 + j) * pitch + m] = (int64_t)key[i][j];
}

// Sum (uf over [k_lo, k_hi]) and max (m_none j-terms over (s, t)) across
// the workgroup.
__device__ inline void block_reduce(uint64_t &sum, int64_t &mx)
{
    __shared__ uint64_t s_sum[4];
    __shared__ int64_t s_max[4];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        sum += (uint64_t)__shfl_xor((long long)sum, off);
        const int64_t o = (int64_t)__shfl_xor((long long)mx, off);
        mx = o > mx ? o : mx;
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        s_sum[wave] = sum;
        s_max[wave] = mx;
    }
    __syncthreads();
    sum = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    mx = s_max[0];
#pragma unroll
    for (int w = 1; w < 4; ++w)
        mx = s_max[w] > mx ? s_max[w] : mx;
}

// Edge splits, C_2 and the gates for the cells a + b = q of every block
// (I, I + D) of one block-diagonal; a workgroup is one cell at 256 budgets.
__global__ __launch_bounds__(256) void edge_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int delta, int q, int a_min,
                                                   int n_q, int64_t *__restrict__ cost, int16_t *__restrict__ dec)
{
    const int c = blockIdx.z;
    const int blk = blockIdx.y / n_q;
    const int a = a_min + (blockIdx.y - blk * n_q);
    const int b = q - a;
    const int I = blk;
    const int J = I + delta;
    const int s = (I + 1) * kT - a;
    const int t = J * kT + 1 + b;
    if (t > L)
        return;  // the whole workgroup, before any barrier
    const int k_lo = (I + 1) * kT;
    const int k_hi = J * kT;
    const ChainRows r = chain_rows(params, L, c);

    uint64_t mid_sum = 0;  // sum of u_f over the middle splits
    int64_t jmax = 0;      // max of the m_none j-terms over (s, t)
    for (int j = k_lo + (int)threadIdx.x; j <= k_hi; j += 256)
        mid_sum += (uint64_t)r.uf[j - 1];
    for (int j = s + 1 + (int)threadIdx.x; j < t; j += 256) {
        const int64_t v = none_term(r, j);
        jmax = v > jmax ? v : jmax;
    }
    block_reduce(mid_sum, jmax);

    const int m = blockIdx.x * 256 + threadIdx.x;
    if (m > M)
        return;
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    const int64_t cell = row_of(L, s, t) * pitch + m;

    // low splits k = s .. k_lo - 1: X from block (I, I), Y from this block
    uint64_t best = ~0ull;
    uint64_t prefix = 0;
    const int64_t *xr = tab + row_of(L, s, s) * pitch;
    const int64_t *yr = tab + row_of(L, s + 1, t) * pitch;
    for (int k = s; k < k_lo; ++k) {
        prefix += (uint64_t)r.uf[k - 1];
        const int ri = m - (int)r.wa[k - 1];
        const uint64_t x = key_of(load_at(xr, m)) + (ri >= 0 ? ((prefix << 16) | (uint64_t)(k + 1)) : kShiftedOut);
        const uint64_t y = key_of(load_at(yr, ri >= 0 ? ri : 0));
        best = umin(best, x + y);
        xr += pitch;
        yr += (int64_t)(L - k - 1) * pitch;
    }
    // middle splits: the stored key counts u_f from k_lo on
    best = umin(best, (uint64_t)load_at(tab + row_of(L, s, t) * pitch, m) + (prefix << 16));
    // high splits k = 16J + 1 .. t - 1: X from this block, Y from block (J, J)
    prefix += mid_sum;
    xr = tab + row_of(L, s, k_hi + 1) * pitch;
    yr = tab + row_of(L, k_hi + 2, t) * pitch;
    for (int k = k_hi + 1; k < t; ++k) {
        prefix += (uint64_t)r.uf[k - 1];
        const int ri = m - (int)r.wa[k - 1];
        const uint64_t x = key_of(load_at(xr, m)) + (ri >= 0 ? ((prefix << 16) | (uint64_t)(k + 1)) : kShiftedOut);
        const uint64_t y = key_of(load_at(yr, ri >= 0 ? ri : 0));
        best = umin(best, x + y);
        xr += pitch;
        yr += (int64_t)(L - k - 1) * pitch;
    }
    if (m < gate_none(r, s, t, jmax))
        best = ~0ull;
    if (m >= gate_all(r, s, t)) {
        const int ri = m - (int)r.wabar[s - 1];
        if (ri >= 0) {
            const uint64_t v = key_of(load_at(tab + row_of(L, s + 1, t) * pitch, ri));
            best = umin(best, v + (((uint64_t)(r.uf[s - 1] + r.ub[s - 1]) << 16) | kAllLow));
        }
    }
    store_cell(tab, dec + (int64_t)c * rows * pitch, cell, best);
}

hipError_t check() { return hipGetLastError(); }

// Pairs (s, s + d) inside one diagonal block of side kT, over all blocks.
uint64_t in_block_pairs(int L, int d)
{
    uint64_t n = 0;
    for (int b0 = 0; b0 < L; b0 += kT) {
        const int len = min(kT, L - b0);
        if (len > d)
            n += (uint64_t)(len - d);
    }
    return n;
}

}  // namespace

hipError_t launch_fill(const Tables &tb, hipStream_t stream, LaunchObserver *obs)
{
    const int L = tb.L;
    const uint64_t W = (uint64_t)tb.M + 1;
    const uint64_t nc = (uint64_t)tb.n_chains;
    const unsigned mb256 = (unsigned)((tb.M + 1 + 255) / 256);
    const unsigned mb64 = (unsigned)((tb.M + 1 + 63) / 64);
    auto launched = [&](KernelClass k, uint64_t c1, uint64_t c2, uint64_t cells) -> hipError_t {
        hipError_t e = check();
        if (e == hipSuccess && obs)
            e = obs->after(k, LaunchWork{c1 * W * nc, c2 * W * nc, cells * W * nc}, stream);
        return e;
    };
    auto before = [&](KernelClass k) -> hipError_t { return obs ? obs->before(k, stream) : hipSuccess; };
    hipError_t e;

    if ((e = before(kLeaf)) != hipSuccess)
        return e;
    leaf_kernel<<<dim3(mb256, L, tb.n_chains), 256, 0, stream>>>(tb.params, L, tb.M, tb.pitch, tb.rows, tb.cost,
                                                                 tb.dec);
    if ((e = launched(kLeaf, 0, 0, (uint64_t)L)) != hipSuccess)
        return e;
    // diagonal blocks
    for (int d = 1; d < kT && d < L; ++d) {
        if ((e = before(kDiag)) != hipSuccess)
            return e;
        diag_kernel<<<dim3(mb256, L - d, tb.n_chains), 256, 0, stream>>>(tb.params, L, tb.M, tb.pitch, tb.rows, d,
                                                                         1, tb.cost, tb.dec);
        const uint64_t pairs = in_block_pairs(L, d);
        if ((e = launched(kDiag, pairs * d, pairs, pairs)) != hipSuccess)
            return e;
    }
    const int nb = (L + kT - 1) / kT;
    for (int delta = 1; delta < nb; ++delta) {
        // pairs of the block-diagonal: full rows of 16, columns up to L
        uint64_t pairs = 0;
        for (int I = 0; I + delta < nb; ++I)
            pairs += (uint64_t)kT * (uint64_t)min(kT, L - (I + delta) * kT);
        if ((e = before(kMiddle)) != hipSuccess)
            return e;
        middle_kernel<<<dim3(mb64, nb - delta, tb.n_chains), 256, 0, stream>>>(tb.params, L, tb.M, tb.pitch,
                                                                               tb.rows, delta, tb.cost);
        if ((e = launched(kMiddle, pairs * (uint64_t)((delta - 1) * kT + 1), 0, 0)) != hipSuccess)
            return e;
        for (int q = 0; q <= 2 * kT - 2; ++q) {
            const int a_min = q - (kT - 1) > 0 ? q - (kT - 1) : 0;
            const int a_max = q < kT - 1 ? q : kT - 1;
            const int n_q = a_max - a_min + 1;
            uint64_t cells = 0;
            for (int I = 0; I + delta < nb; ++I)
                for (int a = a_min; a <= a_max; ++a)
                    cells += ((I + delta) * kT + 1 + (q - a) <= L) ? 1 : 0;
            if ((e = before(kEdge)) != hipSuccess)
                return e;
            edge_kernel<<<dim3(mb256, (nb - delta) * n_q, tb.n_chains), 256, 0, stream>>>(
                tb.params, L, tb.M, tb.pitch, tb.rows, delta, q, a_min, n_q, tb.cost, tb.dec);
            if ((e = launched(kEdge, cells * (uint64_t)q, cells, cells)) != hipSuccess)
                return e;
        }
    }
    return hipSuccess;
}

}  // namespace rotor
