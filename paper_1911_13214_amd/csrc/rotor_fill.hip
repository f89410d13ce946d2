// Table fill of the optimal persistent checkpointing dynamic program
// (Theorem 1, Section 4.2 of Beaumont et al., arXiv 1911.13214) on gfx950.
//
// Recurrence.  For a pair (s, t), t > s, with k = s' - 1 ranging over
// [s, t-1], option C_1 is the min over k of
//     X(s, k) + Y(k, t),   X(s, k) = sum_{j=s}^{k} u_f^j + C(s, k, m),
//                          Y(k, t) = C(k+1, t, m - w_a^k),
// a min-plus product over k, batched over the budget m; option C_2 is
// u_f^s + u_b^s + C(s+1, t, m - w_abar^s).  Every term lies on a strictly
// shorter sub-chain.  Ties go to the smallest s', then to C_1 over C_2.
//
// Saturated budgets.  No schedule of [s, t] takes less than its least time
// LT(s, t) = sum_{j=s}^{t} (u_f^j + u_b^j), every stage forward once and
// backward once, so C >= LT.  C_2 reaches it when m >= m_all(s, t) and
// C(s+1, t, m - w_abar^s) = LT(s+1, t); with G(t, t) = m_all(t, t) and
// G(s, t) = max(m_all(s, t), G(s+1, t) + w_abar^s), induction on t - s
// gives C(s, t, m) = LT(s, t) for every m >= G(s, t).  A C_1 candidate runs
// stages s .. s'-1 forward twice, so it is at least LT(s, t) + u_f^s: when
// u_f^s > 0 the decision there is C_2 alone.  prep_kernel writes G for every
// pair, and a workgroup whose budgets are all at or above G(s, t) (with
// u_f^s > 0) stores LT(s, t) and C_2 without loading an operand: the result
// the relaxation would reach, at the cost of the stores.
//
// Value paths, chosen per block-diagonal by prep_kernel from a bound on
// every finite cost: stage j runs forward at most t - j + 1 times in any
// schedule of the family for [s, t] (induction on the recurrence), so
// V(s, t) = sum_{j=s}^{t} (t - j + 1) u_f^j + sum_{j=s}^{t} u_b^j bounds
// every C_1 or C_2 candidate of the pair, being the time of such a schedule.
// V grows with the sub-chain, so V_D, V over the longest sub-chains of the
// 16 x 16 blocks of block-diagonal D (D = 0: within one block), bounds every
// pair of the block-diagonal and grows with D; a pair's operands are
// sub-chains of it, of block-diagonals up to its own.
//  - narrow, when V_D < 2^32 - 1: operands are read from a compact uint32
//    copy of the table (INT64_MAX stored as 0xFFFFFFFF), which the pairs of
//    narrow block-diagonals write, and added with unsigned saturation (a
//    finite candidate is at most V_D, below the infinity, so no finite sum
//    saturates); the best value and its split are kept side by side and
//    splits are visited in increasing s' with a strict <;
//  - packed (middle products of narrow block-diagonals, when (V_D + 1) << S
//    fits below 2^32 - 1 for the S bits of the block's middle split range):
//    a candidate is one uint32 key (value << S) | (s' - first middle split),
//    so one saturating add and one unsigned min relax it, ties going to the
//    smaller split.  When the range needs more bits than V_D leaves, but at
//    least 7, it is relaxed in runs of 2^S splits, each with its own first
//    split, and the runs' results are merged as (value << 32) | s';
//  - wide, otherwise: operands are the int64 cells and a candidate is one
//    64-bit key (value << 16) | s', so one unsigned min keeps the smallest
//    value and, among equal values, the smallest split.  Finite values are
//    below 2^46 (domain bound 2^44 on costs); a loaded cost is shifted into
//    place with its high word clamped to 2^30, so INT64_MAX lands just above
//    2^62 and a sum of two keys never wraps.
// C_2 is given the split field 0xFFFF (above every split), so C_1 wins ties.
// When V_0 <= 2^15 - 2, the cells of the diagonal blocks are also kept in a
// 2-byte copy (infinity -1), which a sign-extending load turns back into the
// 4-byte form: the pairs inside a block and the edge splits read their
// diagonal-block operands from it.
//
// Schedule.  The triangle of pairs is cut into 16 x 16 blocks (I, J) of stage
// ranges S_I x S_J.  Diagonal blocks (I, I) are filled diagonal by diagonal
// (diag_kernel).  Then, block-diagonal by block-diagonal (D = J - I = 1, 2,
// ...), the split points of a block fall in three ranges:
//   middle  k in [16(I+1), 16J]: X in blocks (I, K) and Y in blocks (K, J)
//           of smaller D -- all finished, the same range for every cell of
//           the block: a register-tiled min-plus product (middle_packed_kernel,
//           operands staged in LDS, for packed keys and runs of them, or
//           middle_kernel for the others);
//   low     k in [s, 16(I+1) - 1]: Y is a cell of the same block further down;
//   high    k in [16J + 1, t - 1]: X is a cell of the same block to the left.
// The low and high ranges hold at most 30 splits per cell and are taken by
// edge_kernel in 30 steps over the block's anti-diagonals a + b = q = 1..30
// (a = 16(I+1) - s low splits, b = t - 16J - 1 high splits), each step
// reading only finished cells; the corner a + b = 0 has neither and is
// finished by the middle kernels.  The middle splits whose operands lie in
// block-diagonals up to D - 2 (all but the first and the last 16) need
// nothing of D - 1: they run on a second stream beside the edges of D - 1
// (latency-bound waves beside VALU-bound ones), and the remaining 32 follow
// those edges, merged by atomic minimum.  A small table is instead filled in the
// streamed order: one launch per diagonal d over all its pairs (diag_kernel,
// or diag_split_kernel with the splits of a pair spread over four waves).
#include <mutex>
#include <type_traits>

#include "rotor_paths.h"

namespace rotor {
namespace {

// The automatic schedule fills small tables diagonal by diagonal: measured on
// MI355X, that is faster up to about 2e9 split candidates for one chain
// (L = 250 at M = 500) and 4e8 for a batch, whose blocked launches are wider,
// and for any single chain with fewer than 64 budgets, which leave most lanes
// of the blocked kernels' 64-budget chunks idle (L = 3000, M = 31: 229
// against 269 ms).
constexpr uint64_t kStreamMaxCandidates1 = 2000000000ull;
constexpr uint64_t kStreamMaxCandidatesN = 400000000ull;
constexpr int kStreamBelowBudgets = 64;
constexpr int kSplitMinD = 16;  // streamed diagonals from this length spread their splits over four waves

// ---------------------------------------------------------------------------

// Gates of every pair, prefix sums of u_f, and the value path and packed key
// width of every block-diagonal.
// Workgroup s - 1 of a chain writes the gate row of s, 64 consecutive t per
// step: m_all(s, t) (peak of F_all^s with delta^t stored, and of B^s with
// delta^s stored) and m_none(s, t) (peak of F_ck^s and F_none^{s+1..t-1} with
// delta^t stored), Section 4.2; delta has the size of a.  The maximum over
// s < j < t in m_none is a running maximum along t: a wave prefix maximum
// per step plus the carry of the steps before.  Workgroup s - 1 also writes
// the saturation budgets G(s, t) of its row (head of this file), from two
// more running maxima along t.  Gates above INT32_MAX are
// clamped: any gate above M < 2^28 is never met.  Workgroup s - 1 also
// writes the shift sizes w_a^s and w_abar^s clamped into [0, M + 1] (see
// ChainRows).  The last workgroup of a chain checks its parameters against
// the domain, scans u_f and u_f + u_b with one wave and bounds the costs of
// each block-diagonal.
__global__ __launch_bounds__(64) void prep_kernel(const int64_t *__restrict__ params, int L, int M, int64_t rows,
                                                  Work w)
{
    const int c = blockIdx.y;
    const int lane = threadIdx.x;
    const ChainParams r = chain_params(params, L, c);
    auto clamp32 = [](int64_t v) { return (int32_t)(v < INT32_MAX ? v : INT32_MAX); };
    if (blockIdx.x == gridDim.x - 1) {
        // the chain's domain status, which rotor_solve_status reports: the
        // fill stays in bounds outside the domain, but its tables are then
        // unspecified
        const bool in_domain = chain_in_domain(params + (int64_t)c * ROTOR_N_ROWS * L, L, lane);
        if (lane == 0)
            w.status[c] = in_domain ? ROTOR_OK : ROTOR_EDOMAIN;
        // prefix sums of u_f and of u_f + u_b: lane l sums a segment of
        // stages, then the segment sums are scanned
        const int seg = (L + 63) / 64;
        const int lo = min(L, lane * seg), hi = min(L, lo + seg);
        uint64_t su = 0, sa = 0;
        for (int l = lo; l < hi; ++l) {
            su += (uint64_t)r.uf[l];
            sa += (uint64_t)r.uf[l] + (uint64_t)r.ub[l];
        }
        uint64_t incl = su, incla = sa;
        for (int off = 1; off < 64; off *= 2) {
            const uint64_t v = __shfl_up(incl, off), va = __shfl_up(incla, off);
            if (lane >= off) {
                incl += v;
                incla += va;
            }
        }
        int64_t *pre = w.pre + (int64_t)c * (L + 1);
        int64_t *preall = w.preall + (int64_t)c * (L + 1);
        uint64_t run = incl - su, runa = incla - sa;
        for (int l = lo; l < hi; ++l) {
            run += (uint64_t)r.uf[l];
            runa += (uint64_t)r.uf[l] + (uint64_t)r.ub[l];
            pre[l + 1] = (int64_t)run;
            preall[l + 1] = (int64_t)runa;
        }
        if (lane == 0) {
            pre[0] = 0;
            preall[0] = 0;
        }
        // Value path and packed key width of every block-diagonal D from V_D,
        // the largest over I of V over [16I + 1, min(16(I + D + 1), L)].  With
        // PP and B the sums of P and of u_b up to a stage,
        // V(x + 1, y) = sum_{l=x+1}^{y} (P[l] - P[x]) + B[y] - B[x]
        //             = PP[y] - PP[x] - (y - x) P[x] + B[y] - B[x];
        // bsum keeps PP and B at the block ends min(16b, L), b = 0..nb.
        const int nb = (L + kT - 1) / kT;
        int32_t *pb = w.pbits + (int64_t)c * nb;
        int64_t *ppb = w.bsum + (int64_t)c * 2 * (nb + 1);
        int64_t *bb = ppb + (nb + 1);
        __syncthreads();  // pre[] of every lane written
        for (int b = 1 + lane; b <= nb; b += 64) {
            const int bhi = min(b * kT, L);
            int64_t sP = 0, sB = 0;
            for (int l = (b - 1) * kT + 1; l <= bhi; ++l) {
                sP += pre[l];
                sB += r.ub[l - 1];
            }
            ppb[b] = sP;
            bb[b] = sB;
        }
        __syncthreads();
        // block sums -> sums up to the block ends, 64 blocks per step
        int64_t carry_p = 0, carry_b = 0;
        for (int b0 = 1; b0 <= nb; b0 += 64) {
            const int b = b0 + lane;
            int64_t vp = b <= nb ? ppb[b] : 0, vb = b <= nb ? bb[b] : 0;
            for (int off = 1; off < 64; off *= 2) {
                const int64_t up = __shfl_up(vp, off), ub = __shfl_up(vb, off);
                if (lane >= off) {
                    vp += up;
                    vb += ub;
                }
            }
            vp += carry_p;
            vb += carry_b;
            if (b <= nb) {
                ppb[b] = vp;
                bb[b] = vb;
            }
            carry_p = __shfl(vp, 63);
            carry_b = __shfl(vb, 63);
        }
        if (lane == 0) {
            ppb[0] = 0;
            bb[0] = 0;
        }
        __syncthreads();
        for (int D = lane; D < nb; D += 64) {
            int64_t vmax = 0;  // below 2^45 in the domain
            for (int I = 0; I + D < nb; ++I) {
                const int x = I * kT, yb = I + D + 1, y = min(yb * kT, L);
                vmax = max(vmax, ppb[yb] - ppb[I] - (int64_t)(y - x) * pre[x] + bb[yb] - bb[I]);
            }
            // (V_D + 1) << S <= 2^32 - 1 leaves S >= 0 bits on the narrow path;
            // -2 marks a 64-bit block-diagonal whose middle keys are exact as
            // doubles, -1 the others
            int bits = (uint64_t)vmax < kNarrowBound
                           ? 63 - __clzll((long long)(0xFFFFFFFFull / ((uint64_t)vmax + 1)))
                           : (uint64_t)vmax < kF64Bound ? -2 : -1;
            // D = 0 has no middle products; its width only says whether the
            // 2-byte copy of the diagonal blocks is used (>= 17), which only
            // the edges of a chain of two blocks or more read
            if (D == 0 && nb < 2)
                bits = min(bits, 16);
            pb[D] = bits;
        }
        return;
    }
    const int s = blockIdx.x + 1;
    if (lane == 0) {
        auto clamp_shift = [&](int64_t v) { return (int32_t)(v < 0 ? 0 : v > (int64_t)M + 1 ? (int64_t)M + 1 : v); };
        int32_t *sh = w.shift + (int64_t)c * 2 * L;
        sh[s - 1] = clamp_shift(r.wa[s - 1]);
        sh[L + s - 1] = clamp_shift(r.wabar[s - 1]);
    }
    int32_t *gn = w.gnone + (int64_t)c * rows;
    int32_t *ga = w.gall + (int64_t)c * rows;
    int32_t *gs = w.gsat + (int64_t)c * rows;
    // The last row s = 16(I + 1) of a block I holds the least G of each
    // block (I, J), J > I (G(s, t) >= G(s + 1, t) in the domain), and its
    // first row s = 16I + 1 the largest: reduced per block J in LDS.
    __shared__ int32_t seg[(ROTOR_MAX_L + kT - 1) / kT];
    const int nb = (L + kT - 1) / kT;
    const int I = (s - 1) / kT;
    const bool last_row = s % kT == 0 && I + 1 < nb, first_row = s % kT == 1;
    if (last_row || first_row) {
        for (int J = lane; J < nb; J += 64)
            seg[J] = last_row ? INT32_MAX : INT32_MIN;
        __syncthreads();
    }
    const int64_t first = r.wa[s - 1] + r.of[s - 1];
    const int64_t bwd = r.wa[s - 1] + r.wabar[s - 1] + r.ob[s - 1];
    const int64_t fpart = r.wabar[s - 1] + r.of[s - 1];
    int64_t carry = 0;  // max over s < j < t0 of w_a^{j-1} + w_a^j + o_f^j
    // G(s, t) = max over s <= j <= t of m_all(j, t) + R(j), with
    // R(j) = sum_{s <= i < j} w_abar^i and m_all(j, t) = max(w_a^t + A_j, B_j),
    // A_j = w_abar^j + o_f^j, B_j = w_a^j + w_abar^j + o_b^j: so
    // G(s, t) = max(w_a^t + max_j (A_j + R(j)), max_j (B_j + R(j))), two
    // running maxima along t like the one of m_none (-1: none yet; every term
    // is >= 0 in the domain)
    int64_t car_r = 0, car_a = -1, car_b = -1;
    int64_t row = row_of(L, s, s);
    for (int t0 = s; t0 <= L; t0 += 64, row += 64) {
        const int t = t0 + lane;
        const bool in = t <= L;
        // the term of j = t - 1, which m_none(s, t) includes when s < t - 1
        int64_t incl = in && t >= s + 2 ? r.wa[t - 3] + r.wa[t - 2] + r.of[t - 2] : 0;
        const int64_t wab_t = in ? r.wabar[t - 1] : 0;
        int64_t rsum = wab_t;  // becomes sum_{t0 <= i <= t} w_abar^i
        for (int off = 1; off < 64; off *= 2) {
            const int64_t v = __shfl_up(incl, off), vr = __shfl_up(rsum, off);
            if (lane >= off) {
                incl = max(incl, v);
                rsum += vr;
            }
        }
        const int64_t rt = car_r + rsum - wab_t;  // R(t)
        int64_t ma = in ? wab_t + r.of[t - 1] + rt : -1;
        int64_t mb = in ? r.wa[t - 1] + wab_t + r.ob[t - 1] + rt : -1;
        for (int off = 1; off < 64; off *= 2) {
            const int64_t va = __shfl_up(ma, off), vb = __shfl_up(mb, off);
            if (lane >= off) {
                ma = max(ma, va);
                mb = max(mb, vb);
            }
        }
        ma = max(car_a, ma);
        mb = max(car_b, mb);
        const int64_t jmax = max(carry, incl);
        if (in) {
            const int64_t wt = r.wa[t - 1];
            const int32_t g = clamp32(max(wt + ma, mb));
            ga[row + lane] = clamp32(max(wt + fpart, bwd));
            gn[row + lane] = t > s ? clamp32(wt + max(first, jmax)) : 0;
            gs[row + lane] = g;
            const int J = (t - 1) / kT;
            if (last_row && J > I)
                atomicMin(&seg[J], g);
            if (first_row)
                atomicMax(&seg[J], g);
        }
        carry = max(carry, __shfl(incl, 63));
        car_r += __shfl(rsum, 63);
        car_a = __shfl(ma, 63);
        car_b = __shfl(mb, 63);
    }
    if (last_row || first_row) {
        __syncthreads();
        // the largest G bounds the block only where every row has u_f > 0
        const int rows_i = min(kT, L - I * kT);
        bool pos = true;
        int64_t wmax = 0;
        for (int i = 0; i < rows_i; ++i) {
            pos = pos && r.uf[I * kT + i] > 0;
            wmax = max(wmax, r.wa[I * kT + i]);
        }
        int32_t *gb = w.gblk + ((int64_t)c * 2 + (first_row ? 1 : 0)) * nb * nb + (int64_t)I * nb;
        for (int J = I + 1 + lane; J < nb; J += 64)
            gb[J - I] = first_row && !pos ? INT32_MAX : seg[J];
        if (first_row && lane == 0) {
            // the diagonal block I (D = 0): its largest G (values only, any
            // u_f), and that plus the largest w_a of its stages in the other
            // plane
            gb[0] = seg[I];
            w.gblk[(int64_t)c * 2 * nb * nb + (int64_t)I * nb] = clamp32((int64_t)seg[I] + wmax);
        }
    }
}

// Eq. (DP:Init): single-stage sub-chains.
__global__ __launch_bounds__(256) void leaf_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int64_t *__restrict__ cost,
                                                   int16_t *__restrict__ dec, Work w)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int m = blockIdx.x * 256 + threadIdx.x;
    if (m > M)
        return;
    const ChainRows r = chain_rows(params, w, L, c);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    const int64_t row = row_of(L, s, s);
    const bool ok = m >= cw.gall[row];
    const int64_t idx = row * pitch + m;
    const int64_t v = r.uf[s - 1] + r.ub[s - 1];
    cost[(int64_t)c * rows * pitch + idx] = ok ? v : kInf;
    dec[(int64_t)c * rows * pitch + idx] = ok ? 0 : -1;
    if (cw.narrow(0))
        cw.shadow[idx] = ok ? (uint32_t)v : kInf32;
    if (cw.diag16())
        cw.half_row(s, s)[m] = ok ? (int16_t)v : (int16_t)-1;
}

// Row cursor of a run of splits of one pair (s, t): the X row (s, k) and the
// Y row (k+1, t) of the next split k, as byte addresses in the table the
// value path reads.  From split k to k + 1 the X row moves one row and the Y
// row L - k - 1 rows; `ystep` holds the latter, in bytes, and shrinks by one
// row per split.
struct RowCursor {
    const char *x;
    const char *y;
    int64_t ystep;
    int64_t row_bytes;
};

template <class P>
__device__ __forceinline__ RowCursor row_cursor(const int64_t *tab, const uint32_t *shadow, int L, int64_t pitch,
                                                int s, int t, int k)
{
    const char *base = P::table(tab, shadow);
    const int64_t rb = pitch * P::kBytes;
    return {base + row_of(L, s, k) * rb, base + row_of(L, k + 1, t) * rb, (int64_t)(L - k - 1) * rb, rb};
}

// Relax the N consecutive splits k = k0 .. k0 + N - 1 at the cursor and
// advance it.  Straight-line code: every load is issued before the first
// relaxation, so their latencies overlap.
template <class P, int N>
__device__ __forceinline__ void relax_fixed(typename P::Acc &acc, const ChainRows &r, int m, int k0, RowCursor &cur,
                                            uint64_t &prefix)
{
    typename P::Raw rx[N], ry[N];
    int ri[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int w = r.wa[k0 + i - 1];
        ri[i] = m - w;
        rx[i] = P::load_at(cur.x, m);
        // a budget shifted below 0 reads budget 0; xop discards the candidate
        ry[i] = P::load_off(cur.y, shifted_off<P::kBytes>((uint32_t)m * P::kBytes, w));
        cur.x += cur.row_bytes;
        cur.y += cur.ystep;
        cur.ystep -= cur.row_bytes;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
        P::relax(acc, P::xop(rx[i], prefix, (uint32_t)(k + 1), ri[i] >= 0), P::yop(ry[i]), (uint32_t)(k + 1));
    }
}

// The same for a run of n <= N splits (n uniform): one branch picks the
// straight-line body of that length.
template <class P, int N>
struct RelaxRun {
    __device__ __forceinline__ static void go(int n, typename P::Acc &acc, const ChainRows &r, int m, int k0,
                                              RowCursor &cur, uint64_t &prefix)
    {
        if (n == N)
            relax_fixed<P, N>(acc, r, m, k0, cur, prefix);
        else
            RelaxRun<P, N - 1>::go(n, acc, r, m, k0, cur, prefix);
    }
};
template <class P>
struct RelaxRun<P, 0> {
    __device__ __forceinline__ static void go(int, typename P::Acc &, const ChainRows &, int, int, RowCursor &,
                                              uint64_t &)
    {
    }
};

template <class P>
__device__ __forceinline__ void relax_run(typename P::Acc &acc, const ChainRows &r, int m, int k0, int n,
                                          RowCursor &cur, uint64_t &prefix)
{
    RelaxRun<P, kT - 1>::go(n, acc, r, m, k0, cur, prefix);
}

// relax_fixed for NB budgets m[0..NB) of one lane: the loads of every split
// and budget are issued first.
template <class P, int N, int NB>
__device__ __forceinline__ void relax_fixed_nb(typename P::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                               int k0, RowCursor &cur, uint64_t &prefix)
{
    typename P::Raw rx[N][NB], ry[N][NB];
    int wa[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        wa[i] = r.wa[k0 + i - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            rx[i][b] = P::load_at(cur.x, m[b]);
            ry[i][b] = P::load_off(cur.y, shifted_off<P::kBytes>((uint32_t)m[b] * P::kBytes, wa[i]));
        }
        cur.x += cur.row_bytes;
        cur.y += cur.ystep;
        cur.ystep -= cur.row_bytes;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b)
            P::relax(acc[b], P::xop(rx[i][b], prefix, (uint32_t)(k + 1), m[b] >= wa[i]), P::yop(ry[i][b]),
                     (uint32_t)(k + 1));
    }
}

template <class P, int N, int NB>
struct RelaxRunNB {
    __device__ __forceinline__ static void go(int n, typename P::Acc (&acc)[NB], const ChainRows &r,
                                              const int (&m)[NB], int k0, RowCursor &cur, uint64_t &prefix)
    {
        if (n == N)
            relax_fixed_nb<P, N, NB>(acc, r, m, k0, cur, prefix);
        else
            RelaxRunNB<P, N - 1, NB>::go(n, acc, r, m, k0, cur, prefix);
    }
};
template <class P, int NB>
struct RelaxRunNB<P, 0, NB> {
    __device__ __forceinline__ static void go(int, typename P::Acc (&)[NB], const ChainRows &, const int (&)[NB], int,
                                              RowCursor &, uint64_t &)
    {
    }
};

// n <= kT - 1 splits from k0 for NB budgets, in straight-line runs of up to
// 8 splits: longer runs of 4-byte operands would hold more registers than the
// runs from the 2-byte copy (101 against 78 VGPRs for the edge kernel).
template <class P, int NB>
__device__ __forceinline__ void relax_run_nb(typename P::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                             int k0, int n, RowCursor &cur, uint64_t &prefix)
{
    constexpr int kRun = 8;
    for (; n > 0; n -= kRun, k0 += kRun)
        RelaxRunNB<P, kRun, NB>::go(n < kRun ? n : kRun, acc, r, m, k0, cur, prefix);
}

// relax_fixed_nb for a run whose X (CX) or Y (!CX) operands are saturated
// rows (head of this file): each is the least time of its pair at every
// budget here, pa[k] - pa_s (X = (s, k), pa_s = pa[s - 1]) or pa_s - pa[k]
// (Y = (k + 1, t), pa_s = pa[t]), so only the other operand is loaded.  The
// cursor moves as in relax_fixed_nb.
template <class P, bool CX, int N, int NB>
__device__ __forceinline__ void relax_sat_fixed_nb(typename P::Acc (&acc)[NB], const ChainRows &r,
                                                   const int (&m)[NB], int k0, RowCursor &cur, uint64_t &prefix,
                                                   const_i64 pa, int64_t pa_s)
{
    typename P::Raw rv[N][NB], c[N];
    int wa[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        wa[i] = r.wa[k - 1];
        c[i] = (typename P::Raw)(CX ? pa[k] - pa_s : pa_s - pa[k]);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            rv[i][b] = CX ? P::load_off(cur.y, shifted_off<P::kBytes>((uint32_t)m[b] * P::kBytes, wa[i]))
                          : P::load_at(cur.x, m[b]);
        }
        cur.x += cur.row_bytes;
        cur.y += cur.ystep;
        cur.ystep -= cur.row_bytes;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const typename P::Raw rx = CX ? c[i] : rv[i][b], ry = CX ? rv[i][b] : c[i];
            P::relax(acc[b], P::xop(rx, prefix, (uint32_t)(k + 1), m[b] >= wa[i]), P::yop(ry), (uint32_t)(k + 1));
        }
    }
}

template <class P, bool CX, int N, int NB>
struct RelaxSatRunNB {
    __device__ __forceinline__ static void go(int n, typename P::Acc (&acc)[NB], const ChainRows &r,
                                              const int (&m)[NB], int k0, RowCursor &cur, uint64_t &prefix,
                                              const_i64 pa, int64_t pa_s)
    {
        if (n == N)
            relax_sat_fixed_nb<P, CX, N, NB>(acc, r, m, k0, cur, prefix, pa, pa_s);
        else
            RelaxSatRunNB<P, CX, N - 1, NB>::go(n, acc, r, m, k0, cur, prefix, pa, pa_s);
    }
};
template <class P, bool CX, int NB>
struct RelaxSatRunNB<P, CX, 0, NB> {
    __device__ __forceinline__ static void go(int, typename P::Acc (&)[NB], const ChainRows &, const int (&)[NB], int,
                                              RowCursor &, uint64_t &, const_i64, int64_t)
    {
    }
};

// relax_run_nb with saturated X (CX) or Y operands, in runs of 8 splits
template <class P, bool CX, int NB>
__device__ __forceinline__ void relax_sat_run_nb(typename P::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                                 int k0, int n, RowCursor &cur, uint64_t &prefix, const_i64 pa,
                                                 int64_t pa_s)
{
    constexpr int kRun = 8;
    for (; n > 0; n -= kRun, k0 += kRun)
        RelaxSatRunNB<P, CX, kRun, NB>::go(n < kRun ? n : kRun, acc, r, m, k0, cur, prefix, pa, pa_s);
}

// Cursor of a narrow run whose X and Y rows come from different copies: X
// moves xstep bytes per split, Y ystep bytes, and ystep shrinks by ydec.
struct MixedCursor {
    const char *x;
    const char *y;
    int64_t xstep;
    int64_t ystep;
    int64_t ydec;
};

// relax_fixed for a MixedCursor: N consecutive splits k0 .. k0 + N - 1, all
// loads issued first.
template <class XL, class YL, int N>
__device__ __forceinline__ void relax_mixed(Narrow::Acc &acc, const ChainRows &r, int m, int k0, MixedCursor &cur,
                                            uint64_t &prefix)
{
    uint32_t rx[N], ry[N];
    int ri[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int w = r.wa[k0 + i - 1];
        ri[i] = m - w;
        rx[i] = XL::at(cur.x, m);
        // a budget shifted below 0 reads budget 0; xop discards the candidate
        ry[i] = YL::at_off(cur.y, shifted_off<YL::kBytes>((uint32_t)m * YL::kBytes, w));
        cur.x += cur.xstep;
        cur.y += cur.ystep;
        cur.ystep -= cur.ydec;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
        Narrow::relax(acc, Narrow::xop(rx[i], prefix, 0, ri[i] >= 0), ry[i], (uint32_t)(k + 1));
    }
}

template <class XL, class YL, int N>
struct MixedRun {
    __device__ __forceinline__ static void go(int n, Narrow::Acc &acc, const ChainRows &r, int m, int k0,
                                              MixedCursor &cur, uint64_t &prefix)
    {
        if (n == N)
            relax_mixed<XL, YL, N>(acc, r, m, k0, cur, prefix);
        else
            MixedRun<XL, YL, N - 1>::go(n, acc, r, m, k0, cur, prefix);
    }
};
template <class XL, class YL>
struct MixedRun<XL, YL, 0> {
    __device__ __forceinline__ static void go(int, Narrow::Acc &, const ChainRows &, int, int, MixedCursor &,
                                              uint64_t &)
    {
    }
};

// relax_mixed for NB budgets m[0..NB) of one lane: the loads of every split
// and budget are issued first.
template <class XL, class YL, int N, int NB>
__device__ __forceinline__ void relax_mixed_nb(Narrow::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                               int k0, MixedCursor &cur, uint64_t &prefix)
{
    uint32_t rx[N][NB], ry[N][NB];
    int wa[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        wa[i] = r.wa[k0 + i - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            rx[i][b] = XL::at(cur.x, m[b]);
            ry[i][b] = YL::at_off(cur.y, shifted_off<YL::kBytes>((uint32_t)m[b] * YL::kBytes, wa[i]));
        }
        cur.x += cur.xstep;
        cur.y += cur.ystep;
        cur.ystep -= cur.ydec;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b)
            Narrow::relax(acc[b], Narrow::xop(rx[i][b], prefix, 0, m[b] >= wa[i]), ry[i][b], (uint32_t)(k + 1));
    }
}

template <class XL, class YL, int N, int NB>
struct MixedRunNB {
    __device__ __forceinline__ static void go(int n, Narrow::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                              int k0, MixedCursor &cur, uint64_t &prefix)
    {
        if (n == N)
            relax_mixed_nb<XL, YL, N, NB>(acc, r, m, k0, cur, prefix);
        else
            MixedRunNB<XL, YL, N - 1, NB>::go(n, acc, r, m, k0, cur, prefix);
    }
};
template <class XL, class YL, int NB>
struct MixedRunNB<XL, YL, 0, NB> {
    __device__ __forceinline__ static void go(int, Narrow::Acc (&)[NB], const ChainRows &, const int (&)[NB], int,
                                              MixedCursor &, uint64_t &)
    {
    }
};

// relax_mixed_nb for a run whose X (CX) or Y (!CX) operands are saturated
// rows (head of this file): each is the least time of its pair at every
// budget here, pa[k] - pa_s (X = (s, k), pa_s = pa[s - 1]) or pa_s - pa[k]
// (Y = (k + 1, t), pa_s = pa[t]), so only the other operand is loaded.  The
// cursor moves as in relax_mixed_nb.
template <class XL, class YL, bool CX, int N, int NB>
__device__ __forceinline__ void relax_mixed_sat_nb(Narrow::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                                   int k0, MixedCursor &cur, uint64_t &prefix, const_i64 pa,
                                                   int64_t pa_s)
{
    uint32_t rv[N][NB], c[N];
    int wa[N];
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        wa[i] = r.wa[k - 1];
        c[i] = (uint32_t)(CX ? pa[k] - pa_s : pa_s - pa[k]);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if constexpr (CX)
                rv[i][b] = YL::at_off(cur.y, shifted_off<YL::kBytes>((uint32_t)m[b] * YL::kBytes, wa[i]));
            else
                rv[i][b] = XL::at(cur.x, m[b]);
        }
        cur.x += cur.xstep;
        cur.y += cur.ystep;
        cur.ystep -= cur.ydec;
    }
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const int k = k0 + i;
        prefix += (uint64_t)r.uf[k - 1];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const uint32_t rx = CX ? c[i] : rv[i][b], ry = CX ? rv[i][b] : c[i];
            Narrow::relax(acc[b], Narrow::xop(rx, prefix, 0, m[b] >= wa[i]), ry, (uint32_t)(k + 1));
        }
    }
}

template <class XL, class YL, bool CX, int N, int NB>
struct MixedSatRunNB {
    __device__ __forceinline__ static void go(int n, Narrow::Acc (&acc)[NB], const ChainRows &r, const int (&m)[NB],
                                              int k0, MixedCursor &cur, uint64_t &prefix, const_i64 pa, int64_t pa_s)
    {
        if (n == N)
            relax_mixed_sat_nb<XL, YL, CX, N, NB>(acc, r, m, k0, cur, prefix, pa, pa_s);
        else
            MixedSatRunNB<XL, YL, CX, N - 1, NB>::go(n, acc, r, m, k0, cur, prefix, pa, pa_s);
    }
};
template <class XL, class YL, bool CX, int NB>
struct MixedSatRunNB<XL, YL, CX, 0, NB> {
    __device__ __forceinline__ static void go(int, Narrow::Acc (&)[NB], const ChainRows &, const int (&)[NB], int,
                                              MixedCursor &, uint64_t &, const_i64, int64_t)
    {
    }
};

// Eq. (DP:mainrec) for one pair (s, t), all splits in straight-line runs of
// up to kT - 1.  Rows (s, s'-1) are consecutive; the row of (s'+1, t) is
// L - s' rows after the row of (s', t).  With H (a pair inside a diagonal
// block, narrow path, ChainWork::diag16) every operand comes from the 2-byte
// copy, where the rows (s'+1, t) are 16 rows apart.
template <class P, bool H, int NB>
__device__ __forceinline__ void diag_body(const ChainRows &r, const ChainWork &cw, int L, int M, int m0, int64_t pitch,
                                          int s, int t, bool sat, int64_t *tab, int16_t *dtab)
{
    const int64_t cell = row_of(L, s, t);
    // the final stores of budget set b, with the 2-byte copy of a diagonal
    // block's cell
    auto store = [&](int b, const typename P::Acc &a) {
        const int mb = m0 + b * kEdgeThreads;
        if (mb <= M) {
            store_cell<P>(tab, dtab, cw.shadow, cell * pitch + mb, a);
            if constexpr (P::kShadow) {
                if (cw.diag16() && block_diag(s, t) == 0)
                    cw.half_row(s, t)[mb] = P::finite(a) ? (int16_t)P::value(a) : (int16_t)-1;
            }
        }
    };
    // every budget of the workgroup saturated
    if (sat) {
        const typename P::Acc a = P::all_only(least_time(cw, s, t));
#pragma unroll
        for (int b = 0; b < NB; ++b)
            store(b, a);
        return;
    }
    // the lane's budgets m0 + b * kEdgeThreads; those past M load budget M
    // and store nothing
    int m[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        m[b] = min(m0 + b * kEdgeThreads, M);
    // the C_2 operand first (the lane's own budget when it is out of reach)
    const int wab = r.wabar[s - 1];
    const int32_t gall = cw.gall[cell];
    const int64_t below = row_of(L, s + 1, t) * pitch;
    typename P::Raw c2[NB];
    bool all_ok[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int ri = m[b] - wab;
        all_ok[b] = m[b] >= gall && ri >= 0;
        if constexpr (H)
            c2[b] = Load16::at((const char *)cw.half_row(s + 1, t), all_ok[b] ? ri : m[b]);
        else
            c2[b] = P::load(tab + below, cw.shadow + below, all_ok[b] ? ri : m[b]);
    }
    typename P::Acc acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        P::init(acc[b]);
    uint64_t prefix = 0;
    if constexpr (H) {
        const int64_t hb = cw.hpitch * 2;
        MixedCursor cur{(const char *)cw.half_row(s, s), (const char *)cw.half_row(s + 1, t), hb, kT * hb, 0};
        MixedRunNB<Load16, Load16, kT - 1, NB>::go(t - s, acc, r, m, s, cur, prefix);  // t - s <= 15
    } else {
        RowCursor cur = row_cursor<P>(tab, cw.shadow, L, pitch, s, t, s);
        relax_run_nb<P, NB>(acc, r, m, s, t - s, cur, prefix);
    }
    const int32_t gnone = cw.gnone[cell];
    const uint64_t ufub = (uint64_t)(r.uf[s - 1] + r.ub[s - 1]);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (m[b] < gnone)
            P::init(acc[b]);
        if (all_ok[b])
            P::relax_all(acc[b], c2[b], ufub);
        store(b, acc[b]);
    }
}

// The pairs (s, s + d): inside the 16 x 16 diagonal blocks only (blocked
// fill), or all of them (streamed fill of a small table, one launch per d).
// NB budgets per lane: kDiagBudgets for the diagonal blocks of the blocked
// order, kEdgeBudgets for the streamed order (small tables, where more and
// smaller workgroups are faster).
template <int NB>
__global__ __launch_bounds__(kEdgeThreads) void diag_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int d, int whole,
                                                   int64_t *__restrict__ cost, int16_t *__restrict__ dec, Work w)
{
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int t = s + d;
    if (!whole && (s - 1) / kT != (t - 1) / kT)
        return;
    const int m0 = blockIdx.x * (kEdgeThreads * NB) + threadIdx.x;
    if (m0 > M)
        return;
    const ChainRows r = chain_rows(params, w, L, c);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    int16_t *dtab = dec + (int64_t)c * rows * pitch;
    const int D = block_diag(s, t);
    // the path and the saturation test first: their scalar loads go together
    const bool narrow = cw.narrow(D), d16 = cw.diag16();
    const bool sat = saturated(r, cw, s, row_of(L, s, t), blockIdx.x * (kEdgeThreads * NB));
    if (!narrow)
        diag_body<Wide, false, NB>(r, cw, L, M, m0, pitch, s, t, sat, tab, dtab);
    else if (D == 0 && d16)
        diag_body<Narrow, true, NB>(r, cw, L, M, m0, pitch, s, t, sat, tab, dtab);
    else
        diag_body<Narrow, false, NB>(r, cw, L, M, m0, pitch, s, t, sat, tab, dtab);
}

// Streamed order for the longer diagonals: the d splits of each pair are
// spread over the four waves of a workgroup (one pair, 64 budgets), wave w
// taking the w-th quarter in increasing order; wave 0 then folds the four
// results in split order (so ties still go to the smallest split), adds C_2
// and the gates, and writes the cell.  Four times the waves of diag_kernel,
// each with a quarter of the dependent loads.
template <class P>
__device__ __forceinline__ void diag_split_body(const ChainRows &r, const ChainWork &cw, int L, int M, int m,
                                                int64_t pitch, int s, int t, int wave, bool sat, int64_t (*part)[64],
                                                int64_t *tab, int16_t *dtab)
{
    const int mc = m <= M ? m : M;  // lanes past M load in bounds and store nothing
    const int lane = threadIdx.x & 63;
    const int64_t cell = row_of(L, s, t);
    // every budget of the workgroup saturated (the same test in its four
    // waves, so all of them leave before the barrier)
    if (sat) {
        if (wave == 0 && m <= M)
            store_cell<P>(tab, dtab, cw.shadow, cell * pitch + m, P::all_only(least_time(cw, s, t)));
        return;
    }
    const int d = t - s;
    const int chunk = (d + 3) / 4;
    const int k0 = s + wave * chunk;
    const int k1 = min(t - 1, k0 + chunk - 1);
    typename P::Acc acc;
    P::init(acc);
    if (k0 <= k1) {
        uint64_t prefix = (uint64_t)(cw.pre[k0 - 1] - cw.pre[s - 1]);
        RowCursor cur = row_cursor<P>(tab, cw.shadow, L, pitch, s, t, k0);
        for (int kk = k0; kk <= k1; kk += kT - 1)
            relax_run<P>(acc, r, mc, kk, min(kT - 1, k1 - kk + 1), cur, prefix);
    }
    part[wave][lane] = P::stored(acc);
    __syncthreads();
    if (wave != 0 || m > M)
        return;
#pragma unroll
    for (int v = 1; v < 4; ++v)
        P::merge_later(acc, part[v][lane]);
    const int ri = m - r.wabar[s - 1];
    const bool all_ok = m >= cw.gall[cell] && ri >= 0;
    const int64_t below = row_of(L, s + 1, t) * pitch;
    const typename P::Raw c2 = P::load(tab + below, cw.shadow + below, all_ok ? ri : m);
    if (m < cw.gnone[cell])
        P::init(acc);
    if (all_ok)
        P::relax_all(acc, c2, (uint64_t)(r.uf[s - 1] + r.ub[s - 1]));
    store_cell<P>(tab, dtab, cw.shadow, cell * pitch + m, acc);
}

__global__ __launch_bounds__(256) void diag_split_kernel(const int64_t *__restrict__ params, int L, int M,
                                                         int64_t pitch, int64_t rows, int d,
                                                         int64_t *__restrict__ cost, int16_t *__restrict__ dec,
                                                         Work w)
{
    __shared__ int64_t part[4][64];
    const int c = blockIdx.z;
    const int s = blockIdx.y + 1;
    const int t = s + d;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int m = blockIdx.x * 64 + (threadIdx.x & 63);
    const ChainRows r = chain_rows(params, w, L, c);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    int16_t *dtab = dec + (int64_t)c * rows * pitch;
    const bool narrow = cw.narrow(block_diag(s, t));
    const bool sat = saturated(r, cw, s, row_of(L, s, t), blockIdx.x * 64);
    if (narrow)
        diag_split_body<Narrow>(r, cw, L, M, m, pitch, s, t, wave, sat, part, tab, dtab);
    else
        diag_split_body<Wide>(r, cw, L, M, m, pitch, s, t, wave, sat, part, tab, dtab);
}

// The corner cell (16I + 16, 16J + 1) of a block (I, J) has no low or high
// splits: its middle result, whose u_f prefix starts at its own s, is its
// whole C_1.  The middle kernels finish it (gates, C_2, final stores), so the
// edge rounds start at a + b = 1.
template <class P>
__device__ inline void finish_corner(const ChainRows &r, const ChainWork &cw, int L, int m, int64_t pitch, int s,
                                     int t, typename P::Acc acc, int64_t *tab, int16_t *dtab)
{
    const int64_t cell = row_of(L, s, t);
    const int ri = m - r.wabar[s - 1];
    const bool all_ok = m >= cw.gall[cell] && ri >= 0;
    const int64_t below = row_of(L, s + 1, t) * pitch;
    const typename P::Raw c2 = P::load(tab + below, cw.shadow + below, all_ok ? ri : m);
    if (m < cw.gnone[cell])
        P::init(acc);
    if (all_ok)
        P::relax_all(acc, c2, (uint64_t)(r.uf[s - 1] + r.ub[s - 1]));
    store_cell<P>(tab, dtab, cw.shadow, cell * pitch + m, acc);
}



// Middle splits of every block (I, I + D) of one block-diagonal
// (middle_packed_kernel, middle_kernel).  A workgroup is one block at 64
// budgets; its four waves hold the four 8 x 8 quarters of the block, one
// accumulator per pair and lane.  For each middle split k the 16 X rows and
// 16 Y rows of the block at the workgroup's budgets are copied into LDS
// (each row fetched once per workgroup), and each wave relaxes its 64
// accumulators with its 8 X and 8 Y operands.  The prefix of u_f starts at
// the first middle split; the edges add the part from s.
//
// Packed middle products.  With S the bit width of
// k - k_lo, a loaded value v becomes v << S by a rotation that leaves
// 0xFFFFFFFF (infinity) unchanged; X also gets (prefix << S) | (k - k_lo) by
// a saturating add, Y nothing more, so a candidate is sat(x + y) and the
// minimum key is the smallest value with, among equal values, the smallest
// split.  A budget shifted below 0 turns the X term of that lane into
// infinity.  The partial key is left in the compact copy of the cell for
// edge_kernel to merge.
__device__ inline uint32_t rot_left(uint32_t v, int S) { return __builtin_amdgcn_alignbit(v, v, (32 - S) & 31); }

// Workgroups are handed to the 8 XCDs in turn (workgroup b of the grid, x
// fastest, to XCD b mod 8), and each XCD has its own L2.  xcd_tile renumbers
// them so that each XCD runs a contiguous range of tiles: neighbouring budget
// chunks of one pair range, whose shifted reads share cache lines, then meet
// in the same L2.
constexpr int kXcds = 8;
struct Tile {
    int x, y, z;
};
__device__ inline Tile xcd_tile()
{
    const int nx = gridDim.x, ny = gridDim.y;
    const int n = nx * ny * gridDim.z;
    const int b = (blockIdx.z * ny + blockIdx.y) * nx + blockIdx.x;
    const int xcd = b % kXcds, slot = b / kXcds;
    const int q = n / kXcds, r = n % kXcds;
    const int id = xcd < r ? xcd * (q + 1) + slot : r * (q + 1) + (xcd - r) * q + slot;
    return {id % nx, (id / nx) % ny, id / (nx * ny)};
}

// The packed kernel stages its operands in LDS.  A stage is kStage splits;
// for each, a slot holds the block's 16 X rows and 16 Y rows at the
// workgroup's 64 budgets (8 KB).  A ring of kRing stages keeps the next
// stage in flight while the current one is relaxed.  Each wave copies 8 of
// the 32 rows of a split straight from global memory into LDS
// (global_load_lds_dword, no registers held), so each row is fetched once
// per workgroup instead of once per wave that uses it; the waves read their
// 8 + 8 operands from LDS.  Two splits per stage let one three-way unsigned
// min fold two candidates into an accumulator.  Measured on MI355X: a ring
// of two such stages (32 KB, four workgroups per CU) beats deeper rings and
// single-split stages.
constexpr int kStage = 2;
constexpr int kRing = 2;
constexpr int kSplitWords = 2 * kT * 64;
constexpr int kDmaPerSplit = 8;  // row copies per wave and split
constexpr int kDmaPerStage = kDmaPerSplit * kStage;
static_assert(kRing >= 2 && (kRing - 2) * kDmaPerStage <= 63, "vmcnt holds at most 63");
// Stages of the packed kernel issue fewer copies where operand rows are
// saturated, so its ring waits for all of them (vmcnt(0)): two stages.
static_assert(kRing == 2, "middle_packed_kernel counts on a ring of two stages");

typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void global_void;

// Wait until at most N of this wave's vector memory operations are
// outstanding and its LDS reads are done, then meet the workgroup.
template <int N>
__device__ __forceinline__ void ring_barrier()
{
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// ring_barrier leaving the copies of the next `later` stages outstanding
// (later uniform, at most kRing - 2)
template <int A>
__device__ __forceinline__ void ring_wait(int later)
{
    if constexpr (A == 0) {
        ring_barrier<0>();
    } else {
        if (later >= A)
            ring_barrier<A * kDmaPerStage>();
        else
            ring_wait<A - 1>(later);
    }
}

// Whether the middle products of block (I, J) at the 64 budgets from `base`
// are needed by no cell: every cell of the block is saturated (head of this
// file) at every budget of the edge workgroups that hold those budgets, from
// the first budget of a 128-budget edge workgroup on (the row edges' 64-budget
// workgroups start no lower), so the edges store least times there without
// reading a middle partial.  prep_kernel keeps the largest G of each block,
// or INT32_MAX when some row has u_f = 0.  Uniform over the workgroup.
__device__ inline bool block_saturated(const ChainWork &cw, int I, int J, int base)
{
    return (base & ~(kEdgeThreads * kEdgeBudgets - 1)) >= block_gmax(cw, I, J - I);
}

// The corner cell of block (I, J) at budget m when its block is saturated:
// the least time and C_2, stored by the middle kernel that finishes corners.
template <class P>
__device__ inline void store_saturated_corner(const ChainWork &cw, int L, int m, int64_t pitch, int I, int J,
                                              int64_t *tab, int16_t *dtab)
{
    const int s = (I + 1) * kT, t = J * kT + 1;
    store_cell<P>(tab, dtab, cw.shadow, row_of(L, s, t) * pitch + m, P::all_only(least_time(cw, s, t)));
}

// The partial slots of the cells of every block of block-diagonal delta, set
// to infinity before a cut middle range merges into them: the packed key in
// the compact copy, or the stored form in the cost table.
__global__ __launch_bounds__(256) void fill_partials_kernel(int L, int M, int64_t pitch, int64_t rows, int delta,
                                                            int64_t *__restrict__ cost, Work w)
{
    const int c = blockIdx.z;
    const int I = blockIdx.y / (kT * kT);
    const int cell = blockIdx.y - I * (kT * kT);
    const int s = I * kT + 1 + cell / kT;
    const int t = (I + delta) * kT + 1 + cell % kT;
    const int m = blockIdx.x * 256 + threadIdx.x;
    if (t > L || m > M)
        return;
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    if (middle_packed(cw, delta, (delta - 1) * kT))
        cw.shadow[row_of(L, s, t) * pitch + m] = kInf32;
    else
        cost[((int64_t)c * rows + row_of(L, s, t)) * pitch + m] = -1;  // all ones: above every stored form
}

// Saturated operand rows of the middle products (head of this file): a row
// whose budgets here (shifted by w_a^k for Y) all lie at or above its G holds
// its least time at each of them, which the wave can write into the ring
// instead of copying the row.  X rows (first + i, k), i < 8, are all
// saturated when the first is (G(s, k) >= G(s + 1, k)); the wave takes that
// for the splits ka .. kx, up to the first that is not.  Y rows (k + 1, t),
// t = first .. first + 7 (at most L), for the splits ky .. kb, from the last
// that is not: G(k + 1, t) falls as k grows.  Both bounds are found once,
// 64 splits per step; wa_v holds the clamped w_a of the chain.
__device__ inline void saturated_splits(const ChainWork &cw, const int32_t *wa_v, int L, bool copies_x, int first,
                                        int ka, int kb, int base, int lane, int &kx, int &ky)
{
    kx = ka - 1;
    ky = kb + 1;
    const int first_c = min(first, L);
    if (copies_x) {
        const int32_t *g_row = cw.gsat + row_of(L, first, ka);  // G(first, k) at g_row[k - ka]
        for (int k0 = ka; k0 <= kb; k0 += 64) {
            const int k = k0 + lane;
            const uint64_t bad = __ballot(k <= kb && g_row[k - ka] > base);
            if (bad) {
                kx = k0 + __ffsll((long long)bad) - 2;
                break;
            }
            kx = min(kb, k0 + 63);
        }
    } else {
        for (int k0 = kb; k0 >= ka; k0 -= 64) {
            const int k = k0 - lane;
            bool bad = false;
            if (k >= ka) {
                const int32_t *g = cw.gsat + row_of(L, k + 1, first_c);
                int32_t gm = g[0];
#pragma unroll
                for (int i = 1; i < kDmaPerSplit; ++i)
                    gm = max(gm, g[min(first + i, L) - first_c]);
                bad = base - wa_v[k - 1] < gm;
            }
            const uint64_t b = __ballot(bad);
            if (b) {
                ky = k0 - (__ffsll((long long)b) - 1) + 1;
                break;
            }
            ky = max(ka, k0 - 63);
        }
    }
}

// Which middle splits of the range [k_lo, k_hi] a launch takes (range) and
// how its workgroups share them (n_part parts).  kMidAll: the whole range.
// kMidInner: all but the first and the last kT splits, the ones whose
// operands lie in blocks up to two block-diagonals back, so that this part
// can run beside the previous block-diagonal's edge rounds; its slots are
// written as with kMidAll.  kMidRim: those 2 kT splits, after the edges, in
// one part that jumps from the first kT to the last kT and merges its
// minimum into the slots the inner part wrote by atomic minimum.  The corner
// is finished by the launch that completes its range: kMidAll in one part,
// or kMidRim (which reads the inner part's slot for it); else its partial is
// stored like any other and the edge round a + b = 0 finishes it.
constexpr int kMidAll = 0, kMidInner = 1, kMidRim = 2;
// Dynamic LDS, unused, that the inner range's packed launches request: it
// caps them at three workgroups per CU (53 of 160 KB each) instead of four,
// which leaves issue slots to the edge waves beside them (measured on MI355X
// at L = 500, M = 5000: 18.34 -> 17.99 ms; two per CU 18.71 ms).
constexpr unsigned kInnerLdsPad = 21 * 1024;
struct MiddleSplits {
    int ka, kb;        // this workgroup's first and last split
    int n_splits;      // splits it takes
    int jump_from;     // after this split the next is jump_to (-1: none)
    int jump_to;
    bool merge;        // atomic minimum into the partial slots
    bool owns_corner;  // finishes the corner cell of the block
};
__device__ inline MiddleSplits middle_splits(int k_lo, int k_hi, int range, int n_part, int part)
{
    MiddleSplits r;
    r.jump_from = -1;
    r.jump_to = -1;
    if (range == kMidRim) {
        r.ka = k_lo;
        r.kb = k_hi;
        r.n_splits = 2 * kT;
        r.jump_from = k_lo + kT - 1;
        r.jump_to = k_hi - kT + 1;
    } else {
        const int ra = range == kMidInner ? k_lo + kT : k_lo;
        const int rb = range == kMidInner ? k_hi - kT : k_hi;
        const int part_len = (rb - ra + n_part) / n_part;
        r.ka = ra + part * part_len;
        r.kb = min(rb, r.ka + part_len - 1);
        r.n_splits = r.kb - r.ka + 1;
    }
    r.merge = n_part > 1 || range == kMidRim;
    r.owns_corner = (n_part == 1 && range == kMidAll) || range == kMidRim;
    return r;
}

// With n_part > 1 (block-diagonals of few blocks, whose launches would leave
// most CUs idle), the middle split range of a block is cut into n_part runs
// taken by different workgroups (x = part * chunks + chunk).  Their keys
// share S and the offset base k_lo, so the unsigned minimum over the runs
// is the minimum over the whole range, ties included: each run merges its
// keys with an atomic minimum into the partial slots, which fill_partials
// has set to infinity, and the corners are left to the edge round a + b = 0.
template <bool RIM>
__global__ __launch_bounds__(256) void middle_packed_kernel(const int64_t *__restrict__ params, int L, int M,
                                                            int64_t pitch, int64_t rows, int delta, int range,
                                                            int n_part, int64_t *__restrict__ cost,
                                                            int16_t *__restrict__ dec, Work w)
{
    __shared__ uint32_t ring[kRing * kStage * kSplitWords];
    const Tile tile = xcd_tile();
    const int c = tile.z;
    const int I = tile.y;
    const int J = I + delta;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int chunks = gridDim.x / n_part;
    const int part = tile.x / chunks;
    const int m = (tile.x - part * chunks) * 64 + lane;
    const int k_lo = (I + 1) * kT;
    const int k_hi = J * kT;
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    // uniform over the workgroup: every wave returns or none does
    const bool full = middle_packed(cw, delta, k_hi - k_lo);
    if (!full && !middle_runs(cw, delta, k_hi - k_lo))
        return;
    // this workgroup's part of the middle splits [ka, kb]
    const MiddleSplits ms = middle_splits(k_lo, k_hi, range, n_part, part);
    const int ka = ms.ka, kb = ms.kb;
    if (ka > kb)
        return;
    const ChainRows r = chain_rows(params, w, L, c);
    if (block_saturated(cw, I, J, m - lane)) {
        if (ms.owns_corner && wave == 0 && m <= M)
            store_saturated_corner<Narrow>(cw, L, m, pitch, I, J, cost + (int64_t)c * rows * pitch,
                                           dec + (int64_t)c * rows * pitch);
        return;
    }
    const int s0 = I * kT + (wave >> 1) * kSub + 1;
    const int t0 = J * kT + (wave & 1) * kSub + 1;
    const int nt = t0 <= L ? min(kSub, L - t0 + 1) : 0;
    // key split bits: the whole range's, or those of a run of 2^S splits
    const int S = full ? (k_hi > k_lo ? 32 - __clz(k_hi - k_lo) : 0) : cw.pbits[delta];
    const int R = full ? INT_MAX : 1 << S;  // splits per run, a multiple of kStage
    const int mc = m <= M ? m : M;
    const int n_stages = (ms.n_splits + kStage - 1) / kStage;

    // rows this wave copies: waves 0, 1 the X rows (s, k) of s = 16I+1+8w ..,
    // waves 2, 3 the Y rows (k+1, t) of t = 16J+1+8(w-2) .. (past L: row L)
    const bool copies_x = wave < 2;
    const int first = copies_x ? I * kT + 1 + wave * kSub : J * kT + 1 + (wave - 2) * kSub;
    const char *src[kDmaPerSplit];  // each copied row at the next split to copy
#pragma unroll
    for (int i = 0; i < kDmaPerSplit; ++i)
        src[i] = (const char *)(cw.shadow + (copies_x ? row_of(L, first + i, ka) * pitch
                                                      : row_of(L, ka + 1, min(first + i, L)) * pitch));
    const int64_t row_bytes = pitch * 4;
    int k_copy = ka;  // next split to copy
    uint32_t *const dst0 = ring + (copies_x ? wave * kSub : kT + (wave - 2) * kSub) * 64;
    int fill = 0;  // ring stage filled next
    // saturated operand rows: X for the splits ka .. kx, Y for ky .. kb
    const int base = m - lane;
    int kx, ky;
    saturated_splits(cw, w.shift + (int64_t)c * 2 * L, L, copies_x, first, ka, RIM ? ms.jump_from : kb, base, lane,
                     kx, ky);
    // the rim's second half has bounds of its own
    int kx2 = 0, ky2 = 0;
    if constexpr (RIM)
        saturated_splits(cw, w.shift + (int64_t)c * 2 * L, L, copies_x, first, ms.jump_to, kb, base, lane, kx2, ky2);
    // the prefixes of u_f + u_b at the rows' other ends (X: s - 1, Y: t),
    // 32 bits suffice for a least time below 2^32 - 1
    const const_i64 pa = (const_i64)cw.preall;
    uint32_t pfx[kDmaPerSplit];
#pragma unroll
    for (int i = 0; i < kDmaPerSplit; ++i)
        pfx[i] = (uint32_t)pa[copies_x ? first + i - 1 : min(first + i, L)];
    // copies of one stage (splits past kb copy split kb again); the ring's
    // barrier waits for every copy and LDS write of the wave
    auto issue = [&]() {
        uint32_t *dst = dst0 + fill * (kStage * kSplitWords);
#pragma unroll
        for (int p = 0; p < kStage; ++p) {
            const int k = k_copy;
            const bool second = RIM && k > ms.jump_from;
            if (copies_x ? k <= (second ? kx2 : kx) : k >= (second ? ky2 : ky)) {
                const uint32_t pk = (uint32_t)pa[k];
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    dst[p * kSplitWords + i * 64 + lane] = copies_x ? pk - pfx[i] : pfx[i] - pk;
            } else {
                const int ri = mc - r.wa[k - 1];
                const uint32_t off = 4u * (uint32_t)(copies_x ? mc : (ri >= 0 ? ri : mc));
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    __builtin_amdgcn_global_load_lds((global_void *)(src[i] + off),
                                                     (lds_void *)(dst + p * kSplitWords + i * 64), 4, 0, 0);
            }
            if (RIM && k == ms.jump_from) {
                k_copy = ms.jump_to;
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    src[i] = (const char *)(cw.shadow + (copies_x ? row_of(L, first + i, k_copy) * pitch
                                                                  : row_of(L, k_copy + 1, min(first + i, L)) * pitch));
            } else if (k < kb) {
                // to split k + 1: X rows advance one row, Y rows L - k - 1 rows
                const int64_t step = copies_x ? row_bytes : (int64_t)(L - k - 1) * row_bytes;
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    src[i] += step;
                ++k_copy;
            }
        }
        fill = fill + 1 == kRing ? 0 : fill + 1;
    };

    uint32_t acc[kSub][kSub];
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j)
            acc[i][j] = kInf32;

#pragma unroll
    for (int st = 0; st < kRing - 1; ++st)
        if (st < n_stages)
            issue();
    // sum of u_f from k_lo to k, at most V
    uint32_t prefix = (uint32_t)(cw.pre[ka - 1] - cw.pre[k_lo - 1]);
    const uint32_t *const x_lds0 = ring + (wave >> 1) * kSub * 64 + lane;
    const uint32_t *const y_lds0 = ring + (kT + (wave & 1) * kSub) * 64 + lane;
    int read = 0;  // ring stage read next
    int k = ka;
    int run_base = full ? k_lo : ka;  // split of key offset 0
    // Runs: at the end of each, the keys become (value << 32) | s' in the
    // cost table: a plain store for the first run when the workgroup owns its
    // cells' slots (no merge), an atomic minimum otherwise (the slots then
    // start at all ones, or hold the inner part).  The corner keeps its best
    // form in registers when this kernel finishes it.
    int64_t *const tab = cost + (int64_t)c * rows * pitch;
    const bool corner = ms.owns_corner && s0 + kSub - 1 == k_lo && t0 == k_hi + 1;
    uint64_t corner_best = ~0ull;
    bool first_flush = true;
    auto flush = [&]() {
        const uint32_t mask = (1u << S) - 1u;
        // the lane's byte offset and the first row, opaque here so that the
        // compiler builds the 64 cell addresses in this rare step rather
        // than holding them in registers across the loop
        uint32_t lane_off = (uint32_t)m * 8u;
        asm volatile("" : "+v"(lane_off));
        int64_t row = row_of(L, s0, t0);
        asm volatile("" : "+s"(row));
#pragma unroll
        for (int i = 0; i < kSub; ++i, row += L - (s0 + i - 1))
#pragma unroll
            for (int j = 0; j < kSub; ++j) {
                const uint32_t key = acc[i][j];
                acc[i][j] = kInf32;
                const uint64_t st = key == kInf32 ? (uint64_t)kInf32 << 32
                                                  : ((uint64_t)(key >> S) << 32) |
                                                        (uint32_t)(run_base + 1 + (int)(key & mask));
                if (i == kSub - 1 && j == 0 && corner) {
                    corner_best = st < corner_best ? st : corner_best;
                } else if (j < nt && m <= M) {
                    // a wave-uniform row base and the lane's 32-bit offset
                    global_u64 slot = (global_u64)((char *)(tab + (row + j) * pitch) + lane_off);
                    if (!ms.merge && first_flush) {
                        *slot = st;
                    } else if (key != kInf32) {
                        __hip_atomic_fetch_min(slot, st, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
            }
        first_flush = false;
    };
    for (int it = 0; it < n_stages; ++it) {
        // this wave's copies of stage it have landed, and so (after the
        // barrier) have every wave's; the stage refilled below was read by
        // every wave before it reached the barrier
        ring_wait<kRing - 2>(n_stages - 1 - it);
        if (it + kRing - 1 < n_stages)
            issue();
        const uint32_t *x_lds = x_lds0 + read * (kStage * kSplitWords);
        const uint32_t *y_lds = y_lds0 + read * (kStage * kSplitWords);
        read = read + 1 == kRing ? 0 : read + 1;
        uint32_t x[kStage][kSub], y[kStage][kSub];
#pragma unroll
        for (int p = 0; p < kStage; ++p, ++k) {
            const bool real = k <= kb;
            const int ri = mc - r.wa[(real ? k : kb) - 1];
            prefix += real ? (uint32_t)r.uf[k - 1] : 0u;
            const uint32_t add = real && ri >= 0 ? (prefix << S) | (uint32_t)(k - run_base) : kInf32;
#pragma unroll
            for (int i = 0; i < kSub; ++i)
                x[p][i] = sat_add(rot_left(x_lds[p * kSplitWords + i * 64], S), add);
#pragma unroll
            for (int j = 0; j < kSub; ++j)
                y[p][j] = rot_left(y_lds[p * kSplitWords + j * 64], S);
        }
#pragma unroll
        for (int i = 0; i < kSub; ++i)
#pragma unroll
            for (int j = 0; j < kSub; ++j)
#pragma unroll
                for (int p = 0; p < kStage; ++p)
                    acc[i][j] = min(acc[i][j], sat_add(x[p][i], y[p][j]));
        if (k - run_base == R) {
            flush();
            run_base = k;
        }
        if (RIM && k == ms.jump_from + 1) {
            // the rim's second half: u_f of the splits skipped joins the prefix
            k = ms.jump_to;
            prefix = (uint32_t)(cw.pre[k - 1] - cw.pre[k_lo - 1]);
            if (!full) {
                flush();
                run_base = k;
            }
        }
    }
    if (!full) {
        if (k > run_base)
            flush();
        if (corner && m <= M) {
            if constexpr (RIM) {
                // the inner part's form in the corner's slot
                const uint64_t inner = (uint64_t)tab[row_of(L, k_lo, k_hi + 1) * pitch + m];
                corner_best = inner < corner_best ? inner : corner_best;
            }
            Narrow::Acc a;
            Narrow::init(a);
            if (corner_best < ((uint64_t)kInf32 << 32)) {
                a.val = (uint32_t)(corner_best >> 32);
                a.sp = (uint32_t)corner_best;
            }
            finish_corner<Narrow>(r, cw, L, m, pitch, k_lo, k_hi + 1, a, tab, dec + (int64_t)c * rows * pitch);
        }
        return;
    }
    if (m > M || nt == 0)
        return;
    // the partial stays a packed key, in the cell's compact copy, which
    // edge_kernel reads once and then overwrites with the final value; used
    // once, it is stored and loaded non-temporally.  The corner cell is
    // finished here when this launch takes the whole range in one part.
    if (ms.merge) {
#pragma unroll
        for (int i = 0; i < kSub; ++i)
#pragma unroll
            for (int j = 0; j < kSub; ++j)
                if (j < nt && !(i == kSub - 1 && j == 0 && corner))
                    atomicMin(&cw.shadow[row_of(L, s0 + i, t0 + j) * pitch + m], acc[i][j]);
        if (!corner)
            return;
    }
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            if (i == kSub - 1 && j == 0 && corner) {
                uint32_t key = acc[i][j];
                if constexpr (RIM) {
                    // the inner part's key in the corner's slot
                    const uint32_t inner =
                        __builtin_nontemporal_load(&cw.shadow[row_of(L, k_lo, k_hi + 1) * pitch + m]);
                    key = inner < key ? inner : key;
                }
                Narrow::Acc a;
                Narrow::init(a);
                if (key != kInf32) {
                    a.val = key >> S;
                    a.sp = (uint32_t)(k_lo + 1) + (key & ((1u << S) - 1u));
                }
                finish_corner<Narrow>(r, cw, L, m, pitch, k_lo, k_hi + 1, a, tab, dec + (int64_t)c * rows * pitch);
            } else if (j < nt && !ms.merge) {
                __builtin_nontemporal_store(acc[i][j], &cw.shadow[row_of(L, s0 + i, t0 + j) * pitch + m]);
            }
        }
}

// The middle products of the chains and block-diagonals that take neither
// packed keys nor packed runs: (value, split) pairs on the narrow path
// (operands from the compact copy, 4 bytes) and 64-bit keys on the wide path
// (operands from the int64 table, copied as two dwords per budget).  Same
// blocks, register tiles, ring of two-split stages and DMA copies into LDS
// as middle_packed_kernel; the partial, counting u_f from the first middle
// split, goes to the cost table in the stored() form ((value << 32) | s' or
// the 64-bit key), merged by atomic minimum when the range is cut
// (n_part > 1, slots set to all ones by fill_partials) or for the rim (the
// slots hold the inner part), and the corner cell is finished here when one
// part takes the whole range.
//
// With F (a block-diagonal whose bound V_D is below 2^38) the accumulators
// are exact doubles instead: a candidate of split k is the key
// value * 2^15 + (k - k_lo), below 2^53, so one double add and one double
// minimum relax it (two instructions against four for the (value, split)
// pairs or the 64-bit keys; the part issues double additions and minima at
// the rate of 32-bit integer ones), and the minimum key is the smallest
// value with, among equal values, the smallest split.  An operand at
// infinity (0xFFFFFFFF, INT64_MAX) gives a key at or above the largest
// finite one plus one, a budget shifted below 0 the key +inf.
// Minimum of two doubles that are never NaN: v_min_f64 itself (the
// compiler's minnum quiets its operands first, one more instruction per
// candidate)
__device__ __forceinline__ double min_f64(double a, double b)
{
    double r;
    asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

__device__ inline double f64_finite_bound(bool narrow)
{
    // narrow: the infinity 0xFFFFFFFF as a value; 64-bit: 2^53
    return narrow ? 4294967295.0 * 32768.0 : 9007199254740992.0;
}

// The stored() form of the path P for a double key of the middle range
// starting at split k_lo + 1.
template <class P>
__device__ inline int64_t f64_stored(double key, int k_lo)
{
    if (!(key < f64_finite_bound(P::kShadow)))
        return P::kShadow ? (int64_t)((uint64_t)kInf32 << 32) : (int64_t)(1ull << 62);
    const double q = __builtin_floor(key * (1.0 / 32768.0));
    const uint64_t v = (uint64_t)q;
    const uint32_t split = (uint32_t)(k_lo + 1) + (uint32_t)(key - q * 32768.0);
    return P::kShadow ? (int64_t)((v << 32) | split) : (int64_t)((v << 16) | split);
}

template <class P>
__device__ inline typename P::Acc f64_acc(double key, int k_lo)
{
    typename P::Acc a;
    P::init(a);
    P::merge_later(a, f64_stored<P>(key, k_lo));
    return a;
}

template <class P, bool F, bool RIM>
__device__ __forceinline__ void middle_lds_body(const ChainRows &r, const ChainWork &cw, int L, int M, int m,
                                                int64_t pitch, int I, int J, int wave, const MiddleSplits &ms,
                                                int k_lo, int k_hi, int64_t *tab, int16_t *dtab, uint32_t *ring)
{
    constexpr int EW = P::kBytes / 4;          // dwords per element
    constexpr int kSW = kSplitWords * EW;      // dwords per split slot: 32 rows of 64 elements
    const int ka = ms.ka, kb = ms.kb;
    const int lane = threadIdx.x & 63;
    const int mc = min(m, M);
    const int m0 = m - lane;                   // the workgroup's first budget
    const int n_stages = (ms.n_splits + kStage - 1) / kStage;
    const int s0 = I * kT + (wave >> 1) * kSub + 1;
    const int t0 = J * kT + (wave & 1) * kSub + 1;
    const int nt = t0 <= L ? min(kSub, L - t0 + 1) : 0;
    // rows this wave copies: waves 0, 1 the X rows (s, k) of s = 16I+1+8w ..,
    // waves 2, 3 the Y rows (k+1, t) of t = 16J+1+8(w-2) .. (past L: row L);
    // a row of 64 elements takes EW copies of 64 dwords, copy e taking
    // elements 32e .. 32e + 31 (two lanes per element) when EW = 2
    const bool copies_x = wave < 2;
    const int first = copies_x ? I * kT + 1 + wave * kSub : J * kT + 1 + (wave - 2) * kSub;
    const char *const base = P::table(tab, cw.shadow);
    const int64_t row_bytes = pitch * P::kBytes;
    const char *src[kDmaPerSplit];
#pragma unroll
    for (int i = 0; i < kDmaPerSplit; ++i)
        src[i] = base + (copies_x ? row_of(L, first + i, ka) : row_of(L, ka + 1, min(first + i, L))) * row_bytes;
    // the element and dword each lane copies in copy e
    int elem_budget[EW];
    uint32_t dword_off[EW];
#pragma unroll
    for (int e = 0; e < EW; ++e) {
        const int el = EW == 1 ? lane : 32 * e + (lane >> 1);
        elem_budget[e] = min(m0 + el, M);
        dword_off[e] = EW == 1 ? 0u : 4u * (uint32_t)(lane & 1);
    }
    int k_copy = ka;  // next split to copy
    uint32_t *const dst0 = ring + (copies_x ? wave * kSub : kT + (wave - 2) * kSub) * 64 * EW;
    int fill = 0;  // ring stage filled next
    // copies of one stage; splits past kb copy split kb again, so every
    // stage issues the same number of copies
    auto issue = [&]() {
        uint32_t *dst = dst0 + fill * (kStage * kSW);
#pragma unroll
        for (int p = 0; p < kStage; ++p) {
            const int k = k_copy;
            const int w_k = r.wa[k - 1];
#pragma unroll
            for (int e = 0; e < EW; ++e) {
                const int mb = elem_budget[e];
                const int ri = mb - w_k;
                const uint32_t off = (uint32_t)P::kBytes * (uint32_t)(copies_x ? mb : (ri >= 0 ? ri : mb)) +
                                     dword_off[e];
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    __builtin_amdgcn_global_load_lds((global_void *)(src[i] + off),
                                                     (lds_void *)(dst + p * kSW + i * 64 * EW + e * 64), 4, 0, 0);
            }
            if (RIM && k == ms.jump_from) {
                k_copy = ms.jump_to;
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    src[i] = base + (copies_x ? row_of(L, first + i, k_copy)
                                              : row_of(L, k_copy + 1, min(first + i, L))) * row_bytes;
            } else if (k < kb) {
                // to split k + 1: X rows advance one row, Y rows L - k - 1 rows
                const int64_t step = copies_x ? row_bytes : (int64_t)(L - k - 1) * row_bytes;
#pragma unroll
                for (int i = 0; i < kDmaPerSplit; ++i)
                    src[i] += step;
                ++k_copy;
            }
        }
        fill = fill + 1 == kRing ? 0 : fill + 1;
    };

    typedef typename std::conditional<F, double, typename P::Acc>::type Acc;
    Acc acc[kSub][kSub];
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            if constexpr (F)
                acc[i][j] = __builtin_inf();
            else
                P::init(acc[i][j]);
        }
#pragma unroll
    for (int st = 0; st < kRing - 1; ++st)
        if (st < n_stages)
            issue();
    uint64_t prefix = (uint64_t)(cw.pre[ka - 1] - cw.pre[k_lo - 1]);  // u_f from k_lo on
    typedef typename P::Raw Raw;
    const Raw *const x_lds0 = (const Raw *)(ring + (wave >> 1) * kSub * 64 * EW) + lane;
    const Raw *const y_lds0 = (const Raw *)(ring + (kT + (wave & 1) * kSub) * 64 * EW) + lane;
    int read = 0;  // ring stage read next
    int k = ka;
    for (int it = 0; it < n_stages; ++it) {
        // this wave's copies of stage it have landed, and so (after the
        // barrier) have every wave's; the stage refilled below was read by
        // every wave before it reached the barrier
        ring_wait<kRing - 2>(n_stages - 1 - it);
        if (it + kRing - 1 < n_stages)
            issue();
        const Raw *x_lds = x_lds0 + read * (kStage * kSplitWords);
        const Raw *y_lds = y_lds0 + read * (kStage * kSplitWords);
        read = read + 1 == kRing ? 0 : read + 1;
        typedef typename std::conditional<F, double, typename P::X>::type XT;
        typedef typename std::conditional<F, double, typename P::Y>::type YT;
        XT x[kStage][kSub];
        YT y[kStage][kSub];
        uint32_t sp[kStage];
#pragma unroll
        for (int p = 0; p < kStage; ++p, ++k) {
            const bool real = k <= kb;
            const int kk = real ? k : kb;
            const int ri = mc - r.wa[kk - 1];
            prefix += real ? (uint64_t)r.uf[k - 1] : 0;
            sp[p] = (uint32_t)(k + 1);
            if constexpr (F) {
                const double add = real && ri >= 0 ? (double)((prefix << 15) + (uint64_t)(k - k_lo)) : __builtin_inf();
                // scaled by ldexp, which the compiler does not fuse into the
                // candidates' additions
#pragma unroll
                for (int i = 0; i < kSub; ++i)
                    x[p][i] = __builtin_ldexp((double)x_lds[p * kSplitWords + i * 64], 15) + add;
#pragma unroll
                for (int j = 0; j < kSub; ++j)
                    y[p][j] = __builtin_ldexp((double)y_lds[p * kSplitWords + j * 64], 15);
            } else {
#pragma unroll
                for (int i = 0; i < kSub; ++i)
                    x[p][i] = P::xop(x_lds[p * kSplitWords + i * 64], prefix, sp[p], real && ri >= 0);
#pragma unroll
                for (int j = 0; j < kSub; ++j)
                    y[p][j] = P::yop(y_lds[p * kSplitWords + j * 64]);
            }
        }
        // splits in increasing order (the narrow pairs keep the first minimum)
#pragma unroll
        for (int p = 0; p < kStage; ++p)
#pragma unroll
            for (int i = 0; i < kSub; ++i)
#pragma unroll
                for (int j = 0; j < kSub; ++j) {
                    if constexpr (F)
                        acc[i][j] = min_f64(acc[i][j], x[p][i] + y[p][j]);
                    else
                        P::relax(acc[i][j], x[p][i], y[p][j], sp[p]);
                }
        if (RIM && k == ms.jump_from + 1) {
            // the rim's second half: u_f of the splits skipped joins the prefix
            k = ms.jump_to;
            prefix = (uint64_t)(cw.pre[k - 1] - cw.pre[k_lo - 1]);
        }
    }
    if (m > M || nt == 0)
        return;
    auto stored = [&](const Acc &a) -> int64_t {
        if constexpr (F)
            return f64_stored<P>(a, k_lo);
        else
            return P::stored(a);
    };
    // the wave whose last row is 16I + 16 and first column 16J + 1 holds the
    // corner
    const bool corner = ms.owns_corner && s0 + kSub - 1 == k_lo && t0 == k_hi + 1;
    if (ms.merge) {
        // a part of a cut range: the stored forms (value << 32) | s' and
        // (value << 16) | s' order by value, then split, as unsigned words
#pragma unroll
        for (int i = 0; i < kSub; ++i)
#pragma unroll
            for (int j = 0; j < kSub; ++j)
                if (j < nt && !(i == kSub - 1 && j == 0 && corner))
                    atomicMin((unsigned long long *)&tab[row_of(L, s0 + i, t0 + j) * pitch + m],
                              (unsigned long long)stored(acc[i][j]));
        if constexpr (RIM) {
            if (corner) {
                // the smaller of the rim's form and the inner part's in the
                // corner's slot completes the corner's middle range
                const uint64_t inner = (uint64_t)tab[row_of(L, k_lo, k_hi + 1) * pitch + m];
                const uint64_t own = (uint64_t)stored(acc[kSub - 1][0]);
                typename P::Acc a;
                P::init(a);
                P::merge_later(a, (int64_t)(inner < own ? inner : own));
                finish_corner<P>(r, cw, L, m, pitch, k_lo, k_hi + 1, a, tab, dtab);
            }
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < kSub; ++i)
#pragma unroll
        for (int j = 0; j < kSub; ++j) {
            if (i == kSub - 1 && j == 0 && corner) {
                if constexpr (F)
                    finish_corner<P>(r, cw, L, m, pitch, k_lo, k_hi + 1, f64_acc<P>(acc[i][j], k_lo), tab, dtab);
                else
                    finish_corner<P>(r, cw, L, m, pitch, k_lo, k_hi + 1, acc[i][j], tab, dtab);
            } else if (j < nt) {
                tab[row_of(L, s0 + i, t0 + j) * pitch + m] = stored(acc[i][j]);
            }
        }
}

template <bool RIM>
__global__ __launch_bounds__(256) void middle_kernel(const int64_t *__restrict__ params, int L, int M,
                                                     int64_t pitch, int64_t rows, int delta, int range, int n_part,
                                                     int64_t *__restrict__ cost, int16_t *__restrict__ dec, Work w)
{
    // a ring of 64-bit elements (the narrow path uses the first half)
    __shared__ __align__(16) uint32_t ring[kRing * kStage * kSplitWords * 2];
    const Tile tile = xcd_tile();
    const int c = tile.z;
    const int I = tile.y;
    const int J = I + delta;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int chunks = gridDim.x / n_part;
    const int part = tile.x / chunks;
    const int m = (tile.x - part * chunks) * 64 + (threadIdx.x & 63);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    const int k_lo = (I + 1) * kT;
    const int k_hi = J * kT;
    // uniform over the workgroup: every wave returns or none does
    if (middle_packed(cw, delta, k_hi - k_lo) || middle_runs(cw, delta, k_hi - k_lo))
        return;  // middle_packed_kernel takes this block-diagonal
    // this workgroup's part of the middle splits, as in middle_packed_kernel
    const MiddleSplits ms = middle_splits(k_lo, k_hi, range, n_part, part);
    if (ms.ka > ms.kb)
        return;
    const ChainRows r = chain_rows(params, w, L, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    int16_t *dtab = dec + (int64_t)c * rows * pitch;
    if (block_saturated(cw, I, J, m - (threadIdx.x & 63))) {
        if (ms.owns_corner && wave == 0 && m <= M) {
            if (cw.narrow(delta))
                store_saturated_corner<Narrow>(cw, L, m, pitch, I, J, tab, dtab);
            else
                store_saturated_corner<Wide>(cw, L, m, pitch, I, J, tab, dtab);
        }
        return;
    }
    if (cw.narrow(delta))
        middle_lds_body<Narrow, true, RIM>(r, cw, L, M, m, pitch, I, J, wave, ms, k_lo, k_hi, tab, dtab, ring);
    else if (cw.f64_keys(delta))
        middle_lds_body<Wide, true, RIM>(r, cw, L, M, m, pitch, I, J, wave, ms, k_lo, k_hi, tab, dtab, ring);
    else
        middle_lds_body<Wide, false, RIM>(r, cw, L, M, m, pitch, I, J, wave, ms, k_lo, k_hi, tab, dtab, ring);
}

// Edge splits, C_2 and the gates for the cells a + b = q of every block
// (I, I + D) of one block-diagonal; a workgroup is one cell at 128 budgets.
// Splits are met in increasing order: low, then the stored middle partial,
// then high.  With H (narrow path, ChainWork::diag16), the operand that lies
// in a diagonal block -- X of a low split, Y of a high one -- comes from the
// 2-byte copy.
template <class P, bool H>
__device__ __forceinline__ void edge_body(const ChainRows &r, const ChainWork &cw, int L, int M, int m0, int64_t pitch,
                                          int s, int t, int k_lo, int k_hi, bool sat, int64_t *tab, int16_t *dtab)
{
    constexpr int NB = kEdgeBudgets;
    const int64_t cell = row_of(L, s, t);
    // every budget of the workgroup saturated
    if (sat) {
        const typename P::Acc a = P::all_only(least_time(cw, s, t));
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int mb = m0 + b * kEdgeThreads;
            if (mb <= M)
                store_cell<P>(tab, dtab, cw.shadow, cell * pitch + mb, a);
        }
        return;
    }
    // the lane's budgets m0 + b * kEdgeThreads; those past M load budget M
    // and store nothing
    int m[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        m[b] = min(m0 + b * kEdgeThreads, M);
    // the diagonal-block operands saturated at every budget of the workgroup
    // (from its first, lane 0's): X of the low splits in block I, Y of the
    // high splits in block J (shifted by at most the block's largest w_a)
    const int base = __builtin_amdgcn_readfirstlane(m0);
    const bool xsat = base >= diag_block_gmax(cw, (s - 1) / kT);
    const bool ysat = base >= diag_block_gyshift(cw, (t - 1) / kT);
    // loads that depend on nothing go first: the stored middle partial (a
    // packed key in the compact copy, or (value << 32) | s' in the cost
    // table) and the C_2 operand (the lane's own budget when C_2 is out of
    // reach)
    const bool packed_partial = P::kShadow && middle_packed(cw, (k_hi - k_lo) / kT + 1, k_hi - k_lo);
    const int wab = r.wabar[s - 1];
    const int32_t gall = cw.gall[cell];
    const int64_t below = row_of(L, s + 1, t) * pitch;
    uint32_t key[NB];
    int64_t stored64[NB];
    typename P::Raw c2[NB];
    bool all_ok[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        key[b] = packed_partial ? __builtin_nontemporal_load(cw.shadow + cell * pitch + m[b]) : 0u;
        stored64[b] = packed_partial ? 0 : load64(tab + cell * pitch, m[b]);
        const int ri = m[b] - wab;
        all_ok[b] = m[b] >= gall && ri >= 0;
        c2[b] = P::load(tab + below, cw.shadow + below, all_ok[b] ? ri : m[b]);
    }
    typename P::Acc acc[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        P::init(acc[b]);
    // low splits k = s .. k_lo - 1: X from block (I, I), Y from this block
    uint64_t prefix = 0;
    const int64_t rb = pitch * 4, hb = cw.hpitch * 2;
    if constexpr (H) {
        // X rows (s, k) of the 2-byte copy are consecutive; all saturated
        // (xsat) when the largest G of diagonal block I is reached
        MixedCursor low{(const char *)cw.half_row(s, s), (const char *)(cw.shadow + row_of(L, s + 1, t) * pitch), hb,
                        (int64_t)(L - s - 1) * rb, rb};
        if (xsat)
            MixedSatRunNB<Load16, Load32, true, kT - 1, NB>::go(k_lo - s, acc, r, m, s, low, prefix,
                                                                 (const_i64)cw.preall, ((const_i64)cw.preall)[s - 1]);
        else
            MixedRunNB<Load16, Load32, kT - 1, NB>::go(k_lo - s, acc, r, m, s, low, prefix);
    } else {
        RowCursor low = row_cursor<P>(tab, cw.shadow, L, pitch, s, t, s);
        if (xsat)
            relax_sat_run_nb<P, true, NB>(acc, r, m, s, k_lo - s, low, prefix, (const_i64)cw.preall,
                                          ((const_i64)cw.preall)[s - 1]);
        else
            relax_run_nb<P, NB>(acc, r, m, s, k_lo - s, low, prefix);
    }
    // middle splits: the stored partial counts u_f from k_lo on
    const int S = k_hi > k_lo ? 32 - __clz(k_hi - k_lo) : 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        int64_t stored = stored64[b];
        if (packed_partial) {
            const uint32_t split = (uint32_t)(k_lo + 1) + (key[b] & ((1u << S) - 1u));
            stored = key[b] == kInf32 ? (int64_t)((uint64_t)kInf32 << 32)
                                      : (int64_t)(((uint64_t)(key[b] >> S) << 32) | split);
        }
        P::merge_stored(acc[b], stored, prefix);
    }
    // high splits k = 16J + 1 .. t - 1: X from this block, Y from block (J, J)
    prefix += (uint64_t)(cw.pre[k_hi] - cw.pre[k_lo - 1]);
    if constexpr (H) {
        // Y rows (k + 1, t) of the 2-byte copy are 16 rows apart; all
        // saturated (ysat) when the largest G of diagonal block J plus the
        // largest w_a^k of its stages is reached
        MixedCursor high{(const char *)(cw.shadow + row_of(L, s, k_hi + 1) * pitch),
                         (const char *)cw.half_row(k_hi + 2, t), rb, kT * hb, 0};
        if (ysat)
            MixedSatRunNB<Load32, Load16, false, kT - 1, NB>::go(t - k_hi - 1, acc, r, m, k_hi + 1, high, prefix,
                                                                  (const_i64)cw.preall, ((const_i64)cw.preall)[t]);
        else
            MixedRunNB<Load32, Load16, kT - 1, NB>::go(t - k_hi - 1, acc, r, m, k_hi + 1, high, prefix);
    } else {
        RowCursor high = row_cursor<P>(tab, cw.shadow, L, pitch, s, t, k_hi + 1);
        if (ysat)
            relax_sat_run_nb<P, false, NB>(acc, r, m, k_hi + 1, t - k_hi - 1, high, prefix, (const_i64)cw.preall,
                                           ((const_i64)cw.preall)[t]);
        else
            relax_run_nb<P, NB>(acc, r, m, k_hi + 1, t - k_hi - 1, high, prefix);
    }
    const int32_t gnone = cw.gnone[cell];
    const uint64_t ufub = (uint64_t)(r.uf[s - 1] + r.ub[s - 1]);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        if (m[b] < gnone)
            P::init(acc[b]);
        if (all_ok[b])
            P::relax_all(acc[b], c2[b], ufub);
        const int mb = m0 + b * kEdgeThreads;
        if (mb <= M)
            store_cell<P>(tab, dtab, cw.shadow, cell * pitch + mb, acc[b]);
    }
}

__global__ __launch_bounds__(kEdgeThreads) void edge_kernel(const int64_t *__restrict__ params, int L, int M,
                                                   int64_t pitch, int64_t rows, int delta, int q, int a_min,
                                                   int n_q, int64_t *__restrict__ cost, int16_t *__restrict__ dec,
                                                   Work w)
{
    const int c = blockIdx.z;
    const int blk = blockIdx.y / n_q;
    const int a = a_min + (blockIdx.y - blk * n_q);
    const int I = blk;
    const int J = I + delta;
    const int s = (I + 1) * kT - a;
    const int t = J * kT + 1 + (q - a);
    const int m0 = blockIdx.x * (kEdgeThreads * kEdgeBudgets) + threadIdx.x;
    if (t > L || m0 > M)
        return;
    const ChainRows r = chain_rows(params, w, L, c);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    int16_t *dtab = dec + (int64_t)c * rows * pitch;
    // the path and the saturation test first: their scalar loads go together
    const bool narrow = cw.narrow(delta), d16 = cw.diag16();
    const bool sat =
        saturated_in_block(r, cw, I, delta, s, row_of(L, s, t), blockIdx.x * (kEdgeThreads * kEdgeBudgets));
    // the 2-byte path first and marked likely, so that the code of the
    // other two paths does not sit in its way
    if (__builtin_expect(narrow && d16, 1))
        edge_body<Narrow, true>(r, cw, L, M, m0, pitch, s, t, (I + 1) * kT, J * kT, sat, tab, dtab);
    else if (!narrow)
        edge_body<Wide, false>(r, cw, L, M, m0, pitch, s, t, (I + 1) * kT, J * kT, sat, tab, dtab);
    else
        edge_body<Narrow, false>(r, cw, L, M, m0, pitch, s, t, (I + 1) * kT, J * kT, sat, tab, dtab);
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

Work work_view(void *base, int n_chains, int L, int64_t pitch)
{
    const WorkLayout wl = work_layout(n_chains, L, pitch);
    char *b = (char *)base;
    Work w;
    w.pre = (int64_t *)(b + wl.pre);
    w.preall = (int64_t *)(b + wl.preall);
    w.pbits = (int32_t *)(b + wl.pbits);
    w.bsum = (int64_t *)(b + wl.bsum);
    w.gnone = (int32_t *)(b + wl.gnone);
    w.gall = (int32_t *)(b + wl.gall);
    w.gsat = (int32_t *)(b + wl.gsat);
    w.gblk = (int32_t *)(b + wl.gblk);
    w.status = (int32_t *)(b + wl.status);
    w.shift = (int32_t *)(b + wl.shift);
    w.shadow = (uint32_t *)(b + wl.shadow);
    w.half = (int16_t *)(b + wl.half);
    return w;
}

// The side stream of a device, for the middle products that run beside the
// edge rounds, and the two events that order it with the caller's stream:
// created on the first solve on the device and kept until the process ends.
// A solve holds side_mutex while it enqueues, so that solves from several
// host threads record and wait the events in turn; their device work still
// overlaps.
struct SideStream {
    hipStream_t stream = nullptr;
    hipEvent_t ready = nullptr, done = nullptr;
};
constexpr int kMaxDevices = 64;
std::mutex side_mutex;
SideStream side_streams[kMaxDevices];

hipError_t device_side_stream(hipStream_t stream, SideStream *&side, std::unique_lock<std::mutex> &lock)
{
    hipDevice_t dev = 0;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    lock = std::unique_lock<std::mutex>(side_mutex);
    SideStream &sd = side_streams[dev];
    if (!sd.stream) {
        int cur = 0;
        if ((e = hipGetDevice(&cur)) != hipSuccess || (cur != dev && (e = hipSetDevice(dev)) != hipSuccess))
            return e;
        SideStream n;
        e = hipStreamCreateWithFlags(&n.stream, hipStreamNonBlocking);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&n.ready, hipEventDisableTiming);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&n.done, hipEventDisableTiming);
        const hipError_t r = cur != dev ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess || r != hipSuccess)
            return e != hipSuccess ? e : r;
        sd = n;
    }
    side = &sd;
    return hipSuccess;
}

hipError_t launch_fill(const Tables &tb, const Work &w, int schedule, hipStream_t stream, LaunchObserver *obs,
                       bool side_stream)
{
    // hipGetLastError also returns an error an earlier runtime call of the
    // caller left behind: clear it, so that the checks below see only these
    // launches
    (void)hipGetLastError();
    const int L = tb.L;
    const uint64_t W = (uint64_t)tb.M + 1;
    const uint64_t nc = (uint64_t)tb.n_chains;
    const unsigned mb256 = (unsigned)((tb.M + 1 + 255) / 256);
    const unsigned mb64 = (unsigned)((tb.M + 1 + 63) / 64);
    const unsigned mb_edge = (unsigned)((tb.M + kEdgeThreads * kEdgeBudgets) / (kEdgeThreads * kEdgeBudgets));
    const unsigned mb_diag = (unsigned)((tb.M + kEdgeThreads * kDiagBudgets) / (kEdgeThreads * kDiagBudgets));
    auto launched_on = [&](hipStream_t st, KernelClass k, uint64_t c1, uint64_t c2, uint64_t cells) -> hipError_t {
        hipError_t e = check();
        if (e == hipSuccess && obs)
            e = obs->after(k, LaunchWork{c1 * W * nc, c2 * W * nc, cells * W * nc}, st);
        return e;
    };
    auto launched = [&](KernelClass k, uint64_t c1, uint64_t c2, uint64_t cells) {
        return launched_on(stream, k, c1, c2, cells);
    };
    auto before_on = [&](hipStream_t st, KernelClass k) -> hipError_t {
        return obs ? obs->before(k, st) : hipSuccess;
    };
    auto before = [&](KernelClass k) { return before_on(stream, k); };
    hipError_t e;

    if ((e = before(kPrep)) != hipSuccess)
        return e;
    prep_kernel<<<dim3(L + 1, tb.n_chains), 64, 0, stream>>>(tb.params, L, tb.M, tb.rows, w);
    if ((e = launched(kPrep, 0, 0, 0)) != hipSuccess)
        return e;
    if ((e = before(kLeaf)) != hipSuccess)
        return e;
    leaf_kernel<<<dim3(mb256, L, tb.n_chains), 256, 0, stream>>>(tb.params, L, tb.M, tb.pitch, tb.rows, tb.cost,
                                                                 tb.dec, w);
    if ((e = launched(kLeaf, 0, 0, (uint64_t)L)) != hipSuccess)
        return e;
    // A small table goes diagonal by diagonal: its launches are few and
    // short, and the blocked fill would need 33 per block-diagonal.
    const uint64_t r_total = ((uint64_t)L * L * L / 6) * W * nc;
    const bool streamed = schedule == ROTOR_SCHEDULE_DIAGONAL ||
                          (schedule == ROTOR_SCHEDULE_AUTO &&
                           (nc == 1 ? r_total <= kStreamMaxCandidates1 || W < (uint64_t)kStreamBelowBudgets
                                    : r_total <= kStreamMaxCandidatesN));
    for (int d = 1; d < (streamed ? L : kT) && d < L; ++d) {
        if ((e = before(kDiag)) != hipSuccess)
            return e;
        if (streamed && d >= kSplitMinD)
            diag_split_kernel<<<dim3(mb64, L - d, tb.n_chains), 256, 0, stream>>>(tb.params, L, tb.M, tb.pitch,
                                                                                  tb.rows, d, tb.cost, tb.dec, w);
        else if (streamed)
            diag_kernel<kEdgeBudgets><<<dim3(mb_edge, L - d, tb.n_chains), kEdgeThreads, 0, stream>>>(
                tb.params, L, tb.M, tb.pitch, tb.rows, d, 1, tb.cost, tb.dec, w);
        else
            diag_kernel<kDiagBudgets><<<dim3(mb_diag, L - d, tb.n_chains), kEdgeThreads, 0, stream>>>(
                tb.params, L, tb.M, tb.pitch, tb.rows, d, 0, tb.cost, tb.dec, w);
        const uint64_t pairs = streamed ? (uint64_t)(L - d) : in_block_pairs(L, d);
        if ((e = launched(kDiag, pairs * d, pairs, pairs)) != hipSuccess)
            return e;
    }
    if (streamed)
        return hipSuccess;
    const int nb = (L + kT - 1) / kT;
    // workgroups of the middle launches: few blocks cut the middle ranges
    // into runs for more workgroups (about 512), each of 32 splits or more
    auto parts_of = [&](int delta) {
        const unsigned wgs = mb64 * (unsigned)(nb - delta) * (unsigned)tb.n_chains;
        const int span = (delta - 1) * kT + 1;
        return wgs < 256 ? max(1, min((int)((512 + wgs - 1) / wgs), span / 32)) : 1;
    };
    // The middle launches of block-diagonal delta over one range: the
    // general kernel and the packed-key one (each chain is taken by one of
    // the two, the other returns at once), slots set to infinity first when
    // the parts merge into them.  Work counts go with the packed kernel's
    // launch (split candidates c1, corner cells finished).
    auto middle_general = [&](int delta, int range, int n_part, hipStream_t st) {
        hipError_t e = before_on(st, kMiddle);
        if (e != hipSuccess)
            return e;
        const dim3 grid(mb64 * n_part, nb - delta, tb.n_chains);
        if (range == kMidRim)
            middle_kernel<true><<<grid, 256, 0, st>>>(tb.params, L, tb.M, tb.pitch, tb.rows, delta, range, n_part,
                                                      tb.cost, tb.dec, w);
        else
            middle_kernel<false><<<grid, 256, 0, st>>>(tb.params, L, tb.M, tb.pitch, tb.rows, delta, range, n_part,
                                                       tb.cost, tb.dec, w);
        return launched_on(st, kMiddle, 0, 0, 0);
    };
    auto middle_packed = [&](int delta, int range, int n_part, hipStream_t st, uint64_t c1, uint64_t corners) {
        hipError_t e = before_on(st, kMiddle);
        if (e != hipSuccess)
            return e;
        const dim3 grid(mb64 * n_part, nb - delta, tb.n_chains);
        if (range == kMidRim)
            middle_packed_kernel<true><<<grid, 256, 0, st>>>(tb.params, L, tb.M, tb.pitch, tb.rows, delta, range,
                                                             n_part, tb.cost, tb.dec, w);
        else
            middle_packed_kernel<false><<<grid, 256, range == kMidInner ? kInnerLdsPad : 0, st>>>(
                tb.params, L, tb.M, tb.pitch, tb.rows, delta, range, n_part, tb.cost, tb.dec, w);
        return launched_on(st, kMiddle, c1, corners, corners);
    };
    auto fill_partials = [&](int delta, hipStream_t st) {
        hipError_t e = before_on(st, kMiddle);
        if (e != hipSuccess)
            return e;
        fill_partials_kernel<<<dim3(mb256, (nb - delta) * kT * kT, tb.n_chains), 256, 0, st>>>(
            L, tb.M, tb.pitch, tb.rows, delta, tb.cost, w);
        return launched_on(st, kMiddle, 0, 0, 0);
    };
    // pairs of block-diagonal delta: full rows of 16, columns up to L
    auto pairs_of = [&](int delta) {
        uint64_t pairs = 0;
        for (int I = 0; I + delta < nb; ++I)
            pairs += (uint64_t)kT * (uint64_t)min(kT, L - (I + delta) * kT);
        return pairs;
    };
    // The inner middle range of block-diagonal delta + 1 (from delta + 1 = 3
    // on) reads only block-diagonals up to delta - 1: it runs on the
    // device's side stream beside the rim and the edges of delta, and its
    // own rim follows them; only beside edges by rounds (the row edges of a
    // batch lose: 4.95 -> 5.06 ms for 256 chains of L = 64).  An observer
    // sees the side stream's launches on that stream.
    bool overlap = side_stream && schedule != ROTOR_SCHEDULE_BLOCKED_SERIAL && nb >= 4;
    SideStream *side = nullptr;
    std::unique_lock<std::mutex> side_lock;
    if (overlap && device_side_stream(stream, side, side_lock) != hipSuccess) {
        // no side stream on this device: everything on the caller's
        // stream (the failed call's error is not this solve's)
        (void)hipGetLastError();
        overlap = false;
        side = nullptr;
        if (side_lock.owns_lock())
            side_lock.unlock();
    }
    bool inner_done = false;  // the inner range of delta ran beside the edges of delta - 1
    auto blocked = [&]() -> hipError_t {
        hipError_t e;
        for (int delta = 1; delta < nb; ++delta) {
            const uint64_t pairs = pairs_of(delta);
            const int span = (delta - 1) * kT + 1;
            const bool rows = schedule == ROTOR_SCHEDULE_BLOCKED_ROWS ||
                              (schedule != ROTOR_SCHEDULE_BLOCKED_ROUNDS &&
                               row_edges((int64_t)(nb - delta) * tb.n_chains));
            // the middle splits of every pair, and C_2 of the corner cell of
            // every block when the middle products finish the corners
            const int n_part = inner_done ? 1 : parts_of(delta);
            const int finish = inner_done || n_part == 1 ? 1 : 0;
            const uint64_t corners = finish ? (uint64_t)(nb - delta) : 0;
            if (inner_done && (e = hipStreamWaitEvent(stream, side->done, 0)) != hipSuccess)
                return e;
            const int range = inner_done ? kMidRim : kMidAll;
            if (n_part > 1 && (e = fill_partials(delta, stream)) != hipSuccess)
                return e;
            // the general kernel first: its workgroups, with their larger LDS
            // ring, would otherwise wait for those of the next inner range even
            // where they return at once
            if ((e = middle_general(delta, range, n_part, stream)) != hipSuccess)
                return e;
            const bool next_inner = overlap && !rows && delta + 1 < nb && delta + 1 >= 3;
            if (next_inner) {
                // the inner splits of every pair of delta + 1: all but 2 kT
                const int np = parts_of(delta + 1);
                const uint64_t inner = pairs_of(delta + 1) * (uint64_t)(delta * kT + 1 - 2 * kT);
                if ((e = hipEventRecord(side->ready, stream)) != hipSuccess ||
                    (e = hipStreamWaitEvent(side->stream, side->ready, 0)) != hipSuccess ||
                    (np > 1 && (e = fill_partials(delta + 1, side->stream)) != hipSuccess) ||
                    (e = middle_packed(delta + 1, kMidInner, np, side->stream, inner, 0)) != hipSuccess ||
                    (e = middle_general(delta + 1, kMidInner, np, side->stream)) != hipSuccess ||
                    (obs && (e = obs->end_stream(side->stream)) != hipSuccess) ||
                    (e = hipEventRecord(side->done, side->stream)) != hipSuccess)
                    return e;
            }
            // the middle splits of every pair (the rim's 2 kT after an inner range)
            const uint64_t c1 = pairs * (uint64_t)(range == kMidRim ? 2 * kT : span);
            if ((e = middle_packed(delta, range, n_part, stream, c1, corners)) != hipSuccess)
                return e;
            inner_done = next_inner;
            if (rows) {
                for (int a = 0; a < kT; ++a) {
                    uint64_t c1 = 0, cells = 0;
                    for (int I = 0; I + delta < nb; ++I) {
                        const int nt = min(kT, L - (I + delta) * kT);
                        for (int j = (a == 0 && finish) ? 1 : 0; j < nt; ++j) {
                            c1 += (uint64_t)(a + j);
                            ++cells;
                        }
                    }
                    if ((e = before(kEdge)) != hipSuccess)
                        return e;
                    launch_edge_row(a, nb - delta, stream, tb, delta, finish, w);
                    if ((e = launched(kEdge, c1, cells, cells)) != hipSuccess)
                        return e;
                }
                continue;
            }
            for (int q = finish; q <= 2 * kT - 2; ++q) {
                const int a_min = q - (kT - 1) > 0 ? q - (kT - 1) : 0;
                const int a_max = q < kT - 1 ? q : kT - 1;
                const int n_q = a_max - a_min + 1;
                uint64_t cells = 0;
                for (int I = 0; I + delta < nb; ++I)
                    for (int a = a_min; a <= a_max; ++a)
                        cells += ((I + delta) * kT + 1 + (q - a) <= L) ? 1 : 0;
                if ((e = before(kEdge)) != hipSuccess)
                    return e;
                edge_kernel<<<dim3(mb_edge, (nb - delta) * n_q, tb.n_chains), kEdgeThreads, 0, stream>>>(
                    tb.params, L, tb.M, tb.pitch, tb.rows, delta, q, a_min, n_q, tb.cost, tb.dec, w);
                if ((e = launched(kEdge, cells * (uint64_t)q, cells, cells)) != hipSuccess)
                    return e;
            }
        }
        return hipSuccess;
    };
    e = blocked();
    if (e != hipSuccess && side) {
        // a failed launch leaves no side-stream work behind the caller's
        // stream: it waits for all of it
        (void)hipEventRecord(side->done, side->stream);
        (void)hipStreamWaitEvent(stream, side->done, 0);
    }
    return e;
}

}  // namespace rotor
