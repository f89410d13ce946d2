// Edges of the blocked fill by rows (Theorem 1, Eq. (DP:mainrec)): the
// kernels, templated on the row's number of low splits.  Their
// instantiations are spread over rotor_rows_*.hip, which compile in
// parallel.  The value paths and the schedule are described at the head of
// rotor_fill.hip.
#pragma once

#include <utility>

#include "rotor_paths.h"

namespace rotor {
namespace {

// ---------------------------------------------------------------------------
// Edges by rows.  The edge splits of a cell (s, t) of block (I, J) read, for
// a low split k, X(s, k) in the diagonal block I (the same for every cell of
// row s) and Y(k + 1, t) further down column t of the block; for a high split
// k, X(s, k) further left in row s of the block and Y(k + 1, t) in the
// diagonal block J.  Row s therefore needs only the rows below it and its
// own cells to the left, at the same budget: one launch per row, bottom-up
// (a = 16(I + 1) - s low splits, the same in every block of the
// block-diagonal), and one workgroup walks a block's row at its budgets from
// left to right, keeping the finished cells of the row, with their u_f
// prefix, in registers as the X operands of the high splits, and the row's
// diagonal-block operands X(s, k) of the low splits loaded once for all 16
// cells.  Each candidate then streams one operand: a 4-byte cell of the
// block for a low split, a 2-byte diagonal-block cell for a high one, about
// half the bytes of the anti-diagonal rounds, in 16 launches instead of 30.
// But a wave walks 16 cells in turn, with at most about 45 loads in flight,
// and a launch has 16 times fewer waves than a round: the rows pay off only
// when a launch holds many blocks (a batch of chains), and the
// anti-diagonal rounds take the others.  Measured on MI355X: the batch of
// 256 chains of L = 64, M = 640 (768 blocks in the first launch) edges 4.89
// -> 4.41 ms; the single chain of L = 500, M = 5000 (31 blocks or fewer)
// 12.9 -> 16.2 ms if it took them.
constexpr int kRowBudgets = 1;  // budgets per lane, 64 apart (two spill registers)
constexpr int kRowMinBlocks = 256;  // blocks of all chains in one launch
constexpr int kRowAhead = 1;  // cells whose loads are in flight ahead of the one relaxed

// f(std::integral_constant<int, i>) for each i of the sequence, in order
template <class F, int... Is>
__device__ __forceinline__ void static_for(F &&f, std::integer_sequence<int, Is...>)
{
    (f(std::integral_constant<int, Is>{}), ...);
}

// A cell of a diagonal block as the value path reads it: from the 2-byte
// copy with H, else from the table the path reads.
template <class P, bool H>
__device__ __forceinline__ typename P::Raw diag_load(const ChainWork &cw, const int64_t *tab, int L, int64_t pitch,
                                                     int s, int t, int m)
{
    if constexpr (H) {
        return Load16::at((const char *)cw.half_row(s, t), m);
    } else {
        const int64_t o = row_of(L, s, t) * pitch;
        return P::load(tab + o, cw.shadow + o, m);
    }
}

// diag_load at budget m - w, or at budget 0 when m < w (the caller's flag
// discards that candidate).
template <class P, bool H>
__device__ __forceinline__ typename P::Raw diag_load_shifted(const ChainWork &cw, const int64_t *tab, int L,
                                                             int64_t pitch, int s, int t, int m, int w)
{
    if constexpr (H) {
        return Load16::at_off((const char *)cw.half_row(s, t), shifted_off<Load16::kBytes>((uint32_t)m * 2u, w));
    } else {
        const int64_t o = row_of(L, s, t) * pitch;
        return P::load_row_off(tab + o, cw.shadow + o, shifted_off<P::kBytes>((uint32_t)m * P::kBytes, w));
    }
}

// A finished cell's cost in the form the path loads it (infinity included).
template <class P>
__device__ __forceinline__ typename P::Raw final_raw(const typename P::Acc &a)
{
    if constexpr (P::kShadow)
        return a.val;
    else
        return P::finite(a) ? P::value(a) : kInf;
}

// Row s = k_lo - A of block (I, J) at the lane's budgets, cells
// t_first .. t_last (the corner, when the middle kernel finished it, is
// only read).  Splits are met in increasing order: low, the stored middle
// partial, high.  The row's scalars (shift sizes, prefix sums, gates) are
// loaded first, all at once; then the loads of cell j + kRowAhead are
// issued before cell j is relaxed and stored, in one straight-line body
// (columns past L read the last column and store nothing).  Scheduling
// barriers keep that order: a load may not pass an earlier store to the
// same table, and hoisting more loads would hold the whole row's operands
// in registers.
// With YS the Y operands of the high splits (diagonal block J) are all
// saturated at the workgroup's budgets (head of rotor_fill.hip): least times,
// not loaded.
template <class P, bool H, bool PP, int A, bool YS>
__device__ __forceinline__ void row_body(const ChainRows &r, const ChainWork &cw, int L, int M, int m0, int64_t pitch,
                                         int s, int J, int t_first, int t_last, int64_t *tab, int16_t *dtab)
{
    constexpr int NB = kRowBudgets;
    const int k_lo = s + A;  // 16(I + 1)
    const int k_hi = J * kT;
    // the lane's budgets m0 + b * 64; those past M load budget M and store nothing
    int m[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b)
        m[b] = min(m0 + b * kEdgeThreads, M);
    // prefix sums and gates through the constant address space (written by
    // prep_kernel, read-only here): scalar loads
    const const_i64 pre = (const_i64)cw.pre;
    const const_i32 gall_c = (const_i32)cw.gall, gnone_c = (const_i32)cw.gnone;
    const int64_t pre_s = pre[s - 1];
    // per low split k = s + i: w_a^k and the u_f prefix from s to k; per
    // column j (t = min(k_hi + 1 + j, L)): w_a^t, the prefix to t, the gates
    int w_lo[A > 0 ? A : 1];
    uint64_t p_lo[A > 0 ? A : 1];
#pragma unroll
    for (int i = 0; i < A; ++i) {
        w_lo[i] = r.wa[s + i - 1];
        p_lo[i] = (uint64_t)(pre[s + i] - pre_s);
    }
    int w_t[kT];
    uint64_t p_t[kT];
    int32_t g_all[kT], g_none[kT];
#pragma unroll
    for (int j = 0; j < kT; ++j) {
        const int t = min(k_hi + 1 + j, L);
        w_t[j] = r.wa[t - 1];
        p_t[j] = (uint64_t)(pre[t] - pre_s);
        const int64_t crow = row_of(L, s, t);
        g_all[j] = gall_c[crow];
        g_none[j] = gnone_c[crow];
    }
    // the stored middle partial counts u_f from k_lo on
    const uint64_t pre_lo = (uint64_t)(pre[k_lo - 1] - pre_s);
    const int wab = r.wabar[s - 1];
    const uint64_t ufub = (uint64_t)(r.uf[s - 1] + r.ub[s - 1]);
    // PP: the middle partial is a packed key in the compact copy (else
    // (value << 32) | s' or a 64-bit key in the cost table)
    const int S = k_hi > k_lo ? 32 - __clz(k_hi - k_lo) : 0;
    // X of the low splits k = s .. k_lo - 1, with the u_f prefix from s
    typename P::X xl[A > 0 ? A : 1][NB];
#pragma unroll
    for (int i = 0; i < A; ++i) {
        const int k = s + i;
#pragma unroll
        for (int b = 0; b < NB; ++b)
            xl[i][b] = P::xop(diag_load<P, H>(cw, tab, L, pitch, s, k, m[b]), p_lo[i], (uint32_t)(k + 1),
                              m[b] >= w_lo[i]);
    }
    // the corner (A = 0, first column) when the middle kernel finished it
    const bool corner_done = A == 0 && t_first > k_hi + 1;
    // X of the high splits: the row's finished cells, with the u_f prefix
    typename P::X xh[kT - 1][NB];
    // the operands of each cell: the stored partial, C_2's, the splits'
    struct Loads {
        uint32_t key[NB];
        int64_t stored64[NB];
        typename P::Raw c2[NB];
        typename P::Raw yl[A > 0 ? A : 1][NB];
        typename P::Raw yh[kT - 1][NB];
    } ld[kT];
    auto load_j = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        const int t = min(k_hi + 1 + j, L);  // columns past L read the last one
        const int64_t cell = row_of(L, s, t) * pitch;
        if constexpr (j == 0 && A == 0) {
            if (corner_done) {
                // the corner's final cost, as X of the high splits
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    ld[0].c2[b] = P::load(tab + cell, cw.shadow + cell, m[b]);
                return;
            }
        }
        const int64_t below = row_of(L, s + 1, t) * pitch;
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            if constexpr (PP)
                ld[j].key[b] = __builtin_nontemporal_load(cw.shadow + cell + m[b]);
            else
                ld[j].stored64[b] = load64(tab + cell, m[b]);
            const int ri = m[b] - wab;
            ld[j].c2[b] = P::load(tab + below, cw.shadow + below, m[b] >= g_all[j] && ri >= 0 ? ri : m[b]);
        }
#pragma unroll
        for (int i = 0; i < A; ++i) {
            const int64_t yrow = row_of(L, s + i + 1, t) * pitch;
#pragma unroll
            for (int b = 0; b < NB; ++b)
                ld[j].yl[i][b] = P::load_row_off(tab + yrow, cw.shadow + yrow,
                                                 shifted_off<P::kBytes>((uint32_t)m[b] * P::kBytes, w_lo[i]));
        }
#pragma unroll
        for (int i = 0; i < j; ++i) {
            // split k = k_hi + 1 + i, Y at (k + 1, t) (within the block for every t <= L)
            const int k1 = min(k_hi + 2 + i, t);
            if constexpr (YS) {
                const const_i64 pa = (const_i64)cw.preall;
                const typename P::Raw lt = (typename P::Raw)(pa[t] - pa[k1 - 1]);
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    ld[j].yh[i][b] = lt;
            } else {
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    ld[j].yh[i][b] = diag_load_shifted<P, H>(cw, tab, L, pitch, k1, t, m[b], w_t[i]);
            }
        }
    };
    auto comp_j = [&](auto jc) {
        constexpr int j = decltype(jc)::value;
        const int t = k_hi + 1 + j;
        if constexpr (j == 0 && A == 0) {
            if (corner_done) {
#pragma unroll
                for (int b = 0; b < NB; ++b)
                    xh[0][b] = P::xop(ld[0].c2[b], p_t[0], (uint32_t)(t + 1), m[b] >= w_t[0]);
                return;
            }
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            typename P::Acc a;
            P::init(a);
#pragma unroll
            for (int i = 0; i < A; ++i)
                P::relax(a, xl[i][b], P::yop(ld[j].yl[i][b]), (uint32_t)(s + i + 1));
            int64_t stored;
            if constexpr (!PP) {
                stored = ld[j].stored64[b];
            } else {
                const uint32_t key = ld[j].key[b];
                const uint32_t split = (uint32_t)(k_lo + 1) + (key & ((1u << S) - 1u));
                stored = key == kInf32 ? (int64_t)((uint64_t)kInf32 << 32)
                                       : (int64_t)(((uint64_t)(key >> S) << 32) | split);
            }
            P::merge_stored(a, stored, pre_lo);
#pragma unroll
            for (int i = 0; i < j; ++i)
                P::relax(a, xh[i][b], P::yop(ld[j].yh[i][b]), (uint32_t)(k_hi + 2 + i));
            if (m[b] < g_none[j])
                P::init(a);
            if (m[b] >= g_all[j] && m[b] >= wab)
                P::relax_all(a, ld[j].c2[b], ufub);
            if constexpr (j + 1 < kT)
                xh[j][b] = P::xop(final_raw<P>(a), p_t[j], (uint32_t)(t + 1), m[b] >= w_t[j]);
            const int mb = m0 + b * kEdgeThreads;
            if (t <= t_last && mb <= M)
                store_cell<P>(tab, dtab, cw.shadow, row_of(L, s, t) * pitch + mb, a);
        }
    };
    static_for([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        if constexpr (j < kRowAhead)
            load_j(std::integral_constant<int, j>{});
    }, std::make_integer_sequence<int, kT>{});
    static_for([&](auto jc) {
        constexpr int j = decltype(jc)::value;
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (j + kRowAhead < kT)
            load_j(std::integral_constant<int, j + kRowAhead>{});
        __builtin_amdgcn_sched_barrier(0);
        comp_j(jc);
    }, std::make_integer_sequence<int, kT>{});
}

// Row 16(I + 1) - A of every block (I, I + delta) of one block-diagonal; a
// workgroup is one wave at 64 kRowBudgets consecutive budgets (kRowBudgets
// per lane, 64 apart) of one block.
// With `finish`, the middle kernels finished the corner (row 16I + 16,
// column 16J + 1).
template <int A>
__global__ __launch_bounds__(kEdgeThreads) void edge_row_kernel(const int64_t *__restrict__ params, int L, int M,
                                                                int64_t pitch, int64_t rows, int delta, int finish,
                                                                int64_t *__restrict__ cost,
                                                                int16_t *__restrict__ dec, Work w)
{
    const int c = blockIdx.z;
    const int I = blockIdx.y;
    const int J = I + delta;
    const int s = (I + 1) * kT - A;
    const int m0 = blockIdx.x * (kEdgeThreads * kRowBudgets) + threadIdx.x;
    if (m0 > M)
        return;
    const int t_first = J * kT + 1 + (A == 0 && finish ? 1 : 0);
    const int t_last = min(J * kT + kT, L);
    const ChainRows r = chain_rows(params, w, L, c);
    const ChainWork cw = chain_work(w, L, rows, pitch, c);
    int64_t *tab = cost + (int64_t)c * rows * pitch;
    int16_t *dtab = dec + (int64_t)c * rows * pitch;
    // every budget of the workgroup saturated in every cell of the row
    // (head of rotor_fill.hip): least times and C_2, nothing loaded; tried
    // only when some cell of the block is saturated there
    const int base = blockIdx.x * (kEdgeThreads * kRowBudgets);
    if (base >= block_gmin(cw, I, delta) && r.uf[s - 1] > 0) {
        const const_i32 gsat = (const_i32)cw.gsat;
        bool all = true;
        for (int t = t_first; t <= t_last; ++t)
            all = all && base >= gsat[row_of(L, s, t)];
        if (all) {
            for (int t = t_first; t <= t_last; ++t) {
                const int64_t idx = row_of(L, s, t) * pitch;
                const int64_t lt = least_time(cw, s, t);
#pragma unroll
                for (int b = 0; b < kRowBudgets; ++b) {
                    const int mb = m0 + b * kEdgeThreads;
                    if (mb > M)
                        continue;
                    if (cw.narrow(delta))
                        store_cell<Narrow>(tab, dtab, cw.shadow, idx + mb, Narrow::all_only(lt));
                    else
                        store_cell<Wide>(tab, dtab, cw.shadow, idx + mb, Wide::all_only(lt));
                }
            }
            return;
        }
    }
    const bool packed = middle_packed(cw, delta, (delta - 1) * kT);
    // the high splits' Y rows, in diagonal block J, all saturated here
    const bool ysat = base >= diag_block_gyshift(cw, J);
    if (cw.narrow(delta) && cw.diag16() && packed && ysat)
        row_body<Narrow, true, true, A, true>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
    else if (!cw.narrow(delta))
        row_body<Wide, false, false, A, false>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
    else if (cw.diag16() && packed)
        row_body<Narrow, true, true, A, false>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
    else if (cw.diag16())
        row_body<Narrow, true, false, A, false>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
    else if (packed)
        row_body<Narrow, false, true, A, false>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
    else
        row_body<Narrow, false, false, A, false>(r, cw, L, M, m0, pitch, s, J, t_first, t_last, tab, dtab);
}

// edge_row_kernel<a> for a launch-time a in [A0, A1]
template <int A0, int A1>
void launch_edge_row_range(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish,
                           const Work &w)
{
    if (a == A0)
        edge_row_kernel<A0><<<grid, kEdgeThreads, 0, stream>>>(tb.params, tb.L, tb.M, tb.pitch, tb.rows, delta,
                                                                finish, tb.cost, tb.dec, w);
    else if constexpr (A0 < A1)
        launch_edge_row_range<A0 + 1, A1>(a, grid, stream, tb, delta, finish, w);
}

}  // namespace

// One range of row lengths each, in rotor_rows_*.hip.
void launch_edge_row_0(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w);
void launch_edge_row_1(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w);
void launch_edge_row_2(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w);
void launch_edge_row_3(int a, dim3 grid, hipStream_t stream, const Tables &tb, int delta, int finish, const Work &w);

}  // namespace rotor
