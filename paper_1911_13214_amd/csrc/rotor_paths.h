// Device-side building blocks of the table fill shared by its kernels
// (rotor_fill.hip, rotor_rows.hip): the chain views, operand loads, the
// narrow and wide value paths and the stores of a finished cell.  The
// recurrence, the value paths and the fill schedules are described at the
// head of rotor_fill.hip.
#pragma once

#include "rotor_internal.h"

namespace rotor {
namespace {

constexpr int64_t kInf = INT64_MAX;
constexpr int kT = kBlock;  // block side, in stages
constexpr int kSub = 8;  // per-wave register tile side
// An edge workgroup is one wave holding kEdgeBudgets budgets per lane, 64
// apart: 128 consecutive budgets, whose loads it issues together (measured on
// MI355X at L = 500, M = 5000, against one budget per lane in 128-thread
// workgroups: edges 13.70 -> 13.24 ms; 128-thread workgroups of two budgets
// per lane 13.53 ms, three or four budgets per lane 14.0-14.4 ms).
constexpr int kEdgeThreads = 64;
constexpr int kEdgeBudgets = 2;
// diag_kernel's workgroups in the blocked order (one wave, like the edges')
// hold four budgets per lane, 256 consecutive budgets (measured on MI355X:
// the batch of 256 chains of L = 64, M = 640, 0.67 -> 0.54 ms of diagonal
// blocks; the edges lose with four, 10.4 -> 12.3 ms at L = 500, M = 5000, and
// so do the small tables of the streamed order, 3-6%)
constexpr int kDiagBudgets = 4;
constexpr uint32_t kAllSplit = 0xFFFF;  // split field of a C_2 candidate
constexpr uint32_t kInf32 = 0xFFFFFFFFu;
constexpr uint64_t kNarrowBound = 0xFFFFFFFFull;  // V_D below: the narrow path
// V_D below: the middle products' keys value * 2^15 + (split offset) stay
// below 2^53, exact as doubles
constexpr uint64_t kF64Bound = 1ull << 38;

// The parameters of one chain as given (stage l at index l-1).
struct ChainParams {
    const int64_t *uf, *ub, *wa, *wabar, *of, *ob;
};

__device__ inline ChainParams chain_params(const int64_t *__restrict__ params, int L, int c)
{
    const int64_t *p = params + (int64_t)c * ROTOR_N_ROWS * L;
    return {p + ROTOR_ROW_UF * L, p + ROTOR_ROW_UB * L, p + ROTOR_ROW_WA * L,
            p + ROTOR_ROW_WABAR * L, p + ROTOR_ROW_OF * L, p + ROTOR_ROW_OB * L};
}

// What the fill kernels read of a chain: the times as given and the two
// sizes that shift operand budgets, w_a and w_abar, as prep_kernel clamped
// them into [0, M + 1] (stage l at index l-1).  In the domain the clamp
// changes nothing the recurrence sees (a shift beyond M puts every operand
// out of reach either way); outside it, every shifted budget m - w stays
// within [m - M - 1, m], so an operand is only ever loaded at a budget in
// [0, M], whatever the parameter values.
// The sizes are read through the constant address space: written by an
// earlier kernel and read-only during the fill, they then take scalar loads
// like the parameters, which the compiler could not assume for a workspace
// pointer the kernel also writes through.
typedef const __attribute__((address_space(4))) int32_t *const_i32;
typedef const __attribute__((address_space(4))) int64_t *const_i64;
struct ChainRows {
    const int64_t *uf, *ub;
    const_i32 wa, wabar;
};

__device__ inline ChainRows chain_rows(const int64_t *__restrict__ params, const Work &w, int L, int c)
{
    const int64_t *p = params + (int64_t)c * ROTOR_N_ROWS * L;
    const_i32 sh = (const_i32)(w.shift + (int64_t)c * 2 * L);
    return {p + ROTOR_ROW_UF * L, p + ROTOR_ROW_UB * L, sh, sh + L};
}

typedef const __attribute__((address_space(1))) int64_t *global_c64;
typedef const __attribute__((address_space(1))) uint32_t *global_c32;
typedef __attribute__((address_space(1))) uint64_t *global_u64;

// Load budget m of a table row: global address space, 32-bit byte offset
// (M < 2^28).
__device__ inline int64_t load64(const int64_t *row, int m)
{
    return *(global_c64)((const char *)row + (uint32_t)m * 8u);
}
__device__ inline uint32_t load32(const uint32_t *row, int m)
{
    return *(global_c32)((const char *)row + (uint32_t)m * 4u);
}

__device__ inline uint32_t sat_add(uint32_t a, uint32_t b) { return __builtin_elementwise_add_sat(a, b); }
__device__ inline uint64_t umin(uint64_t a, uint64_t b) { return b < a ? b : a; }

// Per-chain views of the workspace.
struct ChainWork {
    const int64_t *pre;    // [L+1] prefix sums of u_f
    const int64_t *preall; // [L+1] prefix sums of u_f + u_b
    const int32_t *gnone;  // [rows] m_none(s, t), t > s
    const int32_t *gall;   // [rows] m_all(s, t)
    const int32_t *gsat;   // [rows] G(s, t), the budget from which C_2 reaches the least time
    const int32_t *gblk;   // [2][nb][nb] per block (I, I + D), D >= 1: least G of its cells, then the
                           // largest (INT32_MAX if some row has u_f = 0); D = 0: the diagonal block's
                           // largest G plus its largest w_a, then its largest G
    int nb;
    uint32_t *shadow;      // [rows][pitch] compact copy of the costs (narrow block-diagonals)
    const int32_t *pbits;  // [nb] per block-diagonal D: the largest S with (V_D + 1) << S <= 2^32 - 1,
                           // or, if V_D >= 2^32 - 1 (64-bit path), -2 while V_D < 2^38, else -1
    int16_t *half;         // [16 L][hpitch] 2-byte copy of the diagonal blocks' cells
    int64_t hpitch;
    // whether the pairs of block-diagonal D take the narrow path
    __device__ bool narrow(int D) const { return pbits[D] >= 0; }
    // whether the middle keys value * 2^15 + (split offset) of block-diagonal
    // D are exact as doubles (V_D < 2^38)
    __device__ bool f64_keys(int D) const { return pbits[D] != -1; }
    // whether the diagonal blocks' costs fit the 2-byte copy: (V_0 + 1) << 17
    // <= 2^32 - 1, i.e. V_0 <= 2^15 - 2, so finite values stay positive as
    // int16 and infinity is stored as -1 (0xFFFF)
    __device__ bool diag16() const { return pbits[0] >= 17; }
    // row of the pair (s, t) of a diagonal block in the 2-byte copy:
    // 16 (s - 1) + (t - 1) mod 16
    __device__ int16_t *half_row(int s, int t) const
    {
        return half + ((int64_t)(s - 1) * kT + (t - 1) % kT) * hpitch;
    }
};

// Block-diagonal of the pair (s, t): D = J - I for s in block I, t in block J.
__device__ inline int block_diag(int s, int t) { return (t - 1) / kT - (s - 1) / kT; }

__device__ inline ChainWork chain_work(const Work &w, int L, int64_t rows, int64_t pitch, int c)
{
    ChainWork cw;
    cw.pre = w.pre + (int64_t)c * (L + 1);
    cw.preall = w.preall + (int64_t)c * (L + 1);
    cw.gnone = w.gnone + (int64_t)c * rows;
    cw.gall = w.gall + (int64_t)c * rows;
    cw.gsat = w.gsat + (int64_t)c * rows;
    cw.nb = (L + kT - 1) / kT;
    cw.gblk = w.gblk + (int64_t)c * 2 * cw.nb * cw.nb;
    cw.shadow = w.shadow + (int64_t)c * rows * pitch;
    cw.pbits = w.pbits + (int64_t)c * ((L + kT - 1) / kT);
    cw.hpitch = half_pitch_of(pitch);
    cw.half = w.half + (int64_t)c * L * kT * cw.hpitch;
    return cw;
}

// ---------------------------------------------------------------------------
// Value paths.  X is the left operand with its u_f prefix, Y the shifted
// right operand; relax() folds one candidate into an accumulator.

// A stored cost shifted into the value field of a wide key.
__device__ inline uint64_t key_of(int64_t v)
{
    const uint64_t t = (uint64_t)v << 16;
    const uint32_t hi = min((uint32_t)(t >> 32), 1u << 30);
    return ((uint64_t)hi << 32) | (uint32_t)t;
}

struct Wide {
    typedef int64_t Raw;
    typedef uint64_t X;
    typedef uint64_t Y;
    struct Acc {
        uint64_t key;
    };
    static constexpr bool kShadow = false;
    static constexpr uint64_t kShiftedOut = 1ull << 62;
    static constexpr int kBytes = 8;  // bytes per cell of the table it reads
    __device__ static const char *table(const int64_t *tab, const uint32_t *) { return (const char *)tab; }
    __device__ static Raw load_at(const char *row, int m) { return *(global_c64)(row + (uint32_t)m * 8u); }
    __device__ static Raw load_off(const char *row, uint32_t off) { return *(global_c64)(row + off); }
    __device__ static Raw load(const int64_t *crow, const uint32_t *, int m) { return load64(crow, m); }
    __device__ static Raw load_row_off(const int64_t *crow, const uint32_t *, uint32_t off)
    {
        return *(global_c64)((const char *)crow + off);
    }
    __device__ static void init(Acc &a) { a.key = ~0ull; }
    // ok = false: the budget of Y was shifted below 0, the candidate is infinite
    __device__ static X xop(Raw x, uint64_t prefix, uint32_t sp, bool ok)
    {
        return key_of(x) + (ok ? ((prefix << 16) | sp) : kShiftedOut);
    }
    __device__ static Y yop(Raw y) { return key_of(y); }
    __device__ static void relax(Acc &a, X x, Y y, uint32_t) { a.key = umin(a.key, x + y); }
    // the stored middle partial counts u_f from the first middle split on
    __device__ static void merge_stored(Acc &a, int64_t stored, uint64_t prefix)
    {
        a.key = umin(a.key, (uint64_t)stored + (prefix << 16));
    }
    __device__ static void relax_all(Acc &a, Raw y, uint64_t ufub)
    {
        a.key = umin(a.key, key_of(y) + ((ufub << 16) | kAllSplit));
    }
    __device__ static int64_t stored(const Acc &a) { return (int64_t)a.key; }
    // fold in the stored() form of a result over larger splits
    __device__ static void merge_later(Acc &a, int64_t later) { a.key = umin(a.key, (uint64_t)later); }
    __device__ static bool finite(const Acc &a) { return a.key < (1ull << 62); }
    // the result of a cell whose C_2 alone reaches the finite value v
    __device__ static Acc all_only(int64_t v) { return {((uint64_t)v << 16) | kAllSplit}; }
    __device__ static int64_t value(const Acc &a) { return (int64_t)(a.key >> 16); }
    __device__ static uint32_t split(const Acc &a) { return (uint32_t)(a.key & 0xFFFF); }
};

struct Narrow {
    typedef uint32_t Raw;
    typedef uint32_t X;
    typedef uint32_t Y;
    struct Acc {
        uint32_t val;
        uint32_t sp;
    };
    static constexpr bool kShadow = true;
    static constexpr int kBytes = 4;
    __device__ static const char *table(const int64_t *, const uint32_t *shadow) { return (const char *)shadow; }
    __device__ static Raw load_at(const char *row, int m) { return *(global_c32)(row + (uint32_t)m * 4u); }
    __device__ static Raw load_off(const char *row, uint32_t off) { return *(global_c32)(row + off); }
    __device__ static Raw load(const int64_t *, const uint32_t *srow, int m) { return load32(srow, m); }
    __device__ static Raw load_row_off(const int64_t *, const uint32_t *srow, uint32_t off)
    {
        return *(global_c32)((const char *)srow + off);
    }
    __device__ static void init(Acc &a)
    {
        a.val = kInf32;
        a.sp = 0;
    }
    __device__ static X xop(Raw x, uint64_t prefix, uint32_t, bool ok)
    {
        return sat_add(x, ok ? (uint32_t)prefix : kInf32);
    }
    __device__ static Y yop(Raw y) { return y; }
    // splits are visited in increasing s': a strict < keeps the smallest
    __device__ static void relax(Acc &a, X x, Y y, uint32_t sp)
    {
        const uint32_t v = sat_add(x, y);
        const bool b = v < a.val;
        a.val = b ? v : a.val;
        a.sp = b ? sp : a.sp;
    }
    __device__ static void merge_stored(Acc &a, int64_t stored, uint64_t prefix)
    {
        const uint32_t v = sat_add((uint32_t)((uint64_t)stored >> 32), (uint32_t)prefix);
        const bool b = v < a.val;
        a.val = b ? v : a.val;
        a.sp = b ? (uint32_t)stored : a.sp;
    }
    __device__ static void relax_all(Acc &a, Raw y, uint64_t ufub)
    {
        const uint32_t v = sat_add(y, (uint32_t)ufub);
        const bool b = v < a.val;
        a.val = b ? v : a.val;
        a.sp = b ? kAllSplit : a.sp;
    }
    __device__ static int64_t stored(const Acc &a) { return (int64_t)(((uint64_t)a.val << 32) | a.sp); }
    // fold in the stored() form of a result over larger splits: strict <
    __device__ static void merge_later(Acc &a, int64_t later)
    {
        const uint32_t v = (uint32_t)((uint64_t)later >> 32);
        const bool b = v < a.val;
        a.val = b ? v : a.val;
        a.sp = b ? (uint32_t)later : a.sp;
    }
    __device__ static bool finite(const Acc &a) { return a.val != kInf32; }
    __device__ static Acc all_only(int64_t v) { return {(uint32_t)v, kAllSplit}; }
    __device__ static int64_t value(const Acc &a) { return (int64_t)a.val; }
    __device__ static uint32_t split(const Acc &a) { return a.sp; }
};

// Final cost and decision of a cell, and its compact copy on the narrow path.
// idx is relative to the chain's tables.  On the narrow path the fill never
// reads the int64 cost or the decision of a finished cell back, so they are
// stored non-temporally and leave the caches to the operands (measured on
// MI355X: 25.4 -> 24.7 ms at L = 500, M = 5000); the 64-bit path reads its
// cells as operands and stores them normally.
template <class P>
__device__ inline void store_cell(int64_t *cost, int16_t *dec, uint32_t *shadow, int64_t idx,
                                  const typename P::Acc &a)
{
    const bool fin = P::finite(a);
    const uint32_t sp = P::split(a);
    const int64_t v = fin ? P::value(a) : kInf;
    const int16_t d = fin ? (sp == kAllSplit ? (int16_t)0 : (int16_t)sp) : (int16_t)-1;
    if constexpr (P::kShadow) {
        __builtin_nontemporal_store(v, &cost[idx]);
        __builtin_nontemporal_store(d, &dec[idx]);
        shadow[idx] = fin ? (uint32_t)v : kInf32;
    } else {
        cost[idx] = v;
        dec[idx] = d;
    }
}

// Saturated budgets (head of rotor_fill.hip): whether every budget from
// `base` on of the pair (s, t), whose row is `cell`, has the least time as
// its cost and C_2 as its decision.  Uniform over a wave when base is.
__device__ inline bool saturated(const ChainRows &r, const ChainWork &cw, int s, int64_t cell, int base)
{
    // both loads unconditional, so that they are issued together
    const int64_t uf = r.uf[s - 1];
    const int32_t g = ((const_i32)cw.gsat)[cell];
    return (uf > 0) & (base >= g);
}

// The least and the largest G of the cells of block (I, I + D), D >= 1.
__device__ inline int32_t block_gmin(const ChainWork &cw, int I, int D)
{
    return ((const_i32)cw.gblk)[(int64_t)I * cw.nb + D];
}
__device__ inline int32_t block_gmax(const ChainWork &cw, int I, int D)
{
    return ((const_i32)cw.gblk)[((int64_t)cw.nb + I) * cw.nb + D];
}

// For the diagonal block I (D = 0): the largest G of its pairs, whatever
// the u_f; and that plus the largest w_a of its stages.
__device__ inline int32_t diag_block_gmax(const ChainWork &cw, int I) { return block_gmax(cw, I, 0); }
__device__ inline int32_t diag_block_gyshift(const ChainWork &cw, int I) { return block_gmin(cw, I, 0); }

// saturated() for a cell of block (I, I + D), D >= 1, tried only when some
// cell of the block is saturated from `base` on: a block read by every
// workgroup of the block, then the cell's own bound.
__device__ inline bool saturated_in_block(const ChainRows &r, const ChainWork &cw, int I, int D, int s,
                                          int64_t cell, int base)
{
    return base >= block_gmin(cw, I, D) && saturated(r, cw, s, cell, base);
}

// The least time of the pair (s, t): every stage forward once and backward
// once, sum_{j=s}^{t} (u_f^j + u_b^j).
__device__ inline int64_t least_time(const ChainWork &cw, int s, int t)
{
    const const_i64 pa = (const_i64)cw.preall;
    return pa[t] - pa[s - 1];
}

// Operand loads of the narrow path from the compact copy (4 bytes) or from
// the 2-byte copy of the diagonal blocks (a sign-extending load: finite
// values there are below 2^15, and the infinity 0xFFFF becomes 0xFFFFFFFF).
typedef const __attribute__((address_space(1))) int16_t *global_c16;
struct Load32 {
    static constexpr uint32_t kBytes = 4;
    __device__ static uint32_t at(const char *row, int m) { return *(global_c32)(row + (uint32_t)m * 4u); }
    __device__ static uint32_t at_off(const char *row, uint32_t off) { return *(global_c32)(row + off); }
};
struct Load16 {
    static constexpr uint32_t kBytes = 2;
    __device__ static uint32_t at(const char *row, int m)
    {
        return (uint32_t)(int32_t) * (global_c16)(row + (uint32_t)m * 2u);
    }
    __device__ static uint32_t at_off(const char *row, uint32_t off)
    {
        return (uint32_t)(int32_t) * (global_c16)(row + off);
    }
};

// Byte offset of budget m - w in a row of B-byte cells, from the lane's
// m * B: budget 0 when m < w, where the caller's flag (m >= w) discards the
// candidate.  One saturating subtraction instead of a compare and a select
// before the scaling; in bounds for the shift sizes of ChainRows, which lie
// in [0, M + 1].
template <uint32_t B>
__device__ inline uint32_t shifted_off(uint32_t m_bytes, int w)
{
    return __builtin_elementwise_sub_sat(m_bytes, (uint32_t)w * B);
}

// Whether the middle products of block-diagonal D of a chain, whose middle
// split range has span + 1 splits, use packed keys.
__device__ inline bool middle_packed(const ChainWork &cw, int D, int span)
{
    const int S = span > 0 ? 32 - __clz(span) : 0;
    return cw.narrow(D) && S <= cw.pbits[D];
}

// A narrow block-diagonal whose middle range is too wide for one packed key
// takes packed runs of 2^pbits[D] splits instead (middle_packed_kernel), if
// runs are 128 splits or more; each run's result goes to the cost table as
// (value << 32) | s', the form middle_kernel stores.
constexpr int kMinRunBits = 7;
__device__ inline bool middle_runs(const ChainWork &cw, int D, int span)
{
    return cw.narrow(D) && !middle_packed(cw, D, span) && cw.pbits[D] >= kMinRunBits;
}

}  // namespace
}  // namespace rotor
