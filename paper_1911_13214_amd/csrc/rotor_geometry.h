// Table geometry, workspace layout and the input domain of the library,
// shared by the host-only sources and the kernels.  No HIP header is needed:
// the inline helpers are constexpr, which the HIP compiler also accepts in
// device code, so the host-only sources build with a plain C++ compiler too.
#pragma once

#include <stdint.h>

#include "rotor.h"

namespace rotor {

// Side of the square blocks of pairs of the blocked fill, in stages.
constexpr int kBlock = 16;

// Domain of the library (checked on the host by rotor_check_params and on
// the device by the fill's first kernel): every value >= 0, sizes and
// overheads < 2^30, M < 2^28, and per chain L * sum(u_f) + sum(u_b) < 2^44.
// The cost limit lets the 64-bit value path carry a candidate as one key
// (value << 16) | s'; M < 2^28 keeps byte offsets within a row in 32 bits.
constexpr int64_t kMaxSize = (int64_t)1 << 30;
constexpr int64_t kMaxBudget = (int64_t)1 << 28;
constexpr uint64_t kCostBound = (uint64_t)1 << 44;

// Row of the pair (s, t), 1 <= s <= t <= L, in a chain's table: the upper
// triangle stored s-major, so the rows (s, s), (s, s+1), ..., (s, L) are
// consecutive and the row of (s, t+1) follows the row of (s, t).
constexpr int64_t row_of(int L, int s, int t)
{
    return (int64_t)(s - 1) * L - (int64_t)(s - 1) * (s - 2) / 2 + (t - s);
}

// Row pitch: M + 1 rounded up to 32 elements, so that every row of the int64
// table starts 256 bytes and every row of the 4-byte compact copy 128 bytes
// (one cache line) after an aligned table base.
constexpr int64_t pitch_of(int64_t M) { return (M + 1 + 31) / 32 * 32; }

// Row pitch of the 2-byte copy of the diagonal blocks: a multiple of 64
// elements (128 bytes).
constexpr int64_t half_pitch_of(int64_t pitch) { return (pitch + 63) / 64 * 64; }

// Whether the batch sizes are within what the ABI accepts.
constexpr bool sizes_ok(int32_t n_chains, int32_t L, int64_t M)
{
    return n_chains >= 1 && n_chains <= ROTOR_MAX_CHAINS && L >= 1 && L <= ROTOR_MAX_L && M >= 0 && M < kMaxBudget;
}

// Number of elements of one table, or 0 if its bytes would not fit 63 bits.
uint64_t table_elems(int32_t n_chains, int32_t L, int64_t M);

// Byte offsets of the workspace sections (each 256-byte aligned): prefix
// sums of u_f, per-block-diagonal key widths and the sums they come from,
// the gates m_none and m_all of every pair, a per-chain domain status word,
// the shift sizes the fill reads, the compact uint32 copy of the cost table
// and the 2-byte copy of the diagonal blocks' cells.
struct WorkLayout {
    uint64_t pre, preall, pbits, bsum, gnone, gall, gsat, gblk, status, shift, shadow, half, total;
};
WorkLayout work_layout(int n_chains, int L, int64_t pitch);

}  // namespace rotor
