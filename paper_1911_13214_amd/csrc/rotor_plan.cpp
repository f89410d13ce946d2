// Front end of the solver (host only): discretisation of memory sizes into
// slots (Section 5.2), the memory of the schedule that stores everything,
// equally spaced budgets (the experimental setting of Section 5.3), and the
// time and memory the model predicts for an operation sequence.
#include <stdint.h>

#include <vector>

#include "rotor.h"

namespace {

constexpr int64_t kMaxSlots = (int64_t)1 << 28;
constexpr int64_t kMaxSize = (int64_t)1 << 30;

bool is_size_row(int row)
{
    return row == ROTOR_ROW_WA || row == ROTOR_ROW_WABAR || row == ROTOR_ROW_OF || row == ROTOR_ROW_OB;
}

// ceil(v * slots / mem) in 128-bit arithmetic (v, slots, mem >= 0, mem > 0).
int64_t slots_of(int64_t v, int64_t slots, int64_t mem)
{
    const unsigned __int128 num = (unsigned __int128)(uint64_t)v * (uint64_t)slots;
    const unsigned __int128 q = (num + (uint64_t)mem - 1) / (uint64_t)mem;
    return q >= (unsigned __int128)kMaxSize ? kMaxSize : (int64_t)q;
}

}  // namespace

extern "C" {

int32_t rotor_discretize(const int64_t *h_params, int32_t n_chains, int32_t L, const int64_t *h_mem_bytes,
                         int64_t slots, int64_t *h_out)
{
    if (!h_params || !h_mem_bytes || !h_out || n_chains < 1 || n_chains > ROTOR_MAX_CHAINS || L < 1 ||
        L > ROTOR_MAX_L || slots < 1 || slots >= kMaxSlots)
        return ROTOR_EINVAL;
    for (int32_t c = 0; c < n_chains; ++c)
        if (h_mem_bytes[c] <= 0)
            return ROTOR_EINVAL;
    const int64_t n = (int64_t)n_chains * ROTOR_N_ROWS * L;
    for (int64_t i = 0; i < n; ++i) {
        const int64_t v = h_params[i];
        if (v < 0)
            return ROTOR_EDOMAIN;
        const int row = (int)((i / L) % ROTOR_N_ROWS);
        if (is_size_row(row) && slots_of(v, slots, h_mem_bytes[i / ((int64_t)ROTOR_N_ROWS * L)]) >= kMaxSize)
            return ROTOR_EDOMAIN;
    }
    for (int64_t i = 0; i < n; ++i) {
        const int row = (int)((i / L) % ROTOR_N_ROWS);
        const int64_t mem = h_mem_bytes[i / ((int64_t)ROTOR_N_ROWS * L)];
        h_out[i] = is_size_row(row) ? slots_of(h_params[i], slots, mem) : h_params[i];
    }
    return ROTOR_OK;
}

int32_t rotor_store_all_peak(const int64_t *h_params, int32_t L, int64_t *peak)
{
    if (!h_params || !peak || L < 1 || L > ROTOR_MAX_L)
        return ROTOR_EINVAL;
    for (int64_t i = 0; i < (int64_t)ROTOR_N_ROWS * L; ++i)
        if (h_params[i] < 0)
            return ROTOR_EDOMAIN;
    const int64_t *wa = h_params + (int64_t)ROTOR_ROW_WA * L;
    const int64_t *wabar = h_params + (int64_t)ROTOR_ROW_WABAR * L;
    const int64_t *of = h_params + (int64_t)ROTOR_ROW_OF * L;
    const int64_t *ob = h_params + (int64_t)ROTOR_ROW_OB * L;
    // values are < 2^63 / (3L + 2) in any sane input; saturate otherwise
    auto add = [](int64_t a, int64_t b) { return a > INT64_MAX - b ? INT64_MAX : a + b; };
    int64_t best = 0, kept = 0;  // kept: abar^1 .. abar^{j-1}
    for (int32_t j = 1; j <= L; ++j) {
        const int64_t fwd = add(add(add(wa[L - 1], kept), wabar[j - 1]), of[j - 1]);
        kept = add(kept, wabar[j - 1]);
        const int64_t bwd = add(add(wa[j - 1], kept), ob[j - 1]);
        best = fwd > best ? fwd : best;
        best = bwd > best ? bwd : best;
    }
    *peak = best;
    return ROTOR_OK;
}

int32_t rotor_even_budgets(int64_t top, int32_t n, int64_t *budgets)
{
    if (!budgets || top < 0 || n < 1 || n > (1 << 20))
        return ROTOR_EINVAL;
    for (int32_t i = 1; i <= n; ++i)
        budgets[i - 1] = (int64_t)((unsigned __int128)(uint64_t)top * (uint64_t)i / (uint64_t)n);
    return ROTOR_OK;
}

int32_t rotor_sequence_cost(const int64_t *h_params, int32_t L, const rotor_op *h_ops, int64_t n_ops,
                            int64_t *time, int64_t *peak)
{
    if (!h_params || !time || !peak || L < 1 || L > ROTOR_MAX_L || n_ops < 0 || (n_ops > 0 && !h_ops))
        return ROTOR_EINVAL;
    for (int64_t i = 0; i < (int64_t)ROTOR_N_ROWS * L; ++i)
        if (h_params[i] < 0)
            return ROTOR_EDOMAIN;
    for (int64_t i = 0; i < n_ops; ++i)
        if (h_ops[i].kind < ROTOR_F_CK || h_ops[i].kind > ROTOR_B || h_ops[i].stage < 1 || h_ops[i].stage > L)
            return ROTOR_EINVAL;
    auto row = [&](int r, int l) { return h_params[(int64_t)r * L + (l - 1)]; };
    // what is stored, per index l = 0..L; index 0 (a^0, delta^0) is not counted
    std::vector<char> a(L + 1, 0), abar(L + 1, 0), delta(L + 1, 0);
    auto size_a = [&](int l) { return l == 0 ? (int64_t)0 : row(ROTOR_ROW_WA, l); };
    auto size_abar = [&](int l) { return row(ROTOR_ROW_WABAR, l); };
    a[0] = 1;
    delta[L] = 1;
    int64_t mem = size_a(L), t_sum = 0, p_max = 0;
    for (int64_t i = 0; i < n_ops; ++i) {
        const int kind = h_ops[i].kind, l = h_ops[i].stage;
        if (kind == ROTOR_B) {
            if (!delta[l] || !abar[l] || !(a[l - 1] || abar[l - 1]))
                return ROTOR_ESEQUENCE;
            p_max = p_max > mem + row(ROTOR_ROW_OB, l) ? p_max : mem + row(ROTOR_ROW_OB, l);
            t_sum += row(ROTOR_ROW_UB, l);
            delta[l] = 0;
            abar[l] = 0;
            mem -= size_a(l) + size_abar(l);
            if (!abar[l - 1] && a[l - 1]) {  // a plain input is consumed
                a[l - 1] = 0;
                mem -= size_a(l - 1);
            }
            if (delta[l - 1])
                return ROTOR_ESEQUENCE;
            delta[l - 1] = 1;
            mem += size_a(l - 1);
            continue;
        }
        const bool has_input = a[l - 1] || (kind != ROTOR_F_NONE && abar[l - 1]);
        const bool all = kind == ROTOR_F_ALL;
        if (!has_input || (all ? abar[l] : a[l]))
            return ROTOR_ESEQUENCE;
        const int64_t out = all ? size_abar(l) : size_a(l);
        const int64_t here = mem + out + row(ROTOR_ROW_OF, l);
        p_max = p_max > here ? p_max : here;
        t_sum += row(ROTOR_ROW_UF, l);
        if (kind == ROTOR_F_NONE) {
            a[l - 1] = 0;
            mem -= size_a(l - 1);
        }
        (all ? abar[l] : a[l]) = 1;
        mem += out;
    }
    for (int l = 0; l <= L; ++l)
        if (a[l] || abar[l] || delta[l] != (l == 0))
            return ROTOR_ESEQUENCE;
    *time = t_sum;
    *peak = p_max;
    return ROTOR_OK;
}

}  // extern "C"
