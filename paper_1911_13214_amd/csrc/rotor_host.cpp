// Host-only entry points of include/rotor.h: version, status text, table
// geometry, the workspace layout and the check of host parameters against
// the domain.  No device code and no HIP header: this file also builds with a
// plain C++ compiler (the sanitizer build of the CPU tests).
#include <stdint.h>

#include "rotor_geometry.h"

namespace rotor {

uint64_t table_elems(int32_t n_chains, int32_t L, int64_t M)
{
    const unsigned __int128 e = (unsigned __int128)(uint64_t)n_chains * (uint64_t)((int64_t)L * (L + 1) / 2) *
                                (uint64_t)pitch_of(M);
    if (e * 8 >= ((unsigned __int128)1 << 63))
        return 0;
    return (uint64_t)e;
}

WorkLayout work_layout(int n_chains, int L, int64_t pitch)
{
    auto align = [](uint64_t x) { return (x + 255) / 256 * 256; };
    const uint64_t rows = (uint64_t)L * (L + 1) / 2;
    const uint64_t nc = (uint64_t)n_chains;
    const uint64_t nb = (uint64_t)((L + kBlock - 1) / kBlock);
    WorkLayout wl;
    wl.pre = 0;
    wl.preall = align(wl.pre + 8ull * nc * (uint64_t)(L + 1));
    wl.pbits = align(wl.preall + 8ull * nc * (uint64_t)(L + 1));
    wl.bsum = align(wl.pbits + 4ull * nc * nb);
    wl.gnone = align(wl.bsum + 16ull * nc * (nb + 1));
    wl.gall = align(wl.gnone + 4ull * nc * rows);
    wl.gsat = align(wl.gall + 4ull * nc * rows);
    wl.gblk = align(wl.gsat + 4ull * nc * rows);
    wl.status = align(wl.gblk + 8ull * nc * nb * nb);
    wl.shift = align(wl.status + 4ull * nc);
    wl.shadow = align(wl.shift + 8ull * nc * (uint64_t)L);
    wl.half = align(wl.shadow + 4ull * nc * rows * (uint64_t)pitch);
    const uint64_t half_rows = nb >= 2 ? (uint64_t)L * kBlock : 0;  // no edges in a single block
    wl.total = align(wl.half + 2ull * nc * half_rows * (uint64_t)half_pitch_of(pitch));
    return wl;
}

}  // namespace rotor

using namespace rotor;

extern "C" {

int32_t rotor_version(void) { return ROTOR_VERSION; }

const char *rotor_status_string(int32_t status)
{
    switch (status) {
    case ROTOR_OK: return "ok";
    case ROTOR_EINVAL: return "invalid argument";
    case ROTOR_EDOMAIN: return "chain parameter outside the supported domain";
    case ROTOR_EDEVICE: return "HIP runtime error";
    case ROTOR_INFEASIBLE: return "no sequence fits the memory budget";
    case ROTOR_ECAPACITY: return "output array too small";
    case ROTOR_ECORRUPT: return "decision table inconsistent";
    case ROTOR_ESEQUENCE: return "operation sequence not valid";
    default: return "unknown status";
    }
}

int32_t rotor_layout(int32_t n_chains, int32_t L, int64_t M, int64_t *pitch, int64_t *rows_per_chain,
                     uint64_t *cost_bytes, uint64_t *dec_bytes)
{
    if (!sizes_ok(n_chains, L, M))
        return ROTOR_EINVAL;
    const uint64_t e = table_elems(n_chains, L, M);
    if (e == 0)
        return ROTOR_EINVAL;
    if (pitch)
        *pitch = pitch_of(M);
    if (rows_per_chain)
        *rows_per_chain = (int64_t)L * (L + 1) / 2;
    if (cost_bytes)
        *cost_bytes = e * sizeof(int64_t);
    if (dec_bytes)
        *dec_bytes = e * sizeof(int16_t);
    return ROTOR_OK;
}

int64_t rotor_row_index(int32_t L, int32_t s, int32_t t)
{
    if (L < 1 || L > ROTOR_MAX_L || s < 1 || t < s || t > L)
        return -1;
    return row_of(L, s, t);
}

int32_t rotor_check_params(const int64_t *h_params, int32_t n_chains, int32_t L, int64_t M)
{
    if (!h_params || !sizes_ok(n_chains, L, M))
        return ROTOR_EINVAL;
    for (int32_t c = 0; c < n_chains; ++c) {
        const int64_t *p = h_params + (int64_t)c * ROTOR_N_ROWS * L;
        uint64_t suf = 0, sub = 0;
        for (int32_t l = 0; l < L; ++l) {
            const int64_t uf = p[ROTOR_ROW_UF * L + l], ub = p[ROTOR_ROW_UB * L + l];
            if (uf < 0 || ub < 0 || (uint64_t)uf >= kCostBound || (uint64_t)ub >= kCostBound)
                return ROTOR_EDOMAIN;
            for (int row = ROTOR_ROW_WA; row <= ROTOR_ROW_OB; ++row) {
                const int64_t v = p[row * L + l];
                if (v < 0 || v >= kMaxSize)
                    return ROTOR_EDOMAIN;
            }
            suf += (uint64_t)uf;
            sub += (uint64_t)ub;
            if (suf >= kCostBound || sub >= kCostBound)
                return ROTOR_EDOMAIN;
        }
        // L * suf + sub < 2^44
        if (suf > (kCostBound - sub) / (uint64_t)L)
            return ROTOR_EDOMAIN;
    }
    return ROTOR_OK;
}

int32_t rotor_workspace_bytes(int32_t n_chains, int32_t L, int64_t M, uint64_t *bytes)
{
    if (!sizes_ok(n_chains, L, M) || table_elems(n_chains, L, M) == 0)
        return ROTOR_EINVAL;
    if (bytes)
        *bytes = work_layout(n_chains, L, pitch_of(M)).total;
    return ROTOR_OK;
}

}  // extern "C"
