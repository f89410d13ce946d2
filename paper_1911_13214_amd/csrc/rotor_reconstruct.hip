// Algorithm 2 (OptRec) of Beaumont et al. (arXiv 1911.13214): rebuild the
// optimal persistent sequence of the whole chain from the decision table.
//
// The recursion is unrolled into a walk with an explicit stack kept in LDS:
// one workgroup per requested budget, its first lane walks.  Pending items
// always cover disjoint stage ranges (a split leaves [s, s'-1] pending while
// [s', t] is walked; F_all^s leaves B^s pending while [s+1, t] is walked), so
// the stack never holds more than L frames.
#include "rotor_internal.h"

namespace rotor {
namespace {

// A stack frame: bit 63 set = emit B^s; otherwise solve [s, t] at budget m.
// m < 2^30 in the domain, s and t < 2^15.
__device__ inline uint64_t frame_solve(int s, int t, int64_t m)
{
    return ((uint64_t)s << 47) | ((uint64_t)t << 32) | (uint64_t)(uint32_t)m;
}
__device__ inline uint64_t frame_backward(int s) { return (1ull << 63) | ((uint64_t)s << 47); }

__global__ void walk_kernel(const int64_t *__restrict__ params, int L, int M, int64_t pitch,
                            const int16_t *__restrict__ dec, const int64_t *__restrict__ budgets, int64_t cap,
                            rotor_op *__restrict__ ops, int64_t *__restrict__ count, int32_t *__restrict__ status)
{
    extern __shared__ uint64_t stack[];
    // the whole wave checks the chain's parameters; a table filled from
    // parameters outside the domain is unspecified and is not walked
    const bool in_domain = chain_in_domain(params, L, threadIdx.x);
    if (threadIdx.x != 0)
        return;
    const int b = blockIdx.x;
    if (!in_domain) {
        count[b] = 0;
        status[b] = ROTOR_EDOMAIN;
        return;
    }
    const int64_t *wa = params + (int64_t)ROTOR_ROW_WA * L;
    const int64_t *wabar = params + (int64_t)ROTOR_ROW_WABAR * L;
    rotor_op *out = ops + (int64_t)b * cap;
    const int64_t m0 = budgets[b];
    if (m0 < 0 || m0 > M) {
        count[b] = 0;
        status[b] = ROTOR_EINVAL;
        return;
    }
    int64_t n = 0;
    auto emit = [&](int kind, int stage) {
        if (n < cap)
            out[n] = rotor_op{kind, stage};
        ++n;
    };
    int top = 0;
    stack[top++] = frame_solve(1, L, m0);
    int32_t st = ROTOR_OK;
    bool root = true;
    while (top > 0) {
        const uint64_t f = stack[--top];
        const int s = (int)((f >> 47) & 0x7fff);
        if (f >> 63) {
            emit(ROTOR_B, s);
            continue;
        }
        const int t = (int)((f >> 32) & 0x7fff);
        const int64_t m = (int64_t)(uint32_t)f;
        const int dv = dec[row_of(L, s, t) * pitch + m];
        if (dv < 0) {
            st = root ? ROTOR_INFEASIBLE : ROTOR_ECORRUPT;
            break;
        }
        root = false;
        if (s == t) {
            emit(ROTOR_F_ALL, s);
            emit(ROTOR_B, s);
        } else if (dv > 0) {
            // F_ck^s, F_none^{s+1..s'-1}, then [s', t] with a^{s'-1} stored,
            // then [s, s'-1].
            const int sp = dv;
            if (sp <= s || sp > t) {
                st = ROTOR_ECORRUPT;
                break;
            }
            // a budget outside [0, M] (a negative size: parameters outside
            // the domain) is never read
            const int64_t mr = m - wa[sp - 2];
            if (mr < 0 || mr > M || top + 2 > L + 1) {
                st = ROTOR_ECORRUPT;
                break;
            }
            emit(ROTOR_F_CK, s);
            for (int k = s + 1; k < sp; ++k)
                emit(ROTOR_F_NONE, k);
            stack[top++] = frame_solve(s, sp - 1, m);
            stack[top++] = frame_solve(sp, t, mr);
        } else {
            // F_all^s, then [s+1, t] with abar^s stored, then B^s.
            const int64_t mr = m - wabar[s - 1];
            if (mr < 0 || mr > M || top + 2 > L + 1) {
                st = ROTOR_ECORRUPT;
                break;
            }
            emit(ROTOR_F_ALL, s);
            stack[top++] = frame_backward(s);
            stack[top++] = frame_solve(s + 1, t, mr);
        }
    }
    if (st == ROTOR_OK && n > cap)
        st = ROTOR_ECAPACITY;
    count[b] = (st == ROTOR_OK || st == ROTOR_ECAPACITY) ? n : 0;
    status[b] = st;
}

}  // namespace

hipError_t launch_reconstruct(const int64_t *params, int L, int M, int64_t pitch, int64_t rows,
                              const int16_t *dec_chain, int n_budgets, const int64_t *budgets, int64_t cap,
                              rotor_op *ops, int64_t *count, int32_t *status, hipStream_t stream)
{
    (void)rows;
    (void)hipGetLastError();  // an error the caller's earlier calls left behind is not this launch's
    const size_t lds = sizeof(uint64_t) * (size_t)(L + 1);
    walk_kernel<<<dim3(n_budgets), 64, lds, stream>>>(params, L, M, pitch, dec_chain, budgets, cap, ops, count,
                                                      status);
    return hipGetLastError();
}

}  // namespace rotor
