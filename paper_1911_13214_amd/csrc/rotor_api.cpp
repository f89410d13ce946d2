// C ABI entry points of include/rotor.h that enqueue device work: argument
// checks and the launches.  The arithmetic of the method lives in the
// kernels; the host-only entry points are in rotor_host.cpp.
#include <stdint.h>

#include <map>
#include <vector>

#include "rotor_internal.h"

using namespace rotor;

namespace {

bool solve_args_ok(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, const int64_t *d_cost,
                   const int16_t *d_dec, const void *d_work, uint64_t work_bytes)
{
    if (!d_params || !d_cost || !d_dec || !d_work || !sizes_ok(n_chains, L, M) || table_elems(n_chains, L, M) == 0)
        return false;
    if (work_bytes < work_layout(n_chains, L, pitch_of(M)).total)
        return false;
    return !(((uintptr_t)d_params | (uintptr_t)d_cost | (uintptr_t)d_work) % 8 || (uintptr_t)d_dec % 2);
}

Tables make_tables(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost, int16_t *d_dec)
{
    Tables tb;
    tb.params = d_params;
    tb.cost = d_cost;
    tb.dec = d_dec;
    tb.L = L;
    tb.M = (int)M;
    tb.n_chains = n_chains;
    tb.pitch = pitch_of(M);
    tb.rows = (int64_t)L * (L + 1) / 2;
    return tb;
}

// Adds up the work counts of every launch and times each run of consecutive
// launches of one kernel class on one stream with one pair of HIP events on
// that stream (about two runs per block-diagonal and stream), so the events
// add little to what they measure.  Runs on the side stream overlap those on
// the caller's: the class times then add up to more than the solve.
struct TimingObserver : LaunchObserver {
    struct Run {
        hipEvent_t start, stop;
        KernelClass k;
    };
    std::vector<Run> runs;
    std::map<hipStream_t, size_t> open;  // the run of each stream with no stop recorded yet
    rotor_kernel_stats *stats;

    explicit TimingObserver(rotor_kernel_stats *st) : stats(st)
    {
        for (int k = 0; k < ROTOR_N_KERNEL_CLASSES; ++k)
            stats[k] = rotor_kernel_stats{0, 0.0, 0, 0, 0};
    }
    hipError_t close(hipStream_t s)
    {
        auto it = open.find(s);
        if (it == open.end())
            return hipSuccess;
        const size_t i = it->second;
        open.erase(it);
        return hipEventRecord(runs[i].stop, s);
    }
    hipError_t end_stream(hipStream_t s) override { return close(s); }
    hipError_t before(KernelClass k, hipStream_t s) override
    {
        auto it = open.find(s);
        if (it != open.end() && runs[it->second].k == k)
            return hipSuccess;
        hipError_t e = close(s);
        Run r{nullptr, nullptr, k};
        if (e == hipSuccess)
            e = hipEventCreate(&r.start);
        if (e == hipSuccess)
            e = hipEventCreate(&r.stop);
        if (e == hipSuccess)
            e = hipEventRecord(r.start, s);
        runs.push_back(r);
        if (e == hipSuccess)
            open[s] = runs.size() - 1;
        return e;
    }
    hipError_t after(KernelClass k, const LaunchWork &w, hipStream_t) override
    {
        rotor_kernel_stats &st = stats[k];
        st.launches += 1;
        st.split_candidates += w.split_candidates;
        st.all_candidates += w.all_candidates;
        st.cells += w.cells;
        return hipSuccess;
    }
    hipError_t finish(hipStream_t s)
    {
        // runs still open (a launch failed before its stream joined) close
        // on their own streams, which are then waited for too
        std::vector<hipStream_t> others;
        for (const auto &o : open)
            if (o.first != s)
                others.push_back(o.first);
        hipError_t e = hipSuccess;
        for (hipStream_t o : others)
            if (e == hipSuccess)
                e = close(o);
        if (e == hipSuccess)
            e = close(s);
        if (e == hipSuccess)
            e = hipStreamSynchronize(s);
        for (hipStream_t o : others)
            if (e == hipSuccess)
                e = hipStreamSynchronize(o);
        for (Run &r : runs) {
            float ms = 0.f;
            if (e == hipSuccess && r.start && r.stop)
                e = hipEventElapsedTime(&ms, r.start, r.stop);
            stats[r.k].ms += ms;
        }
        return e;
    }
    ~TimingObserver() override
    {
        for (Run &r : runs) {
            if (r.start)
                (void)hipEventDestroy(r.start);
            if (r.stop)
                (void)hipEventDestroy(r.stop);
        }
    }
};

}  // namespace

extern "C" {

int32_t rotor_solve(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost,
                    int16_t *d_dec, void *d_work, uint64_t work_bytes, void *stream)
{
    if (!solve_args_ok(d_params, n_chains, L, M, d_cost, d_dec, d_work, work_bytes))
        return ROTOR_EINVAL;
    const Tables tb = make_tables(d_params, n_chains, L, M, d_cost, d_dec);
    const Work w = work_view(d_work, n_chains, L, tb.pitch);
    return launch_fill(tb, w, ROTOR_SCHEDULE_AUTO, (hipStream_t)stream) == hipSuccess ? ROTOR_OK : ROTOR_EDEVICE;
}

int32_t rotor_solve_schedule(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost,
                             int16_t *d_dec, void *d_work, uint64_t work_bytes, void *stream, int32_t schedule)
{
    if (schedule < ROTOR_SCHEDULE_AUTO || schedule > ROTOR_SCHEDULE_BLOCKED_SERIAL ||
        !solve_args_ok(d_params, n_chains, L, M, d_cost, d_dec, d_work, work_bytes))
        return ROTOR_EINVAL;
    const Tables tb = make_tables(d_params, n_chains, L, M, d_cost, d_dec);
    const Work w = work_view(d_work, n_chains, L, tb.pitch);
    return launch_fill(tb, w, schedule, (hipStream_t)stream) == hipSuccess ? ROTOR_OK : ROTOR_EDEVICE;
}

int32_t rotor_solve_timed(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, int64_t *d_cost,
                          int16_t *d_dec, void *d_work, uint64_t work_bytes, void *stream,
                          rotor_kernel_stats *stats)
{
    if (!stats || !solve_args_ok(d_params, n_chains, L, M, d_cost, d_dec, d_work, work_bytes))
        return ROTOR_EINVAL;
    const Tables tb = make_tables(d_params, n_chains, L, M, d_cost, d_dec);
    const Work w = work_view(d_work, n_chains, L, tb.pitch);
    TimingObserver obs(stats);
    hipError_t e = launch_fill(tb, w, ROTOR_SCHEDULE_AUTO, (hipStream_t)stream, &obs);
    const hipError_t f = obs.finish((hipStream_t)stream);
    return (e == hipSuccess && f == hipSuccess) ? ROTOR_OK : ROTOR_EDEVICE;
}

int32_t rotor_solve_status(const void *d_work, uint64_t work_bytes, int32_t n_chains, int32_t L, int64_t M,
                           int32_t *h_chain_status, void *stream)
{
    if (!d_work || (uintptr_t)d_work % 8 || !sizes_ok(n_chains, L, M) || table_elems(n_chains, L, M) == 0)
        return ROTOR_EINVAL;
    const WorkLayout wl = work_layout(n_chains, L, pitch_of(M));
    if (work_bytes < wl.total)
        return ROTOR_EINVAL;
    std::vector<int32_t> st(h_chain_status ? 0 : (size_t)n_chains);
    int32_t *dst = h_chain_status ? h_chain_status : st.data();
    const hipStream_t s = (hipStream_t)stream;
    if (hipMemcpyAsync(dst, (const char *)d_work + wl.status, sizeof(int32_t) * (size_t)n_chains,
                       hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return ROTOR_EDEVICE;
    int32_t worst = ROTOR_OK;
    for (int32_t c = 0; c < n_chains; ++c) {
        if (dst[c] != ROTOR_OK && dst[c] != ROTOR_EDOMAIN)
            return ROTOR_EINVAL;  // not a workspace a solve has written
        if (dst[c] == ROTOR_EDOMAIN)
            worst = ROTOR_EDOMAIN;
    }
    return worst;
}

int32_t rotor_reconstruct(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M, const int16_t *d_dec,
                          int32_t chain, int32_t n_budgets, const int64_t *d_budgets, int64_t cap, rotor_op *d_ops,
                          int64_t *d_count, int32_t *d_status, void *stream)
{
    if (!d_params || !d_dec || !d_budgets || !d_count || !d_status || !sizes_ok(n_chains, L, M))
        return ROTOR_EINVAL;
    if (L > ROTOR_MAX_L_RECONSTRUCT || chain < 0 || chain >= n_chains || n_budgets < 1 || cap < 0)
        return ROTOR_EINVAL;
    if (cap > 0 && !d_ops)
        return ROTOR_EINVAL;
    if (table_elems(n_chains, L, M) == 0)
        return ROTOR_EINVAL;
    const int64_t pitch = pitch_of(M);
    const int64_t rows = (int64_t)L * (L + 1) / 2;
    return launch_reconstruct(d_params + (int64_t)chain * ROTOR_N_ROWS * L, L, (int)M, pitch, rows,
                              d_dec + (int64_t)chain * rows * pitch, n_budgets, d_budgets, cap, d_ops, d_count,
                              d_status, (hipStream_t)stream) == hipSuccess
               ? ROTOR_OK
               : ROTOR_EDEVICE;
}

}  // extern "C"
