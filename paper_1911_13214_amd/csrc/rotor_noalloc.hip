// rotor_solve for callers that cannot allocate device memory: the fill's
// workspace is a static device array of fixed size instead of a caller
// buffer.  The kernels are the same as rotor_solve's; they take the array's
// device address as their workspace argument.
#include <mutex>

#include "rotor_internal.h"

namespace rotor {
namespace {

// The workspace of every call on a device.  Each device the library runs on
// holds its own copy of this array until the process ends.
__device__ __align__(256) unsigned char scratch[ROTOR_NOALLOC_WORK_BYTES];

// Device address of `scratch` per device, looked up once per device with
// that device current (the array's name is a host-side stand-in in host
// code, not a device address).
constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void *g_scratch[kMaxDevices];
hipError_t g_lookup[kMaxDevices];

hipError_t scratch_address(int dev, void **ptr)
{
    std::call_once(g_once[dev], [dev] {
        void *p = nullptr;
        g_lookup[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch[dev] = g_lookup[dev] == hipSuccess ? p : nullptr;
    });
    *ptr = g_scratch[dev];
    return g_lookup[dev] == hipSuccess && *ptr ? hipSuccess : hipErrorInvalidSymbol;
}

}  // namespace
}  // namespace rotor

using namespace rotor;

extern "C" int32_t rotor_solve_noalloc(const int64_t *d_params, int32_t n_chains, int32_t L, int64_t M,
                                       int64_t *d_cost, int16_t *d_dec, void *stream)
{
    if (!d_params || !d_cost || !d_dec || !sizes_ok(n_chains, L, M) || table_elems(n_chains, L, M) == 0)
        return ROTOR_EINVAL;
    if (((uintptr_t)d_params | (uintptr_t)d_cost) % 8 || (uintptr_t)d_dec % 2)
        return ROTOR_EINVAL;
    const uint64_t need = work_layout(n_chains, L, pitch_of(M)).total;
    if (need > (uint64_t)ROTOR_NOALLOC_WORK_BYTES)
        return ROTOR_ECAPACITY;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return ROTOR_EDEVICE;
    void *work = nullptr;
    if (scratch_address(dev, &work) != hipSuccess)
        return ROTOR_EDEVICE;
    Tables tb;
    tb.params = d_params;
    tb.cost = d_cost;
    tb.dec = d_dec;
    tb.L = L;
    tb.M = (int)M;
    tb.n_chains = n_chains;
    tb.pitch = pitch_of(M);
    tb.rows = (int64_t)L * (L + 1) / 2;
    // the fill overwrites every workspace word it reads before reading it,
    // so nothing left by an earlier call needs clearing
    const Work w = work_view(work, n_chains, L, tb.pitch);
    // no side stream: creating one on the first call would allocate
    return launch_fill(tb, w, ROTOR_SCHEDULE_AUTO, (hipStream_t)stream, nullptr, false) == hipSuccess ? ROTOR_OK
                                                                                                      : ROTOR_EDEVICE;
}
