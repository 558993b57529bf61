// The on-site entry point that allocates nothing: its workspace is a fixed array in device
// memory, one copy per GPU the library runs on, held until the process ends.
#include <mutex>

#include "internal.h"

namespace {

constexpr int kMaxDevices = 64;

// The scratch array. In host code its name is only a host-side stand-in: every host use goes
// through the device address resolved by noalloc_setup.
static __device__ __align__(256) unsigned char scratch[CGTP_NOALLOC_SCRATCH_BYTES];

std::mutex g_mu;
void *g_ptr[kMaxDevices];
hipError_t g_status[kMaxDevices];
bool g_done[kMaxDevices];

}  // namespace

namespace cgtp {

hipError_t noalloc_setup(int dev)
{
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_done[dev]) {
        void *p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_status[dev] = e;
        g_ptr[dev] = e == hipSuccess ? p : nullptr;
        g_done[dev] = true;
    }
    return g_status[dev];
}

}  // namespace cgtp

extern "C" int cgtp_onsite_noalloc(cgtp_plan plan, int64_t n_nodes, const void *A, const void *B,
                                   const void *U_A, const void *U_B, const void *U_out_even,
                                   const void *U_out_odd, void *out_even, void *out_odd,
                                   void *stream)
{
    cgtp::clear_error();
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return cgtp::report(CGTP_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return cgtp::report(CGTP_ERR_UNSUPPORTED, "device %d beyond the %d with a fixed scratch",
                            dev, kMaxDevices);
    // set up by cgtp_plan_create on the plan's device; resolved here on any other device
    // (the call then fails on the device check)
    e = cgtp::noalloc_setup(dev);
    if (e != hipSuccess)
        return cgtp::report(CGTP_ERR_HIP, "hipGetSymbolAddress(scratch): %s",
                            hipGetErrorString(e));
    void *ptr;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        ptr = g_ptr[dev];
    }
    return cgtp::onsite_fixed_scratch(plan, n_nodes, A, B, U_A, U_B, U_out_even, U_out_odd,
                                      out_even, out_odd, ptr, CGTP_NOALLOC_SCRATCH_BYTES, stream);
}
