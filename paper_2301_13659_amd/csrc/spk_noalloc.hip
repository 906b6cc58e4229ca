// spk_conv_fire_noalloc: spk_conv_fire for callers that cannot allocate
// device memory (code under stream capture, tight serving loops).  The
// scratch that spk_conv_fire takes from a caller workspace (the padded
// channels-last input copy, the packed weight fragments, readout partial
// sums) comes instead from a static device array the library owns, one copy
// per GPU, held until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory: the
// device address of each GPU's copy is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// handed to kernels.
#include <mutex>

#include "spk_internal.h"

namespace {

constexpr size_t kScratchBytes = SPK_CONV_FIRE_NOALLOC_MAX_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`.
spk_status scratch_for_current_device(void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    SPK_REQUIRE(e == hipSuccess, SPK_E_HIP, "spk_conv_fire_noalloc: hipGetDevice: %s",
                hipGetErrorString(e));
    SPK_REQUIRE(dev >= 0 && dev < kMaxDevices, SPK_E_UNSUPPORTED,
                "spk_conv_fire_noalloc: device %d beyond the %d supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        SPK_REQUIRE(e == hipSuccess && p, SPK_E_HIP,
                    "spk_conv_fire_noalloc: hipGetSymbolAddress of the scratch array: %s",
                    hipGetErrorString(e));
        SPK_REQUIRE(((uintptr_t)p & 255u) == 0u, SPK_E_HIP,
                    "spk_conv_fire_noalloc: scratch array not 256-byte aligned");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return SPK_OK;
}

}  // namespace

extern "C" spk_status spk_conv_fire_noalloc(const uint8_t *in_times, int B, int T, int Ci, int Hi,
                                            int Wi, const void *w, spk_dtype w_dtype, int Co, int Kh,
                                            int Kw, int stride, int pad, float theta,
                                            uint8_t *out_times, float *out_vkey, float *potentials,
                                            spk_stream stream)
{
    spk::clear_error();
    // the size check needs only the shapes: a call that cannot fit launches
    // nothing and touches no device state
    const size_t need = spk_conv_fire_workspace_size(B, T, Ci, Hi, Wi, Co, Kh, Kw, stride, pad, theta,
                                                     potentials != nullptr);
    SPK_REQUIRE(need <= kScratchBytes, SPK_E_WORKSPACE,
                "spk_conv_fire_noalloc: this layer needs %zu bytes of scratch, more than the static "
                "%zu; use spk_conv_fire with a workspace",
                need, kScratchBytes);
    void *ws = nullptr;
    if (need > 0) {
        const spk_status st = scratch_for_current_device(&ws);
        if (st != SPK_OK) return st;
    }
    return spk_conv_fire(in_times, B, T, Ci, Hi, Wi, w, w_dtype, Co, Kh, Kw, stride, pad, theta,
                         out_times, out_vkey, potentials, ws, need, stream);
}
