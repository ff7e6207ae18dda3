// Weight gradient of a 3D convolution with no workspace argument: the split
// partial sums and bias-gradient slices live in a file-scope device array
// (`scratch`) instead of a caller-provided workspace, so the call allocates
// nothing.  For callers that cannot allocate device memory (code under HIP
// graph capture, serving loops, harnesses that forbid allocation).
//
// Each GPU holds its own copy of `scratch` for the life of the process.  The
// host never passes the array's name to a kernel (on the host it is only a
// stand-in symbol): its device address is looked up once per device with
// hipGetSymbolAddress, with that device current, and that address is what the
// kernels receive.  Every call on a GPU shares that GPU's array; the kernels
// write every partial before reading it, so nothing needs clearing between
// calls, and calls that overlap on one GPU (two streams) race on it.
#include <mutex>

#include "kernels.hpp"

namespace {

constexpr size_t kScratchBytes = (size_t)32 << 20;  // 32 MiB per device
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this GPU's `scratch` (looked up on first use per device).
rat3d_status scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        rat3d::set_error("conv3d_wgrad_noalloc: no usable current device (%d)", dev);
        return RAT3D_EHIP;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            rat3d::set_error("conv3d_wgrad_noalloc: hipGetSymbolAddress failed on device %d: %s",
                             dev, hipGetErrorString(e));
            return RAT3D_EHIP;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RAT3D_OK;
}

}  // namespace

using namespace rat3d;

extern "C" {

size_t rat3d_conv3d_wgrad_noalloc_max_bytes(void) { return kScratchBytes; }

rat3d_status rat3d_conv3d_wgrad_noalloc(const rat3d_conv3d_desc* desc, const void* x,
                                        const void* dy, float* dw, float* dbias, int accumulate,
                                        void* stream) {
    ConvGeom g;
    rat3d_status s = check_conv_desc(desc, &g);
    if (s != RAT3D_OK) return s;
    if ((s = check_act(x, "x")) != RAT3D_OK || (s = check_act(dy, "dy")) != RAT3D_OK) return s;
    if (!dw) {
        set_error("dw must not be NULL");
        return RAT3D_EINVAL;
    }
    const size_t need = conv_ws_bytes(g, desc->dtype, 2);
    if (need > kScratchBytes) {
        set_error("conv3d_wgrad_noalloc: this shape needs %zu bytes of scratch, more than the "
                  "%zu built in; use rat3d_conv3d_wgrad with a workspace",
                  need, kScratchBytes);
        return RAT3D_EWORKSPACE;
    }
    void* ptr = nullptr;
    if ((s = scratch_address(&ptr)) != RAT3D_OK) return s;
    return conv_wgrad(g, desc->dtype, x, dy, dw, dbias, accumulate ? 1 : 0, ptr, kScratchBytes,
                      (hipStream_t)stream);
}

}  // extern "C"
