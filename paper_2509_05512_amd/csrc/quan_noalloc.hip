// quan_iqbn_forward_noalloc: the IQBN forward pass for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc).
//
// quan_iqbn_forward keeps its per-block partial statistics and per-column
// affine map in a library workspace that it allocates on first use.  This
// entry point runs the same kernels with that scratch in a fixed array of
// device memory, `scratch`, which every GPU the library runs on holds from
// module load until the process ends.  Host code never passes the array's
// name to a kernel: its device address comes from hipGetSymbolAddress, once
// per device with that device current, and is kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "quan.h"
#include "quan_launch.h"

namespace {

// 8 MiB per device.  Its first 64 KiB hold the grid-barrier flags of the
// one-launch IQBN (zero at module load, used by nothing else); the rest holds
// the partial statistics: (2 * blocks + 3) * 4C floats with at most 512
// blocks for the three-launch form (1.0 MiB for 256 real channels), (2 * G +
// 2) * 4C floats for the one-launch form on G compute units.
constexpr size_t kScratchBytes = size_t(8) << 20;
constexpr size_t kFlagBytes = size_t(64) << 10;
static_assert(kFlagBytes >= 512 * 32 * sizeof(unsigned), "room for the barrier flags");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's scratch array.
int scratch_address(void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return quan::report(QUAN_ERR_HIP, "iqbn_forward_noalloc: hipGetDevice: %s (%d)", hipGetErrorString(e),
                            int(e));
    if (dev < 0 || dev >= kMaxDevices)
        return quan::report(QUAN_ERR_UNSUPPORTED, "iqbn_forward_noalloc: device %d beyond the %d supported", dev,
                            kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return quan::report(QUAN_ERR_HIP, "iqbn_forward_noalloc: hipGetSymbolAddress(scratch): %s (%d)",
                                hipGetErrorString(e), int(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return QUAN_OK;
}

}  // namespace

extern "C" QUAN_API int quan_iqbn_forward_noalloc(const void *x, const float *gamma, const float *beta, float eps,
                                                  void *out, float *mean, float *var, int32_t n, int32_t c,
                                                  int32_t h, int32_t w, int32_t dtype, void *stream)
{
    quan::clear_error();
    if (int rc = quan::iqbn_validate(x, gamma, beta, eps, out, mean, var, n, c, h, w, dtype))
        return rc;
    const int64_t pixels = int64_t(n) * h * w;
    const size_t need = quan::iqbn_workspace_bytes(pixels, c) + kFlagBytes;
    if (need > kScratchBytes)
        return quan::report(QUAN_ERR_UNSUPPORTED,
                            "iqbn_forward_noalloc: needs %zu bytes of scratch, the fixed array holds %zu "
                            "(use quan_iqbn_forward)",
                            need, kScratchBytes);
    void *work = nullptr;
    if (int rc = scratch_address(&work))
        return rc;
    unsigned char *base = static_cast<unsigned char *>(work);
    const hipError_t e = quan::iqbn_run(x, gamma, beta, eps, false, out, mean, var, pixels, c,
                                        dtype == QUAN_BF16 ? quan::DType::BF16 : quan::DType::F32,
                                        base + kFlagBytes, reinterpret_cast<unsigned *>(base),
                                        static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return quan::report(QUAN_ERR_HIP, "iqbn_forward_noalloc launch: %s (%d)", hipGetErrorString(e), int(e));
    return QUAN_OK;
}
