// Poincare mapping of RGB images into quaternions (Section III-A, eq. 4) for
// gfx950.  Per pixel, with n2 = r^2 + g^2 + b^2:
//
//   q = ((1 - n2), 2r, 2g, 2b) / (1 + n2)
//
// (the RGB point sent onto the unit quaternion sphere).  Input: the three
// colour planes [N][3][H][W]; output: a one-channel quaternion map in the
// library's activation layout, [N][H][W][4] (components r, i, j, k of a
// pixel contiguous), ready to be the first convolution's input.
//
// Each thread maps four consecutive pixels of a plane when the plane size is
// a multiple of four (one 4-element load per colour plane, the 16
// components leaving as contiguous non-temporal 16-byte stores: the map is
// not read back by this pass; measured 10.2 -> 9.2 us on 64x3x224x224 bf16),
// else one pixel.
// HBM-bound: 3 reads + 4 writes of the element per pixel.  Arithmetic in
// fp32 with an IEEE division, rounded once to the output type.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "quan_launch.h"

namespace quan {
namespace {

constexpr int kThreads = 256;

template <typename T>
struct alignas(4 * sizeof(T)) Quad {
    T v[4];
};

template <typename T>
__device__ __forceinline__ Quad<T> map_pixel(float r, float g, float b)
{
    const float n2 = r * r + g * g + b * b;
    const float den = 1.0f + n2;
    Quad<T> q;
    q.v[0] = T((1.0f - n2) / den);
    q.v[1] = T(2.0f * r / den);
    q.v[2] = T(2.0f * g / den);
    q.v[3] = T(2.0f * b / den);
    return q;
}

// Four pixels per thread: hw % 4 == 0, so a group of four never straddles
// two images.
template <typename T>
__global__ __launch_bounds__(kThreads) void poincare_map4(const T *__restrict__ rgb, T *__restrict__ out,
                                                          int64_t hw, int64_t groups)
{
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= groups)
        return;
    const int64_t p = 4 * i;
    const int64_t img = p / hw, t = p - img * hw;
    const T *src = rgb + img * 3 * hw + t;
    const Quad<T> r = *reinterpret_cast<const Quad<T> *>(src);
    const Quad<T> g = *reinterpret_cast<const Quad<T> *>(src + hw);
    const Quad<T> b = *reinterpret_cast<const Quad<T> *>(src + 2 * hw);
    Quad<T> *dst = reinterpret_cast<Quad<T> *>(out) + p;
    Quad<T> q[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
        q[u] = map_pixel<T>(float(r.v[u]), float(g.v[u]), float(b.v[u]));
    typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
    constexpr int N16 = int(sizeof(q)) / 16;
#pragma unroll
    for (int i = 0; i < N16; ++i) {
        u32x4 v;
        __builtin_memcpy(&v, reinterpret_cast<const unsigned char *>(q) + 16 * i, 16);
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(dst) + i);
    }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void poincare_map1(const T *__restrict__ rgb, T *__restrict__ out,
                                                          int64_t hw, int64_t pixels)
{
    const int64_t p = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (p >= pixels)
        return;
    const int64_t img = p / hw, t = p - img * hw;
    const T *src = rgb + img * 3 * hw + t;
    reinterpret_cast<Quad<T> *>(out)[p] = map_pixel<T>(float(src[0]), float(src[hw]), float(src[2 * hw]));
}

template <typename T>
void launch(const void *rgb, void *out, int64_t hw, int64_t pixels, hipStream_t stream)
{
    const T *in = static_cast<const T *>(rgb);
    T *o = static_cast<T *>(out);
    if (hw % 4 == 0 && reinterpret_cast<uintptr_t>(rgb) % (4 * sizeof(T)) == 0) {
        const int64_t groups = pixels / 4;
        hipLaunchKernelGGL(poincare_map4<T>, dim3(unsigned((groups + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                           stream, in, o, hw, groups);
    } else {
        hipLaunchKernelGGL(poincare_map1<T>, dim3(unsigned((pixels + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                           stream, in, o, hw, pixels);
    }
}

}  // namespace

hipError_t poincare_run(const void *rgb, void *out, int64_t n, int64_t h, int64_t w, DType dt,
                        hipStream_t stream)
{
    const int64_t hw = h * w, pixels = n * hw;
    if (dt == DType::BF16)
        launch<__bf16>(rgb, out, hw, pixels, stream);
    else
        launch<float>(rgb, out, hw, pixels, stream);
    return hipGetLastError();
}

}  // namespace quan
