// C ABI of libquan: argument validation, workspace management and dispatch.
//
// Every entry point validates all of its arguments on the host before the
// first HIP call, so a rejected call never touches the device.  Kernels run
// asynchronously on the caller's stream.
#include <hip/hip_runtime_api.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>

#include "quan.h"
#include "quan_launch.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int fail_hip(hipError_t e, const char *what)
{
    return fail(QUAN_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), int(e));
}

// Library-owned device memory, one buffer per (device, stream, purpose), so
// that calls on different streams never race on a shared scratch buffer.
struct Workspace {
    void *ptr = nullptr;
    size_t bytes = 0;
    unsigned uses = 0;  // calls that took it (the claim buffer's launch tags)
};

std::mutex g_ws_mutex;
std::map<std::pair<int, std::pair<void *, int>>, Workspace> g_ws;

enum Purpose {
    kWeightPack = 0,
    kIqbnPartials = 1,
    kIqbnFold = 2,
    kGradPack = 3,
    kGradStage = 4,
    kWgrad = 5,
    kIqbnBarrier = 6,  // the one-launch IQBN's grid-barrier flags: zeroed once, when allocated
    kConvClaim = 7     // the convolution's tail-block claims: zeroed once, when allocated
};

// Returns a device buffer of at least `bytes` for (current device, stream,
// purpose).  Growing it first waits for the device to finish with the old one.
int workspace(void *stream, Purpose purpose, size_t bytes, void **out, unsigned *uses = nullptr)
{
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return fail_hip(e, "hipGetDevice");
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    Workspace &ws = g_ws[{dev, {stream, int(purpose)}}];
    if (ws.bytes < bytes) {
        if (ws.ptr) {
            e = hipDeviceSynchronize();
            if (e != hipSuccess)
                return fail_hip(e, "hipDeviceSynchronize");
            e = hipFree(ws.ptr);
            ws.ptr = nullptr;
            ws.bytes = 0;
            if (e != hipSuccess)
                return fail_hip(e, "hipFree");
        }
        size_t want = bytes + bytes / 4;  // headroom for slightly larger calls
        want = (want + 4095) & ~size_t(4095);
        e = hipMalloc(&ws.ptr, want);
        if (e != hipSuccess) {
            ws.ptr = nullptr;
            return fail(QUAN_ERR_NOMEM, "hipMalloc(%zu) for workspace: %s", want, hipGetErrorString(e));
        }
        ws.bytes = want;
        if (purpose == kIqbnBarrier || purpose == kConvClaim) {
            e = hipMemsetAsync(ws.ptr, 0, want, static_cast<hipStream_t>(stream));
            if (e != hipSuccess)
                return fail_hip(e, "hipMemsetAsync (barrier flags, claim counter)");
        }
    }
    *out = ws.ptr;
    if (uses != nullptr)
        *uses = ws.uses++;
    return QUAN_OK;
}

// The grid-barrier flags of the one-launch IQBN on this (device, stream).
int iqbn_flags(void *stream, unsigned **out)
{
    void *p = nullptr;
    if (int rc = workspace(stream, kIqbnBarrier, quan::iqbn_barrier_bytes(), &p))
        return rc;
    *out = static_cast<unsigned *>(p);
    return QUAN_OK;
}

// The claim counter and mailboxes of the convolution's tail blocks on this
// (device, stream): every launch leaves the counter zero.
int conv_claim(void *stream, quan::ConvClaim *out)
{
    void *p = nullptr;
    unsigned uses = 0;
    if (int rc = workspace(stream, kConvClaim, quan::qconv2d_claim_bytes(), &p, &uses))
        return rc;
    out->buf = static_cast<unsigned *>(p);
    // each call's launches (up to 16 output phases of an input gradient)
    // take tags from a range of their own
    out->epoch = uses * 17u;
    return QUAN_OK;
}

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

bool misaligned(const void *p, size_t a)
{
    return (reinterpret_cast<uintptr_t>(p) % a) != 0;
}

bool overlaps(const void *a, size_t abytes, const void *b, size_t bbytes)
{
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(a), b0 = reinterpret_cast<uintptr_t>(b);
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

size_t elem_size(int32_t dtype)
{
    return dtype == QUAN_BF16 ? 2 : 4;
}

int check_dtype(int32_t dtype)
{
    if (dtype != QUAN_F32 && dtype != QUAN_BF16)
        return fail(QUAN_ERR_DTYPE, "dtype %d is neither QUAN_F32 (0) nor QUAN_BF16 (1)", dtype);
    return QUAN_OK;
}

quan::DType to_dt(int32_t dtype)
{
    return dtype == QUAN_BF16 ? quan::DType::BF16 : quan::DType::F32;
}

// Validation shared by the two convolution entry points (everything except
// the weights): sizes, output extent, limits, alignment of x/out/bias and
// overlap of out with x and the bias.  Fills the geometry on success.
// rgb_planes: x is the colour planes [n][3][h][w] of a Poincare stem (c_in
// 1), aligned to its element and sized as such.
int check_conv(const void *x, const void *bias, int32_t stride_h, int32_t stride_w, int32_t pad_h,
               int32_t pad_w, int32_t dilation_h, int32_t dilation_w, const void *out, int32_t n,
               int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
               int32_t dtype, quan::ConvGeom *g, size_t *xb, size_t *ob, bool rgb_planes = false)
{
    if (int rc = check_dtype(dtype))
        return rc;
    if (n < 1 || c_in < 1 || h < 1 || w < 1 || c_out < 1 || k_h < 1 || k_w < 1)
        return fail(QUAN_ERR_SHAPE,
                    "qconv2d: sizes must be >= 1 (n=%d c_in=%d h=%d w=%d c_out=%d k=%dx%d)", n, c_in,
                    h, w, c_out, k_h, k_w);
    if (stride_h < 1 || stride_w < 1 || dilation_h < 1 || dilation_w < 1 || pad_h < 0 || pad_w < 0)
        return fail(QUAN_ERR_SHAPE, "qconv2d: stride/dilation must be >= 1 and pad >= 0");
    const int64_t span_h = int64_t(h) + 2 * int64_t(pad_h) - int64_t(dilation_h) * (k_h - 1) - 1;
    const int64_t span_w = int64_t(w) + 2 * int64_t(pad_w) - int64_t(dilation_w) * (k_w - 1) - 1;
    if (span_h < 0 || span_w < 0)
        return fail(QUAN_ERR_SHAPE, "qconv2d: empty output (kernel span exceeds padded input)");
    const int64_t ho = span_h / stride_h + 1, wo = span_w / stride_w + 1;
    const int64_t x_elems = int64_t(n) * h * w * (rgb_planes ? 3 : 4 * c_in);
    const int64_t o_elems = int64_t(n) * ho * wo * 4 * c_out;
    const int64_t w_elems = int64_t(c_out) * c_in * k_h * k_w;
    if (x_elems > kMaxElems || o_elems > kMaxElems || w_elems * 4 * 4 > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "qconv2d: a tensor exceeds 2^31-1 elements");
    const size_t es = elem_size(dtype);
    // A work-group addresses its activations with 32-bit byte offsets from
    // the first image of its tile (at most 256 output pixels, so at most
    // 256 / (ho * wo) + 2 images).
    const int64_t img_bytes = int64_t(h) * w * 4 * c_in * int64_t(es);
    if (img_bytes * (256 / (ho * wo) + 2) > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "qconv2d: images of x too large for 32-bit tile offsets");
    if (misaligned(x, rgb_planes ? es : 16) || misaligned(out, 16))
        return fail(QUAN_ERR_ALIGN, rgb_planes ? "qconv2d: rgb must be aligned to its element, out to 16 bytes"
                                               : "qconv2d: x and out must be 16-byte aligned");
    if (bias && misaligned(bias, es))
        return fail(QUAN_ERR_ALIGN, "qconv2d: weights and bias must be aligned to their element size");
    *xb = size_t(x_elems) * es;
    *ob = size_t(o_elems) * es;
    if (overlaps(out, *ob, x, *xb) || (bias && overlaps(out, *ob, bias, size_t(4) * c_out * es)))
        return fail(QUAN_ERR_ALIAS, "qconv2d: out overlaps x, a kernel or the bias");
    g->n = n;
    g->c_in = c_in;
    g->h = h;
    g->w = w;
    g->c_out = c_out;
    g->k_h = k_h;
    g->k_w = k_w;
    g->s_h = stride_h;
    g->s_w = stride_w;
    g->p_h = pad_h;
    g->p_w = pad_w;
    g->d_h = dilation_h;
    g->d_w = dilation_w;
    g->h_out = int(ho);
    g->w_out = int(wo);
    return QUAN_OK;
}

}  // namespace

namespace quan {

void clear_error()
{
    g_last_error.clear();
}

int report(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int iqbn_validate(const void *x, const float *gamma, const float *beta, float eps, const void *out,
                  const float *mean, const float *var, int32_t n, int32_t c, int32_t h, int32_t w, int32_t dtype)
{
    if (!x || !gamma || !beta || !out || !mean || !var)
        return fail(QUAN_ERR_NULL, "iqbn: x, gamma, beta, out, mean and var must be non-NULL");
    if (int rc = check_dtype(dtype))
        return rc;
    if (n < 1 || c < 1 || h < 1 || w < 1)
        return fail(QUAN_ERR_SHAPE, "iqbn: sizes must be >= 1 (n=%d c=%d h=%d w=%d)", n, c, h, w);
    if (!(eps > 0.0f) || eps != eps)
        return fail(QUAN_ERR_SHAPE, "iqbn: eps must be > 0 (got %g)", double(eps));
    const int64_t pixels = int64_t(n) * h * w;
    const int64_t elems = pixels * 4 * c;
    if (elems > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "iqbn: tensor of %lld elements exceeds 2^31-1",
                    (long long)elems);
    const size_t es = elem_size(dtype);
    if (misaligned(x, 16) || misaligned(out, 16))
        return fail(QUAN_ERR_ALIGN, "iqbn: x and out must be 16-byte aligned");
    if (misaligned(gamma, 4) || misaligned(beta, 4) || misaligned(mean, 4) || misaligned(var, 4))
        return fail(QUAN_ERR_ALIGN, "iqbn: gamma, beta, mean and var must be 4-byte aligned");
    const size_t xbytes = size_t(elems) * es, sbytes = size_t(4) * c * sizeof(float);
    if (out != x && overlaps(out, xbytes, x, xbytes))
        return fail(QUAN_ERR_ALIAS, "iqbn: out partially overlaps x (only out == x is allowed)");
    if (overlaps(mean, sbytes, var, sbytes) || overlaps(mean, sbytes, x, xbytes) ||
        overlaps(var, sbytes, x, xbytes) || overlaps(mean, sbytes, out, xbytes) ||
        overlaps(var, sbytes, out, xbytes))
        return fail(QUAN_ERR_ALIAS, "iqbn: mean/var overlap each other or a tensor");
    return QUAN_OK;
}

}  // namespace quan

namespace {

int iqbn_common(const void *x, const float *gamma, const float *beta, float eps, void *out,
                float *mean, float *var, int32_t n, int32_t c, int32_t h, int32_t w, int32_t dtype,
                void *stream, bool relu)
{
    g_last_error.clear();
    if (int rc = quan::iqbn_validate(x, gamma, beta, eps, out, mean, var, n, c, h, w, dtype))
        return rc;
    const int64_t pixels = int64_t(n) * h * w;
    const quan::DType dt = to_dt(dtype);
    void *work = nullptr;
    if (int rc = workspace(stream, kIqbnPartials, quan::iqbn_workspace_bytes(pixels, c), &work))
        return rc;
    unsigned *flags = nullptr;
    if (int rc = iqbn_flags(stream, &flags))
        return rc;
    hipError_t e = quan::iqbn_run(x, gamma, beta, eps, relu, out, mean, var, pixels, c, dt, work, flags,
                                  static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail_hip(e, "iqbn launch");
    return QUAN_OK;
}

}  // namespace

extern "C" {

namespace {

// The convolution on packed weights (Hamilton, eq. 5, or separable, eq. 7).
int conv_packed(const char *name, bool sep, const void *x, const void *packed, const void *bias,
                int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t dilation_h,
                int32_t dilation_w, void *out, int32_t n, int32_t c_in, int32_t h, int32_t w, int32_t c_out,
                int32_t k_h, int32_t k_w, int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!x || !packed || !out)
        return fail(QUAN_ERR_NULL, "%s: x, packed and out must be non-NULL", name);
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(x, bias, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, out,
                            n, c_in, h, w, c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    const int64_t need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    if (misaligned(packed, 16))
        return fail(QUAN_ERR_ALIGN, "%s: packed must be 16-byte aligned", name);
    if (overlaps(out, ob, packed, size_t(need)))
        return fail(QUAN_ERR_ALIAS, "%s: out overlaps the packed weights", name);
    const quan::DType dt = to_dt(dtype);
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, dt);
    const quan::ConvPlan plan = quan::qconv2d_plan(g, dt, sep ? quan::ConvForm::Separable : quan::ConvForm::Hamilton);
    quan::ConvClaim claim{};
    if (int rc = conv_claim(stream, &claim))
        return rc;
    hipError_t e = quan::qconv2d_run(plan, pg, g, dt, x, packed, bias, out, nullptr, nullptr,
                                     static_cast<hipStream_t>(stream), false, &claim);
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d launch");
    return QUAN_OK;
}

// The convolution on the four real kernels, packed into a library workspace
// first.
int conv_unpacked(const char *name, bool sep, const void *x, const void *w_r, const void *w_i,
                  const void *w_j, const void *w_k, const void *bias, int32_t stride_h, int32_t stride_w,
                  int32_t pad_h, int32_t pad_w, int32_t dilation_h, int32_t dilation_w, void *out, int32_t n,
                  int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype,
                  void *stream)
{
    g_last_error.clear();
    if (!x || !w_r || !w_i || !w_j || !w_k || !out)
        return fail(QUAN_ERR_NULL, "%s: x, w_r, w_i, w_j, w_k and out must be non-NULL", name);
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(x, bias, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, out,
                            n, c_in, h, w, c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    const size_t es = elem_size(dtype);
    if (misaligned(w_r, es) || misaligned(w_i, es) || misaligned(w_j, es) || misaligned(w_k, es))
        return fail(QUAN_ERR_ALIGN, "%s: weights and bias must be aligned to their element size", name);
    const size_t wb = size_t(c_out) * c_in * k_h * k_w * es;
    if (overlaps(out, ob, w_r, wb) || overlaps(out, ob, w_i, wb) || overlaps(out, ob, w_j, wb) ||
        overlaps(out, ob, w_k, wb))
        return fail(QUAN_ERR_ALIAS, "%s: out overlaps x, a kernel or the bias", name);
    const int64_t need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);

    void *wpack = nullptr;
    if (int rc = workspace(stream, kWeightPack, size_t(need), &wpack))
        return rc;
    const quan::DType dt = to_dt(dtype);
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, dt);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = quan::qconv2d_pack_weights(pg, c_in, c_out, k_h, k_w, dt, w_r, w_i, w_j, w_k,
                                              wpack, s);
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d weight pack launch");
    quan::ConvClaim claim{};
    if (int rc = conv_claim(stream, &claim))
        return rc;
    e = quan::qconv2d_run(quan::qconv2d_plan(g, dt, sep ? quan::ConvForm::Separable : quan::ConvForm::Hamilton), pg,
                          g, dt, x, wpack, bias, out, nullptr, nullptr, s, false, &claim);
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d launch");
    return QUAN_OK;
}

}  // namespace

QUAN_API int64_t quan_qconv2d_packed_bytes(int32_t c_in, int32_t c_out, int32_t k_h, int32_t k_w,
                                           int32_t dtype)
{
    g_last_error.clear();
    if (int rc = check_dtype(dtype))
        return rc;
    if (c_in < 1 || c_out < 1 || k_h < 1 || k_w < 1)
        return fail(QUAN_ERR_SHAPE, "qconv2d_packed_bytes: sizes must be >= 1");
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, to_dt(dtype));
    if (pg.bytes > size_t(kMaxElems))
        return fail(QUAN_ERR_UNSUPPORTED, "qconv2d: packed weights exceed 2^31-1 bytes");
    return int64_t(pg.bytes);
}

QUAN_API int quan_qconv2d_pack_weights(const void *w_r, const void *w_i, const void *w_j,
                                       const void *w_k, int32_t c_in, int32_t c_out, int32_t k_h,
                                       int32_t k_w, int32_t dtype, void *packed,
                                       int64_t packed_bytes, void *stream)
{
    g_last_error.clear();
    if (!w_r || !w_i || !w_j || !w_k || !packed)
        return fail(QUAN_ERR_NULL, "qconv2d_pack_weights: w_r..w_k and packed must be non-NULL");
    const int64_t need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    if (packed_bytes < need)
        return fail(QUAN_ERR_SHAPE, "qconv2d_pack_weights: packed holds %lld bytes, needs %lld",
                    (long long)packed_bytes, (long long)need);
    const size_t es = elem_size(dtype);
    if (misaligned(packed, 16))
        return fail(QUAN_ERR_ALIGN, "qconv2d_pack_weights: packed must be 16-byte aligned");
    if (misaligned(w_r, es) || misaligned(w_i, es) || misaligned(w_j, es) || misaligned(w_k, es))
        return fail(QUAN_ERR_ALIGN, "qconv2d_pack_weights: kernels must be aligned to their element size");
    const size_t wb = size_t(c_out) * c_in * k_h * k_w * es;
    if (overlaps(packed, size_t(need), w_r, wb) || overlaps(packed, size_t(need), w_i, wb) ||
        overlaps(packed, size_t(need), w_j, wb) || overlaps(packed, size_t(need), w_k, wb))
        return fail(QUAN_ERR_ALIAS, "qconv2d_pack_weights: packed overlaps a kernel");
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, to_dt(dtype));
    hipError_t e = quan::qconv2d_pack_weights(pg, c_in, c_out, k_h, k_w, to_dt(dtype), w_r, w_i,
                                              w_j, w_k, packed, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d weight pack launch");
    return QUAN_OK;
}

QUAN_API int quan_qconv2d_forward_packed(const void *x, const void *packed, const void *bias,
                                         int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                         int32_t pad_w, int32_t dilation_h, int32_t dilation_w,
                                         void *out, int32_t n, int32_t c_in, int32_t h, int32_t w,
                                         int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype,
                                         void *stream)
{
    return conv_packed("qconv2d_forward_packed", false, x, packed, bias, stride_h, stride_w, pad_h, pad_w,
                       dilation_h, dilation_w, out, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_separable_forward_packed(const void *x, const void *packed, const void *bias,
                                                   int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                                   int32_t pad_w, int32_t dilation_h, int32_t dilation_w,
                                                   void *out, int32_t n, int32_t c_in, int32_t h, int32_t w,
                                                   int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype,
                                                   void *stream)
{
    return conv_packed("qconv2d_separable_forward_packed", true, x, packed, bias, stride_h, stride_w, pad_h,
                       pad_w, dilation_h, dilation_w, out, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_forward(const void *x, const void *w_r, const void *w_i, const void *w_j,
                                  const void *w_k, const void *bias, int32_t stride_h,
                                  int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t dilation_h,
                                  int32_t dilation_w, void *out, int32_t n, int32_t c_in, int32_t h,
                                  int32_t w, int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype,
                                  void *stream)
{
    return conv_unpacked("qconv2d", false, x, w_r, w_i, w_j, w_k, bias, stride_h, stride_w, pad_h, pad_w,
                         dilation_h, dilation_w, out, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_separable_forward(const void *x, const void *w_r, const void *w_i, const void *w_j,
                                            const void *w_k, const void *bias, int32_t stride_h,
                                            int32_t stride_w, int32_t pad_h, int32_t pad_w, int32_t dilation_h,
                                            int32_t dilation_w, void *out, int32_t n, int32_t c_in, int32_t h,
                                            int32_t w, int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype,
                                            void *stream)
{
    return conv_unpacked("qconv2d_separable", true, x, w_r, w_i, w_j, w_k, bias, stride_h, stride_w, pad_h,
                         pad_w, dilation_h, dilation_w, out, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_iqbn_forward(const void *x, const void *packed, const void *bias,
                                       int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                       int32_t dilation_h, int32_t dilation_w, const float *gamma,
                                       const float *beta, float eps, int32_t relu, int32_t stats,
                                       void *out, float *mean, float *var, int32_t n, int32_t c_in,
                                       int32_t h, int32_t w,
                                       int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!x || !packed || !out || !gamma || !beta || !mean || !var)
        return fail(QUAN_ERR_NULL,
                    "qconv2d_iqbn: x, packed, gamma, beta, out, mean and var must be non-NULL");
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(x, bias, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, out,
                            n, c_in, h, w, c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    if (!(eps > 0.0f) || eps != eps)
        return fail(QUAN_ERR_SHAPE, "qconv2d_iqbn: eps must be > 0 (got %g)", double(eps));
    if (relu != 0 && relu != 1)
        return fail(QUAN_ERR_SHAPE, "qconv2d_iqbn: relu must be 0 or 1");
    if (stats != QUAN_STATS_AUTO && stats != QUAN_STATS_EPILOGUE && stats != QUAN_STATS_PASS)
        return fail(QUAN_ERR_SHAPE, "qconv2d_iqbn: stats must be QUAN_STATS_AUTO, _EPILOGUE or _PASS (got %d)",
                    int(stats));
    const int64_t need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    if (misaligned(packed, 16))
        return fail(QUAN_ERR_ALIGN, "qconv2d_iqbn: packed must be 16-byte aligned");
    if (misaligned(gamma, 4) || misaligned(beta, 4) || misaligned(mean, 4) || misaligned(var, 4))
        return fail(QUAN_ERR_ALIGN, "qconv2d_iqbn: gamma, beta, mean and var must be 4-byte aligned");
    const size_t sbytes = size_t(4) * c_out * sizeof(float);
    if (overlaps(out, ob, packed, size_t(need)))
        return fail(QUAN_ERR_ALIAS, "qconv2d_iqbn: out overlaps the packed weights");
    if (overlaps(mean, sbytes, var, sbytes) || overlaps(mean, sbytes, out, ob) ||
        overlaps(var, sbytes, out, ob) || overlaps(mean, sbytes, x, xb) || overlaps(var, sbytes, x, xb))
        return fail(QUAN_ERR_ALIAS, "qconv2d_iqbn: mean/var overlap each other or a tensor");

    const quan::DType dt = to_dt(dtype);
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, dt);
    const quan::ConvPlan plan = quan::qconv2d_plan(g, dt, quan::ConvForm::Hamilton);
    const int64_t pixels = g.m();
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *work = nullptr;
    quan::ConvClaim claim{};
    if (int rc = conv_claim(stream, &claim))
        return rc;
    hipError_t e;
    // AUTO: an IQBN pass after the plain convolution where the tensor takes
    // the one-launch form and is large enough for its fixed cost (two grid
    // barriers and a merge) to matter less than the epilogue's statistics
    // work, or takes the merged two-launch form; else the epilogue.
    // Measured per layer on MI355X: 103 MB tensors (64 x 56 x 56, 64
    // channels) 262.7 us with the pass against 267.5 with the epilogue; 52 MB
    // (16 x 80 x 80, 64 channels, two layers) 162.3 against 160.1; 12.8 MB
    // (32 x 14 x 14, 256 channels, merged form) 133.0 against 137.3.
    constexpr int64_t kPassMinBytes = int64_t(64) << 20;
    const bool big = pixels * 4 * c_out * int64_t(elem_size(dtype)) >= kPassMinBytes;
    const bool pass = (big && quan::iqbn_one_launch(pixels, c_out, dt)) || quan::iqbn_merged(pixels, c_out, dt);
    const bool epilogue = stats == QUAN_STATS_EPILOGUE || (stats == QUAN_STATS_AUTO && !pass);
    if (epilogue && quan::qconv2d_writes_stats(plan, g, dt)) {
        // statistics gathered in the convolution's epilogue
        if (int rc = workspace(stream, kIqbnPartials, quan::iqbn_tile_stats_bytes(plan.stat_tiles, c_out), &work))
            return rc;
        e = quan::qconv2d_run(plan, pg, g, dt, x, packed, bias, out, static_cast<float *>(work), nullptr, s, false,
                              &claim);
        if (e != hipSuccess)
            return fail_hip(e, "qconv2d launch");
        e = quan::iqbn_from_tiles_run(static_cast<const float *>(work), plan.stat_tiles, plan.stat_rows, gamma,
                                      beta, eps, relu != 0, out, mean, var, pixels, c_out, dt, s);
    } else {
        if (int rc = workspace(stream, kIqbnPartials, quan::iqbn_workspace_bytes(pixels, c_out), &work))
            return rc;
        unsigned *flags = nullptr;
        if (int rc = iqbn_flags(stream, &flags))
            return rc;
        e = quan::qconv2d_run(plan, pg, g, dt, x, packed, bias, out, nullptr, nullptr, s, false, &claim);
        if (e != hipSuccess)
            return fail_hip(e, "qconv2d launch");
        e = quan::iqbn_run(out, gamma, beta, eps, relu != 0, out, mean, var, pixels, c_out, dt, work, flags, s);
    }
    if (e != hipSuccess)
        return fail_hip(e, "iqbn launch");
    return QUAN_OK;
}

QUAN_API int quan_qconv2d_iqbn_inference(const void *x, const void *packed, const void *bias,
                                         int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                         int32_t dilation_h, int32_t dilation_w, const float *running_mean,
                                         const float *running_var, const float *gamma, const float *beta,
                                         float eps, int32_t relu, void *out, int32_t n, int32_t c_in,
                                         int32_t h, int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
                                         int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!x || !packed || !out || !running_mean || !running_var || !gamma || !beta)
        return fail(QUAN_ERR_NULL, "qconv2d_iqbn_inference: x, packed, running_mean, running_var, gamma, "
                                   "beta and out must be non-NULL");
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(x, bias, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, out,
                            n, c_in, h, w, c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    if (!(eps > 0.0f) || eps != eps)
        return fail(QUAN_ERR_SHAPE, "qconv2d_iqbn_inference: eps must be > 0 (got %g)", double(eps));
    if (relu != 0 && relu != 1)
        return fail(QUAN_ERR_SHAPE, "qconv2d_iqbn_inference: relu must be 0 or 1");
    const int64_t need = quan_qconv2d_packed_bytes(c_in, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    if (misaligned(packed, 16))
        return fail(QUAN_ERR_ALIGN, "qconv2d_iqbn_inference: packed must be 16-byte aligned");
    if (misaligned(running_mean, 4) || misaligned(running_var, 4) || misaligned(gamma, 4) ||
        misaligned(beta, 4))
        return fail(QUAN_ERR_ALIGN, "qconv2d_iqbn_inference: statistics, gamma and beta must be 4-byte aligned");
    const size_t sbytes = size_t(4) * c_out * sizeof(float);
    if (overlaps(out, ob, packed, size_t(need)) || overlaps(out, ob, running_mean, sbytes) ||
        overlaps(out, ob, running_var, sbytes) || overlaps(out, ob, gamma, sbytes) ||
        overlaps(out, ob, beta, sbytes))
        return fail(QUAN_ERR_ALIAS, "qconv2d_iqbn_inference: out overlaps the weights, statistics or parameters");

    const quan::DType dt = to_dt(dtype);
    const quan::PackGeom pg = quan::qconv2d_pack_geom(c_in, c_out, k_h, k_w, dt);
    hipStream_t s = static_cast<hipStream_t>(stream);
    void *work = nullptr;
    if (int rc = workspace(stream, kIqbnFold, 2 * sbytes, &work))
        return rc;
    float *scale = static_cast<float *>(work), *shift = scale + size_t(4) * c_out;
    hipError_t e = quan::iqbn_fold_run(running_mean, running_var, gamma, beta, bias, eps, c_out, dt, scale,
                                       shift, s);
    if (e != hipSuccess)
        return fail_hip(e, "iqbn fold launch");
    const quan::ConvFold fold{scale, shift, relu != 0};
    quan::ConvClaim claim{};
    if (int rc = conv_claim(stream, &claim))
        return rc;
    e = quan::qconv2d_run(quan::qconv2d_plan(g, dt, quan::ConvForm::Hamilton), pg, g, dt, x, packed, bias, out,
                          nullptr, &fold, s, false, &claim);
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d launch");
    return QUAN_OK;
}

QUAN_API int quan_qconv2d_poincare_forward(const void *rgb, const void *packed, const void *bias,
                                           int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                           int32_t dilation_h, int32_t dilation_w, void *out, int32_t n,
                                           int32_t h, int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
                                           int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!rgb || !packed || !out)
        return fail(QUAN_ERR_NULL, "qconv2d_poincare: rgb, packed and out must be non-NULL");
    // the layer's geometry as a one-channel convolution of the planes
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(rgb, bias, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, out, n, 1, h, w,
                            c_out, k_h, k_w, dtype, &g, &xb, &ob, true))
        return rc;
    const int64_t need = quan_qconv2d_packed_bytes(1, c_out, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    if (misaligned(packed, 16))
        return fail(QUAN_ERR_ALIGN, "qconv2d_poincare: packed must be 16-byte aligned");
    if (overlaps(out, ob, packed, size_t(need)))
        return fail(QUAN_ERR_ALIAS, "qconv2d_poincare: out overlaps the packed weights");
    const quan::DType dt = to_dt(dtype);
    const quan::PackGeom pg = quan::qconv2d_pack_geom(1, c_out, k_h, k_w, dt);
    // the stem kernel where it takes the layer, else the implicit-GEMM
    // kernel with the map in its loads
    hipError_t e = quan::qconv2d_stem_run(pg, g, dt, rgb, packed, bias, out, static_cast<hipStream_t>(stream));
    if (e == hipErrorNotSupported) {
        quan::ConvClaim claim{};
        if (int rc = conv_claim(stream, &claim))
            return rc;
        e = quan::qconv2d_run(quan::qconv2d_plan(g, dt, quan::ConvForm::Hamilton), pg, g, dt, rgb, packed, bias, out,
                              nullptr, nullptr, static_cast<hipStream_t>(stream), true, &claim);
    }
    if (e != hipSuccess)
        return fail_hip(e, "qconv2d_poincare launch");
    return QUAN_OK;
}

QUAN_API int quan_poincare_map(const void *rgb, void *out, int32_t n, int32_t h, int32_t w, int32_t dtype,
                               void *stream)
{
    g_last_error.clear();
    if (!rgb || !out)
        return fail(QUAN_ERR_NULL, "poincare_map: rgb and out must be non-NULL");
    if (int rc = check_dtype(dtype))
        return rc;
    if (n < 1 || h < 1 || w < 1)
        return fail(QUAN_ERR_SHAPE, "poincare_map: sizes must be >= 1 (n=%d h=%d w=%d)", n, h, w);
    const int64_t pixels = int64_t(n) * h * w;
    if (pixels * 4 > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "poincare_map: output of %lld elements exceeds 2^31-1",
                    (long long)(pixels * 4));
    const size_t es = elem_size(dtype);
    if (misaligned(rgb, es) || misaligned(out, 4 * es))
        return fail(QUAN_ERR_ALIGN, "poincare_map: rgb must be aligned to its element, out to four");
    if (overlaps(rgb, size_t(pixels) * 3 * es, out, size_t(pixels) * 4 * es))
        return fail(QUAN_ERR_ALIAS, "poincare_map: out overlaps rgb");
    const hipError_t e = quan::poincare_run(rgb, out, n, h, w, to_dt(dtype), static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail_hip(e, "poincare launch");
    return QUAN_OK;
}

namespace {

// Input gradient of the Hamilton (sep false) or separable (sep true) form.
int backward_data(const char *name, bool sep, const void *dy, const void *w_r, const void *w_i, const void *w_j,
                  const void *w_k, int32_t stride_h, int32_t stride_w, int32_t pad_h, int32_t pad_w,
                  int32_t dilation_h, int32_t dilation_w, void *dx, int32_t n, int32_t c_in, int32_t h, int32_t w,
                  int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!dy || !w_r || !w_i || !w_j || !w_k || !dx)
        return fail(QUAN_ERR_NULL, "%s: dy, w_r, w_i, w_j, w_k and dx must be non-NULL", name);
    // the forward layer's geometry, with dx in the place of x and dy of out
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(dx, nullptr, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, dy, n, c_in, h,
                            w, c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    if (pad_h > dilation_h * (k_h - 1) || pad_w > dilation_w * (k_w - 1))
        return fail(QUAN_ERR_UNSUPPORTED, "%s: padding beyond the dilated kernel span", name);
    const size_t es = elem_size(dtype);
    if (misaligned(w_r, es) || misaligned(w_i, es) || misaligned(w_j, es) || misaligned(w_k, es))
        return fail(QUAN_ERR_ALIGN, "%s: kernels must be aligned to their element size", name);
    const size_t wb = size_t(c_out) * c_in * k_h * k_w * es;
    if (overlaps(dx, xb, w_r, wb) || overlaps(dx, xb, w_i, wb) || overlaps(dx, xb, w_j, wb) ||
        overlaps(dx, xb, w_k, wb))
        return fail(QUAN_ERR_ALIAS, "%s: dx overlaps dy or a kernel", name);
    const quan::DType dt = to_dt(dtype);
    const quan::ConvGeom t = quan::qconv2d_grad_data_geom(g);
    // the gradient convolution's own limits (its input is dy or the staged,
    // zero-inserted dy)
    const int64_t t_img = int64_t(t.h) * t.w * 4 * t.c_in * int64_t(es);
    if (int64_t(t.n) * t.h * t.w * 4 * t.c_in > kMaxElems || t_img * (256 / (int64_t(h) * w) + 2) > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "%s: staged gradient too large for 32-bit offsets", name);
    const int64_t need = quan_qconv2d_packed_bytes(c_out, c_in, k_h, k_w, dtype);
    if (need < 0)
        return int(need);
    void *wpack = nullptr, *stage = nullptr;
    if (int rc = workspace(stream, kGradPack, size_t(need), &wpack))
        return rc;
    const size_t sb = quan::qconv2d_grad_data_stage_bytes(g, dt);
    if (sb > 0) {
        if (int rc = workspace(stream, kGradStage, sb, &stage))
            return rc;
    }
    quan::ConvClaim claim{};
    if (int rc = conv_claim(stream, &claim))
        return rc;
    const hipError_t e = quan::qconv2d_backward_data_run(g, dt, dy, w_r, w_i, w_j, w_k, dx, wpack, stage,
                                                         static_cast<hipStream_t>(stream), sep, &claim);
    if (e != hipSuccess)
        return fail_hip(e, "backward data launch");
    return QUAN_OK;
}

}  // namespace

QUAN_API int quan_qconv2d_backward_data(const void *dy, const void *w_r, const void *w_i, const void *w_j,
                                        const void *w_k, int32_t stride_h, int32_t stride_w, int32_t pad_h,
                                        int32_t pad_w, int32_t dilation_h, int32_t dilation_w, void *dx, int32_t n,
                                        int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h, int32_t k_w,
                                        int32_t dtype, void *stream)
{
    return backward_data("qconv2d_backward_data", false, dy, w_r, w_i, w_j, w_k, stride_h, stride_w, pad_h, pad_w,
                         dilation_h, dilation_w, dx, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_separable_backward_data(const void *dy, const void *w_r, const void *w_i,
                                                  const void *w_j, const void *w_k, int32_t stride_h,
                                                  int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                                  int32_t dilation_h, int32_t dilation_w, void *dx, int32_t n,
                                                  int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h,
                                                  int32_t k_w, int32_t dtype, void *stream)
{
    return backward_data("qconv2d_separable_backward_data", true, dy, w_r, w_i, w_j, w_k, stride_h, stride_w, pad_h,
                         pad_w, dilation_h, dilation_w, dx, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}


namespace {

// Weight and bias gradients of the Hamilton (sep false) or separable form.
int backward_weight(const char *name, bool sep, const void *x, const void *dy, int32_t stride_h, int32_t stride_w,
                    int32_t pad_h, int32_t pad_w, int32_t dilation_h, int32_t dilation_w, float *dw_r, float *dw_i,
                    float *dw_j, float *dw_k, float *db, int32_t n, int32_t c_in, int32_t h, int32_t w,
                    int32_t c_out, int32_t k_h, int32_t k_w, int32_t dtype, void *stream)
{
    g_last_error.clear();
    if (!x || !dy || !dw_r || !dw_i || !dw_j || !dw_k)
        return fail(QUAN_ERR_NULL, "%s: x, dy and dw_r..dw_k must be non-NULL", name);
    quan::ConvGeom g;
    size_t xb = 0, ob = 0;
    if (int rc = check_conv(x, nullptr, stride_h, stride_w, pad_h, pad_w, dilation_h, dilation_w, dy, n, c_in, h, w,
                            c_out, k_h, k_w, dtype, &g, &xb, &ob))
        return rc;
    float *outs[] = {dw_r, dw_i, dw_j, dw_k, db};
    const size_t wb = size_t(c_out) * c_in * k_h * k_w * sizeof(float), bb = size_t(4) * c_out * sizeof(float);
    for (int i = 0; i < 5; ++i) {
        if (!outs[i])
            continue;
        const size_t bi = i < 4 ? wb : bb;
        if (misaligned(outs[i], 4))
            return fail(QUAN_ERR_ALIGN, "%s: dw_* and db must be 4-byte aligned", name);
        if (overlaps(outs[i], bi, x, xb) || overlaps(outs[i], bi, dy, ob))
            return fail(QUAN_ERR_ALIAS, "%s: a gradient overlaps x or dy", name);
        for (int j = 0; j < i; ++j) {
            if (outs[j] && overlaps(outs[i], bi, outs[j], j < 4 ? wb : bb))
                return fail(QUAN_ERR_ALIAS, "%s: gradients overlap each other", name);
        }
    }
    void *work = nullptr;
    if (int rc = workspace(stream, kWgrad, quan::qconv2d_wgrad_work_bytes(g), &work))
        return rc;
    const hipError_t e = quan::qconv2d_backward_weight_run(g, to_dt(dtype), x, dy, dw_r, dw_i, dw_j, dw_k, db, work,
                                                           static_cast<hipStream_t>(stream), sep);
    if (e != hipSuccess)
        return fail_hip(e, "backward weight launch");
    return QUAN_OK;
}

}  // namespace

QUAN_API int quan_qconv2d_backward_weight(const void *x, const void *dy, int32_t stride_h, int32_t stride_w,
                                          int32_t pad_h, int32_t pad_w, int32_t dilation_h, int32_t dilation_w,
                                          float *dw_r, float *dw_i, float *dw_j, float *dw_k, float *db, int32_t n,
                                          int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h,
                                          int32_t k_w, int32_t dtype, void *stream)
{
    return backward_weight("qconv2d_backward_weight", false, x, dy, stride_h, stride_w, pad_h, pad_w, dilation_h,
                           dilation_w, dw_r, dw_i, dw_j, dw_k, db, n, c_in, h, w, c_out, k_h, k_w, dtype, stream);
}

QUAN_API int quan_qconv2d_separable_backward_weight(const void *x, const void *dy, int32_t stride_h,
                                                    int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                                    int32_t dilation_h, int32_t dilation_w, float *dw_r,
                                                    float *dw_i, float *dw_j, float *dw_k, float *db, int32_t n,
                                                    int32_t c_in, int32_t h, int32_t w, int32_t c_out, int32_t k_h,
                                                    int32_t k_w, int32_t dtype, void *stream)
{
    return backward_weight("qconv2d_separable_backward_weight", true, x, dy, stride_h, stride_w, pad_h, pad_w,
                           dilation_h, dilation_w, dw_r, dw_i, dw_j, dw_k, db, n, c_in, h, w, c_out, k_h, k_w, dtype,
                           stream);
}



QUAN_API int quan_iqbn_backward(const void *x, const void *dout, const void *y, const float *mean,
                                const float *var, const float *gamma, float eps, void *dx, float *dgamma,
                                float *dbeta, int32_t n, int32_t c, int32_t h, int32_t w, int32_t dtype,
                                void *stream)
{
    g_last_error.clear();
    if (!x || !dout || !mean || !var || !gamma || !dx || !dgamma || !dbeta)
        return fail(QUAN_ERR_NULL, "iqbn_backward: x, dout, mean, var, gamma, dx, dgamma and dbeta must be non-NULL");
    if (int rc = check_dtype(dtype))
        return rc;
    if (n < 1 || c < 1 || h < 1 || w < 1)
        return fail(QUAN_ERR_SHAPE, "iqbn_backward: sizes must be >= 1 (n=%d c=%d h=%d w=%d)", n, c, h, w);
    if (!(eps > 0.0f) || eps != eps)
        return fail(QUAN_ERR_SHAPE, "iqbn_backward: eps must be > 0 (got %g)", double(eps));
    const int64_t pixels = int64_t(n) * h * w;
    const int64_t elems = pixels * 4 * c;
    if (elems > kMaxElems)
        return fail(QUAN_ERR_UNSUPPORTED, "iqbn_backward: tensor of %lld elements exceeds 2^31-1", (long long)elems);
    const size_t es = elem_size(dtype);
    if (misaligned(x, 16) || misaligned(dout, 16) || misaligned(dx, 16) || (y && misaligned(y, 16)))
        return fail(QUAN_ERR_ALIGN, "iqbn_backward: x, dout, y and dx must be 16-byte aligned");
    if (misaligned(mean, 4) || misaligned(var, 4) || misaligned(gamma, 4) || misaligned(dgamma, 4) ||
        misaligned(dbeta, 4))
        return fail(QUAN_ERR_ALIGN, "iqbn_backward: mean, var, gamma, dgamma and dbeta must be 4-byte aligned");
    const size_t tb = size_t(elems) * es, sb = size_t(4) * c * sizeof(float);
    if (overlaps(dx, tb, x, tb) || (y && overlaps(dx, tb, y, tb)) || (dx != dout && overlaps(dx, tb, dout, tb)))
        return fail(QUAN_ERR_ALIAS, "iqbn_backward: dx overlaps x or y, or partially overlaps dout");
    const void *tensors[] = {x, dout, y, dx};
    for (const void *t : tensors) {
        if (t && (overlaps(dgamma, sb, t, tb) || overlaps(dbeta, sb, t, tb)))
            return fail(QUAN_ERR_ALIAS, "iqbn_backward: dgamma/dbeta overlap a tensor");
    }
    if (overlaps(dgamma, sb, dbeta, sb) || overlaps(dgamma, sb, mean, sb) || overlaps(dgamma, sb, var, sb) ||
        overlaps(dgamma, sb, gamma, sb) || overlaps(dbeta, sb, mean, sb) || overlaps(dbeta, sb, var, sb) ||
        overlaps(dbeta, sb, gamma, sb))
        return fail(QUAN_ERR_ALIAS, "iqbn_backward: dgamma/dbeta overlap each other or the statistics");
    void *work = nullptr;
    if (int rc = workspace(stream, kIqbnPartials, quan::iqbn_workspace_bytes(pixels, c), &work))
        return rc;
    const hipError_t e = quan::iqbn_backward_run(x, dout, y, mean, var, gamma, eps, dx, dgamma, dbeta, pixels, c,
                                                 to_dt(dtype), work, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail_hip(e, "iqbn backward launch");
    return QUAN_OK;
}

QUAN_API int quan_iqbn_forward(const void *x, const float *gamma, const float *beta, float eps,
                               void *out, float *mean, float *var, int32_t n, int32_t c, int32_t h,
                               int32_t w, int32_t dtype, void *stream)
{
    return iqbn_common(x, gamma, beta, eps, out, mean, var, n, c, h, w, dtype, stream, false);
}

QUAN_API int quan_iqbn_relu_forward(const void *x, const float *gamma, const float *beta, float eps,
                                    void *out, float *mean, float *var, int32_t n, int32_t c,
                                    int32_t h, int32_t w, int32_t dtype, void *stream)
{
    return iqbn_common(x, gamma, beta, eps, out, mean, var, n, c, h, w, dtype, stream, true);
}

namespace {

// ---- descriptor entry points: checks of quan_tensor, all on the host ------

int desc_present(const quan_tensor *t, const char *fn, const char *what)
{
    if (t == nullptr || t->data == nullptr)
        return fail(QUAN_ERR_NULL, "%s: %s descriptor or its data pointer is NULL", fn, what);
    return QUAN_OK;
}

// ndim, extents (want[i] < 0: any extent >= 1) and dtype of a descriptor.
int desc_shape(const quan_tensor *t, const char *fn, const char *what, int ndim, const int64_t *want,
               int32_t dtype)
{
    if (t->ndim != ndim)
        return fail(QUAN_ERR_SHAPE, "%s: %s has ndim %d, expected %d", fn, what, t->ndim, ndim);
    for (int i = 0; i < ndim; ++i) {
        if (t->shape[i] < 1)
            return fail(QUAN_ERR_SHAPE, "%s: %s extent %lld on axis %d must be >= 1", fn, what,
                        (long long)t->shape[i], i);
        if (t->shape[i] > INT32_MAX)
            return fail(QUAN_ERR_UNSUPPORTED, "%s: %s extent %lld on axis %d exceeds 2^31-1", fn, what,
                        (long long)t->shape[i], i);
        if (want[i] >= 0 && t->shape[i] != want[i])
            return fail(QUAN_ERR_SHAPE, "%s: %s extent %lld on axis %d, expected %lld", fn, what,
                        (long long)t->shape[i], i, (long long)want[i]);
    }
    if (t->dtype != dtype)
        return fail(QUAN_ERR_DTYPE, "%s: %s has dtype %d, expected %d", fn, what, t->dtype, dtype);
    return QUAN_OK;
}

// Strides against the required ones; an axis of extent 1 is never stepped.
int desc_strides(const quan_tensor *t, const char *fn, const char *what, const int64_t *want,
                 const char *layout)
{
    for (int i = 0; i < t->ndim; ++i)
        if (t->shape[i] != 1 && t->strides[i] != want[i])
            return fail(QUAN_ERR_LAYOUT, "%s: %s is not %s (axis %d: stride %lld, expected %lld)", fn, what,
                        layout, i, (long long)t->strides[i], (long long)want[i]);
    return QUAN_OK;
}

// A quaternion map [N, 4, C, H, W] stored channels-last by component.
int desc_activation(const quan_tensor *t, const char *fn, const char *what, const int64_t *want, int32_t dtype)
{
    if (int rc = desc_present(t, fn, what))
        return rc;
    if (int rc = desc_shape(t, fn, what, 5, want, dtype))
        return rc;
    const int64_t c = t->shape[2], h = t->shape[3], w = t->shape[4];
    const int64_t strides[5] = {h * w * 4 * c, c, 1, w * 4 * c, 4 * c};
    return desc_strides(t, fn, what, strides, "channels-last by component ([N][H][W][4][C] in memory)");
}

// A dense row-major tensor of the given extents.
int desc_dense(const quan_tensor *t, const char *fn, const char *what, int ndim, const int64_t *want,
               int32_t dtype)
{
    if (int rc = desc_present(t, fn, what))
        return rc;
    if (int rc = desc_shape(t, fn, what, ndim, want, dtype))
        return rc;
    int64_t strides[5];
    int64_t step = 1;
    for (int i = ndim - 1; i >= 0; --i) {
        strides[i] = step;
        step *= t->shape[i];
    }
    return desc_strides(t, fn, what, strides, "dense row-major");
}

int iqbn_desc(const char *fn, const quan_tensor *x, const quan_tensor *gamma, const quan_tensor *beta,
              float eps, quan_tensor *out, quan_tensor *mean, quan_tensor *var, void *stream, bool relu)
{
    g_last_error.clear();
    if (int rc = desc_present(x, fn, "x"))
        return rc;
    if (int rc = check_dtype(x->dtype))
        return rc;
    const int64_t any5[5] = {-1, 4, -1, -1, -1};
    if (int rc = desc_activation(x, fn, "x", any5, x->dtype))
        return rc;
    const int64_t stat[2] = {4, x->shape[2]};
    const quan_tensor *params[4] = {gamma, beta, mean, var};
    const char *names[4] = {"gamma", "beta", "mean", "var"};
    for (int i = 0; i < 4; ++i)
        if (int rc = desc_dense(params[i], fn, names[i], 2, stat, QUAN_F32))
            return rc;
    if (int rc = desc_activation(out, fn, "out", x->shape, x->dtype))
        return rc;
    return iqbn_common(x->data, static_cast<const float *>(gamma->data), static_cast<const float *>(beta->data),
                       eps, out->data, static_cast<float *>(mean->data), static_cast<float *>(var->data),
                       int32_t(x->shape[0]), int32_t(x->shape[2]), int32_t(x->shape[3]), int32_t(x->shape[4]),
                       x->dtype, stream, relu);
}

}  // namespace

QUAN_API int quan_qconv2d_forward_desc(const quan_tensor *x, const quan_tensor *w_r, const quan_tensor *w_i,
                                       const quan_tensor *w_j, const quan_tensor *w_k, const quan_tensor *bias,
                                       const int32_t stride[2], const int32_t pad[2], const int32_t dilation[2],
                                       quan_tensor *out, void *stream)
{
    const char *fn = "qconv2d_forward_desc";
    g_last_error.clear();
    if (int rc = desc_present(x, fn, "x"))
        return rc;
    if (int rc = check_dtype(x->dtype))
        return rc;
    const int64_t any5[5] = {-1, 4, -1, -1, -1};
    if (int rc = desc_activation(x, fn, "x", any5, x->dtype))
        return rc;
    if (int rc = desc_present(w_r, fn, "w_r"))
        return rc;
    const int64_t wshape[4] = {w_r->ndim == 4 ? w_r->shape[0] : -1, x->shape[2], w_r->ndim == 4 ? w_r->shape[2] : -1,
                               w_r->ndim == 4 ? w_r->shape[3] : -1};
    const quan_tensor *ws[4] = {w_r, w_i, w_j, w_k};
    const char *wn[4] = {"w_r", "w_i", "w_j", "w_k"};
    for (int i = 0; i < 4; ++i)
        if (int rc = desc_dense(ws[i], fn, wn[i], 4, wshape, x->dtype))
            return rc;
    const int64_t c_out = w_r->shape[0], k_h = w_r->shape[2], k_w = w_r->shape[3];
    if (bias != nullptr) {
        const int64_t bshape[2] = {4, c_out};
        if (int rc = desc_dense(bias, fn, "bias", 2, bshape, x->dtype))
            return rc;
    }
    if (stride == nullptr || pad == nullptr || dilation == nullptr)
        return fail(QUAN_ERR_NULL, "%s: stride, pad and dilation must point to (h, w) pairs", fn);
    int64_t o_hw[2];
    for (int i = 0; i < 2; ++i) {
        const int64_t k = i == 0 ? k_h : k_w, in = x->shape[3 + i];
        if (stride[i] < 1 || dilation[i] < 1 || pad[i] < 0)
            return fail(QUAN_ERR_SHAPE, "%s: stride/dilation must be >= 1 and pad >= 0", fn);
        const int64_t span = in + 2 * int64_t(pad[i]) - int64_t(dilation[i]) * (k - 1) - 1;
        if (span < 0)
            return fail(QUAN_ERR_SHAPE, "%s: empty output (kernel span exceeds padded input)", fn);
        o_hw[i] = span / stride[i] + 1;
    }
    const int64_t oshape[5] = {x->shape[0], 4, c_out, o_hw[0], o_hw[1]};
    if (int rc = desc_activation(out, fn, "out", oshape, x->dtype))
        return rc;
    return conv_unpacked("qconv2d", false, x->data, w_r->data, w_i->data, w_j->data, w_k->data,
                         bias ? bias->data : nullptr, stride[0], stride[1], pad[0], pad[1], dilation[0],
                         dilation[1], out->data, int32_t(x->shape[0]), int32_t(x->shape[2]),
                         int32_t(x->shape[3]), int32_t(x->shape[4]), int32_t(c_out), int32_t(k_h), int32_t(k_w),
                         x->dtype, stream);
}

QUAN_API int quan_iqbn_forward_desc(const quan_tensor *x, const quan_tensor *gamma, const quan_tensor *beta,
                                    float eps, quan_tensor *out, quan_tensor *mean, quan_tensor *var, void *stream)
{
    return iqbn_desc("iqbn_forward_desc", x, gamma, beta, eps, out, mean, var, stream, false);
}

QUAN_API int quan_iqbn_relu_forward_desc(const quan_tensor *x, const quan_tensor *gamma, const quan_tensor *beta,
                                         float eps, quan_tensor *out, quan_tensor *mean, quan_tensor *var,
                                         void *stream)
{
    return iqbn_desc("iqbn_relu_forward_desc", x, gamma, beta, eps, out, mean, var, stream, true);
}

QUAN_API const char *quan_last_error(void)
{
    return g_last_error.c_str();
}

QUAN_API int quan_release(void)
{
    std::lock_guard<std::mutex> lock(g_ws_mutex);
    int rc = QUAN_OK;
    int saved = -1;
    if (hipGetDevice(&saved) != hipSuccess)
        saved = -1;
    for (auto &kv : g_ws) {
        Workspace &ws = kv.second;
        if (!ws.ptr)
            continue;
        hipError_t e = hipSetDevice(kv.first.first);
        if (e == hipSuccess)
            e = hipDeviceSynchronize();
        if (e == hipSuccess)
            e = hipFree(ws.ptr);
        if (e != hipSuccess && rc == QUAN_OK)
            rc = fail_hip(e, "quan_release");
        ws.ptr = nullptr;
        ws.bytes = 0;
    }
    g_ws.clear();
    if (saved >= 0 && hipSetDevice(saved) != hipSuccess && rc == QUAN_OK)
        rc = fail(QUAN_ERR_HIP, "quan_release: hipSetDevice failed");
    return rc;
}

QUAN_API const char *quan_version(void)
{
    return "libquan 0.1 (gfx950)";
}

}  // extern "C"
