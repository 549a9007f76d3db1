// C ABI of the CAT W4A4 linear-layer library: argument validation, launch
// and error mapping for the four device calls.  Every check runs on the
// host before anything is enqueued; nothing falls back silently.
#include <hip/hip_runtime.h>

#include <exception>
#include <mutex>
#include <string>

#include "cat_internal.h"
#include "kernels.h"

namespace {

using cat::fail;

int hip_fail(const char* where, hipError_t err) {
    return fail(CAT_ERR_HIP, std::string(where) + ": " + hipGetErrorString(err));
}

bool valid_dtype(int t) { return t == CAT_F32 || t == CAT_BF16; }

// Checks that a device is present and current before the first launch, so
// that a missing GPU reports CAT_ERR_HIP instead of failing inside HIP.
int require_device(const char* where) {
    int count = 0;
    const hipError_t err = hipGetDeviceCount(&count);
    if (err != hipSuccess) return hip_fail(where, err);
    if (count < 1) return fail(CAT_ERR_HIP, std::string(where) + ": no HIP device");
    return CAT_OK;
}

}  // namespace

extern "C" size_t cat_cov_workspace_bytes(int x_dtype, int64_t n, int64_t d, int mode,
                                          int64_t k) {
    if (!valid_dtype(x_dtype) || n < 1 || d < 1) return 0;
    if (mode != CAT_COV_FULL && mode != CAT_COV_BLOCK_DIAG) return 0;
    if (mode == CAT_COV_BLOCK_DIAG && (!cat::is_pow2(k) || k > CAT_MAX_BLOCK || d % k)) return 0;
    size_t bytes = 0;
    if (catk::cov_workspace_bytes(x_dtype == CAT_BF16, d, mode, k, bytes) != hipSuccess) return 0;
    return bytes;
}

extern "C" int cat_cov_accumulate(const void* X, int x_dtype, int64_t n, int64_t d, int mode,
                                  int64_t k, float* acc, void* workspace, size_t workspace_bytes,
                                  void* stream) {
    const char* fn = "cat_cov_accumulate";
    try {
        if (!X || !acc) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (!valid_dtype(x_dtype)) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad x_dtype");
        if (n < 1 || d < 1) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": n and d must be >= 1");
        if (mode != CAT_COV_FULL && mode != CAT_COV_BLOCK_DIAG)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad mode");
        if (mode == CAT_COV_BLOCK_DIAG) {
            if (!cat::is_pow2(k) || k > CAT_MAX_BLOCK)
                return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": k must be a power of two <= 512");
            if (d % k) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d % k != 0");
        }
        if (!cat::aligned16(X) || !cat::aligned16(acc))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        size_t need = 0;
        hipError_t err = catk::cov_workspace_bytes(x_dtype == CAT_BF16, d, mode, k, need);
        if (err != hipSuccess) return hip_fail(fn, err);
        if (need > 0) {
            if (!workspace) return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace is NULL");
            if (workspace_bytes < need)
                return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace too small (need " +
                                                   std::to_string(need) + " bytes)");
            if (!cat::aligned16(workspace))
                return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": workspace must be 16-byte aligned");
        }
        err = catk::launch_cov_accumulate(X, x_dtype == CAT_BF16, n, d, mode, k, acc, workspace,
                                          workspace_bytes, static_cast<hipStream_t>(stream));
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

extern "C" size_t cat_transform_quant_workspace_bytes(int64_t n, int64_t d, int64_t k) {
    if (n < 1 || d < 1) return 0;
    return catk::tq_workspace_bytes(n, d, k);
}

extern "C" size_t cat_transform_quant_asym_workspace_bytes(int64_t n, int64_t d, int64_t k) {
    if (n < 1 || d < 1 || k < 1) return 0;
    return catk::tq_asym_workspace_bytes(n, d, k);
}

extern "C" size_t cat_transform_quant_flag_offset(int64_t n, int64_t d, int64_t k) {
    (void)k;
    if (n < 1 || d < 1) return 0;
    return catk::tq_flag_offset_bytes(n, d);
}

extern "C" void cat_set_exchange_spin_limit(uint32_t polls) { catk::tq_set_spin_limit(polls); }

// Reads and clears the 32-bit timeout word at ws + flag offset after the
// stream's work so far (the copies are ordered on the stream itself).
static int tq_read_clear_flag(const char* fn, const void* workspace, int64_t n, int64_t d,
                              void* stream) {
    hipStream_t st = static_cast<hipStream_t>(stream);
    uint32_t* word = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(const_cast<void*>(workspace)) +
                                                 catk::tq_flag_offset_bytes(n, d));
    uint32_t v = 0;
    hipError_t err = hipMemcpyAsync(&v, word, sizeof(v), hipMemcpyDeviceToHost, st);
    if (err == hipSuccess) err = hipStreamSynchronize(st);
    if (err != hipSuccess) return hip_fail(fn, err);
    if (v == 0) return CAT_OK;
    const uint32_t zero = 0;
    err = hipMemcpyAsync(word, &zero, sizeof(zero), hipMemcpyHostToDevice, st);
    if (err == hipSuccess) err = hipStreamSynchronize(st);
    if (err != hipSuccess) return hip_fail(fn, err);
    return fail(CAT_ERR_TIMEOUT, std::string(fn) +
                                     ": an exchange wait ran out; the results of the calls "
                                     "concerned are invalid");
}

extern "C" int cat_transform_quant_status(const void* workspace, int64_t n, int64_t d, int64_t k,
                                          void* stream) {
    const char* fn = "cat_transform_quant_status";
    (void)k;
    try {
        if (!workspace) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL workspace");
        if (n < 1 || d < 1) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": n, d >= 1");
        if (int rc = require_device(fn)) return rc;
        return tq_read_clear_flag(fn, workspace, n, d, stream);
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

extern "C" int cat_transform_quant(const void* X, int x_dtype, int64_t n, int64_t d, const void* T,
                                   int t_dtype, int64_t k, int bits, uint8_t* codes, float* s_x,
                                   void* workspace, size_t workspace_bytes, void* stream) {
    const char* fn = "cat_transform_quant";
    try {
        if (!X || !T || !codes || !s_x)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (!valid_dtype(x_dtype) || !valid_dtype(t_dtype))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad dtype");
        if (n < 1 || d < 2) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": need n >= 1, d >= 2");
        if (d % 2) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d must be even");
        if (!cat::is_pow2(k) || k > CAT_MAX_BLOCK)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": k must be a power of two <= 512");
        if (d % k) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d % k != 0");
        if (bits != 4 && bits != 6 && bits != 8)
            return fail(CAT_ERR_UNSUPPORTED, std::string(fn) + ": bits must be 4, 6 or 8");
        if (!cat::aligned16(X) || !cat::aligned16(T) || !cat::aligned16(codes) ||
            !cat::aligned16(s_x))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (!workspace || workspace_bytes < cat_transform_quant_workspace_bytes(n, d, k))
            return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace missing or too small");
        if (!cat::aligned16(workspace))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": workspace must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        const hipError_t err = catk::launch_transform_quant(
            X, x_dtype == CAT_BF16, n, d, T, t_dtype == CAT_BF16, k, bits, codes, s_x,
            static_cast<uint32_t*>(workspace), static_cast<hipStream_t>(stream));
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

// ------------------------------------------------ allocation-free variant
// cat_transform_quant with its workspace in this file-scope device array,
// for callers that cannot allocate (code under graph capture, serving
// loops).  Each GPU holds its own copy until the process ends; its address
// on a device is looked up once, with that device current, and kept, and
// host code only ever hands that address on.  The transform+quant paths
// clear what they need cleared with their own kernels (the two-pass maxima)
// or need nothing cleared (the tagged single-pass words), so the contents a
// previous call left are harmless; calls that overlap on one GPU race.
constexpr size_t kScratchBytes = size_t{16} << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_on_current_device(const char* where, void** out) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return hip_fail(where, err);
    if (dev < 0 || dev >= kMaxDevices)
        return fail(CAT_ERR_UNSUPPORTED, std::string(where) + ": device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return hip_fail(where, err);
        if (!p) return fail(CAT_ERR_HIP, std::string(where) + ": no scratch address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return CAT_OK;
}
}  // namespace

extern "C" size_t cat_transform_quant_noalloc_max_bytes(void) { return kScratchBytes; }

extern "C" int cat_transform_quant_noalloc(const void* X, int x_dtype, int64_t n, int64_t d,
                                           const void* T, int t_dtype, int64_t k, int bits,
                                           uint8_t* codes, float* s_x, void* stream) {
    const char* fn = "cat_transform_quant_noalloc";
    try {
        const size_t need = cat_transform_quant_workspace_bytes(n, d, k);
        if (need > kScratchBytes)
            return fail(CAT_ERR_UNSUPPORTED,
                        std::string(fn) + ": needs " + std::to_string(need) +
                            " bytes of scratch, more than the " + std::to_string(kScratchBytes) +
                            " the library holds per device");
        if (int rc = require_device(fn)) return rc;
        void* ws = nullptr;
        if (int rc = scratch_on_current_device(fn, &ws)) return rc;
        return cat_transform_quant(X, x_dtype, n, d, T, t_dtype, k, bits, codes, s_x, ws,
                                   kScratchBytes, stream);
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

extern "C" int cat_transform_quant_noalloc_status(int64_t n, int64_t d, int64_t k, void* stream) {
    const char* fn = "cat_transform_quant_noalloc_status";
    try {
        if (n < 1 || d < 1) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": n, d >= 1");
        if (cat_transform_quant_workspace_bytes(n, d, k) > kScratchBytes)
            return fail(CAT_ERR_UNSUPPORTED, std::string(fn) + ": shape beyond the scratch array");
        if (int rc = require_device(fn)) return rc;
        void* ws = nullptr;
        if (int rc = scratch_on_current_device(fn, &ws)) return rc;
        return tq_read_clear_flag(fn, ws, n, d, stream);
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

extern "C" int cat_transform_quant_asym(const void* X, int x_dtype, int64_t n, int64_t d,
                                        const void* T, int t_dtype, int64_t k, uint8_t* codes,
                                        float* s_x, float* zmin_x, void* workspace,
                                        size_t workspace_bytes, void* stream) {
    const char* fn = "cat_transform_quant_asym";
    try {
        if (!X || !T || !codes || !s_x || !zmin_x)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (!valid_dtype(x_dtype) || !valid_dtype(t_dtype))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad dtype");
        if (n < 1 || d < 2) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": need n >= 1, d >= 2");
        if (d % 2) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d must be even");
        if (!cat::is_pow2(k) || k > CAT_MAX_BLOCK)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": k must be a power of two <= 512");
        if (d % k) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d % k != 0");
        if (!cat::aligned16(X) || !cat::aligned16(T) || !cat::aligned16(codes) ||
            !cat::aligned16(s_x) || !cat::aligned16(zmin_x))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (!workspace || workspace_bytes < cat_transform_quant_asym_workspace_bytes(n, d, k))
            return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace missing or too small");
        if (!cat::aligned16(workspace))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": workspace must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        const hipError_t err = catk::launch_transform_quant_asym(
            X, x_dtype == CAT_BF16, n, d, T, t_dtype == CAT_BF16, k, codes, s_x, zmin_x,
            static_cast<uint32_t*>(workspace), static_cast<hipStream_t>(stream));
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

extern "C" size_t cat_transform_quant_full_workspace_bytes(int64_t n, int64_t d, int64_t k) {
    if (n < 1 || d < 1 || k < 1) return 0;
    return catk::tq_full_workspace_bytes(n, d);
}

extern "C" int cat_transform_quant_full(const void* X, int x_dtype, int64_t n, int64_t d,
                                        const void* T, int t_dtype, int64_t k, uint8_t* codes,
                                        float* s_x, void* workspace, size_t workspace_bytes,
                                        void* stream) {
    const char* fn = "cat_transform_quant_full";
    try {
        if (!X || !T || !codes || !s_x)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (!valid_dtype(x_dtype) || !valid_dtype(t_dtype))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad dtype");
        if (n < 1 || d < 2 || !cat::is_pow2(k) || k > CAT_MAX_BLOCK || d % k)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": bad sizes");
        if (!catk::tq_full_supported(x_dtype == CAT_BF16, t_dtype == CAT_BF16, d, k))
            return fail(CAT_ERR_UNSUPPORTED, std::string(fn) +
                        ": needs bf16 X and T, k 128 or 256, d/k in {2..64 powers of two, 28, 56, 112}");
        if (!cat::aligned16(X) || !cat::aligned16(T) || !cat::aligned16(codes) || !cat::aligned16(s_x))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (!workspace || workspace_bytes < catk::tq_full_workspace_bytes(n, d))
            return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace missing or too small");
        if (!cat::aligned16(workspace))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": workspace must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        const hipError_t err = catk::launch_transform_quant_full(
            X, n, d, T, k, codes, s_x, static_cast<float*>(workspace), static_cast<hipStream_t>(stream));
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

namespace {

// Shared checks and launch of the two integer GEMM entry points.
int linear_call(const char* fn, bool i8, const void* codes_x, const float* s_x,
                const void* codes_w, const float* s_w, int64_t n, int64_t d_in, int64_t d_out,
                float* y_tilde, int32_t* acc_out, void* stream, bool asym = false,
                const float* zmin_x = nullptr, const int32_t* rsum_w = nullptr) {
    try {
        if (!codes_x || !s_x || !codes_w || !s_w || !y_tilde || (asym && (!zmin_x || !rsum_w)))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (n < 1 || d_out < 1 || d_in < 32)
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": need n, d_out >= 1 and d_in >= 32");
        if (d_in % 32) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": d_in must be a multiple of 32");
        if (d_in > CAT_MAX_D_IN)
            return fail(CAT_ERR_UNSUPPORTED, std::string(fn) + ": d_in exceeds CAT_MAX_D_IN");
        if (!cat::aligned16(codes_x) || !cat::aligned16(codes_w) || !cat::aligned16(s_x) ||
            !cat::aligned16(s_w) || !cat::aligned16(y_tilde) || (acc_out && !cat::aligned16(acc_out)) ||
            (asym && (!cat::aligned16(zmin_x) || !cat::aligned16(rsum_w))))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        const hipStream_t st = static_cast<hipStream_t>(stream);
        const hipError_t err =
            asym ? catk::launch_w4a4_linear_asym(static_cast<const uint8_t*>(codes_x), s_x, zmin_x,
                                                 static_cast<const uint8_t*>(codes_w), s_w, rsum_w,
                                                 n, d_in, d_out, y_tilde, acc_out, st)
            : i8 ? catk::launch_int8_linear(static_cast<const int8_t*>(codes_x), s_x,
                                          static_cast<const int8_t*>(codes_w), s_w, n, d_in, d_out,
                                          y_tilde, acc_out, st)
               : catk::launch_w4a4_linear(static_cast<const uint8_t*>(codes_x), s_x,
                                          static_cast<const uint8_t*>(codes_w), s_w, n, d_in, d_out,
                                          y_tilde, acc_out, st);
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}

}  // namespace

extern "C" int cat_w4a4_linear(const uint8_t* codes_x, const float* s_x, const uint8_t* codes_w,
                               const float* s_w, int64_t n, int64_t d_in, int64_t d_out,
                               float* y_tilde, int32_t* acc_out, void* stream) {
    return linear_call("cat_w4a4_linear", false, codes_x, s_x, codes_w, s_w, n, d_in, d_out,
                       y_tilde, acc_out, stream);
}

extern "C" int cat_w4a4_linear_asym(const uint8_t* codes_x, const float* s_x, const float* zmin_x,
                                    const uint8_t* codes_w, const float* s_w, const int32_t* rsum_w,
                                    int64_t n, int64_t d_in, int64_t d_out, float* y_tilde,
                                    int32_t* acc_out, void* stream) {
    return linear_call("cat_w4a4_linear_asym", false, codes_x, s_x, codes_w, s_w, n, d_in, d_out,
                       y_tilde, acc_out, stream, true, zmin_x, rsum_w);
}

extern "C" int cat_int8_linear(const int8_t* codes_x, const float* s_x, const int8_t* codes_w,
                               const float* s_w, int64_t n, int64_t d_in, int64_t d_out,
                               float* y_tilde, int32_t* acc_out, void* stream) {
    return linear_call("cat_int8_linear", true, codes_x, s_x, codes_w, s_w, n, d_in, d_out,
                       y_tilde, acc_out, stream);
}

extern "C" size_t cat_sqnr_workspace_bytes(int64_t count) {
    if (count < 1) return 0;
    return static_cast<size_t>(catk::sqnr_grid(count)) * 2 * sizeof(double);
}

extern "C" int cat_sqnr(const float* y, const float* y_tilde, int64_t count, void* workspace,
                        size_t workspace_bytes, double* out, void* stream) {
    const char* fn = "cat_sqnr";
    try {
        if (!y || !y_tilde || !out) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": NULL pointer");
        if (count < 1) return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": count must be >= 1");
        if (!cat::aligned16(y) || !cat::aligned16(y_tilde) || !cat::aligned16(out))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": pointers must be 16-byte aligned");
        if (!workspace || workspace_bytes < cat_sqnr_workspace_bytes(count))
            return fail(CAT_ERR_WORKSPACE, std::string(fn) + ": workspace missing or too small");
        if (!cat::aligned16(workspace))
            return fail(CAT_ERR_INVALID_ARG, std::string(fn) + ": workspace must be 16-byte aligned");
        if (int rc = require_device(fn)) return rc;
        const hipError_t err = catk::launch_sqnr(y, y_tilde, count, static_cast<double*>(workspace),
                                                 out, static_cast<hipStream_t>(stream));
        if (err != hipSuccess) return hip_fail(fn, err);
        return CAT_OK;
    } catch (const std::exception& e) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": " + e.what());
    } catch (...) {
        return fail(CAT_ERR_INTERNAL, std::string(fn) + ": unknown error");
    }
}
