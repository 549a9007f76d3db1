// Launchers of the gfx950 kernels (host side).  Arguments are validated by
// the C-ABI layer before any of these is called; each launcher enqueues
// on `stream` and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

#include "../../include/cat.h"

namespace catk {

// ---- SQNR (two passes)
// Pass-1 grid cap: two 256-thread workgroups per CU of a 256-CU part.  A
// sweep of the 8192 x 14336 pair read 6.8 TB/s at 384-512 workgroups and
// 5.5-6.0 TB/s at 1024-2048 (more concurrent streams, worse DRAM locality).
constexpr int kSqnrMaxBlocks = 512;
int sqnr_grid(int64_t count);
hipError_t launch_sqnr(const float* y, const float* yt, int64_t count, double* partials,
                       double* out, hipStream_t stream);

// ---- transform + quantize
// amax_ws: tq_workspace_bytes(n, d, k) bytes of scratch.  bits 4: codes
// [n x d/2] packed INT4; bits 6, 8: codes [n x d] int8.
size_t tq_workspace_bytes(int64_t n, int64_t d, int64_t k);
// byte offset of the 32-bit timeout flag inside that workspace
size_t tq_flag_offset_bytes(int64_t n, int64_t d);
// the asymmetric entry point's workspace: tq_workspace_bytes plus the
// single pass's minimum-key words
size_t tq_asym_workspace_bytes(int64_t n, int64_t d, int64_t k);
// polls after which a single-pass exchange wait gives up (0: the default);
// applies to launches that follow
void tq_set_spin_limit(uint32_t polls);
hipError_t launch_transform_quant(const void* X, int x_bf16, int64_t n, int64_t d,
                                  const void* T, int t_bf16, int64_t k, int bits,
                                  uint8_t* codes, float* s_x, uint32_t* amax_ws,
                                  hipStream_t stream);

// Asymmetric INT4 activations: codes q - 8 packed as INT4, s_x and the
// row minimum zmin_x per token; amax_ws as above (2 n words used).
hipError_t launch_transform_quant_asym(const void* X, int x_bf16, int64_t n, int64_t d,
                                       const void* T, int t_bf16, int64_t k, uint8_t* codes,
                                       float* s_x, float* zmin_x, uint32_t* amax_ws,
                                       hipStream_t stream);

// Full-dimension Hadamard: block transform to fp32 z in zbuf
// (tq_full_workspace_bytes), then the cross-block Hadamard and the
// per-token INT4 quantizer.  Only where tq_full_supported().
bool tq_full_supported(int x_bf16, int t_bf16, int64_t d, int64_t k);
size_t tq_full_workspace_bytes(int64_t n, int64_t d);
hipError_t launch_transform_quant_full(const void* X, int64_t n, int64_t d, const void* T,
                                       int64_t k, uint8_t* codes, float* s_x, float* zbuf,
                                       hipStream_t stream);

// ---- integer GEMM: packed INT4 codes (w4a4) or one int8 per code (int8)
hipError_t launch_w4a4_linear(const uint8_t* codes_x, const float* s_x, const uint8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out,
                              float* y, int32_t* acc_out, hipStream_t stream);
// Asymmetric INT4 activations (codes q - 8, scale s_x, minimum zmin_x) by
// symmetric INT4 weights with row code sums rsum_w.
hipError_t launch_w4a4_linear_asym(const uint8_t* codes_x, const float* s_x, const float* zmin_x,
                                   const uint8_t* codes_w, const float* s_w,
                                   const int32_t* rsum_w, int64_t n, int64_t d_in, int64_t d_out,
                                   float* y, int32_t* acc_out, hipStream_t stream);
hipError_t launch_int8_linear(const int8_t* codes_x, const float* s_x, const int8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out,
                              float* y, int32_t* acc_out, hipStream_t stream);

// ---- second moment accumulation
// Workspace of launch_cov_accumulate on the current device (0 when the
// configuration runs on kernels that need none).
hipError_t cov_workspace_bytes(int x_bf16, int64_t d, int mode, int64_t k, size_t& bytes);
hipError_t launch_cov_accumulate(const void* X, int x_bf16, int64_t n, int64_t d, int mode,
                                 int64_t k, float* acc, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

}  // namespace catk
