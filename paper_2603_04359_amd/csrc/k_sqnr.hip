// SQNR reduction (Sec. 2, eq. 1): S = sum y^2, E = sum (y - y~)^2 in fp64,
// dB = 10 log10(S / E).  Two passes with a fixed reduction order, so the
// result is bit-reproducible:
//   pass 1  a grid of G workgroups streams y and y~ with 16-byte loads,
//           accumulates fp64 per lane, reduces across the wave (shuffles)
//           and the workgroup (LDS) and writes partials[g] = {S_g, E_g};
//   pass 2  one workgroup sums the G partials in index order.
// HBM-bound: 8 bytes read per element.
#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kSqnrThreads = 256;

__device__ __forceinline__ double wave_sum(double v) {
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

__global__ __launch_bounds__(kSqnrThreads) void sqnr_partial_kernel(
    const float* __restrict__ y, const float* __restrict__ yt, int64_t count,
    double* __restrict__ partials) {
    double s = 0.0, e = 0.0;
    const int64_t n4 = count >> 2;
    const f32x4* y4 = reinterpret_cast<const f32x4*>(y);
    const f32x4* t4 = reinterpret_cast<const f32x4*>(yt);
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kSqnrThreads;
    int64_t i = static_cast<int64_t>(blockIdx.x) * kSqnrThreads + threadIdx.x;
    // two independent 16-byte loads per array in flight per iteration
    for (; i + stride < n4; i += 2 * stride) {
        const f32x4 a0 = __builtin_nontemporal_load(y4 + i);
        const f32x4 b0 = __builtin_nontemporal_load(t4 + i);
        const f32x4 a1 = __builtin_nontemporal_load(y4 + i + stride);
        const f32x4 b1 = __builtin_nontemporal_load(t4 + i + stride);
        const float av[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
        const float bv[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const double a = av[q];
            const double d = a - static_cast<double>(bv[q]);
            s += a * a;
            e += d * d;
        }
    }
    for (; i < n4; i += stride) {
        const f32x4 a0 = __builtin_nontemporal_load(y4 + i);
        const f32x4 b0 = __builtin_nontemporal_load(t4 + i);
        const float av[4] = {a0[0], a0[1], a0[2], a0[3]};
        const float bv[4] = {b0[0], b0[1], b0[2], b0[3]};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const double a = av[q];
            const double d = a - static_cast<double>(bv[q]);
            s += a * a;
            e += d * d;
        }
    }
    // scalar tail (count % 4 elements) on workgroup 0
    if (blockIdx.x == 0) {
        const int64_t t = (n4 << 2) + threadIdx.x;
        if (t < count) {
            const double a = y[t];
            const double d = a - static_cast<double>(yt[t]);
            s += a * a;
            e += d * d;
        }
    }
    s = wave_sum(s);
    e = wave_sum(e);
    __shared__ double red[2][kSqnrThreads / kWave];
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        red[0][wave] = s;
        red[1][wave] = e;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double ss = 0.0, ee = 0.0;
        for (int w = 0; w < kSqnrThreads / kWave; ++w) {
            ss += red[0][w];
            ee += red[1][w];
        }
        partials[2 * blockIdx.x] = ss;
        partials[2 * blockIdx.x + 1] = ee;
    }
}

__global__ __launch_bounds__(kSqnrThreads) void sqnr_final_kernel(
    const double* __restrict__ partials, int nparts, double* __restrict__ out) {
    double s = 0.0, e = 0.0;
    for (int g = threadIdx.x; g < nparts; g += kSqnrThreads) {
        s += partials[2 * g];
        e += partials[2 * g + 1];
    }
    __shared__ double rs[kSqnrThreads], re[kSqnrThreads];
    rs[threadIdx.x] = s;
    re[threadIdx.x] = e;
    __syncthreads();
    for (int w = kSqnrThreads / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) {
            rs[threadIdx.x] += rs[threadIdx.x + w];
            re[threadIdx.x] += re[threadIdx.x + w];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double S = rs[0], E = re[0];
        out[0] = S;
        out[1] = E;
        out[2] = 10.0 * log10(S / E);
    }
}

int sqnr_grid(int64_t count) {
    const int64_t n4 = (count + 3) / 4;
    int64_t g = (n4 + kSqnrThreads - 1) / kSqnrThreads;
    if (g > kSqnrMaxBlocks) g = kSqnrMaxBlocks;
    if (g < 1) g = 1;
    return static_cast<int>(g);
}

hipError_t launch_sqnr(const float* y, const float* yt, int64_t count, double* partials,
                       double* out, hipStream_t stream) {
    const int g = sqnr_grid(count);
    hipLaunchKernelGGL(sqnr_partial_kernel, dim3(g), dim3(kSqnrThreads), 0, stream, y, yt,
                       count, partials);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(sqnr_final_kernel, dim3(1), dim3(kSqnrThreads), 0, stream, partials, g,
                       out);
    return hipGetLastError();
}

}  // namespace catk
