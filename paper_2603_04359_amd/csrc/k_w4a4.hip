// W4A4 integer GEMM with fused dequantization (Sec. 3, eq. 5):
//   acc[t, o] = sum_j qx[t, j] qw[o, j]                   (int32, exact)
//   y[t, o]   = fl32(fl32(acc) * s_x[t]) * s_w[o]
//
// gfx950 int8 MFMA (v_mfma_i32_32x32x32_i8) on INT4 codes.  Tiles of packed
// codes (half the bytes of int8) are staged in LDS; each lane reads 16
// packed bytes and widens them in registers to int8 values 16*code with
// two bit operations per dword (low nibbles and high nibbles go to
// separate dwords).  Both operands are widened identically, so each MFMA
// sums the same index pairs (a permutation of the reduction index) and
// the int32 result is 256 * acc; an arithmetic shift by 8 recovers acc
// exactly for d_in <= 131072.
//
// Workgroup: 256 threads (4 waves, 2 x 2), output tile 128 x 128, each
// wave 64 x 64 = 2 x 2 MFMA tiles.  K step 128 codes (64 packed bytes per
// row); the next step's tiles are fetched into registers while the current
// step runs out of the other LDS buffer.  16-byte LDS units are
// XOR-swizzled per row so fragment reads of 16 consecutive rows are
// bank-conflict free.
#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kGemmThreads = 256;
constexpr int kBM = 128;          // tokens per tile
constexpr int kBN = 128;          // outputs per tile
constexpr int kBKB = 64;          // packed bytes per row per K step (128 codes)
constexpr int kUnits = kBKB / 16; // 16-byte units per row per step

__device__ __forceinline__ int gemm_swz(int r) { return (r >> 2) & 3; }

__device__ __forceinline__ i32x4 widen_lo_pair(u32x4 v, int half) {
    // 8 packed bytes (dwords 2*half, 2*half+1) -> 16 int8 values * 16
    const uint32_t w0 = v[2 * half], w1 = v[2 * half + 1];
    return i32x4{static_cast<int>(unpack_lo16(w0)), static_cast<int>(unpack_hi16(w0)),
                 static_cast<int>(unpack_lo16(w1)), static_cast<int>(unpack_hi16(w1))};
}

__global__ __launch_bounds__(kGemmThreads) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ u32x4 lds_a[2][kBM * kUnits];
    __shared__ u32x4 lds_b[2][kBN * kUnits];

    const int64_t tiles_n = (d_out + kBN - 1) / kBN;
    const int64_t tm = blockIdx.x / tiles_n;
    const int64_t tn = blockIdx.x % tiles_n;
    const int64_t m0 = tm * kBM, n0 = tn * kBN;
    const int64_t row_bytes = d_in / 2;
    const int nk = static_cast<int>((row_bytes + kBKB - 1) / kBKB);

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // global -> register staging: each thread moves 2 units of A and 2 of B
    u32x4 ra[2], rb[2];
    auto gload = [&](int kt) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = tid + s * kGemmThreads;
            const int r = i / kUnits, u = i % kUnits;
            const int64_t ga = m0 + r, gb = n0 + r;
            const int64_t off = static_cast<int64_t>(kt) * kBKB + u * 16;
            const bool kin = off < row_bytes;   // ragged last K step: zero codes
            ra[s] = (ga < n && kin) ? *reinterpret_cast<const u32x4*>(qx + ga * row_bytes + off)
                                    : u32x4{0u, 0u, 0u, 0u};
            rb[s] = (gb < d_out && kin)
                        ? *reinterpret_cast<const u32x4*>(qw + gb * row_bytes + off)
                        : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int s = 0; s < 2; ++s) {
            const int i = tid + s * kGemmThreads;
            const int r = i / kUnits, u = i % kUnits;
            lds_a[buf][r * kUnits + (u ^ gemm_swz(r))] = ra[s];
            lds_b[buf][r * kUnits + (u ^ gemm_swz(r))] = rb[s];
        }
    };

    i32x16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = i32x16{};

    gload(0);
    lstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int c2 = 0; c2 < 2; ++c2) {
            // lane half h reads unit 2h + c2 of its row: 32 codes = 2 MFMA steps
            const int u = 2 * h + c2;
            u32x4 a16[2], b16[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int r = wm * 64 + i * 32 + l32;
                a16[i] = lds_a[buf][r * kUnits + (u ^ gemm_swz(r))];
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int r = wn * 64 + j * 32 + l32;
                b16[j] = lds_b[buf][r * kUnits + (u ^ gemm_swz(r))];
            }
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                i32x4 av[2], bv[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) av[i] = widen_lo_pair(a16[i], half);
#pragma unroll
                for (int j = 0; j < 2; ++j) bv[j] = widen_lo_pair(b16[j], half);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(av[i], bv[j], acc[i][j],
                                                                         0, 0, 0);
            }
        }
        if (kt + 1 < nk) {
            lstore(buf ^ 1);
        }
        __syncthreads();
    }

    // epilogue: lane holds column n0 + wn*64 + 32j + l32 and rows
    // m0 + wm*64 + 32i + 8(r/4) + 4h + r%4
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t o = n0 + wn * 64 + j * 32 + l32;
        if (o >= d_out) continue;
        const float sw = s_w[o];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t t = m0 + wm * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
                if (t >= n) continue;
                const int v = acc[i][j][r] >> 8;
                const float yv = (static_cast<float>(v) * s_x[t]) * sw;
                y[t * d_out + o] = yv;
                if (acc_out) acc_out[t * d_out + o] = v;
            }
        }
    }
}

hipError_t launch_w4a4_linear(const uint8_t* codes_x, const float* s_x, const uint8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out, float* y,
                              int32_t* acc_out, hipStream_t stream) {
    const int64_t grid = ((n + kBM - 1) / kBM) * ((d_out + kBN - 1) / kBN);
    hipLaunchKernelGGL(w4a4_gemm_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kGemmThreads), 0,
                       stream, codes_x, s_x, codes_w, s_w, n, d_in, d_out, y, acc_out);
    return hipGetLastError();
}

}  // namespace catk
