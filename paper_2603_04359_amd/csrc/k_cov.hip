// Calibration second moment: acc += X^T X (Sec. 4, Sigma_x = E[x x^T];
// Sec. 6 "Calibration").  The caller divides by the token count.
//
// bf16 path (gfx950 v_mfma_f32_32x32x16_bf16): one workgroup owns one
// TILE x TILE output tile of the upper triangle (mode FULL) or of the upper
// triangle of a diagonal k x k block (mode BLOCK_DIAG) and loops over all
// tokens.  The contraction runs over tokens, i.e. down the columns of the
// row-major X, so each 32-token slab is transposed on its way into LDS:
// every lane loads one channel pair from 8 consecutive tokens (4-byte loads,
// a whole 256-byte row segment per wave instruction), splits the pairs with
// v_perm into two 16-byte runs of 8 tokens and stores them as one LDS unit
// per channel.  Fragments are then 16-byte LDS reads (units XOR-swizzled
// per channel row).  Partial sums stay in registers for at most 4096
// tokens and are then added into acc by the tile's owner (no atomics, so
// results are reproducible); off-diagonal tiles also add their transpose.
//
// fp32 inputs and blocks smaller than 64 use a vector-ALU kernel with the
// same tiling and flush policy.
#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kCovThreads = 256;
constexpr int kCovFlush = 4096;   // tokens per register partial sum
constexpr int kCovTK = 32;        // tokens per LDS slab

// Decode a linear index over the upper triangle of a T x T tile grid.
__device__ __forceinline__ void tri_decode(int64_t idx, int64_t T, int64_t& I, int64_t& J) {
    int64_t i = 0;
    while (idx >= T - i) {
        idx -= T - i;
        ++i;
    }
    I = i;
    J = i + idx;
}

struct CovTile {
    int64_t colbase;  // first channel of the block in X (0 in FULL mode)
    int64_t dim;      // channels of the matrix this tile belongs to
    int64_t I0, J0;   // tile origin (row, col) inside that matrix
    int64_t base;     // offset of that matrix inside acc
};

__device__ __forceinline__ CovTile cov_tile(int64_t work, int tile, int64_t d, int mode,
                                            int64_t k) {
    CovTile c;
    if (mode == CAT_COV_FULL) {
        const int64_t T = (d + tile - 1) / tile;
        int64_t I, J;
        tri_decode(work, T, I, J);
        c.colbase = 0;
        c.dim = d;
        c.I0 = I * tile;
        c.J0 = J * tile;
        c.base = 0;
    } else {
        const int64_t T = (k + tile - 1) / tile;
        const int64_t per = T * (T + 1) / 2;
        const int64_t b = work / per;
        int64_t I, J;
        tri_decode(work % per, T, I, J);
        c.colbase = b * k;
        c.dim = k;
        c.I0 = I * tile;
        c.J0 = J * tile;
        c.base = b * k * k;
    }
    return c;
}

__device__ __forceinline__ int cov_swz(int c) { return (c >> 2) & 3; }

// ------------------------------------------------------------ MFMA (bf16)
template <int TILE>
__global__ __launch_bounds__(kCovThreads) void cov_mfma_kernel(const uint16_t* __restrict__ X,
                                                               int64_t n, int64_t d, int mode,
                                                               int64_t k, float* __restrict__ acc) {
    constexpr int WT = TILE / 2;   // wave tile edge (2 x 2 waves)
    constexpr int NT = WT / 32;    // 32 x 32 MFMA tiles per wave edge
    constexpr int UN = kCovTK / 8; // 16-byte units per channel row
    constexpr int TASKS = 2 * (TILE / 2) * UN;  // (channel pair, token group) x 2 operands
    __shared__ u32x4 lds[2][2][TILE * UN];

    const CovTile ct = cov_tile(blockIdx.x, TILE, d, mode, k);
    const bool diag = ct.I0 == ct.J0;
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    constexpr int PER = (TASKS + kCovThreads - 1) / kCovThreads;
    u32x4 stage[PER][2];

    auto gload = [&](int64_t t0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int task = tid + p * kCovThreads;
            const int op = task / (TASKS / 2);
            const int local = task % (TASKS / 2);
            const int cp = local % (TILE / 2);
            const int g = local / (TILE / 2);
            uint32_t w[8];
            const int64_t lc = (op ? ct.J0 : ct.I0) + 2 * cp;   // channel inside the matrix
            const bool active = task < TASKS && !(op == 1 && diag) && lc < ct.dim;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int64_t t = t0 + 8 * g + i;
                w[i] = (active && t < n)
                           ? *reinterpret_cast<const uint32_t*>(X + t * d + ct.colbase + lc)
                           : 0u;
            }
            // (ch, ch+1) pairs of 8 tokens -> 8 tokens of ch, 8 tokens of ch+1
            stage[p][0] = u32x4{__builtin_amdgcn_perm(w[1], w[0], 0x05040100u),
                                __builtin_amdgcn_perm(w[3], w[2], 0x05040100u),
                                __builtin_amdgcn_perm(w[5], w[4], 0x05040100u),
                                __builtin_amdgcn_perm(w[7], w[6], 0x05040100u)};
            stage[p][1] = u32x4{__builtin_amdgcn_perm(w[1], w[0], 0x07060302u),
                                __builtin_amdgcn_perm(w[3], w[2], 0x07060302u),
                                __builtin_amdgcn_perm(w[5], w[4], 0x07060302u),
                                __builtin_amdgcn_perm(w[7], w[6], 0x07060302u)};
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int task = tid + p * kCovThreads;
            if (task >= TASKS) continue;
            const int op = task / (TASKS / 2);
            if (op == 1 && diag) continue;
            const int local = task % (TASKS / 2);
            const int cp = local % (TILE / 2);
            const int g = local / (TILE / 2);
            const int c0 = 2 * cp, c1 = 2 * cp + 1;
            lds[buf][op][c0 * UN + (g ^ cov_swz(c0))] = stage[p][0];
            lds[buf][op][c1 * UN + (g ^ cov_swz(c1))] = stage[p][1];
        }
    };

    for (int64_t f0 = 0; f0 < n; f0 += kCovFlush) {
        const int64_t f1 = f0 + kCovFlush < n ? f0 + kCovFlush : n;
        f32x16 part[NT][NT];
#pragma unroll
        for (int a = 0; a < NT; ++a)
#pragma unroll
            for (int b = 0; b < NT; ++b) part[a][b] = f32x16{};

        gload(f0);
        lstore(0);
        __syncthreads();
        int buf = 0;
        for (int64_t t0 = f0; t0 < f1; t0 += kCovTK) {
            const bool more = t0 + kCovTK < f1;
            if (more) gload(t0 + kCovTK);
#pragma unroll
            for (int s = 0; s < kCovTK / 16; ++s) {
                const int u = 2 * s + h;
                u32x4 fa[NT], fb[NT];
#pragma unroll
                for (int a = 0; a < NT; ++a) {
                    const int r = wm * WT + 32 * a + l32;
                    fa[a] = lds[buf][0][r * UN + (u ^ cov_swz(r))];
                }
#pragma unroll
                for (int b = 0; b < NT; ++b) {
                    const int r = wn * WT + 32 * b + l32;
                    fb[b] = lds[buf][diag ? 0 : 1][r * UN + (u ^ cov_swz(r))];
                }
#pragma unroll
                for (int a = 0; a < NT; ++a)
#pragma unroll
                    for (int b = 0; b < NT; ++b)
                        part[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            as_bf16x8(fa[a]), as_bf16x8(fb[b]), part[a][b], 0, 0, 0);
            }
            if (more) lstore(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }

        // owner flush: acc[i][j] += part (and the transpose off the diagonal)
#pragma unroll
        for (int a = 0; a < NT; ++a)
#pragma unroll
            for (int b = 0; b < NT; ++b) {
                const int64_t gj = ct.J0 + wn * WT + 32 * b + l32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t gi = ct.I0 + wm * WT + 32 * a + 8 * (r >> 2) + 4 * h + (r & 3);
                    if (gi >= ct.dim || gj >= ct.dim) continue;
                    const float v = part[a][b][r];
                    float* p = acc + ct.base + gi * ct.dim + gj;
                    *p = *p + v;
                    if (!diag) {
                        float* q = acc + ct.base + gj * ct.dim + gi;
                        *q = *q + v;
                    }
                }
            }
    }
}

// ------------------------------------------------------- vector-ALU path
// 64 x 64 tile, 16 x 16 threads each owning 4 x 4 outputs; 16-token slabs
// staged in LDS as fp32.
template <typename XT>
__global__ __launch_bounds__(kCovThreads) void cov_valu_kernel(const XT* __restrict__ X, int64_t n,
                                                               int64_t d, int mode, int64_t k,
                                                               float* __restrict__ acc) {
    constexpr int TILE = 64, TKV = 16;
    __shared__ float xa[TKV][TILE];
    __shared__ float xb[TKV][TILE];
    const CovTile ct = cov_tile(blockIdx.x, TILE, d, mode, k);
    const bool diag = ct.I0 == ct.J0;
    const int ti = threadIdx.x / 16, tj = threadIdx.x % 16;
    for (int64_t f0 = 0; f0 < n; f0 += kCovFlush) {
        const int64_t f1 = f0 + kCovFlush < n ? f0 + kCovFlush : n;
        float part[4][4] = {};
        for (int64_t t0 = f0; t0 < f1; t0 += TKV) {
            for (int e = threadIdx.x; e < TKV * TILE; e += kCovThreads) {
                const int tt = e / TILE, c = e % TILE;
                const int64_t t = t0 + tt;
                const int64_t ci = ct.I0 + c, cj = ct.J0 + c;
                xa[tt][c] = (t < f1 && ci < ct.dim) ? load_as_f32(X, t * d + ct.colbase + ci) : 0.f;
                xb[tt][c] = (t < f1 && cj < ct.dim) ? load_as_f32(X, t * d + ct.colbase + cj) : 0.f;
            }
            __syncthreads();
            for (int tt = 0; tt < TKV; ++tt) {
                float a[4], b[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    a[q] = xa[tt][4 * ti + q];
                    b[q] = xb[tt][4 * tj + q];
                }
#pragma unroll
                for (int p = 0; p < 4; ++p)
#pragma unroll
                    for (int q = 0; q < 4; ++q) part[p][q] = fmaf(a[p], b[q], part[p][q]);
            }
            __syncthreads();
        }
#pragma unroll
        for (int p = 0; p < 4; ++p)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t gi = ct.I0 + 4 * ti + p, gj = ct.J0 + 4 * tj + q;
                if (gi >= ct.dim || gj >= ct.dim) continue;
                float* ptr = acc + ct.base + gi * ct.dim + gj;
                *ptr = *ptr + part[p][q];
                if (!diag) {
                    float* m = acc + ct.base + gj * ct.dim + gi;
                    *m = *m + part[p][q];
                }
            }
    }
}

static int64_t cov_grid(int tile, int64_t d, int mode, int64_t k) {
    if (mode == CAT_COV_FULL) {
        const int64_t T = (d + tile - 1) / tile;
        return T * (T + 1) / 2;
    }
    const int64_t T = (k + tile - 1) / tile;
    return (d / k) * (T * (T + 1) / 2);
}

hipError_t launch_cov_accumulate(const void* X, int x_bf16, int64_t n, int64_t d, int mode,
                                 int64_t k, float* acc, hipStream_t stream) {
    const int64_t dim = mode == CAT_COV_FULL ? d : k;
    if (x_bf16 && dim >= 64 && (dim % 2) == 0 && (d % 2) == 0) {
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        if (dim >= 128) {
            const int64_t g = cov_grid(128, d, mode, k);
            hipLaunchKernelGGL(cov_mfma_kernel<128>, dim3(static_cast<uint32_t>(g)),
                               dim3(kCovThreads), 0, stream, Xb, n, d, mode, k, acc);
        } else {
            const int64_t g = cov_grid(64, d, mode, k);
            hipLaunchKernelGGL(cov_mfma_kernel<64>, dim3(static_cast<uint32_t>(g)),
                               dim3(kCovThreads), 0, stream, Xb, n, d, mode, k, acc);
        }
        return hipGetLastError();
    }
    const int64_t g = cov_grid(64, d, mode, k);
    if (x_bf16)
        hipLaunchKernelGGL(cov_valu_kernel<uint16_t>, dim3(static_cast<uint32_t>(g)),
                           dim3(kCovThreads), 0, stream, static_cast<const uint16_t*>(X), n, d,
                           mode, k, acc);
    else
        hipLaunchKernelGGL(cov_valu_kernel<float>, dim3(static_cast<uint32_t>(g)),
                           dim3(kCovThreads), 0, stream, static_cast<const float*>(X), n, d, mode,
                           k, acc);
    return hipGetLastError();
}

}  // namespace catk
