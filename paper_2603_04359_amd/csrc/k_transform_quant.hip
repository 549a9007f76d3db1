// Block transform fused with symmetric per-token integer quantization.
//
// For each token x (a row of X) and each diagonal block b of the
// block-diagonal transform (Sec. 4, eq. 10):  z_b = T_b x_b.
// The token's scale uses the range of the WHOLE transformed row
// (dynamic per-token range, Lemma 2.2 / Sec. 6):
//   amax = max |z|,  s = amax / qmax,
//   code = clamp(rint(z * (qmax / amax)), -qmax, qmax),
// with qmax = 2^(bits-1) - 1: 7 for INT4 (codes packed two per byte), 31
// and 127 for the 6- and 8-bit comparison widths (one int8 per code).
// Every kernel below takes qmax as the template parameter QM.
//
// The row maximum couples all d/k blocks of a token, while reuse of T_b
// wants many tokens per workgroup.  The work is split by (block, token
// tile), and the kernels differ in how a token's blocks meet:
//   single pass     (bf16, k = 128, d = 2048, 4096, 8192; tq_fused_kernel)
//                   one launch reads X once; workgroups exchange per-token
//                   block maxima through the workspace in two levels;
//   two passes      (every other case) run over the same tiles:
//     pass 1 (amax) computes z and folds max|z| into a per-token word
//                   (LDS atomics, then one atomic max per token on the
//                   float's bit pattern: all values are non-negative, so
//                   unsigned order = float order);
//     pass 2 (quant) recomputes z with the identical instruction sequence,
//                   reads the finished row maximum and writes packed codes.
//   A fill kernel clears the per-token words first (no hipMemset, so the
//   sequence can be captured in a graph).
// Two-pass kernels, by case: tq_group_kernel (bf16, k <= 256, d a multiple
// of 256), tq_ring_kernel (bf16 k = 512, and k = 128 or 256 otherwise),
// tq_mfma_kernel (bf16 k = 32, 64 otherwise) and the vector-ALU kernels
// (fp32 operands or other block sizes).  The asymmetric INT4 variant takes
// the same routes with a row maximum and minimum, except that bf16 k = 32
// and 64 off the group kernel's widths go to the vector ALU.
//
// bf16 kernels run v_mfma_f32_32x32x16_bf16 with A = rows of T_b and B =
// token rows of X, so Z^T tiles come out with one token per lane column;
// the per-token maximum is a register max plus one lane swap.  Where each
// kernel keeps its operands (registers, LDS, DMA rings) is stated at it.
#include <atomic>
#include <type_traits>

#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kTqThreads = 256;
constexpr float kQmax4 = 7.0f;
constexpr int64_t kTqTargetWorkgroups = 512;

__global__ void fill_zero_u32_kernel(uint32_t* p, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

// Quantize one value given inv = qmax/amax (amax > 0); returns the code
// in [-qmax, qmax] as an int.
template <int QM>
__device__ __forceinline__ int quant_code(float z, float inv) {
    constexpr float q = static_cast<float>(QM);
    float u = z * inv;
    u = __builtin_rintf(u);
    u = fminf(fmaxf(u, -q), q);
    return static_cast<int>(u);
}

// Asymmetric INT4 (activations per token, Sec. 6): the row's minimum and
// maximum of z are kept as order-preserving 32-bit keys (larger key =
// larger float; 0 = no value yet), the maximum as a key and the minimum as
// the key's complement, so both fold with an unsigned atomic max.
__device__ __forceinline__ uint32_t fkey(float f) {
    const uint32_t b = __float_as_uint(f);
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float fkey_value(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
// Code q - 8 (q in [0, 15] on the affine grid from the minimum) as a
// signed INT4 value, given inv = fl(15 / r).
__device__ __forceinline__ int asym_code(float z, float zmin, float inv) {
    float u = (z - zmin) * inv;
    u = __builtin_rintf(u);
    u = fminf(fmaxf(u, 0.0f), 15.0f);
    return static_cast<int>(u) - 8;
}
// Scale and inverse from the row's keys (ws_max[t], ws_min[t]).
__device__ __forceinline__ void asym_scale(uint32_t kmax, uint32_t kmin_c, float& zmin, float& s,
                                           float& inv) {
    const float zmax = fkey_value(kmax);
    zmin = fkey_value(~kmin_c);
    const float r = zmax - zmin;
    const bool nz = r > 0.0f;
    s = nz ? __fdiv_rn(r, 15.0f) : 0.0f;
    inv = nz ? __fdiv_rn(15.0f, r) : 0.0f;
}

// ------------------------------------------------------------ generic path
// Vector ALU, for fp32 operands and blocks the MFMA kernels do not take.
// z is summed in fp64 and rounded to fp32 once, so it is fl32 of the exact
// block product up to a rare double rounding: with fp32 sums a block whose
// terms cancel heavily can move a code across a rounding boundary, and at
// k = 256 or 512 with fp32 T the row maximum can drift by more than 1e-6.
template <typename XT, typename TT>
__device__ __forceinline__ float tq_dot(const XT* __restrict__ X, const TT* __restrict__ T,
                                        int64_t t, int64_t d, int64_t k, int64_t c) {
    const int64_t b = c / k;
    const int64_t j = c - b * k;
    const TT* trow = T + (b * k + j) * k;
    const XT* xrow = X + t * d + b * k;
    double acc = 0.0;
    for (int64_t i = 0; i < k; ++i)
        acc = fma(static_cast<double>(load_as_f32(trow, i)), static_cast<double>(load_as_f32(xrow, i)),
                  acc);
    return static_cast<float>(acc);
}

template <typename XT, typename TT>
__global__ __launch_bounds__(kTqThreads) void tq_generic_amax_kernel(
    const XT* __restrict__ X, const TT* __restrict__ T, int64_t n, int64_t d, int64_t k,
    uint32_t* __restrict__ amax_ws) {
    const int64_t pairs = d / 2;
    const int64_t u = static_cast<int64_t>(blockIdx.x) * kTqThreads + threadIdx.x;
    if (u >= n * pairs) return;
    const int64_t t = u / pairs;
    const int64_t c = 2 * (u - t * pairs);
    const float z0 = tq_dot(X, T, t, d, k, c);
    const float z1 = tq_dot(X, T, t, d, k, c + 1);
    const uint32_t m = max(abs_bits(z0), abs_bits(z1));
    if (m) atomicMax(amax_ws + t, m);
}

template <typename XT, typename TT, int QM>
__global__ __launch_bounds__(kTqThreads) void tq_generic_quant_kernel(
    const XT* __restrict__ X, const TT* __restrict__ T, int64_t n, int64_t d, int64_t k,
    const uint32_t* __restrict__ amax_ws, uint8_t* __restrict__ codes, float* __restrict__ s_x) {
    constexpr float qmax = static_cast<float>(QM);
    const int64_t pairs = d / 2;
    const int64_t u = static_cast<int64_t>(blockIdx.x) * kTqThreads + threadIdx.x;
    if (u >= n * pairs) return;
    const int64_t t = u / pairs;
    const int64_t cp = u - t * pairs;
    const float amax = __uint_as_float(amax_ws[t]);
    if (cp == 0) s_x[t] = __fdiv_rn(amax, qmax);
    int q0 = 0, q1 = 0;
    if (amax > 0.0f) {
        const float inv = __fdiv_rn(qmax, amax);
        q0 = quant_code<QM>(tq_dot(X, T, t, d, k, 2 * cp), inv);
        q1 = quant_code<QM>(tq_dot(X, T, t, d, k, 2 * cp + 1), inv);
    }
    if constexpr (QM == 7) {
        codes[t * pairs + cp] = static_cast<uint8_t>((q0 & 0xF) | ((q1 & 0xF) << 4));
    } else {
        // one int8 per code: the pair is two consecutive bytes
        *reinterpret_cast<uint16_t*>(codes + t * d + 2 * cp) =
            static_cast<uint16_t>((q0 & 0xFF) | ((q1 & 0xFF) << 8));
    }
}

template <typename XT, typename TT>
__global__ __launch_bounds__(kTqThreads) void tq_generic_minmax_kernel(
    const XT* __restrict__ X, const TT* __restrict__ T, int64_t n, int64_t d, int64_t k,
    uint32_t* __restrict__ ws) {
    const int64_t pairs = d / 2;
    const int64_t u = static_cast<int64_t>(blockIdx.x) * kTqThreads + threadIdx.x;
    if (u >= n * pairs) return;
    const int64_t t = u / pairs;
    const int64_t c = 2 * (u - t * pairs);
    const uint32_t k0 = fkey(tq_dot(X, T, t, d, k, c));
    const uint32_t k1 = fkey(tq_dot(X, T, t, d, k, c + 1));
    atomicMax(ws + t, max(k0, k1));
    atomicMax(ws + n + t, max(~k0, ~k1));
}

template <typename XT, typename TT>
__global__ __launch_bounds__(kTqThreads) void tq_generic_quant_asym_kernel(
    const XT* __restrict__ X, const TT* __restrict__ T, int64_t n, int64_t d, int64_t k,
    const uint32_t* __restrict__ ws, uint8_t* __restrict__ codes, float* __restrict__ s_x,
    float* __restrict__ zmin_x) {
    const int64_t pairs = d / 2;
    const int64_t u = static_cast<int64_t>(blockIdx.x) * kTqThreads + threadIdx.x;
    if (u >= n * pairs) return;
    const int64_t t = u / pairs;
    const int64_t cp = u - t * pairs;
    float zmin, s, inv;
    asym_scale(ws[t], ws[n + t], zmin, s, inv);
    if (cp == 0) {
        s_x[t] = s;
        zmin_x[t] = zmin;
    }
    const int q0 = asym_code(tq_dot(X, T, t, d, k, 2 * cp), zmin, inv);
    const int q1 = asym_code(tq_dot(X, T, t, d, k, 2 * cp + 1), zmin, inv);
    codes[t * pairs + cp] = static_cast<uint8_t>((q0 & 0xF) | ((q1 & 0xF) << 4));
}

// --------------------------------------------------------------- MFMA path
// Persistent workgroups of 4 waves.  Workgroup w owns output rows
// [jc*JC, jc*JC + JC) of block b (bj = w % NBJ) for the token tiles
// r, r + R, r + 2R, ... (r = w / NBJ; a tile is 128 tokens, 32 per wave).
// Its slice of T_b is staged in LDS once, as 16-byte units with unit u of
// row r stored at position u ^ swz(r), so that 16 lanes reading 16
// consecutive rows at the same unit hit 16 distinct bank groups.  The
// next tile's activations are fetched into registers while the current
// tile is multiplied.  Workgroups sharing a T_b slice are NBJ apart in
// launch order, i.e. on the same XCD whenever NBJ is a multiple of 8.
template <int K>
__device__ __forceinline__ int tq_swz(int r) {
    constexpr int U = K / 8;                   // 16-byte units per row
    constexpr int R = U >= 16 ? 1 : 16 / U;    // rows per 256 bytes
    constexpr int M = (U >= 16 ? 16 : U) - 1;
    return (r / R) & M;
}

template <int K, int JC, bool QUANT, int QM>
__global__ __launch_bounds__(kTqThreads) void tq_mfma_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ T, int64_t n, int64_t d,
    int64_t R, uint32_t* __restrict__ amax_ws, uint8_t* __restrict__ codes,
    float* __restrict__ s_x) {
    static_assert(K % 32 == 0 && JC % 32 == 0 && K % JC == 0, "tile shape");
    constexpr int U = K / 8;
    constexpr int NCHUNK = K / JC;
    constexpr int NM = JC / 32;     // 32-row MFMA tiles per wave
    constexpr int NS = K / 16;      // 16-deep MFMA steps
    constexpr bool PREFETCH = NS <= 16;
    __shared__ u32x4 t_lds[JC * U];

    const int64_t nbj = (d / K) * NCHUNK;
    const int64_t bj = blockIdx.x % nbj;
    const int64_t r0 = blockIdx.x / nbj;
    const int64_t b = bj / NCHUNK;
    const int jc = static_cast<int>(bj % NCHUNK);
    const int64_t ntiles = (n + 127) / 128;

    const u32x4* tg = reinterpret_cast<const u32x4*>(T + (b * K + static_cast<int64_t>(jc) * JC) * K);
    for (int i = threadIdx.x; i < JC * U; i += kTqThreads) {
        const int r = i / U, u = i % U;
        t_lds[r * U + (u ^ tq_swz<K>(r))] = tg[i];
    }
    __syncthreads();

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int col = lane & 31;      // token within the wave's 32
    const int h = lane >> 5;        // which 8-element half of a 16-deep step

    // B operand: 8 consecutive bf16 of the token row per 16-deep step
    auto load_x = [&](int64_t tile, u32x4* xb) {
        const int64_t t = tile * 128 + wave * 32 + col;
        const u32x4* xg = reinterpret_cast<const u32x4*>(X + t * d + b * K);
#pragma unroll
        for (int s = 0; s < NS; ++s) xb[s] = t < n ? xg[2 * s + h] : u32x4{0u, 0u, 0u, 0u};
    };

    u32x4 xb[NS];
    u32x4 xn[PREFETCH ? NS : 1];
    if (r0 < ntiles) load_x(r0, xb);
    for (int64_t tile = r0; tile < ntiles; tile += R) {
        if constexpr (PREFETCH) {
            if (tile + R < ntiles) load_x(tile + R, xn);
        }
        const int64_t t = tile * 128 + wave * 32 + col;
        const bool valid = t < n;

        f32x16 acc[NM];
#pragma unroll
        for (int m = 0; m < NM; ++m) acc[m] = f32x16{};
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                const int r = m * 32 + col;
                const u32x4 a = t_lds[r * U + ((2 * s + h) ^ tq_swz<K>(r))];
                acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), as_bf16x8(xb[s]),
                                                                 acc[m], 0, 0, 0);
            }
        }

        if constexpr (!QUANT) {
            uint32_t m_bits = 0;
#pragma unroll
            for (int m = 0; m < NM; ++m)
#pragma unroll
                for (int q = 0; q < 16; ++q) m_bits = max(m_bits, abs_bits(acc[m][q]));
            m_bits = max(m_bits, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m_bits), 32)));
            if (valid && h == 0 && m_bits) atomicMax(amax_ws + t, m_bits);
        } else if constexpr (QM != 7) {
            // one int8 per code: rows 32m + 8q + 4h + (0..3) of the lane's
            // token are 4 consecutive bytes
            constexpr float qmax = static_cast<float>(QM);
            const float amax = valid ? __uint_as_float(amax_ws[t]) : 0.0f;
            if (valid && h == 0 && b == 0 && jc == 0) s_x[t] = __fdiv_rn(amax, qmax);
            const bool nz = amax > 0.0f;
            const float inv = nz ? __fdiv_rn(qmax, amax) : 0.0f;
            uint32_t* crow = reinterpret_cast<uint32_t*>(codes + t * d + b * K +
                                                         static_cast<int64_t>(jc) * JC);
#pragma unroll
            for (int m = 0; m < NM; ++m)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t p = 0;
                    if (nz) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            p |= static_cast<uint32_t>(quant_code<QM>(acc[m][4 * q + e], inv) & 0xFF)
                                 << (8 * e);
                    }
                    if (valid) crow[(m * 32 + 8 * q + 4 * h) / 4] = p;
                }
        } else {
            const float amax = valid ? __uint_as_float(amax_ws[t]) : 0.0f;
            if (valid && h == 0 && b == 0 && jc == 0) s_x[t] = __fdiv_rn(amax, kQmax4);
            const bool nz = amax > 0.0f;
            const float inv = nz ? __fdiv_rn(kQmax4, amax) : 0.0f;
            uint32_t* crow = reinterpret_cast<uint32_t*>(codes + t * (d / 2) + b * (K / 2) +
                                                         static_cast<int64_t>(jc) * (JC / 2));
#pragma unroll
            for (int m = 0; m < NM; ++m) {
                // v[q]: codes of rows 32m + 8q + 4h + (0..3), packed in 16 bits
                uint32_t v[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t p = 0;
                    if (nz) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            p |= static_cast<uint32_t>(quant_code<7>(acc[m][4 * q + e], inv) & 0xF)
                                 << (4 * e);
                    }
                    v[q] = p;
                }
#pragma unroll
                for (int qp = 0; qp < 4; qp += 2) {
                    // h=0 stores rows 8qp+0..7 of group qp, h=1 those of group qp+1
                    const uint32_t send = h ? v[qp] : v[qp + 1];
                    const uint32_t recv =
                        static_cast<uint32_t>(__shfl_xor(static_cast<int>(send), 32));
                    const uint32_t word = h ? (recv | (v[qp + 1] << 16)) : (v[qp] | (recv << 16));
                    if (valid) crow[(m * 32 + 8 * (qp + h)) / 8] = word;
                }
            }
        }
        if constexpr (PREFETCH) {
#pragma unroll
            for (int s = 0; s < NS; ++s) xb[s] = xn[s];
        } else {
            if (tile + R < ntiles) load_x(tile + R, xb);
        }
    }
}

template <int K, int JC, int QM>
hipError_t launch_tq_mfma(const uint16_t* X, int64_t n, int64_t d, const uint16_t* T,
                          uint8_t* codes, float* s_x, uint32_t* ws, hipStream_t stream) {
    const int64_t tiles = (n + 127) / 128;
    const int64_t nbj = (d / K) * (K / JC);
    // about two resident workgroups per CU, each looping over R token tiles
    int64_t R = (kTqTargetWorkgroups + nbj - 1) / nbj;
    if (R > tiles) R = tiles;
    if (R < 1) R = 1;
    const int64_t grid = nbj * R;
    hipLaunchKernelGGL((tq_mfma_kernel<K, JC, false, 7>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, R, ws, codes, s_x);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((tq_mfma_kernel<K, JC, true, QM>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, R, ws, codes, s_x);
    return hipGetLastError();
}


// ------------------------------------------------------ ring MFMA path
// bf16, k in {128, 256, 512}.  Persistent workgroups of 4 waves, two per
// CU.  Workgroup (bj, r) owns rows [jc*128, jc*128 + 128) of block b and
// the token tiles r, r + R, ...; wave w holds rows jc*128 + 32w .. +31 of
// T_b in registers (the MFMA A operand, loaded once).  Token tiles of TT
// rows stream global -> LDS with global_load_lds_dwordx4 (whole 16-byte
// units, 1 KiB contiguous per wave instruction) into a 2-stage ring: the
// next tile is requested as soon as the previous one has been consumed, so
// it loads during the current tile's MFMAs.  Each wave multiplies its 32
// rows against every token of the tile (B operand read from LDS; 16-byte
// units XOR-swizzled per token row so fragment reads are conflict free).
// Pass 1 folds per-token maxima across the four waves in LDS and issues one
// atomic max per token; pass 2 packs codes straight from the accumulators.
template <int K>
struct TqRing {
    static constexpr int TT = K == 128 ? 128 : (K == 256 ? 64 : 32);   // tokens per tile
    static constexpr int U = K / 8;                // 16-byte units per token row
    static constexpr int NS = K / 16;              // 16-deep MFMA steps
    static constexpr int NSB = TT / 32;            // 32-token subtiles
    static constexpr int STAGE = TT * U;           // units per stage (2048 = 32 KiB)
    static constexpr int LOADS = STAGE / kTqThreads;
    static constexpr int NCHUNK = K / 128;         // 128-row chunks per block
};

template <int K>
__device__ __forceinline__ int tq_xswz(int r) {
    return K == 128 ? ((r ^ (r >> 4)) & 15) : (r & 31);
}

// ASYM: asymmetric INT4 (pass 1 folds the row's max and min keys, pass 2
// writes codes q - 8 and the row minimum to zmin_x).
template <int K, bool QUANT, int QM, bool ASYM = false>
__global__ __launch_bounds__(kTqThreads, 2) void tq_ring_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ T, int64_t n, int64_t d,
    int64_t R, uint32_t* __restrict__ amax_ws, uint8_t* __restrict__ codes,
    float* __restrict__ s_x, float* __restrict__ zmin_x) {
    using C = TqRing<K>;
    __shared__ __attribute__((aligned(16))) u32x4 ring[2][C::STAGE];
    __shared__ uint32_t red[ASYM ? 8 : 4][C::TT];

    // workgroup -> (block, tile row) unit and 128-row chunk; the NCHUNK
    // workgroups of a unit are 8 apart in launch order, so round-robin
    // dispatch puts them on one XCD and the later reads of each X tile hit
    // that XCD's L2
    const int64_t nb = d / K;
    int64_t unit = blockIdx.x;
    int jc = 0;
    if constexpr (C::NCHUNK > 1) {
        const int64_t sq = blockIdx.x >> 3;
        jc = static_cast<int>(sq % C::NCHUNK);
        unit = (sq / C::NCHUNK) * 8 + (blockIdx.x & 7);
    }
    if (unit >= nb * R) return;
    const int64_t b = unit % nb;
    const int64_t r0 = unit / nb;
    const int64_t ntiles = (n + C::TT - 1) / C::TT;
    if (r0 >= ntiles) return;

    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int row0 = jc * 128 + wave * 32;     // first row of T_b this wave owns

    // A operand: row row0 + l32 of T_b, elements 16s + 8h .. +7 per step s
    u32x4 tf[C::NS];
    {
        const u32x4* tg = reinterpret_cast<const u32x4*>(T + (b * K + row0 + l32) * K);
#pragma unroll
        for (int s = 0; s < C::NS; ++s) tf[s] = tg[2 * s + h];
    }

    // slot sl of a stage holds token row sl / U, logical unit (sl % U) ^ swz
    auto issue = [&](int64_t tile, int st) {
        const int64_t t0 = tile * C::TT;
        const uint16_t* base = X + t0 * d + b * K;   // wave-uniform
        const int64_t last = n - 1 - t0;              // last valid row of the tile
#pragma unroll
        for (int q = 0; q < C::LOADS; ++q) {
            const int sl = (q * 4 + wave) * 64 + lane;
            int rr = sl / C::U;
            const int u = (sl % C::U) ^ tq_xswz<K>(rr);
            rr = rr <= last ? rr : static_cast<int>(last);   // rows past the end: never used
            dma16(base, static_cast<uint32_t>((rr * d + u * 8) * 2),
                  lds_addr(&ring[st][(q * 4 + wave) * 64]));
        }
    };

    issue(r0, 0);
    int it = 0;
    for (int64_t tile = r0; tile < ntiles; tile += R, ++it) {
        const int st = it & 1;
        wait_vmcnt<0>();         // this thread's loads of the tile have landed
        lds_barrier();      // ... everyone's; the other stage is free again
        if (tile + R < ntiles) issue(tile + R, st ^ 1);

        f32x16 acc[C::NSB];
#pragma unroll
        for (int sb = 0; sb < C::NSB; ++sb) acc[sb] = f32x16{};
#pragma unroll
        for (int s = 0; s < C::NS; ++s) {
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                const int rr = sb * 32 + l32;
                const u32x4 xf = ring[st][rr * C::U + ((2 * s + h) ^ tq_xswz<K>(rr))];
                acc[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(tf[s]), as_bf16x8(xf),
                                                                  acc[sb], 0, 0, 0);
            }
        }

        if constexpr (!QUANT && ASYM) {
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                uint32_t mx = 0, mn = 0;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const uint32_t kq = fkey(acc[sb][q]);
                    mx = max(mx, kq);
                    mn = max(mn, ~kq);
                }
                mx = max(mx, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mx), 32)));
                mn = max(mn, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mn), 32)));
                if (h == 0) {
                    red[wave][sb * 32 + l32] = mx;
                    red[4 + wave][sb * 32 + l32] = mn;
                }
            }
            lds_barrier();
            for (int idx = threadIdx.x; idx < C::TT; idx += kTqThreads) {
                const uint32_t mx = max(max(red[0][idx], red[1][idx]), max(red[2][idx], red[3][idx]));
                const uint32_t mn = max(max(red[4][idx], red[5][idx]), max(red[6][idx], red[7][idx]));
                const int64_t t = tile * C::TT + idx;
                if (t < n) {
                    atomicMax(amax_ws + t, mx);
                    atomicMax(amax_ws + n + t, mn);
                }
            }
        } else if constexpr (ASYM) {
            // packed like the symmetric INT4 branch below, codes q - 8
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                const int64_t t = tile * C::TT + sb * 32 + l32;
                const bool valid = t < n;
                float zmin = 0.0f, s = 0.0f, inv = 0.0f;
                if (valid) asym_scale(amax_ws[t], amax_ws[n + t], zmin, s, inv);
                if (valid && h == 0 && wave == 0 && b == 0 && jc == 0) {
                    s_x[t] = s;
                    zmin_x[t] = zmin;
                }
                uint32_t v[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t pk = 0;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        pk |= static_cast<uint32_t>(asym_code(acc[sb][4 * q + e], zmin, inv) & 0xF)
                              << (4 * e);
                    v[q] = pk;
                }
                uint32_t* crow =
                    reinterpret_cast<uint32_t*>(codes + t * (d / 2) + (b * K + row0) / 2);
#pragma unroll
                for (int qp = 0; qp < 4; qp += 2) {
                    const uint32_t send = h ? v[qp] : v[qp + 1];
                    const uint32_t recv =
                        static_cast<uint32_t>(__shfl_xor(static_cast<int>(send), 32));
                    const uint32_t word = h ? (recv | (v[qp + 1] << 16)) : (v[qp] | (recv << 16));
                    if (valid) crow[qp + h] = word;
                }
            }
        } else if constexpr (QUANT && QM == 0) {
            // z itself, fp32 (the full-dimension Hadamard path mixes it
            // across blocks afterwards): codes is an [n x d] fp32 buffer
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                const int64_t t = tile * C::TT + sb * 32 + l32;
                if (t >= n) continue;
                float* zrow = reinterpret_cast<float*>(codes) + t * d + b * K + row0;
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    *reinterpret_cast<f32x4*>(zrow + 8 * q + 4 * h) =
                        f32x4{acc[sb][4 * q], acc[sb][4 * q + 1], acc[sb][4 * q + 2], acc[sb][4 * q + 3]};
            }
        } else if constexpr (!QUANT) {
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                uint32_t m = 0;
#pragma unroll
                for (int q = 0; q < 16; ++q) m = max(m, abs_bits(acc[sb][q]));
                m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), 32)));
                if (h == 0) red[wave][sb * 32 + l32] = m;
            }
            lds_barrier();
            for (int idx = threadIdx.x; idx < C::TT; idx += kTqThreads) {
                const uint32_t m = max(max(red[0][idx], red[1][idx]), max(red[2][idx], red[3][idx]));
                const int64_t t = tile * C::TT + idx;
                if (t < n && m) atomicMax(amax_ws + t, m);
            }
        } else if constexpr (QM != 7) {
            // one int8 per code: rows row0 + 8q + 4h + (0..3) of the lane's
            // token are 4 consecutive bytes
            constexpr float qmax = static_cast<float>(QM);
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                const int64_t t = tile * C::TT + sb * 32 + l32;
                const bool valid = t < n;
                const float amax = valid ? __uint_as_float(amax_ws[t]) : 0.0f;
                if (valid && h == 0 && wave == 0 && b == 0 && jc == 0)
                    s_x[t] = __fdiv_rn(amax, qmax);
                const bool nz = amax > 0.0f;
                const float inv = nz ? __fdiv_rn(qmax, amax) : 0.0f;
                uint32_t* crow = reinterpret_cast<uint32_t*>(codes + t * d + b * K + row0);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t pk = 0;
                    if (nz) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            pk |= static_cast<uint32_t>(quant_code<QM>(acc[sb][4 * q + e], inv) & 0xFF)
                                  << (8 * e);
                    }
                    if (valid) crow[2 * q + h] = pk;
                }
            }
        } else {
#pragma unroll
            for (int sb = 0; sb < C::NSB; ++sb) {
                const int64_t t = tile * C::TT + sb * 32 + l32;
                const bool valid = t < n;
                const float amax = valid ? __uint_as_float(amax_ws[t]) : 0.0f;
                if (valid && h == 0 && wave == 0 && b == 0 && jc == 0)
                    s_x[t] = __fdiv_rn(amax, kQmax4);
                const bool nz = amax > 0.0f;
                const float inv = nz ? __fdiv_rn(kQmax4, amax) : 0.0f;
                // v[q]: codes of rows 8q + 4h + (0..3) of the wave's 32, 16 bits
                uint32_t v[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    uint32_t pk = 0;
                    if (nz) {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            pk |= static_cast<uint32_t>(quant_code<7>(acc[sb][4 * q + e], inv) & 0xF)
                                  << (4 * e);
                    }
                    v[q] = pk;
                }
                uint32_t* crow =
                    reinterpret_cast<uint32_t*>(codes + t * (d / 2) + (b * K + row0) / 2);
#pragma unroll
                for (int qp = 0; qp < 4; qp += 2) {
                    // h=0 stores rows 8qp+0..7, h=1 rows 8(qp+1)+0..7
                    const uint32_t send = h ? v[qp] : v[qp + 1];
                    const uint32_t recv =
                        static_cast<uint32_t>(__shfl_xor(static_cast<int>(send), 32));
                    const uint32_t word = h ? (recv | (v[qp + 1] << 16)) : (v[qp] | (recv << 16));
                    if (valid) crow[qp + h] = word;
                }
            }
        }
    }
}

// ------------------------------------------------- single-pass variant
// bf16, k = 128, d = 128 NB with NB = 16, 32 or 64 blocks, one launch, X
// read once.  One workgroup per CU owns block b for the token tiles r,
// r + R, ... (a tile is 64 tokens) and splits its twelve waves by role:
//   waves 0-7  compute: wave w multiplies the 32 rows 32 (w / 2) .. + 31 of
//              T_b (staged in LDS once) with tokens 32 (w % 2) .. + 31 of
//              the tile, read from LDS; two compute waves per SIMD, so one
//              wave's rounding runs beside the other's MFMAs;
//   waves 8-9  copy: stream token tiles into an LDS ring with
//              global_load_lds_dwordx4, kFqAhead tiles ahead;
//   wave 10    gather: reads the per-token maxima other workgroups published;
//   wave 11    publish: writes this workgroup's per-token maxima, and the
//              codes and scales the compute waves leave in LDS (16-byte
//              pieces, 64 contiguous bytes per token).
// Each wave issues one kind of vector-memory traffic only, so every wait is
// exact and no load waits for a store's acknowledgement: the copy waves
// count their own copies, and the compiler tracks the loads of the gather
// wave (the compute waves issue no global memory operation after loading
// T_b, and the stores of the publish wave are never waited for).
//
// The row maximum of a token needs all NB blocks, exchanged in two levels
// through the workspace: every workgroup publishes its block maxima P(b, t)
// of a tile; workgroup b owns the 64 / NB tokens (64 / NB) b, ... of the
// tile, reduces their NB P words each and has the row maxima F(t)
// published; every workgroup then reads F of the tile's 64 tokens (64
// words of reads per workgroup and tile per level instead of 64 NB for all
// P words).  A word is
// (call tag << 32) | maximum bits written with one store, so a reader sees
// either an old word (another tag) or the whole new one and the workspace
// needs no clearing between calls.  Tags have bit 31 set; the two-pass
// paths keep their words in a region of the workspace of their own, so
// nothing they leave behind is read here.  Eager calls take the tag from a host
// counter; a call captured into a graph takes it from a word a one-thread
// kernel advances before every replay (see launch_tq_fused).  P(j, t) lives at
// ((t / 16) * NB + j) * 16 + t % 16 (16 tokens of a block fill one 128-byte
// line), F(t) at NB n' + t (n' = n rounded up to 16).
//
// Steps are separated by one workgroup barrier.  In step s the compute
// waves multiply tile s and leave its per-token maxima in LDS while they
// round tile s - L (L = kFqLag) from the accumulators they kept (seven
// sets rotate); the publish wave writes P of tile s - 1, the codes of tile
// s - L - 1 and, once the gather wave has reduced them, F of tile s - 3;
// the gather wave takes the F words of tile s - L + 1 and the P words of
// tile s - 3 it requested in the last step, reduces P, and requests P of
// tile s - 2 and F of tile s - L + 2.  Every word is thus published a step
// before it is first read and then has a whole step in flight: under a
// full-rate stream a device-scope store takes about a microsecond to
// become visible to a reader on another CU, and workgroups drift apart by
// about as much, so a shorter lag makes reads find stale words and wait a
// further round trip.  Rows of T_b are permuted inside each 32-row MFMA
// group so that lane (token, h) accumulates 16 consecutive output
// channels: its codes are 8 contiguous bytes, no cross-lane exchange.
//
// Progress: the grid never exceeds the device's resident capacity (see
// launch_tq_fused) and every workgroup of a token-tile row visits its tiles
// in the same order, so a workgroup only waits for peers that are running
// or about to run.  Waits are still bounded: after a limit of polls (by
// default kTqSpinLimit; tq_set_spin_limit lowers it for tests that force a
// timeout) the waiting wave records a timeout flag and goes on with a NaN
// maximum, which makes the affected scales NaN.
constexpr uint32_t kTqSpinLimit = 1u << 22;
static std::atomic<uint32_t> g_tq_spin_limit{kTqSpinLimit};
void tq_set_spin_limit(uint32_t polls) {
    g_tq_spin_limit.store(polls == 0 ? kTqSpinLimit : (polls < kTqSpinLimit ? polls : kTqSpinLimit),
                          std::memory_order_relaxed);
}
constexpr int kFqCompute = 8;                   // compute waves
constexpr int kFqCopy = 2;                      // copy waves
constexpr int kFqThreads = (kFqCompute + kFqCopy + 2) * kWave;
constexpr int kFqTT = 64;                       // tokens per tile
constexpr int kFqU = 16;                        // 16-byte units per token row
constexpr int kFqStage = kFqTT * kFqU;          // units per stage (16 KiB)
constexpr int kFqCopyOps = kFqStage / (kFqCopy * kWave);   // copies per lane per tile
constexpr int kFqLag = 6;                       // tile s is rounded in step s + kFqLag
// Copies in flight per CU (kFqAhead tiles of 16 KiB): every load of the CU,
// the exchange reads included, queues behind them, and 16-32 KiB per CU
// already stream X at 5.9-6.1 TB/s.  Three tiles ahead measured the same.
constexpr int kFqAhead = 2;
constexpr int kFqStages = kFqAhead + 1;         // a stage is free once its tile is multiplied
static_assert(kFqCopyOps * kFqAhead < 64, "copies in flight must fit the vmcnt range");
static_assert(kFqStages > kFqAhead, "a stage is refilled only after its tile is multiplied");

struct TqFusedWs {
    uint64_t* pmax;       // P words, then F words (see above)
    uint64_t* pmin;       // asymmetric codes: the same for the complemented minimum keys
    uint32_t* flag;       // timeout flag (0 = fine)
    // The call's tag: the host's when tag_word is NULL, else the word a
    // preceding tq_device_tag_kernel wrote (calls captured into a graph,
    // where every replay must publish under a tag of its own).
    const uint32_t* tag_word;
};

// Advances the device-side tag in the workspace: one per replay of a
// captured call.  Device tags have bits 31 and 30 set, host tags bit 31
// only, so the two never collide; any previous content is a valid start.
__global__ void tq_device_tag_kernel(uint32_t* word) {
    if (threadIdx.x == 0) {
        const uint32_t old = __hip_atomic_load(word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(word, 0xC0000000u | ((old + 1u) & 0x3FFFFFFFu), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
}

// MFMA row i of a 32-row group -> output row within the group
__device__ __forceinline__ int fq_row(int i) {
    return ((i >> 2) & 1) * 16 + (i >> 3) * 4 + (i & 3);
}

// Low bytes of four words -> one word, byte j from word j.
__device__ __forceinline__ uint32_t fq_bytes(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
    return __builtin_amdgcn_perm(b1, b0, 0x0C0C0400u) | __builtin_amdgcn_perm(b3, b2, 0x04000C0Cu);
}

// 16 accumulators (consecutive output channels) -> 16 codes.  u =
// fl(z * inv) is clamped to [-qmax, qmax] and rounded to nearest even by
// adding 1.5 * 2^23 (exact for |u| < 2^22), which leaves the integer in the
// low mantissa bits, two's complement.
template <int QM>
__device__ __forceinline__ void fq_round16(const f32x16& z, float inv, uint32_t (&w)[16]) {
    constexpr float q = static_cast<float>(QM);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        float u = z[r] * inv;
        u = __builtin_amdgcn_fmed3f(u, -q, q);
        w[r] = __float_as_uint(u + 12582912.0f);
    }
}

// INT4: channel 2m in the low nibble of byte m.
__device__ __forceinline__ u32x2 fq_quant16(const f32x16& z, float inv) {
    uint32_t w[16];
    fq_round16<7>(z, inv, w);
    u32x2 out;
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
        const uint32_t* v = w + 8 * hw;
        const uint32_t ev = fq_bytes(v[0], v[2], v[4], v[6]);
        const uint32_t od = fq_bytes(v[1], v[3], v[5], v[7]);
        out[hw] = (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
    }
    return out;
}

// Asymmetric INT4 codes of 16 consecutive channels: q = rint(clamp(fl(fl(z -
// zmin) * inv), 0, 15)) (clamping first gives the same integer, as both
// bounds are integers), stored as q - 8 = q ^ 8, channel 2m in the low
// nibble of byte m.
__device__ __forceinline__ u32x2 fq_quant16_asym(const f32x16& z, float zmin, float inv) {
    uint32_t w[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        float u = (z[r] - zmin) * inv;
        u = __builtin_amdgcn_fmed3f(u, 0.0f, 15.0f);
        w[r] = __float_as_uint(u + 12582912.0f) ^ 8u;
    }
    u32x2 out;
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
        const uint32_t* v = w + 8 * hw;
        const uint32_t ev = fq_bytes(v[0], v[2], v[4], v[6]);
        const uint32_t od = fq_bytes(v[1], v[3], v[5], v[7]);
        out[hw] = (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
    }
    return out;
}

// Asymmetric scale from a row's exchanged keys, as asym_scale, except that
// a range that is NaN (keys of a timed-out exchange are all ones, which
// decode to NaN) keeps s = NaN instead of becoming a zero scale.
__device__ __forceinline__ void fq_asym_scale(uint32_t kmax, uint32_t kmin_c, float& zmin, float& s,
                                              float& inv) {
    const float zmax = fkey_value(kmax);
    zmin = fkey_value(~kmin_c);
    const float r = zmax - zmin;
    const bool nz = !(r <= 0.0f);
    s = nz ? __fdiv_rn(r, 15.0f) : 0.0f;
    inv = nz ? __fdiv_rn(15.0f, r) : 0.0f;
}

// 6- and 8-bit widths: one int8 per channel, channel m in byte m.
template <int QM>
__device__ __forceinline__ u32x4 fq_quant16_i8(const f32x16& z, float inv) {
    uint32_t w[16];
    fq_round16<QM>(z, inv, w);
    return u32x4{fq_bytes(w[0], w[1], w[2], w[3]), fq_bytes(w[4], w[5], w[6], w[7]),
                 fq_bytes(w[8], w[9], w[10], w[11]), fq_bytes(w[12], w[13], w[14], w[15])};
}

// One code's rounding as in fq_round16 (symmetric) or fq_quant16_asym
// (asymmetric, already offset by 8): the integer sits in the low bits.
template <int QM, bool ASYM>
__device__ __forceinline__ uint32_t fq_round1(float z, float inv, float zmin) {
    if constexpr (ASYM) {
        float u = (z - zmin) * inv;
        u = __builtin_amdgcn_fmed3f(u, 0.0f, 15.0f);
        return __float_as_uint(u + 12582912.0f) ^ 8u;
    } else {
        constexpr float q = static_cast<float>(QM);
        float u = z * inv;
        u = __builtin_amdgcn_fmed3f(u, -q, q);
        return __float_as_uint(u + 12582912.0f);
    }
}

// max |z| over 16 values, as float bits.  Read as signed ints, the largest
// value is the largest positive (or, with none, the largest-magnitude
// negative); read as unsigned, it is the largest-magnitude negative (or,
// with none, the largest positive).  The answer is the larger magnitude of
// the two.
__device__ __forceinline__ uint32_t fq_absmax16(const f32x16& z) {
    int32_t mi = static_cast<int32_t>(__float_as_uint(z[0]));
    uint32_t mu = __float_as_uint(z[0]);
#pragma unroll
    for (int r = 1; r < 15; r += 2) {
        const uint32_t a = __float_as_uint(z[r]), c = __float_as_uint(z[r + 1]);
        mi = max(mi, max(static_cast<int32_t>(a), static_cast<int32_t>(c)));
        mu = max(mu, max(a, c));
    }
    mi = max(mi, static_cast<int32_t>(__float_as_uint(z[15])));
    mu = max(mu, __float_as_uint(z[15]));
    return max(static_cast<uint32_t>(mi) & 0x7FFFFFFFu, mu & 0x7FFFFFFFu);
}

// tile t has landed once at most `later` tiles of copies issued after it
// are still in flight
__device__ __forceinline__ void fq_wait_copies(int later) {
    switch (later) {
        case 0: wait_vmcnt<0>(); break;
        case 1: wait_vmcnt<1 * kFqCopyOps>(); break;
        case 2: wait_vmcnt<2 * kFqCopyOps>(); break;
        case 3: wait_vmcnt<3 * kFqCopyOps>(); break;
        case 4: wait_vmcnt<4 * kFqCopyOps>(); break;
        case 5: wait_vmcnt<5 * kFqCopyOps>(); break;
        default: wait_vmcnt<6 * kFqCopyOps>(); break;
    }
}

template <int QM, int NB, bool ASYM>
__global__ __launch_bounds__(kFqThreads, 1) void tq_fused_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ T, int64_t n, int64_t d,
    int64_t R, TqFusedWs ws, uint32_t host_tag, uint32_t spin, uint8_t* __restrict__ codes,
    float* __restrict__ s_x, float* __restrict__ zmin_x) {
    static_assert(!ASYM || QM == 7, "asymmetric codes are INT4");
    const uint32_t tag = ws.tag_word ? __hip_atomic_load(ws.tag_word, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT)
                                     : host_tag;
    constexpr int K = 128;
    constexpr int NS = K / 16;          // 16-deep MFMA steps
    constexpr int L = kFqLag;
    static_assert(L == 6, "seven accumulator sets rotate");
    static_assert(kFqTT == 64 && kFqCompute == 8, "compute waves: 2 token halves x 4 row groups");
    constexpr int CB = QM == 7 ? K / 2 : K;       // code bytes per token and block
    // token stride of the code buffer: 16 bytes of padding put the 16 tokens
    // of one LDS pass on distinct banks (8-byte writes at a 64-byte stride
    // would share 4 banks), and keep every 16-byte piece aligned
    constexpr int CBS = CB + 16;
    __shared__ __attribute__((aligned(16))) u32x4 ring[kFqStages][kFqStage];
    // T_b in MFMA row order: LDS row p holds row (p & ~31) + fq_row(p & 31),
    // 16-byte unit u at position u ^ tq_xswz(p)
    __shared__ __attribute__((aligned(16))) u32x4 tl[K * kFqU];
    __shared__ __attribute__((aligned(16))) uint8_t cbuf[2][kFqTT][CBS];  // codes of a quantized tile
    __shared__ float cscale[2][kFqTT];            // its s_x
    __shared__ float czmin[ASYM ? 2 : 1][ASYM ? kFqTT : 1];
    __shared__ uint32_t red[2][4][kFqTT];         // per-row-group maxima of a step's tile
    __shared__ uint32_t gat[2][kFqTT];            // row maxima of a tile to quantize
    static_assert(NB >= 16 && NB <= kWave && kFqTT % NB == 0, "blocks per token-tile row");
    constexpr int TPO = kFqTT / NB;               // tokens each workgroup reduces per tile
    __shared__ uint32_t fred[2][TPO];             // reduced row maxima of the owned tokens
    __shared__ uint32_t fready;                   // tiles whose fred is complete
    __shared__ uint32_t redn[ASYM ? 2 : 1][4][ASYM ? kFqTT : 1];
    __shared__ uint32_t gatn[ASYM ? 2 : 1][ASYM ? kFqTT : 1];
    __shared__ uint32_t fredn[ASYM ? 2 : 1][ASYM ? TPO : 1];

    const int64_t b = blockIdx.x % NB;
    const int64_t r0 = blockIdx.x / NB;
    const int64_t ntiles = (n + kFqTT - 1) / kFqTT;
    if (r0 >= ntiles) return;           // never taken: the launcher sizes R <= ntiles
    const int64_t nt = (ntiles - r0 + R - 1) / R;
    // step it: tile it multiplied (it < nt), tile it - L quantized into LDS,
    // tile it - L - 1's codes stored
    const int64_t nsteps = nt + L + 1;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    auto tile0 = [&](int64_t it) { return (r0 + it * R) * kFqTT; };   // first token
    if (threadIdx.x == 0) fready = 0;
    // copy waves: tile it of this block into stage it % kFqStages; the first
    // kFqAhead tiles are requested at once, beside the staging of T_b
    const int cw = wave - kFqCompute;
    auto issue = [&](int64_t it) {
        const int64_t t0 = tile0(it);
        const uint16_t* base = X + t0 * d + b * K;
        const int64_t last = n - 1 - t0;
        const int st = static_cast<int>(it % kFqStages);
#pragma unroll
        for (int q = 0; q < kFqCopyOps; ++q) {
            const int first = (cw * kFqCopyOps + q) * kWave;   // first slot of this copy
            const int sl = first + lane;
            int rr = sl / kFqU;
            const int u = (sl % kFqU) ^ tq_xswz<K>(rr);
            rr = rr <= last ? rr : static_cast<int>(last);
            dma16(base, static_cast<uint32_t>((rr * d + u * 8) * 2), lds_addr(&ring[st][first]));
        }
    };
    if (wave >= kFqCompute && wave < kFqCompute + kFqCopy)
        for (int64_t it = 0; it < nt && it < kFqAhead; ++it) issue(it);
    if (threadIdx.x < kFqCompute * kWave) {
        const u32x4* tg = reinterpret_cast<const u32x4*>(T + b * K * K);
#pragma unroll
        for (int i = 0; i < K * kFqU / (kFqCompute * kWave); ++i) {
            const int q = static_cast<int>(threadIdx.x) + i * kFqCompute * kWave;
            const int p = q / kFqU, u = q % kFqU;
            tl[p * kFqU + (u ^ tq_xswz<K>(p))] = tg[((p & ~31) + fq_row(p & 31)) * kFqU + u];
        }
    }
    lds_barrier();

    if (wave >= kFqCompute + kFqCopy) {
        const uint64_t hi = static_cast<uint64_t>(tag) << 32;
        const int64_t n16 = (n + 15) / 16 * 16;
        uint64_t* const fw = ws.pmax + n16 * NB;
        uint64_t* const fwn = ASYM ? ws.pmin + n16 * NB : nullptr;
        auto clampt = [&](int64_t t) { return t < n ? t : n - 1; };
        auto p_word = [&](int64_t t, int64_t j) {
            return ws.pmax + (t >> 4) * (NB * 16) + j * 16 + (t & 15);
        };
        auto pn_word = [&](int64_t t, int64_t j) {
            return ws.pmin + (t >> 4) * (NB * 16) + j * 16 + (t & 15);
        };
        auto store = [&](uint64_t* a, uint32_t m) {
            __hip_atomic_store(a, hi | m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        };
        if (wave == kFqCompute + kFqCopy + 1) {
            // publish: P of tile it-1, the codes (and scales) of tile
            // it-L-1, then F of tile it-3 once the gather wave has reduced it
            for (int64_t it = 0; it < nsteps; ++it) {
                lds_barrier();
                if (it >= 1 && it - 1 < nt) {
                    const int64_t t = tile0(it - 1) + lane;
                    const int sb = static_cast<int>((it - 1) & 1);
                    const uint32_t mm = max(max(red[sb][0][lane], red[sb][1][lane]),
                                            max(red[sb][2][lane], red[sb][3][lane]));
                    if (t < n) store(p_word(t, b), mm);
                    if constexpr (ASYM) {
                        const uint32_t mn = max(max(redn[sb][0][lane], redn[sb][1][lane]),
                                                max(redn[sb][2][lane], redn[sb][3][lane]));
                        if (t < n) store(pn_word(t, b), mn);
                    }
                }
                const int64_t jc = it - L - 1;
                if (jc >= 0 && jc < nt) {
                    const int sb = static_cast<int>(jc & 1);
                    constexpr int PER = CB / 16;          // 16-byte pieces per token
                    constexpr int TPI = kWave / PER;      // tokens per instruction
#pragma unroll
                    for (int q = 0; q < kFqTT / TPI; ++q) {
                        const int tk = q * TPI + lane / PER, pc = lane % PER;
                        const int64_t t = tile0(jc) + tk;
                        const u32x4 v = *reinterpret_cast<const u32x4*>(&cbuf[sb][tk][16 * pc]);
                        if (t < n)
                            *reinterpret_cast<u32x4*>(codes + t * (d * CB / K) + b * CB + 16 * pc) = v;
                    }
                    const int64_t t = tile0(jc) + lane;
                    if (b == 0 && t < n) {
                        s_x[t] = cscale[sb][lane];
                        if constexpr (ASYM) zmin_x[t] = czmin[sb][lane];
                    }
                }
                if (it >= 3 && it - 3 < nt) {
                    // bounded like the gather wave's own waits (an LDS poll
                    // is far shorter than a device read); a wait that runs
                    // out publishes the NaN maximum instead of a stale one
                    const uint32_t want = static_cast<uint32_t>(it - 2);
                    bool ready = true;
                    for (uint32_t polls = 0; __hip_atomic_load(&fready, __ATOMIC_ACQUIRE,
                                                               __HIP_MEMORY_SCOPE_WORKGROUP) < want;) {
                        if (++polls >= 16 * spin) {
                            __hip_atomic_store(ws.flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            ready = false;
                            break;
                        }
                        __builtin_amdgcn_s_sleep(1);
                    }
                    const int64_t t = tile0(it - 3) + TPO * b + lane;
                    const int o = lane < TPO ? lane : 0;
                    const int sb = static_cast<int>((it - 3) & 1);
                    constexpr uint32_t kNaN = ASYM ? 0xFFFFFFFFu : 0x7FC00000u;
                    if (lane < TPO && t < n) {
                        store(fw + t, ready ? fred[sb][o] : kNaN);
                        if constexpr (ASYM) store(fwn + t, ready ? fredn[sb][o] : kNaN);
                    }
                }
            }
            return;
        }
        // gather, step it: take F of tile it-L+1 and P of tile it-3 (both
        // requested in the last step), reduce P into the owned tokens' row
        // maxima, then request P of tile it-2 and F of tile it-L+2 (both
        // published in the last step).  Every read has a whole step in
        // flight; a word that is not there yet is re-read (bounded).
        auto load = [&](const uint64_t* a) {
            return __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        };
        auto await = [&](uint64_t v, const uint64_t* a) {
            for (uint32_t polls = 0; (v >> 32) != tag;) {
                if (++polls >= spin) {
                    __hip_atomic_store(ws.flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    return ASYM ? 0xFFFFFFFFu : 0x7FC00000u;
                }
                __builtin_amdgcn_s_sleep(1);
                v = load(a);
            }
            return static_cast<uint32_t>(v);
        };
        auto f_addr = [&](int64_t j) { return fw + clampt(tile0(j) + lane); };
        auto p_addr = [&](int64_t j) {
            return p_word(clampt(tile0(j) + TPO * b + lane / NB), lane % NB);
        };
        auto fn_addr = [&](int64_t j) { return fwn + clampt(tile0(j) + lane); };
        auto pn_addr = [&](int64_t j) {
            return pn_word(clampt(tile0(j) + TPO * b + lane / NB), lane % NB);
        };
        auto fold = [&](uint32_t m) {
#pragma unroll
            for (int x = 1; x < NB; x <<= 1)
                m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), x)));
            return m;
        };
        uint64_t fv = 0, pv = 0, fvn = 0, pvn = 0;
        for (int64_t it = 0; it < nsteps; ++it) {
            lds_barrier();
            const int64_t jf = it - L + 1, jp = it - 3;
            if (jf >= 0 && jf < nt) {
                gat[jf & 1][lane] = await(fv, f_addr(jf));
                if constexpr (ASYM) gatn[jf & 1][lane] = await(fvn, fn_addr(jf));
            }
            if (jp >= 0 && jp < nt) {
                const uint32_t m = fold(await(pv, p_addr(jp)));
                if (lane % NB == 0) fred[jp & 1][lane / NB] = m;
                if constexpr (ASYM) {
                    const uint32_t mn = fold(await(pvn, pn_addr(jp)));
                    if (lane % NB == 0) fredn[jp & 1][lane / NB] = mn;
                }
                __hip_atomic_store(&fready, static_cast<uint32_t>(jp + 1), __ATOMIC_RELEASE,
                                   __HIP_MEMORY_SCOPE_WORKGROUP);
            }
            if (it >= 2 && it - 2 < nt) {
                pv = load(p_addr(it - 2));
                if constexpr (ASYM) pvn = load(pn_addr(it - 2));
            }
            if (jf + 1 >= 0 && jf + 1 < nt) {
                fv = load(f_addr(jf + 1));
                if constexpr (ASYM) fvn = load(fn_addr(jf + 1));
            }
        }
        return;
    }

    if (wave >= kFqCompute) {
        // ---------------------------------------------------- copy waves
        for (int64_t it = 0; it < nsteps; ++it) {
            if (it < nt) {
                const int64_t hi_t = nt - 1 < it + kFqAhead - 1 ? nt - 1 : it + kFqAhead - 1;
                fq_wait_copies(static_cast<int>(hi_t - it));
            }
            lds_barrier();
            // the stage of tile it + kFqAhead last held tile it + kFqAhead -
            // kFqStages, whose last read (for its multiplication) was in
            // step it + kFqAhead - kFqStages < it
            if (it + kFqAhead < nt) issue(it + kFqAhead);
        }
        return;
    }

    // ------------------------------------------------------ compute waves
    // Wave w multiplies the 32 rows 32 (w / 2) .. + 31 of T_b (read from
    // LDS) with the 32 tokens 32 (w % 2) .. + 31 of a tile; a lane
    // (token, h) accumulates 16 consecutive output channels.  Seven
    // accumulator sets rotate: tile it is multiplied into set it % 7 while
    // tile it - 6 (set (it + 1) % 7) is quantized, its rounding interleaved
    // with the MFMAs.
    const int l32 = lane & 31;
    const int h = lane >> 5;
    const int th = wave & 1;            // token half of the tile
    const int rq = wave >> 1;           // 32-row group of T_b
    const int tok = th * 32 + l32;      // token (within the tile) of this lane
    const int trow = rq * 32 + l32;     // LDS row of this lane's T_b row
    auto tfrag = [&](int s) { return tl[trow * kFqU + ((2 * s + h) ^ tq_xswz<K>(trow))]; };
    using CodeT = std::conditional_t<(QM == 7), u32x2, u32x4>;
    auto keys_out = [&](int64_t it, const f32x16& acc) {
        uint32_t mx, mn = 0;
        if constexpr (ASYM) {
            mx = 0;
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                const uint32_t kq = fkey(acc[q]);
                mx = max(mx, kq);
                mn = max(mn, ~kq);
            }
            mn = max(mn, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mn), 32)));
        } else {
            mx = fq_absmax16(acc);
        }
        mx = max(mx, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mx), 32)));
        const int sb = static_cast<int>(it & 1);
        if (h == 0) {
            red[sb][rq][tok] = mx;
            if constexpr (ASYM) redn[sb][rq][tok] = mn;
        }
    };
    struct Sc {
        float inv, zmin, s;
    };
    auto scale_of = [&](int64_t j) {
        Sc p;
        const int sb = static_cast<int>(j & 1);
        if constexpr (ASYM) {
            fq_asym_scale(gat[sb][tok], gatn[sb][tok], p.zmin, p.s, p.inv);
        } else {
            const float amax = __uint_as_float(gat[sb][tok]);
            p.inv = amax > 0.0f ? __fdiv_rn(static_cast<float>(QM), amax) : 0.0f;
            p.s = __fdiv_rn(amax, static_cast<float>(QM));
            p.zmin = 0.0f;
        }
        return p;
    };
    auto codes_out = [&](int64_t j, const CodeT& c, const Sc& p) {
        const int sb = static_cast<int>(j & 1);
        *reinterpret_cast<CodeT*>(&cbuf[sb][tok][(QM == 7 ? 16 : 32) * rq + (QM == 7 ? 8 : 16) * h]) = c;
        if (rq == 0 && h == 0) {
            cscale[sb][tok] = p.s;
            if constexpr (ASYM) czmin[sb][tok] = p.zmin;
        }
    };
    // rounding of values 2s, 2s + 1 of a set, packed as soon as a word is
    // full; the empty asm keeps each word's packing at this point of the
    // step (the compiler would otherwise sink it next to the LDS store,
    // after every MFMA)
    auto round_piece = [&](int s, const f32x16& z, const Sc& p, uint32_t (&w)[16], CodeT& c) {
        w[2 * s] = fq_round1<QM, ASYM>(z[2 * s], p.inv, p.zmin);
        w[2 * s + 1] = fq_round1<QM, ASYM>(z[2 * s + 1], p.inv, p.zmin);
        if constexpr (QM == 7) {
            if ((s & 3) == 3) {
                const int hw = s >> 2;
                const uint32_t* v = w + 8 * hw;
                const uint32_t ev = fq_bytes(v[0], v[2], v[4], v[6]);
                const uint32_t od = fq_bytes(v[1], v[3], v[5], v[7]);
                uint32_t word = (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
                asm volatile("" : "+v"(word));
                c[hw] = word;
            }
        } else {
            if (s & 1) {
                const int q = s >> 1;
                uint32_t word = fq_bytes(w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]);
                asm volatile("" : "+v"(word));
                c[q] = word;
            }
        }
    };
    auto step = [&](int64_t it, f32x16& cur, const f32x16& old) {
        lds_barrier();
        const bool cd = it < nt, qd = it >= L && it - L < nt;
        const int st = static_cast<int>(it % kFqStages);
        if (cd && qd) {
            // one MFMA and an eighth of the rounding per fenced group, so the
            // vector ALU works while the MFMA runs
            const Sc p = scale_of(it - L);
            uint32_t w[16];
            CodeT c;
            cur = f32x16{};
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const u32x4 xf = ring[st][tok * kFqU + ((2 * s + h) ^ tq_xswz<K>(tok))];
                cur = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(tfrag(s)), as_bf16x8(xf), cur, 0, 0, 0);
                round_piece(s, old, p, w, c);
                __builtin_amdgcn_sched_barrier(0);
            }
            codes_out(it - L, c, p);
            keys_out(it, cur);
        } else if (cd) {
            cur = f32x16{};
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const u32x4 xf = ring[st][tok * kFqU + ((2 * s + h) ^ tq_xswz<K>(tok))];
                cur = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(tfrag(s)), as_bf16x8(xf), cur, 0, 0, 0);
            }
            keys_out(it, cur);
        } else if (qd) {
            const Sc p = scale_of(it - L);
            uint32_t w[16];
            CodeT c;
#pragma unroll
            for (int s = 0; s < NS; ++s) round_piece(s, old, p, w, c);
            codes_out(it - L, c, p);
        }
    };
    f32x16 a0, a1, a2, a3, a4, a5, a6;
    for (int64_t it = 0; it < nsteps; it += 7) {
        step(it, a0, a1);
        if (it + 1 >= nsteps) break;
        step(it + 1, a1, a2);
        if (it + 2 >= nsteps) break;
        step(it + 2, a2, a3);
        if (it + 3 >= nsteps) break;
        step(it + 3, a3, a4);
        if (it + 4 >= nsteps) break;
        step(it + 4, a4, a5);
        if (it + 5 >= nsteps) break;
        step(it + 5, a5, a6);
        if (it + 6 >= nsteps) break;
        step(it + 6, a6, a0);
    }
}

// ------------------------------------------------ group two-pass path
// bf16, k in {32, 64, 128, 256} with d a multiple of 256.  One persistent
// workgroup per CU owns a group of 256 channels (one or more whole blocks)
// for the token tiles r, r + R, ...  Six waves with fixed roles:
//   waves 0-3  compute: wave w holds rows 64 w .. + 63 of the group's T
//              (two 32-row MFMA groups, each in the fq_row order so that a
//              lane ends up with 16 consecutive output channels) in
//              registers and multiplies them with all 64 tokens of the
//              tile, read from LDS; with k >= 64 both row groups share each
//              X fragment, so every fragment read feeds two MFMAs;
//   waves 4-5  copy: stream 32 KiB token tiles (64 tokens x 256 channels)
//              into a 4-stage LDS ring, three tiles ahead, and in pass 2
//              the tile's finished row words beside them.
// The copy waves issue nothing but copies, so their vmcnt waits are exact
// while the compute waves' stores and atomics stay out of the count.
// Pass 1 folds per-token maxima of the four waves with LDS atomics; the
// tile's maxima go to the global per-token words one step later (after the
// next barrier), which needs no barrier of its own.
// (At k = 512 the 64 rows x 512 columns of T a wave would hold do not fit
// its registers; that case runs on the ring kernels.)
constexpr int kTgCompute = 4;
constexpr int kTgCopy = 2;
constexpr int kTgThreads = (kTgCompute + kTgCopy) * kWave;
constexpr int kTgStages = 4;
constexpr int kTgAhead = kTgStages - 1;     // tiles in flight ahead of the one multiplied
constexpr int kTgTT = 64;                   // tokens per tile
constexpr int kTgU = 32;                    // 16-byte units per token row (256 channels)
constexpr int kTgStage = kTgTT * kTgU;      // 16-byte units per stage (32 KiB)
constexpr int kTgCopyOps = kTgStage / (kTgCopy * kWave);   // copies per lane per tile
static_assert(kTgStage % (kTgCopy * kWave) == 0, "copies split evenly");

// tile it has landed once at most `later` tiles issued after it are in flight
template <int OPS>
__device__ __forceinline__ void tg_wait_copies(int later) {
    static_assert((kTgAhead - 1) * OPS < 64, "copies in flight must fit the vmcnt range");
    if (later >= 2) wait_vmcnt<2 * OPS>();
    else if (later == 1) wait_vmcnt<OPS>();
    else wait_vmcnt<0>();
}


// QUANT false: pass 1 (row maxima into ws[t], or for ASYM the max key into
// ws[t] and the complemented min key into ws[n + t]).  QUANT true: pass 2
// (codes and s_x from the finished words; for ASYM also zmin_x).
template <int K, bool QUANT, int QM, bool ASYM>
__global__ __launch_bounds__(kTgThreads, 1) void tq_group_kernel(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ T, int64_t n, int64_t d,
    int64_t R, uint32_t* __restrict__ ws, uint8_t* __restrict__ codes, float* __restrict__ s_x,
    float* __restrict__ zmin_x) {
    static_assert(K == 32 || K == 64 || K == 128 || K == 256, "block size");
    constexpr int NS = K / 16;                          // 16-deep MFMA steps
    constexpr int NSB = kTgTT / 32;                     // 32-token subtiles
    constexpr bool kShare = K >= 64;                    // both row groups in one block
    static_assert(QM == 7 || QM == 31 || QM == 127, "qmax");
    constexpr bool kWordsIn = QUANT;                    // pass 2 reads the row words
    constexpr int OPS = kTgCopyOps + (kWordsIn ? 1 : 0);
    __shared__ __attribute__((aligned(16))) u32x4 ring[kTgStages][kTgStage];
    __shared__ uint32_t words[kWordsIn ? kTgStages : 1][128];
    __shared__ uint32_t red[QUANT ? 1 : 2][ASYM ? 2 : 1][kTgTT];

    const int64_t ngroups = d / 256;
    const int64_t gb = blockIdx.x % ngroups;            // channel group
    const int64_t r0 = blockIdx.x / ngroups;            // first token tile
    const int64_t ntiles = (n + kTgTT - 1) / kTgTT;
    if (r0 >= R || r0 >= ntiles) return;
    const int64_t nt = (ntiles - r0 + R - 1) / R;       // tiles of this workgroup
    const int64_t cb = gb * 256;                        // first channel of the group
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    auto tile0 = [&](int64_t it) { return (r0 + it * R) * kTgTT; };

    if (wave >= kTgCompute) {
        // ---------------------------------------------------- copy waves
        const int cw = wave - kTgCompute;
        auto issue = [&](int64_t it) {
            const int64_t t0 = tile0(it);
            const uint16_t* base = X + t0 * d + cb;
            const int64_t last = n - 1 - t0;            // rows past the end: never used
            const int st = static_cast<int>(it % kTgStages);
#pragma unroll
            for (int q = 0; q < kTgCopyOps; ++q) {
                const int first = (q * kTgCopy + cw) * kWave;
                const int sl = first + lane;
                int rr = sl / kTgU;
                const int u = (sl % kTgU) ^ (rr & 31);
                rr = rr <= last ? rr : static_cast<int>(last);
                dma16(base, static_cast<uint32_t>((rr * d + u * 8) * 2), lds_addr(&ring[st][first]));
            }
            if constexpr (kWordsIn) {
                // symmetric: wave cw brings tokens 32 cw + (lane % 32);
                // asymmetric: wave 0 the max keys, wave 1 the min keys
                int j = ASYM ? lane : cw * 32 + (lane & 31);
                j = j <= last ? j : static_cast<int>(last);
                const uint32_t* src = ws + (ASYM && cw ? n : 0) + t0;
                dma4(src, static_cast<uint32_t>(j * 4), lds_addr(&words[st][cw * 64]));
            }
        };
        for (int64_t it = 0; it < nt && it < kTgAhead; ++it) issue(it);
        for (int64_t it = 0; it < nt; ++it) {
            const int64_t later = nt - 1 - it;
            tg_wait_copies<OPS>(static_cast<int>(later < kTgAhead - 1 ? later : kTgAhead - 1));
            lds_barrier();
            // the stage of tile it + kTgAhead last held tile it - 1, which
            // every compute wave finished before this barrier
            if (it + kTgAhead < nt) issue(it + kTgAhead);
        }
        if constexpr (!QUANT) lds_barrier();
        return;
    }

    // ------------------------------------------------------ compute waves
    const int l32 = lane & 31;
    const int h = lane >> 5;
    int64_t ch[2];               // first output channel of each 32-row group
    int xo[2];                   // first 16-byte unit of its block within the tile row
    u32x4 tf[2][NS];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        ch[g] = cb + wave * 64 + g * 32;
        const int64_t blk = ch[g] / K;
        xo[g] = static_cast<int>((blk * K - cb) / 8);
        const u32x4* tg = reinterpret_cast<const u32x4*>(T + (ch[g] + fq_row(l32)) * K);
#pragma unroll
        for (int s = 0; s < NS; ++s) tf[g][s] = tg[2 * s + h];
    }
    if constexpr (!QUANT) {
        for (int i = threadIdx.x; i < 2 * (ASYM ? 2 : 1) * kTgTT; i += kTgCompute * kWave)
            (&red[0][0][0])[i] = 0u;
    }
    // pass 1: fold a finished tile's LDS maxima into the global words
    auto flush = [&](int64_t it) {
        const int p = static_cast<int>(it & 1);
        const int j = lane;
        const int64_t t = tile0(it) + j;
        const uint32_t m = red[p][0][j];
        red[p][0][j] = 0u;
        if constexpr (ASYM) {
            const uint32_t mn = red[p][1][j];
            red[p][1][j] = 0u;
            if (t < n) {
                atomicMax(ws + t, m);
                atomicMax(ws + n + t, mn);
            }
        } else {
            if (t < n && m) atomicMax(ws + t, m);
        }
    };
    static_assert(kTgTT == kWave, "one token per lane in flush");

    for (int64_t it = 0; it < nt; ++it) {
        lds_barrier();
        if constexpr (!QUANT) {
            if (wave == 0 && it > 0) flush(it - 1);
        }
        const int st = static_cast<int>(it % kTgStages);
        f32x16 acc[2][NSB];
#pragma unroll
        for (int g = 0; g < 2; ++g)
#pragma unroll
            for (int sb = 0; sb < NSB; ++sb) acc[g][sb] = f32x16{};
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
            for (int sb = 0; sb < NSB; ++sb) {
                const int rr = sb * 32 + l32;
                const u32x4 x0 = ring[st][rr * kTgU + ((xo[0] + 2 * s + h) ^ (rr & 31))];
                const u32x4 x1 =
                    kShare ? x0 : ring[st][rr * kTgU + ((xo[1] + 2 * s + h) ^ (rr & 31))];
                acc[0][sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    as_bf16x8(tf[0][s]), as_bf16x8(x0), acc[0][sb], 0, 0, 0);
                acc[1][sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    as_bf16x8(tf[1][s]), as_bf16x8(x1), acc[1][sb], 0, 0, 0);
            }
        }
        // lane (token sb * 32 + l32, h) holds channels ch[g] + 16 h .. + 15
#pragma unroll
        for (int sb = 0; sb < NSB; ++sb) {
            const int j = sb * 32 + l32;
            const int64_t t = tile0(it) + j;
            const bool valid = t < n;
            if constexpr (!QUANT && ASYM) {
                uint32_t mx = 0, mn = 0;
#pragma unroll
                for (int g = 0; g < 2; ++g)
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const uint32_t kq = fkey(acc[g][sb][q]);
                        mx = max(mx, kq);
                        mn = max(mn, ~kq);
                    }
                mx = max(mx, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mx), 32)));
                mn = max(mn, static_cast<uint32_t>(__shfl_xor(static_cast<int>(mn), 32)));
                if (h == 0) {
                    atomicMax(&red[it & 1][0][j], mx);
                    atomicMax(&red[it & 1][1][j], mn);
                }
            } else if constexpr (!QUANT) {
                uint32_t m = max(fq_absmax16(acc[0][sb]), fq_absmax16(acc[1][sb]));
                m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), 32)));
                if (h == 0) atomicMax(&red[it & 1][0][j], m);
            } else if constexpr (ASYM) {
                float zmin = 0.0f, s = 0.0f, inv = 0.0f;
                asym_scale(words[st][j], words[st][64 + j], zmin, s, inv);
                if (valid && h == 0 && wave == 0 && gb == 0) {
                    s_x[t] = s;
                    zmin_x[t] = zmin;
                }
#pragma unroll
                for (int g = 0; g < 2; ++g) {
                    const u32x2 c = fq_quant16_asym(acc[g][sb], zmin, inv);
                    if (valid)
                        *reinterpret_cast<u32x2*>(codes + t * (d / 2) + (ch[g] + 16 * h) / 2) = c;
                }
            } else {
                constexpr float qmax = static_cast<float>(QM);
                const float amax = __uint_as_float(words[st][(j >> 5) * 64 + (j & 31)]);
                if (valid && h == 0 && wave == 0 && gb == 0) s_x[t] = __fdiv_rn(amax, qmax);
                const float inv = amax > 0.0f ? __fdiv_rn(qmax, amax) : 0.0f;
#pragma unroll
                for (int g = 0; g < 2; ++g) {
                    if constexpr (QM == 7) {
                        const u32x2 c = fq_quant16(acc[g][sb], inv);
                        if (valid)
                            *reinterpret_cast<u32x2*>(codes + t * (d / 2) + (ch[g] + 16 * h) / 2) = c;
                    } else {
                        const u32x4 c = fq_quant16_i8<QM>(acc[g][sb], inv);
                        if (valid) *reinterpret_cast<u32x4*>(codes + t * d + ch[g] + 16 * h) = c;
                    }
                }
            }
        }
    }
    if constexpr (!QUANT) {
        lds_barrier();
        if (wave == 0) flush(nt - 1);
    }
}

template <int K, int QM, bool ASYM = false>
hipError_t launch_tq_group(const uint16_t* X, int64_t n, int64_t d, const uint16_t* T,
                           uint8_t* codes, float* s_x, uint32_t* ws, hipStream_t stream,
                           float* zmin_x = nullptr) {
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    const int64_t ntiles = (n + kTgTT - 1) / kTgTT;
    const int64_t ngroups = d / 256;
    // one workgroup per CU: R token-tile rows per channel group, rounded
    // down so that every workgroup is resident at once
    int64_t R = static_cast<int64_t>(cus) / ngroups;
    if (R > ntiles) R = ntiles;
    if (R < 1) R = 1;
    const dim3 grid(static_cast<uint32_t>(ngroups * R)), block(kTgThreads);
    hipLaunchKernelGGL((tq_group_kernel<K, false, 7, ASYM>), grid, block, 0, stream, X, T, n, d, R,
                       ws, codes, s_x, zmin_x);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((tq_group_kernel<K, true, QM, ASYM>), grid, block, 0, stream, X, T, n, d, R,
                       ws, codes, s_x, zmin_x);
    return hipGetLastError();
}

// The group kernels take bf16 k in {32, 64, 128, 256} when d is a multiple
// of 256.
static bool tq_group_fits(int64_t d, int64_t k) {
    return (k == 32 || k == 64 || k == 128 || k == 256) && d % 256 == 0;
}

// Grid of the ring kernels: two resident workgroups per CU, R token-tile
// rows per block rounded down so that every workgroup is resident at once
// (a second round of workgroups would double the time); with NCHUNK > 1
// the units are padded to a multiple of 8 (see the kernel's mapping).
template <int K>
static int64_t tq_ring_grid(int64_t n, int64_t d, int cus, int64_t& R) {
    using C = TqRing<K>;
    const int64_t ntiles = (n + C::TT - 1) / C::TT;
    const int64_t nb = d / K;
    R = (2 * static_cast<int64_t>(cus) / C::NCHUNK) / nb;
    if (R > ntiles) R = ntiles;
    if (R < 1) R = 1;
    const int64_t units = nb * R;
    return C::NCHUNK > 1 ? (units + 7) / 8 * 8 * C::NCHUNK : units;
}

template <int K, int QM, bool ASYM = false>
hipError_t launch_tq_ring(const uint16_t* X, int64_t n, int64_t d, const uint16_t* T,
                          uint8_t* codes, float* s_x, uint32_t* ws, hipStream_t stream,
                          float* zmin_x = nullptr) {
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    int64_t R = 0;
    const int64_t grid = tq_ring_grid<K>(n, d, cus, R);
    hipLaunchKernelGGL((tq_ring_kernel<K, false, 7, ASYM>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, R, ws, codes, s_x, zmin_x);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((tq_ring_kernel<K, true, QM, ASYM>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, R, ws, codes, s_x, zmin_x);
    return hipGetLastError();
}

// Workspace layout (bytes): [0, P) the single-pass exchange words (d/128
// 64-bit tagged block maxima and one tagged row maximum per token, n
// rounded up to 16, P = 8 n' (max(1, d / 128) + 1)); then a 256-byte tail:
// the 32-bit timeout flag at +0 and the device-side tag of captured calls
// at +64; then 8 n bytes for the two-pass paths (one 32-bit running
// maximum per token, or the asymmetric path's two 32-bit keys per token).
// The two regions never overlap, so words one path leaves behind are never
// read by the other: the asymmetric keys can have bit 31 set and could
// otherwise pass for a tagged word.  The asymmetric entry point's workspace
// adds a third region (see tq_asym_min_offset).
static int64_t tq_nbj_max(int64_t d) { return d / 128 > 1 ? d / 128 : 1; }
static size_t tq_flag_offset(int64_t n, int64_t d) {
    return static_cast<size_t>((n + 15) / 16 * 16 * 8 * (tq_nbj_max(d) + 1));
}
static size_t tq_twopass_offset(int64_t n, int64_t d) { return tq_flag_offset(n, d) + 256; }
// asymmetric single pass: the minimum keys' P and F words, laid out like the
// maximum keys', after the two-pass region
static size_t tq_asym_min_offset(int64_t n, int64_t d) {
    return tq_twopass_offset(n, d) + static_cast<size_t>(n) * 8;
}
size_t tq_asym_workspace_bytes(int64_t n, int64_t d, int64_t k) {
    (void)k;
    if (n < 1) return 0;
    return tq_asym_min_offset(n, d) + tq_flag_offset(n, d);
}
size_t tq_flag_offset_bytes(int64_t n, int64_t d) { return tq_flag_offset(n, d); }
size_t tq_workspace_bytes(int64_t n, int64_t d, int64_t k) {
    (void)k;
    if (n < 1) return 0;
    return tq_twopass_offset(n, d) + static_cast<size_t>(n) * 8;
}

static uint32_t next_tq_tag() {
    static std::atomic<uint32_t> tag{0};
    return 0x80000000u | (++tag & 0x3FFFFFFFu);
}

// Resident workgroups of tq_fused_kernel on a device (CUs x blocks per CU
// by its register and LDS use), queried once per device.
template <int QM, int NB, bool ASYM>
static hipError_t tq_fused_resident(int dev, int64_t& resident) {
    constexpr int kMaxDev = 64;
    static std::atomic<int64_t> cache[kMaxDev];   // 0 = not yet known (one table per kernel)
    if (dev >= 0 && dev < kMaxDev) {
        resident = cache[dev].load(std::memory_order_relaxed);
        if (resident > 0) return hipSuccess;
    }
    int cus = 0, per_cu = 0;
    hipError_t err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    err = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, tq_fused_kernel<QM, NB, ASYM>,
                                                       kFqThreads, 0);
    if (err != hipSuccess) return err;
    resident = static_cast<int64_t>(per_cu) * cus;
    if (dev >= 0 && dev < kMaxDev && resident > 0) cache[dev].store(resident, std::memory_order_relaxed);
    return hipSuccess;
}

// Single-pass launch (k = 128, d = 2048, 4096 or 8192) when the grid (d/128
// workgroups per token-tile row, as many rows as fit) can be resident all
// at once; otherwise nothing is launched and the caller takes the two-pass
// path.
// The grid never exceeds the resident capacity, so every workgroup is on
// the device together once other work has drained, and a peer a workgroup
// waits for is always running or about to run.
template <int QM, int NB, bool ASYM>
static hipError_t launch_tq_fused_nb(const uint16_t* X, int64_t n, int64_t d, const uint16_t* T,
                                     uint8_t* codes, float* s_x, uint8_t* ws, hipStream_t stream,
                                     bool& launched, float* zmin_x) {
    launched = false;
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    int64_t resident = 0;
    err = tq_fused_resident<QM, NB, ASYM>(dev, resident);
    if (err != hipSuccess) return err;
    const int64_t ntiles = (n + kFqTT - 1) / kFqTT;
    if (NB > resident) return hipSuccess;
    int64_t R = resident / NB;
    if (R > ntiles) R = ntiles;
    if (R < 1) R = 1;
    TqFusedWs w;
    w.pmax = reinterpret_cast<uint64_t*>(ws);
    w.pmin = ASYM ? reinterpret_cast<uint64_t*>(ws + tq_asym_min_offset(n, d)) : nullptr;
    w.flag = reinterpret_cast<uint32_t*>(ws + tq_flag_offset(n, d));
    w.tag_word = nullptr;
    uint32_t tag = 0;
    hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
    err = hipStreamIsCapturing(stream, &capture);
    if (err != hipSuccess) return err;
    if (capture != hipStreamCaptureStatusNone) {
        // captured: the tag has to change with every replay, so it is made
        // on the device, in the workspace tail next to the timeout flag
        uint32_t* word = reinterpret_cast<uint32_t*>(ws + tq_flag_offset(n, d) + 64);
        hipLaunchKernelGGL(tq_device_tag_kernel, dim3(1), dim3(kWave), 0, stream, word);
        err = hipGetLastError();
        if (err != hipSuccess) return err;
        w.tag_word = word;
    } else {
        tag = next_tq_tag();
    }
    hipLaunchKernelGGL((tq_fused_kernel<QM, NB, ASYM>), dim3(static_cast<uint32_t>(NB * R)),
                       dim3(kFqThreads), 0, stream, X, T, n, d, R, w, tag,
                       g_tq_spin_limit.load(std::memory_order_relaxed), codes, s_x, zmin_x);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    launched = true;
    return hipSuccess;
}

template <int QM, bool ASYM = false>
hipError_t launch_tq_fused(const uint16_t* X, int64_t n, int64_t d, const uint16_t* T,
                           uint8_t* codes, float* s_x, uint8_t* ws, hipStream_t stream,
                           bool& launched, float* zmin_x = nullptr) {
    launched = false;
    switch (d) {
        case 2048:
            return launch_tq_fused_nb<QM, 16, ASYM>(X, n, d, T, codes, s_x, ws, stream, launched, zmin_x);
        case 4096:
            return launch_tq_fused_nb<QM, 32, ASYM>(X, n, d, T, codes, s_x, ws, stream, launched, zmin_x);
        case 8192:
            return launch_tq_fused_nb<QM, 64, ASYM>(X, n, d, T, codes, s_x, ws, stream, launched, zmin_x);
        default: return hipSuccess;
    }
}

template <int QM, typename XT, typename TT>
hipError_t launch_tq_generic(const XT* X, int64_t n, int64_t d, const TT* T, int64_t k,
                             uint8_t* codes, float* s_x, uint32_t* ws, hipStream_t stream) {
    const int64_t units = n * (d / 2);
    const int64_t grid = (units + kTqThreads - 1) / kTqThreads;
    hipLaunchKernelGGL((tq_generic_amax_kernel<XT, TT>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, k, ws);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((tq_generic_quant_kernel<XT, TT, QM>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, k, ws, codes, s_x);
    return hipGetLastError();
}

template <int QM>
static hipError_t launch_tq_qm(const void* X, int x_bf16, int64_t n, int64_t d, const void* T,
                               int t_bf16, int64_t k, uint8_t* codes, float* s_x,
                               uint32_t* amax_ws, hipStream_t stream) {
    if (x_bf16 && t_bf16 && k == 128) {
        bool launched = false;
        const hipError_t e = launch_tq_fused<QM>(static_cast<const uint16_t*>(X), n, d,
                                                 static_cast<const uint16_t*>(T), codes, s_x,
                                                 reinterpret_cast<uint8_t*>(amax_ws), stream,
                                                 launched);
        if (e != hipSuccess || launched) return e;
    }
    amax_ws = reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(amax_ws) +
                                          tq_twopass_offset(n, d));
    hipLaunchKernelGGL(fill_zero_u32_kernel, dim3(static_cast<uint32_t>((n + 255) / 256)),
                       dim3(256), 0, stream, amax_ws, n);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (x_bf16 && t_bf16 && tq_group_fits(d, k)) {
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        const uint16_t* Tb = static_cast<const uint16_t*>(T);
        switch (k) {
            case 32: return launch_tq_group<32, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 64: return launch_tq_group<64, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 128: return launch_tq_group<128, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 256: return launch_tq_group<256, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            default: break;
        }
    }
    if (x_bf16 && t_bf16 && k >= 32) {
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        const uint16_t* Tb = static_cast<const uint16_t*>(T);
        switch (k) {
            case 32: return launch_tq_mfma<32, 32, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 64: return launch_tq_mfma<64, 64, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 128: return launch_tq_ring<128, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 256: return launch_tq_ring<256, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            case 512: return launch_tq_ring<512, QM>(Xb, n, d, Tb, codes, s_x, amax_ws, stream);
            default: break;
        }
    }
    if (x_bf16 && t_bf16)
        return launch_tq_generic<QM>(static_cast<const uint16_t*>(X), n, d,
                                     static_cast<const uint16_t*>(T), k, codes, s_x, amax_ws,
                                     stream);
    if (x_bf16)
        return launch_tq_generic<QM>(static_cast<const uint16_t*>(X), n, d,
                                     static_cast<const float*>(T), k, codes, s_x, amax_ws, stream);
    if (t_bf16)
        return launch_tq_generic<QM>(static_cast<const float*>(X), n, d,
                                     static_cast<const uint16_t*>(T), k, codes, s_x, amax_ws,
                                     stream);
    return launch_tq_generic<QM>(static_cast<const float*>(X), n, d, static_cast<const float*>(T),
                                 k, codes, s_x, amax_ws, stream);
}

hipError_t launch_transform_quant(const void* X, int x_bf16, int64_t n, int64_t d, const void* T,
                                  int t_bf16, int64_t k, int bits, uint8_t* codes, float* s_x,
                                  uint32_t* amax_ws, hipStream_t stream) {
    switch (bits) {
        case 4: return launch_tq_qm<7>(X, x_bf16, n, d, T, t_bf16, k, codes, s_x, amax_ws, stream);
        case 6: return launch_tq_qm<31>(X, x_bf16, n, d, T, t_bf16, k, codes, s_x, amax_ws, stream);
        case 8: return launch_tq_qm<127>(X, x_bf16, n, d, T, t_bf16, k, codes, s_x, amax_ws, stream);
        default: return hipErrorInvalidValue;   // rejected by the caller
    }
}

template <typename XT, typename TT>
static hipError_t launch_tq_generic_asym(const XT* X, int64_t n, int64_t d, const TT* T,
                                         int64_t k, uint8_t* codes, float* s_x, float* zmin_x,
                                         uint32_t* ws, hipStream_t stream) {
    const int64_t units = n * (d / 2);
    const int64_t grid = (units + kTqThreads - 1) / kTqThreads;
    hipLaunchKernelGGL((tq_generic_minmax_kernel<XT, TT>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, k, ws);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL((tq_generic_quant_asym_kernel<XT, TT>), dim3(static_cast<uint32_t>(grid)),
                       dim3(kTqThreads), 0, stream, X, T, n, d, k, ws, codes, s_x, zmin_x);
    return hipGetLastError();
}

// Asymmetric INT4: the single-pass kernel for bf16 with k = 128 and d =
// 2048, 4096 or 8192 (row max and min keys exchanged as two words); else two
// passes (row max and min keys, then codes): the group kernels for bf16
// with k <= 256 and d a multiple of 256, the ring kernels for bf16 with k in
// {128, 256, 512} otherwise, else the vector ALU.
hipError_t launch_transform_quant_asym(const void* X, int x_bf16, int64_t n, int64_t d,
                                       const void* T, int t_bf16, int64_t k, uint8_t* codes,
                                       float* s_x, float* zmin_x, uint32_t* ws,
                                       hipStream_t stream) {
    if (x_bf16 && t_bf16 && k == 128) {
        bool launched = false;
        const hipError_t e = launch_tq_fused<7, true>(
            static_cast<const uint16_t*>(X), n, d, static_cast<const uint16_t*>(T), codes, s_x,
            reinterpret_cast<uint8_t*>(ws), stream, launched, zmin_x);
        if (e != hipSuccess || launched) return e;
    }
    ws = reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(ws) + tq_twopass_offset(n, d));
    hipLaunchKernelGGL(fill_zero_u32_kernel, dim3(static_cast<uint32_t>((2 * n + 255) / 256)),
                       dim3(256), 0, stream, ws, 2 * n);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    if (x_bf16 && t_bf16 && tq_group_fits(d, k)) {
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        const uint16_t* Tb = static_cast<const uint16_t*>(T);
        switch (k) {
            case 32: return launch_tq_group<32, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            case 64: return launch_tq_group<64, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            case 128: return launch_tq_group<128, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            case 256: return launch_tq_group<256, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            default: break;
        }
    }
    if (x_bf16 && t_bf16) {
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        const uint16_t* Tb = static_cast<const uint16_t*>(T);
        switch (k) {
            case 128: return launch_tq_ring<128, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            case 256: return launch_tq_ring<256, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            case 512: return launch_tq_ring<512, 7, true>(Xb, n, d, Tb, codes, s_x, ws, stream, zmin_x);
            default:
                return launch_tq_generic_asym(Xb, n, d, Tb, k, codes, s_x, zmin_x, ws, stream);
        }
    }
    if (x_bf16)
        return launch_tq_generic_asym(static_cast<const uint16_t*>(X), n, d,
                                      static_cast<const float*>(T), k, codes, s_x, zmin_x, ws,
                                      stream);
    if (t_bf16)
        return launch_tq_generic_asym(static_cast<const float*>(X), n, d,
                                      static_cast<const uint16_t*>(T), k, codes, s_x, zmin_x, ws,
                                      stream);
    return launch_tq_generic_asym(static_cast<const float*>(X), n, d,
                                  static_cast<const float*>(T), k, codes, s_x, zmin_x, ws, stream);
}

// ------------------------------------------ full-dimension Hadamard
// T = H_d blockdiag(M_b) with H_d = H_m (x) H_k (m = d / k blocks): the
// block transform T_b = H_k M_b as above, then z' = (H_m (x) I_k) z /
// sqrt(m) across blocks (Sec. 4, T = H M with a full-dimension H), then the
// per-token INT4 quantizer.  H_m is Sylvester for m a power of two, else
// H_28 (x) Sylvester_(m/28), with H_28 from Paley's second construction
// (q = 13): the conference matrix C = [[0, 1^T], [1, Q]], Q_ij = Legendre
// symbol of (i - j) mod 13, and H = C (x) [[1, 1], [1, -1]] + I (x)
// [[1, -1], [-1, -1]].  Row b of H_m splits as b = b1 (m / 28) + b2.
constexpr int legendre13(int a) {
    a = ((a % 13) + 13) % 13;
    return a == 0 ? 0 : (a == 1 || a == 3 || a == 4 || a == 9 || a == 10 || a == 12) ? 1 : -1;
}
constexpr int paley28(int r, int c) {
    const int i = r / 2, j = c / 2, ri = r % 2, cj = c % 2;
    const int conf = (i == 0 && j == 0) ? 0 : (i == 0 || j == 0) ? 1 : legendre13((i - 1) - (j - 1));
    const int a = (ri == 1 && cj == 1) ? -1 : 1;                 // [[1, 1], [1, -1]]
    const int bb = (ri == 0 && cj == 0) ? 1 : -1;                // [[1, -1], [-1, -1]]
    return conf * a + (i == j ? bb : 0);
}

// One workgroup per token, k threads; thread j holds channel j of every
// block (M values), mixes them, and the workgroup reduces the row maximum.
template <int M>
__global__ __launch_bounds__(256) void tq_mix_quant_kernel(const float* __restrict__ z, int64_t n,
                                                          int64_t d, int64_t k,
                                                          uint8_t* __restrict__ codes,
                                                          float* __restrict__ s_x) {
    constexpr bool P28 = (M % 28) == 0;
    constexpr int M2 = P28 ? M / 28 : M;      // Sylvester factor
    __shared__ uint32_t red[4];
    const int64_t t = blockIdx.x;
    const int j = threadIdx.x;
    float v[M];
#pragma unroll
    for (int b = 0; b < M; ++b) v[b] = z[t * d + b * k + j];
    // Sylvester factor over b2 inside each b1 group
#pragma unroll
    for (int hstep = 1; hstep < M2; hstep <<= 1)
#pragma unroll
        for (int b = 0; b < M; ++b)
            if (((b % M2) & hstep) == 0) {
                const float x = v[b], y = v[b + hstep];
                v[b] = x + y;
                v[b + hstep] = x - y;
            }
    if constexpr (P28) {
        // H_28 over b1 for every b2
#pragma unroll
        for (int b2 = 0; b2 < M2; ++b2) {
            float o[28];
#pragma unroll
            for (int a1 = 0; a1 < 28; ++a1) {
                float acc = 0.0f;
#pragma unroll
                for (int b1 = 0; b1 < 28; ++b1) {
                    const int sgn = paley28(a1, b1);
                    acc = sgn > 0 ? acc + v[b1 * M2 + b2] : acc - v[b1 * M2 + b2];
                }
                o[a1] = acc;
            }
#pragma unroll
            for (int a1 = 0; a1 < 28; ++a1) v[a1 * M2 + b2] = o[a1];
        }
    }
    const float norm = 1.0f / __builtin_sqrtf(static_cast<float>(M));
    uint32_t m = 0;
#pragma unroll
    for (int b = 0; b < M; ++b) {
        v[b] *= norm;
        m = max(m, abs_bits(v[b]));
    }
#pragma unroll
    for (int x = 1; x < kWave; x <<= 1)
        m = max(m, static_cast<uint32_t>(__shfl_xor(static_cast<int>(m), x)));
    if ((j & (kWave - 1)) == 0) red[j / kWave] = m;
    __syncthreads();
    const int nw = static_cast<int>(k / kWave);
    m = red[0];
    for (int w = 1; w < nw; ++w) m = max(m, red[w]);
    const float amax = __uint_as_float(m);
    if (j == 0) s_x[t] = __fdiv_rn(amax, kQmax4);
    const float inv = amax > 0.0f ? __fdiv_rn(kQmax4, amax) : 0.0f;
#pragma unroll
    for (int b = 0; b < M; ++b) {
        const int c = amax > 0.0f ? quant_code<7>(v[b], inv) : 0;
        const int other = __shfl_xor(c, 1);
        if ((j & 1) == 0)
            codes[t * (d / 2) + (b * k + j) / 2] = static_cast<uint8_t>((c & 0xF) | ((other & 0xF) << 4));
    }
}

static bool tq_full_supported_m(int64_t m) {
    switch (m) {
        case 2: case 4: case 8: case 16: case 32: case 64: case 28: case 56: case 112: return true;
        default: return false;
    }
}

bool tq_full_supported(int x_bf16, int t_bf16, int64_t d, int64_t k) {
    return x_bf16 && t_bf16 && (k == 128 || k == 256) && d % k == 0 && tq_full_supported_m(d / k);
}

size_t tq_full_workspace_bytes(int64_t n, int64_t d) {
    return static_cast<size_t>(n) * static_cast<size_t>(d) * sizeof(float);
}

hipError_t launch_transform_quant_full(const void* X, int64_t n, int64_t d, const void* T,
                                       int64_t k, uint8_t* codes, float* s_x, float* zbuf,
                                       hipStream_t stream) {
    const uint16_t* Xb = static_cast<const uint16_t*>(X);
    const uint16_t* Tb = static_cast<const uint16_t*>(T);
    uint8_t* zb = reinterpret_cast<uint8_t*>(zbuf);
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    auto zpass = [&](auto kc) -> hipError_t {
        constexpr int K = decltype(kc)::value;
        int64_t R = 0;
        const int64_t grid = tq_ring_grid<K>(n, d, cus, R);
        hipLaunchKernelGGL((tq_ring_kernel<K, true, 0, false>), dim3(static_cast<uint32_t>(grid)),
                           dim3(kTqThreads), 0, stream, Xb, Tb, n, d, R, nullptr, zb, nullptr,
                           nullptr);
        return hipGetLastError();
    };
    // the z pass stays on the ring kernels: writing fp32 z, two workgroups
    // per CU (measured 43 us at 8192 x 4096) beat the group kernel (59 us)
    err = k == 128 ? zpass(std::integral_constant<int, 128>{})
                   : zpass(std::integral_constant<int, 256>{});
    if (err != hipSuccess) return err;
    const dim3 grid(static_cast<uint32_t>(n)), block(static_cast<uint32_t>(k));
    switch (d / k) {
#define CAT_MIX(MM) case MM: hipLaunchKernelGGL(tq_mix_quant_kernel<MM>, grid, block, 0, stream, zbuf, n, d, k, codes, s_x); break;
        CAT_MIX(2) CAT_MIX(4) CAT_MIX(8) CAT_MIX(16) CAT_MIX(32) CAT_MIX(64) CAT_MIX(28) CAT_MIX(56) CAT_MIX(112)
#undef CAT_MIX
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace catk
