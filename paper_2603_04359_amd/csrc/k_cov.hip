// Calibration second moment: acc += X^T X (Sec. 4, Sigma_x = E[x x^T];
// Sec. 6 "Calibration").  The caller divides by the token count.
//
// Matrices of at least 256 channels (bf16, channel count a multiple of 32)
// run cov_sk_kernel: 256 x 256 upper-triangle tiles, token slabs streamed
// HBM -> LDS in X's own layout and transposed by ds_read_tr16_b64 on the
// way into v_mfma_f32_32x32x16_bf16, work split evenly over the CUs
// (stream-K over (tile, slab) units), partial sums added with fp32
// atomics.  The design notes are at that kernel.
//
// Smaller bf16 matrices (64 or 128 channels, or widths that are not a
// multiple of 32) run cov_mfma_kernel: one workgroup per 128 x 128 (or
// 64 x 64) upper-triangle tile looping over all tokens; each 32-token slab
// is transposed on its way into LDS (4-byte loads of channel pairs split
// with v_perm into 16-byte runs of 8 tokens per channel).  Partial sums
// stay in registers for at most 4096 tokens and are then added into acc by
// the tile's owner together with the transpose.
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

// ------------------------------------------- 256 x 256 tiles, stream-K
// For matrices of at least 256 channels (bf16, channel count a multiple
// of 8).  Each workgroup (4 waves, one per SIMD) owns a 256 x 256 tile of
// the upper triangle; every wave keeps 128 x 128 fp32 partial sums (4 x 4
// v_mfma_f32_32x32x16_bf16 accumulators).  Token slabs of 32 rows go from
// HBM straight into a 3-stage LDS ring with global_load_lds_dwordx4, in
// X's own row-major order (no transposition on the way in): 512 bytes of
// each token row per operand, 16-byte units XOR-swizzled by row.  The
// MFMA operands need 8 consecutive tokens of one channel; ds_read_tr16_b64
// performs that transposition on the LDS read: within 16 lanes, lane
// 4e + q addresses token row e, channels 4q..4q+3, and lane i receives
// channel i of the 4 rows.
//
// The work is the list of (tile, 32-token slab) units over all tiles; each
// workgroup takes one contiguous share of it (stream-K), so every CU gets
// the same number of MFMAs whatever the tile count.  A tile processed by a
// single workgroup from its first to its last slab is added into acc with
// plain read-modify-write stores; a tile split between workgroups is added
// with fp32 atomics (so the last bit of such tiles may differ between
// runs).  Off-diagonal tiles also add their transpose (16-byte runs: each
// lane holds 4 consecutive rows of one column); diagonal tiles are
// computed whole and written as is.
constexpr int kSkT = 256;                        // tile edge
constexpr int kSkSlab = 32;                      // tokens per ring stage
constexpr int kSkStages = 3;
constexpr int kSkRowUnits = kSkT / 8;            // 16-byte units per token row (32)
constexpr int kSkOpUnits = kSkSlab * kSkRowUnits;  // units per operand and stage (1024)
constexpr int kSkLoads = kSkOpUnits / kCovThreads; // direct loads per thread and operand (4)
constexpr int kSkFlushSlabs = 256;               // at most 8192 tokens per register partial

struct SkGeom {
    int64_t dim;     // channels of one matrix (d in FULL mode, k in BLOCK_DIAG mode)
    int64_t T;       // tiles along one edge of a matrix
    int64_t tri;     // upper-triangle tiles per matrix
    int64_t S;       // slabs per tile (= token slabs)
    int64_t U;       // total units = matrices * tri * S
};

typedef short sk_v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) sk_v4i16 sk_lds_v4i16;

// Eight consecutive tokens of one channel from two transposing reads
// (4 tokens each) at byte offsets off and off + 4 rows.
__device__ __forceinline__ bf16x8 sk_frag(const char __attribute__((address_space(3))) * base,
                                          uint32_t off) {
    const sk_v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((sk_lds_v4i16*)(base + off));
    const sk_v4i16 hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((sk_lds_v4i16*)(base + off + 4 * kSkT * 2));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8, v);
}

__global__ __launch_bounds__(kCovThreads, 1) void cov_sk_kernel(const uint16_t* __restrict__ X,
                                                                int64_t n, int64_t d, int mode,
                                                                int64_t k, SkGeom g,
                                                                float* __restrict__ acc) {
    __shared__ __attribute__((aligned(16))) u32x4 ring[kSkStages][2][kSkOpUnits];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave >> 1, wn = wave & 1;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // contiguous share of the unit list; consecutive shares on one XCD
    const int64_t G = gridDim.x;
    int64_t w = blockIdx.x;
    if (G % 8 == 0) w = (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8;
    const int64_t u_begin = g.U * w / G, u_end = g.U * (w + 1) / G;

    // direct-load geometry: load q of this thread fills unit (q*4+wave)*64+lane
    // of an operand stage, i.e. token row 8q + rr, swizzled position l32.
    const int rr = 2 * wave + h;
    const int unit = l32 ^ ((rr & 3) << 2);      // global 16-byte unit of the row
    const uint32_t row_bytes = static_cast<uint32_t>(d) * 2u;

    // fragment-read geometry (bytes inside one operand stage)
    const int i16 = lane & 15, e = i16 >> 2, qq = i16 & 3, gg = (lane >> 4) & 1;
    uint32_t offA[4], offB[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int row = 8 * h + e;                 // token row inside the 16-token step
        const int ua = (wm * 16 + 4 * a + 2 * gg + (qq >> 1)) ^ ((row & 3) << 2);
        const int ub = (wn * 16 + 4 * a + 2 * gg + (qq >> 1)) ^ ((row & 3) << 2);
        offA[a] = row * (kSkT * 2) + 16 * ua + 8 * (qq & 1);
        offB[a] = row * (kSkT * 2) + 16 * ub + 8 * (qq & 1);
    }

    for (int64_t u = u_begin; u < u_end;) {
        const int64_t tile = u / g.S;
        const int64_t s0 = u % g.S;
        int64_t s1 = (g.S < s0 + (u_end - u)) ? g.S : s0 + (u_end - u);
        const int64_t cend = (s0 / kSkFlushSlabs + 1) * kSkFlushSlabs;   // register partial limit
        s1 = s1 < cend ? s1 : cend;
        u += s1 - s0;

        const int64_t mat = tile / g.tri;
        int64_t I, J;
        tri_decode(tile % g.tri, g.T, I, J);
        const int64_t colbase = mode == CAT_COV_FULL ? 0 : mat * k;
        const int64_t I0 = I * kSkT, J0 = J * kSkT;
        const bool diag = I == J;
        float* accm = acc + (mode == CAT_COV_FULL ? 0 : mat * k * k);

        // per-thread source byte offsets inside a slab (columns clamped into
        // the matrix when the last tile is ragged: those rows/columns of the
        // result are discarded)
        int64_t ca = I0 + 8 * unit, cb = J0 + 8 * unit;
        if (ca >= g.dim) ca = I0;
        if (cb >= g.dim) cb = J0;
        const uint32_t oa = static_cast<uint32_t>(rr) * row_bytes + static_cast<uint32_t>(colbase + ca) * 2u;
        const uint32_t ob = static_cast<uint32_t>(rr) * row_bytes + static_cast<uint32_t>(colbase + cb) * 2u;

        auto issue = [&](int64_t s, int st) {
            const int64_t t0 = s * kSkSlab;
            const char* base = reinterpret_cast<const char*>(X + t0 * d);
            if (t0 + kSkSlab <= n) {
#pragma unroll
                for (int q = 0; q < kSkLoads; ++q)
                    __builtin_amdgcn_global_load_lds(
                        (const void*)(base + (oa + q * 8u * row_bytes)),
                        (lds_void_t*)&ring[st][0][(q * 4 + wave) * 64], 16, 0, 0);
                if (!diag) {
#pragma unroll
                    for (int q = 0; q < kSkLoads; ++q)
                        __builtin_amdgcn_global_load_lds(
                            (const void*)(base + (ob + q * 8u * row_bytes)),
                            (lds_void_t*)&ring[st][1][(q * 4 + wave) * 64], 16, 0, 0);
                }
            } else {
                // ragged last slab: rows past n load row n-1 (zeroed once landed)
#pragma unroll
                for (int q = 0; q < kSkLoads; ++q) {
                    const int64_t t = t0 + 8 * q + rr;
                    const uint32_t back = t < n ? 0u : static_cast<uint32_t>(t - (n - 1)) * row_bytes;
                    __builtin_amdgcn_global_load_lds(
                        (const void*)(base + (oa + q * 8u * row_bytes - back)),
                        (lds_void_t*)&ring[st][0][(q * 4 + wave) * 64], 16, 0, 0);
                    if (!diag)
                        __builtin_amdgcn_global_load_lds(
                            (const void*)(base + (ob + q * 8u * row_bytes - back)),
                            (lds_void_t*)&ring[st][1][(q * 4 + wave) * 64], 16, 0, 0);
                }
            }
        };

        f32x16 part[4][4];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) part[a][b] = f32x16{};

        issue(s0, 0);
        if (s0 + 1 < s1) issue(s0 + 1, 1);
        int st = 0;
        for (int64_t s = s0; s < s1; ++s) {
            if (s + 1 < s1) {
                if (diag) wait_vmcnt<kSkLoads>();
                else wait_vmcnt<2 * kSkLoads>();
            } else {
                wait_vmcnt<0>();
            }
            const int64_t t0 = s * kSkSlab;
            if (t0 + kSkSlab > n) {
#pragma unroll
                for (int q = 0; q < kSkLoads; ++q) {
                    if (t0 + 8 * q + rr >= n) {
                        ring[st][0][(q * 4 + wave) * 64 + lane] = u32x4{0u, 0u, 0u, 0u};
                        if (!diag) ring[st][1][(q * 4 + wave) * 64 + lane] = u32x4{0u, 0u, 0u, 0u};
                    }
                }
            }
            lds_barrier();   // slab s landed for every thread; slab s-1 consumed
            if (s + 2 < s1) issue(s + 2, st == 0 ? 2 : st - 1);

            const char __attribute__((address_space(3)))* baseA =
                (const char __attribute__((address_space(3)))*)&ring[st][0][0];
            const char __attribute__((address_space(3)))* baseB =
                (const char __attribute__((address_space(3)))*)&ring[st][diag ? 0 : 1][0];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
                bf16x8 fa[4], fb[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) fa[a] = sk_frag(baseA, offA[a] + kk * 16 * kSkT * 2);
#pragma unroll
                for (int b = 0; b < 4; ++b) fb[b] = sk_frag(baseB, offB[b] + kk * 16 * kSkT * 2);
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int b = 0; b < 4; ++b)
                        part[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[a], fb[b],
                                                                             part[a][b], 0, 0, 0);
            }
            st = st == 2 ? 0 : st + 1;
        }

        // Add the partial sums into acc with fp32 atomics (no return value):
        // each wave instruction covers two 128-byte row segments.  The
        // transpose for the mirror tile goes through LDS (a 32 x 33 float
        // pad per wave) so its atomics are row segments too.  32-bit element
        // offsets from the matrix base; the empty asm keeps them from being
        // precomputed outside the loop.
        lds_barrier();   // the ring is free: every wave has finished reading it
        uint32_t dimu = static_cast<uint32_t>(g.dim);
        uint32_t rowb = static_cast<uint32_t>(I0 + wm * 128 + 4 * h);
        uint32_t colb = static_cast<uint32_t>(J0 + wn * 128 + l32);
        asm volatile("" : "+v"(rowb), "+v"(colb), "+s"(dimu));
        const uint32_t row_u = static_cast<uint32_t>(I0 + wm * 128);
        const uint32_t col_u = static_cast<uint32_t>(J0 + wn * 128);
        float* pad = reinterpret_cast<float*>(&ring[0][0][0]) + wave * (32 * 33);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                if (row_u + 32 * a >= dimu || col_u + 32 * b >= dimu) continue;
                const uint32_t up = (rowb + 32 * a) * dimu + colb + 32 * b;
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    unsafeAtomicAdd(accm + up + (8 * (r >> 2) + (r & 3)) * dimu, part[a][b][r]);
                if (!diag) {
                    // element (R, C) of the 32 x 32 block -> pad[C][R]; read back
                    // as (R, C) of the transposed block
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        pad[l32 * 33 + 8 * (r >> 2) + 4 * h + (r & 3)] = part[a][b][r];
                    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
                    const uint32_t mi = (colb - l32 + 32 * b + 4 * h) * dimu +
                                        (rowb - 4 * h + 32 * a + l32);
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int R = 8 * (r >> 2) + 4 * h + (r & 3);
                        unsafeAtomicAdd(accm + mi + (8 * (r >> 2) + (r & 3)) * dimu,
                                        pad[R * 33 + l32]);
                    }
                    __builtin_amdgcn_s_waitcnt(0xC07F);
                }
            }
        lds_barrier();   // every wave is done with the ring before the next tile refills it
    }
}

static bool cov_sk_geometry(int64_t n, int64_t d, int mode, int64_t k, SkGeom& g) {
    g.dim = mode == CAT_COV_FULL ? d : k;
    const int64_t nmat = mode == CAT_COV_FULL ? 1 : d / k;
    g.T = (g.dim + kSkT - 1) / kSkT;
    g.tri = g.T * (g.T + 1) / 2;
    g.S = (n + kSkSlab - 1) / kSkSlab;
    g.U = nmat * g.tri * g.S;
    return g.U > 0;
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
    if (x_bf16 && dim >= kSkT && (d % 8) == 0 && (dim % 32) == 0) {
        SkGeom g;
        if (!cov_sk_geometry(n, d, mode, k, g)) return hipSuccess;
        int dev = 0, cus = 0;
        hipError_t err = hipGetDevice(&dev);
        if (err != hipSuccess) return err;
        err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (err != hipSuccess) return err;
        const int64_t grid = g.U < cus ? g.U : cus;
        hipLaunchKernelGGL(cov_sk_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kCovThreads), 0,
                           stream, static_cast<const uint16_t*>(X), n, d, mode, k, g, acc);
        return hipGetLastError();
    }
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
