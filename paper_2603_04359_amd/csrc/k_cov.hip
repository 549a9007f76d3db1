// Calibration second moment: acc += X^T X (Sec. 4, Sigma_x = E[x x^T];
// Sec. 6 "Calibration").  The caller divides by the token count.
//
// Matrices of at least 256 channels (bf16, channel count a multiple of 32)
// run cov_sk_kernel: 256 x 256 upper-triangle tiles, token slabs streamed
// HBM -> LDS in X's own layout and transposed by ds_read_tr16_b64 on the
// way into v_mfma_f32_32x32x16_bf16, work split evenly over the CUs
// (stream-K over (tile, slab) units), pieces of split tiles combined in a
// fixed order.  Diagonal blocks of 32, 64 or 128 channels also run there
// when the width is a multiple of 256: each 256-channel group is one
// diagonal tile, of which only the diagonal blocks are stored (the MFMAs
// of the rest are spent to keep the CUs streaming; the path is bound by
// the X stream, not by the matrix cores).  The design notes are at that
// kernel.
//
// Other small bf16 matrices (64 to 255 channels, or widths that are not a
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
// staged in LDS as fp32.  The partial sums are fp64 and reach acc rounded
// once per flush: with fp32 running sums over thousands of tokens, a column
// of heavy-tailed values (say Student-t with two degrees of freedom) left
// its sum of squares about 1e-5 off.
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
        double part[4][4] = {};
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
                    for (int q = 0; q < 4; ++q)
                        part[p][q] = fma(static_cast<double>(a[p]), static_cast<double>(b[q]),
                                         part[p][q]);
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
                *ptr = static_cast<float>(*ptr + part[p][q]);
                if (!diag) {
                    float* m = acc + ct.base + gj * ct.dim + gi;
                    *m = static_cast<float>(*m + part[p][q]);
                }
            }
    }
}

// ------------------------------------------- 256 x 256 tiles, stream-K
// For matrices of at least 256 channels (bf16, channel count a multiple
// of 32).  Each workgroup (8 waves in a 2 x 4 grid, two per SIMD) works on
// 256 x 256 tiles of the upper triangle; every wave keeps 128 x 64 fp32
// partial sums (4 x 2 v_mfma_f32_32x32x16_bf16 accumulators).  Waves 0-3
// and 4-7 (one of each per SIMD) run a ping-pong schedule one phase apart:
// in a load phase a wave requests its operand's slab three slabs ahead
// and reads all fragments of its next slab; in a compute phase it issues
// that slab's 16 MFMAs at raised priority.  Token slabs of 32 rows go from
// HBM straight into a 4-stage LDS ring with global_load_lds_dwordx4, in
// X's own row-major order (no transposition on the way in): 512 bytes of
// each token row per operand, 16-byte units XOR-swizzled by row.  The
// MFMA operands need 8 consecutive tokens of one channel; ds_read_tr16_b64
// performs that transposition on the LDS read: within 16 lanes, lane
// 4e + q addresses token row e, channels 4q..4q+3, and lane i receives
// channel i of the 4 rows.
//
// Work split (stream-K): the (tile, slab) units of all tiles, tile-major
// with tiles in super-tile order, are cut into one contiguous share per
// workgroup, so every CU gets the same number of MFMAs whatever the tile
// count.  A workgroup processes its tiles in order of their first slab
// (its share's head tile first), so the workgroups of one XCD stream
// nearly the same token slabs at the same time and share them in L2.
// A tile covered whole by one workgroup is added into acc directly; the
// pieces of a split tile go to per-workgroup slots of the workspace with
// plain stores, and cov_combine_kernel adds them into acc in a fixed order
// (deterministic, no atomics) and writes every tile's mirror image.
constexpr int kSkT = 256;                        // tile edge
constexpr int kSkSlab = 32;                      // tokens per ring stage
constexpr int kSkStages = 4;
static_assert(kSkStages >= 2 && kSkStages <= 4, "wait counts cover at most 2 slabs ahead");
constexpr int kSkRowUnits = kSkT / 8;            // 16-byte units per token row (32)
constexpr int kSkOpUnits = kSkSlab * kSkRowUnits;  // units per operand and stage (1024)
constexpr int kSkThreads = 512;                  // 8 waves: 2 x 4 over the tile
constexpr int kSkMaxSlabs = 256;                 // slabs per launch (8192 tokens)
constexpr int64_t kSkSlotFloats = int64_t(kSkT) * kSkT;   // one 256 x 256 fp32 tile

// A launch covers nmat matrices of dim channels each, X columns
// mat * dim .. mat * dim + dim - 1 for matrix mat: the whole d x d matrix
// (FULL), one k x k block (BLOCK_DIAG, k >= 256), or, for blocks of
// 32 .. 128 channels, one 256-channel group of 256 / k blocks ("packed":
// the group's 256 x 256 square is computed and only its diagonal k x k
// blocks are stored).
struct SkGeom {
    int64_t dim;     // channels of one matrix
    int64_t T;       // tiles along one edge of a matrix
    int64_t tri;     // upper-triangle tiles per matrix
    int64_t tiles;   // tiles over all matrices
    int64_t S;       // 32-token slabs of this launch
    int64_t U;       // units = tiles * S
    int64_t G;       // workgroups
    // output addressing (sk_out): matrix mat starts at acc + mat * mbase;
    // element (r, c) lies in diagonal block r >> lsub (lsub = 62 when the
    // matrix is stored whole), which starts bsz floats into the matrix per
    // block and has row stride `stride`
    int64_t mbase;
    int64_t bsz;
    int64_t stride;
    int lsub;
};

// Element offset in acc of entry (r, c) of matrix mat, or -1 for an entry
// off the block diagonal of a packed group (not stored).
__device__ __forceinline__ int64_t sk_out(const SkGeom& g, int64_t mat, int64_t r, int64_t c) {
    const int64_t br = r >> g.lsub;
    if (br != (c >> g.lsub)) return -1;
    const int64_t o = br << g.lsub;
    return mat * g.mbase + br * g.bsz + (r - o) * g.stride + (c - o);
}

// First unit of workgroup w's share (w = G gives U).
__device__ __forceinline__ int64_t sk_begin(const SkGeom& g, int64_t w) { return g.U * w / g.G; }

// The k-th upper-triangle tile of a T x T tile grid in super-tile order:
// 8 x 8 groups of tiles (row-major over the upper triangle of groups),
// row-major inside a group.  Consecutive tiles then share few distinct
// 256-channel blocks of X, which is what one XCD's L2 holds.
__device__ __forceinline__ void st_decode(int64_t r, int64_t T, int64_t& I, int64_t& J) {
    const int64_t Ts = (T + 7) / 8;
    for (int64_t P = 0; P < Ts; ++P)
        for (int64_t Q = P; Q < Ts; ++Q) {
            const int64_t i0 = 8 * P, i1 = (8 * P + 8 < T) ? 8 * P + 8 : T;
            const int64_t j0 = 8 * Q, j1 = (8 * Q + 8 < T) ? 8 * Q + 8 : T;
            const int64_t m = i1 - i0;
            const int64_t cnt = P == Q ? m * (m + 1) / 2 : m * (j1 - j0);
            if (r < cnt) {
                if (P == Q) {
                    int64_t i = 0;
                    while (r >= m - i) {
                        r -= m - i;
                        ++i;
                    }
                    I = i0 + i;
                    J = i0 + i + r;
                } else {
                    I = i0 + r / (j1 - j0);
                    J = j0 + r % (j1 - j0);
                }
                return;
            }
            r -= cnt;
        }
    I = J = 0;   // not reached for r < T (T + 1) / 2
}

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

__global__ __launch_bounds__(kSkThreads, 1) void cov_sk_kernel(const uint16_t* __restrict__ X,
                                                                int64_t n, int64_t d, SkGeom g,
                                                                float* __restrict__ acc,
                                                                float* __restrict__ ws) {
    __shared__ __attribute__((aligned(16))) u32x4 ring[kSkStages][2][kSkOpUnits];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // uniform: SGPR branches
    const int wm = wave >> 2, wn = wave & 3;   // wave tile 128 x 64
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // this workgroup's share of the unit list (XCD-major numbering: the
    // 32 consecutive shares of one XCD cover neighbouring tiles)
    const int64_t G = g.G;
    int64_t w = blockIdx.x;
    if (G % 8 == 0) w = (blockIdx.x % 8) * (G / 8) + blockIdx.x / 8;
    const int64_t u_begin = sk_begin(g, w), u_end = sk_begin(g, w + 1);
    const int64_t t_first = u_begin / g.S, t_last = (u_end - 1) / g.S;
    const bool head_first = (u_begin % g.S) != 0 && t_last > t_first;

    // Ping-pong: waves 0-3 (rows 0-127 of the tile, one per SIMD) and waves
    // 4-7 (rows 128-255) are one phase apart.  In a load phase a wave
    // requests its operand's slab three slabs ahead (waves 0-3 operand A,
    // waves 4-7 operand B, which a diagonal tile does not load) and reads
    // all fragments of its next slab; in a compute phase it issues that
    // slab's 16 MFMAs.  On every SIMD one wave computes while the other
    // loads.
    const int grp = wave >> 2, w4 = wave & 3;
    // direct-load geometry: load q of this thread fills unit (4q+w4)*64+lane
    // of its operand's stage, i.e. token row 8q + rr, swizzled position l32.
    const int rr = 2 * w4 + h;
    const int unit = l32 ^ ((rr & 3) << 2);      // global 16-byte unit of the row
    const uint32_t row_bytes = static_cast<uint32_t>(d) * 2u;
    constexpr int kPpLoads = kSkOpUnits / (kSkThreads / 2);   // 4

    for (int64_t idx = 0; u_begin < u_end && idx <= t_last - t_first; ++idx) {
        // tiles in order of their first slab: t_first + 1 .. t_last, then t_first
        const int64_t tile = head_first ? (idx < t_last - t_first ? t_first + 1 + idx : t_first)
                                        : t_first + idx;
        const int64_t s0 = tile == t_first ? u_begin % g.S : 0;
        const int64_t s1 = tile == t_last ? (u_end - 1) % g.S + 1 : g.S;
        const bool whole = s0 == 0 && s1 == g.S;
        const int64_t mat = tile / g.tri;
        int64_t I, J;
        st_decode(tile % g.tri, g.T, I, J);
        const int64_t colbase = mat * g.dim;
        const int64_t I0 = I * kSkT, J0 = J * kSkT;
        const bool diag = I == J;
        // this wave's operand: A (rows I0..) for group 0, B (J0..) for group 1
        const bool loads = grp == 0 || !diag;
        const int op = grp;

        // per-thread source byte offset inside a slab (columns clamped into
        // the matrix when the last tile is ragged: those rows/columns of the
        // result are discarded)
        int64_t cx = (grp == 0 ? I0 : J0) + 8 * unit;
        if (cx >= g.dim) cx = grp == 0 ? I0 : J0;
        const uint32_t ox = static_cast<uint32_t>(rr) * row_bytes + static_cast<uint32_t>(colbase + cx) * 2u;
        const uint32_t lx = static_cast<uint32_t>(
            __builtin_amdgcn_readfirstlane(lds_addr(&ring[0][op][w4 * 64])));

        auto issue = [&](int64_t s, int st) {
            if (!loads) return;
            const int64_t t0 = s * kSkSlab;
            const char* base = reinterpret_cast<const char*>(X + t0 * d);
            const uint32_t l = lx + static_cast<uint32_t>(st) * (2 * kSkOpUnits * 16);
            if (t0 + kSkSlab <= n) {
#pragma unroll
                for (int q = 0; q < kPpLoads; ++q) dma16(base, ox + q * 8u * row_bytes, l + q * 4096u);
            } else {
                // ragged last slab: rows past n load row n-1 (zeroed once landed)
#pragma unroll
                for (int q = 0; q < kPpLoads; ++q) {
                    const int64_t t = t0 + 8 * q + rr;
                    const uint32_t back = t < n ? 0u : static_cast<uint32_t>(t - (n - 1)) * row_bytes;
                    dma16(base, ox + q * 8u * row_bytes - back, l + q * 4096u);
                }
            }
        };
        // this thread's loads of slab s have landed once at most those of the
        // slabs issued after it (up to `last`) are outstanding; rows past n of
        // a ragged slab are then zeroed by the thread that loaded them
        auto wait_slab = [&](int64_t s, int64_t last) {
            if (!loads || s >= s1) return;
            const int64_t ahead = last - s;
            if (ahead >= 2) wait_vmcnt<2 * kPpLoads>();
            else if (ahead == 1) wait_vmcnt<kPpLoads>();
            else wait_vmcnt<0>();
            const int64_t t0 = s * kSkSlab;
            if (t0 + kSkSlab > n) {
                const int sl = static_cast<int>((s - s0) % kSkStages);
#pragma unroll
                for (int q = 0; q < kPpLoads; ++q)
                    if (t0 + 8 * q + rr >= n)
                        ring[sl][op][(q * 4 + w4) * 64 + lane] = u32x4{0u, 0u, 0u, 0u};
            }
        };
        auto last_issued = [&](int64_t s) {   // last slab requested once slab s's load phase ran
            return (s + kSkStages - 1 < s1 - 1) ? s + kSkStages - 1 : s1 - 1;
        };
        typedef const char __attribute__((address_space(3))) * lds_cptr;
        bf16x8 fa[2][4], fb[2][2];
        auto read_frags = [&](int sl) {
            // fragment-read geometry (bytes inside one operand stage),
            // recomputed per call from a lane index the compiler cannot
            // hoist: kept live across the loop it would spill
            int el = lane;
            asm volatile("" : "+v"(el));
            const int i16 = el & 15, e = i16 >> 2, qq = i16 & 3, gg = (el >> 4) & 1, hh = el >> 5;
            const int row = 8 * hh + e;             // token row inside the 16-token step
            const uint32_t rowoff = static_cast<uint32_t>(row * (kSkT * 2) + 8 * (qq & 1));
            const int usw = (row & 3) << 2;
            lds_cptr baseA = (lds_cptr)&ring[sl][0][0];
            lds_cptr baseB = (lds_cptr)&ring[sl][diag ? 0 : 1][0];
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    const int ua = (wm * 16 + 4 * a + 2 * gg + (qq >> 1)) ^ usw;
                    fa[kk][a] = sk_frag(baseA, rowoff + 16 * ua + kk * 16 * kSkT * 2);
                }
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int ub = (wn * 8 + 4 * b + 2 * gg + (qq >> 1)) ^ usw;
                    fb[kk][b] = sk_frag(baseB, rowoff + 16 * ub + kk * 16 * kSkT * 2);
                }
            }
        };
        f32x16 part[4][2];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b) part[a][b] = f32x16{};
        auto mfmas = [&]() {
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int kk = 0; kk < 2; ++kk)
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int b = 0; b < 2; ++b)
                        part[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk][a], fb[kk][b],
                                                                             part[a][b], 0, 0, 0);
            __builtin_amdgcn_s_setprio(0);
        };
        auto phase_end = [&]() {
            __builtin_amdgcn_sched_barrier(0);
            lds_barrier();
            __builtin_amdgcn_sched_barrier(0);
        };

        // prologue: slabs s0 .. s0 + 2 requested, s0 landed and published
#pragma unroll
        for (int p = 0; p < kSkStages - 1; ++p)
            if (s0 + p < s1) issue(s0 + p, p);
        wait_slab(s0, (s0 + kSkStages - 2 < s1 - 1) ? s0 + kSkStages - 2 : s1 - 1);
        lds_barrier();
        // 2 (s1 - s0) + 1 phases: group 0 loads slab i in phase 2i and computes
        // it in phase 2i + 1; group 1 one phase later
        if (grp == 0) {
            for (int64_t s = s0; s < s1; ++s) {
                const int st = static_cast<int>((s - s0) % kSkStages);
                if (s + kSkStages - 1 < s1)
                    issue(s + kSkStages - 1, st == 0 ? kSkStages - 1 : st - 1);
                read_frags(st);
                phase_end();
                mfmas();
                wait_slab(s + 1, last_issued(s));          // A of the next slab
                phase_end();
            }
            phase_end();
        } else {
            phase_end();
            for (int64_t s = s0; s < s1; ++s) {
                const int st = static_cast<int>((s - s0) % kSkStages);
                if (s + kSkStages - 1 < s1)
                    issue(s + kSkStages - 1, st == 0 ? kSkStages - 1 : st - 1);
                read_frags(st);
                wait_slab(s + 1, last_issued(s));          // B of the next slab
                phase_end();
                mfmas();
                phase_end();
            }
        }

        // Partial sums out.  A whole tile is added into acc (upper tile,
        // both triangles of a diagonal tile) in 4 chunks of 64 values per
        // lane; a split tile's piece is stored to its slot, a 256 x 256
        // row-major fp32 tile (slot 0: the share's first tile, slot 1: its
        // last).  32-bit element offsets; the empty asm statements keep the
        // offsets from being precomputed outside the loop and the chunks
        // apart.
        uint32_t rowb = static_cast<uint32_t>(wm * 128 + 4 * h);
        uint32_t colb = static_cast<uint32_t>(wn * 64 + l32);
        asm volatile("" : "+v"(rowb), "+v"(colb));
        if (whole) {
            // Through LDS (the ring is free once every wave is past its last
            // fragment read): the 128 x 256 half of the tile that the four
            // waves with wm == half hold is written row-major into LDS, then
            // all 512 threads add it into acc with 16-byte row accesses.  This
            // keeps the read-modify-write of acc out of the accumulator
            // registers.
            float* stage = reinterpret_cast<float*>(&ring[0][0][0]);   // 128 x 256 fp32
            const int64_t dimv = g.dim;
            const bool rows_ok = I0 + kSkT <= dimv, cols_ok = J0 + kSkT <= dimv;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                lds_barrier();
                if (wm == half) {
                    // one base per 32-row group keeps every offset inside the
                    // 64 KiB immediate range of an LDS store
                    int el = lane;
                    asm volatile("" : "+v"(el));
#pragma unroll
                    for (int a = 0; a < 4; ++a) {
                        float* sa = stage + (32 * a + 4 * (el >> 5)) * kSkT + wn * 64 + (el & 31);
#pragma unroll
                        for (int b = 0; b < 2; ++b)
#pragma unroll
                            for (int r = 0; r < 16; ++r)
                                sa[(8 * (r >> 2) + (r & 3)) * kSkT + 32 * b] = part[a][b][r];
                    }
                }
                lds_barrier();
                // 128 rows x 64 float4 per row; thread tid takes column group
                // tid % 64 of rows tid / 64 + 8 j
                const int cg = tid & 63;
                const int64_t col = J0 + 4 * cg;
                if (cols_ok || col < dimv) {
#pragma unroll
                    for (int j0 = 0; j0 < 16; j0 += 8) {
                        f32x4 old[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            const int row = (tid >> 6) + 8 * (j0 + j);
                            const int64_t grow = I0 + 128 * half + row;
                            const int64_t o = (rows_ok || grow < dimv) ? sk_out(g, mat, grow, col) : -1;
                            old[j] = o >= 0 ? *reinterpret_cast<const f32x4*>(acc + o)
                                            : f32x4{0.f, 0.f, 0.f, 0.f};
                        }
#pragma unroll
                        for (int j = 0; j < 8; ++j) {
                            const int row = (tid >> 6) + 8 * (j0 + j);
                            const int64_t grow = I0 + 128 * half + row;
                            const f32x4 add = *reinterpret_cast<const f32x4*>(stage + row * kSkT + 4 * cg);
                            const int64_t o = (rows_ok || grow < dimv) ? sk_out(g, mat, grow, col) : -1;
                            if (o >= 0) *reinterpret_cast<f32x4*>(acc + o) = old[j] + add;
                        }
                    }
                }
            }
        } else {
            float* slot = ws + (w * 2 + (tile == t_first ? 0 : 1)) * kSkSlotFloats;
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    // a packed group keeps only its diagonal blocks (each
                    // 32 x 32 accumulator lies inside one block)
                    if ((int64_t(wm * 128 + 32 * a) >> g.lsub) != (int64_t(wn * 64 + 32 * b) >> g.lsub))
                        continue;
#pragma unroll
                    for (int r = 0; r < 16; ++r)
                        slot[(rowb + 32 * a + 8 * (r >> 2) + (r & 3)) * kSkT + colb + 32 * b] =
                            part[a][b][r];
                }
        }
        lds_barrier();   // every wave is done with the ring before the next tile refills it
    }
}

// The workgroup whose share holds unit u.
__device__ __forceinline__ int64_t sk_owner(const SkGeom& g, int64_t u) {
    int64_t w = u * g.G / g.U;
    while (w + 1 < g.G && sk_begin(g, w + 1) <= u) ++w;
    while (w > 0 && sk_begin(g, w) > u) --w;
    return w;
}

// After cov_sk_kernel: every split tile's pieces are added into acc in
// share order (acc + piece of the lowest workgroup + ... ), and every
// off-diagonal tile's transpose is written below the diagonal.  One
// workgroup per 64 x 64 sub-block of a tile: coalesced 16-byte row reads,
// transposition through LDS, coalesced 16-byte row writes.
__global__ __launch_bounds__(kCovThreads) void cov_combine_kernel(float* __restrict__ acc, SkGeom g,
                                                                  const float* __restrict__ ws) {
    __shared__ float tr[64][65];
    const int64_t tile = blockIdx.x / 16;
    const int sub = static_cast<int>(blockIdx.x % 16);
    const int64_t mat = tile / g.tri;
    int64_t I, J;
    st_decode(tile % g.tri, g.T, I, J);
    const int sr = (sub >> 2) * 64, sc = (sub & 3) * 64;   // sub-block origin inside the tile
    const int64_t r0 = I * kSkT + sr, c0 = J * kSkT + sc;
    if (r0 >= g.dim || c0 >= g.dim) return;
    // a packed group's sub-blocks off its block diagonal are not stored
    const int lb = g.lsub > 6 ? g.lsub : 6;
    if ((r0 >> lb) != (c0 >> lb)) return;
    const int64_t w_lo = sk_owner(g, tile * g.S), w_hi = sk_owner(g, (tile + 1) * g.S - 1);
    const bool whole = w_lo == w_hi && sk_begin(g, w_lo) <= tile * g.S &&
                       sk_begin(g, w_lo + 1) >= (tile + 1) * g.S;
    if (whole && I == J) return;   // added in place by the main kernel, no mirror
    const int tid = threadIdx.x;
    const int rl = tid >> 4, cl = 4 * (tid & 15);
    f32x4 v[4];
    int64_t o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = rl + 16 * i;
        const bool ok = r0 + row < g.dim && c0 + cl < g.dim;
        o[i] = ok ? sk_out(g, mat, r0 + row, c0 + cl) : -1;
        v[i] = o[i] >= 0 ? *reinterpret_cast<const f32x4*>(acc + o[i]) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    if (!whole) {
        auto slot_of = [&](int64_t w) {
            const int64_t t_first = sk_begin(g, w) / g.S;
            return ws + (w * 2 + (tile == t_first ? 0 : 1)) * kSkSlotFloats;
        };
        int64_t w = w_lo;
        // two pieces per round: all their loads in flight before the adds,
        // which keep the share order
        for (; w + 1 <= w_hi; w += 2) {
            const float* s0 = slot_of(w);
            const float* s1 = slot_of(w + 1);
            f32x4 p0[4], p1[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p0[i] = *reinterpret_cast<const f32x4*>(s0 + (sr + rl + 16 * i) * kSkT + sc + cl);
                p1[i] = *reinterpret_cast<const f32x4*>(s1 + (sr + rl + 16 * i) * kSkT + sc + cl);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] += p0[i];
                v[i] += p1[i];
            }
        }
        if (w <= w_hi) {
            const float* s0 = slot_of(w);
#pragma unroll
            for (int i = 0; i < 4; ++i)
                v[i] += *reinterpret_cast<const f32x4*>(s0 + (sr + rl + 16 * i) * kSkT + sc + cl);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (o[i] >= 0) *reinterpret_cast<f32x4*>(acc + o[i]) = v[i];
    }
    if (I == J) return;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = rl + 16 * i;
#pragma unroll
        for (int e = 0; e < 4; ++e) tr[row][cl + e] = v[i][e];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = rl + 16 * i;   // row of the lower block = column of the upper one
        if (c0 + row >= g.dim || r0 + cl >= g.dim) continue;
        const f32x4 t = {tr[cl][row], tr[cl + 1][row], tr[cl + 2][row], tr[cl + 3][row]};
        *reinterpret_cast<f32x4*>(acc + sk_out(g, mat, c0 + row, r0 + cl)) = t;   // whole matrix
    }
}

// Geometry of one launch over n <= kSkMaxSlabs * 32 tokens.
// Blocks of 32 .. 128 channels in whole 256-channel groups run packed.
static bool cov_sk_packed(int64_t d, int mode, int64_t k) {
    return mode == CAT_COV_BLOCK_DIAG && k >= 32 && k < kSkT && (d % kSkT) == 0;
}

static bool cov_sk_geometry(int64_t n, int64_t d, int mode, int64_t k, int64_t cus, SkGeom& g) {
    const bool packed = cov_sk_packed(d, mode, k);
    g.dim = packed ? kSkT : (mode == CAT_COV_FULL ? d : k);
    const int64_t nmat = mode == CAT_COV_FULL ? 1 : d / g.dim;
    if (packed) {
        int l = 0;
        while ((int64_t(1) << l) < k) ++l;   // k is a power of two
        g.lsub = l;
        g.bsz = k * k;
        g.stride = k;
        g.mbase = kSkT * k;
    } else {
        g.lsub = 62;
        g.bsz = 0;
        g.stride = g.dim;
        g.mbase = g.dim * g.dim;
    }
    g.T = (g.dim + kSkT - 1) / kSkT;
    g.tri = g.T * (g.T + 1) / 2;
    g.tiles = nmat * g.tri;
    g.S = (n + kSkSlab - 1) / kSkSlab;
    g.U = g.tiles * g.S;
    g.G = g.U < cus ? g.U : cus;
    return g.U > 0;
}

static bool cov_uses_sk(int x_bf16, int64_t d, int mode, int64_t k) {
    const int64_t dim = mode == CAT_COV_FULL ? d : k;
    return x_bf16 && (d % 8) == 0 &&
           ((dim >= kSkT && (dim % 32) == 0) || cov_sk_packed(d, mode, k));
}

static hipError_t device_cus(int& cus) {
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    return hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
}

hipError_t cov_workspace_bytes(int x_bf16, int64_t d, int mode, int64_t k, size_t& bytes) {
    bytes = 0;
    if (!cov_uses_sk(x_bf16, d, mode, k)) return hipSuccess;
    int cus = 0;
    hipError_t err = device_cus(cus);
    if (err != hipSuccess) return err;
    bytes = static_cast<size_t>(cus) * 2 * kSkSlotFloats * sizeof(float);
    return hipSuccess;
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
                                 int64_t k, float* acc, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
    const int64_t dim = mode == CAT_COV_FULL ? d : k;
    if (cov_uses_sk(x_bf16, d, mode, k)) {
        int cus = 0;
        hipError_t err = device_cus(cus);
        if (err != hipSuccess) return err;
        if (workspace_bytes < static_cast<size_t>(cus) * 2 * kSkSlotFloats * sizeof(float))
            return hipErrorInvalidValue;   // checked by the caller; never reached
        const uint16_t* Xb = static_cast<const uint16_t*>(X);
        // one launch pair per 8192 tokens: each register partial covers at
        // most that many tokens, and the pieces are combined before the
        // workspace is reused
        for (int64_t t0 = 0; t0 < n; t0 += int64_t(kSkMaxSlabs) * kSkSlab) {
            const int64_t nc = (n - t0 < int64_t(kSkMaxSlabs) * kSkSlab) ? n - t0
                                                                       : int64_t(kSkMaxSlabs) * kSkSlab;
            SkGeom g;
            if (!cov_sk_geometry(nc, d, mode, k, cus, g)) return hipSuccess;
            hipLaunchKernelGGL(cov_sk_kernel, dim3(static_cast<uint32_t>(g.G)), dim3(kSkThreads),
                               0, stream, Xb + t0 * d, nc, d, g, acc,
                               static_cast<float*>(workspace));
            err = hipGetLastError();
            if (err != hipSuccess) return err;
            hipLaunchKernelGGL(cov_combine_kernel, dim3(static_cast<uint32_t>(g.tiles * 16)),
                               dim3(kCovThreads), 0, stream, acc, g,
                               static_cast<const float*>(workspace));
            err = hipGetLastError();
            if (err != hipSuccess) return err;
        }
        return hipSuccess;
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
