// W4A4 integer GEMM with fused dequantization (Sec. 3, eq. 5):
//   acc[t, o] = sum_j qx[t, j] qw[o, j]                   (int32, exact)
//   y[t, o]   = fl32(fl32(acc) * s_x[t]) * s_w[o]
//
// gfx950 int8 MFMA (v_mfma_i32_32x32x32_i8) on INT4 codes.
//
// Tiles: 256 x 256 outputs per workgroup of 512 threads = 8 waves in a
// 2 x 4 grid, each wave 128 x 64 = 4 x 2 MFMA tiles with int32
// accumulators; one workgroup per CU (two waves per SIMD, 144 KiB of LDS).
// One K step covers 128 codes (64 packed bytes per row); a tile reads
// 32 KiB of packed codes per step.  When 256-token tiles would leave CUs
// idle (fewer tiles than workgroup slots) and 128-token tiles take no more
// rounds of the grid, the launch uses 128 x 256 tiles instead: each wave
// 64 x 64 (2 x 2 MFMA tiles), the same ring and schedule, 24 KiB per step
// spread as three direct loads per wave.
//
// Ping-pong schedule: waves 0-3 (rows 0-127 of the tile, one wave per
// SIMD) and waves 4-7 (rows 128-255, the other wave of each SIMD) are
// offset by one phase.  In a compute phase a wave issues the 32 MFMAs of
// one K step at raised priority; in a load phase it requests the direct
// loads of a later step and reads the next step's fragments from LDS.  A
// workgroup barrier separates phases, so on every SIMD one wave computes
// while the other loads.  Per tile: 2 nk + 2 phases; group 0 stores its
// half of the tile while group 1 computes the last step, group 1 one phase
// later.  Each group runs its own straight-line loop.
//
// Operand path: packed INT4 tiles go straight from global memory into an
// LDS ring of kStages (4) steps with global_load_lds_dwordx4 (no register
// staging, no LDS store instructions), requested kStages-1 steps ahead;
// waves 0-3 load operand A (codes_x), waves 4-7 operand B (codes_w) (with
// 128-token tiles waves 0-3 also load B's first 64 rows).  The
// barrier waits for LDS traffic only (a plain workgroup barrier would also
// drain the loads in flight); each wave waits for its own loads of the next
// step (vmcnt) before the barrier that publishes it.  Each lane reads 16
// packed bytes (32 codes, two MFMA steps) per fragment and widens them in
// registers to int8 values 16*code: a packed dword (8 codes) becomes one
// dword of its low nibbles and one of its high nibbles.  B is widened in
// the load phase, A in the compute phase (registers: 128 accumulators,
// 32 packed A and 32 widened B per lane).  Both operands are widened
// identically, so each MFMA sums the same index pairs (a permutation of the
// reduction index) and the int32 result is 256 * acc; an arithmetic shift
// by 8 recovers acc exactly for d_in <= 131072.
//
// LDS layout: each operand stage is rows x 4 units of 16 bytes; unit u of
// row r sits at slot 4r + (u ^ swz(r)), with swz(r) built from bits 2 and 3
// of r.  A fragment read covers 32 consecutive rows at one unit (lanes
// 0-31) and the same rows at unit u ^ 2 (lanes 32-63).  Rows r, r+4, r+8,
// r+12 get four different swz values, and swz(r+4) always differs from
// swz(r) in bit 0, so both 16 consecutive lanes and lanes {i..i+7} with
// {i+32..i+39} land on 16 distinct 16-byte bank groups of a 64-bank LDS.
// The direct loads fill 64 consecutive slots per wave instruction, so each
// lane loads the global unit that belongs in its slot (a permutation inside
// each 64-byte row segment).  Rows past the end of a matrix load a clamped
// in-bounds row (their outputs are never stored); units past d_in in a
// ragged last step load any in-bounds unit and the loading thread clears
// them in A before the barrier that publishes the step, which zeroes their
// products.
//
// Persistent launch: one workgroup per CU walks a list of tiles in an
// XCD-aware order (workgroups are dealt to the 8 XCDs round-robin; those of
// XCD x walk one contiguous range of tiles, in groups of kGroupM row
// panels, so tiles resident on one XCD share panels in its L2).  The
// operand steps of consecutive tiles form one stream through the ring, and
// each tile's scales are staged in LDS with its first step, so the
// epilogue reads no global memory.  The epilogue of a full tile is
// straight-line code with a wave-uniform row base per accumulator row: it
// runs once per tile, so its instruction footprint is what it costs.
#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kGemmWaves = 8;
constexpr int kGemmThreads = kGemmWaves * 64;
constexpr int kBM = 256;           // tokens per tile (the LDS layout's maximum)
constexpr int kBN = 256;           // outputs per tile
constexpr int kKBP = 64;           // packed bytes per row per K step (128 codes)
constexpr int kUP = kKBP / 16;     // 16-byte units per row per step
constexpr int kStages = 4;         // LDS ring depth (steps)
constexpr int kWgPerCu = 1;
static_assert(kStages >= 2 && kStages <= 4, "waits cover at most 2 steps ahead");
constexpr int kGroupM = 4;         // row panels per tile group
constexpr int kXcd = 8;

__device__ __forceinline__ int gemm_swz(int r) {
    return ((r >> 2) & 1) | ((((r >> 2) ^ (r >> 3)) & 1) << 1);
}

struct GemmTile {
    int64_t m0, n0;
};

template <int BM>
__device__ __forceinline__ bool gemm_tile(int64_t k, int64_t n, int64_t d_out, GemmTile& t) {
    const int64_t tiles_m = (n + BM - 1) / BM;
    const int64_t tiles_n = (d_out + kBN - 1) / kBN;
    const int64_t T = tiles_m * tiles_n;
    const int64_t per_xcd = (T + kXcd - 1) / kXcd;
    const int64_t wg_per_xcd = gridDim.x / kXcd;
    const int64_t x = blockIdx.x % kXcd, j = blockIdx.x / kXcd;
    const int64_t local = j + k * wg_per_xcd;
    if (local >= per_xcd) return false;
    const int64_t tau = x * per_xcd + local;
    if (tau >= T) return false;
    const int64_t group = tau / (kGroupM * tiles_n);
    const int64_t first_m = group * kGroupM;
    const int64_t gm = (tiles_m - first_m) < kGroupM ? (tiles_m - first_m) : kGroupM;
    const int64_t in_group = tau % (kGroupM * tiles_n);
    t.m0 = (first_m + in_group % gm) * BM;
    t.n0 = (in_group / gm) * kBN;
    return true;
}

__device__ __forceinline__ i32x4 widen8(u32x4 v, int half) {
    const uint32_t w0 = v[2 * half], w1 = v[2 * half + 1];
    return i32x4{static_cast<int>(unpack_lo16(w0)), static_cast<int>(unpack_hi16(w0)),
                 static_cast<int>(unpack_lo16(w1)), static_cast<int>(unpack_hi16(w1))};
}

constexpr int kPpUnits = kBM * kUP;                        // units per operand stage
// direct loads (64-slot instructions) per wave and step: 4 with 256-token
// tiles (group 0 loads A, group 1 B); 3 with 128-token tiles (A's 8
// chunks and B's first 4 from group 0, B's other 12 from group 1)
template <int BM>
constexpr int gemm_loads() { return BM == kBM ? 4 : 3; }
// scale slots: a tile's slot is reused 8 tiles later, after both groups'
// epilogues of the earlier tile even when every tile is one K step
constexpr int kScaleSlots = 8;
static_assert(kBM == kBN, "both operands share the stage layout");
static_assert(kPpUnits / (kGemmThreads / 2) == 4, "four 64-slot instructions per wave per step");

// ring[o][stage]: operand o (0 = A, 1 = B), kStages steps deep.
// sscale[slot]: s_x of a tile's rows and s_w of its outputs; slot = tile
// index % kScaleSlots.
typedef u32x4 GemmRing[2][kStages][kPpUnits];
typedef float GemmScales[kScaleSlots][kBM + kBN];

// I8: codes are one int8 per element (rows of d_in bytes), used by the
// MFMA as they are; otherwise packed INT4 (rows of d_in / 2 bytes), widened
// to 16 * code in registers.  A K step is 64 bytes of a row either way:
// 128 INT4 codes (4 MFMA sub-steps) or 64 int8 codes (2).
// ASYM (INT4 only): asymmetric activations stored as q - 8 with the row
// minimum zmin_x, weights with row code sums rsum_w: the epilogue adds
// 8 R_o back (int32, exact) and forms
// y = fl(fl(fl(acc) s_x) + fl(zmin fl(R_o))) s_w.
template <bool I8, bool ASYM, int BM>
__device__ __forceinline__ void gemm_body(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out, GemmRing& ring,
    GemmScales& sscale, const float* __restrict__ zmin_x, const int32_t* __restrict__ rsum_w,
    GemmScales* sasym) {
    static_assert(!(I8 && ASYM), "asymmetric codes are INT4");
    static_assert(BM == kBM || BM == kBM / 2, "256- or 128-token tiles");
    constexpr int IM = BM / 64;            // 32-row accumulator groups per wave
    constexpr int NL = gemm_loads<BM>();
    const int64_t row_bytes = I8 ? d_in : d_in / 2;
    const int nk = static_cast<int>((row_bytes + kKBP - 1) / kKBP);

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);   // uniform: SGPR branches
    const int grp = wave >> 2;                 // 0: rows 0-127, loads A; 1: rows 128-255, loads B
    const int wm = grp, wn = wave & 3;         // 2 x 4 waves, each 128 x 64
    const int w4 = wave & 3;
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // tiles of this workgroup and total steps
    int n_tiles = 0;
    {
        GemmTile t;
        while (gemm_tile<BM>(n_tiles, n, d_out, t)) ++n_tiles;
    }
    if (n_tiles == 0) return;
    const int G = n_tiles * nk;

    // Direct loads: instruction q of this wave fills chunk ch(q) (64 slots,
    // 16 rows) of operand op(q)'s stage; slot s of a chunk holds row s / 4
    // of the chunk, logical unit (s % 4) ^ swz(row).  swz(row) depends on
    // lane bits 4-5 only.  256-token tiles: group 0 loads A, group 1 B,
    // chunk 4q + w4.  128-token tiles: group 0 loads A's chunks 2 w4, 2 w4
    // + 1 and B's chunk w4, group 1 B's chunks 4 + 3 w4 + q.
    auto ld_op = [&](int q) { return BM == kBM ? grp : (grp == 1 || q == 2 ? 1 : 0); };
    auto ld_ch = [&](int q) {
        if constexpr (BM == kBM) return 4 * q + w4;
        return grp == 0 ? (q < 2 ? 2 * w4 + q : w4) : 4 + 3 * w4 + q;
    };
    const uint8_t* base_a = qx;
    const uint8_t* base_b = qw;
    uint32_t src_off[NL];
    const int u_off = ((lane % kUP) ^ gemm_swz(lane / kUP)) * 16;
    // row offsets inside a tile are below 256 * 65536 bytes: 32-bit
    const uint32_t rb32 = static_cast<uint32_t>(row_bytes);
    auto set_rows = [&](const GemmTile& tl) {
        base_a = qx + tl.m0 * row_bytes;
        base_b = qw + tl.n0 * row_bytes;
        const int left_a = static_cast<int>(n - tl.m0 < BM ? n - tl.m0 : BM);
        const int left_b = static_cast<int>(d_out - tl.n0 < kBN ? d_out - tl.n0 : kBN);
        int el = lane;
        asm volatile("" : "+v"(el));
#pragma unroll
        for (int q = 0; q < NL; ++q) {
            const int r = ld_ch(q) * (64 / kUP) + el / kUP;
            const int left = ld_op(q) == 0 ? left_a : left_b;
            const int rr = r < left ? r : left - 1;   // clamped rows: never stored
            src_off[q] = static_cast<uint32_t>(rr) * rb32;
        }
    };
    uint32_t lds_q[NL];
#pragma unroll
    for (int q = 0; q < NL; ++q)
        lds_q[q] = static_cast<uint32_t>(
            __builtin_amdgcn_readfirstlane(lds_addr(&ring[ld_op(q)][0][ld_ch(q) * 64])));
    auto issue_step = [&](int kt, int st) {
        const int64_t k0 = static_cast<int64_t>(kt) * kKBP;
        int64_t col = k0 + u_off;
        col = col < row_bytes ? col : 0;      // past the row end: any in-bounds unit
        const uint32_t cu = static_cast<uint32_t>(col);
        const uint32_t so = static_cast<uint32_t>(st) * (kPpUnits * 16);
#pragma unroll
        for (int q = 0; q < NL; ++q)
            dma16(ld_op(q) == 0 ? base_a : base_b, src_off[q] + cu, lds_q[q] + so);
    };
    // s_x (group 0) or s_w (group 1) of a tile into its scale slot (s_x at
    // [0, BM), s_w at [kBM, kBM + kBN)): rows / outputs past the end load
    // the last one (never stored).  With 128-token tiles waves 0 and 1 load
    // s_x and waves 2 and 3 load none.
    const int64_t src_rows = grp == 0 ? n : d_out;
    const bool ld_scales = grp == 1 || 64 * w4 < BM;
    auto issue_scales = [&](const GemmTile& tl, int slot) {
        if (!ld_scales) return;
        const int64_t r = (grp == 0 ? tl.m0 : tl.n0) + 64 * w4 + lane;
        dma4(grp == 0 ? s_x : s_w, static_cast<uint32_t>((r < src_rows ? r : src_rows - 1) * 4),
             lds_addr(&sscale[slot][grp * kBM + 64 * w4]));
        if constexpr (ASYM) {
            // the rows' minima (group 0) and the outputs' weight code sums
            // (group 1), staged like the scales; older than the step's
            // loads, so the step's wait covers them too
            const void* a = grp == 0 ? static_cast<const void*>(zmin_x)
                                     : static_cast<const void*>(rsum_w);
            dma4(a, static_cast<uint32_t>((r < src_rows ? r : src_rows - 1) * 4),
                 lds_addr(&(*sasym)[slot][grp * kBM + 64 * w4]));
        }
    };
    // A units of a ragged last step past d_in: zeroed by the threads that loaded them
    auto clear_ragged = [&](int kt, int st) {
        if (grp == 0 && kt == nk - 1 && (row_bytes % kKBP) != 0) {
#pragma unroll
            for (int q = 0; q < NL; ++q)
                if (ld_op(q) == 0 && static_cast<int64_t>(kt) * kKBP + u_off >= row_bytes)
                    ring[0][st][ld_ch(q) * 64 + lane] = u32x4{0u, 0u, 0u, 0u};
        }
    };

    i32x16 acc[IM][2];
    // Fragments of one K step, read in the load phase: unit u = 2h + c of
    // each row (c = 0, 1), 32 codes each; sub-step s = 2c + half covers
    // codes [32 s, 32 s + 32) of the step (a permutation of the reduction
    // index shared by both operands).  A stays packed until the compute
    // phase; B is widened in the load phase.
    u32x4 pa[2][IM];
    i32x4 fb[4][2];
    // Row r = base + 32 i + l32 of a fragment has swz(r) = swz(l32) (bits 2
    // and 3 of r come from l32), so each unit's address is one per-lane
    // base plus immediate offsets.
    const int frag_lane = l32 * kUP;
    const int frag_u0 = (2 * h) ^ gemm_swz(l32);
    // (int8 codes: unit c of the lane is sub-step c as it is; fb[0..1] hold
    // B's two units)
    auto load_frags = [&](int st) {
        const u32x4* ra = &ring[0][st][wm * (BM / 2) * kUP + frag_lane];
        const u32x4* rb = &ring[1][st][wn * 64 * kUP + frag_lane];
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int uo = frag_u0 ^ c;
#pragma unroll
            for (int i = 0; i < IM; ++i) pa[c][i] = ra[i * 32 * kUP + uo];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const u32x4 pbj = rb[j * 32 * kUP + uo];
                if constexpr (I8) {
                    fb[c][j] = __builtin_bit_cast(i32x4, pbj);
                } else {
                    fb[2 * c][j] = widen8(pbj, 0);
                    fb[2 * c + 1][j] = widen8(pbj, 1);
                }
            }
        }
    };
    auto compute_step = [&]() {
        // the computing wave's instructions go first on its SIMD (the other
        // wave there is in its load phase)
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int s = 0; s < (I8 ? 2 : 4); ++s) {
            i32x4 wa[IM];
#pragma unroll
            for (int i = 0; i < IM; ++i)
                wa[i] = I8 ? __builtin_bit_cast(i32x4, pa[s][i]) : widen8(pa[s >> 1][i], s & 1);
            const i32x4* wb = fb[s];
#pragma unroll
            for (int i = 0; i < IM; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wa[i], wb[j], acc[i][j], 0,
                                                                     0, 0);
        }
        __builtin_amdgcn_s_setprio(0);
    };
    // lane holds column n0 + wn*64 + 32j + l32 and rows m0 + wm*128 + 32i +
    // 8(r/4) + 4h + r%4.  Widened INT4 products carry a factor 256.
    constexpr int kShift = I8 ? 0 : 8;
    auto epilogue = [&](const GemmTile& tl, int slot) {
        // lane-derived values are recomputed here: hoisted out of the loop
        // they would stay live next to the fragments and accumulators
        int el = lane;
        asm volatile("" : "+v"(el));
        const int l32 = el & 31, h = el >> 5;
        const float* sc = sscale[slot];
        float sw[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) sw[j] = sc[kBM + wn * 64 + j * 32 + l32];
        const int64_t tile_off = tl.m0 * d_out + tl.n0;
        float* yt = y + tile_off;
        int32_t* at = acc_out ? acc_out + tile_off : nullptr;
        const int rows_left = static_cast<int>(n - tl.m0 < BM ? n - tl.m0 : BM);
        const int cols_left = static_cast<int>(d_out - tl.n0 < kBN ? d_out - tl.n0 : kBN);
        if (rows_left == BM && cols_left == kBN && !at && d_out < (int64_t{1} << 29)) {
            // full tile: straight-line code, a wave-uniform row base per
            // accumulator row plus a 32-bit per-lane offset (row 4h, column
            // of fragment j; below 2^32 for d_out < 2^29), no bounds checks
            const uint32_t dout = static_cast<uint32_t>(d_out);
            uint32_t voff[2];
#pragma unroll
            for (int j = 0; j < 2; ++j)
                voff[j] = static_cast<uint32_t>(4 * h) * dout + static_cast<uint32_t>(wn * 64 + j * 32 + l32);
            int rs[2] = {0, 0};
            const float* za = ASYM ? (*sasym)[slot] : nullptr;
            if constexpr (ASYM) {
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    rs[j] = __float_as_int(za[kBM + wn * 64 + j * 32 + l32]);
            }
#pragma unroll
            for (int i = 0; i < IM; ++i) {
                float sx[16], zm[16];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x4 v = *reinterpret_cast<const f32x4*>(sc + wm * (BM / 2) + i * 32 + 8 * q + 4 * h);
#pragma unroll
                    for (int e = 0; e < 4; ++e) sx[4 * q + e] = v[e];
                    if constexpr (ASYM) {
                        const f32x4 z = *reinterpret_cast<const f32x4*>(
                            za + wm * (BM / 2) + i * 32 + 8 * q + 4 * h);
#pragma unroll
                        for (int e = 0; e < 4; ++e) zm[4 * q + e] = z[e];
                    }
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float* yr = yt + static_cast<int64_t>(wm * (BM / 2) + i * 32 + 8 * (r >> 2) + (r & 3)) * d_out;
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const int v = acc[i][j][r] >> kShift;
                        if constexpr (ASYM) {
                            const float t1 = static_cast<float>(v + 8 * rs[j]) * sx[r];
                            const float t2 = zm[r] * static_cast<float>(rs[j]);
                            __builtin_nontemporal_store((t1 + t2) * sw[j], yr + voff[j]);
                        } else {
                            __builtin_nontemporal_store((static_cast<float>(v) * sx[r]) * sw[j], yr + voff[j]);
                        }
                    }
                }
            }
            return;
        }
#pragma unroll
        for (int i = 0; i < IM; ++i) {
            const int rb = wm * (BM / 2) + i * 32 + 4 * h;
            float sx[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(sc + wm * (BM / 2) + i * 32 + 8 * q + 4 * h);
#pragma unroll
                for (int e = 0; e < 4; ++e) sx[4 * q + e] = v[e];
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int col = wn * 64 + j * 32 + l32;
                if (col >= cols_left) continue;
                const int rsj = ASYM ? __float_as_int((*sasym)[slot][kBM + col]) : 0;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = rb + 8 * (r >> 2) + (r & 3);
                    if (row >= rows_left) continue;
                    const int64_t off = static_cast<int64_t>(row) * d_out + col;
                    int v = acc[i][j][r] >> kShift;
                    float yv;
                    if constexpr (ASYM) {
                        v += 8 * rsj;
                        const float t1 = static_cast<float>(v) * sx[r];
                        const float t2 = (*sasym)[slot][row] * static_cast<float>(rsj);
                        yv = (t1 + t2) * sw[j];
                    } else {
                        yv = (static_cast<float>(v) * sx[r]) * sw[j];
                    }
                    __builtin_nontemporal_store(yv, yt + off);
                    if (at) at[off] = v;
                }
            }
        }
    };

    // issue cursor: the next step whose direct loads are requested
    int is_g = 0, is_kt = 0, is_ti = 0;
    GemmTile is_tile;
    gemm_tile<BM>(0, n, d_out, is_tile);
    set_rows(is_tile);
    auto issue_next = [&]() {
        if (is_g >= G) return;
        if (is_kt == 0) issue_scales(is_tile, is_ti % kScaleSlots);
        issue_step(is_kt, is_g % kStages);
        ++is_g;
        if (++is_kt == nk && is_g < G) {
            is_kt = 0;
            ++is_ti;
            gemm_tile<BM>(is_ti, n, d_out, is_tile);
            set_rows(is_tile);
        }
    };
    // waits until this thread's loads of step g have landed, given that the
    // steps after it up to is_g - 1 have been requested
    auto wait_step = [&](int g) {
        if (g >= G) return;
        const int newer = is_g - 1 - g;
        if (newer >= 2) wait_vmcnt<2 * NL>();
        else if (newer == 1) wait_vmcnt<NL>();
        else wait_vmcnt<0>();
    };

    // A phase boundary: the barrier, with nothing scheduled across it (an
    // s_barrier does not stop the compiler from moving MFMAs or ALU work)
    auto phase_end = [&]() {
        __builtin_amdgcn_sched_barrier(0);
        lds_barrier();
        __builtin_amdgcn_sched_barrier(0);
    };

    // prologue: the first kStages - 1 steps, visible to both groups
    const int pre = G < kStages - 1 ? G : kStages - 1;
    for (int g = 0; g < pre; ++g) issue_next();
    wait_vmcnt<0>();
    {
        int kt = 0;
        for (int g = 0; g < pre; ++g) {
            clear_ragged(kt, g % kStages);
            if (++kt == nk) kt = 0;
        }
    }
    lds_barrier();

    // Per tile, 2 nk + 2 phases separated by barriers.  Group 0 loads step i
    // in phase 2i and computes it in phase 2i + 1; group 1 does the same one
    // phase later.  Group 0 stores its half of the tile in phase 2 nk (while
    // group 1 computes the last step), group 1 in phase 2 nk + 1.  Each
    // group runs its own straight-line loop (same barrier count per tile).
    auto zero_acc = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = i32x16{};
    };
    if (grp == 0) {
        int g = 0;   // global index of the tile's first step
        for (int ti = 0; ti < n_tiles; ++ti) {
            GemmTile tl;
            gemm_tile<BM>(ti, n, d_out, tl);
            zero_acc();
            for (int i = 0; i < nk; ++i) {
                issue_next();                        // phase 2i
                load_frags((g + i) % kStages);
                phase_end();
                compute_step();                      // phase 2i + 1
                wait_step(g + i + 1);                // A of the next step
                clear_ragged(i + 1 < nk ? i + 1 : 0, (g + i + 1) % kStages);
                phase_end();
            }
            epilogue(tl, ti % kScaleSlots);          // phase 2 nk
            phase_end();
            phase_end();                             // phase 2 nk + 1
            g += nk;
        }
    } else {
        int g = 0;
        for (int ti = 0; ti < n_tiles; ++ti) {
            GemmTile tl;
            gemm_tile<BM>(ti, n, d_out, tl);
            zero_acc();
            phase_end();                             // phase 0
            for (int i = 0; i < nk; ++i) {
                issue_next();                        // phase 2i + 1
                load_frags((g + i) % kStages);
                wait_step(g + i + 1);                // B of the next step
                phase_end();
                compute_step();                      // phase 2i + 2
                phase_end();
            }
            epilogue(tl, ti % kScaleSlots);          // phase 2 nk + 1
            phase_end();
            g += nk;
        }
    }
}

template <int BM>
__global__ __launch_bounds__(kGemmThreads, kWgPerCu) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ __attribute__((aligned(16))) GemmRing ring;
    __shared__ __attribute__((aligned(16))) GemmScales sscale;
    gemm_body<false, false, BM>(qx, s_x, qw, s_w, n, d_in, d_out, y, acc_out, ring, sscale, nullptr,
                            nullptr, nullptr);
}

template <int BM>
__global__ __launch_bounds__(kGemmThreads, kWgPerCu) void int8_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ __attribute__((aligned(16))) GemmRing ring;
    __shared__ __attribute__((aligned(16))) GemmScales sscale;
    gemm_body<true, false, BM>(qx, s_x, qw, s_w, n, d_in, d_out, y, acc_out, ring, sscale, nullptr,
                           nullptr, nullptr);
}

template <int BM>
__global__ __launch_bounds__(kGemmThreads, kWgPerCu) void w4a4_asym_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out,
    const float* __restrict__ zmin_x, const int32_t* __restrict__ rsum_w) {
    __shared__ __attribute__((aligned(16))) GemmRing ring;
    __shared__ __attribute__((aligned(16))) GemmScales sscale;
    // zmin of a tile's rows and the code sums of its outputs, slots as sscale
    __shared__ __attribute__((aligned(16))) GemmScales sasym;
    gemm_body<false, true, BM>(qx, s_x, qw, s_w, n, d_in, d_out, y, acc_out, ring, sscale, zmin_x,
                           rsum_w, &sasym);
}

static hipError_t launch_gemm(bool i8, const uint8_t* codes_x, const float* s_x,
                              const uint8_t* codes_w, const float* s_w, int64_t n, int64_t d_in,
                              int64_t d_out, float* y, int32_t* acc_out, hipStream_t stream,
                              const float* zmin_x = nullptr, const int32_t* rsum_w = nullptr) {
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    // 256 x 256 tiles, or 128 x 256 when the 256-token tiles leave CUs idle
    // and the 128-token ones still take no more rounds of the grid
    const int64_t tiles_n = (d_out + kBN - 1) / kBN;
    const int64_t T256 = ((n + kBM - 1) / kBM) * tiles_n;
    const int64_t T128 = ((n + kBM / 2 - 1) / (kBM / 2)) * tiles_n;
    // kWgPerCu resident workgroups per CU, a multiple of the XCD count
    const int64_t slots = (static_cast<int64_t>(cus) * kWgPerCu / kXcd) * kXcd;
    const bool small = T256 < slots && (T128 + slots - 1) / slots <= (T256 + slots - 1) / slots;
    const int64_t T = small ? T128 : T256;
    int64_t grid = slots;
    const int64_t t_pad = ((T + kXcd - 1) / kXcd) * kXcd;
    if (grid > t_pad) grid = t_pad;
    if (grid < kXcd) grid = kXcd;
    const dim3 g(static_cast<uint32_t>(grid)), blk(kGemmThreads);
    if (zmin_x) {
        if (small)
            hipLaunchKernelGGL(w4a4_asym_gemm_kernel<kBM / 2>, g, blk, 0, stream, codes_x, s_x,
                               codes_w, s_w, n, d_in, d_out, y, acc_out, zmin_x, rsum_w);
        else
            hipLaunchKernelGGL(w4a4_asym_gemm_kernel<kBM>, g, blk, 0, stream, codes_x, s_x,
                               codes_w, s_w, n, d_in, d_out, y, acc_out, zmin_x, rsum_w);
    } else if (i8) {
        if (small)
            hipLaunchKernelGGL(int8_gemm_kernel<kBM / 2>, g, blk, 0, stream, codes_x, s_x,
                               codes_w, s_w, n, d_in, d_out, y, acc_out);
        else
            hipLaunchKernelGGL(int8_gemm_kernel<kBM>, g, blk, 0, stream, codes_x, s_x, codes_w,
                               s_w, n, d_in, d_out, y, acc_out);
    } else {
        if (small)
            hipLaunchKernelGGL(w4a4_gemm_kernel<kBM / 2>, g, blk, 0, stream, codes_x, s_x,
                               codes_w, s_w, n, d_in, d_out, y, acc_out);
        else
            hipLaunchKernelGGL(w4a4_gemm_kernel<kBM>, g, blk, 0, stream, codes_x, s_x, codes_w,
                               s_w, n, d_in, d_out, y, acc_out);
    }
    return hipGetLastError();
}

hipError_t launch_w4a4_linear(const uint8_t* codes_x, const float* s_x, const uint8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out, float* y,
                              int32_t* acc_out, hipStream_t stream) {
    return launch_gemm(false, codes_x, s_x, codes_w, s_w, n, d_in, d_out, y, acc_out, stream);
}

hipError_t launch_w4a4_linear_asym(const uint8_t* codes_x, const float* s_x, const float* zmin_x,
                                   const uint8_t* codes_w, const float* s_w,
                                   const int32_t* rsum_w, int64_t n, int64_t d_in, int64_t d_out,
                                   float* y, int32_t* acc_out, hipStream_t stream) {
    return launch_gemm(false, codes_x, s_x, codes_w, s_w, n, d_in, d_out, y, acc_out, stream,
                       zmin_x, rsum_w);
}

hipError_t launch_int8_linear(const int8_t* codes_x, const float* s_x, const int8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out, float* y,
                              int32_t* acc_out, hipStream_t stream) {
    return launch_gemm(true, reinterpret_cast<const uint8_t*>(codes_x), s_x,
                       reinterpret_cast<const uint8_t*>(codes_w), s_w, n, d_in, d_out, y, acc_out,
                       stream);
}

}  // namespace catk
