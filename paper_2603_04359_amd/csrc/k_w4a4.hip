// W4A4 integer GEMM with fused dequantization (Sec. 3, eq. 5):
//   acc[t, o] = sum_j qx[t, j] qw[o, j]                   (int32, exact)
//   y[t, o]   = fl32(fl32(acc) * s_x[t]) * s_w[o]
//
// gfx950 int8 MFMA (v_mfma_i32_32x32x32_i8) on INT4 codes.
//
// Tiles: 256 x 256 outputs per workgroup of 512 threads = 8 waves in a
// 2 x 4 grid, each wave 128 x 64 = 4 x 2 MFMA tiles with int32
// accumulators; one workgroup per CU (two waves per SIMD, 132 KiB of LDS).
// One K step covers 128 codes (64 packed bytes per row); a tile reads
// 32 KiB of packed codes per step.
//
// Operand path: packed INT4 tiles go straight from global memory into an
// LDS ring of kStages (4) steps with global_load_lds_dwordx4 (no register
// staging, no LDS store instructions), issued kStages-1 steps ahead of
// use, with one barrier per step that waits for LDS traffic only (a plain
// workgroup barrier would also drain the loads in flight).  Each lane reads
// 16 packed bytes (32 codes, two MFMA steps) per fragment and widens them
// in registers to int8 values 16*code: a packed dword (8 codes) becomes one
// dword of its low nibbles and one of its high nibbles, two bit operations
// each.  The widening of the next 32-code step is independent of the MFMAs
// of the current one, so it co-issues with them.  Both operands are widened
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
// lane loads the global unit that belongs in its slot
// (a permutation inside each 64-byte row segment).  Rows past the end of a
// matrix load a clamped in-bounds row (their outputs are never stored);
// units past d_in in a ragged last step load any in-bounds unit and the
// loading thread clears them in LDS before the step's barrier, which
// zeroes their products.
//
// Persistent launch: kWgPerCu workgroups per CU walk lists of tiles in an
// XCD-aware order (workgroups are dealt to the 8 XCDs round-robin; those of
// XCD x walk one contiguous range of tiles, in groups of kGroupM row
// panels, so tiles resident on one XCD share panels in its L2).  The
// operand steps of consecutive tiles form one stream through the ring, and
// the tile's scales are staged in LDS with the first step, so the epilogue
// reads no global memory and the next tile never waits behind the output
// stores.  Output rows stream out with nontemporal stores.
#include "device_common.h"
#include "kernels.h"

namespace catk {

constexpr int kGemmWaves = 8;
constexpr int kGemmThreads = kGemmWaves * 64;
constexpr int kBM = 256;           // tokens per tile
constexpr int kBN = 256;           // outputs per tile
constexpr int kKBP = 64;           // packed bytes per row per K step (128 codes)
constexpr int kUP = kKBP / 16;     // 16-byte units per row per step
constexpr int kStages = 4;         // LDS ring depth (steps)
constexpr int kAUnits = kBM * kUP;                   // A units per stage
constexpr int kBUnits = kBN * kUP;                   // B units per stage
constexpr int kLoadsA = kAUnits / kGemmThreads;      // direct loads per thread, A
constexpr int kLoadsB = kBUnits / kGemmThreads;      // direct loads per thread, B
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

__device__ __forceinline__ bool gemm_tile(int64_t k, int64_t n, int64_t d_out, GemmTile& t) {
    const int64_t tiles_m = (n + kBM - 1) / kBM;
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
    t.m0 = (first_m + in_group % gm) * kBM;
    t.n0 = (in_group / gm) * kBN;
    return true;
}

__device__ __forceinline__ i32x4 widen8(u32x4 v, int half) {
    const uint32_t w0 = v[2 * half], w1 = v[2 * half + 1];
    return i32x4{static_cast<int>(unpack_lo16(w0)), static_cast<int>(unpack_hi16(w0)),
                 static_cast<int>(unpack_lo16(w1)), static_cast<int>(unpack_hi16(w1))};
}

__global__ __launch_bounds__(kGemmThreads, kWgPerCu) void w4a4_gemm_kernel(
    const uint8_t* __restrict__ qx, const float* __restrict__ s_x,
    const uint8_t* __restrict__ qw, const float* __restrict__ s_w, int64_t n, int64_t d_in,
    int64_t d_out, float* __restrict__ y, int32_t* __restrict__ acc_out) {
    __shared__ __attribute__((aligned(16))) u32x4 ring_a[kStages][kAUnits];
    __shared__ __attribute__((aligned(16))) u32x4 ring_b[kStages][kBUnits];
    // s_x of the tile's rows and s_w of its outputs, double-buffered by tile
    __shared__ __attribute__((aligned(16))) float sscale[2][kBM + kBN];

    const int64_t row_bytes = d_in / 2;
    const int nk = static_cast<int>((row_bytes + kKBP - 1) / kKBP);

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1);
    const int wave = tid / kWave;
    const int wm = wave >> 2, wn = wave & 3;   // 2 x 4 waves, each 128 x 64
    const int l32 = lane & 31;
    const int h = lane >> 5;

    // Direct loads: instruction q of wave w fills slots [64 I, 64 I + 64)
    // with I = q * 8 + w (16 rows of 64 bytes); slot s holds row s / 4,
    // logical unit (s % 4) ^ swz(row).  32-bit offsets from the tile's
    // first row.
    const uint8_t* a_base = qx;
    const uint8_t* b_base = qw;
    uint32_t a_off[kLoadsA], b_off[kLoadsB];
    // the byte offset of a thread's unit inside its row segment is the same
    // for every load q (64 slots per instruction keep row / 8 and slot % 8)
    const int u_off = ((lane % kUP) ^ gemm_swz((wave * 64 + lane) / kUP)) * 16;
    static_assert((64 / kUP) % 16 == 0, "swz(row) must not depend on the instruction");
    auto set_rows = [&](const GemmTile& tl) {
        a_base = qx + tl.m0 * row_bytes;
        b_base = qw + tl.n0 * row_bytes;
#pragma unroll
        for (int q = 0; q < kLoadsA; ++q) {
            const int r = ((q * kGemmWaves + wave) * 64 + lane) / kUP;
            const int64_t ra = tl.m0 + r < n ? r : n - 1 - tl.m0;   // clamped rows: never stored
            a_off[q] = static_cast<uint32_t>(ra * row_bytes);
        }
#pragma unroll
        for (int q = 0; q < kLoadsB; ++q) {
            const int r = ((q * kGemmWaves + wave) * 64 + lane) / kUP;
            const int64_t rb = tl.n0 + r < d_out ? r : d_out - 1 - tl.n0;
            b_off[q] = static_cast<uint32_t>(rb * row_bytes);
        }
    };
    // LDS byte addresses of this wave's first slot in stage 0 (wave-uniform)
    const uint32_t lds_a0 = static_cast<uint32_t>(
        __builtin_amdgcn_readfirstlane(lds_addr(&ring_a[0][wave * 64])));
    const uint32_t lds_b0 = static_cast<uint32_t>(
        __builtin_amdgcn_readfirstlane(lds_addr(&ring_b[0][wave * 64])));
    auto issue = [&](int kt, int st) {
        const int64_t k0 = static_cast<int64_t>(kt) * kKBP;
        const uint32_t la = lds_a0 + static_cast<uint32_t>(st) * (kAUnits * 16);
        const uint32_t lb = lds_b0 + static_cast<uint32_t>(st) * (kBUnits * 16);
        if (k0 + kKBP <= row_bytes) {
            const uint32_t k0u = static_cast<uint32_t>(k0);
#pragma unroll
            for (int q = 0; q < kLoadsA; ++q)
                dma16(a_base, a_off[q] + k0u + u_off, la + q * (kGemmWaves * 1024u));
#pragma unroll
            for (int q = 0; q < kLoadsB; ++q)
                dma16(b_base, b_off[q] + k0u + u_off, lb + q * (kGemmWaves * 1024u));
        } else {
#pragma unroll
            for (int q = 0; q < kLoadsA; ++q) {
                int64_t col = k0 + u_off;
                col = col < row_bytes ? col : 0;     // past the row end: any in-bounds unit
                dma16(a_base, a_off[q] + static_cast<uint32_t>(col), la + q * (kGemmWaves * 1024u));
            }
#pragma unroll
            for (int q = 0; q < kLoadsB; ++q) {
                int64_t col = k0 + u_off;
                col = col < row_bytes ? col : 0;
                dma16(b_base, b_off[q] + static_cast<uint32_t>(col), lb + q * (kGemmWaves * 1024u));
            }
        }
    };
    constexpr int kLoadsPerStep = kLoadsA + kLoadsB;

    i32x16 acc[4][2];

    // Fragments: lane half h reads logical units 2h and 2h+1 (c = 0, 1) of
    // its row; each unit feeds two MFMA steps (its low and high 8 bytes).
    // Both operands use the same assignment, so the reduction index is only
    // permuted.
    struct Packed {
        u32x4 a[4], b[2];
    };
    struct Wide {
        i32x4 a[4], b[2];
    };
    auto read_packed = [&](Packed& p, int st, int c) {
        const int u = 2 * h + c;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = wm * 128 + i * 32 + l32;
            p.a[i] = ring_a[st][r * kUP + (u ^ gemm_swz(r))];
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int r = wn * 64 + j * 32 + l32;
            p.b[j] = ring_b[st][r * kUP + (u ^ gemm_swz(r))];
        }
    };
    auto widen = [&](Wide& w, const Packed& p, int half) {
#pragma unroll
        for (int i = 0; i < 4; ++i) w.a[i] = widen8(p.a[i], half);
#pragma unroll
        for (int j = 0; j < 2; ++j) w.b[j] = widen8(p.b[j], half);
    };
    auto mfma16 = [&](const Wide& w) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(w.a[i], w.b[j], acc[i][j], 0, 0,
                                                                 0);
    };
    // one K step = 4 MFMA steps of 32 codes; the widening of MFMA step
    // m+1 is issued before the 16 MFMAs of step m
    auto compute = [&](int st) {
        Packed p;
        Wide w0, w1;
        read_packed(p, st, 0);
        widen(w0, p, 0);
        widen(w1, p, 1);
#pragma unroll
        for (int c = 1; c < kUP / 2; ++c) {
            read_packed(p, st, c);
            mfma16(w0);
            widen(w0, p, 0);
            mfma16(w1);
            widen(w1, p, 1);
        }
        mfma16(w0);
        mfma16(w1);
    };

    // s_x / s_w of a tile into its scale slot: 64 dwords per wave
    // instruction (rows / outputs past the end load the last one; their
    // outputs are never stored).  Issued before the tile's first operand
    // step, so waiting for that step covers them.
    auto issue_scales = [&](const GemmTile& tl, int slot) {
        if (wave < 4) {
            const int64_t r = tl.m0 + 64 * wave + lane;
            dma4(s_x, static_cast<uint32_t>((r < n ? r : n - 1) * 4),
                 lds_addr(&sscale[slot][64 * wave]));
        } else {
            const int64_t o = tl.n0 + 64 * (wave - 4) + lane;
            dma4(s_w, static_cast<uint32_t>((o < d_out ? o : d_out - 1) * 4),
                 lds_addr(&sscale[slot][kBM + 64 * (wave - 4)]));
        }
    };

    // The operand steps of consecutive tiles form one stream through the
    // ring: during a tile's last steps the first steps of the next tile
    // (and its scales) are already requested, and they have landed before
    // the tile's output is stored, so the next tile starts without waiting
    // behind those stores.
    GemmTile cur;
    if (!gemm_tile(0, n, d_out, cur)) return;
    const int pre_n = nk < kStages - 1 ? nk : kStages - 1;   // steps requested ahead of a tile
    int sp = 0;      // scale slot of the current tile
    int base = 0;    // ring stage of the current tile's step 0
    set_rows(cur);
    issue_scales(cur, sp);
    for (int j = 0; j < pre_n; ++j) issue(j, j);
    wait_vmcnt<0>();
    lds_barrier();

    for (int64_t k = 0;; ++k) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = i32x16{};
        GemmTile nxt;
        const bool more = gemm_tile(k + 1, n, d_out, nxt);
        int nx_issued = 0;   // steps of the next tile requested so far

        for (int kt = 0; kt < nk; ++kt) {
            const int st = (base + kt) % kStages;
            if (kt >= pre_n) {
                // this thread's loads of step kt have landed once at most the
                // loads of the one step requested after it are outstanding
                const int last = nk - 1 + (more ? pre_n : 0);   // last step requested in this tile
                const int issued = kt + kStages - 2 < last ? kt + kStages - 2 : last;
                const int ahead = issued - kt;
                if (ahead >= 2) wait_vmcnt<2 * kLoadsPerStep>();
                else if (ahead == 1) wait_vmcnt<kLoadsPerStep>();
                else wait_vmcnt<0>();
            }
            if (kt == nk - 1 && (row_bytes % kKBP) != 0) {
                // ragged last step: codes past d_in read garbage; zero them in
                // A (each thread clears the slots its own loads filled)
#pragma unroll
                for (int q = 0; q < kLoadsA; ++q)
                    if (static_cast<int64_t>(kt) * kKBP + u_off >= row_bytes)
                        ring_a[st][(q * kGemmWaves + wave) * 64 + lane] = u32x4{0u, 0u, 0u, 0u};
            }
            lds_barrier();     // all threads' loads of step kt landed; step kt-1 consumed
            const int tgt = kt + kStages - 1;
            if (tgt < nk) {
                issue(tgt, (base + tgt) % kStages);
            } else if (more && nx_issued < pre_n && nx_issued <= tgt - nk) {
                // the next tile's steps, in order; step j's stage last held
                // this tile's step nk + j - kStages <= kt - 1 (consumed)
                const int j = nx_issued;
                if (j == 0) {
                    set_rows(nxt);
                    issue_scales(nxt, sp ^ 1);
                }
                issue(j, (base + nk + j) % kStages);
                nx_issued = j + 1;
            }
            compute(st);
        }
        if (more) {
            for (int j = nx_issued; j < pre_n; ++j) {   // only when nk < kStages - 1
                if (j == 0) {
                    set_rows(nxt);
                    issue_scales(nxt, sp ^ 1);
                }
                issue(j, (base + nk + j) % kStages);
            }
            wait_vmcnt<0>();   // the next tile's first steps and scales have landed
        }
        lds_barrier();         // stages of this tile consumed; next tile's first steps visible

        // ---- epilogue: lane holds column n0 + wn*64 + 32j + l32 and rows
        // m0 + wm*128 + 32i + 8(r/4) + 4h + r%4
        const float* sc = sscale[sp];
        float sw[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) sw[j] = sc[kBM + wn * 64 + j * 32 + l32];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t tb = cur.m0 + wm * 128 + i * 32 + 4 * h;
            float sx[16];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(sc + wm * 128 + i * 32 + 8 * q + 4 * h);
#pragma unroll
                for (int e = 0; e < 4; ++e) sx[4 * q + e] = v[e];
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int64_t o = cur.n0 + wn * 64 + j * 32 + l32;
                if (o >= d_out) continue;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int64_t t = tb + 8 * (r >> 2) + (r & 3);
                    if (t >= n) continue;
                    const int v = acc[i][j][r] >> 8;
                    const float yv = (static_cast<float>(v) * sx[r]) * sw[j];
                    __builtin_nontemporal_store(yv, y + t * d_out + o);
                    if (acc_out) acc_out[t * d_out + o] = v;
                }
            }
        }
        if (!more) break;
        cur = nxt;
        sp ^= 1;
        base = (base + nk) % kStages;
    }
}

hipError_t launch_w4a4_linear(const uint8_t* codes_x, const float* s_x, const uint8_t* codes_w,
                              const float* s_w, int64_t n, int64_t d_in, int64_t d_out, float* y,
                              int32_t* acc_out, hipStream_t stream) {
    int dev = 0, cus = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    err = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (err != hipSuccess) return err;
    const int64_t T = ((n + kBM - 1) / kBM) * ((d_out + kBN - 1) / kBN);
    // kWgPerCu resident workgroups per CU, a multiple of the XCD count
    int64_t grid = (static_cast<int64_t>(cus) * kWgPerCu / kXcd) * kXcd;
    const int64_t t_pad = ((T + kXcd - 1) / kXcd) * kXcd;
    if (grid > t_pad) grid = t_pad;
    if (grid < kXcd) grid = kXcd;
    hipLaunchKernelGGL(w4a4_gemm_kernel, dim3(static_cast<uint32_t>(grid)), dim3(kGemmThreads), 0,
                       stream, codes_x, s_x, codes_w, s_w, n, d_in, d_out, y, acc_out);
    return hipGetLastError();
}

}  // namespace catk
