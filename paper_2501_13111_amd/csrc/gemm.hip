// Prefill projections: tiled GEMM  C[M, N] = X[M, K] . W[N, K]^T on MFMA, with the
// weight tile dequantised while it is staged into LDS and the layer's elementwise
// work fused into the epilogue.
//
// Prefill (the fingerprint's time to first token, paper Sec. 5.3) runs every
// prompt token through the projections at once, so it is a dense contraction
// and belongs on the matrix cores.  Weight-only quantised tiles (Sec. 3.2) are
// converted to 16-bit on the way into LDS (small tiling) or per MFMA fragment
// after the LDS read (large tiling, where LDS holds the packed codes):
//   bf16 W: copied; A operand bf16                   (bf16 MFMA)
//   int8 W: codes -> exact fp16; per-row scale in the epilogue    (fp16 MFMA)
//   int4 W: small tiling fp16((q - z) * s), one rounding per weight; large tiling
//           exact q - z with the group scale on the fp32 accumulators  (fp16 MFMA)
// Epilogues: fp32 store (q, k, v before the rotary embedding), residual
// out = bf16(resid + acc), and SwiGLU a = bf16(silu(gate) * up) where each wave
// holds gate and up columns of the same f (dual tiles over [gate; up]).
//
// Weights are read from the fragment-major layout (1 KiB blocks of 16 rows x one
// K-step), so each 64-thread group of a tile load reads contiguous memory.
//
// Two tilings:
//  * small problems (few 256 x 256 tiles): 128 (or 64) x 128 x 64 tiles, 4 waves in
//    2 x 2, each 64 (32) x 64; the next K tiles are loaded into a ring of registers
//    (and dequantised on the way to LDS) while the current one is multiplied;
//  * large problems: 256 x 256 tiles, 8 waves in 2 x 4, each 128 x 64, operands
//    copied global -> LDS by buffer loads that write LDS directly, two LDS stages.
// Both multiply with 32x32x16 MFMAs, which run at about 1.4x the rate of 16x16x32
// on this part.
// Both map workgroups to tiles XCD-aware: workgroups are dealt to the 8 XCDs
// round-robin, and each XCD takes a contiguous range of a grouped raster so its
// L2 sees the same A row tiles and weight column tiles again.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

constexpr int GBN = 128, GBK = 64, GPAD = 8;
#ifndef GEMM_BIG_MIN_TILES
#define GEMM_BIG_MIN_TILES 128   // 256 x 256 tiles from this many
#endif
#ifndef GEMM_GM
#define GEMM_GM 2                // tile rows per group of the grouped raster (256-row tiles: a
                                 // group keeps 2 activation row-tiles per XCD in flight)
#endif
#ifndef GEMM_SMALL_TILES
#define GEMM_SMALL_TILES 256
#endif
constexpr int GLD = GBK + GPAD;   // LDS row (u16)

// BM = 128 (waves 2 x 2 of 64 x 64) or 64 (waves 2 x 2 of 32 x 64, for problems with
// too few 128-row tiles to fill the GPU)
template <int WF, int EPI, int BM, int RD>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a) {
    static_assert(RD % 2 == 0, "the LDS buffer parity of a tile is fixed within the unrolled ring");
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    constexpr int TI = BM / 64;                 // 32-row MFMA tiles per wave
    constexpr int NA = BM / 32;                 // 16-byte A loads per thread per K tile
    __shared__ __attribute__((aligned(16))) uint16_t Asb[2][BM * GLD];
    __shared__ __attribute__((aligned(16))) uint16_t Bsb[2][GBN * GLD];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int wm = w >> 1, wn = w & 1;
    // tile of this workgroup: XCD-aware, grouped raster.  Workgroups are dealt to the
    // 8 XCDs round-robin; each XCD takes a contiguous range of the grouped tile order
    // so that its L2 sees the same A row tiles and B column tiles again.
    int mt, nb;
    {
        const int T = a.tiles_m * a.tiles_n, bid = blockIdx.x;
        const int x = bid & 7, j = bid >> 3, q = T >> 3, rm = T & 7;
        const int t = x * q + (x < rm ? x : rm) + j;
        const int GM = GEMM_GM;
        const int grp = t / (GM * a.tiles_n);
        const int gm0 = grp * GM;
        const int gsz = min(GM, a.tiles_m - gm0);
        const int tt = t - grp * GM * a.tiles_n;
        mt = gm0 + tt % gsz;
        nb = tt / gsz;
    }
    const int m0 = mt * BM;

    // global row of B-tile row lr (plain: n0 + lr; dual: gate / up rows of 64 f's)
    auto brow = [&](int lr, bool& valid) -> int {
        if constexpr (EPI == EPI_SWIGLU) {
            const int wnn = lr >> 6, ni = (lr & 63) >> 4, rr = lr & 15;
            const int f = nb * 64 + 32 * wnn + 16 * (ni & 1) + rr;
            valid = f < a.F;
            return (ni >> 1) * a.F + f;
        } else {
            const int n = nb * GBN + lr;
            valid = n < a.N;
            return n;
        }
    };

    // ---- register staging of one K tile
    constexpr int BCH = (WF == W_BF16) ? 4 : (WF == W_INT8 ? 2 : 1);   // 16-byte B loads per thread
    struct Stage {
        u32x4 ra[NA], rb[BCH];
        uint32_t sz;              // int4: scale | zero << 16 of the lane's row and group
    };
    // Loads are unconditional (clamped addresses) so the compiler can count them across
    // the loop and keep several tiles in flight: rows past M or N only feed outputs that
    // are never stored; activation pieces past K are zeroed (the weights there are
    // padding or a clamped copy), which only happens in a ragged last tile.
    auto load_tile = [&](int k0, Stage& sg) {
        u32x4* ra = sg.ra;
        u32x4* rb = sg.rb;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + 256 * i;
            const int row = c >> 3, kc = (c & 7) * 8;
            const int m = min(m0 + row, a.M - 1), k = min(k0 + kc, a.K - 8);
            ra[i] = *(const u32x4*)(a.X + (int64_t)m * a.K + k);
        }
        if (k0 + GBK > a.K) {
#pragma unroll
            for (int i = 0; i < NA; ++i)
                if (k0 + ((tid + 256 * i) & 7) * 8 >= a.K) ra[i] = u32x4{0u, 0u, 0u, 0u};
        }
        // B: fragment-major tiles -- each 64-thread group reads one contiguous 1 KiB block
        // (16 rows x one K-step); chunk L = r + 16 g holds row r, k-slice g of the block.
        const u32x4* Wt = (const u32x4*)a.W;
        if constexpr (WF == W_BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {                  // 8 subtiles x 2 K-steps of 32
                const int c = tid + 256 * i;
                const int blk = c >> 6, L = c & 63, ntl = blk >> 1, kst = blk & 1;
                const int lr = 16 * ntl + (L & 15);
                bool v;
                int n = brow(lr, v);
                n = v ? n : 0;
                rb[i] = Wt[((int64_t)(n >> 4) * a.kst + min((k0 + 32 * kst) / 32, a.kst - 1)) * 64 + L];
            }
        } else if constexpr (WF == W_INT8) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {                  // 8 subtiles x 1 K-step of 64
                const int c = tid + 256 * i;
                const int ntl = c >> 6, L = c & 63;
                const int lr = 16 * ntl + (L & 15);
                bool v;
                int n = brow(lr, v);
                n = v ? n : 0;
                rb[i] = Wt[((int64_t)(n >> 4) * a.kst + min(k0 / 64, a.kst - 1)) * 64 + L];
            }
        } else {                                           // 8 subtiles x half a K-step of 128
            const int ntl = tid >> 5, j = tid & 31;
            const int lr = 16 * ntl + (j & 15);
            const int gg = j >> 4, g = gg + 2 * ((k0 >> 6) & 1);
            bool v;
            int n = brow(lr, v);
            n = v ? n : 0;
            rb[0] = Wt[((int64_t)(n >> 4) * a.kst + k0 / 128) * 64 + (j & 15) + 16 * g];
            sg.sz = a.sz[(int64_t)(k0 / 128) * a.N + n];
        }
    };
    auto store_tile = [&](uint16_t* As, uint16_t* Bs, const Stage& sg) {
        const u32x4* ra = sg.ra;
        const u32x4* rb = sg.rb;
#pragma unroll
        for (int i = 0; i < NA; ++i) {
            const int c = tid + 256 * i;
            *(u32x4*)(As + (c >> 3) * GLD + (c & 7) * 8) = ra[i];
        }
        if constexpr (WF == W_BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int c = tid + 256 * i;
                const int blk = c >> 6, L = c & 63;
                *(u32x4*)(Bs + (16 * (blk >> 1) + (L & 15)) * GLD + 32 * (blk & 1) + 8 * (L >> 4)) = rb[i];
            }
        } else if constexpr (WF == W_INT8) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int c = tid + 256 * i;
                const int L = c & 63;
                uint16_t* dst = Bs + (16 * (c >> 6) + (L & 15)) * GLD + 16 * (L >> 4);
                const u32x2 c0 = i8x4_to_f16x4(rb[i].x), c1 = i8x4_to_f16x4(rb[i].y);
                const u32x2 c2 = i8x4_to_f16x4(rb[i].z), c3 = i8x4_to_f16x4(rb[i].w);
                *(u32x4*)(dst) = u32x4{c0.x, c0.y, c1.x, c1.y};
                *(u32x4*)(dst + 8) = u32x4{c2.x, c2.y, c3.x, c3.y};
            }
        } else {
            uint16_t* dst = Bs + (16 * (tid >> 5) + (tid & 15)) * GLD + 32 * ((tid >> 4) & 1);
            const _Float16 bz = (_Float16)(1024.0f + h2f((uint16_t)(sg.sz >> 16)));
            const f16x2 bias = {bz, bz};
            const _Float16 sh = __builtin_bit_cast(_Float16, (uint16_t)(sg.sz & 0xFFFFu));
            const f16x2 sc = {sh, sh};
            const uint32_t wd[4] = {rb[0].x, rb[0].y, rb[0].z, rb[0].w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const u32x4 q = i4x8_to_f16x8(wd[j], bias);   // exact (q - z)
                *(u32x4*)(dst + 8 * j) =
                    u32x4{mul_h2(q.x, sc), mul_h2(q.y, sc), mul_h2(q.z, sc), mul_h2(q.w, sc)};
            }
        }
    };

    // 32x32 MFMA tiles: TI (rows) x 2 (columns) per wave; lane l holds column l % 32
    f32x16 acc[TI][2];
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

    const int l32 = lane & 31, h32 = lane >> 5;
    const int nk = (a.K + GBK - 1) / GBK;
    auto compute = [&](const uint16_t* As, const uint16_t* Bs) {
#pragma unroll
        for (int kk = 0; kk < GBK / 16; ++kk) {
            u32x4 af[TI], bf[2];
#pragma unroll
            for (int i = 0; i < TI; ++i)
                af[i] = *(const u32x4*)(As + (wm * (BM / 2) + 32 * i + l32) * GLD + 16 * kk + 8 * h32);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[j] = *(const u32x4*)(Bs + (wn * 64 + 32 * j + l32) * GLD + 16 * kk + 8 * h32);
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32<AF>(af[i], bf[j], acc[i][j]);
        }
    };
    // LDS writes done, then a bare barrier: the global loads in flight are not drained
    auto barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

    // K tiles are loaded into a ring of RD register stages, RD tiles ahead, and written
    // to the other LDS buffer while the current one is multiplied (tile t lives in
    // stage t % RD)
    // Every trip issues the same memory operations (tile indexes past the end are
    // clamped, their copies never read), so the compiler's wait counts stay exact and
    // the ring stays in flight; only the MFMA work is skipped past the last tile.
    Stage st[RD];
#pragma unroll
    for (int q = 0; q < RD; ++q) load_tile(min(q, nk - 1) * GBK, st[q]);
    store_tile(Asb[0], Bsb[0], st[0]);
    load_tile(min(RD, nk - 1) * GBK, st[0]);
    barrier();
    for (int kt0 = 0; kt0 < nk; kt0 += RD) {
#pragma unroll
        for (int q = 0; q < RD; ++q) {
            const int kt = kt0 + q;
            const int nq = (q + 1) % RD;
            if (kt < nk) compute(Asb[q & 1], Bsb[q & 1]);
            store_tile(Asb[(q + 1) & 1], Bsb[(q + 1) & 1], st[nq]);
            load_tile(min(kt + 1 + RD, nk - 1) * GBK, st[nq]);
            barrier();
        }
    }

    // ---- epilogue (accumulator element e of lane l: row 8 (e / 4) + 4 (l / 32) + e % 4 of
    // the 32x32 tile, column l % 32); dual tiles: column tile 0 is gate, 1 is up, same f
    if constexpr (EPI == EPI_SWIGLU) {
        const int f = nb * 64 + 32 * wn + l32;
        if (f < a.F) {
            float sg = 1.f, su = 1.f;
            if constexpr (WF == W_INT8) {
                sg = h2f(a.scales[f]);
                su = h2f(a.scales[a.F + f]);
            }
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int m = m0 + wm * (BM / 2) + 32 * i + 8 * (e >> 2) + 4 * h32 + (e & 3);
                    if (m >= a.M) continue;
                    const float gv = acc[i][0][e] * sg, uv = acc[i][1][e] * su;
                    a.out16[(int64_t)m * a.F + f] = act_store(bfround(silu_f(gv) * uv), a.out_fmt);
                }
        }
    } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = nb * GBN + wn * 64 + 32 * j + l32;
            if (n >= a.N) continue;
            float sn = 1.f;
            if constexpr (WF == W_INT8) sn = h2f(a.scales[n]);
#pragma unroll
            for (int i = 0; i < TI; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int m = m0 + wm * (BM / 2) + 32 * i + 8 * (e >> 2) + 4 * h32 + (e & 3);
                    if (m >= a.M) continue;
                    const float v = acc[i][j][e] * sn;
                    if constexpr (EPI == EPI_F32) a.out32[(int64_t)m * a.N + n] = v;
                    else a.out16[(int64_t)m * a.N + n] = f2bf(bf2f(a.resid[(int64_t)m * a.N + n]) + v);
                }
        }
    }
}

// register ring depth: deeper for 64-row tiles (one workgroup per CU, nothing else to
// hide the load latency)
#ifndef GEMM_RD64
#define GEMM_RD64 4
#endif
#ifndef GEMM_RD128
#define GEMM_RD128 2
#endif
template <int WF, int BM, int RD = (BM == 64 ? GEMM_RD64 : GEMM_RD128)>
static hipError_t launch_wm(const GemmArgs& a, int epi, hipStream_t st) {
    GemmArgs b = a;
    b.tiles_n = (epi == EPI_SWIGLU) ? (a.F + 63) / 64 : (a.N + GBN - 1) / GBN;
    b.tiles_m = (a.M + BM - 1) / BM;
    dim3 grid(b.tiles_n * b.tiles_m);
    switch (epi) {
        case EPI_F32: FP_LAUNCH((gemm_kernel<WF, EPI_F32, BM, RD>), grid, dim3(256), 0, st, b); break;
        case EPI_RESID: FP_LAUNCH((gemm_kernel<WF, EPI_RESID, BM, RD>), grid, dim3(256), 0, st, b); break;
        case EPI_SWIGLU: FP_LAUNCH((gemm_kernel<WF, EPI_SWIGLU, BM, RD>), grid, dim3(256), 0, st, b); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// 64-row tiles when 128-row tiles would leave most of the 256 CUs idle
template <int WF>
static hipError_t launch_w(const GemmArgs& a, int epi, hipStream_t st) {
    const int tn = (epi == EPI_SWIGLU) ? (a.F + 63) / 64 : (a.N + GBN - 1) / GBN;
    const int t128 = tn * ((a.M + 127) / 128);
    if (t128 < GEMM_SMALL_TILES) return launch_wm<WF, 64>(a, epi, st);
    return launch_wm<WF, 128>(a, epi, st);
}

hipError_t launch_gemm_small(const GemmArgs& a, int wf, int epi, hipStream_t st) {
    switch (wf) {
        case W_BF16: return launch_w<W_BF16>(a, epi, st);
        case W_INT8: return launch_w<W_INT8>(a, epi, st);
        case W_INT4: return launch_w<W_INT4>(a, epi, st);
        default: return hipErrorInvalidValue;
    }
}


// ---------------------------------------------------------------------------
// Large prefill GEMMs: 256 x 256 tiles, 8 waves of 128 x 64 (4 x 2 32x32 MFMA tiles),
// operands copied global -> LDS by buffer loads that write LDS directly (16 B per
// lane), two LDS stages; the next stage's copies are issued in parts between the
// MFMA steps of the first half of the current stage.  A rows are stored with an XOR swizzle of their 16-byte
// chunks so that MFMA fragment reads are free of bank conflicts; weight blocks
// keep their fragment-major order, so a fragment is one contiguous 1 KiB read.
// Quantised weights stay packed in LDS and are converted to fp16 per fragment.  For the
// int4 qkv projection (fp32 output, whose K / V rows become cache codes) the fragments hold
// the exact integers q - z, and the group scale goes to the fp32 accumulators instead: a
// stage is one 128-input group, and a lane's accumulators of a 32x32 tile all belong to
// one output column (one scale), so before each stage the lane re-expresses them in units
// of that stage's scale (acc *= s_prev / s_cur) and the epilogue multiplies by the last
// one; no weight is rounded to fp16.  The other int4 projections (o, [gate; up], down)
// multiply the exact q - z by the group scale in fp16 instead -- the dequantised weight
// rounded once to fp16, relative error at most 2^-11 -- which takes one packed multiply
// per two weights instead of the rescaling of 128 accumulators per lane every stage.  The
// fragments take one shift per word (i4x8_to_f16x8_q).

// int4 projections other than qkv: weights (q - z) * s rounded to fp16 (0: every int4
// projection takes the exact scheme)
#ifndef GEMM_FASTQ
#define GEMM_FASTQ 1
#endif
constexpr int BT = 256;
template <int WF>
struct BigT {
    static constexpr int TK = (WF == W_INT4) ? 128 : 64;                             // k per stage
    static constexpr int KSW = (WF == W_BF16) ? 32 : (WF == W_INT8 ? 64 : 128);     // weight K-step
    static constexpr int NBLK = TK / KSW;                                            // blocks per row-block per stage
    static constexpr int A_BYTES = BT * TK * 2;
    static constexpr int B_BYTES = 16 * NBLK * 1024;
    static constexpr int STAGE = A_BYTES + B_BYTES;
    static constexpr int CPR = TK / 8;                                               // 16-byte chunks per A row
    static constexpr int NSUB = TK / 32;                                             // MFMA k-steps per stage
    // LDS: two stages, reused by the epilogue (the residual epilogue stages 8 waves x 64 rows
    // x 72 floats; one workgroup per CU either way)
    static constexpr int EPI_BYTES = 8 * 64 * 72 * 4;
    static constexpr int SMEM = 2 * STAGE > EPI_BYTES ? 2 * STAGE : EPI_BYTES;
};

// Eight int4 codes of one word (device nibble order) -> exact fp16 q - z, one shift: the
// nibbles in bits 0-3 of each 16-bit half become fp16 1024 + q (exponent 0x64), those in bits
// 4-7 become 64 + q (exponent 0x54, whose ulp is 1/16); b1024 = 1024 + z, b64 = 64 + z.
// Same values, in the same order, as i4x8_to_f16x8.
__device__ __forceinline__ u32x4 i4x8_to_f16x8_q(uint32_t w, f16x2 b1024, f16x2 b64) {
    const uint32_t w8 = w >> 8;
    const uint32_t p0 = and_or(w, 0x000F000Fu, 0x64006400u);
    const uint32_t p1 = and_or(w, 0x00F000F0u, 0x54005400u);
    const uint32_t p2 = and_or(w8, 0x000F000Fu, 0x64006400u);
    const uint32_t p3 = and_or(w8, 0x00F000F0u, 0x54005400u);
    u32x4 r;
    r.x = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p0) - b1024);
    r.y = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p1) - b64);
    r.z = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p2) - b1024);
    r.w = __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, p3) - b64);
    return r;
}

template <int CPR>
__device__ __forceinline__ int a_swz(int row) { return CPR == 8 ? ((row >> 1) & 7) : (row & 15); }

template <int WF, int EPI, bool DUAL>
__global__ void __launch_bounds__(512, 1) gemm_big_kernel(GemmArgs a) {
    using T = BigT<WF>;
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    static_assert(DUAL == (EPI == EPI_SWIGLU) || EPI == EPI_PART, "dual tiling");
    __shared__ __attribute__((aligned(1024))) char smem[T::SMEM];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int wm = w >> 2, wn = w & 3;      // 2 x 4 waves, each 128 x 64
    int mt, nt;
    {
        const int Tn = a.tiles_m * a.tiles_n, bid = blockIdx.x;
        const int x = bid & 7, j = bid >> 3, q = Tn >> 3, rm = Tn & 7;
        const int t = x * q + (x < rm ? x : rm) + j;
        const int GM = GEMM_GM;
        const int grp = t / (GM * a.tiles_n);
        const int gm0 = grp * GM;
        const int gsz = min(GM, a.tiles_m - gm0);
        const int tt = t - grp * GM * a.tiles_n;
        mt = gm0 + tt % gsz;
        nt = tt / gsz;
    }
    const int m0 = mt * BT;
    const int nrb = DUAL ? a.F / 16 : (a.N + 15) / 16;    // valid (gate) row-blocks

    // global row-block of LDS row-block rb
    auto grow_block = [&](int rb, bool& v) -> int {
        if constexpr (DUAL) {
            const int fb = nt * 8 + (rb & 7);
            v = fb < nrb;
            return rb < 8 ? fb : nrb + fb;
        } else {
            const int b = nt * 16 + rb;
            v = b < nrb;
            return b;
        }
    };
    // LDS row-block of this wave's column tile j
    auto col_rb = [&](int j) -> int {
        if constexpr (DUAL) return j < 2 ? wn * 2 + j : 8 + wn * 2 + (j - 2);
        else return wn * 4 + j;
    };

    uint32_t nsz[2], csz[2];       // int4: scale | zero << 16 of the lane's two columns, next / current stage
    float s_unit[2] = {1.f, 1.f};  // int4: the scale the lane's accumulators of column tile j are in
    f16x2 qbias[2], qbias64[2];    // int4: fp16 1024 + z and 64 + z of the current group
    f16x2 qs2[2];                  // int4, rounded weights: the group scale, twice
    constexpr bool EXQ = !GEMM_FASTQ || EPI == EPI_F32;   // int4: exact scheme (qkv)

    // Copies of one stage, issued in parts from inside the previous stage's MFMA loop so
    // that no wave stalls on a burst of copies.  They go through buffer resources: rows
    // past M and blocks past the matrix read past the resource's end and land as zeros,
    // so the per-thread source offsets are fixed and only advance with k.
    constexpr int NA = BT * T::CPR / 512;            // A copies per thread per stage
    constexpr int NB = 16 * T::NBLK / 8;             // B copies per thread per stage
    constexpr int NPART = T::TK / 16;                // parts = 16-k MFMA steps of a stage
    uint32_t aoff[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) {
        const int pp = (i * 8 + w) * 64 + lane;
        const int row = pp / T::CPR, slot = pp % T::CPR;
        const int kc = (slot ^ a_swz<T::CPR>(row)) * 8;
        aoff[i] = m0 + row < a.M ? (uint32_t)(((int64_t)(m0 + row) * a.K + kc) * 2) : BUF_OOB;
    }
    uint32_t boff[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) {
        const int blk = i * 8 + w;
        bool v;
        const int gb = grow_block(blk / T::NBLK, v);
        boff[i] = v ? (uint32_t)((((int64_t)gb * a.kst + blk % T::NBLK) * 64 + lane) * 16) : BUF_OOB;
    }
    // int4: the lane's column of each column tile in the group-major scale / zero words
    // (-1: past the matrix)
    int szcol[2] = {-1, -1};
    if constexpr (WF == W_INT4) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            bool v;
            const int gb = grow_block(col_rb(2 * j + ((lane & 31) >> 4)), v);
            szcol[j] = v ? gb * 16 + r : -1;
        }
    }
    // K is a whole number of stages (the launcher sends other K to the small tiling), so
    // every k of every stage exists: the k advance goes into the buffer resources (uniform:
    // base moved forward, size cut by as much) and the per-lane offsets stay fixed; the
    // past-the-end offsets of rows past M and of blocks past the matrix stay past the end.
    // The LDS destinations are wave-uniform (scalar arithmetic, no per-copy VALU work).
    const uint32_t xbytes = (uint32_t)min((int64_t)a.M * a.K * 2, (int64_t)0xFFFFFFF0);
    const uint32_t wbytes = (uint32_t)min((int64_t)(DUAL ? 2 * nrb : nrb) * a.kst * 1024, (int64_t)0xFFFFFFF0);
    const int wu = __builtin_amdgcn_readfirstlane(w);
    auto issue_part = [&](int stage, int k0, int q) {
        char* sA = smem + stage * T::STAGE;
        char* sB = sA + T::A_BYTES;
        const uint32_t xadv = 2u * (uint32_t)k0;
        const uint32_t wadv = (uint32_t)(k0 / T::KSW) * 1024u;
        const __amdgpu_buffer_rsrc_t xr = buf_rsrc((const char*)a.X + xadv, xbytes - xadv);
        const __amdgpu_buffer_rsrc_t wr = buf_rsrc((const char*)a.W + wadv, wbytes - wadv);
#pragma unroll
        for (int i = 0; i < NA; ++i)
            if ((i * NPART) / NA == q) {
                // through a local: an array element passed straight to the builtin left the
                // kernels' host stubs unemitted (no diagnostic; the link caught it)
                const uint32_t off = aoff[i];
                __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lvoid_t*)(sA + (i * 8 + wu) * 1024), 16, off, 0, 0, 0);
            }
#pragma unroll
        for (int i = 0; i < NB; ++i)
            if ((i * NPART) / NB == q) {
                const uint32_t off = boff[i];
                __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lvoid_t*)(sB + (i * 8 + wu) * 1024), 16, off, 0, 0, 0);
            }
        if constexpr (WF == W_INT4) {
            if (q == 0) {
                // raw words, not converted here: a conversion would wait for them (and
                // for the stage's copies issued before them)
                const uint32_t* szg = a.sz + (int64_t)(k0 / 128) * a.N;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    nsz[j] = 0u;
                    if (szcol[j] >= 0) nsz[j] = szg[szcol[j]];
                }
            }
        }
    };
    auto issue = [&](int stage, int k0) {
#pragma unroll
        for (int q = 0; q < NPART; ++q) issue_part(stage, k0, q);
    };

    // 32x32 MFMA tiles: 4 (rows) x 2 (columns) per wave.  Column tile j covers the
    // wave's LDS row-blocks col_rb(2 j) and col_rb(2 j + 1); lane l holds column l % 32.
    f32x16 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

    const int l32 = lane & 31, h32 = lane >> 5;
    // multiply stage `stage` out of LDS; with nk0 >= 0, issue the copies of the stage at
    // k offset nk0 into the other buffer, two parts per 16-k step over the first half of
    // the steps (the second half covers their latency before the stage's closing wait)
    // int4: the stage is one group; the accumulators go to units of its scale, and the
    // biases that turn the extracted nibbles into q - z are set (two per column: nibbles in
    // bits 0-3 of an fp16 half read as 1024 + q, in bits 4-7 with exponent 0x54 as 64 + q)
    // A group whose scale is zero (its weights dequantise to zero) gets the unit 2^-64: the
    // accumulators are scaled up by s_prev * 2^64 and the group's own contribution, taken in
    // that unit, ends up 2^-64 / s_next of the value -- some 1e-18 of it, far below the
    // accumulators' rounding -- with no per-fragment work.
    auto regroup = [&]() {
        if constexpr (!EXQ) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const float z = h2f((uint16_t)(csz[j] >> 16));
                const _Float16 b0 = (_Float16)(1024.0f + z), b1 = (_Float16)(64.0f + z);
                qbias[j] = f16x2{b0, b0};
                qbias64[j] = f16x2{b1, b1};
                const _Float16 sc = __builtin_bit_cast(_Float16, (uint16_t)(csz[j] & 0xFFFFu));
                qs2[j] = f16x2{sc, sc};
            }
            return;
        }
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const float sc = h2f((uint16_t)(csz[j] & 0xFFFFu));
            const float s_new = sc == 0.f ? 0x1p-64f : sc;
            const float ratio = s_unit[j] * __builtin_amdgcn_rcpf(s_new);   // within 1 ulp
            s_unit[j] = s_new;
            const float z = h2f((uint16_t)(csz[j] >> 16));
            const _Float16 b0 = (_Float16)(1024.0f + z), b1 = (_Float16)(64.0f + z);
            qbias[j] = f16x2{b0, b0};
            qbias64[j] = f16x2{b1, b1};
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i][j] *= ratio;
        }
    };
    auto compute = [&](int stage, int nk0) {
        const char* sA = smem + stage * T::STAGE;
        const char* sB = sA + T::A_BYTES;
        u32x2 wd2[2];                                        // int4: the 32-k step's two words
        u32x4 wd4[2];                                        // int8: the 32-k step's 16 codes
#pragma unroll
        for (int kk = 0; kk < T::TK / 16; ++kk) {            // 16-k MFMA steps
            if (nk0 >= 0 && kk < T::TK / 32) {
                issue_part(stage ^ 1, nk0, 2 * kk);
                issue_part(stage ^ 1, nk0, 2 * kk + 1);
            }
            const int s = kk >> 1, hh = kk & 1;              // 32-k sub-step, half
            u32x4 af[4], bop[2];
            // 16-byte chunk of the A row: k 8 c .. 8 c + 7 for chunk c.  int4 lanes take the
            // k of the weight word they hold (below), so the chunk follows it: the MFMA only needs
            // both operands to agree on k
            const int chunk = WF != W_BF16 ? 4 * s + 2 * h32 + hh : 2 * kk + h32;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm * 128 + 32 * i + l32;
                af[i] = *(const u32x4*)(sA + row * (T::CPR * 16) + ((chunk ^ a_swz<T::CPR>(row)) * 16));
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int rb = col_rb(2 * j + (l32 >> 4)), rr = lane & 15;
                if constexpr (WF == W_BF16) {
                    // block (rb, s): lane r + 16 g holds k 8 g .. 8 g + 7 of the 32-k step
                    bop[j] = *(const u32x4*)(sB + (rb * 2 + s) * 1024 + (rr + 16 * (2 * hh + h32)) * 16);
                } else if constexpr (WF == W_INT8) {
                    // one 64-k block: lane r + 16 g holds k 16 g .. 16 g + 15.  A lane half h32
                    // takes piece g = 2 s + h32 whole at the step's first half (k 32 s + 16 h32
                    // + 8 hh ..): one 16-byte read per 32-k step
                    if (hh == 0) wd4[j] = *(const u32x4*)(sB + rb * 1024 + (rr + 16 * (2 * s + h32)) * 16);
                    const u32x2 c = hh ? u32x2{wd4[j].z, wd4[j].w} : u32x2{wd4[j].x, wd4[j].y};
                    const u32x2 c0 = i8x4_to_f16x4(c.x), c1 = i8x4_to_f16x4(c.y);
                    bop[j] = u32x4{c0.x, c0.y, c1.x, c1.y};
                } else {
                    // one 128-k block: lane r + 16 g holds k 32 g .. 32 g + 31, 8 per dword.  A
                    // lane half h32 takes words 2 h32 and 2 h32 + 1 of the 32-k step (k 32 s +
                    // 16 h32 + 8 hh ..), both in one 8-byte read at the step's first half: one LDS
                    // read where two 4-byte reads at a 16-byte lane stride met bank conflicts.
                    // Exact q - z
                    if (hh == 0) wd2[j] = *(const u32x2*)(sB + rb * 1024 + (rr + 16 * s) * 16 + 8 * h32);
                    const uint32_t wd = hh ? wd2[j].y : wd2[j].x;
                    bop[j] = i4x8_to_f16x8_q(wd, qbias[j], qbias64[j]);
                    if constexpr (!EXQ) {
                        const u32x4 d = bop[j];
                        bop[j] = u32x4{mul_h2(d.x, qs2[j]), mul_h2(d.y, qs2[j]), mul_h2(d.z, qs2[j]), mul_h2(d.w, qs2[j])};
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = mfma32<AF>(af[i], bop[j], acc[i][j]);
            // quantised weights: the compiler's interleaving strategy 1 for the step's LDS reads,
            // unpacking and MFMAs (measured 1.5-4% faster; bf16 weights are faster without it)
            if constexpr (WF != W_BF16) __builtin_amdgcn_iglp_opt(1);
        }
    };

    // k-range of this workgroup (the whole of K unless the GEMM is split)
    const int kb = EPI == EPI_PART ? blockIdx.y * a.krange : 0;
    const int ke = EPI == EPI_PART ? min(a.K, kb + a.krange) : a.K;
    const int nk = (ke - kb + T::TK - 1) / T::TK;
    issue(0, kb);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        if constexpr (WF == W_INT4) {
#pragma unroll
            for (int j = 0; j < 2; ++j) csz[j] = nsz[j];
        }
        const int nk0 = kt + 1 < nk ? kb + (kt + 1) * T::TK : -1;
        if constexpr (WF == W_INT4) regroup();
        compute(kt & 1, nk0);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
    }

    // ---- epilogue (accumulator element e of lane l: row 8 (e / 4) + 4 (l / 32) + e % 4 of
    // the 32x32 tile, column l % 32)
    if constexpr (EPI == EPI_PART) {
        const int ncols = DUAL ? 2 * a.F : a.N;
        float* out = a.out32 + (int64_t)blockIdx.y * a.M * ncols;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            int n;
            if constexpr (DUAL) n = (j == 0 ? 0 : a.F) + nt * 128 + wn * 32 + l32;
            else n = nt * 256 + wn * 64 + 32 * j + l32;
            if (DUAL ? nt * 128 + wn * 32 + l32 >= a.F : n >= a.N) continue;
            float sn = 1.f;
            if constexpr (WF == W_INT8) sn = h2f(a.scales[n]);
            if constexpr (WF == W_INT4) sn = s_unit[j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int m = m0 + wm * 128 + 32 * i + 8 * (e >> 2) + 4 * h32 + (e & 3);
                    if (m < a.M) out[(int64_t)m * ncols + n] = acc[i][j][e] * sn;
                }
        }
    } else if constexpr (DUAL) {
        // SwiGLU: a = act(bf16(silu(gate) * up)) per (m, f); the tile's 256 x 128 outputs are
        // staged in LDS (the stage buffers are free now) and written as 16-byte pieces of
        // whole 256-byte rows
        constexpr int FS = 136;                               // LDS row stride (u16)
        static_assert(256 * FS * 2 <= T::SMEM, "SwiGLU staging fits the LDS");
        uint16_t* st16 = (uint16_t*)smem;
        const int fl = wn * 32 + l32;                         // the lane's column in the tile
        const int f = nt * 128 + fl;
        float sg = 1.f, su = 1.f;
        if constexpr (WF == W_INT8) {
            if (f < a.F) {
                sg = h2f(a.scales[f]);
                su = h2f(a.scales[a.F + f]);
            }
        }
        if constexpr (WF == W_INT4) {
            sg = s_unit[0];
            su = s_unit[1];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = wm * 128 + 32 * i + 8 * (e >> 2) + 4 * h32 + (e & 3);
                const float gv = acc[i][0][e] * sg, uv = acc[i][1][e] * su;
                st16[row * FS + fl] = act_store(bfround(silu_f(gv) * uv), a.out_fmt);
            }
        __syncthreads();
#pragma unroll
        for (int t = 0; t < 8; ++t) {                         // 256 rows x 16 pieces of 8 columns
            const int idx = t * 512 + tid, row = idx >> 4, c = (idx & 15) * 8;
            const int m = m0 + row, f0 = nt * 128 + c;
            if (m < a.M && f0 < a.F)
                *(u32x4*)(a.out16 + (int64_t)m * a.F + f0) = *(const u32x4*)(st16 + row * FS + c);
        }
    } else if constexpr (EPI == EPI_F32) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = nt * 256 + wn * 64 + 32 * j + l32;
            if (n >= a.N) continue;
            float sn = 1.f;
            if constexpr (WF == W_INT8) sn = h2f(a.scales[n]);
            if constexpr (WF == W_INT4) sn = s_unit[j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int m = m0 + wm * 128 + 32 * i + 8 * (e >> 2) + 4 * h32 + (e & 3);
                    if (m < a.M) a.out32[(int64_t)m * a.N + n] = acc[i][j][e] * sn;
                }
        }
    } else {
        // residual: out = bf16(resid + acc).  Each wave stages its 128 x 64 results in two
        // passes of 64 rows through its own LDS region (fp32), then reads 8 consecutive
        // columns per lane and writes them, with the matching resid piece, as 16-byte
        // pieces of 128-byte row segments; a pass's resid loads go out first.
        constexpr int ES = 72;                                // LDS row stride (floats): rows r, r + 4 are 32 banks apart
        static_assert(8 * 64 * ES * 4 <= T::SMEM, "residual staging fits the LDS");
        float* reg = (float*)smem + w * 64 * ES;
        float sn[2];
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = nt * 256 + wn * 64 + 32 * j + l32;
            sn[j] = 1.f;
            if constexpr (WF == W_INT8) sn[j] = n < a.N ? h2f(a.scales[n]) : 0.f;
            if constexpr (WF == W_INT4) sn[j] = s_unit[j];
        }
        const int rl = lane >> 3, c8 = (lane & 7) * 8;        // 8 rows x 8 pieces per instruction
        const int n8 = nt * 256 + wn * 64 + c8;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            u32x4 rv[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int m = m0 + wm * 128 + 64 * p + 8 * t + rl;
                rv[t] = u32x4{0u, 0u, 0u, 0u};
                if (m < a.M && n8 < a.N) rv[t] = *(const u32x4*)(a.resid + (int64_t)m * a.N + n8);
            }
#pragma unroll
            for (int ii = 0; ii < 2; ++ii)
#pragma unroll
                for (int j = 0; j < 2; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        const int row = 32 * ii + 8 * (e >> 2) + 4 * h32 + (e & 3);
                        reg[row * ES + 32 * j + l32] = acc[2 * p + ii][j][e] * sn[j];
                    }
            __syncthreads();
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                const int row = 8 * t + rl, m = m0 + wm * 128 + 64 * p + row;
                if (m >= a.M || n8 >= a.N) continue;
                const f32x4 v0 = *(const f32x4*)(reg + row * ES + c8), v1 = *(const f32x4*)(reg + row * ES + c8 + 4);
                const uint32_t r4[4] = {rv[t].x, rv[t].y, rv[t].z, rv[t].w};
                const float vv[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
                uint32_t o[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    o[q] = (uint32_t)f2bf(bf2f(r4[q] & 0xFFFFu) + vv[2 * q]) |
                           ((uint32_t)f2bf(bf2f(r4[q] >> 16) + vv[2 * q + 1]) << 16);
                *(u32x4*)(a.out16 + (int64_t)m * a.N + n8) = u32x4{o[0], o[1], o[2], o[3]};
            }
            __syncthreads();                                  // before the next pass overwrites the region
        }
    }
}

template <int WF>
static hipError_t launch_big(const GemmArgs& a, int epi, hipStream_t st) {
    GemmArgs b = a;
    b.tiles_n = (epi == EPI_SWIGLU) ? (a.F + 127) / 128 : (a.N + BT - 1) / BT;
    b.tiles_m = (a.M + BT - 1) / BT;
    dim3 grid(b.tiles_n * b.tiles_m);
    switch (epi) {
        case EPI_F32: FP_LAUNCH((gemm_big_kernel<WF, EPI_F32, false>), grid, dim3(512), 0, st, b); break;
        case EPI_RESID: FP_LAUNCH((gemm_big_kernel<WF, EPI_RESID, false>), grid, dim3(512), 0, st, b); break;
        case EPI_SWIGLU: FP_LAUNCH((gemm_big_kernel<WF, EPI_SWIGLU, true>), grid, dim3(512), 0, st, b); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int WF>
static hipError_t launch_big_split(const GemmArgs& a, bool dual, int ks, hipStream_t st) {
    GemmArgs b = a;
    b.tiles_n = dual ? (a.F + 127) / 128 : (a.N + BT - 1) / BT;
    b.tiles_m = (a.M + BT - 1) / BT;
    dim3 grid(b.tiles_n * b.tiles_m, ks);
    if (dual) FP_LAUNCH((gemm_big_kernel<WF, EPI_PART, true>), grid, dim3(512), 0, st, b);
    else FP_LAUNCH((gemm_big_kernel<WF, EPI_PART, false>), grid, dim3(512), 0, st, b);
    return hipGetLastError();
}

static int big_tk(int wf) { return wf == W_INT4 ? BigT<W_INT4>::TK : BigT<W_BF16>::TK; }

#ifndef GEMM_SPLIT_MAX
#define GEMM_SPLIT_MAX 16
#endif
int gemm_split_factor(int M, int N, int K, int dual_F, int wf, int* krange) {
    const int tiles = ((M + BT - 1) / BT) * (dual_F > 0 ? (dual_F + 127) / 128 : (N + BT - 1) / BT);
    const int tk = big_tk(wf);
    const int stages = (K + tk - 1) / tk;
    *krange = stages * tk;
    if (M < BT || tiles >= 256 || K % tk != 0) return 1;
    // one round of workgroups (one per compute unit), at least four stages per split
    int ks = 256 / tiles;
    if (ks > GEMM_SPLIT_MAX) ks = GEMM_SPLIT_MAX;
    if (ks > stages / 4) ks = stages / 4;
    if (ks < 2) return 1;
    const int per = (stages + ks - 1) / ks;
    *krange = per * tk;
    return (stages + per - 1) / per;
}

hipError_t launch_gemm_split(const GemmArgs& a, int wf, bool dual, int ks, hipStream_t st) {
    if (ks < 1 || a.krange <= 0 || a.krange % big_tk(wf) != 0 || a.K % big_tk(wf) != 0 || (int64_t)ks * a.krange < a.K ||
        (int64_t)(ks - 1) * a.krange >= a.K)
        return hipErrorInvalidValue;
    switch (wf) {
        case W_BF16: return launch_big_split<W_BF16>(a, dual, ks, st);
        case W_INT8: return launch_big_split<W_INT8>(a, dual, ks, st);
        case W_INT4: return launch_big_split<W_INT4>(a, dual, ks, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_big(const GemmArgs& a, int wf, int epi, hipStream_t st) {
    if (a.K % big_tk(wf) != 0) return hipErrorInvalidValue;     // whole stages only
    switch (wf) {
        case W_BF16: return launch_big<W_BF16>(a, epi, st);
        case W_INT8: return launch_big<W_INT8>(a, epi, st);
        case W_INT4: return launch_big<W_INT4>(a, epi, st);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm(const GemmArgs& a, int wf, int epi, hipStream_t st) {
    const int tiles = ((a.M + BT - 1) / BT) * ((epi == EPI_SWIGLU) ? (a.F + 127) / 128 : (a.N + BT - 1) / BT);
    if (tiles >= GEMM_BIG_MIN_TILES && a.K % big_tk(wf) == 0) return launch_gemm_big(a, wf, epi, st);
    return launch_gemm_small(a, wf, epi, st);
}

}  // namespace fpk
