// Prefill projections: tiled GEMM  C[M, N] = X[M, K] . W[N, K]^T on MFMA, with the
// weight tile dequantised while it is staged into LDS and the layer's elementwise
// work fused into the epilogue.
//
// Prefill (the fingerprint's time to first token, paper Sec. 5.3) runs every
// prompt token through the projections at once, so it is a dense contraction
// and belongs on the matrix cores.  Weight-only quantised tiles (Sec. 3.2) are
// converted to 16-bit once per workgroup tile, amortised over its 128 rows:
//   bf16 W: copied; A operand bf16                   (bf16 MFMA)
//   int8 W: codes -> exact fp16; per-row scale in the epilogue    (fp16 MFMA)
//   int4 W: fp16((q - z) * s), one rounding per weight            (fp16 MFMA)
// Epilogues: fp32 store (q, k, v before the rotary embedding), residual
// out = bf16(resid + acc), and SwiGLU a = bf16(silu(gate) * up) where each wave
// holds gate and up columns of the same f (dual tiles over [gate; up]).
//
// Weights are read from the fragment-major layout (1 KiB blocks of 16 rows x one
// K-step), so each 64-thread group of a tile load reads contiguous memory.
//
// Tile 128 x 128 x 64, 4 waves in 2 x 2, each wave 64 x 64 = 4 x 4 MFMA 16x16x32
// tiles; the next K tile is loaded into registers while the current one is
// multiplied out of LDS.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

constexpr int GBM = 128, GBN = 128, GBK = 64, GPAD = 8;
constexpr int GLD = GBK + GPAD;   // LDS row (u16)

template <int WF, int EPI>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs a) {
    constexpr int AF = (WF == W_BF16) ? ACT_BF16 : ACT_F16;
    __shared__ __attribute__((aligned(16))) uint16_t As[GBM * GLD];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[GBN * GLD];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int wm = w >> 1, wn = w & 1;
    const int m0 = blockIdx.y * GBM;
    const int nb = blockIdx.x;

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
    u32x4 ra[4], rb[BCH];
    float bs_scale = 0.f, bs_zero = 0.f;
    auto load_tile = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 256 * i;
            const int row = c >> 3, kc = (c & 7) * 8;
            const int m = m0 + row, k = k0 + kc;
            ra[i] = u32x4{0u, 0u, 0u, 0u};
            if (m < a.M && k < a.K) ra[i] = *(const u32x4*)(a.X + (int64_t)m * a.K + k);
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
                const int n = brow(lr, v);
                const int kabs = k0 + 32 * kst;
                rb[i] = u32x4{0u, 0u, 0u, 0u};
                if (v && kabs + 8 * (L >> 4) < a.K)
                    rb[i] = Wt[((int64_t)(n >> 4) * a.kst + kabs / 32) * 64 + L];
            }
        } else if constexpr (WF == W_INT8) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {                  // 8 subtiles x 1 K-step of 64
                const int c = tid + 256 * i;
                const int ntl = c >> 6, L = c & 63;
                const int lr = 16 * ntl + (L & 15);
                bool v;
                const int n = brow(lr, v);
                rb[i] = u32x4{0u, 0u, 0u, 0u};
                if (v && k0 + 16 * (L >> 4) < a.K)
                    rb[i] = Wt[((int64_t)(n >> 4) * a.kst + k0 / 64) * 64 + L];
            }
        } else {                                           // 8 subtiles x half a K-step of 128
            const int ntl = tid >> 5, j = tid & 31;
            const int lr = 16 * ntl + (j & 15);
            const int gg = j >> 4, g = gg + 2 * ((k0 >> 6) & 1);
            bool v;
            const int n = brow(lr, v);
            rb[0] = u32x4{0u, 0u, 0u, 0u};
            bs_scale = 0.f;
            bs_zero = 0.f;
            if (v && k0 < a.K) {
                rb[0] = Wt[((int64_t)(n >> 4) * a.kst + k0 / 128) * 64 + (j & 15) + 16 * g];
                const int grp = k0 / 128;
                bs_scale = h2f(a.scales[(int64_t)n * (a.K / 128) + grp]);
                bs_zero = h2f(a.zeros[(int64_t)n * (a.K / 128) + grp]);
            }
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
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
            const _Float16 bz = (_Float16)(1024.0f + bs_zero);
            const f16x2 bias = {bz, bz};
            const _Float16 sh = (_Float16)bs_scale;
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

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int nk = (a.K + GBK - 1) / GBK;
    load_tile(0);
    store_tile();
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk) load_tile((kt + 1) * GBK);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            u32x4 af[4], bf[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                af[i] = *(const u32x4*)(As + (wm * 64 + 16 * i + r) * GLD + 32 * ks + 8 * g);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bf[j] = *(const u32x4*)(Bs + (wn * 64 + 16 * j + r) * GLD + 32 * ks + 8 * g);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = mfma16<AF>(af[i], bf[j], acc[i][j]);
        }
        __syncthreads();
        if (kt + 1 < nk) {
            store_tile();
            __syncthreads();
        }
    }

    // ---- epilogue
    if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int f = nb * 64 + 32 * wn + 16 * j + r;
            if (f >= a.F) continue;
            float sg = 1.f, su = 1.f;
            if constexpr (WF == W_INT8) {
                sg = h2f(a.scales[f]);
                su = h2f(a.scales[a.F + f]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = m0 + wm * 64 + 16 * i + 4 * g + e;
                    if (m >= a.M) continue;
                    const float gv = acc[i][j][e] * sg, uv = acc[i][j + 2][e] * su;
                    a.out16[(int64_t)m * a.F + f] = act_store(bfround(silu_f(gv) * uv), a.out_fmt);
                }
        }
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = nb * GBN + wn * 64 + 16 * j + r;
            if (n >= a.N) continue;
            float sn = 1.f;
            if constexpr (WF == W_INT8) sn = h2f(a.scales[n]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int m = m0 + wm * 64 + 16 * i + 4 * g + e;
                    if (m >= a.M) continue;
                    const float v = acc[i][j][e] * sn;
                    if constexpr (EPI == EPI_F32) a.out32[(int64_t)m * a.N + n] = v;
                    else a.out16[(int64_t)m * a.N + n] = f2bf(bf2f(a.resid[(int64_t)m * a.N + n]) + v);
                }
        }
    }
}

template <int WF>
static hipError_t launch_w(const GemmArgs& a, int epi, hipStream_t st) {
    const int nt = (epi == EPI_SWIGLU) ? (a.F + 63) / 64 : (a.N + GBN - 1) / GBN;
    dim3 grid(nt, (a.M + GBM - 1) / GBM);
    switch (epi) {
        case EPI_F32: FP_LAUNCH((gemm_kernel<WF, EPI_F32>), grid, dim3(256), 0, st, a); break;
        case EPI_RESID: FP_LAUNCH((gemm_kernel<WF, EPI_RESID>), grid, dim3(256), 0, st, a); break;
        case EPI_SWIGLU: FP_LAUNCH((gemm_kernel<WF, EPI_SWIGLU>), grid, dim3(256), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemm(const GemmArgs& a, int wf, int epi, hipStream_t st) {
    switch (wf) {
        case W_BF16: return launch_w<W_BF16>(a, epi, st);
        case W_INT8: return launch_w<W_INT8>(a, epi, st);
        case W_INT4: return launch_w<W_INT4>(a, epi, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace fpk
