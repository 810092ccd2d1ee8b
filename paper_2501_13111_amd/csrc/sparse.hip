// 2:4 semi-structured sparse weights (the pruning of paper Sec. 3.3 and Table A.1: two
// of every four weights zero) on the sparse matrix cores of gfx950.
//
// Mask: in each group of 4 consecutive inputs of a row, the 2 weights of largest
// magnitude are kept (the lower input first among equal magnitudes); kept weights stay
// bf16.  The sparse MFMA v_smfmac_f32_32x32x32_bf16 multiplies a 2:4-sparse 32 x 32
// operand, given as its 32 x 16 kept values plus 2-bit positions, by a dense 32 x 32
// operand: half the multiply work and half the weight bytes of a dense bf16 MFMA.  The
// sparse operand must be the first one, so the weights play A and the activations B:
// C^T[n, m] = sum_k W[n, k] X[m, k].
//
// Operand layout of that instruction (lane l):
//   sparse A: row l % 32, 8 kept values of 4 groups, groups 0 and 1 covering inputs
//             8 s .. 8 s + 7 and groups 2 and 3 covering 16 + 8 s .. 16 + 8 s + 7, s = l / 32;
//             value i's position in its group in bits 2i + 1 .. 2i of the index word
//   dense B:  column l % 32, inputs 16 s .. 16 s + 15
//   C / D:    column l % 32, rows 8 (e / 4) + 4 s + e % 4 for accumulator element e
// Storage: weights in 32-row x 32-input blocks; block (rb, kb) holds the 64 lanes'
// 16-byte value pieces contiguously (1 KiB, lane l at l * 16) and the lanes' 16-bit index
// words in a separate 128-byte block, rb-major over kb, so a wave's operand load is one
// contiguous 1 KiB read.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void lvoid_t;

__device__ __forceinline__ f32x16 smfmac(u32x4 a, u32x4 b0, u32x4 b1, uint32_t idx, f32x16 c) {
    const u32x4 bb[2] = {b0, b1};
    return __builtin_amdgcn_smfmac_f32_32x32x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x16, bb),
                                                      c, (int)idx, 0, 0);
}

// Dense input k (0..31 within a block) of kept value group g (0..3) of slice s.
__host__ __device__ inline int sp24_group_k(int g, int s) { return (g < 2 ? 0 : 16) + 8 * s + 4 * (g & 1); }

// ---------------------------------------------------------------- mask and compression
// One thread per (row, 32-input block, slice): 4 groups of 4 bf16 weights -> 8 kept values
// and a 16-bit index word.  Magnitudes compare as the bf16 bits without the sign (finite
// values only), exactly, so the mask is a pure function of the weights.
__global__ void __launch_bounds__(256) sp24_compress_kernel(const uint16_t* __restrict__ w, int n, int K,
                                                             uint16_t* __restrict__ vals, uint16_t* __restrict__ idx,
                                                             int row0) {
    const int kst = K / 32;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * kst * 2) return;
    const int s = (int)(t & 1);
    const int kb = (int)((t >> 1) % kst);
    const int r = (int)((t >> 1) / kst);
    const uint16_t* src = w + (int64_t)r * K + kb * 32;
    uint32_t v[4];
    uint32_t word = 0;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int k0 = sp24_group_k(g, s);
        uint32_t m[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) m[p] = src[k0 + p] & 0x7FFFu;
        // the first kept: the largest, lowest position on ties; the second: the same over the rest
        int a = 0;
#pragma unroll
        for (int p = 1; p < 4; ++p)
            if (m[p] > m[a]) a = p;
        int b = a == 0 ? 1 : 0;
#pragma unroll
        for (int p = 0; p < 4; ++p)
            if (p != a && m[p] > m[b]) b = p;
        const int p0 = a < b ? a : b, p1 = a < b ? b : a;
        v[g] = (uint32_t)src[k0 + p0] | ((uint32_t)src[k0 + p1] << 16);
        word |= (uint32_t)(p0 | (p1 << 2)) << (4 * g);
    }
    const int grow = row0 + r;
    const int64_t blk = (int64_t)(grow / 32) * kst + kb;
    const int lane = (grow % 32) + 32 * s;
    *(u32x4*)(vals + blk * 512 + lane * 8) = u32x4{v[0], v[1], v[2], v[3]};
    idx[blk * 64 + lane] = (uint16_t)word;
}

hipError_t launch_sp24_compress(const uint16_t* w, int n, int K, uint16_t* vals, uint16_t* idx, int row0,
                                hipStream_t st) {
    if (n % 32 != 0 || row0 % 32 != 0 || K % 32 != 0) return hipErrorInvalidValue;
    const int64_t threads = (int64_t)n * (K / 32) * 2;
    FP_LAUNCH(sp24_compress_kernel, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st, w, n, K, vals, idx,
              row0);
    return hipGetLastError();
}

// ---------------------------------------------------------------- decode projection
// part[s, m, n] = sum_{k in split s} X[m, k] W[n, k], M <= 64 tokens.  A workgroup of 4
// waves takes 128 weight rows (32 per wave) over one k-range; its slice of X (rows past M
// zero) is staged once in LDS.  Each wave streams its 32-row blocks with SP_RING blocks in
// flight (buffer loads: past the range they return zeros without memory traffic).
constexpr int SP_RING = 8;
constexpr int SP_LDS_BYTES = 64 * 1024;
constexpr int SP_PAD = 8;

template <int MT>
__global__ void __launch_bounds__(256) sp24_gemv_kernel(Sp24Args a) {
    extern __shared__ __attribute__((aligned(16))) uint16_t Xs[];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int s = lane >> 5, c32 = lane & 31;
    const int kb = blockIdx.y * a.krange;
    const int ke = min(a.K, kb + a.krange);
    const int klen = ke - kb;
    const int ld = a.krange + SP_PAD;
    const int n0 = blockIdx.x * 128 + w * 32;
    const bool live = n0 < a.N;
    const int nsteps = klen / 32;
    const int64_t blk0 = live ? (int64_t)(n0 / 32) * a.kst + kb / 32 : 0;
    const __amdgpu_buffer_rsrc_t vres = buf_rsrc(a.Wv, (uint32_t)((a.N / 32) * (int64_t)a.kst * 1024));
    u32x4 rv[SP_RING];
    uint32_t ri[SP_RING];
    auto load = [&](int t, int d) {
        rv[d] = buf_load_nt(vres, off_or_oob(live && t < nsteps, (uint32_t)((blk0 + t) * 1024 + lane * 16)));
        ri[d] = a.Wi[(blk0 + min(t, nsteps - 1)) * 64 + lane];
    };
    // the first weight blocks go out before the activation slice is staged
#pragma unroll
    for (int d = 0; d < SP_RING; ++d) load(d, d);
    {
        const int cpr = klen / 8;
        for (int i = tid; i < 32 * MT * cpr; i += 256) {
            const int row = i / cpr, c = i % cpr;
            u32x4 v = u32x4{0u, 0u, 0u, 0u};
            if (row < a.M) v = *(const u32x4*)(a.X + (int64_t)row * a.K + kb + c * 8);
            *(u32x4*)(Xs + row * ld + c * 8) = v;
        }
    }
    __syncthreads();
    if (!live) return;
    f32x16 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x16{};
    for (int t0 = 0; t0 < nsteps; t0 += SP_RING) {
#pragma unroll
        for (int d = 0; d < SP_RING; ++d) {
            const int kl = min(t0 + d, nsteps - 1) * 32 + 16 * s;   // past the range the weights are zero
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint16_t* xr = Xs + (32 * mt + c32) * ld + kl;
                acc[mt] = smfmac(rv[d], *(const u32x4*)xr, *(const u32x4*)(xr + 8), ri[d], acc[mt]);
            }
            load(t0 + d + SP_RING, d);
        }
    }
    // lane: token 32 mt + c32, rows n0 + 8 q + 4 s .. + 3 (accumulator elements 4 q .. 4 q + 3)
    float* out = a.part + (int64_t)blockIdx.y * a.M * a.N;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = 32 * mt + c32;
        if (m >= a.M) continue;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *(f32x4*)(out + (int64_t)m * a.N + n0 + 8 * q + 4 * s) =
                f32x4{acc[mt][4 * q], acc[mt][4 * q + 1], acc[mt][4 * q + 2], acc[mt][4 * q + 3]};
    }
}

int sp24_max_krange(int M) {
    const int rows = M > 32 ? 64 : 32;
    int kr = SP_LDS_BYTES / (rows * 2) - SP_PAD;
    return kr - kr % 128;
}

hipError_t launch_sp24_gemv(const Sp24Args& a, int ks, hipStream_t st) {
    if (a.M < 1 || a.M > 64 || a.N % 32 != 0 || a.K % 32 != 0 || a.krange % 32 != 0) return hipErrorInvalidValue;
    if (a.krange > sp24_max_krange(a.M) || (int64_t)ks * a.krange < a.K || (int64_t)(ks - 1) * a.krange >= a.K)
        return hipErrorInvalidValue;
    if ((int64_t)(a.N / 32) * a.kst * 1024 >= ((int64_t)1 << 32) - 16) return hipErrorInvalidValue;
    const dim3 grid((a.N + 127) / 128, ks);
    const size_t lds = (size_t)(a.M > 32 ? 64 : 32) * (a.krange + SP_PAD) * 2;
    if (a.M > 32) FP_LAUNCH(sp24_gemv_kernel<2>, grid, dim3(256), lds, st, a);
    else FP_LAUNCH(sp24_gemv_kernel<1>, grid, dim3(256), lds, st, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------- prefill projection
// C^T tiles of TN weight rows x TM tokens: waves of NBW 32-row weight blocks x MW 32-token
// tiles (NBW x MW sparse 32x32x32 MFMA tiles), 64 inputs per stage.  Large products take
// 256 x 256 tiles of 8 waves with 4 x 2 tiles each (per 32 inputs a wave reads 4 weight
// fragments and 4 activation pieces for 8 MFMAs); smaller ones take 128 x 128 tiles of 4
// waves with 2 x 2, so that more workgroups fill the GPU.  Activation rows (128 B per
// stage), weight value blocks and the blocks' index words are copied into LDS by buffer
// loads that write LDS directly (rows past M and blocks past the matrix land as zeros),
// activation chunks stored with an XOR swizzle so that fragment reads are free of bank
// conflicts.  Three LDS stages: a stage's copies are issued two stages ahead (a stage holds
// only 16 MFMAs per wave, too few to cover a copy's latency on its own), and each wave waits
// for all but the newest stage's copies, an exact count since they are its only
// vector-memory instructions in the loop.  A lane's accumulators hold one token and runs of
// 4 consecutive weight rows, so the epilogues write 16- and 8-byte pieces of the [M, N]
// outputs directly; the SwiGLU tiling gives each wave gate blocks and the matching up blocks.
constexpr int SG_TK = 64;

template <int TM, int TN, int MW, int NBW>
struct SgT {
    static constexpr int WGM = TM / (32 * MW), WGN = TN / (32 * NBW);   // waves along m and n
    static constexpr int NW = WGM * WGN, NT = 64 * NW;
    static constexpr int X_BYTES = TM * SG_TK * 2;
    static constexpr int W_BYTES = (TN / 32) * (SG_TK / 32) * 1024;
    static constexpr int I_BYTES = (TN / 32) * 256;                    // index words: 2 k-blocks x 64 lanes per row-block
    static constexpr int STAGE = X_BYTES + W_BYTES + I_BYTES;
    static constexpr int NX = X_BYTES / 1024 / NW;                     // activation copies per thread
    static constexpr int NWB = W_BYTES / 1024 / NW;                    // weight-block copies per thread
    static constexpr int LPS = NX + NWB + 1;                           // copies per thread per stage (one of index words)
    static_assert(NX * NW * 1024 == X_BYTES && NWB * NW * 1024 == W_BYTES && TN / 32 == NW, "copy split");
};

__device__ __forceinline__ int sg_swz(int row) { return (row >> 1) & 7; }

template <int EPI, int TM, int TN, int MW, int NBW>
__global__ void __launch_bounds__(64 * (TM / (32 * MW)) * (TN / (32 * NBW))) gemm_sp24_kernel(Sp24Args a) {
    using T = SgT<TM, TN, MW, NBW>;
    constexpr bool DUAL = EPI == EPI_SWIGLU;
    constexpr int RB = TN / 32;                     // weight row-blocks of a tile
    static_assert(!DUAL || NBW % 2 == 0, "SwiGLU: gate and up blocks in pairs");
    constexpr int NS = 3;                           // LDS stages: copies run two stages ahead
    __shared__ __attribute__((aligned(1024))) char smem[NS * T::STAGE];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int s = lane >> 5, c32 = lane & 31;
    const int wn = w / T::WGM, wm = w % T::WGM;
    int mt, nt;
    {
        const int Tn = a.tiles_m * a.tiles_n, bid = blockIdx.x;
        const int x = bid & 7, j = bid >> 3, q = Tn >> 3, rm = Tn & 7;
        const int t = x * q + (x < rm ? x : rm) + j;
        const int GM = 8;
        const int grp = t / (GM * a.tiles_n);
        const int gm0 = grp * GM;
        const int gsz = min(GM, a.tiles_m - gm0);
        const int tt = t - grp * GM * a.tiles_n;
        mt = gm0 + tt % gsz;
        nt = tt / gsz;
    }
    const int m0 = mt * TM;
    const int nrb = a.N / 32;                       // row-blocks of the matrix
    // global row-block of the tile's row-block rb: plain, or [gate RB/2 | up RB/2] for SwiGLU
    auto grb = [&](int rb, bool& v) -> int {
        if constexpr (DUAL) {
            const int fb = nt * (RB / 2) + (rb % (RB / 2));
            v = fb < a.F / 32;
            return (rb < RB / 2 ? 0 : a.F / 32) + fb;
        } else {
            const int b = nt * RB + rb;
            v = b < nrb;
            return b;
        }
    };
    // the tile row-block of this wave's n-block bn (SwiGLU: gate blocks, then their up blocks)
    auto wrb = [&](int bn) -> int {
        if constexpr (DUAL) return bn < NBW / 2 ? wn * (NBW / 2) + bn : RB / 2 + wn * (NBW / 2) + (bn - NBW / 2);
        else return wn * NBW + bn;
    };

    const __amdgpu_buffer_rsrc_t xres = buf_rsrc(a.X, (uint32_t)min((int64_t)a.M * a.K * 2, (int64_t)0xFFFFFFF0));
    const __amdgpu_buffer_rsrc_t wres = buf_rsrc(a.Wv, (uint32_t)min((int64_t)nrb * a.kst * 1024, (int64_t)0xFFFFFFF0));
    const __amdgpu_buffer_rsrc_t ires = buf_rsrc(a.Wi, (uint32_t)min((int64_t)nrb * a.kst * 128, (int64_t)0xFFFFFFF0));
    // per-thread copy slots: NX activation pieces and NWB weight blocks (1 KiB wave copies)
    uint32_t xoff[T::NX];
#pragma unroll
    for (int i = 0; i < T::NX; ++i) {
        const int p = (i * T::NW + w) * 64 + lane;
        const int row = p >> 3, slot = p & 7;
        const int kc = (slot ^ sg_swz(row)) * 8;
        xoff[i] = m0 + row < a.M ? (uint32_t)(((int64_t)(m0 + row) * a.K + kc) * 2) : BUF_OOB;
    }
    uint32_t woff[T::NWB];
#pragma unroll
    for (int i = 0; i < T::NWB; ++i) {
        const int b = i * T::NW + w, rb = b >> 1, kb = b & 1;
        bool v;
        const int g = grb(rb, v);
        woff[i] = v ? (uint32_t)((((int64_t)g * a.kst + kb) * 64 + lane) * 16) : BUF_OOB;
    }
    // the index words of tile row-block w (one per wave): the two k-blocks of a stage are 256
    // contiguous bytes, one dword per lane
    uint32_t ioff;
    {
        bool v;
        const int g = grb(w, v);
        ioff = v ? (uint32_t)((int64_t)g * a.kst * 128 + lane * 4) : BUF_OOB;
    }
    const int wu = __builtin_amdgcn_readfirstlane(w);
    auto issue = [&](int sl, int k0) {
        char* sX = smem + sl * T::STAGE;
        char* sW = sX + T::X_BYTES;
        char* sI = sW + T::W_BYTES;
#pragma unroll
        for (int i = 0; i < T::NX; ++i) {
            const uint32_t off = xoff[i] != BUF_OOB ? xoff[i] + 2u * k0 : BUF_OOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(xres, (lvoid_t*)(sX + (i * T::NW + wu) * 1024), 16, off, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < T::NWB; ++i) {
            const uint32_t off = woff[i] != BUF_OOB ? woff[i] + (uint32_t)(k0 / 32) * 1024u : BUF_OOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wres, (lvoid_t*)(sW + (i * T::NW + wu) * 1024), 16, off, 0, 0, 0);
        }
        const uint32_t off = ioff != BUF_OOB ? ioff + (uint32_t)(k0 / 32) * 128u : BUF_OOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ires, (lvoid_t*)(sI + wu * 256), 4, off, 0, 0, 0);
    };

    f32x16 acc[NBW][MW];
#pragma unroll
    for (int bn = 0; bn < NBW; ++bn)
#pragma unroll
        for (int bm = 0; bm < MW; ++bm) acc[bn][bm] = f32x16{};

    // stage sl: multiply it out of LDS (the index words come from its LDS region too)
    auto compute = [&](int sl) {
        const char* sX = smem + sl * T::STAGE;
        const char* sW = sX + T::X_BYTES;
        const char* sI = sW + T::W_BYTES;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            u32x4 af[NBW], b0[MW], b1[MW];
            uint32_t ix[NBW];
#pragma unroll
            for (int bn = 0; bn < NBW; ++bn) {
                af[bn] = *(const u32x4*)(sW + (wrb(bn) * 2 + kk) * 1024 + lane * 16);
                ix[bn] = *(const uint16_t*)(sI + wrb(bn) * 256 + kk * 128 + lane * 2);
            }
#pragma unroll
            for (int bm = 0; bm < MW; ++bm) {
                const int row = wm * 32 * MW + bm * 32 + c32;
                const int ch = 4 * kk + 2 * s;
                b0[bm] = *(const u32x4*)(sX + row * 128 + ((ch ^ sg_swz(row)) * 16));
                b1[bm] = *(const u32x4*)(sX + row * 128 + (((ch + 1) ^ sg_swz(row)) * 16));
            }
#pragma unroll
            for (int bn = 0; bn < NBW; ++bn)
#pragma unroll
                for (int bm = 0; bm < MW; ++bm) acc[bn][bm] = smfmac(af[bn], b0[bm], b1[bm], ix[bn], acc[bn][bm]);
        }
    };
    // the copies of a stage are the wave's only vector-memory instructions in the loop, LPS of
    // them, so "all but the last stage's" is an exact wait count
    auto wait_all_but_one_stage = [&]() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(T::LPS) : "memory"); };
    auto wait_all = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
    auto barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

    const int nk = a.K / SG_TK;
    issue(0, 0);
    if (nk > 1) {
        issue(1, SG_TK);
        wait_all_but_one_stage();
    } else {
        wait_all();
    }
    barrier();
    // trip kt: copies of stage kt + 2 into the slot stage kt - 1 used, multiply stage kt, then
    // wait for stage kt + 1 (the slots are kt % 3: three trips per loop turn)
    auto trip = [&](int kt, int sl) {
        if (kt + 2 < nk) issue((sl + 2) % NS, (kt + 2) * SG_TK);
        compute(sl);
        if (kt + 2 < nk) wait_all_but_one_stage();
        else wait_all();
        barrier();
    };
    int kt = 0;
    for (; kt + NS <= nk; kt += NS) {
        trip(kt, 0);
        trip(kt + 1, 1);
        trip(kt + 2, 2);
    }
    if (kt < nk) trip(kt, 0);
    if (kt + 1 < nk) trip(kt + 1, 1);

    // epilogue: lane holds token m = m0 + 32 MW wm + 32 bm + c32 and, per q, rows
    // r0 + 8 q + 4 s .. + 3 of its n-block (accumulator elements 4 q .. 4 q + 3)
#pragma unroll
    for (int bm = 0; bm < MW; ++bm) {
        const int m = m0 + wm * 32 * MW + bm * 32 + c32;
        if (m >= a.M) continue;
        if constexpr (DUAL) {
#pragma unroll
            for (int jg = 0; jg < NBW / 2; ++jg) {
                bool v;
                const int g = grb(wrb(jg), v);          // gate row-block; up is g + F / 32
                if (!v) continue;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int f = g * 32 + 8 * q + 4 * s;
                    uint32_t o[2];
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        const float g0 = acc[jg][bm][4 * q + 2 * h], u0 = acc[jg + NBW / 2][bm][4 * q + 2 * h];
                        const float g1 = acc[jg][bm][4 * q + 2 * h + 1], u1 = acc[jg + NBW / 2][bm][4 * q + 2 * h + 1];
                        o[h] = (uint32_t)act_store(bfround(silu_f(g0) * u0), a.out_fmt) |
                               ((uint32_t)act_store(bfround(silu_f(g1) * u1), a.out_fmt) << 16);
                    }
                    *(u32x2*)(a.out16 + (int64_t)m * a.F + f) = u32x2{o[0], o[1]};
                }
            }
        } else {
#pragma unroll
            for (int bn = 0; bn < NBW; ++bn) {
                bool v;
                const int g = grb(wrb(bn), v);
                if (!v) continue;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int n = g * 32 + 8 * q + 4 * s;
                    const f32x4 r = f32x4{acc[bn][bm][4 * q], acc[bn][bm][4 * q + 1], acc[bn][bm][4 * q + 2],
                                          acc[bn][bm][4 * q + 3]};
                    if constexpr (EPI == EPI_F32) {
                        *(f32x4*)(a.out32 + (int64_t)m * a.N + n) = r;
                    } else {
                        const u32x2 rs = *(const u32x2*)(a.resid + (int64_t)m * a.N + n);
                        const uint32_t o0 = (uint32_t)f2bf(bf2f(rs.x & 0xFFFFu) + r[0]) |
                                            ((uint32_t)f2bf(bf2f(rs.x >> 16) + r[1]) << 16);
                        const uint32_t o1 = (uint32_t)f2bf(bf2f(rs.y & 0xFFFFu) + r[2]) |
                                            ((uint32_t)f2bf(bf2f(rs.y >> 16) + r[3]) << 16);
                        *(u32x2*)(a.out16 + (int64_t)m * a.N + n) = u32x2{o0, o1};
                    }
                }
            }
        }
    }
}

template <int EPI, int TM, int TN, int MW, int NBW>
static void launch_sg_shape(const Sp24Args& a, hipStream_t st) {
    Sp24Args b = a;
    b.tiles_m = (a.M + TM - 1) / TM;
    b.tiles_n = EPI == EPI_SWIGLU ? (a.F + TN / 2 - 1) / (TN / 2) : (a.N + TN - 1) / TN;
    FP_LAUNCH((gemm_sp24_kernel<EPI, TM, TN, MW, NBW>), dim3(b.tiles_m * b.tiles_n), dim3(SgT<TM, TN, MW, NBW>::NT), 0,
              st, b);
}

// the large tiling from this many 256 x 256 tiles (fewer: 128 x 128 tiles, four times as many)
#ifndef SG_BIG_MIN_TILES
#define SG_BIG_MIN_TILES 128
#endif
template <int EPI>
static void launch_sg(const Sp24Args& a, hipStream_t st) {
    const int big = ((a.M + 255) / 256) * (EPI == EPI_SWIGLU ? (a.F + 127) / 128 : (a.N + 255) / 256);
    if (big >= SG_BIG_MIN_TILES) launch_sg_shape<EPI, 256, 256, 2, 4>(a, st);
    else launch_sg_shape<EPI, 128, 128, 2, 2>(a, st);
}

hipError_t launch_gemm_sp24(const Sp24Args& a, int epi, hipStream_t st) {
    if (a.K % SG_TK != 0 || a.N % 32 != 0 || a.kst != a.K / 32 || a.M < 1) return hipErrorInvalidValue;
    if ((int64_t)a.M * a.K * 2 >= ((int64_t)1 << 32) - 16) return hipErrorInvalidValue;   // 32-bit buffer offsets
    if (epi == EPI_SWIGLU && (a.F % 32 != 0 || a.N != 2 * a.F)) return hipErrorInvalidValue;
    if ((int64_t)(a.N / 32) * a.kst * 1024 >= ((int64_t)1 << 32) - 16) return hipErrorInvalidValue;
    switch (epi) {
        case EPI_F32: launch_sg<EPI_F32>(a, st); break;
        case EPI_RESID: launch_sg<EPI_RESID>(a, st); break;
        case EPI_SWIGLU: launch_sg<EPI_SWIGLU>(a, st); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace fpk
