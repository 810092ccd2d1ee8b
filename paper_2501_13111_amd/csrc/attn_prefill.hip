// Prefill attention: causal attention of a whole prompt, reading K / V back from
// the cache the rotary/append kernel has just written (bf16, or int8 codes with
// per-(position, kv head) scales -- the INT8 KV cache of paper Sec. 3.2), so
// that prefill sees exactly what later decode steps see.
//
// Flash-style on MFMA 32x32x16, written in the transposed form
//     S^T = K Q^T          (A = key rows from LDS, B = the wave's 32 queries)
//     O^T += V^T P^T       (A = value columns from LDS, B = the probabilities already
//                           in the lanes)
// so the probabilities never leave registers: after S^T, lane l holds the scores of
// 16 keys of a 32-key block for its query column l % 32 (element e: key
// 8 (e / 4) + 4 (l / 32) + e % 4).  A 16-key P.V step j takes elements 4j .. 4j+3
// and 4j+8 .. 4j+11, whose keys sit in slots 16 j + 8 (l / 32) .. + 7 of the value
// cache's transposed 32-position blocks (vt_slot order), so each value fragment is one
// contiguous 16-byte piece.
//
// Keys go in 32-key blocks; the LDS holds each block in fragment-major order (one 1 KiB
// chunk per MFMA operand, lane l's 16 bytes at 16 l), so every fragment read is one
// conflict-free ds_read_b128.  Blocks are brought in through registers two blocks ahead
// (loaded at the top of a trip, written to LDS at its end) and the waves meet once per
// block.  Two waves per SIMD; within a wave, the MFMAs of S for block s + 1 are issued
// beside the softmax of block s.
//
// Softmax in the base-2 domain against a fixed reference: each query's maximum over its
// first key block (taken exactly, across the two lane halves) is the reference m for all
// later blocks, whose probabilities exp2(s - m) may then exceed 1.  Softmax does not
// depend on m and bf16 probabilities keep their relative precision over the fp32 range, so
// only overflow matters: a block with a probability above a.pmax (2^64: bf16 probabilities,
// fp32 accumulators) records its exact maximum, and the workgroup repeats the prompt once
// with the larger reference.  The loop never rescales the accumulators, and its P.V MFMAs
// sit on a single path, so they accumulate in place.  Each lane half keeps its own partial
// sum, added once at the end.
//
// int8 caches: K codes are scaled into fp16 on the way to LDS (code * s_k / kappa, kappa =
// the largest key scale of the prompt; fp16 MFMA with the queries in fp16, kappa folded
// into the score scale) and V codes into bf16 (code * s_v / sigma, sigma likewise; sigma
// multiplies the output).  Workgroups of NW waves hold HPW heads that share one kv head
// (GQA: the blocks are staged once for all of them) times NW / HPW consecutive 32-query
// blocks; the heaviest (latest) query tiles are launched first.
#include <type_traits>

#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

constexpr int PK = 32;          // keys per block (= VT_BLK: one value-cache block)

__device__ __forceinline__ uint32_t mul_f16x2(uint32_t x, uint32_t y) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, x) * __builtin_bit_cast(f16x2, y));
}

template <int D, bool KV8, int NW, int HPW>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) attn_prefill_kernel(AttnPreArgs a) {
    static_assert(NW % HPW == 0 && PK == VT_BLK, "workgroup shape");
    constexpr int NT = 64 * NW;
    constexpr int QW = NW / HPW;                // waves (32-query blocks) per head
    // LDS blocks: the one being multiplied, the next one, and the one being written (the
    // buffer of block s is s & (NBUF - 1))
    constexpr int NBUF = 4;
    constexpr int AQ = KV8 ? ACT_F16 : ACT_BF16;  // S = K Q^T operands; P.V runs on bf16
    constexpr int NKC = D / 16;                 // K chunks per block (MFMA k-steps)
    constexpr int NVC = 2 * (D / 32);           // V chunks per block (2 key steps x dim tiles)
    constexpr int CH = NKC + NVC;
    constexpr int SB = CH * 1024;               // LDS bytes per block
    // pieces per thread per block: int8, 4D 8-code pieces of K and as many of V; bf16, one
    // 16-byte piece per lane of each chunk
    constexpr int NPT = KV8 ? (4 * D + NT - 1) / NT : (CH * 64 + NT - 1) / NT;
    __shared__ __attribute__((aligned(1024))) char smem[NBUF * SB];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);     // wave index (uniform)
    const int l32 = lane & 31, h32 = lane >> 5;
    const int ngrp = a.nh / HPW;
    const int b = blockIdx.x / ngrp, hg = blockIdx.x % ngrp;
    const int nqt = (a.P + 32 * QW - 1) / (32 * QW);
    const int qt = nqt - 1 - (int)blockIdx.y;          // heaviest first (y varies slowest)
    const int h = hg * HPW + w % HPW;
    const int kvh = (hg * HPW * a.nkv) / a.nh;         // shared by the HPW heads
    const int q0 = qt * 32 * QW;
    const int wq0 = q0 + 32 * (w / HPW);               // this wave's first query
    const int wglast = min(a.P - 1, q0 + 32 * QW - 1);
    const int ns = wglast / PK + 1;                    // key blocks of the workgroup
    const int wlast = wq0 < a.P ? min(a.P - 1, wq0 + 31) / PK : -1;   // last block of the wave
    const float sl2 = a.scale * 1.4426950408889634f;   // scores in the base-2 domain

    // Q^T fragments for the D/16 k-steps: lane l supplies query l % 32, dims
    // 16 j + 8 (l / 32) .. + 7
    u32x4 qf[D / 16];
    const int qpos = wq0 + l32;
    {
        const bool qv = qpos < a.P;
        const float* qrow = a.q + ((int64_t)b * a.P + (qv ? qpos : 0)) * a.nh * D + h * D;
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (qv) {
                const float4 x0 = *(const float4*)(qrow + 16 * j + 8 * h32);
                const float4 x1 = *(const float4*)(qrow + 16 * j + 8 * h32 + 4);
                if constexpr (KV8) {
                    v[0] = pack_f16_hw(x0.x, x0.y); v[1] = pack_f16_hw(x0.z, x0.w);
                    v[2] = pack_f16_hw(x1.x, x1.y); v[3] = pack_f16_hw(x1.z, x1.w);
                } else {
                    v[0] = pack_bf16_hw(x0.x, x0.y); v[1] = pack_bf16_hw(x0.z, x0.w);
                    v[2] = pack_bf16_hw(x1.x, x1.y); v[3] = pack_bf16_hw(x1.z, x1.w);
                }
            }
            qf[j] = u32x4{v[0], v[1], v[2], v[3]};
        }
    }

    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.kv_stride;   // key row of position 0
    const int64_t vblk0 = ((int64_t)b * a.nkv + kvh) * a.nblk;        // value block of position 0

    // int8: kappa and sigma = the largest key and value scales over the prompt (1 if all
    // are zero); the staged values are code * scale / kappa (or sigma), at most 127
    float kappa = 1.f, sigma = 1.f;
    if constexpr (KV8) {
        float mk = 0.f, mv = 0.f;
        for (int p0 = 0; p0 < a.P; p0 += 512) {      // 8 independent loads per lane and array
            uint16_t kk[8], vv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int p = p0 + 64 * i + lane;
                kk[i] = p < a.P ? a.k_scales[crow0 + p] : (uint16_t)0;
                vv[i] = p < a.P ? a.v_scales[crow0 + p] : (uint16_t)0;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                mk = fmaxf(mk, h2f(kk[i]));
                mv = fmaxf(mv, h2f(vv[i]));
            }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            mk = fmaxf(mk, __shfl_xor(mk, o, 64));
            mv = fmaxf(mv, __shfl_xor(mv, o, 64));
        }
        kappa = mk > 0.f ? mk : 1.f;
        sigma = mv > 0.f ? mv : 1.f;
    }
    const float kinv = 1.0f / kappa, vinv = 1.0f / sigma;
    const float kmul = KV8 ? kappa * sl2 : sl2;        // score = S * kmul (base-2 domain)

    // ---- staging of key block s into buffer s & (NBUF - 1).  Chunk j < NKC: K fragment
    // of k-step j (lane l: key l % 32, dims 16 j + 8 (l / 32) .. + 7); chunk NKC + t,
    // t = j2 (D / 32) + dt: V^T fragment of key step j2, dims 32 dt + l % 32, slots
    // 16 j2 + 8 (l / 32) .. + 7 of the value block.
    const __amdgpu_buffer_rsrc_t kr =
        buf_rsrc((const char*)a.kc + crow0 * D * (KV8 ? 1 : 2), (uint32_t)((int64_t)a.kv_stride * D * (KV8 ? 1 : 2)));
    const __amdgpu_buffer_rsrc_t vr =
        buf_rsrc((const char*)a.vc + vblk0 * D * VT_BLK * (KV8 ? 1 : 2), (uint32_t)((int64_t)a.nblk * D * VT_BLK * (KV8 ? 1 : 2)));
    // bf16: piece p = chunk p / 64, lane slot p % 64, loaded into registers and written to
    // its place in the chunk
    struct RegsB {
        u32x4 v[NPT];
    };
    auto load_bf = [&](int s, RegsB& r) {
#pragma unroll
        for (int i = 0; i < NPT; ++i) {
            const int p = tid + NT * i;
            if (p >= CH * 64) break;
            const int c = p / 64, l = p % 64;
            if (c < NKC) {
                r.v[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    kr, (uint32_t)(((s * PK + l % 32) * D + 16 * c + 8 * (l / 32)) * 2), 0, 0);
            } else {
                const int t = c - NKC, j2 = t / (D / 32), dt = t % (D / 32);
                r.v[i] = __builtin_amdgcn_raw_buffer_load_b128(
                    vr, (uint32_t)((((s * D + 32 * dt + l % 32) * VT_BLK) + 16 * j2 + 8 * (l / 32)) * 2), 0, 0);
            }
        }
    };
    auto store_bf = [&](int s, const RegsB& r) {
        char* base = smem + (s & (NBUF - 1)) * SB;
#pragma unroll
        for (int i = 0; i < NPT; ++i) {
            const int p = tid + NT * i;
            if (p >= CH * 64) break;
            *(u32x4*)(base + p * 16) = r.v[i];
        }
    };
    // int8: 8-code pieces through registers, scaled on the way to LDS (one rounding); each
    // thread takes pieces of both kinds.  K piece p: key p % 32, dims 8 (p / 32) .. + 7, times
    // the key's scale over kappa, fp16.  V piece p: dim p % D, slots 8 o .. 8 o + 7
    // (o = p / D), which hold positions 4 o .. + 3 and 16 + 4 o .. + 3 of the block
    // (vt_slot order), each times its scale over sigma, bf16.  The value scales over sigma
    // (32 per block) are staged in LDS one block ahead of their codes by threads 0 .. 31.
    __shared__ __attribute__((aligned(16))) float vsl[KV8 ? NBUF : 1][PK];
    struct Regs {
        u32x2 k[NPT], v[NPT];
        uint16_t ks[NPT];
        uint16_t vs;
    };
    auto load_codes = [&](int s, Regs& r) {
#pragma unroll
        for (int i = 0; i < NPT; ++i) {
            const int p = tid + NT * i;
            if (p >= 4 * D) break;
            r.k[i] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(
                                                   kr, (uint32_t)((s * PK + p % 32) * D + 8 * (p / 32)), 0, 0));
            r.ks[i] = a.k_scales[crow0 + s * PK + p % 32];
            r.v[i] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(
                                                   vr, (uint32_t)((s * D + p % D) * VT_BLK + 8 * (p / D)), 0, 0));
        }
    };
    auto load_vscale = [&](int s, Regs& r) {
        if (tid < PK) r.vs = a.v_scales[crow0 + s * PK + tid];
    };
    auto store_vscale = [&](int s, const Regs& r) {
        if (tid < PK) vsl[s & (NBUF - 1)][tid] = h2f(r.vs) * vinv;
    };
    auto store_codes = [&](int s, const Regs& r) {
        char* base = smem + (s & (NBUF - 1)) * SB;
        const float* sv = vsl[s & (NBUF - 1)];
#pragma unroll
        for (int i = 0; i < NPT; ++i) {
            const int p = tid + NT * i;
            if (p >= 4 * D) break;
            {
                const int o = p / 32;
                const u32x2 c0 = i8x4_to_f16x4(r.k[i].x), c1 = i8x4_to_f16x4(r.k[i].y);
                const uint32_t k1 = f2h(h2f(r.ks[i]) * kinv), k2 = k1 | (k1 << 16);
                *(u32x4*)(base + (o >> 1) * 1024 + ((p % 32) + 32 * (o & 1)) * 16) =
                    u32x4{mul_f16x2(c0.x, k2), mul_f16x2(c0.y, k2), mul_f16x2(c1.x, k2), mul_f16x2(c1.y, k2)};
            }
            {
                const int o = p / D, dim = p % D;
                const f32x4 sa = *(const f32x4*)(sv + 4 * o), sb = *(const f32x4*)(sv + 16 + 4 * o);
                // code j of a dword: signed byte j, times its position's scale, to bf16
                auto cv = [](uint32_t wd, const f32x4& sc) {
                    return u32x2{pack_bf16_hw((float)(int8_t)wd * sc[0], (float)(int8_t)(wd >> 8) * sc[1]),
                                 pack_bf16_hw((float)(int8_t)(wd >> 16) * sc[2], (float)(int8_t)(wd >> 24) * sc[3])};
                };
                const u32x2 e0 = cv(r.v[i].x, sa), e1 = cv(r.v[i].y, sb);
                *(u32x4*)(base + (NKC + (o >> 1) * (D / 32) + dim / 32) * 1024 + ((dim % 32) + 32 * (o & 1)) * 16) =
                    u32x4{e0.x, e0.y, e1.x, e1.y};
            }
        }
    };

    // ---- softmax helpers.  Element e of a lane holds key offset 8 (e / 4) + e % 4 + 4 h32
    // of the block; it is live when that offset (less 4 h32) is at most lim (the key passes
    // neither the query nor the prompt).
    auto koff = [](int e) { return 8 * (e >> 2) + (e & 3); };
    auto limit = [&](int s) { return min(qpos, a.P - 1) - s * PK - 4 * h32; };
    // probability fragment words: elements e, e + 1 (e even) go to step (e / 4) % 2, word
    // (e % 4) / 2 + 2 (e / 8)
    auto put_pair = [&](u32x4 (&pf)[2], int e, float x0, float x1) {
        pf[(e >> 2) & 1][((e & 3) >> 1) + 2 * (e >> 3)] = pack_bf16_hw(x0, x1);
    };
    // exact maximum of the block's live scores (base-2 domain), across the lane halves
    auto block_max = [&](int s, const f32x16& acc, bool masked) {
        const int lim = masked ? limit(s) : PK;
        float t = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) t = fmaxf(t, koff(e) <= lim ? acc[e] * kmul : -INFINITY);
        return fmaxf(t, __shfl_xor(t, 32, 64));
    };

    f32x16 oacc[D / 32];                            // O^T: dim 32 dt + 8 (e / 4) + 4 (l / 32) + e % 4
    float m_ref = -INFINITY, l_run = 0.f, m_seen = -INFINITY;
    bool over = false;

    auto qk = [&](int s) {
        const char* kb = smem + (s & (NBUF - 1)) * SB + lane * 16;
        f32x16 acc = f32x16{};
#pragma unroll
        for (int j = 0; j < D / 16; ++j) acc = mfma32<AQ>(*(const u32x4*)(kb + j * 1024), qf[j], acc);
        return acc;
    };
    auto pv = [&](int s, const u32x4 (&pf)[2]) {
        const char* vb = smem + (s & (NBUF - 1)) * SB + NKC * 1024 + lane * 16;
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt)
                oacc[dt] = mfma32<ACT_BF16>(*(const u32x4*)(vb + (j2 * (D / 32) + dt) * 1024), pf[j2], oacc[dt]);
    };
    // block 0: its exact maximum (at least the reference carried over) becomes the reference
    auto first_block = [&](bool masked, const f32x16& acc, u32x4 (&pf)[2]) {
        m_ref = fmaxf(m_ref, block_max(0, acc, masked));
        const float ms = m_ref == -INFINITY ? 0.f : m_ref;
        const int lim = masked ? limit(0) : PK;
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            const float x0 = koff(e) <= lim ? __builtin_amdgcn_exp2f(fmaf(acc[e], kmul, -ms)) : 0.f;
            const float x1 = koff(e + 1) <= lim ? __builtin_amdgcn_exp2f(fmaf(acc[e + 1], kmul, -ms)) : 0.f;
            psum += x0 + x1;
            put_pair(pf, e, x0, x1);
        }
        l_run += psum;
    };
    // later blocks: probabilities against the reference, while the MFMAs of S for the
    // next block (into nxt) run
    auto next_block = [&](int s, auto dm, const f32x16& acc, f32x16& nxt, u32x4 (&pf)[2]) {
        constexpr bool DM = decltype(dm)::value;
        nxt = qk(s + 1);
        int lim = 0;
        if constexpr (DM) lim = limit(s);
        float pmax = 0.f, psum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            float v0 = fmaf(acc[e], kmul, -m_ref), v1 = fmaf(acc[e + 1], kmul, -m_ref);
            if constexpr (DM) {
                v0 = koff(e) <= lim ? v0 : -INFINITY;
                v1 = koff(e + 1) <= lim ? v1 : -INFINITY;
            }
            const float x0 = __builtin_amdgcn_exp2f(v0), x1 = __builtin_amdgcn_exp2f(v1);
            pmax = fmaxf(pmax, fmaxf(x0, x1));
            psum += x0 + x1;
            put_pair(pf, e, x0, x1);
        }
        if (__ballot(!(pmax <= a.pmax))) {
            asm volatile("" ::: "memory");     // a real branch: never computed speculatively
            m_seen = fmaxf(m_seen, block_max(s, acc, DM));
            over = true;
        }
        l_run += psum;
    };
    using T_ = std::integral_constant<bool, true>;
    using F_ = std::integral_constant<bool, false>;
    auto masked_block = [&](int s) { return s * PK + PK - 1 > wq0 || s * PK + PK > a.P; };

    // ---- block loop: block s is multiplied while block s + 2 is brought in through
    // registers (int8: and the value scales of block s + 3); the waves meet after each block.
    using Stage = typename std::conditional<KV8, Regs, RegsB>::type;
    Stage rg;
    auto load_block = [&](int s) {
        if constexpr (KV8) load_codes(s, rg);
        else load_bf(s, rg);
    };
    auto store_block = [&](int s) {
        if constexpr (KV8) store_codes(s, rg);
        else store_bf(s, rg);
    };
    auto sync_after = [&](int s) {
        if (s + 2 < ns) store_block(s + 2);
        if constexpr (KV8) {
            if (s + 3 < ns) store_vscale(s + 3, rg);
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    };
    auto prefetch = [&](int s) {
        if (s + 2 < ns) load_block(s + 2);
        if constexpr (KV8) {
            if (s + 3 < ns) load_vscale(s + 3, rg);
        }
    };

    // at most two passes: the second only if a probability left the range, with the
    // largest maximum seen as the reference
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
        l_run = 0.f;
        over = false;
        if constexpr (KV8) {
            // value scales of blocks 0 .. 2 first: a block's codes are scaled with them
            for (int t = 0; t < 3 && t < ns; ++t) {
                load_vscale(t, rg);
                store_vscale(t, rg);
            }
            asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        }
        for (int t = 0; t < 2 && t < ns; ++t) {
            load_block(t);
            store_block(t);
        }
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        // S of block s + 1 is computed in trip s, beside the softmax of block s; the two S
        // registers alternate (two trips per loop turn)
        f32x16 accA, accB;
        prefetch(0);
        {
            u32x4 pf[2] = {u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}};
            if (0 <= wlast) {
                accA = qk(0);
                accB = qk(1);
                first_block(masked_block(0), accA, pf);
            }
            pv(0, pf);
        }
        sync_after(0);
        // the P.V MFMAs stay on one path, so they accumulate in place
        auto trip = [&](int s, const f32x16& cur, f32x16& nxt) {
            prefetch(s);
            u32x4 pf[2];
            if (masked_block(s)) next_block(s, T_{}, cur, nxt, pf);
            else next_block(s, F_{}, cur, nxt, pf);
            pv(s, pf);
            sync_after(s);
        };
        int s = 1;
        for (; s + 1 <= wlast; s += 2) {
            trip(s, accB, accA);
            trip(s + 1, accA, accB);
        }
        if (s <= wlast) trip(s++, accB, accA);
        for (; s < ns; ++s) {                  // a wave past its queries keeps staging blocks
            prefetch(s);
            sync_after(s);
        }
        if (!__syncthreads_or(over)) break;
        m_ref = fmaxf(m_ref, m_seen);
    }

    const float lt = l_run + __shfl_xor(l_run, 32, 64);
    if (qpos >= a.P) return;
    const float inv = (KV8 ? sigma : 1.f) / lt;
    uint16_t* orow = a.out + ((int64_t)b * a.P + qpos) * a.nh * D + h * D;
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4) {
            uint16_t v[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = act_store(bfround(oacc[dt][4 * e4 + i] * inv), a.out_fmt);
            *(u32x2*)(orow + 32 * dt + 8 * e4 + 4 * h32) =
                u32x2{(uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16)};
        }
}

// Workgroups: 32 queries per wave; HPW = the largest of 8, 4, 2, 1 that divides both the
// heads per kv head and the waves; 8 waves (two per SIMD).  bf16 caches drop to 4, 2 or 1
// wave while the grid is under 128 workgroups (a single short prompt: more, smaller
// workgroups spread the causal critical path over more CUs).
template <int D, bool KV8, int NW, int HPW>
static void launch_shape(const AttnPreArgs& a, int B, hipStream_t st) {
    const int wq = 32 * (NW / HPW);
    FP_LAUNCH((attn_prefill_kernel<D, KV8, NW, HPW>), dim3((unsigned)(a.nh / HPW * B), (unsigned)((a.P + wq - 1) / wq)),
              dim3(64 * NW), 0, st, a);
}

template <int D, bool KV8, int NW>
static void launch_nw(const AttnPreArgs& a, int B, int hpw, hipStream_t st) {
    if constexpr (NW >= 8) {
        if (hpw >= 8) return launch_shape<D, KV8, NW, 8>(a, B, st);
    }
    if constexpr (NW >= 4) {
        if (hpw >= 4) return launch_shape<D, KV8, NW, 4>(a, B, st);
    }
    if constexpr (NW >= 2) {
        if (hpw >= 2) return launch_shape<D, KV8, NW, 2>(a, B, st);
    }
    launch_shape<D, KV8, NW, 1>(a, B, st);
}

template <int D, bool KV8>
static hipError_t launch_ap(const AttnPreArgs& a, int B, hipStream_t st) {
    const int gq = a.nh / a.nkv;
    const int hmax = gq % 8 == 0 ? 8 : gq % 4 == 0 ? 4 : gq % 2 == 0 ? 2 : 1;
    auto grid = [&](int n) {
        const int hp = hmax < n ? hmax : n, wq = 32 * (n / hp);
        return (int64_t)((a.P + wq - 1) / wq) * (a.nh / hp) * B;
    };
    int nw = 8;
    if constexpr (!KV8)
        while (nw > 1 && grid(nw) < 128) nw /= 2;
    const int hpw = hmax < nw ? hmax : nw;
    if ((int64_t)(a.nh / hpw) * B > INT_MAX) return hipErrorInvalidValue;
    if (nw == 8) launch_nw<D, KV8, 8>(a, B, hpw, st);
    else if (nw == 4) launch_nw<D, KV8, 4>(a, B, hpw, st);
    else if constexpr (!KV8) {
        if (nw == 2) launch_nw<D, KV8, 2>(a, B, hpw, st);
        else launch_nw<D, KV8, 1>(a, B, hpw, st);
    }
    return hipGetLastError();
}

hipError_t launch_attn_prefill(const AttnPreArgs& a, int B, hipStream_t st) {
    if (B < 1 || a.P < 1 || a.nkv < 1 || a.nh % a.nkv != 0) return hipErrorInvalidValue;
    // every key block of the prompt lies inside the cache rows of its (sequence, kv head)
    if (a.nblk * VT_BLK < a.P || a.kv_stride < a.nblk * VT_BLK) return hipErrorInvalidValue;
    if (a.d == 128) return a.kv_int8 ? launch_ap<128, true>(a, B, st) : launch_ap<128, false>(a, B, st);
    if (a.d == 64) return a.kv_int8 ? launch_ap<64, true>(a, B, st) : launch_ap<64, false>(a, B, st);
    return hipErrorInvalidValue;
}

}  // namespace fpk
