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
// conflict-free ds_read_b128.  The waves meet once per block.  Four waves per workgroup
// and two workgroups per CU (two waves per SIMD, from workgroups that run out of step);
// within a wave, the MFMAs of S for block s + 1 are issued beside the softmax of block s.
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
// Blocks reach the LDS by buffer-to-LDS copies, so no thread holds them in registers:
// each 1 KiB fragment chunk is one copy, issued three blocks ahead into a ring of four
// slots.  int8 caches are first dequantised once per block of the prompt by
// attn_stage_kernel into the same fragment-major layout: K codes into fp16
// (code * s_k / kappa_b, kappa_b the largest key scale of the block's keys inside the
// prompt, so at most 127 in size; fp16 MFMA with the queries in fp16, kappa_b folded into
// the block's score scale and copied with the block) and V codes into bf16 (code * s_v).
// Every workgroup that reads a block then copies it as it would a bf16 cache block, instead
// of dequantising it again.  The copies are issued in asm with explicit wait counts: the
// compiler cannot tell a copy's target slot from the slots being read, and would wait for
// every copy in flight before each LDS read.  Workgroups of NW waves hold HPW heads that
// share one kv head (GQA: the blocks are staged once for all of them) times NW / HPW
// consecutive 32-query blocks; the heaviest (latest) query tiles are launched first.
#include <type_traits>

#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

constexpr int PK = 32;          // keys per block (= VT_BLK: one value-cache block)

__device__ __forceinline__ uint32_t mul_f16x2(uint32_t x, uint32_t y) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(f16x2, x) * __builtin_bit_cast(f16x2, y));
}

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

// The four words of a raw buffer resource over [base, base + bytes): no stride, 32-bit data
// format (the resource __builtin_amdgcn_make_buffer_rsrc builds), for copies written in asm.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
    const uint64_t p = (uint64_t)base;
    return i32x4{(int32_t)(uint32_t)p, (int32_t)((uint32_t)(p >> 32) & 0xFFFFu), (int32_t)bytes, 0x00020000};
}

// Buffer-to-LDS copy: lane l's W bytes (16 or 4) at voff + soff of the resource land at LDS
// address lds + W l (past the resource's end: zeros).  M0 carries the LDS address and is
// restored afterwards; one wait state separates its write from the copy.
template <int W>
__device__ __forceinline__ void lds_copy(const i32x4& r, uint32_t voff, uint32_t soff, uint32_t lds) {
    uint32_t keep;
    if constexpr (W == 16)
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                     "buffer_load_dwordx4 %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
                     : "=&s"(keep) : "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory");
    else
        asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                     "buffer_load_dword %2, %3, %4 offen lds\n\ts_mov_b32 m0, %0"
                     : "=&s"(keep) : "s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory");
}

template <int D, bool KV8, int NW, int HPW>
__global__ void __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) attn_prefill_kernel(AttnPreArgs a) {
    static_assert(NW % HPW == 0 && PK == VT_BLK, "workgroup shape");
    constexpr int NT = 64 * NW;
    constexpr int QW = NW / HPW;                // waves (32-query blocks) per head
    constexpr int AQ = KV8 ? ACT_F16 : ACT_BF16;  // S = K Q^T operands; P.V runs on bf16
    constexpr int NKC = D / 16;                 // K chunks per block (MFMA k-steps)
    constexpr int NVC = 2 * (D / 32);           // V chunks per block (2 key steps x dim tiles)
    constexpr int CH = NKC + NVC;
    constexpr int SB = CH * 1024;               // LDS bytes per staged block
    // fragment ring: copies land 3 blocks ahead (4 slots, block b in slot b & 3)
    constexpr int NBF = 4;
    constexpr int AHEAD = 3;                    // copies of block s + AHEAD start in trip s
    // copy jobs per block and wave: the CH chunks; int8, also the block's kappa (a 4-byte
    // copy by every wave, into the slot's kappa row)
    static_assert(CH % NW == 0, "copy jobs spread evenly over the waves");
    constexpr int JPW = CH / NW + (KV8 ? 1 : 0);
    constexpr int SBK = SB + 256;               // int8: bytes per staged block (kappa row last)
    __shared__ __attribute__((aligned(1024))) char smem[NBF * SB];
    __shared__ __attribute__((aligned(16))) float kap[KV8 ? NBF : 1][64];   // int8: kappa rows

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);     // wave index (uniform)
    const int l32 = lane & 31, h32 = lane >> 5;
    // workgroup -> (sequence, kv head, head group, query tile); a unit is a head group times
    // a query tile of one (sequence, kv head).  Workgroup i runs on XCD i % 8: each XCD takes
    // its own kv heads, W at a time (W = 8, 4, 2 or 1, whichever divides its share), and
    // runs the W heads' units heaviest first across the W (the latest query tiles of all W,
    // then the next ones, ...).  The units of a kv head then stream the same blocks at about
    // the same time through that XCD's L2, and the W heads keep its CUs balanced.  Grids
    // whose kv heads do not split evenly over the XCDs go heaviest first over the whole grid.
    const int hgs = a.nh / a.nkv / HPW;                // head groups per kv head
    const int nqt = (a.P + 32 * QW - 1) / (32 * QW);
    const int units = hgs * nqt;
    const int ngroups = (int)gridDim.x / units;       // sequences x kv heads
    const int L = blockIdx.x;
    int g, u;
    if (ngroups % 8 == 0) {
        const int per = ngroups / 8;
        const int W = per % 8 == 0 ? 8 : per % 4 == 0 ? 4 : per % 2 == 0 ? 2 : 1;
        const int k = L >> 3, nwin = W * units, idx = k % nwin;
        g = ((k / nwin) * W + idx % W) * 8 + (L & 7);
        u = idx / W;
    } else {
        const int hgi = L % hgs;
        g = (L / hgs) % ngroups;
        u = L / (hgs * ngroups) * hgs + hgi;
    }
    const int b = g / a.nkv, kvh = g % a.nkv;
    const int qt = nqt - 1 - u / hgs;
    const int h = (kvh * hgs + u % hgs) * HPW + w % HPW;
    const int q0 = qt * 32 * QW;
    const int wq0 = q0 + 32 * (w / HPW);               // this wave's first query
    const int wglast = min(a.P - 1, q0 + 32 * QW - 1);
    const int ns = wglast / PK + 1;                    // key blocks of the workgroup
    const int wlast = wq0 < a.P ? min(a.P - 1, wq0 + 31) / PK : -1;   // last block of the wave
    const float sl2 = a.scale * 1.4426950408889634f;   // scores in the base-2 domain

    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.kv_stride;   // key row of position 0
    const int64_t vblk0 = ((int64_t)b * a.nkv + kvh) * a.nblk;        // value block of position 0
    const int nsb = (a.P + PK - 1) / PK;               // int8: staged blocks per (sequence, kv head)
    i32x4 rk, rv;
    if constexpr (KV8) {
        rk = rsrc_words((const char*)a.staged + (int64_t)g * nsb * SBK, (uint32_t)((int64_t)nsb * SBK));
        rv = rk;
    } else {
        rk = rsrc_words((const char*)a.kc + crow0 * D * 2, (uint32_t)((int64_t)a.kv_stride * D * 2));
        rv = rsrc_words((const char*)a.vc + vblk0 * D * VT_BLK * 2, (uint32_t)((int64_t)a.nblk * D * VT_BLK * 2));
    }
    // the wave's copy jobs (job j = w + NW i): kind, per-lane offset, place in the slot
    // (wave-uniform)
    uint32_t jv[JPW];
    int jkind[JPW];                                    // 0 K, 1 V, 2 kappa row
    uint32_t jl[JPW];
#pragma unroll
    for (int i = 0; i < JPW; ++i) {
        const int j = w + NW * i;
        if (KV8 && i == JPW - 1) {
            jkind[i] = 2;
            jv[i] = (uint32_t)(SB + 4 * lane);
            jl[i] = 0;
        } else if constexpr (KV8) {                    // staged blocks are fragment-major already
            jkind[i] = 0;
            jv[i] = (uint32_t)(j * 1024 + 16 * lane);
            jl[i] = (uint32_t)(j * 1024);
        } else {
            jl[i] = (uint32_t)(j * 1024);
            if (j < NKC) {       // key l % 32, dims 16 j + 8 (l / 32) .. + 7
                jkind[i] = 0;
                jv[i] = (uint32_t)(((lane % 32) * D + 16 * j + 8 * (lane / 32)) * 2);
            } else {             // value dims 32 dt + l % 32, slots 16 j2 + 8 (l / 32) .. + 7
                const int t = j - NKC, j2 = t / (D / 32), dt = t % (D / 32);
                jkind[i] = 1;
                jv[i] = (uint32_t)((((32 * dt + lane % 32) * VT_BLK) + 16 * j2 + 8 * (lane / 32)) * 2);
            }
        }
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lvoid_t*)smem;
    const uint32_t kap0 = (uint32_t)(uintptr_t)(lvoid_t*)&kap[0][0];
    auto slot = [](int bb) { return bb & (NBF - 1); };
    // copies of block bb (past the workgroup's blocks: of its last block, into bb's free
    // slot, so that every wave issues JPW copies per block and the wait counts stay exact)
    auto issue = [&](int bb) {
        const int bc = min(bb, ns - 1);
#pragma unroll
        for (int i = 0; i < JPW; ++i) {
            const int k = jkind[i];
            if (k == 2) {
                lds_copy<4>(rk, jv[i], (uint32_t)(bc * SBK), kap0 + (uint32_t)slot(bb) * 256u);
            } else {
                const uint32_t dst = (uint32_t)__builtin_amdgcn_readfirstlane(lds0 + slot(bb) * SB + jl[i]);
                if constexpr (KV8) lds_copy<16>(rk, jv[i], (uint32_t)(bc * SBK), dst);
                else if (k == 0) lds_copy<16>(rk, jv[i], (uint32_t)(bc * PK * D * 2), dst);
                else lds_copy<16>(rv, jv[i], (uint32_t)(bc * D * VT_BLK * 2), dst);
            }
        }
    };
    // all but the copies issued in the current trip are complete
    auto wait_older_copies = [&]() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(JPW) : "memory"); };
    auto wait_all_copies = [&]() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
    auto barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

    // the first blocks' copies go out before the queries are read
    issue(0);
    issue(1);
    issue(2);

    // Q^T fragments for the D/16 k-steps (the rotary step wrote them in the operand
    // format): lane l supplies query l % 32, dims 16 j + 8 (l / 32) .. + 7.  Every load is
    // issued before any is used (one round trip); lanes past the prompt read row 0 and
    // keep zeros.
    u32x4 qf[D / 16];
    const int qpos = wq0 + l32;
    {
        const bool qv = qpos < a.P;
        const uint16_t* qrow = a.q + (((int64_t)b * a.nh + h) * a.P + (qv ? qpos : 0)) * D;
        u32x4 x[D / 16];
#pragma unroll
        for (int j = 0; j < D / 16; ++j) x[j] = *(const u32x4*)(qrow + 16 * j + 8 * h32);
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
            qf[j] = qv ? x[j] : u32x4{0u, 0u, 0u, 0u};
            // the loads are complete here: the compiler does not see the asm waits, and its
            // own wait for them would otherwise sit inside the block loop (before the first
            // MFMA of every trip) and drain the block copies in flight
            asm volatile("" : "+v"(qf[j]));
        }
    }
    // score multiplier of block bb (base-2 domain): int8, times the block's kappa
    auto kmul_of = [&](int bb) { return KV8 ? kap[slot(bb)][0] * sl2 : sl2; };

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
    auto block_max = [&](int s, const f32x16& acc, bool masked, float km) {
        const int lim = masked ? limit(s) : PK;
        float t = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) t = fmaxf(t, koff(e) <= lim ? acc[e] * km : -INFINITY);
        return fmaxf(t, __shfl_xor(t, 32, 64));
    };

    f32x16 oacc[D / 32];                            // O^T: dim 32 dt + 8 (e / 4) + 4 (l / 32) + e % 4
    float m_ref = -INFINITY, l_run = 0.f, m_seen = -INFINITY;
    bool over = false;

    auto qk = [&](int s) {
        const char* kb = smem + slot(s) * SB + lane * 16;
        f32x16 acc = f32x16{};
#pragma unroll
        for (int j = 0; j < D / 16; ++j) acc = mfma32<AQ>(*(const u32x4*)(kb + j * 1024), qf[j], acc);
        return acc;
    };
    auto pv = [&](int s, const u32x4 (&pf)[2]) {
        const char* vb = smem + slot(s) * SB + NKC * 1024 + lane * 16;
#pragma unroll
        for (int j2 = 0; j2 < 2; ++j2)
#pragma unroll
            for (int dt = 0; dt < D / 32; ++dt)
                oacc[dt] = mfma32<ACT_BF16>(*(const u32x4*)(vb + (j2 * (D / 32) + dt) * 1024), pf[j2], oacc[dt]);
    };
    // block 0: its exact maximum (at least the reference carried over) becomes the reference
    auto first_block = [&](bool masked, const f32x16& acc, u32x4 (&pf)[2]) {
        const float km = kmul_of(0);
        m_ref = fmaxf(m_ref, block_max(0, acc, masked, km));
        const float ms = m_ref == -INFINITY ? 0.f : m_ref;
        const int lim = masked ? limit(0) : PK;
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            const float x0 = koff(e) <= lim ? __builtin_amdgcn_exp2f(fmaf(acc[e], km, -ms)) : 0.f;
            const float x1 = koff(e + 1) <= lim ? __builtin_amdgcn_exp2f(fmaf(acc[e + 1], km, -ms)) : 0.f;
            psum += x0 + x1;
            put_pair(pf, e, x0, x1);
        }
        l_run += psum;
    };
    // later blocks: probabilities against the reference, while the MFMAs of S for the
    // next block (into nxt) run
    auto next_block = [&](int s, auto dm, const f32x16& acc, f32x16& nxt, u32x4 (&pf)[2]) {
        constexpr bool DM = decltype(dm)::value;
        const float km = kmul_of(s);
        nxt = qk(s + 1);
        int lim = 0;
        if constexpr (DM) lim = limit(s);
        float pmax = 0.f, psum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            float v0 = fmaf(acc[e], km, -m_ref), v1 = fmaf(acc[e + 1], km, -m_ref);
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
            m_seen = fmaxf(m_seen, block_max(s, acc, DM, km));
            over = true;
        }
        l_run += psum;
    };
    using T_ = std::integral_constant<bool, true>;
    using F_ = std::integral_constant<bool, false>;
    auto masked_block = [&](int s) { return s * PK + PK - 1 > wq0 || s * PK + PK > a.P; };

    // ---- block loop.  Trip s multiplies block s (and S of block s + 1) while the copies of
    // block s + AHEAD are in flight; at its end the copies of the previous trip are complete,
    // and the waves meet.
    auto trip_begin = [&](int s) { issue(s + AHEAD); };
    auto trip_end = [&](int s) {
        wait_older_copies();
        barrier();
    };

    // at most two passes: the second only if a probability left the range, with the
    // largest maximum seen as the reference
    for (int pass = 0; pass < 2; ++pass) {
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
        l_run = 0.f;
        over = false;
        if (pass > 0) {                  // copies left by the first pass go to free slots
            wait_all_copies();
            barrier();
            issue(0);
            issue(1);
            issue(2);
        }
        wait_all_copies();
        barrier();
        // S of block s + 1 is computed in trip s, beside the softmax of block s; the two S
        // registers alternate (two trips per loop turn)
        f32x16 accA, accB;
        trip_begin(0);
        {
            u32x4 pf[2] = {u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}};
            if (0 <= wlast) {
                accA = qk(0);
                accB = qk(1);
                first_block(masked_block(0), accA, pf);
            }
            pv(0, pf);
        }
        trip_end(0);
        // the P.V MFMAs stay on one path, so they accumulate in place
        auto trip = [&](int s, const f32x16& cur, f32x16& nxt) {
            trip_begin(s);
            u32x4 pf[2];
            if (masked_block(s)) next_block(s, T_{}, cur, nxt, pf);
            else next_block(s, F_{}, cur, nxt, pf);
            pv(s, pf);
            trip_end(s);
        };
        int s = 1;
        for (; s + 1 <= wlast; s += 2) {
            trip(s, accB, accA);
            trip(s + 1, accA, accB);
        }
        if (s <= wlast) trip(s++, accB, accA);
        for (; s < ns; ++s) {                  // a wave past its queries keeps staging blocks
            trip_begin(s);
            trip_end(s);
        }
        if (!__syncthreads_or(over)) break;
        m_ref = fmaxf(m_ref, m_seen);
    }
    wait_all_copies();                         // no copy outlives the workgroup

    const float lt = l_run + __shfl_xor(l_run, 32, 64);
    if (qpos >= a.P) return;
    const float inv = 1.f / lt;
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

// Short prompts with bf16 caches (a grid of fewer workgroups than CUs in the layout
// above: one sequence, few heads): the layout above leaves most SIMDs empty and the
// latest query tile walks every key block alone.  Here a workgroup takes one 32-query
// block of one head and its four waves split the key blocks (wave w takes blocks w, w + 4,
// ...), so the chain of dependent blocks is a quarter as long and the grid four times
// larger.  Each wave loads its blocks' MFMA fragments straight into registers (block s + 4
// is in flight while block s is multiplied) and keeps an online softmax: a running
// maximum m per query, the accumulators and the sum rescaled by exp2(m_old - m_new) when
// m grows.  The four partial (m, l, O) then merge through LDS: M = max m_w, O = sum
// O_w exp2(m_w - M), l likewise, and the output is O / l rounded to bf16: the same causal
// softmax attention as the kernel above, up to rounding order.
template <int D>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) attn_prefill_ks_kernel(AttnPreArgs a) {
    constexpr int NKC = D / 16;                 // K fragment chunks per block
    constexpr int NVC = 2 * (D / 32);           // V fragment chunks per block
    constexpr int RS = D + 4;                   // LDS row stride of a partial (floats)
    __shared__ __attribute__((aligned(16))) float po[4][32 * RS];
    __shared__ float pm[4][32], pl[4][32];

    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, h32 = lane >> 5;
    // workgroup -> (query block, sequence, head): the first half of the grid takes the
    // latest query blocks first, the second half the earliest first, so that the two
    // workgroups a CU holds at a time (i and i + half the grid) carry about equal work
    const int nqb = (a.P + 31) / 32;
    const int nbh = (int)gridDim.x / nqb;       // sequences x heads
    const int L = blockIdx.x;
    const int u = L / nbh, hq = (nqb + 1) / 2;
    const int qb = u < hq ? nqb - 1 - u : u - hq;
    const int b = (L % nbh) / a.nh, h = (L % nbh) % a.nh;
    const int kvh = h / (a.nh / a.nkv);
    const int q0 = 32 * qb;
    const int nb = min(a.P - 1, q0 + 31) / PK + 1;     // key blocks of the query block
    const int nmine = nb > w ? (nb - w + 3) / 4 : 0;   // this wave's blocks: w + 4 i
    const float sl2 = a.scale * 1.4426950408889634f;

    const uint16_t* kbase = (const uint16_t*)a.kc + ((int64_t)b * a.nkv + kvh) * a.kv_stride * D;
    const uint16_t* vbase = (const uint16_t*)a.vc + ((int64_t)b * a.nkv + kvh) * a.nblk * D * VT_BLK;
    // fragment pieces of lane l: K key l % 32, dims 16 j + 8 (l / 32) .. + 7; V dims
    // 32 dt + l % 32, keys 16 j2 + 8 (l / 32) .. + 7 (chunk j2 (D / 32) + dt)
    const int koffl = l32 * D + 8 * h32;
    const int voffl = l32 * VT_BLK + 8 * h32;
    struct Blk {
        u32x4 k[NKC], v[NVC];
    };
    // loads of the wave's i-th block (past its last: the last again, from L2; nothing is
    // loaded by a wave without blocks)
    auto load = [&](int i, Blk& x) {
        const int s = w + 4 * min(i, nmine - 1);
        const uint16_t* kp = kbase + (int64_t)s * PK * D + koffl;
        const uint16_t* vp = vbase + (int64_t)s * D * VT_BLK + voffl;
#pragma unroll
        for (int j = 0; j < NKC; ++j) x.k[j] = *(const u32x4*)(kp + 16 * j);
#pragma unroll
        for (int t = 0; t < NVC; ++t) x.v[t] = *(const u32x4*)(vp + (t % (D / 32)) * 32 * VT_BLK + 16 * (t / (D / 32)));
    };

    // Q^T fragments: lane l supplies query l % 32, dims 16 j + 8 (l / 32) .. + 7; lanes
    // past the prompt keep zeros
    u32x4 qf[NKC];
    const int qpos = q0 + l32;
    {
        const bool qv = qpos < a.P;
        const uint16_t* qrow = a.q + (((int64_t)b * a.nh + h) * a.P + (qv ? qpos : 0)) * D;
#pragma unroll
        for (int j = 0; j < NKC; ++j) {
            const u32x4 x = *(const u32x4*)(qrow + 16 * j + 8 * h32);
            qf[j] = qv ? x : u32x4{0u, 0u, 0u, 0u};
        }
    }

    // element e of a lane's scores holds key 8 (e / 4) + e % 4 + 4 h32 of the block; it is
    // live when that key passes neither the query nor the prompt
    auto koff = [](int e) { return 8 * (e >> 2) + (e & 3); };
    f32x16 oacc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;
    auto block = [&](int i, const Blk& x) {
        const int s = w + 4 * i;
        f32x16 acc = f32x16{};
#pragma unroll
        for (int j = 0; j < NKC; ++j) acc = mfma32<ACT_BF16>(x.k[j], qf[j], acc);
        const int lim = min(qpos, a.P - 1) - s * PK - 4 * h32;
        float t = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            acc[e] = koff(e) <= lim ? acc[e] * sl2 : -INFINITY;
            t = fmaxf(t, acc[e]);
        }
        const float m_new = fmaxf(m_run, fmaxf(t, __shfl_xor(t, 32, 64)));
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);     // 0 on the first block
        m_run = m_new;
        u32x4 pf[2];
        float psum = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            const float x0 = __builtin_amdgcn_exp2f(acc[e] - m_new), x1 = __builtin_amdgcn_exp2f(acc[e + 1] - m_new);
            psum += x0 + x1;
            pf[(e >> 2) & 1][((e & 3) >> 1) + 2 * (e >> 3)] = pack_bf16_hw(x0, x1);
        }
        l_run = l_run * alpha + psum;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
            oacc[dt] *= alpha;
#pragma unroll
            for (int j2 = 0; j2 < 2; ++j2) oacc[dt] = mfma32<ACT_BF16>(x.v[j2 * (D / 32) + dt], pf[j2], oacc[dt]);
        }
    };
    if (nmine > 0) {
        Blk xa, xb;
        load(0, xa);
        load(1, xb);
        int i = 0;
        for (; i + 2 <= nmine; i += 2) {
            block(i, xa);
            load(i + 2, xa);
            block(i + 1, xb);
            load(i + 3, xb);
        }
        if (i < nmine) block(i, xa);
    }

    // merge the four waves' partials
    const float lt = l_run + __shfl_xor(l_run, 32, 64);
    if (h32 == 0) {
        pm[w][l32] = m_run;
        pl[w][l32] = lt;
    }
    __syncthreads();
    float mm = pm[0][l32];
#pragma unroll
    for (int v = 1; v < 4; ++v) mm = fmaxf(mm, pm[v][l32]);
    const float f = nmine > 0 ? __builtin_amdgcn_exp2f(m_run - mm) : 0.f;
    // O^T element (dt, e) of lane l: dim 32 dt + 8 (e / 4) + 4 h32 + e % 4, query l % 32
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int e4 = 0; e4 < 4; ++e4)
            *(f32x4*)&po[w][l32 * RS + 32 * dt + 8 * e4 + 4 * h32] =
                f32x4{oacc[dt][4 * e4] * f, oacc[dt][4 * e4 + 1] * f, oacc[dt][4 * e4 + 2] * f, oacc[dt][4 * e4 + 3] * f};
    __syncthreads();
    // thread t writes query t / 8, dims D / 8 (t % 8) .. + D / 8 - 1
    constexpr int DPT = D / 8;
    const int oq = tid >> 3, d0 = DPT * (tid & 7);
    if (q0 + oq >= a.P) return;
    float mq = pm[0][oq];
#pragma unroll
    for (int v = 1; v < 4; ++v) mq = fmaxf(mq, pm[v][oq]);
    float lsum = 0.f;
#pragma unroll
    for (int v = 0; v < 4; ++v) lsum += v < nb ? pl[v][oq] * __builtin_amdgcn_exp2f(pm[v][oq] - mq) : 0.f;
    const float inv = 1.f / lsum;
    uint16_t* orow = a.out + ((int64_t)b * a.P + q0 + oq) * a.nh * D + h * D + d0;
#pragma unroll
    for (int c = 0; c < DPT; c += 8) {
        uint32_t wd[4];
#pragma unroll
        for (int i2 = 0; i2 < 8; i2 += 2) {
            float o0 = 0.f, o1 = 0.f;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                o0 += po[v][oq * RS + d0 + c + i2];
                o1 += po[v][oq * RS + d0 + c + i2 + 1];
            }
            wd[i2 / 2] = (uint32_t)act_store(bfround(o0 * inv), a.out_fmt) |
                         ((uint32_t)act_store(bfround(o1 * inv), a.out_fmt) << 16);
        }
        *(u32x4*)(orow + c) = u32x4{wd[0], wd[1], wd[2], wd[3]};
    }
}

// int8 caches: dequantise block blk of the prompt of (sequence, kv head) g into the
// fragment-major layout attn_prefill_kernel copies: K chunk c, lane l = key l % 32, dims
// 16 c + 8 (l / 32) .. + 7 as fp16 code * s_k / kappa_b; V chunk NKC + t (t = j2 (D / 32) +
// dt), lane l = dim 32 dt + l % 32, slots 16 j2 + 8 (l / 32) .. + 7 as bf16 code * s_v
// (slots 8 o .. 8 o + 7 hold positions 4 o .. + 3 and 16 + 4 o .. + 3, vt_slot order); then
// kappa_b 64 times.  Positions past the prompt become zeros.
template <int D>
__global__ void __launch_bounds__(256) attn_stage_kernel(AttnPreArgs a) {
    constexpr int NKC = D / 16, NVC = 2 * (D / 32), CH = NKC + NVC, SBK = CH * 1024 + 256;
    const int blk = blockIdx.x, g = blockIdx.y, nsb = gridDim.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int64_t crow0 = (int64_t)g * a.kv_stride;
    const int p0 = blk * PK;
    char* out = (char*)a.staged + ((int64_t)g * nsb + blk) * SBK;
    // kappa_b: lanes l and l + 32 of every wave take key l % 32 (the key of all their K items)
    const int key = lane & 31;
    const float ks0 = h2f(a.k_scales[crow0 + p0 + key]);
    const float ks = p0 + key < a.P ? ks0 : 0.f;
    float km = ks;
#pragma unroll
    for (int o = 16; o >= 1; o >>= 1) km = fmaxf(km, __shfl_xor(km, o, 32));
    const float kappa = km > 0.f ? km : 1.f;
    if (tid < 64) ((float*)(out + CH * 1024))[tid] = kappa;
    const uint32_t k1 = f2h(ks / kappa), k2 = k1 | (k1 << 16);
    for (int it = tid; it < NKC * 64; it += 256) {
        const int c = it / 64;
        const u32x2 code = *(const u32x2*)((const int8_t*)a.kc + (crow0 + p0 + key) * D + 16 * c + 8 * (lane / 32));
        const u32x2 c0 = i8x4_to_f16x4(code.x), c1 = i8x4_to_f16x4(code.y);
        *(u32x4*)(out + c * 1024 + lane * 16) =
            u32x4{mul_f16x2(c0.x, k2), mul_f16x2(c0.y, k2), mul_f16x2(c1.x, k2), mul_f16x2(c1.y, k2)};
    }
    const uint16_t* vs = a.v_scales + crow0 + p0;
    for (int it = tid; it < NVC * 64; it += 256) {
        const int t = it / 64, j2 = t / (D / 32), dt = t % (D / 32);
        const int dim = 32 * dt + lane % 32, o = 2 * j2 + lane / 32;
        const u32x2 code = *(const u32x2*)((const int8_t*)a.vc + (((int64_t)g * a.nblk + blk) * D + dim) * VT_BLK + 8 * o);
        // positions 4 o .. + 3 and 16 + 4 o .. + 3: whole 8-byte words inside the cache rows
        // (rows are whole blocks), positions past the prompt zeroed after the load
        const u32x2 sa = *(const u32x2*)(vs + 4 * o), sb = *(const u32x2*)(vs + 16 + 4 * o);
        const uint32_t sw[4] = {sa.x, sa.y, sb.x, sb.y};
        float sc[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int pos = p0 + (i < 4 ? 4 * o + i : 16 + 4 * o + i - 4);
            const float v = h2f((uint16_t)(sw[i / 2] >> (16 * (i & 1))));
            sc[i] = pos < a.P ? v : 0.f;
        }
        auto cv = [&](uint32_t wd, int i0) {
            return u32x2{pack_bf16_hw((float)(int8_t)wd * sc[i0], (float)(int8_t)(wd >> 8) * sc[i0 + 1]),
                         pack_bf16_hw((float)(int8_t)(wd >> 16) * sc[i0 + 2], (float)(int8_t)(wd >> 24) * sc[i0 + 3])};
        };
        const u32x2 e0 = cv(code.x, 0), e1 = cv(code.y, 4);
        *(u32x4*)(out + (NKC + t) * 1024 + lane * 16) = u32x4{e0.x, e0.y, e1.x, e1.y};
    }
}

size_t attn_stage_bytes(int B, int P, int nkv, int d) {
    return (size_t)B * nkv * ((P + PK - 1) / PK) * (size_t)(4 * d / 16 * 1024 + 256);
}

hipError_t launch_attn_stage(const AttnPreArgs& a, int B, hipStream_t st) {
    if (!a.kv_int8 || a.staged == nullptr || B < 1 || a.P < 1 || a.nkv < 1) return hipErrorInvalidValue;
    if (a.nblk * VT_BLK < a.P || a.kv_stride < a.nblk * VT_BLK || a.kv_stride % 4 != 0) return hipErrorInvalidValue;
    const dim3 grid((unsigned)((a.P + PK - 1) / PK), (unsigned)(B * a.nkv));
    if (a.d == 128) FP_LAUNCH(attn_stage_kernel<128>, grid, dim3(256), 0, st, a);
    else if (a.d == 64) FP_LAUNCH(attn_stage_kernel<64>, grid, dim3(256), 0, st, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// Workgroups: 32 queries per wave; HPW = the largest of 4, 2, 1 that divides both the heads
// per kv head and the waves; 4 waves, two workgroups per CU.  bf16 caches drop to 2 or 1
// wave while the grid is under 128 workgroups (a single short prompt: more, smaller
// workgroups spread the causal critical path over more CUs).
template <int D, bool KV8, int NW, int HPW>
static void launch_shape(const AttnPreArgs& a, int B, hipStream_t st) {
    const int wq = 32 * (NW / HPW);
    const int64_t n = (int64_t)B * (a.nh / HPW) * ((a.P + wq - 1) / wq);
    FP_LAUNCH((attn_prefill_kernel<D, KV8, NW, HPW>), dim3((unsigned)n), dim3(64 * NW), 0, st, a);
}

template <int D, bool KV8, int NW>
static void launch_nw(const AttnPreArgs& a, int B, int hpw, hipStream_t st) {
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
    const int hmax = gq % 4 == 0 ? 4 : gq % 2 == 0 ? 2 : 1;
    auto grid = [&](int n) {
        const int hp = hmax < n ? hmax : n, wq = 32 * (n / hp);
        return (int64_t)((a.P + wq - 1) / wq) * (a.nh / hp) * B;
    };
    if constexpr (!KV8) {
        // fewer workgroups than CUs: split each query block's keys over four waves
        if (grid(4) < 256) {
            const int64_t n = (int64_t)((a.P + 31) / 32) * a.nh * B;
            if (n > INT_MAX) return hipErrorInvalidValue;
            FP_LAUNCH(attn_prefill_ks_kernel<D>, dim3((unsigned)n), dim3(256), 0, st, a);
            return hipGetLastError();
        }
    }
    const int nw = 4;
    const int hpw = hmax < nw ? hmax : nw;
    if ((int64_t)(a.nh / hpw) * B * ((a.P + 31) / 32) > INT_MAX) return hipErrorInvalidValue;
    launch_nw<D, KV8, 4>(a, B, hpw, st);
    return hipGetLastError();
}

hipError_t launch_attn_prefill(const AttnPreArgs& a, int B, hipStream_t st) {
    if (B < 1 || a.P < 1 || a.nkv < 1 || a.nh % a.nkv != 0) return hipErrorInvalidValue;
    if (a.kv_int8 && a.staged == nullptr) return hipErrorInvalidValue;
    // every key block of the prompt lies inside the cache rows of its (sequence, kv head)
    if (a.nblk * VT_BLK < a.P || a.kv_stride < a.nblk * VT_BLK) return hipErrorInvalidValue;
    if (a.d == 128) return a.kv_int8 ? launch_ap<128, true>(a, B, st) : launch_ap<128, false>(a, B, st);
    if (a.d == 64) return a.kv_int8 ? launch_ap<64, true>(a, B, st) : launch_ap<64, false>(a, B, st);
    return hipErrorInvalidValue;
}

}  // namespace fpk
