// Prefill attention: causal attention of a whole prompt, reading K / V back from
// the cache the rotary/append kernel has just written (bf16, or int8 codes with
// per-(position, kv head) scales -- the INT8 KV cache of paper Sec. 3.2), so
// that prefill sees exactly what later decode steps see.
//
// Flash-style on MFMA 32x32x16, written in the transposed form
//     S^T = K Q^T          (A = key rows from LDS, B = the wave's 32 queries)
//     O^T += V^T P^T       (A = value columns, B = the probabilities already in
//                           the lanes)
// so the probabilities never leave registers: after S^T, lane l holds the scores of
// 16 keys of a 32-key subtile for its query column l % 32 (element e: key
// 8 (e / 4) + 4 (l / 32) + e % 4).  A 16-key P.V step j takes elements 4j .. 4j+3
// and 4j+8 .. 4j+11, whose keys sit in slots 16 j + 8 (l / 32) .. + 7 of the
// value cache's transposed 32-position blocks (vt_slot order), so each value
// fragment is one contiguous 16-byte LDS read.
// Online softmax per query column (max / sum across the two lane halves by one
// shuffle).  int8 caches: codes are exact in fp16; s_k scales the scores and s_v
// the probabilities.  Heaviest (latest) query tiles are launched first.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

// Workgroup = NW waves x 32 queries of one head (8 waves, or 4 when 8-wave workgroups
// would leave CUs idle); key tiles of 64 are staged in LDS
// (double buffered: the next tile is loaded into registers while the current one is
// multiplied, then written to the other buffer; a bare barrier keeps those loads in
// flight).  A bf16 cache runs on bf16 MFMA; an int8 cache is converted to exact fp16
// codes while staging and runs on fp16 MFMA (queries and probabilities in fp16).
// Scores are kept in the base-2 domain (scaled by log2 e) so each probability is
// one exp2; the causal mask is applied only on tiles that reach past the wave's
// first query.
constexpr int PKT = 64;          // keys per tile

template <int D, bool KV8, int NW>
__global__ void __launch_bounds__(64 * NW, 8 / NW) attn_prefill_kernel(AttnPreArgs a) {
    constexpr int NT = 64 * NW;   // threads
    constexpr int PQ = 32 * NW;   // queries per workgroup
    constexpr int AF = KV8 ? ACT_F16 : ACT_BF16;
    constexpr int KP = D + 8;     // padded row of the key tile (u16)
    constexpr int VP = PKT + 8;   // padded row of the value tile (u16), slots in vt_slot order
    constexpr int KSZ = PKT * KP, VSZ = D * VP;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][KSZ];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[2][VSZ];
    __shared__ float ksc[2][PKT], vsc[2][PKT];
    // register staging: 16-byte pieces of the K tile and of the two value blocks
    constexpr int KPC = PKT * D * (KV8 ? 1 : 2) / 16;
    constexpr int NKP = (KPC + NT - 1) / NT;
    constexpr int EPP = KV8 ? 16 : 8;            // elements per piece

    const int nqt = (a.P + PQ - 1) / PQ;
    const int qt = nqt - 1 - (int)blockIdx.x;     // heaviest (latest) query tiles first
    const int h = blockIdx.y, b = blockIdx.z;
    const int kvh = (h * a.nkv) / a.nh;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int l32 = lane & 31, h32 = lane >> 5;
    const int p0 = qt * PQ;
    const int qpos = p0 + 32 * w + l32;           // this lane's query column
    const bool qvalid = qpos < a.P;
    const int wfirst = p0 + 32 * w;               // first and last query of this wave
    const int wlast = min(a.P - 1, wfirst + 31);
    const float sl2 = a.scale * 1.4426950408889634f;   // scores in the base-2 domain

    // Q^T fragments for the D/16 MFMA k-steps: lane l supplies query l % 32, dims
    // 16 s + 8 (l / 32) .. + 7
    u32x4 qf[D / 16];
    {
        const float* qrow = a.q + ((int64_t)b * a.P + (qvalid ? qpos : 0)) * a.nh * D + h * D;
#pragma unroll
        for (int j = 0; j < D / 16; ++j) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (qvalid) {
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

    f32x16 oacc[D / 32];                          // O^T: dim 32 dt + 8 (e / 4) + 4 (l / 32) + e % 4
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt) oacc[dt] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.kv_stride; // key row of position 0
    const int64_t vblk0 = ((int64_t)b * a.nkv + kvh) * a.nblk;      // value block of position 0
    const int kend = min(a.P, p0 + PQ);
    const int ntiles = (kend + PKT - 1) / PKT;

    // ---- staging of key tile kt: global -> registers.  K piece c: key c / (D / EPP);
    // V piece c: dim (c / (VPD)) % D of block c / (VPD * D), VPD pieces per dim and block
    constexpr int VPD = 32 / EPP;
    struct Stage {
        u32x4 k[NKP], v[NKP];
        uint16_t sc;
    };
    auto load = [&](int kt, Stage& sg) {
#pragma unroll
        for (int i = 0; i < NKP; ++i) {
            const int c = tid + NT * i;
            sg.k[i] = u32x4{0u, 0u, 0u, 0u};
            sg.v[i] = u32x4{0u, 0u, 0u, 0u};
            if (c < KPC) {
                const int key = c / (D / EPP), dc = (c % (D / EPP)) * EPP;
                const int kpos = kt * PKT + key;
                if (kpos < a.P) sg.k[i] = *(const u32x4*)((const char*)a.kc + ((crow0 + kpos) * D + dc) * (KV8 ? 1 : 2));
                const int q = c % VPD, dd = (c / VPD) % D, blk = c / (VPD * D);
                const int gb = 2 * kt + blk;
                if (gb < a.nblk)
                    sg.v[i] = *(const u32x4*)((const char*)a.vc + (((vblk0 + gb) * D + dd) * VT_BLK + EPP * q) * (KV8 ? 1 : 2));
            }
        }
        if constexpr (KV8) {
            sg.sc = 0;
            if (tid < 2 * PKT) {
                const int kpos = kt * PKT + (tid & (PKT - 1));
                if (kpos < a.P) sg.sc = tid < PKT ? a.k_scales[crow0 + kpos] : a.v_scales[crow0 + kpos];
            }
        }
    };
    // ---- registers -> LDS buffer st (int8 codes become exact fp16 values)
    auto store = [&](int st, const Stage& sg) {
#pragma unroll
        for (int i = 0; i < NKP; ++i) {
            const int c = tid + NT * i;
            if (c < KPC) {
                const int key = c / (D / EPP), dc = (c % (D / EPP)) * EPP;
                const int q = c % VPD, dd = (c / VPD) % D, blk = c / (VPD * D);
                uint16_t* kd = &Ks[st][key * KP + dc];
                uint16_t* vd = &Vt[st][dd * VP + 32 * blk + EPP * q];
                if constexpr (KV8) {
                    const u32x2 k0 = i8x4_to_f16x4(sg.k[i].x), k1 = i8x4_to_f16x4(sg.k[i].y);
                    const u32x2 k2 = i8x4_to_f16x4(sg.k[i].z), k3 = i8x4_to_f16x4(sg.k[i].w);
                    *(u32x4*)(kd) = u32x4{k0.x, k0.y, k1.x, k1.y};
                    *(u32x4*)(kd + 8) = u32x4{k2.x, k2.y, k3.x, k3.y};
                    const u32x2 v0 = i8x4_to_f16x4(sg.v[i].x), v1 = i8x4_to_f16x4(sg.v[i].y);
                    const u32x2 v2 = i8x4_to_f16x4(sg.v[i].z), v3 = i8x4_to_f16x4(sg.v[i].w);
                    *(u32x4*)(vd) = u32x4{v0.x, v0.y, v1.x, v1.y};
                    *(u32x4*)(vd + 8) = u32x4{v2.x, v2.y, v3.x, v3.y};
                } else {
                    *(u32x4*)(kd) = sg.k[i];
                    *(u32x4*)(vd) = sg.v[i];
                }
            }
        }
        if constexpr (KV8) {
            if (tid < 2 * PKT) {
                if (tid < PKT) ksc[st][tid] = h2f(sg.sc) * sl2;
                else vsc[st][tid - PKT] = h2f(sg.sc);
            }
        }
    };

    auto compute = [&](int kt, int st, bool masked) {
        // ---- S^T = K Q^T for the two 32-key subtiles (base-2 domain)
        f32x16 sc[2];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
            f32x16 acc = f32x16{};
#pragma unroll
            for (int j = 0; j < D / 16; ++j) {
                const u32x4 ka = *(const u32x4*)(&Ks[st][(32 * kk + l32) * KP + 16 * j + 8 * h32]);
                acc = mfma32<AF>(ka, qf[j], acc);
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int key = 32 * kk + 8 * (e >> 2) + 4 * h32 + (e & 3);
                float v;
                if constexpr (KV8) v = acc[e] * ksc[st][key];
                else v = acc[e] * sl2;
                if (masked) {
                    const int kpos = kt * PKT + key;
                    v = (kpos <= qpos && kpos < a.P) ? v : -INFINITY;
                }
                acc[e] = v;
            }
            sc[kk] = acc;
        }
        // ---- online softmax for this lane's query column (the other 32 keys of the tile
        // are in lane l ^ 32)
        float tmax = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, sc[kk][e]);
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float m_new = fmaxf(m_run, tmax);
        const float alpha = exp2f(m_run - m_new);
        float psum = 0.f;
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float p = exp2f(sc[kk][e] - m_new);
                sc[kk][e] = p;
                psum += p;
            }
        psum += __shfl_xor(psum, 32, 64);
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) oacc[dt] *= alpha;

        // ---- O^T += V^T P^T, two 16-key steps per subtile
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                float pv[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[i] = sc[kk][4 * j + i];
                    pv[4 + i] = sc[kk][4 * j + 8 + i];
                }
                if constexpr (KV8) {
#pragma unroll
                    for (int i = 0; i < 8; ++i)
                        pv[i] *= vsc[st][32 * kk + 8 * (j + 2 * (i >> 2)) + 4 * h32 + (i & 3)];
                }
                u32x4 pfrag;
                if constexpr (KV8)
                    pfrag = u32x4{pack_f16_hw(pv[0], pv[1]), pack_f16_hw(pv[2], pv[3]), pack_f16_hw(pv[4], pv[5]),
                                  pack_f16_hw(pv[6], pv[7])};
                else
                    pfrag = u32x4{pack_bf16_hw(pv[0], pv[1]), pack_bf16_hw(pv[2], pv[3]), pack_bf16_hw(pv[4], pv[5]),
                                  pack_bf16_hw(pv[6], pv[7])};
#pragma unroll
                for (int dt = 0; dt < D / 32; ++dt) {
                    const u32x4 vf = *(const u32x4*)(&Vt[st][(32 * dt + l32) * VP + 32 * kk + 16 * j + 8 * h32]);
                    oacc[dt] = mfma32<AF>(vf, pfrag, oacc[dt]);
                }
            }
    };
    auto barrier = [&]() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); };

    Stage sg;
    load(0, sg);
    store(0, sg);
    if (ntiles > 1) load(1, sg);
    barrier();
    for (int kt = 0; kt < ntiles; ++kt) {
        if (kt * PKT <= wlast) {                  // tiles past the wave's queries: nothing
            if ((kt + 1) * PKT - 1 > wfirst || (kt + 1) * PKT > a.P) compute(kt, kt & 1, true);
            else compute(kt, kt & 1, false);
        }
        if (kt + 1 < ntiles) store((kt + 1) & 1, sg);
        if (kt + 2 < ntiles) load(kt + 2, sg);
        barrier();
    }

    if (!qvalid) return;
    const float inv = 1.0f / l_run;
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

template <int D, bool KV8>
static void launch_ap(const AttnPreArgs& a, int B, hipStream_t st) {
    // 8 waves (256 queries) per workgroup when that still gives every CU a workgroup;
    // 4 waves otherwise (2-wave workgroups measured slower still)
    if ((int64_t)((a.P + 255) / 256) * a.nh * B >= 256)
        FP_LAUNCH((attn_prefill_kernel<D, KV8, 8>), dim3((a.P + 255) / 256, a.nh, B), dim3(512), 0, st, a);
    else
        FP_LAUNCH((attn_prefill_kernel<D, KV8, 4>), dim3((a.P + 127) / 128, a.nh, B), dim3(256), 0, st, a);
}

hipError_t launch_attn_prefill(const AttnPreArgs& a, int B, hipStream_t st) {
    if (a.d == 128) {
        if (a.kv_int8) launch_ap<128, true>(a, B, st);
        else launch_ap<128, false>(a, B, st);
    } else if (a.d == 64) {
        if (a.kv_int8) launch_ap<64, true>(a, B, st);
        else launch_ap<64, false>(a, B, st);
    } else {
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace fpk
