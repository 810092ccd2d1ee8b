// Prefill attention: causal attention of a whole prompt, reading K / V back from
// the cache the rotary/append kernel has just written (bf16, or int8 codes with
// per-(position, kv head) scales -- the INT8 KV cache of paper Sec. 3.2), so
// that prefill sees exactly what later decode steps see.
//
// Flash-style on bf16 MFMA 16x16x32, written in the transposed form
//     S^T = K Q^T          (A = key rows from LDS, B = the wave's 16 queries)
//     O^T += V^T P^T       (A = value columns, B = the probabilities already in
//                           the lanes)
// so the probabilities never leave registers: after S^T, lane (q, g) holds the
// scores of keys 16t + 4g + i for its query column q, which are exactly the 8
// k-values it must supply as B for a 32-key MFMA step (subtiles t, t+1).  The
// value cache is stored transposed in 32-position blocks whose slots follow that
// order (vt_slot), so the value tile is copied into LDS as it is and each A
// fragment is one contiguous 16-byte LDS read.
// Online softmax per query column (max / sum across the 4 lane groups by
// shuffles).  int8 caches: codes are exact in bf16; s_k scales the scores and
// s_v the probabilities.  Workgroup = 4 waves x 16 queries of one head; key
// tiles of 64; heaviest (latest) query tiles are launched first.
#include "fp_device.h"
#include "fp_internal.h"

namespace fpk {

template <int D>
__global__ void __launch_bounds__(256) attn_prefill_kernel(AttnPreArgs a) {
    constexpr int KT = 64;
    constexpr int KP = D + 8;     // padded row of the key tile (u16)
    constexpr int VP = KT + 8;    // padded row of the transposed value tile (u16)
    __shared__ __attribute__((aligned(16))) uint16_t Ks[KT * KP];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VP];
    __shared__ float ksc[KT], vsc[KT];

    const int nqt = (a.P + 63) / 64;
    const int qt = nqt - 1 - (int)blockIdx.x;
    const int h = blockIdx.y, b = blockIdx.z;
    const int kvh = (h * a.nkv) / a.nh;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int p0 = qt * 64;
    const int qpos = p0 + 16 * w + r;           // this lane's query column
    const bool qvalid = qpos < a.P;

    // Q^T fragments (bf16) for the D/32 MFMA k-steps
    u32x4 qf[D / 32];
    {
        const float* qrow = a.q + ((int64_t)b * a.P + (qvalid ? qpos : 0)) * a.nh * D + h * D;
#pragma unroll
        for (int j = 0; j < D / 32; ++j) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (qvalid) {
                const float4 x0 = *(const float4*)(qrow + 32 * j + 8 * g);
                const float4 x1 = *(const float4*)(qrow + 32 * j + 8 * g + 4);
                v[0] = (uint32_t)f2bf(x0.x) | ((uint32_t)f2bf(x0.y) << 16);
                v[1] = (uint32_t)f2bf(x0.z) | ((uint32_t)f2bf(x0.w) << 16);
                v[2] = (uint32_t)f2bf(x1.x) | ((uint32_t)f2bf(x1.y) << 16);
                v[3] = (uint32_t)f2bf(x1.z) | ((uint32_t)f2bf(x1.w) << 16);
            }
            qf[j] = u32x4{v[0], v[1], v[2], v[3]};
        }
    }

    f32x4 oacc[D / 16];
#pragma unroll
    for (int dd = 0; dd < D / 16; ++dd) oacc[dd] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -INFINITY, l_run = 0.f;

    const int64_t crow0 = ((int64_t)b * a.nkv + kvh) * a.kv_stride; // key row of position 0
    const int64_t vblk0 = ((int64_t)b * a.nkv + kvh) * a.nblk;      // value block of position 0
    const int kend = min(a.P, p0 + 64);
    const int ntiles = (kend + KT - 1) / KT;
    for (int kt = 0; kt < ntiles; ++kt) {
        __syncthreads();
        // ---- stage the K tile (row-major) and the two value blocks of the tile, bf16
        if (a.kv_int8) {
            constexpr int CPR = D / 16;            // 16-code chunks per key row
            for (int c = tid; c < KT * CPR; c += 256) {
                const int key = c / CPR, dc = (c % CPR) * 16;
                const int kpos = kt * KT + key;
                u32x4 kr = u32x4{0u, 0u, 0u, 0u};
                if (kpos < a.P) kr = *(const u32x4*)((const int8_t*)a.kc + (crow0 + kpos) * D + dc);
                const uint32_t kw[4] = {kr.x, kr.y, kr.z, kr.w};
                uint32_t o[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {     // codes are exact in bf16
                    const float f0 = (float)(int8_t)((kw[e >> 1] >> (16 * (e & 1))) & 0xFF);
                    const float f1 = (float)(int8_t)((kw[e >> 1] >> (16 * (e & 1) + 8)) & 0xFF);
                    o[e] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xFFFF0000u);
                }
                *(u32x4*)(Ks + key * KP + dc) = u32x4{o[0], o[1], o[2], o[3]};
                *(u32x4*)(Ks + key * KP + dc + 8) = u32x4{o[4], o[5], o[6], o[7]};
            }
            for (int c = tid; c < 2 * D * 2; c += 256) {   // 2 blocks x D dims x 2 chunks of 16 codes
                const int half = c & 1, dd = (c >> 1) % D, blk = c / (2 * D);
                const int gb = 2 * kt + blk;
                u32x4 vr = u32x4{0u, 0u, 0u, 0u};
                if (gb < a.nblk) vr = *(const u32x4*)((const int8_t*)a.vc + ((vblk0 + gb) * D + dd) * VT_BLK + 16 * half);
                const uint32_t vw[4] = {vr.x, vr.y, vr.z, vr.w};
                uint32_t o[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float f0 = (float)(int8_t)((vw[e >> 1] >> (16 * (e & 1))) & 0xFF);
                    const float f1 = (float)(int8_t)((vw[e >> 1] >> (16 * (e & 1) + 8)) & 0xFF);
                    o[e] = (__float_as_uint(f0) >> 16) | (__float_as_uint(f1) & 0xFFFF0000u);
                }
                uint16_t* dst = Vt + dd * VP + 32 * blk + 16 * half;
                *(u32x4*)(dst) = u32x4{o[0], o[1], o[2], o[3]};
                *(u32x4*)(dst + 8) = u32x4{o[4], o[5], o[6], o[7]};
            }
            if (tid < KT) {
                const int kpos = kt * KT + tid;
                ksc[tid] = kpos < a.P ? h2f(a.k_scales[crow0 + kpos]) : 0.f;
                vsc[tid] = kpos < a.P ? h2f(a.v_scales[crow0 + kpos]) : 0.f;
            }
        } else {
            constexpr int CPR = D / 8;             // 8-value chunks per key row
            for (int c = tid; c < KT * CPR; c += 256) {
                const int key = c / CPR, dc = (c % CPR) * 8;
                const int kpos = kt * KT + key;
                u32x4 kr = u32x4{0u, 0u, 0u, 0u};
                if (kpos < a.P) kr = *(const u32x4*)((const uint16_t*)a.kc + (crow0 + kpos) * D + dc);
                *(u32x4*)(Ks + key * KP + dc) = kr;
            }
            for (int c = tid; c < 2 * D * 4; c += 256) {   // 2 blocks x D dims x 4 chunks of 8 values
                const int q4 = c & 3, dd = (c >> 2) % D, blk = c / (4 * D);
                const int gb = 2 * kt + blk;
                u32x4 vr = u32x4{0u, 0u, 0u, 0u};
                if (gb < a.nblk) vr = *(const u32x4*)((const uint16_t*)a.vc + ((vblk0 + gb) * D + dd) * VT_BLK + 8 * q4);
                *(u32x4*)(Vt + dd * VP + 32 * blk + 8 * q4) = vr;
            }
        }
        __syncthreads();

        // ---- S^T = K Q^T for the 4 key subtiles
        float s[4][4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < D / 32; ++j) {
                const u32x4 ka = *(const u32x4*)(Ks + (16 * kk + r) * KP + 32 * j + 8 * g);
                acc = mfma_bf16(ka, qf[j], acc);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = 16 * kk + 4 * g + i;
                const int kpos = kt * KT + key;
                float v = acc[i] * a.scale;
                if (a.kv_int8) v *= ksc[key];
                s[kk][i] = (kpos <= qpos && kpos < a.P) ? v : -INFINITY;
            }
        }
        // ---- online softmax for this lane's query column
        float tmax = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i) tmax = fmaxf(tmax, s[kk][i]);
        tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
        const float m_new = fmaxf(m_run, tmax);
        const float alpha = __expf(m_run - m_new);
        float psum = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float p = __expf(s[kk][i] - m_new);
                s[kk][i] = p;
                psum += p;
            }
        psum += __shfl_xor(psum, 16, 64);
        psum += __shfl_xor(psum, 32, 64);
        l_run = l_run * alpha + psum;
        m_run = m_new;
#pragma unroll
        for (int dd = 0; dd < D / 16; ++dd) oacc[dd] *= alpha;

        // ---- O^T += V^T P^T, two 32-key steps
#pragma unroll
        for (int k2 = 0; k2 < 2; ++k2) {
            uint32_t pb[4];
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int kk = 2 * k2 + half;
                float pv[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pv[i] = s[kk][i];
                    if (a.kv_int8) pv[i] *= vsc[16 * kk + 4 * g + i];
                }
                pb[2 * half] = (uint32_t)f2bf(pv[0]) | ((uint32_t)f2bf(pv[1]) << 16);
                pb[2 * half + 1] = (uint32_t)f2bf(pv[2]) | ((uint32_t)f2bf(pv[3]) << 16);
            }
            const u32x4 pfrag = u32x4{pb[0], pb[1], pb[2], pb[3]};
#pragma unroll
            for (int dd = 0; dd < D / 16; ++dd) {
                const u32x4 vf = *(const u32x4*)(Vt + (16 * dd + r) * VP + 32 * k2 + 8 * g);
                oacc[dd] = mfma_bf16(vf, pfrag, oacc[dd]);
            }
        }
    }

    if (!qvalid) return;
    const float inv = 1.0f / l_run;
    uint16_t* orow = a.out + ((int64_t)b * a.P + qpos) * a.nh * D + h * D;
#pragma unroll
    for (int dd = 0; dd < D / 16; ++dd) {
        uint16_t v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = act_store(bfround(oacc[dd][i] * inv), a.out_fmt);
        *(u32x2*)(orow + 16 * dd + 4 * g) =
            u32x2{(uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16)};
    }
}

hipError_t launch_attn_prefill(const AttnPreArgs& a, int B, hipStream_t st) {
    const int nqt = (a.P + 63) / 64;
    dim3 grid(nqt, a.nh, B);
    if (a.d == 128) FP_LAUNCH(attn_prefill_kernel<128>, grid, dim3(256), 0, st, a);
    else if (a.d == 64) FP_LAUNCH(attn_prefill_kernel<64>, grid, dim3(256), 0, st, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace fpk
