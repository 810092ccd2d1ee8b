// Internal interface between the host runtime (fp_host.cpp) and the kernels.
#pragma once
#include "fp.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fpk {

// Per-kernel timing of a profiled step.  While a timer is armed on the calling thread,
// each launch stamps the stop event with its own end of execution, and the first launch
// after arming stamps the start event with its own start (hipExtLaunchKernel takes both
// from the dispatch itself), so an interval covers kernel execution only, not the
// queue gaps around it.
struct LaunchTimer {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
extern thread_local LaunchTimer g_launch_timer;

#define FP_LAUNCH(kern, grid, block, shmem, st, ...)                                           \
    do {                                                                                       \
        if (::fpk::g_launch_timer.stop) {                                                      \
            hipExtLaunchKernelGGL(kern, grid, block, shmem, st, ::fpk::g_launch_timer.start,   \
                                  ::fpk::g_launch_timer.stop, 0, __VA_ARGS__);                 \
            ::fpk::g_launch_timer.start = nullptr;                                             \
        } else {                                                                               \
            hipLaunchKernelGGL(kern, grid, block, shmem, st, __VA_ARGS__);                     \
        }                                                                                      \
    } while (0)

enum WFmt { W_BF16 = 0, W_INT8 = 1, W_INT4 = 2, W_SP24 = 3 };
// EPI_PART: fp32 partial sums of one k-split, [ks, M, N] (or [ks, M, 2F] for the
// [gate; up] matrix), multiplied by the int8 row scales; a reduction kernel finishes.
enum Epi { EPI_F32 = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_PART = 3 };
// Activation format of a GEMM's A operand: bf16 for bf16 weights, fp16 for quantised
// weights (the fp16 copy of a bf16-rounded value is exact in fp16's normal range).
enum ActFmt { ACT_BF16 = 0, ACT_F16 = 1 };

// Weight rows per workgroup of the decode skinny GEMM = 64 * SKINNY_NS.
#ifndef SKINNY_NS
#define SKINNY_NS 2
#endif

// How the decode skinny GEMM forms its A operand while staging it in LDS.
enum XForm {
    XF_COPY = 0,     // A = X (activation format already)
    XF_NORM = 1,     // A = act(bf16(X * r[m] * gain)), X bf16, r from ssq block sums
    XF_SWIGLU = 2,   // A = act(bf16(silu(G) * U)) from gate|up partial sums
    XF_MERGE = 3     // A = attention output merged from its context-split partials
};

// Decode skinny GEMM: part[s, m, col] = sum_{k in split s} A[m, k] W[col, k]
// (times the row scale for int8).  W rows are output columns; dual_F > 0 selects
// the SwiGLU tiling over the concatenated [gate; up] matrix of 2 * dual_F rows.
struct SkinnyArgs {
    const uint16_t* X;        // XF_COPY: act [M, K]; XF_NORM: bf16 [M, K]
    const void* W;            // fragment-major tiles (bf16 / int8 / int4 in device nibble order)
    const uint16_t* scales;   // fp16: int8 [N]; int4 [N, K/128]
    const uint16_t* zeros;    // fp16 [N, K/128] (int4)
    const uint32_t* sz;       // int4: scale | zero << 16 per (row, group), group-major [K/128, N]
    int M, N, K;
    int kst;                  // K-steps per 16-row block row of W (ceil(K / KS))
    int dual_F;
    int krange;               // k per split (multiple of the format's K-step)
    float* part;              // [ks, M, N] fp32
    int xf;                   // XForm
    const uint16_t* gain;     // XF_NORM: bf16 [K]
    const float* ssq;         // XF_NORM: [M, ssq_blocks] sums of squares of X rows; NULL: the
                              // workgroup sums the squares of its rows itself
    int ssq_blocks;
    float eps;
    const float* src_part;    // XF_SWIGLU: [src_ks, M, 2K] gate|up partial sums
    int src_ks;
    const float* att_ws;      // XF_MERGE: [M, K / head_dim, att_nsplit, head_dim + 4]
    int att_nsplit, att_kps, head_dim;
    const int* d_pos;         // XF_MERGE: position of the newest token
};

struct GemmArgs {
    const uint16_t* X;        // activations [M, K]
    const void* W;            // fragment-major tiles
    const uint16_t* scales;
    const uint16_t* zeros;
    const uint32_t* sz;       // int4: scale | zero << 16 per (row, group), group-major [K/128, N]
    int M, N, K, F;           // F: SwiGLU width (N = 2F rows of [gate; up])
    int kst;                  // K-steps per 16-row block row of W
    float* out32;             // EPI_F32: [M, N]
    uint16_t* out16;          // EPI_RESID: bf16 [M, N]; EPI_SWIGLU: act [M, F]
    const uint16_t* resid;    // EPI_RESID: bf16 [M, N]
    int out_fmt;              // EPI_SWIGLU activation format
    int krange;               // EPI_PART: k per split (multiple of the large tiling's k per stage)
    int tiles_m, tiles_n;     // set by the launcher
};

// Value cache layout: blocks of VT_BLK positions per (sequence, kv head), each stored
// transposed as [head_dim][VT_BLK]; inside a block, position kb sits in slot
// vt_slot(kb), the order in which the decode and prefill attention kernels supply
// probabilities as the B operand of a 32-key MFMA step (lane group g holds keys
// 4g..4g+3 and 16+4g..16+4g+3).  Key cache: [B, nkv, max_seq, head_dim] row-major.
constexpr int VT_BLK = 32;
__host__ __device__ inline int vt_slot(int kb) { return 8 * ((kb & 15) >> 2) + 4 * (kb >> 4) + (kb & 3); }
inline int vt_blocks(int max_seq) { return (max_seq + VT_BLK - 1) / VT_BLK; }
// Rows of the key cache (and of the int8 scales) per (sequence, kv head): max_seq
// rounded up to whole VT_BLK blocks, so every 32-key chunk of a context can be loaded
// without a bounds test (rows past the current length are masked, never used).
inline int kv_row_stride(int max_seq) { return vt_blocks(max_seq) * VT_BLK; }

struct RopeKvArgs {
    const float* part;        // [ks, M, Nqkv]
    int ks, M, T, nh, nkv, d;
    const int* d_pos;         // NULL -> positions start at 0
    const float* cos_t;
    const float* sin_t;
    int max_seq, nblk;        // nblk: value blocks per (sequence, kv head)
    int kv_stride;            // key / scale rows per (sequence, kv head)
    uint16_t* qout;           // [M / T, nh, T, d] rotated queries: fp16 with an int8 cache, else bf16
    void* kc;
    void* vc;
    uint16_t* ks_out;
    uint16_t* vs_out;
    int kv_int8;
    float* dump;              // NULL or [2, M, nkv, d]
};

struct AttnDecArgs {
    // q|k|v of the new tokens as split-K partial sums [ks, B, (nh + 2 nkv) d], before the
    // rotary embedding; the kernel rotates q and k and appends k, v to the cache
    const float* qkv_part;
    int ks;
    const float* cos_t;       // [max_seq, d/2]
    const float* sin_t;
    float* dump;              // NULL or [2, B, nkv, d] pre-quantisation K, V
    void* kc;                 // layer cache [B, nkv, max_seq, d]
    void* vc;
    uint16_t* k_scales;       // [B, nkv, max_seq] (int8)
    uint16_t* v_scales;
    int kv_int8, nh, nkv, d, max_seq, nblk;
    int kv_stride;            // key / scale rows per (sequence, kv head)
    const int* d_pos;         // current position (the new token's index)
    float scale;              // float32(1/sqrt(d))
    int keys_per_split;       // context keys per split (multiple of VT_BLK)
    int batch;                // B
    int skip_merge;           // leave split partials in ws (the consumer merges them)
    float* ws;                // [B, nh, nsw, d + 4] workgroup partials when nsw > 1 (m at d, l at d + 1)
    uint16_t* out;            // [B, nh*d] activation format out_fmt
    int out_fmt;
};

struct AttnPreArgs {
    const uint16_t* q;        // [B, nh, P, d] rotated queries: fp16 with an int8 cache, else bf16
    const void* kc;
    const void* vc;
    const uint16_t* k_scales;
    const uint16_t* v_scales;
    void* staged;             // int8: the prompt's blocks dequantised by attn_stage_kernel
    int kv_int8, P, nh, nkv, d, max_seq, nblk;
    int kv_stride;            // key / scale rows per (sequence, kv head)
    float scale;
    float pmax;               // largest probability against the reference before a repeat
    uint16_t* out;            // [B*P, nh*d]
    int out_fmt;
};

// bytes of the int8 prompt staging buffer for B sequences of P tokens (0 for bf16 caches)
size_t attn_stage_bytes(int B, int P, int nkv, int d);
hipError_t launch_attn_stage(const AttnPreArgs& a, int B, hipStream_t st);
hipError_t launch_fill_bf16(uint16_t* dst, int64_t n, uint64_t key, float mean, float sigma,
                            hipStream_t st);
// Fragment-major weight layout (see tile_kernel): KS = k per 1 KiB block row-slice (2:4 sparse
// weights: 32 rows x 32 inputs per 1 KiB block, see sparse.hip).
inline int weight_kstep(int wf) { return wf == W_BF16 ? 32 : (wf == W_INT8 ? 64 : (wf == W_INT4 ? 128 : 32)); }
inline int weight_ebits(int wf) { return wf == W_BF16 ? 16 : (wf == W_INT8 ? 8 : 4); }
hipError_t launch_tile(const void* src, int n, int K, int ebits, int KS, void* dst, int row0, hipStream_t st);
hipError_t launch_quant_int8(const uint16_t* w, int N, int K, int8_t* codes, uint16_t* scales,
                             hipStream_t st);
hipError_t launch_quant_int4(const uint16_t* w, int N, int K, uint32_t* codes, uint16_t* scales,
                             uint16_t* zeros, hipStream_t st);
hipError_t launch_pack_sz(const uint16_t* scales, const uint16_t* zeros, int N, int ng, uint32_t* sz,
                          hipStream_t st);

hipError_t launch_rmsnorm(const uint16_t* x, int M, int H, const uint16_t* g, float eps, uint16_t* out,
                          int out_fmt, hipStream_t st);
// Decode epilogue: out = bf16(resid + sum of ks partials) (skipped when ks == 0: the
// row is resid itself); then, if g != NULL, nout = act(bf16(row * rsqrt(mean(row^2) + eps) * g)).
// ssq: scratch of M * resid_ssq_blocks(N) floats.  inc_pos (optional): position counter
// the kernel increments once after its work.
hipError_t launch_resid_norm(const float* part, int ks, int M, int N, const uint16_t* resid,
                             uint16_t* out, const uint16_t* g, float eps, uint16_t* nout, int nfmt,
                             float* ssq, int* inc_pos, hipStream_t st);
int resid_ssq_blocks(int N);
hipError_t launch_swiglu(const float* part, int ks, int M, int F, uint16_t* a, int afmt,
                         hipStream_t st);
hipError_t launch_rope_kv(const RopeKvArgs& a, hipStream_t st);
hipError_t launch_set_pos(int* d_pos, int v, hipStream_t st);
hipError_t launch_inc_pos(int* d_pos, hipStream_t st);

int skinny_kstep(int wf);
int skinny_max_krange(int M);
int skinny_tiles(int N, int dual_F, int M);
hipError_t launch_skinny(const SkinnyArgs& a, int wf, int ks, hipStream_t st);
// Batched decode projections (XF_COPY, M <= 64): k-range walked in staged chunks of
// skinny_batch_chunk() values; krange a multiple of it, ks * krange >= K.
int skinny_batch_rows(int N, int dual_F, int wf);   // weight rows per workgroup
int skinny_batch_tiles(int N, int dual_F, int wf);
int skinny_batch_chunk();
hipError_t launch_skinny_batch(const SkinnyArgs& a, int wf, int ks, hipStream_t st);
hipError_t launch_gemm(const GemmArgs& a, int wf, int epi, hipStream_t st);
// Split-K on the large tiling for prefill GEMMs with too few 256 x 256 tiles to fill
// the GPU: the split factor (1: no split) and k per split for an [M, N] x [N, K]
// product (dual_F > 0: the [gate; up] matrix), and the launch writing EPI_PART partials.
int gemm_split_factor(int M, int N, int K, int dual_F, int wf, int* krange);
hipError_t launch_gemm_split(const GemmArgs& a, int wf, bool dual, int ks, hipStream_t st);

int attn_decode_max_splits(int max_seq);
int attn_decode_partials(int nsplit);
void attn_decode_split(int max_seq, int B, int nkv, int group, int* nsplit, int* keys_per_split);
bool attn_decode_supported(int d, int group);
hipError_t launch_attn_decode(const AttnDecArgs& a, int B, hipStream_t st);
hipError_t launch_attn_prefill(const AttnPreArgs& a, int B, hipStream_t st);

// 2:4 sparse weights (sparse.hip): values in 32-row x 32-input blocks of 1 KiB (the 64
// lanes' 16-byte operand pieces of the sparse MFMA) and 16-bit index words in 128-byte
// blocks, both block-row-major over K / 32 blocks.
struct Sp24Args {
    const uint16_t* X;        // activations bf16 [M, K]
    const uint16_t* Wv;       // value blocks
    const uint16_t* Wi;       // index blocks
    int M, N, K, F;           // F: SwiGLU width (N = 2F rows of [gate; up])
    int kst;                  // blocks per 32-row block row (K / 32)
    int krange;               // decode: k per split (multiple of 32)
    float* part;              // decode: [ks, M, N]
    float* out32;             // prefill EPI_F32: [M, N]
    uint16_t* out16;          // prefill EPI_RESID: bf16 [M, N]; EPI_SWIGLU: act [M, F]
    const uint16_t* resid;    // prefill EPI_RESID: bf16 [M, N]
    int out_fmt;
    int tiles_m, tiles_n;     // set by the launcher
};
hipError_t launch_sp24_compress(const uint16_t* w, int n, int K, uint16_t* vals, uint16_t* idx, int row0,
                                hipStream_t st);
int sp24_max_krange(int M);
hipError_t launch_sp24_gemv(const Sp24Args& a, int ks, hipStream_t st);
hipError_t launch_gemm_sp24(const Sp24Args& a, int epi, hipStream_t st);

// The blocks outside the hidden layers (head.hip).
hipError_t launch_embed(const int* ids, int64_t M, const uint16_t* E, int V, int H, uint16_t* x, hipStream_t st);
hipError_t launch_head_norm(const uint16_t* y, int B, int T, int H, const uint16_t* g, float eps, uint16_t* out,
                            hipStream_t st);
int head_logit_blocks(int V);
hipError_t launch_logits_argmax(const float* part, int ks, int B, int V, float* logits, float* bval, int* bidx,
                                int* out_ids, hipStream_t st);

// Host runtime hooks for the allocation-free decode step (noalloc.hip): one eager decode
// step whose scratch buffers live in [scratch, scratch + bytes), and setting the
// thread's last-error message.
fp_status decode_step_scratch(fp_layer* h, const void* x, void* y, hipStream_t st, void* scratch, size_t bytes);
fp_status report_error(fp_status s, const char* msg);
bool layer_unbacked(const fp_layer* h);

}  // namespace fpk
