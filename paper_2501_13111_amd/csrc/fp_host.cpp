// Host runtime of the fingerprint forward pass: handle, validation, allocation,
// weight synthesis, the prefill / decode schedules, graph replay of decode steps,
// export and error reporting.  See include/fp.h for the contract of each call.
//
// Dataflow of one hidden layer (the paper names the components -- attention,
// normalisation, activation -- Sec. 5.1; their Llama-style math is the reading):
//   prefill, M = B*P tokens:
//     rmsnorm(x) -> gemm[qkv] -> rope + KV append -> causal attention over the
//     cache -> gemm[o] + residual -> rmsnorm -> gemm[gate|up] + SwiGLU ->
//     gemm[down] + residual
//   decode, M = B tokens at position pos:
//     skinny[qkv] -> rope + KV append at pos -> split-context attention + merge
//     -> skinny[o] -> residual + next rmsnorm -> skinny[gate|up] -> SwiGLU ->
//     skinny[down] -> residual + next layer's rmsnorm
// All weights of a layer live in three fused matrices: [q; k; v], o, [gate; up],
// down, each [N, K] row-major (out x in).
#include "fp.h"
#include "fp_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <tuple>
#include <string>
#include <utility>
#include <vector>

using namespace fpk;

thread_local LaunchTimer fpk::g_launch_timer;

namespace {

// Prefill attention takes probabilities against a fixed reference per query and repeats a
// prompt once if one would pass this limit (2^64).  FP_ATTN_PROB_LIMIT_LOG2 (1 .. 64)
// lowers it, so that tests can drive the repeat on ordinary inputs.
float attn_prob_limit() {
    const char* e = std::getenv("FP_ATTN_PROB_LIMIT_LOG2");
    int v = e ? std::atoi(e) : 64;
    v = v < 1 ? 1 : v > 64 ? 64 : v;
    return std::ldexp(1.0f, v);
}


thread_local std::string g_err;

fp_status fail(fp_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

#define HIPCHK(expr)                                                                       \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail(FP_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
    } while (0)

constexpr uint64_t GAMMA = 0x9E3779B97F4A7C15ull;
uint64_t mix64(uint64_t z) {
    z ^= z >> 30; z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27; z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}
uint64_t stream_key(uint64_t seed, int32_t layer, int32_t tensor) {
    const uint64_t id = ((uint64_t)(int64_t)(layer + 1) << 8) | (uint64_t)(uint32_t)tensor;
    return mix64(mix64(seed) + GAMMA * id);
}

constexpr int KSMAX = 64;         // max split-K factor of the decode projections
#ifndef FP_TARGET_WG
#define FP_TARGET_WG 512
#endif
constexpr int TARGET_WG = FP_TARGET_WG;   // decode workgroups per projection the split-K aims for
#ifndef SPLIT_WIDE_N
#define SPLIT_WIDE_N 8192
#endif

struct Mat {
    int wf = 0;                   // weight format (W_BF16 / W_INT8 / W_INT4)
    void* codes = nullptr;        // fragment-major tiles of bf16 / int8 / int4 (device nibble order)
    uint16_t* scales = nullptr;
    uint16_t* zeros = nullptr;
    uint32_t* sz = nullptr;       // int4: scale | zero << 16 per (row, group)
    uint16_t* sidx = nullptr;     // 2:4 sparse: 16-bit index words, 128-byte blocks (codes: value blocks)
    int N = 0, K = 0;
    int kst = 0;                  // K-steps (1 KiB blocks) per 16-row block row
};

struct LayerW {
    uint16_t* attn_norm = nullptr;
    uint16_t* mlp_norm = nullptr;
    Mat qkv, o, gu, down;
};

// Kernel-timed intervals of a profiled step: mark() opens an interval of the given kind,
// and the launches enqueued until the next mark() or end() stamp its start / stop
// events from their own dispatches (FP_LAUNCH).
struct Prof {
    std::vector<hipEvent_t> t0, t1;
    std::vector<int> kind, layer;
    hipStream_t st = nullptr;
    bool on = false;
    void mark(int k, int l) {
        if (!on) return;
        hipEvent_t a = nullptr, b = nullptr;
        if (hipEventCreate(&a) != hipSuccess) return;
        if (hipEventCreate(&b) != hipSuccess) {
            (void)hipEventDestroy(a);
            return;
        }
        t0.push_back(a);
        t1.push_back(b);
        kind.push_back(k);
        layer.push_back(l);
        g_launch_timer.start = a;
        g_launch_timer.stop = b;
    }
    void end() { g_launch_timer = LaunchTimer{}; }
    void clear() {
        for (auto e : t0) (void)hipEventDestroy(e);
        for (auto e : t1) (void)hipEventDestroy(e);
        t0.clear();
        t1.clear();
        kind.clear();
        layer.clear();
        on = false;
        g_launch_timer = LaunchTimer{};
    }
};

}  // namespace

struct fp_layer {
    fp_shape s{};
    int wq = 0, kvq = 0;
    uint64_t seed = 0;
    bool unbacked = false;
    int act_fmt = ACT_BF16;
    int q_dim = 0, kv_dim = 0, nqkv = 0;
    std::vector<LayerW> L;
    std::vector<void*> kc, vc;
    std::vector<uint16_t*> ksc, vsc;
    float* cos_t = nullptr;
    float* sin_t = nullptr;
    // workspace
    uint16_t* act_in = nullptr;   // normalised inputs of qkv / gate|up  [Mmax, H]
    uint16_t* act_o = nullptr;    // attention output                     [Mmax, q_dim]
    uint16_t* act_f = nullptr;    // SwiGLU output                        [Mmax, F]
    uint16_t* hbuf = nullptr;     // h = x + attention projection         [Mmax, H]
    uint16_t* xbuf = nullptr;     // inter-layer hidden state              [Mmax, H]
    float* qkv32 = nullptr;       // prefill q|k|v before rotary          [Mmax, Nqkv]
    uint16_t* q16 = nullptr;      // rotated queries (fp16 / bf16)        [Mmax, q_dim]
    void* stage = nullptr;        // int8 caches: the prompt's K / V blocks dequantised for
                                  // prefill attention (act_f when that is large enough: it is
                                  // idle between the rotary step and the gate/up projection)
    float* part = nullptr;        // decode split-K partials              [KSMAX, Bmax, Ncol]
    float* part2 = nullptr;       // gate|up partials (read while down writes part)
    float* ppart = nullptr;       // prefill split-K partials (GEMMs with too few large tiles)
    float* attn_ws = nullptr;     // decode attention partials
    float* ssq = nullptr;         // decode row-norm block sums         [Bmax, nblk]
    int* d_pos = nullptr;
    // blocks outside the hidden layers (vocab > 0)
    uint16_t* embed = nullptr;    // token embedding, bf16 [vocab, H] row-major
    uint16_t* final_norm = nullptr;
    Mat lm;                       // LM head, bf16 [vocab, H] fragment-major
    float* hpart = nullptr;       // LM head split-K partials            [ks, Bmax, vocab]
    float* hbval = nullptr;       // best logit per 2048-logit block     [Bmax, nblk]
    int* hbidx = nullptr;
    uint16_t* hnorm = nullptr;    // final-normalised rows (batches)     [Bmax, H]
    uint16_t* tok_x = nullptr;    // embedded tokens of a request        [Mmax, H]
    uint16_t* tok_y = nullptr;    // layer-stack output of a request     [Mmax, H]
    // state
    int pos = 0, B = 0;
    bool prefilled = false;
    bool use_graph = true;
    float* dump = nullptr;
    uint16_t* ldump = nullptr;      // per-layer outputs [n_layers, B, T, hidden] (debug)
    hipStream_t cap_stream = nullptr;
    // Captured decode graphs.  A capture bakes in the buffers and everything that depends
    // on the active batch (grids, split factors, the single-sequence or batch schedule,
    // the rows written), so both caches are keyed by the batch too, and a prefill that
    // changes the batch drops them.  At most GRAPH_CACHE_MAX entries each.
    std::map<std::tuple<const void*, void*, int>, hipGraphExec_t> graphs;     // (x, y, B)
    std::map<std::tuple<void*, void*, int, int>, hipGraphExec_t> mgraphs;     // (x, y, n, B)
    // fp_generate's decode loop: (out_ids, logits, force_ids, n_out, B)
    std::map<std::tuple<int32_t*, float*, const int32_t*, int, int>, hipGraphExec_t> ggraphs;
    Prof prof;
    size_t bytes_w = 0, bytes_kv = 0, bytes_ws = 0;
    std::vector<void*> allocs;
};

namespace {

fp_status dev_alloc(fp_layer* h, void** p, size_t bytes, size_t* counter) {
    if (bytes == 0) bytes = 256;
    if (h->unbacked) {               // validation-only handle: count the bytes, allocate nothing
        *p = nullptr;
        *counter += bytes;
        return FP_OK;
    }
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        return fail(e == hipErrorOutOfMemory ? FP_ERR_OOM : FP_ERR_HIP, "hipMalloc(%zu) failed: %s",
                    bytes, hipGetErrorString(e));
    }
    h->allocs.push_back(*p);
    *counter += bytes;
    return FP_OK;
}

template <typename T>
fp_status alloc_t(fp_layer* h, T** p, size_t count, size_t* counter) {
    void* v = nullptr;
    fp_status st = dev_alloc(h, &v, count * sizeof(T), counter);
    *p = (T*)v;
    return st;
}

constexpr size_t GRAPH_CACHE_MAX = 16;

// Destroy every captured decode graph.  A replay may still be in flight on some stream,
// so the device is synchronised first (only when there is something to destroy).
void drop_graphs(fp_layer* h) {
    if (h->graphs.empty() && h->mgraphs.empty() && h->ggraphs.empty()) return;
    (void)hipDeviceSynchronize();
    for (auto& kv : h->graphs) (void)hipGraphExecDestroy(kv.second);
    h->graphs.clear();
    for (auto& kv : h->mgraphs) (void)hipGraphExecDestroy(kv.second);
    h->mgraphs.clear();
    for (auto& kv : h->ggraphs) (void)hipGraphExecDestroy(kv.second);
    h->ggraphs.clear();
}

void free_all(fp_layer* h) {
    drop_graphs(h);
    if (h->cap_stream) (void)hipStreamDestroy(h->cap_stream);
    h->cap_stream = nullptr;
    for (void* p : h->allocs) (void)hipFree(p);
    h->allocs.clear();
}

fp_status validate_shape(const fp_shape* s, int wq, int kvq) {
    if (!s) return fail(FP_ERR_INVALID_ARG, "shape is NULL");
    if (wq < FP_WQ_BF16 || wq > FP_WQ_BF16_2OF4) return fail(FP_ERR_INVALID_ARG, "bad weight quant %d", wq);
    if (kvq < FP_KV_BF16 || kvq > FP_KV_INT8) return fail(FP_ERR_INVALID_ARG, "bad kv quant %d", kvq);
    if (s->n_layers <= 0 || s->hidden <= 0 || s->n_heads <= 0 || s->n_kv_heads <= 0 ||
        s->head_dim <= 0 || s->ffn <= 0 || s->max_batch <= 0 || s->max_prompt <= 0 || s->max_seq <= 0)
        return fail(FP_ERR_INVALID_ARG, "shape fields must be positive");
    if (s->n_heads % s->n_kv_heads != 0)
        return fail(FP_ERR_INVALID_ARG, "n_heads %d not a multiple of n_kv_heads %d", s->n_heads, s->n_kv_heads);
    if (s->head_dim % 2 != 0) return fail(FP_ERR_INVALID_ARG, "head_dim must be even");
    if (s->max_seq < s->max_prompt) return fail(FP_ERR_INVALID_ARG, "max_seq < max_prompt");
    if (!(s->rms_eps > 0.f) || !(s->rope_theta > 0.f)) return fail(FP_ERR_INVALID_ARG, "rms_eps and rope_theta must be > 0");
    if (s->vocab < 0 || s->vocab % 16 != 0)
        return fail(FP_ERR_INVALID_ARG, "vocab %d must be 0 or a positive multiple of 16", s->vocab);
    const int q_dim = s->n_heads * s->head_dim;
    const int mult = (wq == FP_WQ_INT4_G128) ? 128 : (wq == FP_WQ_BF16_2OF4 ? 64 : 16);
    if (s->hidden % mult || q_dim % mult || s->ffn % mult)
        return fail(FP_ERR_INVALID_ARG, "hidden (%d), n_heads*head_dim (%d) and ffn (%d) must be multiples of %d",
                    s->hidden, q_dim, s->ffn, mult);
    if (s->head_dim != 64 && s->head_dim != 128)
        return fail(FP_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", s->head_dim);
    if (!attn_decode_supported(s->head_dim, s->n_heads / s->n_kv_heads))
        return fail(FP_ERR_UNSUPPORTED, "query group size %d not supported (1 to 16)",
                    s->n_heads / s->n_kv_heads);
    if (s->max_batch > 64) return fail(FP_ERR_UNSUPPORTED, "max_batch %d > 64", s->max_batch);
    if ((int64_t)s->max_batch * s->max_prompt > (1 << 24))
        return fail(FP_ERR_UNSUPPORTED, "max_batch * max_prompt too large");
    return FP_OK;
}

size_t act_elems(const fp_layer* h) { return (size_t)h->s.max_batch * h->s.max_prompt; }

// Allocate the storage of a [N, K] weight in format wf.
fp_status alloc_mat(fp_layer* h, Mat* m, int N, int K, int wf) {
    m->wf = wf;
    m->N = N;
    m->K = K;
    const int KS = weight_kstep(wf);
    m->kst = (K + KS - 1) / KS;
    const size_t nk = (size_t)N * K;
    fp_status st;
    if (wf == W_SP24) {        // 32-row x 32-input blocks: 1 KiB of values, 128 B of index words
        if ((st = dev_alloc(h, &m->codes, (size_t)(N / 32) * m->kst * 1024, &h->bytes_w))) return st;
        return alloc_t(h, &m->sidx, (size_t)(N / 32) * m->kst * 64, &h->bytes_w);
    }
    if ((st = dev_alloc(h, &m->codes, (size_t)(N / 16) * m->kst * 1024, &h->bytes_w))) return st;
    if (wf == W_INT8) return alloc_t(h, &m->scales, (size_t)N, &h->bytes_w);
    if (wf == W_INT4) {
        if ((st = alloc_t(h, &m->scales, nk / 128, &h->bytes_w))) return st;
        if ((st = alloc_t(h, &m->sz, nk / 128, &h->bytes_w))) return st;
        return alloc_t(h, &m->zeros, nk / 128, &h->bytes_w);
    }
    return FP_OK;
}

// Synthesise rows [row0, row0 + n) of matrix m from stream (seed, layer, tensor),
// quantise them (row-major, in tmpq) and write them into the fragment-major tiles.
// tmp holds >= n * K bf16 values, tmpq >= n * K bytes.
fp_status synth_rows(fp_layer* h, Mat* m, int row0, int n, int layer, int tensor, uint16_t* tmp, void* tmpq) {
    const uint64_t key = stream_key(h->seed, layer, tensor);
    const int K = m->K;
    const int64_t cnt = (int64_t)n * K;
    const int KS = weight_kstep(m->wf), eb = weight_ebits(m->wf);
    HIPCHK(launch_fill_bf16(tmp, cnt, key, 0.f, 0.02f, 0));
    if (m->wf == W_SP24) {
        HIPCHK(launch_sp24_compress(tmp, n, K, (uint16_t*)m->codes, m->sidx, row0, 0));
        return FP_OK;
    }
    const void* src = tmp;
    if (m->wf == W_INT8) {
        HIPCHK(launch_quant_int8(tmp, n, K, (int8_t*)tmpq, m->scales + row0, 0));
        src = tmpq;
    } else if (m->wf == W_INT4) {
        HIPCHK(launch_quant_int4(tmp, n, K, (uint32_t*)tmpq, m->scales + (int64_t)row0 * (K / 128),
                                 m->zeros + (int64_t)row0 * (K / 128), 0));
        src = tmpq;
    }
    HIPCHK(launch_tile(src, n, K, eb, KS, m->codes, row0, 0));
    return FP_OK;
}

// Split-K factor and k-range for a decode projection: aim for TARGET_WG workgroups,
// within the LDS bound on the staged activation slice.
void choose_split(int tiles, int K, int M, int wf, int target, int* ks, int* krange) {
    const int KS = skinny_kstep(wf);
    const int nsteps = (K + KS - 1) / KS;
    int k = (target + tiles - 1) / tiles;
    int kmax = nsteps / 4;             // keep at least four K-steps per workgroup
    if (kmax < 1) kmax = 1;
    if (k > kmax) k = kmax;
    if (k < 1) k = 1;
    int per = (nsteps + k - 1) / k;
    const int maxsteps = skinny_max_krange(M) / KS;
    if (per > maxsteps) per = maxsteps;
    *krange = per * KS;
    *ks = (K + *krange - 1) / *krange;
}

struct XIn {
    int xf = XF_COPY;
    const uint16_t* gain = nullptr;
    const float* ssq = nullptr;
    int ssq_blocks = 0;
    const float* src_part = nullptr;
    int src_ks = 0;
    int att_nsplit = 0, att_kps = 0;
};

// Split of a single-sequence decode projection: wide matrices (qkv, gate/up) stream
// faster with twice the workgroups.
void plan_skinny(const fp_layer* h, const Mat& m, int M, int dual_F, int* ks, int* kr) {
    (void)h;
    const int ncols = dual_F > 0 ? 2 * dual_F : m.N;
    choose_split(skinny_tiles(m.N, dual_F, M), m.K, M, m.wf, ncols >= SPLIT_WIDE_N ? 2 * TARGET_WG : TARGET_WG, ks,
                 kr);
}

fp_status run_skinny(fp_layer* h, const uint16_t* X, const Mat& m, int M, int dual_F, const XIn& xin,
                     float* part, int* ks_out, hipStream_t st) {
    SkinnyArgs a{};
    a.X = X;
    a.W = m.codes;
    a.scales = m.scales;
    a.zeros = m.zeros;
    a.sz = m.sz;
    a.M = M;
    a.N = m.N;
    a.K = m.K;
    a.kst = m.kst;
    a.dual_F = dual_F;
    a.part = part;
    a.xf = xin.xf;
    a.gain = xin.gain;
    a.ssq = xin.ssq;
    a.ssq_blocks = xin.ssq_blocks;
    a.eps = h->s.rms_eps;
    a.src_part = xin.src_part;
    a.src_ks = xin.src_ks;
    a.att_ws = h->attn_ws;
    a.att_nsplit = xin.att_nsplit;
    a.att_kps = xin.att_kps;
    a.head_dim = h->s.head_dim;
    a.d_pos = h->d_pos;
    int ks, kr;
    plan_skinny(h, m, M, dual_F, &ks, &kr);
    if (ks > KSMAX) return fail(FP_ERR_UNSUPPORTED, "split-K factor %d exceeds %d", ks, KSMAX);
    a.krange = kr;
    HIPCHK(launch_skinny(a, m.wf, ks, st));
    *ks_out = ks;
    return FP_OK;
}

// Batched decode projection: the workgroup walks its k-range in staged chunks, so the
// split-K factor only has to fill the GPU and stays small.  The kernels hold one
// workgroup per compute unit, so the factor is chosen by a cost model in units of one
// workgroup's chunk time: rounds of resident workgroups times (chunks per workgroup +
// a start-up cost of about two chunks), plus the partial sums each extra split writes
// and the consumer reads back (ks * M * N floats each way, at about 5 TB/s, against a
// chunk time of the workgroup's weight bytes at about 25 GB/s per compute unit).
constexpr int NCU = 256;
void plan_sp24(const Mat& m, int M, int* ks_out, int* kr_out);

// Bytes of one split of the qkv projection's partial sums that batch decode attention
// reads beyond their one read: every attention workgroup of a (sequence, kv head) reduces
// the sums of the group's queries itself.
double qkv_reread(const fp_layer* h, int B) {
    const fp_shape& s = h->s;
    int nsplit = 0, kps = 0;
    attn_decode_split(s.max_seq, B, s.n_kv_heads, s.n_heads / s.n_kv_heads, &nsplit, &kps);
    const int nsw = attn_decode_partials(nsplit);
    return (double)B * s.n_kv_heads * (nsw - 1) * s.n_heads / s.n_kv_heads * s.head_dim * 4.0;
}

void plan_skinny_batch(const fp_layer* h, const Mat& m, int M, int dual_F, int* ks_out, int* kr_out, double reread = 0.0) {
    if (m.wf == W_SP24) {
        plan_sp24(m, M, ks_out, kr_out);
        return;
    }
    const int KC = skinny_batch_chunk();
    const int nch = (m.K + KC - 1) / KC;
    (void)h;
    const int tiles = skinny_batch_tiles(m.N, dual_F, m.wf);
    const int rows = skinny_batch_rows(m.N, dual_F, m.wf);
    const double bpw = m.wf == W_BF16 ? 2.0 : (m.wf == W_INT8 ? 1.0 : 0.5);
    const double chunk_s = rows * KC * bpw / 25e9;
    // each split's partials are written and read once, and `reread` more bytes by a
    // consumer that reads them several times (decode attention re-reads the queries' sums)
    const double split_s = ((double)M * (dual_F > 0 ? 2.0 * dual_F : m.N) * 8.0 + reread) / 5e12;
    int per = nch;
    double best = 1e30;
    for (int k = 1; k <= std::min(nch, KSMAX); ++k) {
        const int p = (nch + k - 1) / k;
        const int ksk = (nch + p - 1) / p;
        const int rounds = (tiles * ksk + NCU - 1) / NCU;
        const double cost = rounds * (p + 2.0) * chunk_s + ksk * split_s;
        if (cost < best - 1e-12) { best = cost; per = p; }
    }
    *kr_out = per * KC;
    *ks_out = (nch + per - 1) / per;
}

// Split of a 2:4 sparse decode projection: about TARGET_WG workgroups of 128 rows, within
// the LDS bound on the staged activation slice.
void plan_sp24(const Mat& m, int M, int* ks_out, int* kr_out) {
    const int nsteps = m.K / 32;
    const int tiles = (m.N + 127) / 128;
    const int maxsteps = sp24_max_krange(M) / 32;
    int ks = std::max(1, std::min((TARGET_WG + tiles - 1) / tiles, std::max(1, nsteps / 4)));
    int per = (nsteps + ks - 1) / ks;
    if (per > maxsteps) per = maxsteps;
    *kr_out = per * 32;
    *ks_out = (nsteps + per - 1) / per;
}

fp_status run_skinny_batch(fp_layer* h, const uint16_t* X, const Mat& m, int M, int dual_F, float* part,
                           int* ks_out, hipStream_t st, double reread = 0.0) {
    if (m.wf == W_SP24) {      // the [gate; up] matrix is a plain [2F, K] matrix here
        Sp24Args a{};
        a.X = X;
        a.Wv = (const uint16_t*)m.codes;
        a.Wi = m.sidx;
        a.M = M;
        a.N = m.N;
        a.K = m.K;
        a.kst = m.kst;
        a.part = part;
        int ks;
        plan_sp24(m, M, &ks, &a.krange);
        if (ks > KSMAX) return fail(FP_ERR_UNSUPPORTED, "split-K factor %d exceeds %d", ks, KSMAX);
        HIPCHK(launch_sp24_gemv(a, ks, st));
        *ks_out = ks;
        return FP_OK;
    }
    SkinnyArgs a{};
    a.X = X;
    a.W = m.codes;
    a.scales = m.scales;
    a.zeros = m.zeros;
    a.sz = m.sz;
    a.M = M;
    a.N = m.N;
    a.K = m.K;
    a.kst = m.kst;
    a.dual_F = dual_F;
    a.part = part;
    a.xf = XF_COPY;
    int ks;
    plan_skinny_batch(h, m, M, dual_F, &ks, &a.krange, reread);
    if (ks > KSMAX) return fail(FP_ERR_UNSUPPORTED, "split-K factor %d exceeds %d", ks, KSMAX);
    HIPCHK(launch_skinny_batch(a, m.wf, ks, st));
    *ks_out = ks;
    return FP_OK;
}

fp_status run_gemm(fp_layer* h, const uint16_t* X, const Mat& m, int M, int epi, float* out32,
                   uint16_t* out16, const uint16_t* resid, hipStream_t st) {
    if (m.wf == W_SP24) {
        Sp24Args a{};
        a.X = X;
        a.Wv = (const uint16_t*)m.codes;
        a.Wi = m.sidx;
        a.M = M;
        a.N = m.N;
        a.K = m.K;
        a.F = h->s.ffn;
        a.kst = m.kst;
        a.out32 = out32;
        a.out16 = out16;
        a.resid = resid;
        a.out_fmt = h->act_fmt;
        HIPCHK(launch_gemm_sp24(a, epi, st));
        return FP_OK;
    }
    GemmArgs a{};
    a.X = X;
    a.W = m.codes;
    a.scales = m.scales;
    a.zeros = m.zeros;
    a.sz = m.sz;
    a.M = M;
    a.N = m.N;
    a.K = m.K;
    a.kst = m.kst;
    a.F = h->s.ffn;
    a.out32 = out32;
    a.out16 = out16;
    a.resid = resid;
    a.out_fmt = h->act_fmt;
    HIPCHK(launch_gemm(a, h->wq, epi, st));
    return FP_OK;
}

RopeKvArgs rope_args(fp_layer* h, int l, const float* part, int ks, int M, int T, const int* d_pos,
                     float* dump) {
    RopeKvArgs r{};
    r.part = part;
    r.ks = ks;
    r.M = M;
    r.T = T;
    r.nh = h->s.n_heads;
    r.nkv = h->s.n_kv_heads;
    r.d = h->s.head_dim;
    r.d_pos = d_pos;
    r.cos_t = h->cos_t;
    r.sin_t = h->sin_t;
    r.max_seq = h->s.max_seq;
    r.nblk = vt_blocks(h->s.max_seq);
    r.kv_stride = kv_row_stride(h->s.max_seq);
    r.qout = h->q16;
    r.kc = h->kc[l];
    r.vc = h->vc[l];
    r.ks_out = h->ksc[l];
    r.vs_out = h->vsc[l];
    r.kv_int8 = h->kvq == FP_KV_INT8;
    r.dump = dump;
    return r;
}

// Split factor of a prefill GEMM on the large tiling (1: no split).  Splits are used
// for the residual and SwiGLU GEMMs only, whose reductions (resid_norm_row_kernel,
// swiglu_kernel) also finish the epilogue; the residual reduction keeps a row in one
// workgroup, which bounds the hidden size.
int prefill_split(const fp_layer* h, int M, int N, int K, int dual_F, int* krange) {
    const int H = h->s.hidden;
    if (H % 8 != 0 || H > 16384 || h->wq == FP_WQ_BF16_2OF4) return 1;
    return gemm_split_factor(M, N, K, dual_F, h->wq, krange);
}

fp_status run_gemm_split(fp_layer* h, const uint16_t* X, const Mat& m, int M, int dual_F, int ks, int krange,
                         float* part, hipStream_t st) {
    GemmArgs a{};
    a.X = X;
    a.W = m.codes;
    a.scales = m.scales;
    a.zeros = m.zeros;
    a.sz = m.sz;
    a.M = M;
    a.N = m.N;
    a.K = m.K;
    a.kst = m.kst;
    a.F = h->s.ffn;
    a.out32 = part;
    a.krange = krange;
    HIPCHK(launch_gemm_split(a, h->wq, dual_F > 0, ks, st));
    return FP_OK;
}

fp_status enqueue_prefill(fp_layer* h, const uint16_t* x, int B, int P, uint16_t* y, hipStream_t st) {
    const fp_shape& s = h->s;
    const int M = B * P;
    const float scale = (float)(1.0 / std::sqrt((double)s.head_dim));
    fp_status rc;
    const int H = s.hidden, F = s.ffn;
    int kr_o, kr_g, kr_d;
    const int ks_o = prefill_split(h, M, H, h->q_dim, 0, &kr_o);
    const int ks_g = prefill_split(h, M, 2 * F, H, F, &kr_g);
    const int ks_d = prefill_split(h, M, H, F, 0, &kr_d);
    bool normed = false;    // act_in already holds this layer's normalised input
    for (int l = 0; l < s.n_layers; ++l) {
        const LayerW& W = h->L[l];
        const bool last = l == s.n_layers - 1;
        const uint16_t* in = (l == 0) ? x : h->xbuf;
        uint16_t* out = last ? y : h->xbuf;
        float* dump = h->dump ? h->dump + (size_t)l * 2 * M * h->kv_dim : nullptr;
        if (!normed) {
            h->prof.mark(FP_K_RMSNORM, l);
            HIPCHK(launch_rmsnorm(in, M, s.hidden, W.attn_norm, s.rms_eps, h->act_in, h->act_fmt, st));
        }
        normed = false;
        h->prof.mark(FP_K_QKV, l);
        if ((rc = run_gemm(h, h->act_in, W.qkv, M, EPI_F32, h->qkv32, nullptr, nullptr, st))) return rc;
        h->prof.mark(FP_K_ROPE_KV, l);
        HIPCHK(launch_rope_kv(rope_args(h, l, h->qkv32, 1, M, P, nullptr, dump), st));
        AttnPreArgs aa{};
        aa.q = h->q16;
        aa.kc = h->kc[l];
        aa.vc = h->vc[l];
        aa.k_scales = h->ksc[l];
        aa.v_scales = h->vsc[l];
        aa.staged = h->stage;
        aa.kv_int8 = h->kvq == FP_KV_INT8;
        aa.P = P;
        aa.nh = s.n_heads;
        aa.nkv = s.n_kv_heads;
        aa.d = s.head_dim;
        aa.max_seq = s.max_seq;
        aa.nblk = vt_blocks(s.max_seq);
        aa.kv_stride = kv_row_stride(s.max_seq);
        aa.scale = scale;
        aa.pmax = attn_prob_limit();
        aa.out = h->act_o;
        aa.out_fmt = h->act_fmt;
        h->prof.mark(FP_K_ATTN, l);
        if (aa.kv_int8) HIPCHK(launch_attn_stage(aa, B, st));
        HIPCHK(launch_attn_prefill(aa, B, st));
        h->prof.mark(FP_K_O, l);
        if (ks_o > 1) {
            // split-K partials; the residual add and the MLP RMSNorm in one row kernel
            if ((rc = run_gemm_split(h, h->act_o, W.o, M, 0, ks_o, kr_o, h->ppart, st))) return rc;
            HIPCHK(launch_resid_norm(h->ppart, ks_o, M, H, in, h->hbuf, W.mlp_norm, s.rms_eps, h->act_in,
                                     h->act_fmt, nullptr, nullptr, st));
        } else {
            if ((rc = run_gemm(h, h->act_o, W.o, M, EPI_RESID, nullptr, h->hbuf, in, st))) return rc;
            h->prof.mark(FP_K_RMSNORM, l);
            HIPCHK(launch_rmsnorm(h->hbuf, M, s.hidden, W.mlp_norm, s.rms_eps, h->act_in, h->act_fmt, st));
        }
        h->prof.mark(FP_K_GATE_UP, l);
        if (ks_g > 1) {
            if ((rc = run_gemm_split(h, h->act_in, W.gu, M, F, ks_g, kr_g, h->ppart, st))) return rc;
            HIPCHK(launch_swiglu(h->ppart, ks_g, M, F, h->act_f, h->act_fmt, st));
        } else {
            if ((rc = run_gemm(h, h->act_in, W.gu, M, EPI_SWIGLU, nullptr, h->act_f, nullptr, st))) return rc;
        }
        h->prof.mark(FP_K_DOWN, l);
        if (ks_d > 1) {
            // the residual add, and the next layer's attention RMSNorm
            if ((rc = run_gemm_split(h, h->act_f, W.down, M, 0, ks_d, kr_d, h->ppart, st))) return rc;
            HIPCHK(launch_resid_norm(h->ppart, ks_d, M, H, h->hbuf, out, last ? nullptr : h->L[l + 1].attn_norm,
                                     s.rms_eps, h->act_in, h->act_fmt, nullptr, nullptr, st));
            normed = !last;
        } else {
            if ((rc = run_gemm(h, h->act_f, W.down, M, EPI_RESID, nullptr, out, h->hbuf, st))) return rc;
        }
        if (h->ldump) HIPCHK(hipMemcpyAsync(h->ldump + (size_t)l * M * s.hidden, out, (size_t)M * s.hidden * 2,
                                            hipMemcpyDeviceToDevice, st));
    }
    h->prof.mark(FP_K_POS, -1);
    HIPCHK(launch_set_pos(h->d_pos, P, st));
    h->prof.end();
    return FP_OK;
}

AttnDecArgs attn_args(fp_layer* h, int l, int ks, int B, float* dump) {
    const fp_shape& s = h->s;
    AttnDecArgs ad{};
    ad.qkv_part = h->part;
    ad.ks = ks;
    ad.cos_t = h->cos_t;
    ad.sin_t = h->sin_t;
    ad.dump = dump;
    ad.kc = h->kc[l];
    ad.vc = h->vc[l];
    ad.k_scales = h->ksc[l];
    ad.v_scales = h->vsc[l];
    ad.kv_int8 = h->kvq == FP_KV_INT8;
    ad.nh = s.n_heads;
    ad.nkv = s.n_kv_heads;
    ad.d = s.head_dim;
    ad.max_seq = s.max_seq;
    ad.nblk = vt_blocks(s.max_seq);
    ad.kv_stride = kv_row_stride(s.max_seq);
    ad.d_pos = h->d_pos;
    ad.scale = (float)(1.0 / std::sqrt((double)s.head_dim));
    int nsplit;
    attn_decode_split(s.max_seq, B, s.n_kv_heads, s.n_heads / s.n_kv_heads, &nsplit, &ad.keys_per_split);
    ad.batch = B;
    ad.ws = h->attn_ws;
    ad.out = h->act_o;
    ad.out_fmt = h->act_fmt;
    return ad;
}

// One sequence: the RMSNorms and the SwiGLU are applied while the projections stage
// their inputs (layer 0 sums the squares of its input row itself), attention rotates
// and appends the new K / V itself, and a light kernel per residual add reduces the
// split-K partials and the row's sum of squares.
fp_status enqueue_decode_single(fp_layer* h, const uint16_t* x, uint16_t* y, hipStream_t st) {
    const fp_shape& s = h->s;
    const int B = h->B;
    const int ssq_blocks = resid_ssq_blocks(s.hidden);
    fp_status rc;
    int ks;
    for (int l = 0; l < s.n_layers; ++l) {
        const LayerW& W = h->L[l];
        const uint16_t* in = (l == 0) ? x : h->xbuf;
        uint16_t* out = (l == s.n_layers - 1) ? y : h->xbuf;
        float* dump = h->dump ? h->dump + (size_t)l * 2 * B * h->kv_dim : nullptr;
        XIn xq;
        xq.xf = XF_NORM;
        xq.gain = W.attn_norm;
        xq.ssq = (l == 0) ? nullptr : h->ssq;    // layer 0: the projection sums the squares itself
        xq.ssq_blocks = ssq_blocks;
        h->prof.mark(FP_K_QKV, l);
        if ((rc = run_skinny(h, in, W.qkv, B, 0, xq, h->part, &ks, st))) return rc;
        AttnDecArgs ad = attn_args(h, l, ks, B, dump);
        const int nsw = attn_decode_partials((s.max_seq + ad.keys_per_split - 1) / ad.keys_per_split);
        XIn xo;
        if (nsw > 1) {                  // the o projection merges the attention partials
            ad.skip_merge = 1;
            xo.xf = XF_MERGE;
            xo.att_nsplit = nsw;
            xo.att_kps = 4 * ad.keys_per_split;
        }
        h->prof.mark(FP_K_ATTN, l);
        HIPCHK(launch_attn_decode(ad, B, st));
        h->prof.mark(FP_K_O, l);
        if ((rc = run_skinny(h, h->act_o, W.o, B, 0, xo, h->part, &ks, st))) return rc;
        h->prof.mark(FP_K_RESID_NORM, l);
        HIPCHK(launch_resid_norm(h->part, ks, B, s.hidden, in, h->hbuf, nullptr, s.rms_eps, nullptr, h->act_fmt,
                                 h->ssq, nullptr, st));
        XIn xg;
        xg.xf = XF_NORM;
        xg.gain = W.mlp_norm;
        xg.ssq = h->ssq;
        xg.ssq_blocks = ssq_blocks;
        h->prof.mark(FP_K_GATE_UP, l);
        if ((rc = run_skinny(h, h->hbuf, W.gu, B, s.ffn, xg, h->part2, &ks, st))) return rc;
        XIn xd;
        xd.xf = XF_SWIGLU;
        xd.src_part = h->part2;
        xd.src_ks = ks;
        h->prof.mark(FP_K_DOWN, l);
        if ((rc = run_skinny(h, nullptr, W.down, B, 0, xd, h->part, &ks, st))) return rc;
        // the last residual kernel also advances the position (every reader has run)
        h->prof.mark(FP_K_RESID_NORM, l);
        HIPCHK(launch_resid_norm(h->part, ks, B, s.hidden, h->hbuf, out, nullptr, s.rms_eps, nullptr, h->act_fmt,
                                 h->ssq, (l == s.n_layers - 1) ? h->d_pos : nullptr, st));
        if (h->ldump) HIPCHK(hipMemcpyAsync(h->ldump + (size_t)l * B * s.hidden, out, (size_t)B * s.hidden * 2,
                                            hipMemcpyDeviceToDevice, st));
    }
    h->prof.end();
    return FP_OK;
}

// A batch: the RMSNorm of each projection input and the SwiGLU are formed once
// (every workgroup re-forming them from B rows would cost more than the weights).  The last
// layer's residual kernel also normalises the step's output with layer 0's gain, so a step
// whose input is the previous step's output (chained: n steps in one call) starts from that
// (the same kernel computes it from the same bf16 row, so the result is bit for bit the one
// the step's own first RMSNorm would give).
fp_status enqueue_decode_batch(fp_layer* h, const uint16_t* x, uint16_t* y, hipStream_t st, bool chained) {
    const fp_shape& s = h->s;
    const int B = h->B;
    fp_status rc;
    int ks;
    if (!chained) {
        h->prof.mark(FP_K_RMSNORM, 0);
        HIPCHK(launch_resid_norm(nullptr, 0, B, s.hidden, x, nullptr, h->L[0].attn_norm, s.rms_eps, h->act_in,
                                 h->act_fmt, h->ssq, nullptr, st));
    }
    for (int l = 0; l < s.n_layers; ++l) {
        const LayerW& W = h->L[l];
        const uint16_t* in = (l == 0) ? x : h->xbuf;
        uint16_t* out = (l == s.n_layers - 1) ? y : h->xbuf;
        float* dump = h->dump ? h->dump + (size_t)l * 2 * B * h->kv_dim : nullptr;
        h->prof.mark(FP_K_QKV, l);
        if ((rc = run_skinny_batch(h, h->act_in, W.qkv, B, 0, h->part, &ks, st, qkv_reread(h, B)))) return rc;
        h->prof.mark(FP_K_ATTN, l);
        HIPCHK(launch_attn_decode(attn_args(h, l, ks, B, dump), B, st));
        h->prof.mark(FP_K_O, l);
        if ((rc = run_skinny_batch(h, h->act_o, W.o, B, 0, h->part, &ks, st))) return rc;
        h->prof.mark(FP_K_RESID_NORM, l);
        HIPCHK(launch_resid_norm(h->part, ks, B, s.hidden, in, h->hbuf, W.mlp_norm, s.rms_eps, h->act_in,
                                 h->act_fmt, h->ssq, nullptr, st));
        h->prof.mark(FP_K_GATE_UP, l);
        if ((rc = run_skinny_batch(h, h->act_in, W.gu, B, s.ffn, h->part2, &ks, st))) return rc;
        h->prof.mark(FP_K_SWIGLU, l);
        HIPCHK(launch_swiglu(h->part2, ks, B, s.ffn, h->act_f, h->act_fmt, st));
        h->prof.mark(FP_K_DOWN, l);
        if ((rc = run_skinny_batch(h, h->act_f, W.down, B, 0, h->part, &ks, st))) return rc;
        const bool last = (l == s.n_layers - 1);
        h->prof.mark(FP_K_RESID_NORM, l);
        HIPCHK(launch_resid_norm(h->part, ks, B, s.hidden, h->hbuf, out, h->L[last ? 0 : l + 1].attn_norm,
                                 s.rms_eps, h->act_in, h->act_fmt, h->ssq, last ? h->d_pos : nullptr, st));
        if (h->ldump) HIPCHK(hipMemcpyAsync(h->ldump + (size_t)l * B * s.hidden, out, (size_t)B * s.hidden * 2,
                                            hipMemcpyDeviceToDevice, st));
    }
    h->prof.end();
    return FP_OK;
}

// 2:4 sparse weights run every batch size, one sequence included, on the batch schedule
// (their projection kernel stages plain activations).
fp_status enqueue_decode(fp_layer* h, const uint16_t* x, uint16_t* y, hipStream_t st, bool chained = false) {
    return h->B == 1 && h->wq != FP_WQ_BF16_2OF4 ? enqueue_decode_single(h, x, y, st)
                                                 : enqueue_decode_batch(h, x, y, st, chained);
}

// Final RMSNorm, LM head and greedy argmax of position T - 1 of each of B sequences of
// y [B, T, H].  One sequence: the projection normalises its row while staging it (the
// workgroup sums the row's squares itself); batches: a row kernel normalises first.
fp_status enqueue_head(fp_layer* h, const uint16_t* y, int B, int T, float* logits, int32_t* ids, hipStream_t st) {
    const int H = h->s.hidden;
    fp_status rc;
    int ks;
    if (B == 1) {
        XIn xn;
        xn.xf = XF_NORM;
        xn.gain = h->final_norm;
        xn.ssq = nullptr;
        if ((rc = run_skinny(h, y + (size_t)(T - 1) * H, h->lm, 1, 0, xn, h->hpart, &ks, st))) return rc;
    } else {
        HIPCHK(launch_head_norm(y, B, T, H, h->final_norm, h->s.rms_eps, h->hnorm, st));
        if ((rc = run_skinny_batch(h, h->hnorm, h->lm, B, 0, h->hpart, &ks, st))) return rc;
    }
    HIPCHK(launch_logits_argmax(h->hpart, ks, B, h->s.vocab, logits, h->hbval, h->hbidx, ids, st));
    return FP_OK;
}

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = (const char*)a;
    const char* pb = (const char*)b;
    return pa < pb + nb && pb < pa + na;
}

// Floats of the decode step's scratch buffers at batch B: split-K partials of the qkv / o /
// down projections (part) and of [gate; up] (part2), attention partials and row-norm
// block sums.  The same split plans the launchers use.
void decode_scratch_floats(const fp_layer* h, int B, size_t* part, size_t* part2, size_t* att, size_t* ssq) {
    const fp_shape& s = h->s;
    const LayerW& W = h->L[0];
    int kq, ko, kg, kd, kr;
    if (B == 1 && h->wq != FP_WQ_BF16_2OF4) {
        plan_skinny(h, W.qkv, B, 0, &kq, &kr);
        plan_skinny(h, W.o, B, 0, &ko, &kr);
        plan_skinny(h, W.gu, B, s.ffn, &kg, &kr);
        plan_skinny(h, W.down, B, 0, &kd, &kr);
    } else {
        plan_skinny_batch(h, W.qkv, B, 0, &kq, &kr, qkv_reread(h, B));
        plan_skinny_batch(h, W.o, B, 0, &ko, &kr);
        plan_skinny_batch(h, W.gu, B, s.ffn, &kg, &kr);
        plan_skinny_batch(h, W.down, B, 0, &kd, &kr);
    }
    *part = std::max({(size_t)kq * B * h->nqkv, (size_t)ko * B * s.hidden, (size_t)kd * B * s.hidden});
    *part2 = (size_t)kg * B * 2 * s.ffn;
    *att = (size_t)B * s.n_heads * attn_decode_max_splits(s.max_seq) * (s.head_dim + 4);
    *ssq = (size_t)B * resid_ssq_blocks(s.hidden);
}

}  // namespace

// One decode step, launched kernel by kernel (no graph capture, no allocation), with its
// scratch buffers carved from the caller-provided device region [scratch, scratch + bytes)
// instead of the handle's workspace.  FP_ERR_CAPACITY when the step needs more than bytes.
fp_status fpk::decode_step_scratch(fp_layer* h, const void* x, void* y, hipStream_t st, void* scratch,
                                   size_t bytes) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!x || !y) return fail(FP_ERR_INVALID_ARG, "x and y must be device pointers");
    if (!h->prefilled) return fail(FP_ERR_STATE, "decode step before prefill");
    if (h->pos >= h->s.max_seq) return fail(FP_ERR_CAPACITY, "position %d reached max_seq %d", h->pos, h->s.max_seq);
    const size_t xbytes = (size_t)h->B * h->s.hidden * 2;
    if (overlap(x, xbytes, y, xbytes)) return fail(FP_ERR_INVALID_ARG, "x and y overlap");
    size_t np, np2, na, ns;
    decode_scratch_floats(h, h->B, &np, &np2, &na, &ns);
    auto up = [](size_t floats) { return (floats * sizeof(float) + 255) / 256 * 256; };
    const size_t need = up(np) + up(np2) + up(na) + up(ns);
    if (need > bytes)
        return fail(FP_ERR_CAPACITY, "decode step at batch %d needs %zu bytes of scratch, the static region holds %zu",
                    h->B, need, bytes);
    if (!h->unbacked) {
        if (!scratch) return fail(FP_ERR_INVALID_ARG, "scratch region is NULL");
        char* p = (char*)scratch;
        float* part = (float*)p;
        float* part2 = (float*)(p += up(np));
        float* att = (float*)(p += up(np2));
        float* ssq = (float*)(p += up(na));
        std::swap(h->part, part);
        std::swap(h->part2, part2);
        std::swap(h->attn_ws, att);
        std::swap(h->ssq, ssq);
        const fp_status rc = enqueue_decode(h, (const uint16_t*)x, (uint16_t*)y, st);
        std::swap(h->part, part);
        std::swap(h->part2, part2);
        std::swap(h->attn_ws, att);
        std::swap(h->ssq, ssq);
        if (rc) return rc;
    }
    h->pos += 1;
    return FP_OK;
}

fp_status fpk::report_error(fp_status s, const char* msg) { return fail(s, "%s", msg); }
bool fpk::layer_unbacked(const fp_layer* h) { return h->unbacked; }

// ============================================================================ C ABI
extern "C" {

const char* fp_status_str(fp_status s) {
    switch (s) {
        case FP_OK: return "FP_OK";
        case FP_ERR_INVALID_ARG: return "FP_ERR_INVALID_ARG";
        case FP_ERR_STATE: return "FP_ERR_STATE";
        case FP_ERR_CAPACITY: return "FP_ERR_CAPACITY";
        case FP_ERR_OOM: return "FP_ERR_OOM";
        case FP_ERR_HIP: return "FP_ERR_HIP";
        case FP_ERR_UNSUPPORTED: return "FP_ERR_UNSUPPORTED";
    }
    return "FP_ERR_UNKNOWN";
}

const char* fp_last_error(void) { return g_err.c_str(); }

// Allocate the handle's weights, KV cache and workspace (an unbacked handle only counts
// the bytes: fp_memory_bytes then reports what a real handle of the shape holds).
fp_status alloc_storage(fp_layer* h) {
    const fp_shape& s = h->s;
    const int kvq = h->kvq;
    fp_status st;
    const int H = s.hidden, F = s.ffn;
    h->L.resize(s.n_layers);
    for (auto& W : h->L) {
        if ((st = alloc_t(h, &W.attn_norm, H, &h->bytes_w))) return st;
        if ((st = alloc_t(h, &W.mlp_norm, H, &h->bytes_w))) return st;
        if ((st = alloc_mat(h, &W.qkv, h->nqkv, H, h->wq))) return st;
        if ((st = alloc_mat(h, &W.o, H, h->q_dim, h->wq))) return st;
        if ((st = alloc_mat(h, &W.gu, 2 * F, H, h->wq))) return st;
        if ((st = alloc_mat(h, &W.down, H, F, h->wq))) return st;
    }
    // KV cache
    // keys [Bmax, nkv, kv_stride, d]; values in transposed blocks [Bmax, nkv, nblk, d, VT_BLK];
    // int8 scales [Bmax, nkv, kv_stride]
    const size_t esz = kvq == FP_KV_INT8 ? 1 : 2;
    const size_t kvs = (size_t)kv_row_stride(s.max_seq);
    const size_t kv_bytes = (size_t)s.max_batch * s.n_kv_heads * kvs * s.head_dim * esz;
    const size_t v_bytes = (size_t)s.max_batch * s.n_kv_heads * vt_blocks(s.max_seq) * VT_BLK * s.head_dim * esz;
    const size_t sc_elems = (size_t)s.max_batch * s.n_kv_heads * kvs;
    h->kc.assign(s.n_layers, nullptr);
    h->vc.assign(s.n_layers, nullptr);
    h->ksc.assign(s.n_layers, nullptr);
    h->vsc.assign(s.n_layers, nullptr);
    for (int l = 0; l < s.n_layers; ++l) {
        if ((st = dev_alloc(h, &h->kc[l], kv_bytes, &h->bytes_kv))) return st;
        if ((st = dev_alloc(h, &h->vc[l], v_bytes, &h->bytes_kv))) return st;
        if (kvq == FP_KV_INT8) {
            if ((st = alloc_t(h, &h->ksc[l], sc_elems, &h->bytes_kv))) return st;
            if ((st = alloc_t(h, &h->vsc[l], sc_elems, &h->bytes_kv))) return st;
        }
    }
    // workspace
    const size_t Mmax = std::max(act_elems(h), (size_t)s.max_batch);
    const int ncol = std::max({h->nqkv, H, 2 * F});
    if ((st = alloc_t(h, &h->act_in, Mmax * H, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->act_o, Mmax * h->q_dim, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->act_f, Mmax * F, &h->bytes_ws))) return st;
    if (kvq == FP_KV_INT8) {
        const size_t need = attn_stage_bytes(s.max_batch, s.max_prompt, s.n_kv_heads, s.head_dim);
        if (need <= Mmax * F * sizeof(uint16_t)) h->stage = h->act_f;
        else if ((st = dev_alloc(h, &h->stage, need, &h->bytes_ws))) return st;
    }
    if ((st = alloc_t(h, &h->hbuf, Mmax * H, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->xbuf, Mmax * H, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->qkv32, Mmax * h->nqkv, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->q16, Mmax * h->q_dim, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->part, (size_t)KSMAX * s.max_batch * ncol, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->part2, (size_t)KSMAX * s.max_batch * 2 * F, &h->bytes_ws))) return st;
    {
        // the largest split-K partial buffer any prefill size up to Mmax asks for (the split
        // factor depends on the number of 256-row tiles, so the worst case is at a whole tile)
        size_t pp = 0;
        const int Mp = (int)act_elems(h);
        for (int tm = 1; (int64_t)(tm - 1) * 256 < Mp; ++tm) {
            const int M = std::min(tm * 256, Mp);
            int kr;
            const int ko = prefill_split(h, M, H, h->q_dim, 0, &kr);
            const int kg = prefill_split(h, M, 2 * F, H, F, &kr);
            const int kd = prefill_split(h, M, H, F, 0, &kr);
            pp = std::max({pp, (size_t)(ko > 1 ? ko : 0) * M * H, (size_t)(kg > 1 ? kg : 0) * M * 2 * F,
                           (size_t)(kd > 1 ? kd : 0) * M * H});
        }
        if (pp > 0 && (st = alloc_t(h, &h->ppart, pp, &h->bytes_ws))) return st;
    }
    const size_t nch = attn_decode_max_splits(s.max_seq);
    if ((st = alloc_t(h, &h->attn_ws, (size_t)s.max_batch * s.n_heads * nch * (s.head_dim + 4), &h->bytes_ws)))
        return st;
    if ((st = alloc_t(h, &h->d_pos, 1, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->ssq, (size_t)s.max_batch * resid_ssq_blocks(H), &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->cos_t, (size_t)s.max_seq * s.head_dim / 2, &h->bytes_ws))) return st;
    if ((st = alloc_t(h, &h->sin_t, (size_t)s.max_seq * s.head_dim / 2, &h->bytes_ws))) return st;

    if (s.vocab > 0) {
        // embedding, final norm and LM head (bf16 under every weight format), and the head's
        // workspace: split-K partials for the largest batch's split, block bests, normalised
        // rows, and the embedded tokens / outputs of a request
        const int V = s.vocab;
        if ((st = alloc_t(h, &h->embed, (size_t)V * H, &h->bytes_w))) return st;
        if ((st = alloc_t(h, &h->final_norm, H, &h->bytes_w))) return st;
        if ((st = alloc_mat(h, &h->lm, V, H, W_BF16))) return st;
        size_t hp = 0;
        for (int b = 1; b <= s.max_batch; ++b) {
            int ks, kr;
            if (b == 1) plan_skinny(h, h->lm, b, 0, &ks, &kr);
            else plan_skinny_batch(h, h->lm, b, 0, &ks, &kr);
            hp = std::max(hp, (size_t)ks * b * V);
        }
        if ((st = alloc_t(h, &h->hpart, hp, &h->bytes_ws))) return st;
        if ((st = alloc_t(h, &h->hbval, (size_t)s.max_batch * head_logit_blocks(V), &h->bytes_ws))) return st;
        if ((st = alloc_t(h, &h->hbidx, (size_t)s.max_batch * head_logit_blocks(V), &h->bytes_ws))) return st;
        if ((st = alloc_t(h, &h->hnorm, (size_t)s.max_batch * H, &h->bytes_ws))) return st;
        if ((st = alloc_t(h, &h->tok_x, Mmax * H, &h->bytes_ws))) return st;
        if ((st = alloc_t(h, &h->tok_y, Mmax * H, &h->bytes_ws))) return st;
    }
    return FP_OK;
}

static fp_status create_impl(const fp_shape* shape, fp_weight_quant wq, fp_kv_quant kvq, uint64_t seed,
                             fp_layer** out, bool unbacked) {
    if (!out) return fail(FP_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    fp_status st = validate_shape(shape, wq, kvq);
    if (st) return st;
    fp_layer* h = new fp_layer();
    h->s = *shape;
    h->wq = wq;
    h->kvq = kvq;
    h->seed = seed;
    h->unbacked = unbacked;
    h->act_fmt = (wq == FP_WQ_BF16 || wq == FP_WQ_BF16_2OF4) ? ACT_BF16 : ACT_F16;
    const fp_shape& s = h->s;
    h->q_dim = s.n_heads * s.head_dim;
    h->kv_dim = s.n_kv_heads * s.head_dim;
    h->nqkv = h->q_dim + 2 * h->kv_dim;
    if (unbacked) {
        if ((st = alloc_storage(h))) {   // counts bytes only
            delete h;
            return st;
        }
        *out = h;
        return FP_OK;
    }

    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev == 0) {
        delete h;
        return fail(FP_ERR_HIP, "no HIP device available");
    }
    int dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess) {
        delete h;
        return fail(FP_ERR_HIP, "cannot query the current HIP device");
    }
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
        delete h;
        return fail(FP_ERR_UNSUPPORTED, "device %s is not gfx950", prop.gcnArchName);
    }

    auto bail = [&](fp_status code) {
        free_all(h);
        delete h;
        return code;
    };
    if ((st = alloc_storage(h))) return bail(st);
    const int H = s.hidden, F = s.ffn;
    const size_t maxrows = std::max<size_t>({(size_t)h->q_dim * H, (size_t)H * h->q_dim, (size_t)F * H,
                                             (size_t)H * F, (size_t)s.vocab * H});
    const size_t esz = kvq == FP_KV_INT8 ? 1 : 2;
    const size_t kvs = (size_t)kv_row_stride(s.max_seq);
    const size_t kv_bytes = (size_t)s.max_batch * s.n_kv_heads * kvs * s.head_dim * esz;
    const size_t v_bytes = (size_t)s.max_batch * s.n_kv_heads * vt_blocks(s.max_seq) * VT_BLK * s.head_dim * esz;
    const size_t sc_elems = (size_t)s.max_batch * s.n_kv_heads * kvs;

    // rotary tables: angle(p, i) = p * theta^(-2i/d) in double, rounded once to float
    {
        const int half = s.head_dim / 2;
        std::vector<float> c((size_t)s.max_seq * half), sn((size_t)s.max_seq * half);
        for (int i = 0; i < half; ++i) {
            const double inv = std::pow((double)s.rope_theta, -2.0 * i / s.head_dim);
            for (int p = 0; p < s.max_seq; ++p) {
                const double ang = (double)p * inv;
                c[(size_t)p * half + i] = (float)std::cos(ang);
                sn[(size_t)p * half + i] = (float)std::sin(ang);
            }
        }
        if (hipMemcpy(h->cos_t, c.data(), c.size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
            hipMemcpy(h->sin_t, sn.data(), sn.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
            return bail(fail(FP_ERR_HIP, "rotary table upload failed"));
    }

    // weights
    uint16_t* tmp = nullptr;
    void* tmpq = nullptr;
    size_t tmp_bytes = 0;
    if ((st = alloc_t(h, &tmp, maxrows, &tmp_bytes))) return bail(st);
    if ((st = dev_alloc(h, &tmpq, maxrows, &tmp_bytes))) return bail(st);
    for (int l = 0; l < s.n_layers; ++l) {
        LayerW& W = h->L[l];
        auto chk = [&](hipError_t e) { return e == hipSuccess ? FP_OK : fail(FP_ERR_HIP, "weight synthesis: %s", hipGetErrorString(e)); };
        if ((st = chk(launch_fill_bf16(W.attn_norm, H, stream_key(seed, l, FP_T_ATTN_NORM), 1.f, 0.02f, 0)))) return bail(st);
        if ((st = chk(launch_fill_bf16(W.mlp_norm, H, stream_key(seed, l, FP_T_MLP_NORM), 1.f, 0.02f, 0)))) return bail(st);
        if ((st = synth_rows(h, &W.qkv, 0, h->q_dim, l, FP_T_Q, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.qkv, h->q_dim, h->kv_dim, l, FP_T_K, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.qkv, h->q_dim + h->kv_dim, h->kv_dim, l, FP_T_V, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.o, 0, H, l, FP_T_O, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.gu, 0, F, l, FP_T_GATE, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.gu, F, F, l, FP_T_UP, tmp, tmpq))) return bail(st);
        if ((st = synth_rows(h, &W.down, 0, H, l, FP_T_DOWN, tmp, tmpq))) return bail(st);
        if (h->wq == FP_WQ_INT4_G128) {
            for (Mat* m : {&W.qkv, &W.o, &W.gu, &W.down})
                if ((st = chk(launch_pack_sz(m->scales, m->zeros, m->N, m->K / 128, m->sz, 0)))) return bail(st);
        }
    }
    if (s.vocab > 0) {
        auto chk = [&](hipError_t e) { return e == hipSuccess ? FP_OK : fail(FP_ERR_HIP, "head synthesis: %s", hipGetErrorString(e)); };
        if ((st = chk(launch_fill_bf16(h->embed, (int64_t)s.vocab * H, stream_key(seed, -1, FP_T_EMBED), 0.f, 0.02f, 0))))
            return bail(st);
        if ((st = chk(launch_fill_bf16(h->final_norm, H, stream_key(seed, -1, FP_T_FINAL_NORM), 1.f, 0.02f, 0))))
            return bail(st);
        if ((st = synth_rows(h, &h->lm, 0, s.vocab, -1, FP_T_LM_HEAD, tmp, tmpq))) return bail(st);
    }
    if (hipDeviceSynchronize() != hipSuccess) return bail(fail(FP_ERR_HIP, "weight synthesis failed"));
    for (void* p : {(void*)tmp, tmpq}) {
        (void)hipFree(p);
        h->allocs.erase(std::find(h->allocs.begin(), h->allocs.end(), p));
    }
    // zero the KV cache so exports of unwritten positions are deterministic
    for (int l = 0; l < s.n_layers; ++l) {
        if (hipMemset(h->kc[l], 0, kv_bytes) != hipSuccess || hipMemset(h->vc[l], 0, v_bytes) != hipSuccess)
            return bail(fail(FP_ERR_HIP, "kv clear failed"));
        if (kvq == FP_KV_INT8 && (hipMemset(h->ksc[l], 0, sc_elems * 2) != hipSuccess ||
                                   hipMemset(h->vsc[l], 0, sc_elems * 2) != hipSuccess))
            return bail(fail(FP_ERR_HIP, "kv clear failed"));
    }
    if (hipStreamCreateWithFlags(&h->cap_stream, hipStreamNonBlocking) != hipSuccess)
        return bail(fail(FP_ERR_HIP, "stream creation failed"));
    if (hipDeviceSynchronize() != hipSuccess) return bail(fail(FP_ERR_HIP, "create failed"));
    *out = h;
    return FP_OK;
}

fp_status fp_layer_create(const fp_shape* shape, fp_weight_quant wq, fp_kv_quant kvq, uint64_t seed,
                          fp_layer** out) {
    return create_impl(shape, wq, kvq, seed, out, false);
}

fp_status fp_layer_create_unbacked(const fp_shape* shape, fp_weight_quant wq, fp_kv_quant kvq,
                                   uint64_t seed, fp_layer** out) {
    return create_impl(shape, wq, kvq, seed, out, true);
}

fp_status fp_layer_destroy(fp_layer* h) {
    if (!h) return FP_OK;
    if (!h->unbacked) {
        (void)hipDeviceSynchronize();
        free_all(h);
    }
    delete h;
    return FP_OK;
}

fp_status fp_prefill(fp_layer* h, const void* x, int32_t B, int32_t P, void* y, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!x || !y) return fail(FP_ERR_INVALID_ARG, "x and y must be device pointers");
    if (B < 1 || P < 1) return fail(FP_ERR_INVALID_ARG, "B and P must be >= 1 (got %d, %d)", B, P);
    if (B > h->s.max_batch) return fail(FP_ERR_CAPACITY, "B %d > max_batch %d", B, h->s.max_batch);
    if (P > h->s.max_prompt) return fail(FP_ERR_CAPACITY, "P %d > max_prompt %d", P, h->s.max_prompt);
    const size_t bytes = (size_t)B * P * h->s.hidden * 2;
    if (overlap(x, bytes, y, bytes)) return fail(FP_ERR_INVALID_ARG, "x and y overlap");
    if (!h->unbacked) {
        if (B != h->B) drop_graphs(h);   // captured for another batch: never valid again
        fp_status st = enqueue_prefill(h, (const uint16_t*)x, B, P, (uint16_t*)y, (hipStream_t)stream);
        if (st) {
            h->prefilled = false;
            return st;
        }
    }
    h->B = B;
    h->pos = P;
    h->prefilled = true;
    return FP_OK;
}

fp_status fp_decode_step(fp_layer* h, const void* x, void* y, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!x || !y) return fail(FP_ERR_INVALID_ARG, "x and y must be device pointers");
    if (!h->prefilled) return fail(FP_ERR_STATE, "decode step before prefill");
    if (h->pos >= h->s.max_seq) return fail(FP_ERR_CAPACITY, "position %d reached max_seq %d", h->pos, h->s.max_seq);
    const size_t bytes = (size_t)h->B * h->s.hidden * 2;
    if (overlap(x, bytes, y, bytes)) return fail(FP_ERR_INVALID_ARG, "x and y overlap");
    if (!h->unbacked) {
        hipStream_t st = (hipStream_t)stream;
        fp_status rc;
        if (h->use_graph && !h->dump && !h->ldump) {
            const auto key = std::make_tuple(x, y, h->B);
            auto it = h->graphs.find(key);
            if (it == h->graphs.end()) {
                if (h->graphs.size() >= GRAPH_CACHE_MAX) drop_graphs(h);
                hipGraph_t g = nullptr;
                hipGraphExec_t ge = nullptr;
                HIPCHK(hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal));
                rc = enqueue_decode(h, (const uint16_t*)x, (uint16_t*)y, h->cap_stream);
                hipError_t e = hipStreamEndCapture(h->cap_stream, &g);
                if (rc) {
                    if (g) (void)hipGraphDestroy(g);
                    return rc;
                }
                if (e != hipSuccess) return fail(FP_ERR_HIP, "graph capture failed: %s", hipGetErrorString(e));
                e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
                (void)hipGraphDestroy(g);
                if (e != hipSuccess) return fail(FP_ERR_HIP, "graph instantiate failed: %s", hipGetErrorString(e));
                it = h->graphs.emplace(key, ge).first;
            }
            HIPCHK(hipGraphLaunch(it->second, st));
        } else {
            if ((rc = enqueue_decode(h, (const uint16_t*)x, (uint16_t*)y, st))) return rc;
        }
    }
    h->pos += 1;
    return FP_OK;
}

fp_status fp_decode_steps(fp_layer* h, void* x, void* y, int32_t n, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!x || !y) return fail(FP_ERR_INVALID_ARG, "x and y must be device pointers");
    if (n < 1) return fail(FP_ERR_INVALID_ARG, "n = %d steps", n);
    if (!h->prefilled) return fail(FP_ERR_STATE, "decode steps before prefill");
    if (h->pos + (int64_t)n > h->s.max_seq)
        return fail(FP_ERR_CAPACITY, "%d steps from position %d pass max_seq %d", n, h->pos, h->s.max_seq);
    const size_t bytes = (size_t)h->B * h->s.hidden * 2;
    if (overlap(x, bytes, y, bytes)) return fail(FP_ERR_INVALID_ARG, "x and y overlap");
    if (!h->unbacked) {
        // the step kernels advance the device-side position, so the steps chain as they are
        auto run = [&](hipStream_t s) -> fp_status {
            for (int i = 0; i < n; ++i) {
                const uint16_t* src = (const uint16_t*)((i & 1) ? y : x);
                uint16_t* dst = (uint16_t*)((i & 1) ? x : y);
                fp_status rc = enqueue_decode(h, src, dst, s, i > 0);   // step i > 0 reads step i - 1's output
                if (rc) return rc;
            }
            return FP_OK;
        };
        hipStream_t st = (hipStream_t)stream;
        fp_status rc;
        if (h->use_graph && !h->dump && !h->ldump) {
            const auto key = std::make_tuple(x, y, (int)n, h->B);
            auto it = h->mgraphs.find(key);
            if (it == h->mgraphs.end()) {
                if (h->mgraphs.size() >= GRAPH_CACHE_MAX) drop_graphs(h);
                hipGraph_t g = nullptr;
                hipGraphExec_t ge = nullptr;
                HIPCHK(hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal));
                rc = run(h->cap_stream);
                hipError_t e = hipStreamEndCapture(h->cap_stream, &g);
                if (rc) {
                    if (g) (void)hipGraphDestroy(g);
                    return rc;
                }
                if (e != hipSuccess) return fail(FP_ERR_HIP, "graph capture failed: %s", hipGetErrorString(e));
                e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
                (void)hipGraphDestroy(g);
                if (e != hipSuccess) return fail(FP_ERR_HIP, "graph instantiate failed: %s", hipGetErrorString(e));
                it = h->mgraphs.emplace(key, ge).first;
            }
            HIPCHK(hipGraphLaunch(it->second, st));
        } else {
            if ((rc = run(st))) return rc;
        }
    }
    h->pos += n;
    return FP_OK;
}

static fp_status collect_profile(fp_layer* h, fp_kernel_time* out, int32_t cap, int32_t* count) {
    fp_status rc = FP_OK;
    if (hipStreamSynchronize(h->prof.st) != hipSuccess) rc = fail(FP_ERR_HIP, "profile synchronise failed");
    int n = 0;
    for (size_t i = 0; rc == FP_OK && i < h->prof.t0.size(); ++i) {
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, h->prof.t0[i], h->prof.t1[i]) != hipSuccess) {
            rc = fail(FP_ERR_HIP, "event timing failed");
            break;
        }
        if (n < cap) out[n++] = fp_kernel_time{h->prof.kind[i], h->prof.layer[i], ms};
    }
    if (count) *count = n;
    h->prof.clear();
    return rc;
}

fp_status fp_profile_prefill(fp_layer* h, const void* x, int32_t B, int32_t P, void* y, void* stream,
                             fp_kernel_time* out, int32_t cap, int32_t* count) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!out || cap <= 0) return fail(FP_ERR_INVALID_ARG, "no output records");
    if (h->unbacked) return fail(FP_ERR_STATE, "handle has no device storage");
    h->prof.clear();
    h->prof.on = true;
    h->prof.st = (hipStream_t)stream;
    fp_status rc = fp_prefill(h, x, B, P, y, stream);
    if (rc) {
        h->prof.clear();
        return rc;
    }
    return collect_profile(h, out, cap, count);
}

fp_status fp_profile_decode_step(fp_layer* h, const void* x, void* y, void* stream, fp_kernel_time* out,
                                 int32_t cap, int32_t* count) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (!out || cap <= 0) return fail(FP_ERR_INVALID_ARG, "no output records");
    if (h->unbacked) return fail(FP_ERR_STATE, "handle has no device storage");
    const bool g = h->use_graph;
    h->use_graph = false;            // launch kernel by kernel
    h->prof.clear();
    h->prof.on = true;
    h->prof.st = (hipStream_t)stream;
    fp_status rc = fp_decode_step(h, x, y, stream);
    h->use_graph = g;
    if (rc) {
        h->prof.clear();
        return rc;
    }
    return collect_profile(h, out, cap, count);
}

fp_status fp_embed(fp_layer* h, const int32_t* ids, int64_t M, void* x, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (h->s.vocab == 0) return fail(FP_ERR_STATE, "the handle has no embedding (vocab = 0)");
    if (!ids || !x) return fail(FP_ERR_INVALID_ARG, "ids and x must be device pointers");
    if (M < 1 || M > (int64_t)1 << 30) return fail(FP_ERR_INVALID_ARG, "M = %lld tokens", (long long)M);
    if (h->unbacked) return FP_OK;
    HIPCHK(launch_embed((const int*)ids, M, h->embed, h->s.vocab, h->s.hidden, (uint16_t*)x, (hipStream_t)stream));
    return FP_OK;
}

fp_status fp_head(fp_layer* h, const void* y, int32_t B, int32_t T, float* logits, int32_t* next_ids, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (h->s.vocab == 0) return fail(FP_ERR_STATE, "the handle has no LM head (vocab = 0)");
    if (!y || !next_ids) return fail(FP_ERR_INVALID_ARG, "y and next_ids must be device pointers");
    if (B < 1 || T < 1) return fail(FP_ERR_INVALID_ARG, "B and T must be >= 1 (got %d, %d)", B, T);
    if (B > h->s.max_batch) return fail(FP_ERR_CAPACITY, "B %d > max_batch %d", B, h->s.max_batch);
    if (h->unbacked) return FP_OK;
    return enqueue_head(h, (const uint16_t*)y, B, T, logits, next_ids, (hipStream_t)stream);
}

fp_status fp_generate(fp_layer* h, const int32_t* prompt_ids, int32_t B, int32_t P, int32_t n_out, int32_t* out_ids,
                      float* logits, const int32_t* force_ids, float* elapsed_ms, void* stream) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (h->s.vocab == 0) return fail(FP_ERR_STATE, "the handle has no embedding / LM head (vocab = 0)");
    if (!prompt_ids || !out_ids) return fail(FP_ERR_INVALID_ARG, "prompt_ids and out_ids must be device pointers");
    if (B < 1 || P < 1 || n_out < 0)
        return fail(FP_ERR_INVALID_ARG, "B, P >= 1 and n_out >= 0 required (got %d, %d, %d)", B, P, n_out);
    if (B > h->s.max_batch) return fail(FP_ERR_CAPACITY, "B %d > max_batch %d", B, h->s.max_batch);
    if (P > h->s.max_prompt) return fail(FP_ERR_CAPACITY, "P %d > max_prompt %d", P, h->s.max_prompt);
    if ((int64_t)P + n_out > h->s.max_seq)
        return fail(FP_ERR_CAPACITY, "P %d + n_out %d > max_seq %d", P, n_out, h->s.max_seq);
    if (h->unbacked) {
        h->B = B;
        h->pos = P + n_out;
        h->prefilled = true;
        return FP_OK;
    }
    hipStream_t st = (hipStream_t)stream;
    if (B != h->B) drop_graphs(h);
    const int H = h->s.hidden, V = h->s.vocab;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (elapsed_ms) {
        HIPCHK(hipEventCreate(&e0));
        if (hipEventCreate(&e1) != hipSuccess) {
            (void)hipEventDestroy(e0);
            return fail(FP_ERR_HIP, "event creation failed");
        }
    }
    auto finish = [&](fp_status rc) {
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
        return rc;
    };
    if (e0 && hipEventRecord(e0, st) != hipSuccess) return finish(fail(FP_ERR_HIP, "event record failed"));
    fp_status rc;
    h->prefilled = false;
    // the prompt: embed, prefill, head -> token 0
    if (hipError_t e = launch_embed((const int*)prompt_ids, (int64_t)B * P, h->embed, V, H, h->tok_x, st))
        return finish(fail(FP_ERR_HIP, "embedding launch failed: %s", hipGetErrorString(e)));
    if ((rc = enqueue_prefill(h, h->tok_x, B, P, h->tok_y, st))) return finish(rc);
    if ((rc = enqueue_head(h, h->tok_y, B, P, logits, out_ids, st))) return finish(rc);
    h->B = B;
    h->pos = P;
    h->prefilled = true;
    // n_out decode steps: embed token i - 1, decode, head -> token i
    auto loop = [&](hipStream_t s) -> fp_status {
        for (int i = 1; i <= n_out; ++i) {
            const int32_t* src = force_ids ? force_ids + (size_t)(i - 1) * B : out_ids + (size_t)(i - 1) * B;
            if (hipError_t e = launch_embed((const int*)src, B, h->embed, V, H, h->tok_x, s))
                return fail(FP_ERR_HIP, "embedding launch failed: %s", hipGetErrorString(e));
            fp_status r = enqueue_decode(h, h->tok_x, h->tok_y, s);
            if (r) return r;
            r = enqueue_head(h, h->tok_y, B, 1, logits ? logits + (size_t)i * B * V : nullptr, out_ids + (size_t)i * B, s);
            if (r) return r;
        }
        return FP_OK;
    };
    if (n_out > 0) {
        if (h->use_graph && !h->dump && !h->ldump) {
            const auto key = std::make_tuple(out_ids, logits, force_ids, (int)n_out, B);
            auto it = h->ggraphs.find(key);
            if (it == h->ggraphs.end()) {
                if (h->ggraphs.size() >= GRAPH_CACHE_MAX) drop_graphs(h);
                hipGraph_t g = nullptr;
                hipGraphExec_t ge = nullptr;
                if (hipStreamBeginCapture(h->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
                    return finish(fail(FP_ERR_HIP, "graph capture failed to start"));
                rc = loop(h->cap_stream);
                hipError_t e = hipStreamEndCapture(h->cap_stream, &g);
                if (rc) {
                    if (g) (void)hipGraphDestroy(g);
                    return finish(rc);
                }
                if (e != hipSuccess) return finish(fail(FP_ERR_HIP, "graph capture failed: %s", hipGetErrorString(e)));
                e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
                (void)hipGraphDestroy(g);
                if (e != hipSuccess) return finish(fail(FP_ERR_HIP, "graph instantiate failed: %s", hipGetErrorString(e)));
                it = h->ggraphs.emplace(key, ge).first;
            }
            if (hipGraphLaunch(it->second, st) != hipSuccess) return finish(fail(FP_ERR_HIP, "graph launch failed"));
        } else if ((rc = loop(st))) {
            return finish(rc);
        }
    }
    h->pos = P + n_out;
    if (e1) {
        float ms = 0.f;
        if (hipEventRecord(e1, st) != hipSuccess || hipEventSynchronize(e1) != hipSuccess ||
            hipEventElapsedTime(&ms, e0, e1) != hipSuccess)
            return finish(fail(FP_ERR_HIP, "request timing failed"));
        *elapsed_ms = ms;
    }
    return finish(FP_OK);
}

fp_status fp_set_decode_graph(fp_layer* h, int32_t enable) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    h->use_graph = enable != 0;
    return FP_OK;
}

fp_status fp_fill_normal(void* dst, int64_t n, uint64_t seed, int32_t layer, int32_t tensor, float mean,
                         float sigma, void* stream) {
    if (!dst && n > 0) return fail(FP_ERR_INVALID_ARG, "dst is NULL");
    if (n < 0) return fail(FP_ERR_INVALID_ARG, "n < 0");
    if (tensor < 0 || tensor > 255) return fail(FP_ERR_INVALID_ARG, "tensor id out of range");
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev == 0) return fail(FP_ERR_HIP, "no HIP device available");
    HIPCHK(launch_fill_bf16((uint16_t*)dst, n, stream_key(seed, layer, tensor), mean, sigma, (hipStream_t)stream));
    return FP_OK;
}

fp_status fp_export_weight(fp_layer* h, int32_t l, int32_t tensor, void* codes, void* scales, void* zeros) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    const bool head = tensor == FP_T_EMBED || tensor == FP_T_FINAL_NORM || tensor == FP_T_LM_HEAD;
    if (head ? l != -1 : (l < 0 || l >= h->s.n_layers))
        return fail(FP_ERR_INVALID_ARG, "layer index %d out of range for tensor %d", l, tensor);
    if (head && h->s.vocab == 0) return fail(FP_ERR_STATE, "the handle has no embedding / LM head (vocab = 0)");
    if (!codes) return fail(FP_ERR_INVALID_ARG, "codes is NULL");
    if (h->unbacked) return fail(FP_ERR_STATE, "handle has no device storage");
    const int H = h->s.hidden;
    if (tensor == FP_T_ATTN_NORM || tensor == FP_T_MLP_NORM || tensor == FP_T_FINAL_NORM || tensor == FP_T_EMBED) {
        const uint16_t* src = tensor == FP_T_ATTN_NORM ? h->L[l].attn_norm
                            : tensor == FP_T_MLP_NORM  ? h->L[l].mlp_norm
                            : tensor == FP_T_FINAL_NORM ? h->final_norm : h->embed;
        const size_t n = tensor == FP_T_EMBED ? (size_t)h->s.vocab * H : (size_t)H;
        HIPCHK(hipDeviceSynchronize());
        HIPCHK(hipMemcpy(codes, src, n * 2, hipMemcpyDeviceToHost));
        return FP_OK;
    }
    const Mat* m = nullptr;
    int row0 = 0, n = 0;
    switch (tensor) {
        case FP_T_Q: m = &h->L[l].qkv; row0 = 0; n = h->q_dim; break;
        case FP_T_K: m = &h->L[l].qkv; row0 = h->q_dim; n = h->kv_dim; break;
        case FP_T_V: m = &h->L[l].qkv; row0 = h->q_dim + h->kv_dim; n = h->kv_dim; break;
        case FP_T_O: m = &h->L[l].o; row0 = 0; n = H; break;
        case FP_T_GATE: m = &h->L[l].gu; row0 = 0; n = h->s.ffn; break;
        case FP_T_UP: m = &h->L[l].gu; row0 = h->s.ffn; n = h->s.ffn; break;
        case FP_T_DOWN: m = &h->L[l].down; row0 = 0; n = H; break;
        case FP_T_LM_HEAD: m = &h->lm; row0 = 0; n = h->s.vocab; break;
        default: return fail(FP_ERR_INVALID_ARG, "unknown tensor id %d", tensor);
    }
    const int K = m->K, wf = m->wf;
    if (wf == W_SP24) {
        // value and index blocks -> dense bf16 rows (pruned weights zero)
        HIPCHK(hipDeviceSynchronize());
        const size_t nblk = (size_t)(n / 32) * m->kst;
        std::vector<uint16_t> vals(nblk * 512), idx(nblk * 64);
        HIPCHK(hipMemcpy(vals.data(), (const uint16_t*)m->codes + (size_t)(row0 / 32) * m->kst * 512, vals.size() * 2,
                         hipMemcpyDeviceToHost));
        HIPCHK(hipMemcpy(idx.data(), m->sidx + (size_t)(row0 / 32) * m->kst * 64, idx.size() * 2,
                         hipMemcpyDeviceToHost));
        uint16_t* dst = (uint16_t*)codes;
        std::memset(dst, 0, (size_t)n * K * 2);
        for (int rb = 0; rb < n / 32; ++rb)
            for (int kb = 0; kb < m->kst; ++kb)
                for (int L = 0; L < 64; ++L) {
                    const size_t b = (size_t)rb * m->kst + kb;
                    const int r = 32 * rb + (L & 31), s = L >> 5;
                    const uint32_t word = idx[b * 64 + L];
                    for (int i = 0; i < 8; ++i) {
                        const int g = i / 2, pos = (word >> (2 * i)) & 3;
                        const int k = 32 * kb + (g < 2 ? 0 : 16) + 8 * s + 4 * (g & 1) + pos;
                        dst[(size_t)r * K + k] = vals[b * 512 + L * 8 + i];
                    }
                }
        return FP_OK;
    }
    if (wf != W_BF16 && !scales) return fail(FP_ERR_INVALID_ARG, "scales is NULL");
    if (wf == W_INT4 && !zeros) return fail(FP_ERR_INVALID_ARG, "zeros is NULL");
    HIPCHK(hipDeviceSynchronize());
    // fragment-major tiles -> row-major canonical layout
    const int KS = weight_kstep(wf), eb = weight_ebits(wf);
    const size_t blk_bytes = 1024, nblk = (size_t)(n / 16) * m->kst;
    std::vector<uint8_t> tiles(nblk * blk_bytes);
    HIPCHK(hipMemcpy(tiles.data(), (const uint8_t*)m->codes + (size_t)(row0 / 16) * m->kst * blk_bytes,
                     tiles.size(), hipMemcpyDeviceToHost));
    const size_t rowbytes = (size_t)K * eb / 8, chunk = 16;
    uint8_t* dst = (uint8_t*)codes;
    for (int nt = 0; nt < n / 16; ++nt)
        for (int st = 0; st < m->kst; ++st)
            for (int L = 0; L < 64; ++L) {
                const int r = L & 15, g = L >> 4;
                const int k0 = st * KS + g * (KS / 4);
                if (k0 >= K) continue;
                std::memcpy(dst + (size_t)(16 * nt + r) * rowbytes + (size_t)k0 * eb / 8,
                            tiles.data() + ((size_t)nt * m->kst + st) * blk_bytes + (size_t)L * chunk, chunk);
            }
    if (wf == W_BF16) return FP_OK;
    if (wf == W_INT8) {
        HIPCHK(hipMemcpy(scales, m->scales + row0, (size_t)n * 2, hipMemcpyDeviceToHost));
        return FP_OK;
    }
    // int4: device nibble order -> canonical (nibble j holds column 8w + j)
    uint32_t* wds = (uint32_t*)codes;
    const size_t words = (size_t)n * K / 8;
    for (size_t i = 0; i < words; ++i) {
        const uint32_t wv = wds[i];
        uint32_t c = 0;
        for (int p = 0; p < 8; ++p) {
            const int col = (p < 4) ? 2 * p : 2 * (p - 4) + 1;
            c |= ((wv >> (4 * p)) & 0xFu) << (4 * col);
        }
        wds[i] = c;
    }
    HIPCHK(hipMemcpy(scales, m->scales + (size_t)row0 * (K / 128), (size_t)n * (K / 128) * 2, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(zeros, m->zeros + (size_t)row0 * (K / 128), (size_t)n * (K / 128) * 2, hipMemcpyDeviceToHost));
    return FP_OK;
}

fp_status fp_export_kv(fp_layer* h, int32_t l, void* k, void* v, void* k_scales, void* v_scales) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (l < 0 || l >= h->s.n_layers) return fail(FP_ERR_INVALID_ARG, "layer index %d out of range", l);
    if (!k || !v) return fail(FP_ERR_INVALID_ARG, "k and v must be host buffers");
    if (h->unbacked) return fail(FP_ERR_STATE, "handle has no device storage");
    if (!h->prefilled) return fail(FP_ERR_STATE, "no prefill yet");
    const fp_shape& s = h->s;
    const size_t esz = h->kvq == FP_KV_INT8 ? 1 : 2;
    const int D = s.head_dim, nblk = vt_blocks(s.max_seq);
    const size_t kvs = (size_t)kv_row_stride(s.max_seq), nbh = (size_t)h->B * s.n_kv_heads;
    HIPCHK(hipDeviceSynchronize());
    // keys: rows of kv_stride -> [B, nkv, max_seq, d]
    HIPCHK(hipMemcpy2D(k, (size_t)s.max_seq * D * esz, h->kc[l], kvs * D * esz, (size_t)s.max_seq * D * esz, nbh,
                       hipMemcpyDeviceToHost));
    // values: transposed blocks -> [B, nkv, max_seq, d]
    std::vector<uint8_t> vt((size_t)h->B * s.n_kv_heads * nblk * VT_BLK * D * esz);
    HIPCHK(hipMemcpy(vt.data(), h->vc[l], vt.size(), hipMemcpyDeviceToHost));
    uint8_t* vd = (uint8_t*)v;
    for (size_t bh = 0; bh < (size_t)h->B * s.n_kv_heads; ++bh)
        for (int p = 0; p < s.max_seq; ++p)
            for (int dd = 0; dd < D; ++dd) {
                const size_t src = ((bh * nblk + p / VT_BLK) * D + dd) * VT_BLK + vt_slot(p % VT_BLK);
                std::memcpy(vd + ((bh * s.max_seq + p) * D + dd) * esz, vt.data() + src * esz, esz);
            }
    if (h->kvq == FP_KV_INT8) {
        if (!k_scales || !v_scales) return fail(FP_ERR_INVALID_ARG, "scale buffers are NULL");
        HIPCHK(hipMemcpy2D(k_scales, (size_t)s.max_seq * 2, h->ksc[l], kvs * 2, (size_t)s.max_seq * 2, nbh,
                           hipMemcpyDeviceToHost));
        HIPCHK(hipMemcpy2D(v_scales, (size_t)s.max_seq * 2, h->vsc[l], kvs * 2, (size_t)s.max_seq * 2, nbh,
                           hipMemcpyDeviceToHost));
    }
    return FP_OK;
}

fp_status fp_set_debug_kv_dump(fp_layer* h, void* dev_f32) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    h->dump = (float*)dev_f32;
    return FP_OK;
}

fp_status fp_set_debug_layer_dump(fp_layer* h, void* dev_bf16) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    h->ldump = (uint16_t*)dev_bf16;
    return FP_OK;
}

fp_status fp_memory_bytes(const fp_layer* h, size_t* weights, size_t* kv, size_t* workspace) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (weights) *weights = h->bytes_w;
    if (kv) *kv = h->bytes_kv;
    if (workspace) *workspace = h->bytes_ws;
    return FP_OK;
}

fp_status fp_get_position(const fp_layer* h, int32_t* pos, int32_t* batch) {
    if (!h) return fail(FP_ERR_INVALID_ARG, "layer is NULL");
    if (pos) *pos = h->prefilled ? h->pos : 0;
    if (batch) *batch = h->prefilled ? h->B : 0;
    return FP_OK;
}

}  // extern "C"
