// Latency and memory estimation from fingerprints (paper Sec. 5.2 and Sec. 5.3): the
// arithmetic that turns a few fingerprint observations into the estimate for a stack of
// any number of hidden layers.  Host only.
//
//   Eq. 1   latency = TTFT + output_length * TPOT
//   Eq. 2   TTFT = num_layers * TTFT_layer + TTFT_other
//   Eq. 3   TPOT = num_layers * TPOT_layer + TPOT_other
// L2 observes two fingerprints (layer counts n_a, n_b), each at two output lengths: a 2x2
// system of Eq. 1 per fingerprint, then a 4x4 system of Eq. 2 and Eq. 3.  M2 extrapolates
// fingerprint footprints linearly in the layer count.
#include "fp_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>

namespace {

// Solve A x = b for n <= 4 by Gaussian elimination with partial pivoting.  Returns false
// for a (numerically) singular A: a pivot below 1e-12 of the largest |A| entry.
bool solve(int n, double A[4][4], double b[4], double x[4]) {
    double amax = 0.0;
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j) amax = std::fmax(amax, std::fabs(A[i][j]));
    if (!(amax > 0.0)) return false;
    for (int c = 0; c < n; ++c) {
        int p = c;
        for (int r = c + 1; r < n; ++r)
            if (std::fabs(A[r][c]) > std::fabs(A[p][c])) p = r;
        if (!(std::fabs(A[p][c]) > 1e-12 * amax)) return false;
        if (p != c) {
            for (int j = 0; j < n; ++j) std::swap(A[p][j], A[c][j]);
            std::swap(b[p], b[c]);
        }
        for (int r = c + 1; r < n; ++r) {
            const double f = A[r][c] / A[c][c];
            for (int j = c; j < n; ++j) A[r][j] -= f * A[c][j];
            b[r] -= f * b[c];
        }
    }
    for (int r = n - 1; r >= 0; --r) {
        double v = b[r];
        for (int j = r + 1; j < n; ++j) v -= A[r][j] * x[j];
        x[r] = v / A[r][r];
    }
    return true;
}

}  // namespace

extern "C" {

fp_status fp_fit_ttft_tpot(const int32_t n_out[2], const double latency[2], double* ttft, double* tpot) {
    if (!n_out || !latency || !ttft || !tpot) return fpk::report_error(FP_ERR_INVALID_ARG, "NULL argument");
    double A[4][4] = {{1.0, (double)n_out[0]}, {1.0, (double)n_out[1]}};
    double b[4] = {latency[0], latency[1]}, x[4] = {};
    if (!solve(2, A, b, x))
        return fpk::report_error(FP_ERR_INVALID_ARG, "Eq. 1 needs two distinct output lengths");
    *ttft = x[0];
    *tpot = x[1];
    return FP_OK;
}

fp_status fp_fit_latency_l2(const int32_t layers[2], const int32_t n_out[2], const double latency[4],
                            fp_latency_model* model) {
    if (!layers || !n_out || !latency || !model) return fpk::report_error(FP_ERR_INVALID_ARG, "NULL argument");
    double t[2], p[2];
    for (int i = 0; i < 2; ++i) {
        const fp_status st = fp_fit_ttft_tpot(n_out, latency + 2 * i, &t[i], &p[i]);
        if (st) return st;
    }
    // unknowns (TTFT_layer, TPOT_layer, TTFT_other, TPOT_other); rows: Eq. 2 for both
    // fingerprints, then Eq. 3 for both
    const double na = layers[0], nb = layers[1];
    double A[4][4] = {{na, 0.0, 1.0, 0.0}, {nb, 0.0, 1.0, 0.0}, {0.0, na, 0.0, 1.0}, {0.0, nb, 0.0, 1.0}};
    double b[4] = {t[0], t[1], p[0], p[1]}, x[4] = {};
    if (!solve(4, A, b, x))
        return fpk::report_error(FP_ERR_INVALID_ARG, "Eq. 2 and Eq. 3 need two distinct layer counts");
    model->ttft_layer = x[0];
    model->tpot_layer = x[1];
    model->ttft_other = x[2];
    model->tpot_other = x[3];
    return FP_OK;
}

fp_status fp_predict_latency(const fp_latency_model* m, int32_t n_layers, int32_t n_out, double* ttft, double* tpot,
                             double* latency) {
    if (!m) return fpk::report_error(FP_ERR_INVALID_ARG, "model is NULL");
    if (n_layers < 0 || n_out < 0) return fpk::report_error(FP_ERR_INVALID_ARG, "negative layer count or length");
    const double t = n_layers * m->ttft_layer + m->ttft_other;
    const double p = n_layers * m->tpot_layer + m->tpot_other;
    if (ttft) *ttft = t;
    if (tpot) *tpot = p;
    if (latency) *latency = t + n_out * p;
    return FP_OK;
}

fp_status fp_extrapolate_layers(const int32_t layers[2], const double values[2], int32_t n_layers, double* value) {
    if (!layers || !values || !value) return fpk::report_error(FP_ERR_INVALID_ARG, "NULL argument");
    if (layers[0] == layers[1]) return fpk::report_error(FP_ERR_INVALID_ARG, "two distinct layer counts are needed");
    const double slope = (values[1] - values[0]) / (double)(layers[1] - layers[0]);
    *value = values[0] + (double)(n_layers - layers[0]) * slope;
    return FP_OK;
}

fp_status fp_device_memory(size_t* used, size_t* total) {
    size_t fr = 0, tot = 0;
    if (hipMemGetInfo(&fr, &tot) != hipSuccess) return fpk::report_error(FP_ERR_HIP, "hipMemGetInfo failed");
    if (used) *used = tot - fr;
    if (total) *total = tot;
    return FP_OK;
}

}  // extern "C"
