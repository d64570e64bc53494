// Internal launch interface between the C ABI (cd_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cdk {

enum Variant { kMono = 0, kDualIdeal = 1, kDualPred = 2, kDense = 3, kCats = 4, kDualTern = 5 };

// Arguments of the coefficient kernels: dense coefficient projection,
// threshold, and (mono / pred) the gathered gate (mono) or gate+up (pred)
// rows of the active neurons. One wave per neuron.
struct CoefArgs {
    const uint16_t *x;   // [nb][d_model] bf16
    int nb;              // tokens in this call
    const uint16_t *Wg;  // [d_ff][d_model]
    const uint16_t *Wu;  // [d_ff][d_model]
    const uint16_t *Bt;  // [d_ff][d_rank] (pred only)
    const float *lat;    // [nb][d_rank] fp32 latent (pred only)
    const uint32_t *Tp;  // packed ternary predictor (tern only)
    int d_model, d_ff, d_rank;
    float thld;
    int *act;            // [d_ff] 1 if the neuron is in IDX
    float *s;            // [nb][d_ff] s of the active neurons (others untouched)
    float *coef;         // optional [nb][d_ff] dense coefficient vector
    float *y;            // [nb][d_model], zeroed here for the down kernel
};

struct DownArgs {
    const int *act;      // [d_ff]
    const float *s;      // [nb][d_ff]
    int nb;
    const uint16_t *Wd;  // [d_ff][d_model]
    int d_model, d_ff;
    int gc, gr;          // column chunks x neuron ranges (set by launch_down)
    int rows_per_group;  // ceil(d_ff / gr)
    float *y;            // [nb][d_model], accumulated (or written from part)
    float *part;         // [gr][nb][d_model] per-range partial sums, summed into y in
                         // ascending range order by a second kernel (bit-reproducible
                         // y); NULL: each range adds into y with fp32 atomics
};

// Residual stream between stacked layers (not part of the paper's method):
// h_out = h_in + y_prev, x_out = bf16(h_out / sqrt(mean(h_out^2) + eps)).
struct NormArgs {
    const float *h_in;    // [nb][d_model]
    const float *y_prev;  // [nb][d_model] or NULL (no residual add)
    float *h_out;         // [nb][d_model], distinct from h_in
    uint16_t *x_out;      // [nb][d_model] bf16
    int nb, d_model;
    float eps;
};

// 32-bit words of the packed ternary predictor per neuron row
int tern_row_words(int d_model);

// Smallest supported template widths for a call.
int batch_tile(int B);        // 1, 2, 4 or 8
int col_tile(int d_model);    // chunks of 512 columns: 1, 2, 4, 8 or 16
size_t down_lds_bytes(int rows_per_group, int bt);

hipError_t launch_coef(int variant, const CoefArgs &a, hipStream_t s);
hipError_t launch_latent(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                         float *lat, hipStream_t s);
hipError_t launch_down(const DownArgs &a, hipStream_t s);
// floats of DownArgs::part a call of batch tile bt needs at this shape
size_t down_part_floats(int d_model, int d_ff, int bt);
// x_out / h_out of the residual stream (one workgroup)
hipError_t launch_norm(const NormArgs &n, hipStream_t s);
// the same fused with the predictor latent: every workgroup normalises, the first writes
hipError_t launch_latent_norm(const NormArgs &n, const uint16_t *At, int d_rank, float *lat,
                              hipStream_t s);
// Flat ascending IDX / |IDX| / compact s from the per-neuron arrays (any output may be NULL).
hipError_t launch_export(const int *act, const float *s_rows, int nb, int d_ff, int *idx_dst,
                         int *n_dst, float *s_dst, hipStream_t s);
// Per-token threshold path after a dense coefficient kernel (a.coef holds
// [nb][d_ff]): q[b] = Quantile(k, c_b), then act / s of the neurons above
// their tokens' thresholds (gathering W_gate, or W_gate and W_up). For ideal
// D-CountDown the select sets act and s stays in a.coef. d_ff <= 32768.
hipError_t launch_topk(int variant, const CoefArgs &a, double k, double *q, hipStream_t s);
// Per-token ideal D-CountDown of one token: select, flags and down projection in
// one launch (after the coefficient kernel wrote the dense s to coef and zeroed y),
// when topk_down_fused(a) holds: one token, d_model <= 4096, d_ff <= 16384, no
// per-range partials (deterministic plans keep the separate kernels).
bool topk_down_fused(const DownArgs &a);
hipError_t launch_topk_down1(const DownArgs &a, const float *coef, int *act, double k,
                             double *q, hipStream_t s);
constexpr int kTopkMaxDff = 32768;
// Per-token linear-interpolation quantile of coef rows [T][ld] (n used entries).
hipError_t launch_select(const float *coef, int ld, int n, int T, int use_abs, double k,
                         double *q_out, hipStream_t s);
hipError_t launch_mean(const double *q, int T, float *out, hipStream_t s);
// Measurement aid: plain streaming read of bytes (a multiple of 16) at src.
hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *sink, hipStream_t s);

} // namespace cdk
