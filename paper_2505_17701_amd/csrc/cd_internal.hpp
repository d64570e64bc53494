// Internal launch interface between the C ABI (cd_api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cdk {

enum Variant { kMono = 0, kDualIdeal = 1, kDualPred = 2, kDense = 3 };

// Arguments of the coefficient kernels: dense coefficient projection,
// threshold, per-block ordered compaction, and (mono / pred) the gathered
// gate (mono) or gate+up (pred) rows of the active neurons.
struct CoefArgs {
    const uint16_t *x;   // [nb][d_model] bf16
    int nb;              // tokens in this call
    const uint16_t *Wg;  // [d_ff][d_model]
    const uint16_t *Wu;  // [d_ff][d_model]
    const uint16_t *Bt;  // [d_ff][d_rank] (pred only)
    const float *lat;    // [nb][d_rank] fp32 latent (pred only)
    int d_model, d_ff, d_rank;
    int R;               // rows per workgroup (<= 64)
    float thld;
    int *cnt;            // [nblk] active rows per workgroup
    int *lidx;           // [nblk * R] neuron ids, slot blk * R + j
    float *ls;           // [nb][ls_stride] coefficient s of slot
    int ls_stride;
    float *coef;         // optional [nb][d_ff] dense coefficient vector
    float *y;            // [nb][d_model], zeroed here for the down kernel
};

struct DownArgs {
    const int *cnt;
    int nblk, R;
    const int *lidx;
    const float *ls;
    int ls_stride;
    int nb;
    const uint16_t *Wd;  // [d_ff][d_model]
    int d_model, d_ff;
    int gc, gr;          // column chunks x row groups (grid = gc * gr)
    float *y;            // [nb][d_model], accumulated
    int *idx_out;        // [d_ff] ascending IDX
    float *s_out;        // [nb][d_ff] compact s aligned with IDX
    int *n_out;          // [1]
};

// Smallest supported template widths for a call.
int batch_tile(int B);        // 1, 2, 4 or 8
int col_tile(int d_model);    // chunks of 512 columns: 1, 2, 4, 8 or 16
size_t coef_lds_bytes(int variant, int bt, int nk, int d_rank);
size_t down_lds_bytes(int nblk);

hipError_t launch_coef(int variant, const CoefArgs &a, int grid, hipStream_t s);
hipError_t launch_latent(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                         float *lat, hipStream_t s);
hipError_t launch_down(const DownArgs &a, hipStream_t s);
// Per-token linear-interpolation quantile of coef rows [T][ld] (n used entries).
hipError_t launch_select(const float *coef, int ld, int n, int T, int use_abs, double k,
                         double *q_out, hipStream_t s);
hipError_t launch_mean(const double *q, int T, float *out, hipStream_t s);

} // namespace cdk
