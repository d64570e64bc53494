// gfx950 kernels of the COUNTDOWN sparse Gated-MLP FFN (arXiv 2505.17701).
//
// Path for one call (Sec. 3 Eq. 2-6, Sec. 4):
//   coefficient kernel: one workgroup per block of R neurons. It streams the
//     dense coefficient rows (W_up for M-CountDown, W_gate and W_up for ideal
//     D-CountDown, B_t for the predictor), thresholds the coefficient of every
//     neuron (union over the batch), compacts the active neurons of the block
//     in ascending order with one wave ballot, then reads the W_gate (mono)
//     or W_gate and W_up (pred) rows of just those neurons and forms
//     s = u * SiLU(g). It writes the block's active count and its (neuron, s)
//     list, and zeroes y for the next kernel.
//   down kernel: every workgroup scans the per-block counts in LDS, takes a
//     contiguous range of active positions and one 512-column chunk,
//     accumulates s * W_down[i, chunk] over its rows in fp32 and adds the
//     result into y with fp32 atomics. Column-chunk-0 workgroups also write
//     the flat ascending IDX and the compact s.
// Rows are read as 16-byte chunks, 64 lanes x 16 B = one contiguous 1 KB
// segment per wave instruction. x is staged once per workgroup in LDS.
#include "cd_device.hpp"
#include "cd_internal.hpp"

namespace cdk {

// x (bf16) -> LDS as packed pairs, each token padded with zeros to NK*512 columns
template <int B, int NK>
__device__ __forceinline__ void stage_x(uint32_t *xs, const uint16_t *__restrict__ x, int nb,
                                        int d_model)
{
    constexpr int kCols = NK * kColsPerLoad;
    constexpr int kChunksPerTok = kCols / 8;
    for (int c = threadIdx.x; c < B * kChunksPerTok; c += kBlock) {
        const int b = c / kChunksPerTok;
        const int col = (c % kChunksPerTok) * 8;
        u32x4 v = zero16();
        if (b < nb && col < d_model)
            v = load16(x + (size_t)b * d_model + col);
        *reinterpret_cast<u32x4 *>(xs + (size_t)b * (kCols / 2) + col / 2) = v;
    }
}

template <int NK>
__device__ __forceinline__ void load_row(u32x4 (&w)[NK], const uint16_t *__restrict__ row,
                                         int d_model, int lane)
{
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int col = k * kColsPerLoad + lane * 8;
        w[k] = (col < d_model) ? load16(row + col) : zero16();
    }
}

// per-lane partial dot products of one row chunk set with the B staged tokens
template <int B, int NK>
__device__ __forceinline__ void dot_row(const u32x4 (&w)[NK], const uint32_t *xs, int lane,
                                        float (&acc)[B])
{
    constexpr int kStride = NK * kColsPerLoad / 2;
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int c2 = (k * kColsPerLoad + lane * 8) / 2;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const u32x4 xv = *reinterpret_cast<const u32x4 *>(xs + b * kStride + c2);
            acc[b] = dot8(w[k], xv, acc[b]);
        }
    }
}

__device__ __forceinline__ void zero_y(float *y, int n)
{
    for (int i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock)
        y[i] = 0.0f;
}

// Wave 0 turns the per-row flags of the block into the ascending list of
// active local rows (spos) and publishes the count.
__device__ __forceinline__ void compact_local(const int *sflag, int R, int *spos, int *snact,
                                              int *cnt_out)
{
    if (threadIdx.x < kWave) {
        const int lane = threadIdx.x;
        const bool f = lane < R && sflag[lane] != 0;
        const uint64_t m = ballot(f);
        if (f)
            spos[lanes_below(m)] = lane;
        if (lane == 0) {
            const int n = __popcll(m);
            *snact = n;
            *cnt_out = n;
        }
    }
}

// rows of one wave loop iteration, sized so that ~16 KB per wave are in flight
template <int NK, int MATS>
constexpr int rows_per_iter()
{
    return (NK * MATS >= 16) ? 1 : (NK * MATS >= 8 ? 2 : 4);
}

// Gather phase shared by mono and pred: for the nact active local rows (spos)
// read the W_gate row (and the W_up row when UP) and form s = u * SiLU(g),
// with u from su when !UP. Writes slot lists.
template <int B, int NK, bool UP>
__device__ __forceinline__ void gather_gate(const CoefArgs &a, const uint32_t *xs, int row0,
                                            const int *spos, int nact, const float (*su)[kMaxRowsPerBlock],
                                            int wave, int lane)
{
    constexpr int RPI = rows_per_iter<NK, UP ? 2 : 1>();
    for (int j0 = wave; j0 < nact; j0 += kWavesPerBlock * RPI) {
        u32x4 wg[RPI][NK];
        u32x4 wu[UP ? RPI : 1][UP ? NK : 1];
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int j = j0 + q * kWavesPerBlock;
            if (j < nact) {
                const size_t off = (size_t)(row0 + spos[j]) * a.d_model;
                load_row<NK>(wg[q], a.Wg + off, a.d_model, lane);
                if constexpr (UP)
                    load_row<NK>(wu[q], a.Wu + off, a.d_model, lane);
            }
        }
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int j = j0 + q * kWavesPerBlock;
            if (j >= nact)
                continue;
            const int lr = spos[j];
            const int slot = blockIdx.x * a.R + j;
            float ag[B], au[B];
#pragma unroll
            for (int b = 0; b < B; ++b) {
                ag[b] = 0.0f;
                au[b] = 0.0f;
            }
            dot_row<B, NK>(wg[q], xs, lane, ag);
            if constexpr (UP)
                dot_row<B, NK>(wu[q], xs, lane, au);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const float g = wave_sum(ag[b]);
                float u;
                if constexpr (UP)
                    u = wave_sum(au[b]);
                else
                    u = su[b][lr];
                if (b < a.nb && lane == 0)
                    a.ls[(size_t)b * a.ls_stride + slot] = u * silu(g);
            }
            if (lane == 0)
                a.lidx[slot] = row0 + lr;
        }
    }
}

// M-CountDown coefficient kernel (Eq. 6b): u = x.W_up, |u| > thld, then gate.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_coef_mono(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ float su[B][kMaxRowsPerBlock];
    __shared__ int sflag[kMaxRowsPerBlock];
    __shared__ int spos[kMaxRowsPerBlock];
    __shared__ int snact;
    constexpr int RPI = rows_per_iter<NK, 1>();
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row0 = blockIdx.x * a.R;

    zero_y(a.y, a.nb * a.d_model);
    stage_x<B, NK>(xs, a.x, a.nb, a.d_model);
    __syncthreads();

    for (int base = wave; base < a.R; base += kWavesPerBlock * RPI) {
        u32x4 w[RPI][NK];
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int lr = base + q * kWavesPerBlock, row = row0 + lr;
            if (lr < a.R && row < a.d_ff)
                load_row<NK>(w[q], a.Wu + (size_t)row * a.d_model, a.d_model, lane);
        }
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int lr = base + q * kWavesPerBlock, row = row0 + lr;
            if (lr >= a.R)
                continue;
            bool act = false;
            if (row < a.d_ff) {
                float acc[B];
#pragma unroll
                for (int b = 0; b < B; ++b)
                    acc[b] = 0.0f;
                dot_row<B, NK>(w[q], xs, lane, acc);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const float u = wave_sum(acc[b]);
                    if (b < a.nb) {
                        act = act || (fabsf(u) > a.thld);
                        if (lane == 0) {
                            su[b][lr] = u;
                            if (a.coef)
                                a.coef[(size_t)b * a.d_ff + row] = u;
                        }
                    }
                }
            }
            if (lane == 0)
                sflag[lr] = act ? 1 : 0;
        }
    }
    __syncthreads();
    compact_local(sflag, a.R, spos, &snact, a.cnt + blockIdx.x);
    __syncthreads();
    gather_gate<B, NK, false>(a, xs, row0, spos, snact, su, wave, lane);
}

// Ideal D-CountDown coefficient kernel (Eq. 6c): s = (x.W_up) * SiLU(x.W_gate)
// over all rows, |s| > thld. DENSE keeps every row (Eq. 1).
template <int B, int NK, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_coef_dual(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ float ss[B][kMaxRowsPerBlock];
    __shared__ int sflag[kMaxRowsPerBlock];
    __shared__ int spos[kMaxRowsPerBlock];
    __shared__ int snact;
    constexpr int RPI = rows_per_iter<NK, 2>();
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row0 = blockIdx.x * a.R;

    zero_y(a.y, a.nb * a.d_model);
    stage_x<B, NK>(xs, a.x, a.nb, a.d_model);
    __syncthreads();

    for (int base = wave; base < a.R; base += kWavesPerBlock * RPI) {
        u32x4 wg[RPI][NK], wu[RPI][NK];
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int lr = base + q * kWavesPerBlock, row = row0 + lr;
            if (lr < a.R && row < a.d_ff) {
                load_row<NK>(wg[q], a.Wg + (size_t)row * a.d_model, a.d_model, lane);
                load_row<NK>(wu[q], a.Wu + (size_t)row * a.d_model, a.d_model, lane);
            }
        }
#pragma unroll
        for (int q = 0; q < RPI; ++q) {
            const int lr = base + q * kWavesPerBlock, row = row0 + lr;
            if (lr >= a.R)
                continue;
            bool act = false;
            if (row < a.d_ff) {
                float ag[B], au[B];
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    ag[b] = 0.0f;
                    au[b] = 0.0f;
                }
                dot_row<B, NK>(wg[q], xs, lane, ag);
                dot_row<B, NK>(wu[q], xs, lane, au);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const float g = wave_sum(ag[b]);
                    const float u = wave_sum(au[b]);
                    const float s = u * silu(g);
                    if (b < a.nb) {
                        act = act || DENSE || (fabsf(s) > a.thld);
                        if (lane == 0) {
                            ss[b][lr] = s;
                            if (a.coef)
                                a.coef[(size_t)b * a.d_ff + row] = s;
                        }
                    }
                }
            }
            if (lane == 0)
                sflag[lr] = act ? 1 : 0;
        }
    }
    __syncthreads();
    compact_local(sflag, a.R, spos, &snact, a.cnt + blockIdx.x);
    __syncthreads();
    const int nact = snact;
    for (int j = threadIdx.x; j < nact; j += kBlock) {
        const int lr = spos[j];
        const int slot = blockIdx.x * a.R + j;
        a.lidx[slot] = row0 + lr;
        for (int b = 0; b < a.nb; ++b)
            a.ls[(size_t)b * a.ls_stride + slot] = ss[b][lr];
    }
}

// Predictor scores s_hat = latent . B_t[row] for the block's rows, with
// 2^LOG lanes per B_t row (64 >> LOG rows per wave instruction); sets the
// signed-threshold flags (union over the batch).
template <int B, int LOG>
__device__ __forceinline__ void score_rows(const CoefArgs &a, const float *lat_s, int row0,
                                           int *sflag, int wave, int lane)
{
    constexpr int LPR = 1 << LOG;
    constexpr int RW = kWave / LPR;
    const int nch = a.d_rank > kColsPerLoad ? a.d_rank / kColsPerLoad : 1;
    const int sub = lane / LPR;
    const int e0 = (lane % LPR) * 8;
    const bool last = (lane % LPR) == LPR - 1;
    for (int base = wave * RW; base < a.R; base += kWavesPerBlock * RW) {
        const int lr = base + sub, row = row0 + lr;
        const bool ok = lr < a.R && row < a.d_ff;
        float acc[B];
#pragma unroll
        for (int b = 0; b < B; ++b)
            acc[b] = 0.0f;
        for (int ch = 0; ch < nch; ++ch) {
            const int e = ch * kColsPerLoad + e0;
            const u32x4 w = ok ? load16(a.Bt + (size_t)row * a.d_rank + e) : zero16();
            const float wf[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                                 bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const float *l = lat_s + b * a.d_rank + e;
#pragma unroll
                for (int t = 0; t < 8; ++t)
                    acc[b] = fmaf(wf[t], l[t], acc[b]);
            }
        }
        bool act = false;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const float v = segment_sum<LOG>(acc[b]);
            if (b < a.nb && ok) {
                act = act || (v > a.thld);
                if (last && a.coef)
                    a.coef[(size_t)b * a.d_ff + row] = v;
            }
        }
        if (last && lr < a.R)
            sflag[lr] = (ok && act) ? 1 : 0;
    }
}

// Practical D-CountDown coefficient kernel (Sec. 4): predictor score, signed
// threshold, then gate and up rows of the active neurons.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_coef_pred(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ int sflag[kMaxRowsPerBlock];
    __shared__ int spos[kMaxRowsPerBlock];
    __shared__ int snact;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row0 = blockIdx.x * a.R;
    float *lat_s = reinterpret_cast<float *>(xs + B * NK * kColsPerLoad / 2);

    zero_y(a.y, a.nb * a.d_model);
    stage_x<B, NK>(xs, a.x, a.nb, a.d_model);
    for (int i = threadIdx.x; i < B * a.d_rank; i += kBlock)
        lat_s[i] = (i / a.d_rank) < a.nb ? a.lat[i] : 0.0f;
    __syncthreads();

    switch (a.d_rank) {
    case 8: score_rows<B, 0>(a, lat_s, row0, sflag, wave, lane); break;
    case 16: score_rows<B, 1>(a, lat_s, row0, sflag, wave, lane); break;
    case 32: score_rows<B, 2>(a, lat_s, row0, sflag, wave, lane); break;
    case 64: score_rows<B, 3>(a, lat_s, row0, sflag, wave, lane); break;
    case 128: score_rows<B, 4>(a, lat_s, row0, sflag, wave, lane); break;
    case 256: score_rows<B, 5>(a, lat_s, row0, sflag, wave, lane); break;
    default: score_rows<B, 6>(a, lat_s, row0, sflag, wave, lane); break;  // 512, 1024
    }
    __syncthreads();
    compact_local(sflag, a.R, spos, &snact, a.cnt + blockIdx.x);
    __syncthreads();
    gather_gate<B, NK, true>(a, xs, row0, spos, snact, nullptr, wave, lane);
}

// latent = x . theta_A for the predictor: one row of A_t per wave iteration
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_latent(const uint16_t *__restrict__ x, int nb,
                                                   const uint16_t *__restrict__ At, int d_model,
                                                   int d_rank, float *__restrict__ lat)
{
    extern __shared__ __align__(16) uint32_t xs[];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    stage_x<B, NK>(xs, x, nb, d_model);
    __syncthreads();
    const int r = blockIdx.x * kWavesPerBlock + wave;
    if (r >= d_rank)
        return;
    u32x4 w[NK];
    load_row<NK>(w, At + (size_t)r * d_model, d_model, lane);
    float acc[B];
#pragma unroll
    for (int b = 0; b < B; ++b)
        acc[b] = 0.0f;
    dot_row<B, NK>(w, xs, lane, acc);
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float v = wave_sum(acc[b]);
        if (b < nb && lane == 0)
            lat[(size_t)b * d_rank + r] = v;
    }
}

// exclusive scan of cnt[0..n) into pre[0..n]; pre[n] = total (256 threads)
__device__ __forceinline__ void block_scan_counts(const int *__restrict__ cnt, int n, int *pre,
                                                  int *part)
{
    const int t = threadIdx.x;
    const int per = (n + kBlock - 1) / kBlock;
    const int lo = min(n, t * per), hi = min(n, lo + per);
    int sum = 0;
    for (int i = lo; i < hi; ++i)
        sum += cnt[i];
    part[t] = sum;
    __syncthreads();
    for (int off = 1; off < kBlock; off <<= 1) {
        const int v = t >= off ? part[t - off] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    int run = part[t] - sum;  // exclusive prefix of this thread's segment
    for (int i = lo; i < hi; ++i) {
        pre[i] = run;
        run += cnt[i];
    }
    if (t == kBlock - 1)
        pre[n] = part[t];
    __syncthreads();
}

// largest blk in [0, n) with pre[blk] <= p (pre ascending, pre[0] = 0 <= p)
__device__ __forceinline__ int find_block(const int *pre, int n, int p, int top)
{
    int lo = 0;
    for (int step = top; step > 0; step >>= 1) {
        const int cand = lo + step;
        if (cand < n && pre[cand] <= p)
            lo = cand;
    }
    return lo;
}

// Gathered down projection (Eq. 5): y_b += sum_{p in range} s_b[p] W_down[IDX[p], chunk]
template <int B>
__global__ __launch_bounds__(kBlock) void k_down(const DownArgs a)
{
    extern __shared__ __align__(16) int dsm[];
    __shared__ int part[kBlock];
    constexpr int U = 4;  // rows in flight per wave
    int *pre = dsm;                                                  // nblk + 1
    float *red = reinterpret_cast<float *>(dsm + ((a.nblk + 4) & ~3)); // [4][512]
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;

    block_scan_counts(a.cnt, a.nblk, pre, part);
    const int n = pre[a.nblk];
    if (blockIdx.x == 0 && threadIdx.x == 0)
        *a.n_out = n;

    const int c = blockIdx.x % a.gc, g = blockIdx.x / a.gc;
    const int p_begin = (int)(((long long)n * g) / a.gr);
    const int p_end = (int)(((long long)n * (g + 1)) / a.gr);
    if (p_begin >= p_end)
        return;  // uniform for the workgroup
    const int col = c * kColsPerLoad + lane * 8;
    const bool colok = col < a.d_model;
    int top = 1;
    while (top * 2 < a.nblk)
        top <<= 1;

    float acc[B][8];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            acc[b][e] = 0.0f;

    for (int p0 = p_begin + wave; p0 < p_end; p0 += kWavesPerBlock * U) {
        int row[U];
        float s[U][B];
        u32x4 w[U];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int p = p0 + q * kWavesPerBlock;
            row[q] = 0;
#pragma unroll
            for (int b = 0; b < B; ++b)
                s[q][b] = 0.0f;
            if (p < p_end) {
                const int blk = find_block(pre, a.nblk, p, top);
                const int slot = blk * a.R + (p - pre[blk]);
                row[q] = a.lidx[slot];
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (b < a.nb)
                        s[q][b] = a.ls[(size_t)b * a.ls_stride + slot];
            }
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int p = p0 + q * kWavesPerBlock;
            w[q] = (p < p_end && colok) ? load16(a.Wd + (size_t)row[q] * a.d_model + col) : zero16();
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const float wf[8] = {bf16_lo(w[q].x), bf16_hi(w[q].x), bf16_lo(w[q].y), bf16_hi(w[q].y),
                                 bf16_lo(w[q].z), bf16_hi(w[q].z), bf16_lo(w[q].w), bf16_hi(w[q].w)};
#pragma unroll
            for (int b = 0; b < B; ++b)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc[b][e] = fmaf(s[q][b], wf[e], acc[b][e]);
            const int p = p0 + q * kWavesPerBlock;
            if (c == 0 && lane == 0 && p < p_end) {
                a.idx_out[p] = row[q];
#pragma unroll
                for (int b = 0; b < B; ++b)
                    if (b < a.nb)
                        a.s_out[(size_t)b * a.d_ff + p] = s[q][b];
            }
        }
    }

    // reduce the four waves' partials in LDS, then one atomic add per column
#pragma unroll
    for (int b = 0; b < B; ++b) {
        if (b >= a.nb)
            break;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < 8; ++e)
            red[wave * kColsPerLoad + lane * 8 + e] = acc[b][e];
        __syncthreads();
        for (int cc = threadIdx.x; cc < kColsPerLoad; cc += kBlock) {
            const int gcol = c * kColsPerLoad + cc;
            if (gcol < a.d_model) {
                const float v = red[cc] + red[kColsPerLoad + cc] + red[2 * kColsPerLoad + cc] +
                                red[3 * kColsPerLoad + cc];
                unsafeAtomicAdd(a.y + (size_t)b * a.d_model + gcol, v);
            }
        }
    }
}

// ------------------------------------------------------------- calibration

// order-preserving uint32 key of a float (|v| when use_abs)
__device__ __forceinline__ uint32_t order_key(float v, int use_abs)
{
    uint32_t u = __float_as_uint(v);
    if (use_abs)
        return u & 0x7fffffffu;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t k, int use_abs)
{
    if (use_abs)
        return __uint_as_float(k);
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

constexpr int kSelThreads = 1024;

// key of rank r (0-based, ascending) among keys[0..n): 4 passes of 8-bit radix select
__device__ uint32_t radix_select(const uint32_t *keys, int n, int r, int *hist, int *sh)
{
    uint32_t prefix = 0, mask = 0;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = threadIdx.x; i < 256; i += kSelThreads)
            hist[i] = 0;
        __syncthreads();
        for (int i = threadIdx.x; i < n; i += kSelThreads) {
            const uint32_t k = keys[i];
            if ((k & mask) == prefix)
                atomicAdd(&hist[(k >> shift) & 0xffu], 1);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            int cum = 0, bin = 0;
            for (; bin < 256; ++bin) {
                if (cum + hist[bin] > r)
                    break;
                cum += hist[bin];
            }
            sh[0] = bin;
            sh[1] = r - cum;
        }
        __syncthreads();
        prefix |= (uint32_t)sh[0] << shift;
        mask |= 0xffu << shift;
        r = sh[1];
        __syncthreads();
    }
    return prefix;
}

// One workgroup per token: q[t] = v[lo] + (h - lo)(v[lo+1] - v[lo]), h = k (n - 1)
__global__ __launch_bounds__(kSelThreads) void k_select_quantile(const float *__restrict__ coef,
                                                                int ld, int n, int use_abs,
                                                                double k, double *__restrict__ q)
{
    extern __shared__ uint32_t keys[];
    __shared__ int hist[256];
    __shared__ int sh[2];
    const float *c = coef + (size_t)blockIdx.x * ld;
    for (int i = threadIdx.x; i < n; i += kSelThreads)
        keys[i] = order_key(c[i], use_abs);
    __syncthreads();
    const double h = k * (double)(n - 1);
    int lo = (int)floor(h);
    if (lo > n - 1)
        lo = n - 1;
    const uint32_t k0 = radix_select(keys, n, lo, hist, sh);
    double v0 = (double)key_value(k0, use_abs);
    double v1 = v0;
    if (lo + 1 < n)
        v1 = (double)key_value(radix_select(keys, n, lo + 1, hist, sh), use_abs);
    if (threadIdx.x == 0)
        q[blockIdx.x] = v0 + (h - (double)lo) * (v1 - v0);
}

__global__ void k_mean(const double *__restrict__ q, int T, float *__restrict__ out)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double s = 0.0;
        for (int t = 0; t < T; ++t)
            s += q[t];
        *out = (float)(s / (double)T);
    }
}

// ------------------------------------------------------------------ launchers

// kernels staging more than 64 KB in LDS opt in to the larger gfx950 limit
template <class K>
static void allow_lds(K kernel, size_t bytes)
{
    if (bytes > 65536)
        (void)hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

int batch_tile(int B) { return B <= 1 ? 1 : B <= 2 ? 2 : B <= 4 ? 4 : 8; }

int col_tile(int d_model)
{
    const int chunks = (d_model + kColsPerLoad - 1) / kColsPerLoad;
    return chunks <= 1 ? 1 : chunks <= 2 ? 2 : chunks <= 4 ? 4 : chunks <= 8 ? 8 : 16;
}

size_t coef_lds_bytes(int variant, int bt, int nk, int d_rank)
{
    size_t b = (size_t)bt * nk * kColsPerLoad * 2;
    if (variant == kDualPred)
        b += (size_t)bt * d_rank * 4;
    return b;
}

size_t down_lds_bytes(int nblk)
{
    return (size_t)((nblk + 4) & ~3) * 4 + (size_t)kWavesPerBlock * kColsPerLoad * 4;
}

template <int B, int NK>
static hipError_t coef_bn(int variant, const CoefArgs &a, int grid, hipStream_t s)
{
    const size_t lds = coef_lds_bytes(variant, B, NK, a.d_rank);
    switch (variant) {
    case kMono:
        allow_lds(k_coef_mono<B, NK>, lds);
        k_coef_mono<B, NK><<<grid, kBlock, lds, s>>>(a);
        break;
    case kDualIdeal:
        allow_lds(k_coef_dual<B, NK, false>, lds);
        k_coef_dual<B, NK, false><<<grid, kBlock, lds, s>>>(a);
        break;
    case kDense:
        allow_lds(k_coef_dual<B, NK, true>, lds);
        k_coef_dual<B, NK, true><<<grid, kBlock, lds, s>>>(a);
        break;
    case kDualPred:
        allow_lds(k_coef_pred<B, NK>, lds);
        k_coef_pred<B, NK><<<grid, kBlock, lds, s>>>(a);
        break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int B>
static hipError_t coef_b(int variant, const CoefArgs &a, int grid, hipStream_t s)
{
    switch (col_tile(a.d_model)) {
    case 1: return coef_bn<B, 1>(variant, a, grid, s);
    case 2: return coef_bn<B, 2>(variant, a, grid, s);
    case 4: return coef_bn<B, 4>(variant, a, grid, s);
    case 8: return coef_bn<B, 8>(variant, a, grid, s);
    default:
        // B * d_model is capped at 32768 by the plan checks: no 8 x 8192 tile
        if constexpr (B * 16 <= 64)
            return coef_bn<B, 16>(variant, a, grid, s);
        return hipErrorInvalidValue;
    }
}

hipError_t launch_coef(int variant, const CoefArgs &a, int grid, hipStream_t s)
{
    switch (batch_tile(a.nb)) {
    case 1: return coef_b<1>(variant, a, grid, s);
    case 2: return coef_b<2>(variant, a, grid, s);
    case 4: return coef_b<4>(variant, a, grid, s);
    default: return coef_b<8>(variant, a, grid, s);
    }
}

template <int B, int NK>
static hipError_t latent_bn(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                            float *lat, hipStream_t s)
{
    const int grid = (d_rank + kWavesPerBlock - 1) / kWavesPerBlock;
    const size_t lds = (size_t)B * NK * kColsPerLoad * 2;
    allow_lds(k_latent<B, NK>, lds);
    k_latent<B, NK><<<grid, kBlock, lds, s>>>(x, nb, At, d_model, d_rank, lat);
    return hipGetLastError();
}

template <int B>
static hipError_t latent_b(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                           float *lat, hipStream_t s)
{
    switch (col_tile(d_model)) {
    case 1: return latent_bn<B, 1>(x, nb, At, d_model, d_rank, lat, s);
    case 2: return latent_bn<B, 2>(x, nb, At, d_model, d_rank, lat, s);
    case 4: return latent_bn<B, 4>(x, nb, At, d_model, d_rank, lat, s);
    case 8: return latent_bn<B, 8>(x, nb, At, d_model, d_rank, lat, s);
    default:
        if constexpr (B * 16 <= 64)
            return latent_bn<B, 16>(x, nb, At, d_model, d_rank, lat, s);
        return hipErrorInvalidValue;
    }
}

hipError_t launch_latent(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                         float *lat, hipStream_t s)
{
    switch (batch_tile(nb)) {
    case 1: return latent_b<1>(x, nb, At, d_model, d_rank, lat, s);
    case 2: return latent_b<2>(x, nb, At, d_model, d_rank, lat, s);
    case 4: return latent_b<4>(x, nb, At, d_model, d_rank, lat, s);
    default: return latent_b<8>(x, nb, At, d_model, d_rank, lat, s);
    }
}

hipError_t launch_down(const DownArgs &a, hipStream_t s)
{
    const size_t lds = down_lds_bytes(a.nblk);
    const int grid = a.gc * a.gr;
    switch (batch_tile(a.nb)) {
    case 1: k_down<1><<<grid, kBlock, lds, s>>>(a); break;
    case 2: k_down<2><<<grid, kBlock, lds, s>>>(a); break;
    case 4: k_down<4><<<grid, kBlock, lds, s>>>(a); break;
    default: k_down<8><<<grid, kBlock, lds, s>>>(a); break;
    }
    return hipGetLastError();
}

hipError_t launch_select(const float *coef, int ld, int n, int T, int use_abs, double k,
                         double *q_out, hipStream_t s)
{
    allow_lds(k_select_quantile, (size_t)n * 4);
    k_select_quantile<<<T, kSelThreads, (size_t)n * 4, s>>>(coef, ld, n, use_abs, k, q_out);
    return hipGetLastError();
}

hipError_t launch_mean(const double *q, int T, float *out, hipStream_t s)
{
    k_mean<<<1, 64, 0, s>>>(q, T, out);
    return hipGetLastError();
}

} // namespace cdk
