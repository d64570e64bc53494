// gfx950 kernels of the COUNTDOWN sparse Gated-MLP FFN (arXiv 2505.17701).
//
// One call (Sec. 3 Eq. 2-6, Sec. 4) runs two kernels (three with the predictor):
//   coefficient kernel, M-CountDown and ideal D-CountDown: one wave per
//     neuron. The wave streams the neuron's coefficient row(s) -- W_up, or
//     W_gate and W_up -- with non-temporal 16-byte loads (64 lanes x 16 B =
//     one contiguous 1 KB segment per instruction), takes the dot products
//     against x (registers for one token, and for two of d_model <= 4096 in
//     the two-row kernel; otherwise an LDS copy per workgroup) with
//     v_dot2_f32_bf16, reduces across the wave with DPP and applies the
//     strict threshold (union over the batch). For M-CountDown an active
//     neuron's wave immediately reads its W_gate row and forms s = u *
//     SiLU(g). Results land in per-neuron arrays act[d_ff] and s[B][d_ff];
//     there are no barriers between waves. The kernel also zeroes y.
//   predictor (practical D-CountDown): the latent x . theta_A (one workgroup
//     per A_t row), then a coefficient kernel over blocks of 32 neurons: B_t
//     scores, signed threshold, and the block's active neurons dealt to its
//     waves for the W_gate / W_up gather (v_dot2 up to 4 tokens, MFMA tiles
//     of 16 neurons with the rows staged through LDS for 5-8). The ternary
//     predictor scores from its 2-bit packed theta instead, with no latent.
//   down kernel: workgroup (c, g) owns a column chunk c and a contiguous
//     neuron range g. One round trip reads act and s of the range, a wave
//     ballot compacts the active neurons in ascending order into LDS; for 1-2
//     tokens each wave then keeps 16 W_down rows in flight on the VALU, for
//     4-8 the rows feed MFMA (S as bf16 hi + lo); partial sums are added in
//     LDS and go to y with one fp32 atomic per column and token.
//   per-token threshold: the coefficient kernel writes the dense
//     coefficients, one workgroup per token selects its quantile (one wide
//     radix pass, then the few keys of the two bins ranked by counting), a
//     gather kernel thresholds and gathers. A single token runs select,
//     flags and gather in one launch: every workgroup selects on its own and
//     gathers its slice, its rows loaded as soon as the select's first pass
//     bounds the active set.
// The residual stream of a layer stack (h += y, x = bf16(RMSNorm(h))) is a
// small kernel of its own, or part of the latent kernel with the predictor.
#include "cd_device.hpp"
#include "cd_internal.hpp"

namespace cdk {

// weight rows are read exactly once per call: non-temporal loads
__device__ __forceinline__ u32x4 load16_stream(const uint16_t *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}

// Lanes whose chunk lies past the end of a row (ragged d_model) or of the
// token batch load these 16 zero bytes instead: an address select before the
// load rather than a select of the loaded data, which would make the compiler
// wait for each load on its own.
__device__ __align__(16) uint32_t kZeroChunk[4] = {0u, 0u, 0u, 0u};  // never written

template <class T>
__device__ __forceinline__ const T *or_zero(bool ok, const T *p)
{
    return ok ? p : reinterpret_cast<const T *>(kZeroChunk);
}

template <int NK>
__device__ __forceinline__ void load_row(u32x4 (&w)[NK], const uint16_t *__restrict__ row,
                                         int d_model, int lane)
{
#pragma unroll
    for (int k = 0; k < NK; ++k) {
        const int col = k * kColsPerLoad + lane * 8;
        w[k] = load16_stream(or_zero(col < d_model, row + col));
    }
}

// Token operand of the dot products: registers (XREG) or the LDS copy.
template <int B, int NK, bool XREG>
struct Tokens {
    static constexpr int kCols = NK * kColsPerLoad;
    static constexpr int kChunksPerTok = kCols / 8;
    static constexpr int kTotal = B * kChunksPerTok;  // 16-byte chunks of the LDS copy
    static constexpr int kIter = XREG ? 1 : (kTotal + kBlock - 1) / kBlock;
    u32x4 r[XREG ? B : 1][XREG ? NK : 1];
    u32x4 stage[kIter];  // LDS path: this thread's share of the copy, in flight
    const uint32_t *lds;

    // Issue every global load of the tokens (this lane's chunks, or this
    // thread's share of the LDS copy, padded with zeros to NK * 512 columns).
    // A scheduling barrier keeps the loads ahead of whatever follows.
    __device__ __forceinline__ void issue(const uint16_t *__restrict__ x, int nb, int d_model,
                                          int lane)
    {
        if constexpr (XREG) {
#pragma unroll
            for (int b = 0; b < B; ++b)
#pragma unroll
                for (int k = 0; k < NK; ++k) {
                    const int col = k * kColsPerLoad + lane * 8;
                    r[b][k] = load16(or_zero(b < nb && col < d_model, x + (size_t)b * d_model + col));
                }
        } else {
#pragma unroll
            for (int i = 0; i < kIter; ++i) {
                const int c = threadIdx.x + i * kBlock;
                const int b = c / kChunksPerTok;
                const int col = (c % kChunksPerTok) * 8;
                stage[i] = load16(or_zero(c < kTotal && b < nb && col < d_model,
                                          x + (size_t)b * d_model + col));
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }

    // LDS path: write this thread's share of the copy to smem (the caller
    // synchronises the workgroup before reading it). Register path: nothing.
    __device__ __forceinline__ void write(uint32_t *smem)
    {
        if constexpr (!XREG) {
#pragma unroll
            for (int i = 0; i < kIter; ++i) {
                const int c = threadIdx.x + i * kBlock;
                if (c < kTotal)
                    *reinterpret_cast<u32x4 *>(smem + (size_t)(c / kChunksPerTok) * (kCols / 2) +
                                               (c % kChunksPerTok) * 4) = stage[i];
            }
            lds = smem;
        }
    }

    // write() and a workgroup barrier on the LDS path (every thread must call this)
    __device__ __forceinline__ void commit(uint32_t *smem)
    {
        if constexpr (!XREG) {
            write(smem);
            __syncthreads();
        }
    }

    // Address of this lane's 16 bytes of token b, chunk k, in the LDS copy. The
    // offset goes through an empty asm so that a second pass over the tokens
    // reads LDS again instead of keeping B x NK chunks alive in registers.
    __device__ __forceinline__ const u32x4 *lds_chunk(int b, int k, int lane, int off) const
    {
        constexpr int kStride = NK * kColsPerLoad / 2;
        return reinterpret_cast<const u32x4 *>(lds + off + b * kStride +
                                               (k * kColsPerLoad + lane * 8) / 2);
    }

    static __device__ __forceinline__ int opaque_zero()
    {
        int z = 0;
        asm volatile("" : "+s"(z));
        return z;
    }

    // Materialise the accumulators here: keeps the dot products of one chunk
    // from being deferred (with their token operands held live) past the next.
    static __device__ __forceinline__ void settle(float (&acc)[B])
    {
#pragma unroll
        for (int b = 0; b < B; ++b)
            asm volatile("" : "+v"(acc[b]));
    }

    // acc[b] += w . x_b over this lane's chunks
    __device__ __forceinline__ void dot(const u32x4 (&w)[NK], int lane, float (&acc)[B]) const
    {
        if constexpr (XREG) {
#pragma unroll
            for (int k = 0; k < NK; ++k)
#pragma unroll
                for (int b = 0; b < B; ++b)
                    acc[b] = dot8(w[k], r[b][k], acc[b]);
        } else {
            const int off = opaque_zero();
#pragma unroll
            for (int k = 0; k < NK; ++k) {
#pragma unroll
                for (int b = 0; b < B; ++b)
                    acc[b] = dot8(w[k], *lds_chunk(b, k, lane, off), acc[b]);
                settle(acc);
            }
        }
    }

    // ag[b] += wg . x_b and au[b] += wu . x_b, one read of each x chunk for both rows
    __device__ __forceinline__ void dot2(const u32x4 (&wg)[NK], const u32x4 (&wu)[NK], int lane,
                                         float (&ag)[B], float (&au)[B]) const
    {
        if constexpr (XREG) {
#pragma unroll
            for (int k = 0; k < NK; ++k)
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    ag[b] = dot8(wg[k], r[b][k], ag[b]);
                    au[b] = dot8(wu[k], r[b][k], au[b]);
                }
        } else {
            const int off = opaque_zero();
#pragma unroll
            for (int k = 0; k < NK; ++k) {
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const u32x4 xv = *lds_chunk(b, k, lane, off);
                    ag[b] = dot8(wg[k], xv, ag[b]);
                    au[b] = dot8(wu[k], xv, au[b]);
                }
                settle(ag);
                settle(au);
            }
        }
    }
};

__device__ __forceinline__ void zero_y(float *y, int n)
{
    for (int i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock)
        y[i] = 0.0f;
}

template <int B>
__device__ __forceinline__ void zero_acc(float (&acc)[B])
{
#pragma unroll
    for (int b = 0; b < B; ++b)
        acc[b] = 0.0f;
}

// Single-projection coefficient kernel. M-CountDown (Eq. 6b): u = x.W_up,
// |u| > thld, then the active neuron's W_gate row and s = u * SiLU(g) (Eq. 2
// restricted to IDX). CATS (Eq. 6a, the comparison method): h = SiLU(x.W_gate),
// |h| > thld, then the active neuron's W_up row and s = u * h. The stored
// coefficient is u (M) or h (CATS).
template <int B, int NK, bool XREG, bool CATS>
__global__ __launch_bounds__(kBlock) void k_coef_mono(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row = blockIdx.x * kWavesPerBlock + wave;
    const bool live = row < a.d_ff;
    const uint16_t *first = CATS ? a.Wg : a.Wu;   // the coefficient's projection
    const uint16_t *second = CATS ? a.Wu : a.Wg;  // gathered for the active neurons
    u32x4 w[NK];
    load_row<NK>(w, first + (size_t)(live ? row : 0) * a.d_model, a.d_model, lane);
    Tokens<B, NK, XREG> tok;
    tok.issue(a.x, a.nb, a.d_model, lane);
    zero_y(a.y, a.nb * a.d_model);
    tok.commit(xs);
    if (!live)
        return;

    float acc[B], c[B];
    zero_acc(acc);
    tok.dot(w, lane, acc);
    bool act = false;
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float p = wave_sum(acc[b]);
        c[b] = CATS ? silu(p) : p;
        if (b < a.nb) {
            act = act || (fabsf(c[b]) > a.thld);
            if (a.coef && lane == 0)
                a.coef[(size_t)b * a.d_ff + row] = c[b];
        }
    }
    if (act) {
        load_row<NK>(w, second + (size_t)row * a.d_model, a.d_model, lane);
        zero_acc(acc);
        tok.dot(w, lane, acc);
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const float p = wave_sum(acc[b]);
            if (b < a.nb && lane == 0)
                a.s[(size_t)b * a.d_ff + row] = CATS ? p * c[b] : c[b] * silu(p);
        }
    }
    if (lane == 0)
        a.act[row] = act ? 1 : 0;
}

// Ideal D-CountDown coefficient kernel (Eq. 6c): s = (x.W_up) * SiLU(x.W_gate)
// for every neuron, |s| > thld. DENSE keeps every neuron (Eq. 1).
template <int B, int NK, bool XREG, bool DENSE>
__global__ __launch_bounds__(kBlock) void k_coef_dual(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row = blockIdx.x * kWavesPerBlock + wave;
    const bool live = row < a.d_ff;
    u32x4 wg[NK], wu[NK];
    const size_t roff = (size_t)(live ? row : 0) * a.d_model;
    load_row<NK>(wg, a.Wg + roff, a.d_model, lane);
    load_row<NK>(wu, a.Wu + roff, a.d_model, lane);
    Tokens<B, NK, XREG> tok;
    tok.issue(a.x, a.nb, a.d_model, lane);
    zero_y(a.y, a.nb * a.d_model);
    tok.commit(xs);
    if (!live)
        return;

    float ag[B], au[B];
    zero_acc(ag);
    zero_acc(au);
    tok.dot2(wg, wu, lane, ag, au);
    bool act = DENSE;
    float s[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float g = wave_sum(ag[b]);
        const float u = wave_sum(au[b]);
        s[b] = u * silu(g);
        if (b < a.nb) {
            act = act || (fabsf(s[b]) > a.thld);
            if (a.coef && lane == 0)
                a.coef[(size_t)b * a.d_ff + row] = s[b];
        }
    }
    if (lane == 0) {
        if (act)
#pragma unroll
            for (int b = 0; b < B; ++b)
                if (b < a.nb)
                    a.s[(size_t)b * a.d_ff + row] = s[b];
        a.act[row] = act ? 1 : 0;
    }
}

constexpr int kPredRowsPerWave = 8;
constexpr int kPredRows = kPredRowsPerWave * kWavesPerBlock;  // neurons per workgroup

// The predictor latent [B][d_rank] fp32 on its way to LDS: the part a rank of up
// to 256 needs is loaded with the kernel's other loads (issue), written after
// (write); larger ranks take a second, plain pass. The caller synchronises.
template <int B>
struct LatentStage {
    static constexpr int kFast = (B * 256 / 4 + kBlock - 1) / kBlock;
    u32x4 v[kFast];  // 4 fp32 each, as raw bits

    __device__ __forceinline__ void issue(const float *lat, int nb, int d_rank)
    {
        const int q4 = d_rank / 4;
        const u32x4 *g = reinterpret_cast<const u32x4 *>(lat);
#pragma unroll
        for (int t = 0; t < kFast; ++t) {
            const int i = threadIdx.x + t * kBlock;
            v[t] = *or_zero(i < B * q4 && i / q4 < nb, g + i);
        }
    }

    __device__ __forceinline__ void write(u32x4 *dst, const float *lat, int nb, int d_rank) const
    {
        const int q4 = d_rank / 4;
        const u32x4 *g = reinterpret_cast<const u32x4 *>(lat);
#pragma unroll
        for (int t = 0; t < kFast; ++t) {
            const int i = threadIdx.x + t * kBlock;
            if (i < B * q4)
                dst[i] = v[t];
        }
        for (int i = threadIdx.x + kFast * kBlock; i < B * q4; i += kBlock)
            dst[i] = *or_zero(i / q4 < nb, g + i);
    }
};

// Shape of one wave's B_t work at rank d_rank = 8 << LCPR: its kPredRowsPerWave
// rows are one flat run of 16-byte chunks, chunk f on lane f % 64, kLoads per
// lane. A row is a segment of min(cpr, 64) lanes (summed by DPP) spread over
// kJpr consecutive loads when it is longer than 64 chunks.
template <int LCPR>
struct PredShape {
    static constexpr int kCpr = 1 << LCPR;  // 16-byte chunks per B_t row
    static constexpr int kLoads = kCpr * kPredRowsPerWave >= kWave ? kCpr * kPredRowsPerWave / kWave : 1;
    static constexpr int kJpr = kCpr > kWave ? kCpr / kWave : 1;
    static constexpr int kSegLog = LCPR < 6 ? LCPR : 6;
    static constexpr int kSeg = 1 << kSegLog;
};

template <int LCPR>
__device__ __forceinline__ void pred_issue_bt(u32x4 (&wb)[PredShape<LCPR>::kLoads],
                                              const CoefArgs &a, int wr0, int lane)
{
    using S = PredShape<LCPR>;
#pragma unroll
    for (int j = 0; j < S::kLoads; ++j) {
        const int f = j * kWave + lane;
        const int rw = f >> LCPR;
        wb[j] = zero16();
        if (rw < kPredRowsPerWave && wr0 + rw < a.d_ff)
            wb[j] = load16_stream(a.Bt + (size_t)(wr0 + rw) * a.d_rank + (f & (S::kCpr - 1)) * 8);
    }
}

// The latent entries a lane multiplies. Up to rank 512 a lane meets the same
// 8 entries of each token in every one of its B_t loads, so they are loaded
// once, from global memory, with the kernel's first loads; rank 1024 rows
// read the LDS copy instead.
template <int B, int LCPR>
struct LatentRegs {
    static constexpr bool kRegs = PredShape<LCPR>::kCpr <= kWave;
    u32x4 v[kRegs ? B : 1][2];  // 8 fp32 per token as raw bits

    __device__ __forceinline__ void issue(const float *lat, int nb, int d_rank, int lane)
    {
        if constexpr (kRegs) {
            const int e = (lane & (PredShape<LCPR>::kCpr - 1)) * 8;
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const u32x4 *p = reinterpret_cast<const u32x4 *>(lat + (size_t)b * d_rank + e);
                v[b][0] = *or_zero(b < nb, p);
                v[b][1] = *or_zero(b < nb, p + 1);
            }
        }
    }

    __device__ __forceinline__ float get(int b, int q) const
    {
        return __uint_as_float(v[b][q / 4][q % 4]);
    }
};

// s_hat_b = latent_b . B_t[row] for the wave's rows (latent from lr, or from
// the LDS copy lat for rank 1024), the signed threshold with the union over
// the batch, act[] and (optionally) the coefficients. Returns the
// wave-uniform mask of its active rows.
template <int B, int LCPR>
__device__ __forceinline__ uint32_t pred_score(const u32x4 (&wb)[PredShape<LCPR>::kLoads],
                                               const LatentRegs<B, LCPR> &lr, const float *lat,
                                               const CoefArgs &a, int wr0, int lane)
{
    using S = PredShape<LCPR>;
    const bool seg_end = (lane & (S::kSeg - 1)) == S::kSeg - 1;
    float acc[B];
    zero_acc(acc);
    uint32_t wmask = 0;
#pragma unroll
    for (int j = 0; j < S::kLoads; ++j) {
        const int f = j * kWave + lane;
        const int e = (f & (S::kCpr - 1)) * 8;
        const u32x4 w = wb[j];
        const float wf[8] = {bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y),
                             bf16_lo(w.z), bf16_hi(w.z), bf16_lo(w.w), bf16_hi(w.w)};
#pragma unroll
        for (int b = 0; b < B; ++b) {
            if (b < a.nb) {
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    acc[b] = fmaf(wf[q],
                                  LatentRegs<B, LCPR>::kRegs ? lr.get(b, q) : lat[b * a.d_rank + e + q],
                                  acc[b]);
            }
        }
        if ((j + 1) % S::kJpr != 0)
            continue;
        // the segment ends of this load close its rows
        const int rw = f >> LCPR;
        const int row = wr0 + rw;
        const bool live = seg_end && rw < kPredRowsPerWave && row < a.d_ff;
        bool act = false;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const float v = segment_sum<S::kSegLog>(acc[b]);
            acc[b] = 0.0f;
            if (b < a.nb) {
                act = act || (v > a.thld);
                if (a.coef && live)
                    a.coef[(size_t)b * a.d_ff + row] = v;
            }
        }
        if (live)
            a.act[row] = act ? 1 : 0;
        const uint64_t m = ballot(live && act);
#pragma unroll
        for (int i = 0; i < kWave / S::kSeg; ++i) {
            const int end = (i + 1) * S::kSeg - 1;        // lane of segment i's sum
            const int rwi = (j * kWave + end) >> LCPR;    // its row within the wave
            if (rwi < kPredRowsPerWave)
                wmask |= (uint32_t)((m >> end) & 1u) << rwi;
        }
    }
    return wmask;
}

// s = u * SiLU(g) of one active neuron from its W_gate and W_up rows
template <int B, int NK, bool XREG>
__device__ __forceinline__ void pred_finish(const CoefArgs &a, const Tokens<B, NK, XREG> &tok,
                                            const u32x4 (&wg)[NK], const u32x4 (&wu)[NK], int row,
                                            int lane)
{
    float ag[B], au[B];
    zero_acc(ag);
    zero_acc(au);
    tok.dot2(wg, wu, lane, ag, au);
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float g = wave_sum(ag[b]);
        const float u = wave_sum(au[b]);
        if (b < a.nb && lane == 0)
            a.s[(size_t)b * a.d_ff + row] = u * silu(g);
    }
}

// Next neuron of this wave's share of the block mask (every fourth active
// neuron), or -1; advances the mask past it.
template <int NW = kWavesPerBlock>
__device__ __forceinline__ int pred_next(uint32_t &m)
{
    if (!m)
        return -1;
    const int r = __builtin_ctz(m);
#pragma unroll
    for (int k = 0; k < NW; ++k)
        m &= m - 1;
    return r;
}

// This wave's share of the block's active neurons: the waves' masks are
// joined (one barrier) and every fourth active neuron, starting at number
// `wave`, is kept.
template <int NW = kWavesPerBlock>
__device__ __forceinline__ uint32_t block_share(uint32_t *wflag, uint32_t wmask, int wave, int lane)
{
    if (lane == 0 && wave < kWavesPerBlock)  // the scoring waves
        wflag[wave] = wmask;
    __syncthreads();
    uint32_t m = 0;
#pragma unroll
    for (int v = 0; v < kWavesPerBlock; ++v)
        m |= wflag[v] << (v * kPredRowsPerWave);
    for (int v = 0; v < wave; ++v)
        m &= m - 1;
    return m;
}

// Gather of the wave's share m of the block's active neurons (block base r0):
// W_gate and W_up rows, s = u * SiLU(g), the next neuron's rows in flight
// while the current one is reduced.
template <int B, int NK, bool XREG, int NW = kWavesPerBlock>
__device__ __forceinline__ void gather_rr(const CoefArgs &a, const Tokens<B, NK, XREG> &tok,
                                          uint32_t m, int r0, int lane)
{
    // the next neuron's W_gate + W_up rows in flight while the current one is
    // reduced, for 1-2 tokens; at 4 the second buffer cost occupancy (168 against
    // 100 VGPRs) and one buffer measured 1.5-4% faster (8B shape)
    constexpr bool kPrefetch = NK <= 8 && B <= 2;
    int ra = pred_next<NW>(m);
    if (ra < 0)
        return;
    u32x4 ga[NK], ua[NK];
    load_row<NK>(ga, a.Wg + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
    load_row<NK>(ua, a.Wu + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
    if constexpr (kPrefetch) {
        u32x4 gb[NK], ub[NK];
        for (;;) {
            const int rb = pred_next<NW>(m);
            if (rb >= 0) {
                load_row<NK>(gb, a.Wg + (size_t)(r0 + rb) * a.d_model, a.d_model, lane);
                load_row<NK>(ub, a.Wu + (size_t)(r0 + rb) * a.d_model, a.d_model, lane);
            }
            pred_finish<B, NK, XREG>(a, tok, ga, ua, r0 + ra, lane);
            if (rb < 0)
                break;
            ra = pred_next<NW>(m);
            if (ra >= 0) {
                load_row<NK>(ga, a.Wg + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
                load_row<NK>(ua, a.Wu + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
            }
            pred_finish<B, NK, XREG>(a, tok, gb, ub, r0 + rb, lane);
            if (ra < 0)
                break;
        }
    } else {
        for (;;) {
            pred_finish<B, NK, XREG>(a, tok, ga, ua, r0 + ra, lane);
            ra = pred_next<NW>(m);
            if (ra < 0)
                break;
            load_row<NK>(ga, a.Wg + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
            load_row<NK>(ua, a.Wu + (size_t)(r0 + ra) * a.d_model, a.d_model, lane);
        }
    }
}

// Practical D-CountDown coefficient kernel (Sec. 4). A workgroup owns a block
// of kPredRows neurons (kPredRowsPerWave per wave). One round of loads brings
// the wave's B_t rows, the tokens (registers for batches of 1-2, this
// thread's share of an LDS copy for 4-8) and the latent (staged in LDS).
// Each wave scores its rows (s_hat = latent . B_t[row], signed threshold,
// union over the batch); the block's active neurons are then dealt
// round-robin to the four waves, which gather their W_gate and W_up rows
// (for 1-2 tokens the next row's loads in flight while the current one is
// reduced) and write s = u * SiLU(g).
template <int B, int NK, bool XREG, int LCPR, int NWV = kWavesPerBlock>
__global__ __launch_bounds__(NWV * kWave) void k_coef_pred(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];  // [tokens [B][NK * 256]], latent [B][d_rank]
    __shared__ uint32_t wflag[kWavesPerBlock];
    using S = PredShape<LCPR>;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // NWV 8: the first four waves score the block's rows; the others score
    // nothing (their rows start past d_ff) and join the gather
    const bool scorer = NWV == kWavesPerBlock || wave < kWavesPerBlock;  // wave-uniform
    const int r0 = blockIdx.x * kPredRows;
    const int wr0 = scorer ? r0 + wave * kPredRowsPerWave : a.d_ff;

    // loads in the order they are needed: B_t and the latent for the scores,
    // then the tokens, which only the gather reads
    using LR = LatentRegs<B, LCPR>;
    u32x4 wb[S::kLoads];
    pred_issue_bt<LCPR>(wb, a, wr0, lane);
    LR lr;
    lr.issue(a.lat, a.nb, a.d_rank, lane);
    LatentStage<LR::kRegs ? 1 : B> ls;  // the LDS copy, rank 1024 only
    if constexpr (!LR::kRegs)
        if (scorer)
            ls.issue(a.lat, a.nb, a.d_rank);
    Tokens<B, NK, XREG> tok;
    if (XREG || scorer)  // the LDS copy: the first kBlock threads
        tok.issue(a.x, a.nb, a.d_model, lane);
    if (scorer)
        zero_y(a.y, a.nb * a.d_model);
    uint32_t *latw = xs + (XREG ? 0 : B * NK * kColsPerLoad / 2);
    if constexpr (!LR::kRegs) {
        if (scorer)
            ls.write(reinterpret_cast<u32x4 *>(latw), a.lat, a.nb, a.d_rank);
        __syncthreads();
    }

    const uint32_t wmask =
        scorer ? pred_score<B, LCPR>(wb, lr, reinterpret_cast<const float *>(latw), a, wr0, lane)
               : 0u;
    if (scorer)
        tok.write(xs);  // (block_share's barrier publishes the LDS copy)
    else
        tok.lds = xs;
    uint32_t m = block_share<NWV>(wflag, wmask, wave, lane);
    gather_rr<B, NK, XREG, NWV>(a, tok, m, r0, lane);
}

// ------------------------------------------- MFMA gather for batches of 5-8
// For 4-8 tokens the gathered products are small dense contractions: a tile
// of 16 active neurons times the batch, on v_mfma_f32_16x16x32_bf16. Lane
// l = i + 16 g (i = l % 16, g = l / 16) supplies row i of the tile (A operand)
// and token i of the batch (B operand, zero for i >= B), each with the 8
// columns 32 s + 8 g + [0, 8) of step s, so both operands use the same
// column order. The four waves take a quarter of the steps each and add
// their 16 x 16 partial sums in LDS; lane l holds D[4 (l / 16) + r][l % 16].

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kTile = 16;

__device__ __forceinline__ f32x4_t mfma16(const u32x4 &a, const u32x4 &b, f32x4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                    __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// LDS token rows for the MFMA kernel: a 16-byte pad per row keeps the 16
// tokens of one step on distinct banks; one zero chunk serves tokens >= B.
template <int NK>
struct MfmaTokLayout {
    static constexpr int kCols = NK * kColsPerLoad;
    static constexpr int kStride = kCols / 2 + 4;  // u32 per token row
};

template <int B, int NK>
__host__ __device__ constexpr size_t mfma_lds_tokens_u32()
{
    return (size_t)B * MfmaTokLayout<NK>::kStride + 4;
}

// The tokens of the MFMA kernels: every thread's share of the LDS copy is
// loaded with the kernel's first loads (issue) and written after (write);
// the caller synchronises the workgroup before the copy is read.
template <int B, int NK>
struct MfmaTokens {
    using TL = MfmaTokLayout<NK>;
    static constexpr int kChunksPerTok = TL::kCols / 8;
    static constexpr int kTotal = B * kChunksPerTok;
    static constexpr int kIter = (kTotal + kBlock - 1) / kBlock;
    u32x4 stage[kIter];

    __device__ __forceinline__ void issue(const CoefArgs &a)
    {
#pragma unroll
        for (int t = 0; t < kIter; ++t) {
            const int c = threadIdx.x + t * kBlock;
            const int b = c / kChunksPerTok, col = (c % kChunksPerTok) * 8;
            stage[t] = load16(or_zero(c < kTotal && b < a.nb && col < a.d_model,
                                      a.x + (size_t)b * a.d_model + col));
        }
    }

    // the rows [B][kStride] and, after them, one zero chunk (returned)
    __device__ __forceinline__ uint32_t *write(uint32_t *xs) const
    {
#pragma unroll
        for (int t = 0; t < kIter; ++t) {
            const int c = threadIdx.x + t * kBlock;
            if (c < kTotal)
                *reinterpret_cast<u32x4 *>(xs + (size_t)(c / kChunksPerTok) * TL::kStride +
                                           (c % kChunksPerTok) * 4) = stage[t];
        }
        uint32_t *zchunk = xs + (size_t)B * TL::kStride;
        if (threadIdx.x == 0)
            *reinterpret_cast<u32x4 *>(zchunk) = zero16();
        return zchunk;
    }
};

// MFMA gather with the weight rows staged in LDS. Loads in the MFMA operand
// layout (16 rows x 64 B per instruction) reach about 60% of the HBM rate of
// row-contiguous loads on gathered rows (measured), so a wave loads each
// batch of STEPS steps (32 columns each) of its tile's 16 W_gate and W_up rows
// with 4 STEPS lanes on each row's piece (256 B of a row per load at 4 steps,
// 512 B at 8), writes them to its own LDS tile (rows padded by 16 B) and
// reads the A operands back; the token operand (L2-resident) is loaded with
// the batch.
template <int STEPS>
struct WtShape {
    static constexpr int kCols = STEPS * 32;              // columns of a batch
    static constexpr int kStride = kCols + 8;             // bf16 per tile row
    static constexpr int kWaveElems = 2 * kTile * kStride;  // bf16 per wave: W_gate and W_up tiles
    static constexpr int kLanesPerRow = kCols / 8;        // lanes on one row's piece
    static constexpr int kRowsPerLoad = kWave / kLanesPerRow;
    static constexpr int kLoads = kTile / kRowsPerLoad;   // loads per lane and matrix
};

// batch widths: the low-rank kernel's 256 columns with one batch in flight
// per wave measured 1-1.5% faster at 5-8 tokens than 128 columns with two in
// flight (two 256-column batches take 254 VGPRs, one wave per SIMD); the
// ternary kernel, and the low-rank one at rank 1024 (latent in LDS), keep
// 128-column batches, two in flight (with 256 columns the ternary layer took
// 80.7 against 64.4 us at 8 tokens)
constexpr int kWtStepsWide = 8;
constexpr int kWtStepsNarrow = 4;

template <int STEPS>
struct WtBatch {
    using W = WtShape<STEPS>;
    u32x4 w[2 * W::kLoads];  // W_gate rows kRowsPerLoad q + lane / kLanesPerRow, then W_up
    u32x4 x[STEPS];
};

template <int STEPS>
__device__ __forceinline__ void wt_load(WtBatch<STEPS> &bt, const CoefArgs &a,
                                        const int (&row)[WtShape<STEPS>::kLoads], uint32_t have,
                                        const uint16_t *xrow, bool xreal, int s, int s1, int lane)
{
    using W = WtShape<STEPS>;
    const int g = lane / kTile;
    const int col = s * 32 + (lane % W::kLanesPerRow) * 8;
    const bool colok = col < s1 * 32 && col < a.d_model;
#pragma unroll
    for (int q = 0; q < W::kLoads; ++q) {
        bt.w[q] = zero16();
        bt.w[W::kLoads + q] = zero16();
        if (((have >> q) & 1u) && colok) {
            bt.w[q] = load16_stream(a.Wg + (size_t)row[q] * a.d_model + col);
            bt.w[W::kLoads + q] = load16_stream(a.Wu + (size_t)row[q] * a.d_model + col);
        }
    }
    // a batch inside the row needs no column checks; lanes past the batch read
    // token 0 there (xrow), which only feeds output columns that are never
    // stored (MFMA output column j depends on B column j alone)
    if ((s + STEPS) * 32 <= a.d_model) {  // uniform
#pragma unroll
        for (int q = 0; q < STEPS; ++q)
            bt.x[q] = load16(xrow + (s + q) * 32 + g * 8);
    } else {
#pragma unroll
        for (int q = 0; q < STEPS; ++q) {
            const int xc = (s + q) * 32 + g * 8;
            bt.x[q] = load16(or_zero(xreal && xc < a.d_model, xrow + xc));
        }
    }
}

template <int STEPS>
__device__ __forceinline__ void wt_consume(uint16_t *wt, const WtBatch<STEPS> &bt, int s, int s1,
                                           int lane, f32x4_t &dg, f32x4_t &du)
{
    using W = WtShape<STEPS>;
    const int i = lane % kTile, g = lane / kTile;
    const int c = (lane % W::kLanesPerRow) * 8, rr0 = lane / W::kLanesPerRow;
#pragma unroll
    for (int q = 0; q < W::kLoads; ++q) {
        const int rr = W::kRowsPerLoad * q + rr0;
        *reinterpret_cast<u32x4 *>(wt + rr * W::kStride + c) = bt.w[q];
        *reinterpret_cast<u32x4 *>(wt + (kTile + rr) * W::kStride + c) = bt.w[W::kLoads + q];
    }
#pragma unroll
    for (int q = 0; q < STEPS; ++q) {
        if (s + q < s1) {  // uniform
            const u32x4 ga = *reinterpret_cast<const u32x4 *>(wt + i * W::kStride + q * 32 + g * 8);
            const u32x4 ua =
                *reinterpret_cast<const u32x4 *>(wt + (kTile + i) * W::kStride + q * 32 + g * 8);
            dg = mfma16(ga, bt.x[q], dg);
            du = mfma16(ua, bt.x[q], du);
        }
    }
}

// The block's active neurons (bits of M, rows r0 + bit) in tiles of 16 on MFMA:
// each tile's column steps are split among 4 / ntiles waves, which add their
// 16 x 16 partial sums in `part` (LDS [4][2][256] fp32) and write s = u * SiLU(g).
// wtiles: LDS [4 waves][WtShape<STEPS>::kWaveElems] bf16; lrow: LDS [32] rows
// of the active neurons. INTERLEAVE: wave kw of a tile takes batches kw,
// kw + wpt, ... of STEPS steps, so the tile's waves read adjacent pieces of
// each row together (after the low-rank score: 57.5 -> 56.7 us per 8B layer at
// 8 tokens); otherwise each takes one contiguous run of steps (the ternary
// kernel: interleaved, its layer took 68.2 against 65.4 us). A wave keeps two
// batches in flight at 4 steps, one at 8.
template <int B, int NK, bool INTERLEAVE, int STEPS>
__device__ __forceinline__ void gather_mfma_lds(const CoefArgs &a, uint16_t *wtiles, float *part,
                                                int *lrow, uint32_t M, int r0, int wave, int lane)
{
    using W = WtShape<STEPS>;
    constexpr int kWtSteps = STEPS, kWtLoads = W::kLoads;
    const int n = __builtin_popcount(M);
    if (threadIdx.x < kPredRows && ((M >> threadIdx.x) & 1u))
        lrow[__builtin_popcount(M & ((1u << threadIdx.x) - 1u))] = r0 + threadIdx.x;
    __syncthreads();  // lrow visible; the LDS scratch is free

    const int ntiles = (n + kTile - 1) / kTile;  // 0, 1 or 2
    if (ntiles == 0)
        return;
    const int wpt = kWavesPerBlock / ntiles;
    const int t0 = (wave / wpt) * kTile, kw = wave % wpt;
    const int i = lane % kTile, g = lane / kTile;
    const int steps = (a.d_model + 31) / 32;
    const int nbat = (steps + kWtSteps - 1) / kWtSteps;  // batches of kWtSteps steps
    (void)nbat;
    const bool xreal = i < a.nb;
    const uint16_t *xrow = a.x + (size_t)(xreal ? i : 0) * a.d_model;
    int row[kWtLoads];
    uint32_t have = 0u;
#pragma unroll
    for (int q = 0; q < kWtLoads; ++q) {
        const int k = t0 + W::kRowsPerLoad * q + lane / W::kLanesPerRow;
        row[q] = k < n ? lrow[k] : r0;
        have |= (k < n ? 1u : 0u) << q;
    }
    uint16_t *wt = wtiles + (size_t)wave * W::kWaveElems;
    f32x4_t dg = {0.0f, 0.0f, 0.0f, 0.0f}, du = {0.0f, 0.0f, 0.0f, 0.0f};
    WtBatch<STEPS> b0, b1;  // 4 steps: the next batch is in flight while this one is consumed
    if constexpr (INTERLEAVE && STEPS >= kWtStepsWide) {
        for (int j = kw; j < nbat; j += wpt) {
            wt_load(b0, a, row, have, xrow, xreal, j * kWtSteps, steps, lane);
            wt_consume(wt, b0, j * kWtSteps, steps, lane, dg, du);
        }
    } else if constexpr (INTERLEAVE) {
        if (kw < nbat)
            wt_load(b0, a, row, have, xrow, xreal, kw * kWtSteps, steps, lane);
        for (int j = kw; j < nbat; j += 2 * wpt) {
            const int jb = j + wpt;
            if (jb < nbat)
                wt_load(b1, a, row, have, xrow, xreal, jb * kWtSteps, steps, lane);
            wt_consume(wt, b0, j * kWtSteps, steps, lane, dg, du);
            if (jb >= nbat)
                break;
            if (jb + wpt < nbat)
                wt_load(b0, a, row, have, xrow, xreal, (jb + wpt) * kWtSteps, steps, lane);
            wt_consume(wt, b1, jb * kWtSteps, steps, lane, dg, du);
        }
    } else {
        const int sw = (steps + wpt - 1) / wpt;  // this wave's steps [s0, s1)
        const int s0 = min(steps, kw * sw), s1 = min(steps, s0 + sw);
        wt_load(b0, a, row, have, xrow, xreal, s0, s1, lane);
        for (int s = s0; s < s1; s += 2 * kWtSteps) {
            const int sb = s + kWtSteps;
            if (sb < s1)
                wt_load(b1, a, row, have, xrow, xreal, sb, s1, lane);
            wt_consume(wt, b0, s, s1, lane, dg, du);
            if (sb >= s1)
                break;
            if (sb + kWtSteps < s1)
                wt_load(b0, a, row, have, xrow, xreal, sb + kWtSteps, s1, lane);
            wt_consume(wt, b1, sb, s1, lane, dg, du);
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int e = (4 * g + r) * kTile + i;  // D[4g + r][i]
        part[(wave * 2 + 0) * 256 + e] = dg[r];
        part[(wave * 2 + 1) * 256 + e] = du[r];
    }
    __syncthreads();
    const int ti = threadIdx.x / kTile, tj = threadIdx.x % kTile;  // D[ti][tj] of each tile
    for (int tile = 0; tile < ntiles; ++tile) {
        float gs = 0.0f, us = 0.0f;
        for (int v = tile * wpt; v < (tile + 1) * wpt; ++v) {
            gs += part[(v * 2 + 0) * 256 + threadIdx.x];
            us += part[(v * 2 + 1) * 256 + threadIdx.x];
        }
        const int rank = tile * kTile + ti;
        if (rank < n && tj < a.nb)
            a.s[(size_t)tj * a.d_ff + lrow[rank]] = us * silu(gs);
    }
}

// Practical D-CountDown coefficient kernel for batches of 4-8 (Sec. 4): the
// scoring of k_coef_pred, then the block's active neurons in tiles of 16 on MFMA.
template <int B, int NK, int LCPR>
__global__ __launch_bounds__(kBlock) void k_coef_pred_mfma(const CoefArgs a)
{
    // LDS: the waves' weight tiles [4][kWaveElems] bf16, then the latent [B][d_rank]
    // fp32 (rank 1024 only), whose space later holds the partial sums [4][2][16 x 16]
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ uint32_t wflag[kWavesPerBlock];
    __shared__ int lrow[kPredRows];
    using S = PredShape<LCPR>;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int r0 = blockIdx.x * kPredRows;
    const int wr0 = r0 + wave * kPredRowsPerWave;

    using LR = LatentRegs<B, LCPR>;
    u32x4 wb[S::kLoads];
    pred_issue_bt<LCPR>(wb, a, wr0, lane);
    LR lr;
    lr.issue(a.lat, a.nb, a.d_rank, lane);
    LatentStage<LR::kRegs ? 1 : B> ls;  // the LDS copy, rank 1024 only
    if constexpr (!LR::kRegs)
        ls.issue(a.lat, a.nb, a.d_rank);
    __builtin_amdgcn_sched_barrier(0);
    zero_y(a.y, a.nb * a.d_model);
    uint16_t *wtiles = reinterpret_cast<uint16_t *>(xs);
    constexpr int STEPS = LR::kRegs ? kWtStepsWide : kWtStepsNarrow;
    uint32_t *latw = xs + kWavesPerBlock * WtShape<STEPS>::kWaveElems / 2;
    if constexpr (!LR::kRegs) {
        ls.write(reinterpret_cast<u32x4 *>(latw), a.lat, a.nb, a.d_rank);
        __syncthreads();
    }

    const uint32_t wmask = pred_score<B, LCPR>(wb, lr, reinterpret_cast<const float *>(latw), a,
                                               wr0, lane);
    if (lane == 0)
        wflag[wave] = wmask;
    __syncthreads();
    uint32_t M = 0;
#pragma unroll
    for (int v = 0; v < kWavesPerBlock; ++v)
        M |= wflag[v] << (v * kPredRowsPerWave);
    // the latent is no longer read once gather_mfma_lds's first barrier has passed
    gather_mfma_lds<B, NK, true, STEPS>(a, wtiles, reinterpret_cast<float *>(latw), lrow, M, r0,
                                        wave, lane);
}

// ------------------------------------------------ ternary predictor
// The TernaryLinear predictor of the paper's appendix: s_hat = x . theta with
// theta in {-1, 0, +1}^{d_model x d_ff}, thresholded like the low-rank score
// (signed, union over the batch), then the same gather. theta is stored
// neuron-major at 2 bits per weight in a layout that matches the token
// chunks of the lanes: row i is 64 * kWords 32-bit words, lane l owning words
// [l * kWords, (l + 1) * kWords). Unit j < NK of lane l holds the 8 weights
// of columns j * 512 + 8 l + [0, 8) (the columns of the lane's token chunk
// j); word k holds units 2k ("A") and 2k + 1 ("B"). In a word, bits 2m..2m+1
// of byte 1 / byte 3 are A's weights 2m / 2m + 1, and of byte 0 / byte 2 are
// B's weights 2m / 2m + 1 (m = 0..3). Codes: 0 -> 0, 1 -> +1, 2 -> -1.
//
// Decoding: a shift and a mask put the two codes of one weight pair in
// bytes 1 and 3 of a v_perm_b32 selector (bytes 0 and 2 zero); the table
// kTernLut maps code c to the high byte of a bf16 (0, +0.5, -0.5) and the
// zero selectors give the low bytes, so one v_perm yields a packed bf16 pair
// for v_dot2_f32_bf16. The products are half the weights', and doubling
// the fp32 sum at the end is exact.
template <int NK>
struct TernShape {
    static constexpr int kWords = NK >= 2 ? NK / 2 : 1;  // per lane and row
};

constexpr uint32_t kTernLut = 0x00BF3F00u;  // bytes: code 0 -> 0x00, 1 -> 0x3F, 2 -> 0xBF
constexpr uint32_t kTernPairMask = 0x03000300u;

template <int NK>
struct TernRows {
    static constexpr int kW = TernShape<NK>::kWords;
    uint32_t w[kPredRowsPerWave][kW];

    // the wave's kPredRowsPerWave rows starting at wr0 (rows past d_ff read zeros)
    __device__ __forceinline__ void issue(const CoefArgs &a, int wr0, int lane)
    {
#pragma unroll
        for (int r = 0; r < kPredRowsPerWave; ++r) {
            const bool ok = wr0 + r < a.d_ff;
            const uint32_t *p = a.Tp + ((size_t)(ok ? wr0 + r : 0) * kWave + lane) * kW;
            if constexpr (kW >= 4) {
#pragma unroll
                for (int q = 0; q < kW / 4; ++q) {
                    const u32x4 v = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x4 *>(or_zero(ok, p + 4 * q)));
                    w[r][4 * q + 0] = v.x;
                    w[r][4 * q + 1] = v.y;
                    w[r][4 * q + 2] = v.z;
                    w[r][4 * q + 3] = v.w;
                }
            } else if constexpr (kW == 2) {
                const uint64_t v = __builtin_nontemporal_load(
                    reinterpret_cast<const uint64_t *>(or_zero(ok, p)));
                w[r][0] = (uint32_t)v;
                w[r][1] = (uint32_t)(v >> 32);
            } else {
                w[r][0] = __builtin_nontemporal_load(or_zero(ok, p));
            }
        }
    }
};

// bf16 pair (weights 2m, 2m + 1 of unit j's half of word W), each 0 or +-0.5
// (j and m are compile-time constants after unrolling)
__device__ __forceinline__ uint32_t tern_pair(uint32_t W, int j, int m)
{
    const uint32_t sel = (j & 1) ? (W << (8 - 2 * m)) & kTernPairMask : (W >> (2 * m)) & kTernPairMask;
    return __builtin_amdgcn_perm(0u, kTernLut, sel);
}

// s_hat_b = x_b . theta[:, row] for the wave's rows (xget(b, j) = this lane's
// 16-byte chunk j of token b), the signed threshold with the union over the
// batch, act[] and (optionally) the coefficients. Returns the wave-uniform
// mask of its active rows. With LDS tokens (SETTLE) the accumulators are
// materialised after every chunk and xget addresses LDS through an opaque
// offset, so the reads of chunk j + 1 cannot be hoisted above the products of
// chunk j (hoisting them all costs 4 * B * NK registers).
template <int B, int NK, bool SETTLE, class XF>
__device__ __forceinline__ uint32_t tern_score(const TernRows<NK> &t, XF xget, const CoefArgs &a,
                                               int wr0, int lane)
{
    constexpr int R = kPredRowsPerWave;
    float acc[R][B];
#pragma unroll
    for (int r = 0; r < R; ++r)
        zero_acc(acc[r]);
#pragma unroll
    for (int j = 0; j < NK; ++j) {
        u32x4 xv[B];
#pragma unroll
        for (int b = 0; b < B; ++b)
            xv[b] = xget(b, j);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint32_t W = t.w[r][j >> 1];
            const uint32_t p0 = tern_pair(W, j, 0), p1 = tern_pair(W, j, 1);
            const uint32_t p2 = tern_pair(W, j, 2), p3 = tern_pair(W, j, 3);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                acc[r][b] = dot2_bf16(p0, xv[b].x, acc[r][b]);
                acc[r][b] = dot2_bf16(p1, xv[b].y, acc[r][b]);
                acc[r][b] = dot2_bf16(p2, xv[b].z, acc[r][b]);
                acc[r][b] = dot2_bf16(p3, xv[b].w, acc[r][b]);
            }
        }
        if constexpr (SETTLE) {
#pragma unroll
            for (int r = 0; r < R; ++r)
#pragma unroll
                for (int b = 0; b < B; ++b)
                    asm volatile("" : "+v"(acc[r][b]));
        }
    }
    uint32_t wmask = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int row = wr0 + r;
        bool act = false;
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const float v = 2.0f * wave_sum(acc[r][b]);
            if (b < a.nb) {
                act = act || (v > a.thld);
                if (a.coef && lane == 0 && row < a.d_ff)
                    a.coef[(size_t)b * a.d_ff + row] = v;
            }
        }
        if (row < a.d_ff) {
            if (lane == 0)
                a.act[row] = act ? 1 : 0;
            if (act)
                wmask |= 1u << r;
        }
    }
    return wmask;
}

// The ternary score of a wave's kPredRowsPerWave rows on MFMA, for batches of
// 5-8 and d_model 4096 (one 16-byte block of packed theta per lane and row):
// s_hat = theta . x is a dense product with weights in {-1, 0, +1}. Lane
// (n, g) = (lane % 16, lane / 16) reads block 4 t + g of row n (rows past the
// wave's 8 read zeros) for t = 0 .. 15; unit j of that block, decoded by
// tern_pair into 8 bf16 weights of +-0.5 or 0, is the A operand of one
// v_mfma_f32_16x16x32_bf16 step whose B operand is token n's columns
// 512 j + 8 (4 t + g) + [0, 8) from the LDS copy, so A and B agree on the
// column order and the 128 steps cover every column once. D[row][token] is
// half the score. Threshold, union and stores as in tern_score.
template <int NK>
struct TernMfmaRows {
    static_assert(NK == 8, "one 16-byte block per lane and row");
    static constexpr int kW = TernShape<NK>::kWords;  // 4
    u32x4 blk[16];

    __device__ __forceinline__ void issue(const CoefArgs &a, int wr0, int lane)
    {
        const int n = lane % kTile, g = lane / kTile;
        const int row = wr0 + n;
        const bool ok = n < kPredRowsPerWave && row < a.d_ff;
        const uint32_t *rp = a.Tp + (size_t)(ok ? row : 0) * kWave * kW;
#pragma unroll
        for (int t = 0; t < 16; ++t)
            blk[t] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4 *>(or_zero(ok, rp + (4 * t + g) * kW)));
    }
};

// xcol(col): this lane's token (lane % 16) at columns col .. col + 7, zeros
// past the batch
template <int NK, class XC>
__device__ __forceinline__ uint32_t tern_score_mfma(const TernMfmaRows<NK> &tr, XC xcol,
                                                    const CoefArgs &a, int wr0, int lane)
{
    const int n = lane % kTile, g = lane / kTile;
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int t = 0; t < 16; ++t) {
        const u32x4 w = tr.blk[t];
#pragma unroll
        for (int j = 0; j < NK; ++j) {
            const uint32_t W = w[j >> 1];
            u32x4 wa;
            wa.x = tern_pair(W, j, 0);
            wa.y = tern_pair(W, j, 1);
            wa.z = tern_pair(W, j, 2);
            wa.w = tern_pair(W, j, 3);
            acc = mfma16(wa, xcol(j * kColsPerLoad + 8 * (4 * t + g)), acc);
        }
    }
    // lane l holds D[4 g + r][l % 16]: rows 4 g + r of the wave (g < 2), token l % 16
    uint32_t wmask = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int rw = 4 * g + r;
        const int row = wr0 + rw;
        const bool live = rw < kPredRowsPerWave && row < a.d_ff && n < a.nb;
        const float v = 2.0f * acc[r];
        if (a.coef && live)
            a.coef[(size_t)n * a.d_ff + row] = v;
        const uint64_t m = ballot(live && v > a.thld);
        const bool act0 = (m & 0xffffull) != 0, act1 = ((m >> 16) & 0xffffull) != 0;
        if (lane == 0 && wr0 + r < a.d_ff)
            a.act[wr0 + r] = act0 ? 1 : 0;
        if (lane == kTile && wr0 + 4 + r < a.d_ff)
            a.act[wr0 + 4 + r] = act1 ? 1 : 0;
        wmask |= (act0 && wr0 + r < a.d_ff ? 1u : 0u) << r;
        wmask |= (act1 && wr0 + 4 + r < a.d_ff ? 1u : 0u) << (4 + r);
    }
    return wmask;
}

// Ternary-predictor coefficient kernel for batches of 1-4: k_coef_pred with
// the ternary score in place of the latent . B_t one (no latent kernel).
template <int B, int NK, bool XREG, int NWV = kWavesPerBlock>
__global__ __launch_bounds__(NWV * kWave) void k_coef_tern(const CoefArgs a)
{
    extern __shared__ __align__(16) uint32_t xs[];  // tokens [B][NK * 256] (LDS path)
    __shared__ uint32_t wflag[kWavesPerBlock];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // NWV 8: as in k_coef_pred, the waves past the fourth only gather
    const bool scorer = NWV == kWavesPerBlock || wave < kWavesPerBlock;  // wave-uniform
    const int r0 = blockIdx.x * kPredRows;
    const int wr0 = scorer ? r0 + wave * kPredRowsPerWave : a.d_ff;

    TernRows<NK> tr;
    tr.issue(a, wr0, lane);
    Tokens<B, NK, XREG> tok;
    if (XREG || scorer)  // the LDS copy: the first kBlock threads
        tok.issue(a.x, a.nb, a.d_model, lane);
    if (scorer)
        zero_y(a.y, a.nb * a.d_model);
    if constexpr (!XREG) {
        if (scorer)
            tok.write(xs);
        else
            tok.lds = xs;
        __syncthreads();
    }
    uint32_t wmask = 0;
    if (!scorer) {
        // no rows to score
    } else if constexpr (XREG) {
        wmask = tern_score<B, NK, false>(tr, [&](int b, int j) { return tok.r[b][j]; }, a, wr0,
                                         lane);
    } else {
        wmask = tern_score<B, NK, true>(
            tr,
            [&](int b, int j) {
                return *tok.lds_chunk(b, j, lane, Tokens<B, NK, XREG>::opaque_zero());
            },
            a, wr0, lane);
    }
    const uint32_t m = block_share<NWV>(wflag, wmask, wave, lane);
    gather_rr<B, NK, XREG, NWV>(a, tok, m, r0, lane);
}

// LDS bytes of the ternary MFMA kernel: the token copy, which the gather's
// weight tiles reuse once the scores are in, then the partial sums
template <int B, int NK>
__host__ __device__ constexpr size_t tern_mfma_front_u32()
{
    constexpr size_t kTiles = (size_t)kWavesPerBlock * WtShape<kWtStepsNarrow>::kWaveElems / 2;
    return mfma_lds_tokens_u32<B, NK>() > kTiles ? mfma_lds_tokens_u32<B, NK>() : kTiles;
}

// Ternary-predictor coefficient kernel for batches of 5-8: the ternary score
// (on MFMA at d_model 4096, tern_score_mfma; v_dot2 otherwise), then the MFMA
// gather with LDS-staged weight rows.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_coef_tern_mfma(const CoefArgs a)
{
    // LDS: tokens [B][kStride] (+ zero chunk), overlaid by the weight tiles after
    // the scores, then the partial sums [4 waves][2][16 x 16]
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ uint32_t wflag[kWavesPerBlock];
    __shared__ int lrow[kPredRows];
    using TL = MfmaTokLayout<NK>;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int r0 = blockIdx.x * kPredRows;
    const int wr0 = r0 + wave * kPredRowsPerWave;

    // the score on MFMA at d_model 4096 (8B layer at 8 tokens: 64.4 -> 58.0 us,
    // at 5: 54.3 -> 49.0); v_dot2 for the other widths. (At 3-4 tokens, in
    // k_coef_tern, it measured no faster: 38.5 against 38.2 us at 4.)
    constexpr bool kMfmaScore = NK == 8;
    using TR = std::conditional_t<kMfmaScore, TernMfmaRows<8>, TernRows<NK>>;
    TR tr;
    tr.issue(a, wr0, lane);
    MfmaTokens<B, NK> mt;
    mt.issue(a);
    __builtin_amdgcn_sched_barrier(0);
    zero_y(a.y, a.nb * a.d_model);
    const uint32_t *zchunk = mt.write(xs);
    __syncthreads();

    uint32_t wmask;
    if constexpr (kMfmaScore) {
        const int n = lane % kTile;
        const uint32_t *xt =
            n < a.nb ? xs + Tokens<B, NK, false>::opaque_zero() + (size_t)n * TL::kStride : zchunk;
        // past the batch the zero chunk for every column: a mask on the offset,
        // not a pointer select per step (the select cost 1.7 us at 8 tokens)
        const int cm = n < a.nb ? ~0 : 0;
        wmask = tern_score_mfma<NK>(
            tr, [&](int col) { return *reinterpret_cast<const u32x4 *>(xt + ((col / 2) & cm)); }, a,
            wr0, lane);
    } else {
        wmask = tern_score<B, NK, true>(
            tr,
            [&](int b, int j) {
                return *reinterpret_cast<const u32x4 *>(xs + Tokens<B, NK, false>::opaque_zero() +
                                                        (size_t)b * TL::kStride +
                                                        (j * kColsPerLoad + lane * 8) / 2);
            },
            a, wr0, lane);
    }
    if (lane == 0)
        wflag[wave] = wmask;
    __syncthreads();
    uint32_t M = 0;
#pragma unroll
    for (int v = 0; v < kWavesPerBlock; ++v)
        M |= wflag[v] << (v * kPredRowsPerWave);
    (void)zchunk;
    // (the barrier above ends the token reads: the tiles may overwrite them)
    gather_mfma_lds<B, NK, false, kWtStepsNarrow>(a, reinterpret_cast<uint16_t *>(xs),
                           reinterpret_cast<float *>(xs + tern_mfma_front_u32<B, NK>()), lrow, M,
                           r0, wave, lane);
}

// latent = x . theta_A for the predictor: one workgroup per row of A_t, the
// four waves take every fourth 512-column chunk (tokens read straight from
// global memory, each lane only its own chunks) and add up in LDS.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_latent(const uint16_t *__restrict__ x, int nb,
                                                   const uint16_t *__restrict__ At, int d_model,
                                                   int d_rank, float *__restrict__ lat)
{
    constexpr int KW = (NK + kWavesPerBlock - 1) / kWavesPerBlock;  // chunks per wave
    __shared__ float part[kWavesPerBlock][B];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int r = blockIdx.x;
    const uint16_t *row = At + (size_t)r * d_model;
    u32x4 w[KW];
#pragma unroll
    for (int t = 0; t < KW; ++t) {
        const int col = (wave + t * kWavesPerBlock) * kColsPerLoad + lane * 8;
        w[t] = col < d_model ? load16_stream(row + col) : zero16();
    }
    float acc[B];
    zero_acc(acc);
#pragma unroll
    for (int b = 0; b < B; ++b) {
        if (b < nb) {
#pragma unroll
            for (int t = 0; t < KW; ++t) {
                const int col = (wave + t * kWavesPerBlock) * kColsPerLoad + lane * 8;
                acc[b] = dot8(w[t], load16(or_zero(col < d_model, x + (size_t)b * d_model + col)),
                              acc[b]);
            }
        }
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float v = wave_sum(acc[b]);
        if (lane == 0)
            part[wave][b] = v;
    }
    __syncthreads();
    if (threadIdx.x < nb) {
        float v = 0.0f;
#pragma unroll
        for (int q = 0; q < kWavesPerBlock; ++q)
            v += part[q][threadIdx.x];
        lat[(size_t)threadIdx.x * d_rank + r] = v;
    }
}

// ----------------------------------------------------- residual + RMSNorm
// Joins the layers of a stack of FFNs (the paper's method stops at one layer):
// per token h = h_in + y_prev (fp32) and x = bf16(h / sqrt(mean(h^2) + eps)),
// round to nearest even. A 256-thread workgroup holds a token's values in the
// column layout of the latent product: wave w, lane l owns the 8 columns
// (w + 4t) * 512 + 8l + [0, 8), t < KW.

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    const uint32_t l = __builtin_bit_cast(uint16_t, static_cast<__bf16>(lo));
    const uint32_t h = __builtin_bit_cast(uint16_t, static_cast<__bf16>(hi));
    return l | (h << 16);
}

__device__ __forceinline__ float f32_of(uint32_t v) { return __uint_as_float(v); }

// Normalised tokens of this thread's columns, xq[b][t] (8 bf16 each). With
// WRITE the thread also stores its columns of h_out and x_out. red: LDS
// [kWavesPerBlock][B] floats. Every thread of the workgroup must call this.
template <int B, int KW, bool WRITE>
__device__ __forceinline__ void residual_norm(const NormArgs &n, int lane, int wave, float *red,
                                              u32x4 (&xq)[B][KW])
{
    u32x4 hv[B][KW][2];  // 8 fp32 of h per (token, chunk), raw bits
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
        for (int t = 0; t < KW; ++t) {
            const int col = (wave + t * kWavesPerBlock) * kColsPerLoad + lane * 8;
            const bool ok = b < n.nb && col < n.d_model;
            const size_t off = (size_t)b * n.d_model + col;
            const u32x4 *hp = reinterpret_cast<const u32x4 *>(n.h_in + off);
            hv[b][t][0] = *or_zero(ok, hp);
            hv[b][t][1] = *or_zero(ok, hp + 1);
            if (n.y_prev) {
                const u32x4 *yp = reinterpret_cast<const u32x4 *>(n.y_prev + off);
                const u32x4 y0 = *or_zero(ok, yp), y1 = *or_zero(ok, yp + 1);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    hv[b][t][0][q] = __float_as_uint(f32_of(hv[b][t][0][q]) + f32_of(y0[q]));
                    hv[b][t][1][q] = __float_as_uint(f32_of(hv[b][t][1][q]) + f32_of(y1[q]));
                }
            }
        }
    float ss[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
        float v = 0.0f;
#pragma unroll
        for (int t = 0; t < KW; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                v += f32_of(hv[b][t][0][q]) * f32_of(hv[b][t][0][q]) +
                     f32_of(hv[b][t][1][q]) * f32_of(hv[b][t][1][q]);
        ss[b] = wave_sum(v);
    }
    if (lane == 0)
#pragma unroll
        for (int b = 0; b < B; ++b)
            red[wave * B + b] = ss[b];
    __syncthreads();
#pragma unroll
    for (int b = 0; b < B; ++b) {
        float tot = 0.0f;
#pragma unroll
        for (int v = 0; v < kWavesPerBlock; ++v)
            tot += red[v * B + b];
        const float inv = 1.0f / sqrtf(tot / (float)n.d_model + n.eps);
#pragma unroll
        for (int t = 0; t < KW; ++t) {
            const u32x4 h0 = hv[b][t][0], h1 = hv[b][t][1];
            xq[b][t] = u32x4{pack_bf16(f32_of(h0.x) * inv, f32_of(h0.y) * inv),
                             pack_bf16(f32_of(h0.z) * inv, f32_of(h0.w) * inv),
                             pack_bf16(f32_of(h1.x) * inv, f32_of(h1.y) * inv),
                             pack_bf16(f32_of(h1.z) * inv, f32_of(h1.w) * inv)};
            if constexpr (WRITE) {
                const int col = (wave + t * kWavesPerBlock) * kColsPerLoad + lane * 8;
                if (b < n.nb && col < n.d_model) {
                    const size_t off = (size_t)b * n.d_model + col;
                    u32x4 *ho = reinterpret_cast<u32x4 *>(n.h_out + off);
                    ho[0] = h0;
                    ho[1] = h1;
                    *reinterpret_cast<u32x4 *>(n.x_out + off) = xq[b][t];
                }
            }
        }
    }
}

// Residual stream step alone (variants without a latent product): one workgroup.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_norm(const NormArgs n)
{
    constexpr int KW = (NK + kWavesPerBlock - 1) / kWavesPerBlock;
    __shared__ float red[kWavesPerBlock * B];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    u32x4 xq[B][KW];
    residual_norm<B, KW, true>(n, lane, wave, red, xq);
}

// Residual stream step fused with latent = x . theta_A: one workgroup per row
// of A_t; each normalises the tokens itself (the first also writes h_out and
// x_out for the kernels that follow) and takes the dot products with its row.
template <int B, int NK>
__global__ __launch_bounds__(kBlock) void k_latent_norm(const NormArgs n,
                                                        const uint16_t *__restrict__ At,
                                                        int d_rank, float *__restrict__ lat)
{
    constexpr int KW = (NK + kWavesPerBlock - 1) / kWavesPerBlock;
    __shared__ float red[kWavesPerBlock * B];
    __shared__ float part[kWavesPerBlock][B];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int r = blockIdx.x;
    const uint16_t *row = At + (size_t)r * n.d_model;
    u32x4 w[KW];
#pragma unroll
    for (int t = 0; t < KW; ++t) {
        const int col = (wave + t * kWavesPerBlock) * kColsPerLoad + lane * 8;
        w[t] = col < n.d_model ? load16_stream(row + col) : zero16();
    }
    u32x4 xq[B][KW];
    if (blockIdx.x == 0)
        residual_norm<B, KW, true>(n, lane, wave, red, xq);
    else
        residual_norm<B, KW, false>(n, lane, wave, red, xq);
    float acc[B];
    zero_acc(acc);
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
        for (int t = 0; t < KW; ++t)
            acc[b] = dot8(w[t], xq[b][t], acc[b]);  // chunks past d_model hold zeros in w
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float v = wave_sum(acc[b]);
        if (lane == 0)
            part[wave][b] = v;
    }
    __syncthreads();
    if (threadIdx.x < n.nb) {
        float v = 0.0f;
#pragma unroll
        for (int q = 0; q < kWavesPerBlock; ++q)
            v += part[q][threadIdx.x];
        lat[(size_t)threadIdx.x * d_rank + r] = v;
    }
}

// A range without active neurons still owns its slice of the per-range partial
// sums in deterministic mode: zeros for columns [c0, c0 + w) of every token.
__device__ __forceinline__ void zero_part(const DownArgs &a, int g, int c0, int w)
{
    for (int i = threadIdx.x; i < a.nb * w; i += kBlock) {
        const int b = i / w, col = c0 + i % w;
        if (col < a.d_model)
            a.part[((size_t)g * a.nb + b) * a.d_model + col] = 0.0f;
    }
}

// y[b][col] = sum over the gr ranges, in ascending order, of their partial sums:
// the down projection's reduction in a fixed order (deterministic mode).
__global__ __launch_bounds__(kBlock) void k_reduce_parts(const float *__restrict__ part, int gr,
                                                         int n, float *__restrict__ y)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n)
        return;
    // all of a column's partial sums in flight at once (64 ranges at 1-2 tokens);
    // the additions stay in range order
    constexpr int U = 64;
    float v = 0.0f;
    for (int g0 = 0; g0 < gr; g0 += U) {
        float t[U];
#pragma unroll
        for (int q = 0; q < U; ++q)
            t[q] = g0 + q < gr ? part[(size_t)(g0 + q) * n + i] : 0.0f;
#pragma unroll
        for (int q = 0; q < U; ++q)
            v += t[q];  // + 0 past gr leaves v unchanged
    }
    y[i] = v;
}

// Gathered down projection (Eq. 5). Workgroup (c, g) owns a 512-column chunk
// c and a contiguous neuron range g: one round trip reads act and s of the
// range, a wave ballot compacts the active neurons in ascending order into
// LDS, each wave then keeps U rows in flight (1 KB of a row per load), the
// four waves reduce in LDS and add the chunk to y with one fp32 atomic per
// column and token. U = 16 against 8: the same time at 90% sparsity, 5% less
// at 50% (7B shape), where a wave has about 20 rows to read; 24 and 32 cost
// occupancy and measured no better (7B at 50%: 32.7 / 32.5 against 31.8 us).
template <int B>
__global__ __launch_bounds__(kBlock) void k_down(const DownArgs a)
{
    constexpr int U = 16;
    extern __shared__ __align__(16) int dsm[];
    __shared__ int wcnt[kWavesPerBlock];
    const int cap = a.rows_per_group;
    int *lrow = dsm;                                                 // [cap]
    float *lsv = reinterpret_cast<float *>(dsm + cap);               // [B][cap]
    float *red = reinterpret_cast<float *>(dsm + cap * (1 + B));     // [4][512]
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int c = blockIdx.x % a.gc, g = blockIdx.x / a.gc;
    const int r0 = g * cap;
    const int r1 = min(a.d_ff, r0 + cap);

    // four consecutive neurons per thread: 16-byte flag and s loads, one pass
    // per 1024 neurons (ranges are multiples of 4 neurons, so a quad is whole)
    int nl = 0;
    for (int t0 = r0; t0 < r1; t0 += 4 * kBlock) {
        const int row = t0 + 4 * threadIdx.x;
        const bool ok = row < r1;
        const int4 av = *or_zero(ok, reinterpret_cast<const int4 *>(a.act + row));
        const int f[4] = {av.x != 0, av.y != 0, av.z != 0, av.w != 0};
        float sv[B][4];
#pragma unroll
        for (int b = 0; b < B; ++b) {
            const float4 v =
                *or_zero(ok && b < a.nb, reinterpret_cast<const float4 *>(a.s + (size_t)b * a.d_ff + row));
            sv[b][0] = v.x;
            sv[b][1] = v.y;
            sv[b][2] = v.z;
            sv[b][3] = v.w;
        }
        int below = 0, tot = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint64_t m = ballot(f[k] != 0);
            below += lanes_below(m);
            tot += __popcll(m);
        }
        if (lane == 0)
            wcnt[wave] = tot;
        __syncthreads();
        int pos = nl + below;
        for (int v = 0; v < wave; ++v)
            pos += wcnt[v];
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (f[k]) {
                lrow[pos] = row + k;
#pragma unroll
                for (int b = 0; b < B; ++b)
                    lsv[b * cap + pos] = sv[b][k];
                ++pos;
            }
        nl += wcnt[0] + wcnt[1] + wcnt[2] + wcnt[3];
        __syncthreads();
    }
    if (nl == 0) {  // uniform for the workgroup
        if (a.part)
            zero_part(a, g, c * kColsPerLoad, kColsPerLoad);
        return;
    }

    const int col = c * kColsPerLoad + lane * 8;
    const bool colok = col < a.d_model;
    float acc[B][8];
#pragma unroll
    for (int b = 0; b < B; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            acc[b][e] = 0.0f;

    for (int q0 = wave; q0 < nl; q0 += kWavesPerBlock * U) {
        u32x4 w[U];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int r = q0 + q * kWavesPerBlock;
            w[q] = (r < nl && colok) ? load16_stream(a.Wd + (size_t)lrow[r] * a.d_model + col)
                                     : zero16();
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const int r = q0 + q * kWavesPerBlock;
            if (r >= nl)
                break;
            const float wf[8] = {bf16_lo(w[q].x), bf16_hi(w[q].x), bf16_lo(w[q].y), bf16_hi(w[q].y),
                                 bf16_lo(w[q].z), bf16_hi(w[q].z), bf16_lo(w[q].w), bf16_hi(w[q].w)};
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const float sv = lsv[b * cap + r];
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc[b][e] = fmaf(sv, wf[e], acc[b][e]);
            }
        }
    }

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
                if (a.part)
                    a.part[((size_t)g * a.nb + b) * a.d_model + gcol] = v;
                else
                    unsafeAtomicAdd(a.y + (size_t)b * a.d_model + gcol, v);
            }
        }
    }
}

// passes of 4 * kBlock neurons in the MFMA down kernel's flag scan (ranges of
// at most 2048 neurons, a multiple of 4)
constexpr int kDownScanPasses = 2;

// Gathered down projection for batches of 4-8 on MFMA. The product
// Y[B x d_model] = S[B x n] . W_down[IDX, :] is a dense contraction over the
// active neurons: v_mfma_f32_16x16x32_bf16 with A = S (row i = token i, zero
// rows past the batch) and B = the W_down rows. Workgroup (c, g) owns 128
// columns c and neuron range g (compacted as in k_down); its waves take every
// fourth step of 32 list positions and add their 16 x 128 results in LDS
// before the atomics. In a step, lane l = j + 16 q loads rows
// 8 q .. 8 q + 7 of the step at columns 8 j .. 8 j + 7 (one 16-byte load per
// row); v_perm then regroups them per column e into the B operand of an
// MFMA whose output columns are 8 j + e, so the loaded data needs no LDS
// transpose. S enters as bf16 hi + lo (s - hi rounded again), two MFMAs per
// operand, so each product keeps about 16 mantissa bits.
template <int BT>
__global__ __launch_bounds__(kBlock) void k_down_mfma(const DownArgs a)
{
    constexpr int T = kDownScanPasses;
    extern __shared__ __align__(16) int dsm[];
    __shared__ int wcnt[T][kWavesPerBlock];
    const int cap = a.rows_per_group;
    const int capp = (cap + 31) & ~31;                                     // padded list length
    int *lrow = dsm;                                                       // [capp]
    uint16_t *shi = reinterpret_cast<uint16_t *>(dsm + capp);              // [BT][capp] bf16
    uint16_t *slo = shi + (size_t)BT * capp;                               // [BT][capp] bf16
    uint32_t *zrow = reinterpret_cast<uint32_t *>(slo + (size_t)BT * capp);  // 16 zero bytes
    float *out = reinterpret_cast<float *>(zrow + 4);                      // [4 waves][BT][128]
    constexpr int kStep = 32, kWc = 128;  // list positions per step, columns per workgroup
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int c = blockIdx.x % a.gc, g = blockIdx.x / a.gc;
    const int r0 = g * cap;
    const int r1 = min(a.d_ff, r0 + cap);

    // flags and s of four consecutive neurons per thread (16-byte loads: a
    // quarter of the load instructions of one neuron per thread, which at
    // batch 8 took about 1.4 us more per call); the list stays ascending
    int f[T][4], below[T];
    float sv[T][BT][4];
#pragma unroll
    for (int t = 0; t < T; ++t) {
        const int row = r0 + t * 4 * kBlock + 4 * threadIdx.x;
        const bool ok = t * 4 * kBlock < cap && row < r1;  // r0, r1 multiples of 4 (host)
        const int4 av = *or_zero(ok, reinterpret_cast<const int4 *>(a.act + row));
        f[t][0] = av.x != 0;
        f[t][1] = av.y != 0;
        f[t][2] = av.z != 0;
        f[t][3] = av.w != 0;
#pragma unroll
        for (int b = 0; b < BT; ++b) {
            const float4 v =
                *or_zero(ok && b < a.nb, reinterpret_cast<const float4 *>(a.s + (size_t)b * a.d_ff + row));
            sv[t][b][0] = v.x;
            sv[t][b][1] = v.y;
            sv[t][b][2] = v.z;
            sv[t][b][3] = v.w;
        }
        int tot = 0;
        below[t] = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint64_t m = ballot(f[t][k] != 0);
            below[t] += lanes_below(m);
            tot += __popcll(m);
        }
        if (lane == 0)
            wcnt[t][wave] = tot;
    }
    if (threadIdx.x < 4)
        zrow[threadIdx.x] = 0u;
    __syncthreads();
    int nl = 0;
#pragma unroll
    for (int t = 0; t < T; ++t) {
        int pos = nl + below[t];
        for (int v = 0; v < wave; ++v)
            pos += wcnt[t][v];
        const int row = r0 + t * 4 * kBlock + 4 * threadIdx.x;
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (f[t][k]) {
                lrow[pos] = row + k;
#pragma unroll
                for (int b = 0; b < BT; ++b) {
                    const __bf16 h = (__bf16)sv[t][b][k];
                    const __bf16 l = (__bf16)(sv[t][b][k] - (float)h);
                    shi[b * capp + pos] = __builtin_bit_cast(uint16_t, h);
                    slo[b * capp + pos] = __builtin_bit_cast(uint16_t, l);
                }
                ++pos;
            }
        nl += wcnt[t][0] + wcnt[t][1] + wcnt[t][2] + wcnt[t][3];
    }
    // zero coefficients (and a valid row) for the padding of the last step
    const int nlp = (nl + 31) & ~31;
    for (int p = nl + threadIdx.x; p < nlp; p += kBlock) {
        lrow[p] = r0;
#pragma unroll
        for (int b = 0; b < BT; ++b) {
            shi[b * capp + p] = 0;
            slo[b * capp + p] = 0;
        }
    }
    __syncthreads();
    if (nl == 0) {  // uniform for the workgroup
        if (a.part)
            zero_part(a, g, c * kWc, kWc);
        return;
    }

    const int j = lane % 16, q = lane / 16;
    const int col = c * kWc + j * 8;
    const bool colok = col < a.d_model;
    // A operand source: token j's coefficients (zero row past the batch)
    const bool real = j < a.nb;
    f32x4_t acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        acc[e] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    u32x4 cur[8], nxt[8];
    auto load_step = [&](u32x4 (&w)[8], int p0) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int p = p0 + 8 * q + r;
            w[r] = zero16();
            if (p < nl && colok)
                w[r] = load16_stream(a.Wd + (size_t)lrow[p] * a.d_model + col);
        }
    };
    auto consume = [&](const u32x4 (&w)[8], int p0) {
        const int pa = p0 + 8 * q;
        const u32x4 ah = *reinterpret_cast<const u32x4 *>(real ? shi + (size_t)j * capp + pa
                                                               : reinterpret_cast<uint16_t *>(zrow));
        const u32x4 al = *reinterpret_cast<const u32x4 *>(real ? slo + (size_t)j * capp + pa
                                                               : reinterpret_cast<uint16_t *>(zrow));
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            // column 8 j + e of the lane's 8 rows: 16-bit halves of word e / 2
            const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
            u32x4 bw;
            bw.x = __builtin_amdgcn_perm(w[1][e / 2], w[0][e / 2], sel);
            bw.y = __builtin_amdgcn_perm(w[3][e / 2], w[2][e / 2], sel);
            bw.z = __builtin_amdgcn_perm(w[5][e / 2], w[4][e / 2], sel);
            bw.w = __builtin_amdgcn_perm(w[7][e / 2], w[6][e / 2], sel);
            acc[e] = mfma16(ah, bw, acc[e]);
            acc[e] = mfma16(al, bw, acc[e]);
        }
    };
    // this wave's steps start at positions wave * kStep + k * 4 * kStep
    constexpr int kStride = kWavesPerBlock * kStep;
    const int pw = wave * kStep;
    if (pw < nl) {  // uniform per wave
        load_step(cur, pw);
        for (int p0 = pw; p0 < nl; p0 += 2 * kStride) {
            const bool more = p0 + kStride < nl;  // uniform
            if (more)
                load_step(nxt, p0 + kStride);
            consume(cur, p0);
            if (!more)
                break;
            if (p0 + 2 * kStride < nl)
                load_step(cur, p0 + 2 * kStride);
            consume(nxt, p0 + kStride);
        }
    }

    // D[token 4 q + r][column 8 j + e] of the four waves -> LDS, summed, then
    // one contiguous fp32 atomic per column and token
    float *ow = out + (size_t)wave * BT * kWc;
#pragma unroll
    for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int tok = 4 * q + r;
            if (tok < BT)
                ow[tok * kWc + j * 8 + e] = acc[e][r];
        }
    __syncthreads();
    for (int i = threadIdx.x; i < BT * kWc; i += kBlock) {
        const int b = i / kWc, cc = i % kWc;
        const int gcol = c * kWc + cc;
        if (b < a.nb && gcol < a.d_model) {
            const float v = out[i] + out[BT * kWc + i] + out[2 * BT * kWc + i] +
                            out[3 * BT * kWc + i];
            if (a.part)
                a.part[((size_t)g * a.nb + b) * a.d_model + gcol] = v;
            else
                unsafeAtomicAdd(a.y + (size_t)b * a.d_model + gcol, v);
        }
    }
}

// batches from which the down projection runs on MFMA (measured: at 2 the
// VALU kernel is faster, at 4 and 8 the MFMA one)
constexpr int kDownMfmaMinBatch = 4;

size_t down_mfma_lds_bytes(int rows_per_group, int bt)
{
    const size_t capp = (size_t)((rows_per_group + 31) & ~31);
    return capp * 4 + 2 * (size_t)bt * capp * 2 + 16 + (size_t)kWavesPerBlock * bt * 128 * 4;
}

constexpr int kExportThreads = 1024;

// Flat ascending IDX, |IDX| and compact s of the last call (one workgroup):
// scan of the per-neuron flags, then every thread writes its neurons.
__global__ __launch_bounds__(kExportThreads) void k_export(const int *__restrict__ act,
                                                           const float *__restrict__ s, int nb,
                                                           int d_ff, int *idx_dst, int *n_dst,
                                                           float *s_dst)
{
    __shared__ int part[kExportThreads];
    const int t = threadIdx.x;
    const int per = (d_ff + kExportThreads - 1) / kExportThreads;
    const int lo = min(d_ff, t * per), hi = min(d_ff, lo + per);
    int sum = 0;
    for (int i = lo; i < hi; ++i)
        sum += act[i] != 0;
    part[t] = sum;
    __syncthreads();
    for (int off = 1; off < kExportThreads; off <<= 1) {
        const int v = t >= off ? part[t - off] : 0;
        __syncthreads();
        part[t] += v;
        __syncthreads();
    }
    if (t == kExportThreads - 1 && n_dst)
        *n_dst = part[t];
    int pos = part[t] - sum;
    for (int i = lo; i < hi; ++i) {
        if (!act[i])
            continue;
        if (idx_dst)
            idx_dst[pos] = i;
        if (s_dst)
            for (int b = 0; b < nb; ++b)
                s_dst[(size_t)b * d_ff + pos] = s[(size_t)b * d_ff + i];
        ++pos;
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

// ------------------------------------------------- per-token threshold path
// The per-token form of Eq. 6: each token's threshold is the quantile of its
// own coefficients. The coefficient kernel first writes the dense
// coefficients (threshold +inf, nothing gathered); k_topk_select finds each
// token's quantile; k_gather_topk thresholds against it and gathers.

constexpr int kTopkThreads = 1024;
constexpr int kTopkPerThread = 32;  // keys per thread: d_ff <= 32768

// One workgroup per token: q = v[lo] + (h - lo)(v[lo + 1] - v[lo]), h = k (n - 1).
// Both order statistics (ranks lo and lo + 1) are found together from
// order-preserving keys held in registers. The first radix pass histograms the
// top 15 significant key bits (sign, exponent and the leading mantissa bits)
// into 32768 LDS bins, so a bin spans a relative width of 2^-7 (2^-6 for
// signed keys) and the bins of the two ranks typically hold a few dozen keys.
// The count each key's atomic returns is its slot within its bin, so those
// keys are placed into an LDS list without a second scan, and the thread
// holding each candidate counts the candidates below it and equal to it: the
// rank of every candidate is exact, ties included. When the two bins hold more
// than kSelList keys (many equal values, or a narrow cluster), two radix passes
// of 11 bits and of the rest fix every remaining bit instead, with one
// histogram per rank once the ranks part. Slots past the row hold a key above
// every finite value, which lands in the top bin. Every VALU instruction per
// key costs the one CU about 16 cycles at 1024 threads, so the per-key work is
// kept to the first pass and the placement. Scans use DPP within waves and
// one barrier across them; fp64 interpolation.
constexpr int kSelBits0 = 15;
constexpr int kSelBins0 = 1 << kSelBits0;               // first pass
constexpr int kSelPer0 = kSelBins0 / kTopkThreads;      // 32 consecutive bins per thread
constexpr int kSelPad0 = kSelPer0 + 4;                  // their LDS words: lanes on different banks
constexpr int kSelWords0 = kSelPad0 * kTopkThreads;
constexpr int kSelBins = 2048;                          // later passes (11 bits)
constexpr int kSelList = 512;                           // candidates ranked by counting
constexpr uint32_t kSelNoKey = 0xffffffffu;             // slot past the row: above every finite key

// LDS word of first-pass bin d
__device__ __forceinline__ uint32_t sel_word(uint32_t d) { return d + 4u * (d >> 5); }

// Order-preserving key of a coefficient: the bits of |c| (am = ~0, |c| keys) or
// the signed float's bits mapped to an unsigned order (am = 0); the select
// kernel's keys, written out there the same way
__device__ __forceinline__ uint32_t sel_key(float c, uint32_t am)
{
    const uint32_t u = __float_as_uint(c);
    const uint32_t sk = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
    return ((u & 0x7fffffffu) & am) | (sk & ~am);
}

// A caller's hook into the select after the first pass, or nothing
struct NoFirstPassHook {
    __device__ __forceinline__ void operator()(uint32_t, uint32_t, int) const {}
};

// inclusive prefix sum over the 64 lanes (DPP row shifts, then row broadcasts)
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v)
{
    v += __builtin_amdgcn_update_dpp(0u, v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0u, v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0u, v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0u, v, 0x118, 0xF, 0xF, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0u, v, kDppBcast15, 0xA, 0xF, false);
    v += __builtin_amdgcn_update_dpp(0u, v, kDppBcast31, 0xC, 0xF, false);
    return v;
}

// Exclusive prefix of v over the workgroup (thread order) and the total; one barrier.
// wsum: LDS [16]. Every thread must call this.
__device__ __forceinline__ void block_scan(uint32_t v, uint32_t *wsum, uint32_t &excl,
                                           uint32_t &total)
{
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const uint32_t inc = wave_incl_scan(v);
    if (lane == kWave - 1)
        wsum[wave] = inc;
    __syncthreads();
    const uint32_t ws = lane < kTopkThreads / kWave ? wsum[lane] : 0u;
    const uint32_t wi = wave_incl_scan(ws);
    const uint32_t before = wave > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)wi, wave - 1) : 0u;
    total = (uint32_t)__builtin_amdgcn_readlane((int)wi, kTopkThreads / kWave - 1);
    excl = before + inc - v;
}

// The bin that holds rank r among this thread's 32 first-pass bins (LDS words
// mine[0, 36), groups of 4 at 4 g summing to gs[g]), given base <= r < base +
// sum(gs): out = {bin, rank within it, its count}. Only the group found is
// read back.
__device__ __forceinline__ void find_bin(const uint32_t *mine, const uint32_t (&gs)[kSelPer0 / 4],
                                         uint32_t base, uint32_t r, uint32_t *out)
{
    uint32_t cum = base, gbase = base;
    int gi = kSelPer0 / 4 - 1;
    bool found = false;
#pragma unroll
    for (int i = 0; i < kSelPer0 / 4; ++i) {
        const bool here = !found && r < cum + gs[i];
        gi = here ? i : gi;
        gbase = here ? cum : gbase;
        found = found || here;
        cum += gs[i];
    }
    const uint4 v = *reinterpret_cast<const uint4 *>(mine + 4 * gi);
    uint32_t o = 3, before = gbase + v.x + v.y + v.z, cnt = v.w;
    if (r < gbase + v.x) {
        o = 0, before = gbase, cnt = v.x;
    } else if (r < gbase + v.x + v.y) {
        o = 1, before = gbase + v.x, cnt = v.y;
    } else if (r < gbase + v.x + v.y + v.z) {
        o = 2, before = gbase + v.x + v.y, cnt = v.z;
    }
    out[0] = kSelPer0 * threadIdx.x + 4 * gi + o;
    out[1] = r - before;
    out[2] = cnt;
}

// The quantile q of one row c[0, n) for the whole workgroup: every thread
// returns the same q (both order statistics end up in every thread, which
// interpolates them itself, so no broadcast is needed). key[] keeps this
// thread's keys, slots threadIdx.x + j * kTopkThreads, for callers that
// flag the row's neurons afterwards. hook(binA, binB, sh0) runs in every
// thread once the first pass has found the bins of ranks lo and lo + 1: a key
// whose first-pass bin (key >> sh0 within the 15 bits) lies below binB is at
// most the rank-lo value, so not above q. ALL_SLOTS: every key slot loads,
// slots past the row reading the zero chunk; otherwise only the slots in use
// load, each under a uniform branch, which saves the select kernel 0.14 us at
// 11008 keys but, in a caller that keeps more registers live, lets the
// compiler wait for each branch's load in turn.
template <int KPT, bool ALL_SLOTS, class Hook>
__device__ __forceinline__ double topk_row(const float *__restrict__ c, int n, int use_abs, double k,
                                           uint32_t (&key)[KPT], const Hook &hook)
{
    constexpr int kWaves = kTopkThreads / kWave;
    extern __shared__ __align__(16) uint32_t sm[];
    uint32_t *hA = sm;                    // first pass: bin d at word sel_word(d); later: [kSelBins] rank lo
    uint32_t *hB = sm + kSelBins;         // later passes: [kSelBins] rank lo + 1, once apart
    uint32_t *list = sm + kSelWords0;     // [kSelList] candidate keys, then kSelNoKey
    uint32_t *dump = list + kSelList;     // [64] stores of the other keys (never read)
    __shared__ uint32_t wsum[kWaves];
    __shared__ uint32_t sel[2][3];        // [rank][bin, rank within bin, keys in bin]
    __shared__ uint32_t val[2];
    const int lane = threadIdx.x % kWave;
    const int jn = (n + kTopkThreads - 1) / kTopkThreads;  // key slots in use (uniform)
    float cv[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const int i = threadIdx.x + j * kTopkThreads;
        if constexpr (ALL_SLOTS) {
            cv[j] = *or_zero(i < n, c + i);
        } else {
            cv[j] = 0.0f;
            if (j < jn)  // uniform
                cv[j] = *or_zero(i < n, c + i);
        }
    }
    for (int i = threadIdx.x; i < kSelWords0 / 4; i += kTopkThreads)
        reinterpret_cast<uint4 *>(sm)[i] = make_uint4(0u, 0u, 0u, 0u);
    if (threadIdx.x < kSelList)
        list[threadIdx.x] = kSelNoKey;
    // sel_key written out: through the helper the compiler no longer folds the
    // absolute value into its select (one more VALU per key, 0.1 us)
    const uint32_t am = use_abs ? ~0u : 0u;
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const uint32_t u = __float_as_uint(cv[j]);
        const uint32_t sk = u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
        key[j] = threadIdx.x + j * kTopkThreads < n ? ((u & 0x7fffffffu) & am) | (sk & ~am)
                                                    : kSelNoKey;
    }
    const double h = k * (double)(n - 1);
    int lo = (int)floor(h);
    if (lo > n - 1)
        lo = n - 1;
    const bool two = lo + 1 < n;  // rank lo + 1 exists
    const uint32_t rlo = (uint32_t)lo, rhi = two ? rlo + 1u : rlo;
    const int sh0 = use_abs ? 16 : 17;  // |c| keys have bit 31 clear
    __syncthreads();

    // first pass; the returned count is the key's slot within its bin
    uint32_t pos[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        pos[j] = 0u;
        if (j < jn)  // uniform
            pos[j] = atomicAdd(hA + sel_word((key[j] >> sh0) & (uint32_t)(kSelBins0 - 1)), 1u);
    }
    __syncthreads();
    {
        const uint32_t *mine = hA + kSelPad0 * threadIdx.x;
        uint32_t gs[kSelPer0 / 4];
        uint32_t sum = 0u;
#pragma unroll
        for (int i = 0; i < kSelPer0 / 4; ++i) {
            const uint4 g = reinterpret_cast<const uint4 *>(mine)[i];
            gs[i] = g.x + g.y + g.z + g.w;
            sum += gs[i];
        }
        uint32_t e, tot;
        block_scan(sum, wsum, e, tot);
        if (rlo >= e && rlo < e + sum)
            find_bin(mine, gs, e, rlo, sel[0]);
        if (rhi >= e && rhi < e + sum)
            find_bin(mine, gs, e, rhi, sel[1]);
        __syncthreads();
    }
    const uint32_t binA = sel[0][0], binB = sel[1][0];
    hook(binA, binB, sh0);
    uint32_t rA = sel[0][1], rB = sel[1][1];
    const uint32_t cA = sel[0][2];
    const bool apart = binA != binB;  // then rank lo is the last of its bin, lo + 1 the first of its
    const uint32_t cnt = cA + (apart ? sel[1][2] : 0u);
    uint32_t kA, kB;
    if (cnt <= (uint32_t)kSelList) {  // uniform
        // bin A's keys fill list[0, cA), bin B's follow
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            if (j < jn) {  // uniform
                const uint32_t d = (key[j] >> sh0) & (uint32_t)(kSelBins0 - 1);
                const uint32_t at = d == binA ? pos[j] : cA + pos[j];
                const bool m = (d == binA || d == binB) && at < (uint32_t)kSelList;
                *(m ? list + at : dump + lane) = key[j];
            }
        }
        __syncthreads();
        const uint32_t tA = rA, tB = apart ? cA + rB : rB;
        if (threadIdx.x < cnt) {
            const uint32_t me = list[threadIdx.x];
            const uint4 *l4 = reinterpret_cast<const uint4 *>(list);
            uint32_t less = 0u, leq = 0u;
#pragma unroll 1
            for (uint32_t j = 0; j < cnt; j += 8) {  // the list is kSelNoKey past cnt
                const uint4 o = l4[j / 4], p = l4[j / 4 + 1];
                less += (o.x < me ? 1u : 0u) + (o.y < me ? 1u : 0u) + (o.z < me ? 1u : 0u) +
                        (o.w < me ? 1u : 0u) + (p.x < me ? 1u : 0u) + (p.y < me ? 1u : 0u) +
                        (p.z < me ? 1u : 0u) + (p.w < me ? 1u : 0u);
                leq += (o.x <= me ? 1u : 0u) + (o.y <= me ? 1u : 0u) + (o.z <= me ? 1u : 0u) +
                       (o.w <= me ? 1u : 0u) + (p.x <= me ? 1u : 0u) + (p.y <= me ? 1u : 0u) +
                       (p.z <= me ? 1u : 0u) + (p.w <= me ? 1u : 0u);
            }
            if (less <= tA && tA < leq)
                val[0] = me;
            if (less <= tB && tB < leq)
                val[1] = me;
        }
        __syncthreads();
        kA = val[0];
        kB = val[1];
    } else {
        // many keys in the bins: radix passes over the remaining bits (11, then
        // the rest); the bins of both histograms are cleared as they are read
        reinterpret_cast<uint4 *>(sm)[threadIdx.x] = make_uint4(0u, 0u, 0u, 0u);  // hA, hB
        __syncthreads();
        uint32_t pA = binA << sh0, pB = binB << sh0;
        uint32_t mask = (uint32_t)(kSelBins0 - 1) << sh0;
#pragma unroll 1
        for (int pass = 1; pass < 3; ++pass) {
            const bool ap = pA != pB;  // uniform
            const int shift = pass == 1 ? sh0 - 11 : 0;
            const uint32_t dmask = pass == 1 ? 0x7ffu : (1u << (sh0 - 11)) - 1u;
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                if (j < jn) {  // uniform
                    const uint32_t d = (key[j] >> shift) & dmask;
                    const uint32_t pk = key[j] & mask;
                    uint32_t *dst = dump + lane;
                    dst = ap && pk == pB ? hB + d : dst;
                    dst = pk == pA ? hA + d : dst;
                    atomicAdd(dst, 1u);
                }
            }
            __syncthreads();
            // thread t owns bins 2t and 2t + 1
            const uint32_t a0 = hA[2 * threadIdx.x], a1 = hA[2 * threadIdx.x + 1];
            hA[2 * threadIdx.x] = 0u;
            hA[2 * threadIdx.x + 1] = 0u;
            uint32_t ea, ta;
            block_scan(a0 + a1, wsum, ea, ta);
            uint32_t b0 = a0, b1 = a1, eb = ea;
            if (ap) {
                b0 = hB[2 * threadIdx.x];
                b1 = hB[2 * threadIdx.x + 1];
                hB[2 * threadIdx.x] = 0u;
                hB[2 * threadIdx.x + 1] = 0u;
                uint32_t tb;
                __syncthreads();  // wsum is read by every thread before it is rewritten
                block_scan(b0 + b1, wsum, eb, tb);
            }
            if (rA >= ea && rA < ea + a0) {
                sel[0][0] = 2 * threadIdx.x, sel[0][1] = rA - ea;
            } else if (rA >= ea + a0 && rA < ea + a0 + a1) {
                sel[0][0] = 2 * threadIdx.x + 1, sel[0][1] = rA - ea - a0;
            }
            if (rB >= eb && rB < eb + b0) {
                sel[1][0] = 2 * threadIdx.x, sel[1][1] = rB - eb;
            } else if (rB >= eb + b0 && rB < eb + b0 + b1) {
                sel[1][0] = 2 * threadIdx.x + 1, sel[1][1] = rB - eb - b0;
            }
            __syncthreads();
            pA |= sel[0][0] << shift;
            pB |= sel[1][0] << shift;
            mask |= dmask << shift;
            rA = sel[0][1];
            rB = sel[1][1];
        }
        kA = pA;  // every bit is fixed
        kB = pB;
    }
    const double v0 = (double)key_value(kA, use_abs);
    const double v1 = (double)key_value(two ? kB : kA, use_abs);
    return v0 + (h - (double)lo) * (v1 - v0);
}

// One workgroup per token. With act set (ideal D-CountDown, |s| keys), the
// workgroup also flags its token's neurons with |c| > q: act starts at 0 (the
// coefficient kernel with threshold +inf wrote it) and every token stores the
// same 1, so the union needs no atomics and no gather kernel follows (s is the
// coefficient itself).
template <int KPT>
__global__ __launch_bounds__(kTopkThreads) void k_topk_select(const float *__restrict__ coef, int ld,
                                                              int n, int use_abs, double k,
                                                              double *__restrict__ q,
                                                              int *__restrict__ act)
{
    uint32_t key[KPT];
    const double qv = topk_row<KPT, false>(coef + (size_t)blockIdx.x * ld, n, use_abs, k, key,
                                    NoFirstPassHook{});
    if (threadIdx.x == 0)
        q[blockIdx.x] = qv;
    if (act) {  // uniform; |s| keys (use_abs): the key's bits are |c|
        const int jn = (n + kTopkThreads - 1) / kTopkThreads;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int i = threadIdx.x + j * kTopkThreads;
            if (j < jn && i < n && (double)__uint_as_float(key[j]) > qv)
                act[i] = 1;
        }
    }
}

static size_t topk_select_lds_bytes()
{
    return ((size_t)kSelWords0 + kSelList + kWave) * 4;
}

// s of one active neuron of a single-projection variant from its second row
// (W_gate for M-CountDown: s = u * SiLU(g); W_up for CATS: s = u * h), the
// first factor from the dense coefficients
template <int B, int NK, bool XREG, bool CATS>
__device__ __forceinline__ void mono_finish(const CoefArgs &a, const Tokens<B, NK, XREG> &tok,
                                            const u32x4 (&w2)[NK], int row, int lane)
{
    float ag[B];
    zero_acc(ag);
    tok.dot(w2, lane, ag);
#pragma unroll
    for (int b = 0; b < B; ++b) {
        const float p = wave_sum(ag[b]);
        const float c = a.coef[(size_t)b * a.d_ff + row];
        if (b < a.nb && lane == 0)
            a.s[(size_t)b * a.d_ff + row] = CATS ? p * c : c * silu(p);
    }
}

// Per-token threshold and gather for batches of 4-8: a workgroup owns kPredRows neurons; its
// first kPredRows threads test them against every token's own threshold
// (|u|, |s| or signed s_hat > q_b, union over the batch) and set act; the
// active neurons are dealt round-robin to the four waves, which gather W_gate
// (mono) or W_gate and W_up (pred) and write s; ideal D-CountDown copies s.
template <int B, int NK, bool XREG, int VARIANT, int NWV = kWavesPerBlock>
__global__ __launch_bounds__(NWV * kWave) void k_gather_topk(const CoefArgs a, const double *__restrict__ q)
{
    extern __shared__ __align__(16) uint32_t xs[];
    __shared__ uint32_t mask;
    constexpr bool kGather = VARIANT != kDualIdeal;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // NWV 8: the first kBlock threads stage the tokens and zero y; all gather
    const bool first = NWV == kWavesPerBlock || threadIdx.x < kBlock;  // wave-uniform
    const int r0 = blockIdx.x * kPredRows;
    Tokens<B, NK, XREG> tok;
    if constexpr (kGather)
        if (XREG || first)
            tok.issue(a.x, a.nb, a.d_model, lane);
    bool act = false;
    const int row = r0 + threadIdx.x;
    if (threadIdx.x < kPredRows && row < a.d_ff) {
#pragma unroll
        for (int b = 0; b < B; ++b) {
            if (b < a.nb) {
                const float c = a.coef[(size_t)b * a.d_ff + row];
                act = act || ((double)(VARIANT == kDualPred ? c : fabsf(c)) > q[b]);
            }
        }
        a.act[row] = act ? 1 : 0;
        if (VARIANT == kDualIdeal && act)
#pragma unroll
            for (int b = 0; b < B; ++b)
                if (b < a.nb)
                    a.s[(size_t)b * a.d_ff + row] = a.coef[(size_t)b * a.d_ff + row];
    }
    const uint64_t m = ballot(act);
    if (threadIdx.x == 0)
        mask = (uint32_t)m;  // the first kPredRows threads are lanes 0..31 of wave 0
    if (first)
        zero_y(a.y, a.nb * a.d_model);
    if constexpr (kGather) {
        if (first)
            tok.write(xs);
        else
            tok.lds = xs;
        __syncthreads();
        uint32_t mm = mask;
        for (int v = 0; v < wave; ++v)
            mm &= mm - 1;
        for (int r = pred_next<NWV>(mm); r >= 0; r = pred_next<NWV>(mm)) {
            u32x4 wg[NK];
            const uint16_t *w2 = VARIANT == kCats ? a.Wu : a.Wg;
            load_row<NK>(wg, w2 + (size_t)(r0 + r) * a.d_model, a.d_model, lane);
            if constexpr (VARIANT == kMono || VARIANT == kCats) {
                mono_finish<B, NK, XREG, VARIANT == kCats>(a, tok, wg, r0 + r, lane);
            } else {
                u32x4 wu[NK];
                load_row<NK>(wu, a.Wu + (size_t)(r0 + r) * a.d_model, a.d_model, lane);
                pred_finish<B, NK, XREG>(a, tok, wg, wu, r0 + r, lane);
            }
        }
    }
}

// Per-token threshold and gather for batches of 1-2: one wave per neuron.
// Lane b reads token b's coefficient and threshold; an inactive neuron's wave
// only writes its flag, an active one issues its token loads with its weight
// rows at once (W_gate for mono, W_gate and W_up for pred) and writes s, so
// every active row of the call is in flight together.
template <int B, int NK, int VARIANT>
__global__ __launch_bounds__(kBlock) void k_gather_topk_w(const CoefArgs a, const double *__restrict__ q)
{
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int row = blockIdx.x * kWavesPerBlock + wave;
    zero_y(a.y, a.nb * a.d_model);
    if (row >= a.d_ff)
        return;
    float cb = 0.0f;
    bool mine = false;
    if (lane < a.nb) {
        cb = a.coef[(size_t)lane * a.d_ff + row];
        mine = (double)(VARIANT == kDualPred ? cb : fabsf(cb)) > q[lane];
    }
    const bool act = ballot(mine) != 0;
    if (lane == 0)
        a.act[row] = act ? 1 : 0;
    if (!act)
        return;
    if constexpr (VARIANT == kDualIdeal) {
        if (lane < a.nb)
            a.s[(size_t)lane * a.d_ff + row] = cb;  // s itself is the coefficient
    } else {
        u32x4 wg[NK];
        load_row<NK>(wg, (VARIANT == kCats ? a.Wu : a.Wg) + (size_t)row * a.d_model, a.d_model,
                     lane);
        u32x4 wu[VARIANT == kDualPred ? NK : 1];
        if constexpr (VARIANT == kDualPred)
            load_row<NK>(wu, a.Wu + (size_t)row * a.d_model, a.d_model, lane);
        Tokens<B, NK, true> tok;
        tok.issue(a.x, a.nb, a.d_model, lane);
        float ag[B];
        zero_acc(ag);
        if constexpr (VARIANT == kDualPred) {
            float au[B];
            zero_acc(au);
            tok.dot2(wg, wu, lane, ag, au);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const float g = wave_sum(ag[b]);
                const float u = wave_sum(au[b]);
                if (b < a.nb && lane == 0)
                    a.s[(size_t)b * a.d_ff + row] = u * silu(g);
            }
        } else {
            tok.dot(wg, lane, ag);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const float p = wave_sum(ag[b]);
                const float cv = __builtin_bit_cast(
                    float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cb), b));
                if (b < a.nb && lane == 0)  // M: u * SiLU(g); CATS: u * h
                    a.s[(size_t)b * a.d_ff + row] = VARIANT == kCats ? p * cv : cv * silu(p);
            }
        }
    }
}

// Per-token threshold, flags and gather of a single token in one launch (mono,
// CATS and, TWO, the W_gate + W_up gather of the predictors). Every workgroup
// (one per CU: the select's LDS fills it) finds the token's quantile itself,
// the same way k_topk_select does, so no workgroup waits for another, and then
// flags its own contiguous slice of at most 64 neurons. Every wave holds the
// whole slice (lane l: neuron l) and takes the same ballots, so work is dealt
// to the 16 waves without a barrier. Once the select's first pass has found
// the bins of ranks lo and lo + 1, every active neuron has its key in the bin
// of rank lo + 1 or above (keys in lower bins are at most the rank-lo value,
// hence at most q), so the slice's candidates are known: the neurons of those
// bins, in order, candidate p going to wave p % 16. Each wave issues the first
// row of its first candidate there, so its HBM round trip overlaps the rest of
// the select; after q it finishes the candidates that are active (the other
// rows stay unused). The predictors' W_up row follows q: both rows in flight
// through the select would spill registers. The token is loaded with the keys
// and copied into LDS the select no longer uses after its first pass. The dot
// products and reductions are those of k_gather_topk_w (the same order, so s
// and act are the same bits). Workgroup 0 stores q.
constexpr int kFusedTopkGrid = 256;        // one workgroup per CU of the MI355X
constexpr int kFusedTopkSlice = kWave;     // neurons per workgroup at most
constexpr int kFusedTokWord = 2 * kSelBins;  // token copy: past the later passes' bins

// position n (from 0) among the set bits of m (n < popcount(m))
__device__ __forceinline__ int nth_set_bit(uint64_t m, int n)
{
    for (int i = 0; i < n; ++i)
        m &= m - 1;
    return __builtin_ctzll(m);
}

template <int NK, bool TWO>
__global__ __launch_bounds__(kTopkThreads) void k_topk_gather1(const CoefArgs a, int cats, double k,
                                                               double *__restrict__ q)
{
    constexpr int KPT = 16;  // d_ff <= kFusedTopkGrid * kFusedTopkSlice
    static_assert(kFusedTokWord + NK * kColsPerLoad / 2 <= kSelWords0, "token copy in LDS");
    constexpr int kWaves = kTopkThreads / kWave;
    extern __shared__ __align__(16) uint32_t sm[];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int per = (a.d_ff + (int)gridDim.x - 1) / (int)gridDim.x;  // <= kWave (host)
    const int lo = blockIdx.x * per;
    const int row = lo + lane;
    const bool mine = lane < per && row < a.d_ff;
    const float c = mine ? a.coef[row] : 0.0f;
    const uint16_t *w1 = cats ? a.Wu : a.Wg;
    constexpr int kTokChunks = NK * kColsPerLoad / 8;  // 16-byte chunks of the padded token
    const bool xt = threadIdx.x < kTokChunks;
    const u32x4 xv = xt ? load16(or_zero((int)threadIdx.x * 8 < a.d_model, a.x + threadIdx.x * 8))
                        : zero16();

    u32x4 wg[NK], wu[TWO ? NK : 1];
    uint64_t cand = 0;  // the slice's candidates: keys in the bin of rank lo + 1 or above
    const auto early = [&](uint32_t, uint32_t binB, int sh0) {
        if (xt)
            *reinterpret_cast<u32x4 *>(sm + kFusedTokWord + 4 * threadIdx.x) = xv;
        const uint32_t key = sel_key(c, TWO ? 0u : ~0u);
        cand = ballot(mine && ((key >> sh0) & (uint32_t)(kSelBins0 - 1)) >= binB);
        if (wave < __builtin_popcountll(cand))
            load_row<NK>(wg, w1 + (size_t)(lo + nth_set_bit(cand, wave)) * a.d_model, a.d_model,
                         lane);
    };
    uint32_t key[KPT];
    const double qv = topk_row<KPT, true>(a.coef, a.d_ff, TWO ? 0 : 1, k, key, early);
    if (blockIdx.x == 0 && threadIdx.x == 0)
        q[0] = qv;
    for (int i = blockIdx.x * kTopkThreads + threadIdx.x; i < a.d_model; i += gridDim.x * kTopkThreads)
        a.y[i] = 0.0f;
    const bool act = mine && (double)(TWO ? c : fabsf(c)) > qv;
    if (wave == 0 && mine)
        a.act[row] = act ? 1 : 0;
    const uint64_t am = ballot(act);  // within cand
    const int ncand = __builtin_popcountll(cand);
    Tokens<1, NK, false> tok;
    tok.lds = sm + kFusedTokWord;  // written before the select's later barriers
    for (int p = wave; p < ncand; p += kWaves) {
        const int i = nth_set_bit(cand, p);
        if (!((am >> i) & 1u))
            continue;
        const int r = lo + i;
        if (p != wave)  // the first candidate's row is in flight already
            load_row<NK>(wg, w1 + (size_t)r * a.d_model, a.d_model, lane);
        if constexpr (TWO)
            load_row<NK>(wu, a.Wu + (size_t)r * a.d_model, a.d_model, lane);
        if constexpr (TWO)
            pred_finish<1, NK, false>(a, tok, wg, wu, r, lane);
        else if (cats)
            mono_finish<1, NK, false, true>(a, tok, wg, r, lane);
        else
            mono_finish<1, NK, false, false>(a, tok, wg, r, lane);
    }
}

// Per-token ideal D-CountDown for a single token in one launch. s is the dense
// coefficient already, so after the select only the flags and the down
// projection remain, and for a neuron range both need nothing but q. Every
// workgroup (one per CU) selects on its own, as k_topk_gather1 does, then
// takes neuron range g and 512-column chunk c of y: it flags the range (the
// workgroups of chunk 0 store the flags), compacts the active neurons into LDS
// in ascending order, keeps kFusedDownRows W_down rows in flight per wave,
// adds the 16 waves' partial sums per column in LDS and adds them to y with
// one fp32 atomic per column (y was zeroed by the coefficient kernel).
// Workgroup 0 stores q.
constexpr int kFusedDownRows = 16;  // W_down rows in flight per wave

__global__ __launch_bounds__(kTopkThreads) void k_topk_down1(const DownArgs a,
                                                             const float *__restrict__ coef,
                                                             int *__restrict__ act_out, double k,
                                                             double *__restrict__ q)
{
    constexpr int kWaves = kTopkThreads / kWave;
    constexpr int U = kFusedDownRows;
    extern __shared__ __align__(16) uint32_t sm[];
    __shared__ int wcnt[kWaves];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    uint32_t key[16];
    const double qv = topk_row<16, true>(coef, a.d_ff, 1, k, key, NoFirstPassHook{});
    if (blockIdx.x == 0 && threadIdx.x == 0)
        q[0] = qv;
    __syncthreads();  // the select's LDS is free from here on
    int *lrow = reinterpret_cast<int *>(sm);                                 // [kTopkThreads]
    float *lsv = reinterpret_cast<float *>(sm + kTopkThreads);               // [kTopkThreads]
    float *red = reinterpret_cast<float *>(sm + 2 * kTopkThreads);           // [kWaves][512]
    const int c = blockIdx.x % a.gc, g = blockIdx.x / a.gc;
    const int r0 = g * a.rows_per_group;  // rows_per_group <= kTopkThreads (host)
    const int r1 = min(a.d_ff, r0 + a.rows_per_group);
    const int row = r0 + threadIdx.x;
    float sv = 0.0f;
    bool act = false;
    if (row < r1) {  // threadIdx.x < rows_per_group included
        sv = coef[row];
        act = (double)fabsf(sv) > qv;
        if (c == 0)
            act_out[row] = act ? 1 : 0;
    }
    const uint64_t m = ballot(act);
    if (lane == 0)
        wcnt[wave] = __popcll(m);
    __syncthreads();
    int base = 0, nl = 0;
    for (int v = 0; v < kWaves; ++v) {
        base += v < wave ? wcnt[v] : 0;
        nl += wcnt[v];
    }
    if (act) {
        const int pos = base + lanes_below(m);
        lrow[pos] = row;
        lsv[pos] = sv;
    }
    __syncthreads();
    if (nl == 0)  // uniform for the workgroup
        return;

    const int col = c * kColsPerLoad + lane * 8;
    const bool colok = col < a.d_model;
    float acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        acc[e] = 0.0f;
    for (int q0 = wave; q0 < nl; q0 += kWaves * U) {
        u32x4 w[U];
#pragma unroll
        for (int t = 0; t < U; ++t) {
            const int r = q0 + t * kWaves;
            w[t] = (r < nl && colok) ? load16_stream(a.Wd + (size_t)lrow[r] * a.d_model + col)
                                     : zero16();
        }
#pragma unroll
        for (int t = 0; t < U; ++t) {
            const int r = q0 + t * kWaves;
            if (r >= nl)
                break;
            const float wf[8] = {bf16_lo(w[t].x), bf16_hi(w[t].x), bf16_lo(w[t].y), bf16_hi(w[t].y),
                                 bf16_lo(w[t].z), bf16_hi(w[t].z), bf16_lo(w[t].w), bf16_hi(w[t].w)};
            const float s_r = lsv[r];
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc[e] = fmaf(s_r, wf[e], acc[e]);
        }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
        red[wave * kColsPerLoad + lane * 8 + e] = acc[e];
    __syncthreads();
    if (threadIdx.x < kColsPerLoad) {
        const int gcol = c * kColsPerLoad + threadIdx.x;
        if (gcol < a.d_model) {
            float v = 0.0f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w)
                v += red[w * kColsPerLoad + threadIdx.x];
            unsafeAtomicAdd(a.y + gcol, v);
        }
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

int tern_row_words(int d_model)
{
    const int nk = col_tile(d_model);
    return kWave * (nk >= 2 ? nk / 2 : 1);
}

// tokens live in registers up to a batch of 2, in LDS beyond
// Whether the coefficient kernels keep the tokens in registers (else one LDS
// copy per workgroup). Registers hold 4 * B * NK VGPRs of tokens: at two tokens
// of d_model 8192 that left the two-row and predictor kernels one wave per SIMD,
// and the LDS copy measured 8-20% faster there (70B shape: ideal D, low-rank and
// ternary predictors, dense); at one token, and two of d_model <= 4096, the
// registers are as fast or faster.
constexpr bool tokens_in_regs(int bt, int nk) { return bt == 1 || (bt == 2 && nk <= 8); }

static size_t token_lds_bytes(int bt, int nk)
{
    return tokens_in_regs(bt, nk) ? 0 : (size_t)bt * nk * kColsPerLoad * 2;
}

size_t down_lds_bytes(int rows_per_group, int bt)
{
    return (size_t)rows_per_group * 4 * (1 + bt) + (size_t)kWavesPerBlock * kColsPerLoad * 4;
}

// Down-kernel grid: 512-column chunks x 56 neuron ranges up to 8 chunks
// (d_model 4096), 64 beyond, of at least 16 neurons each, more ranges when a
// range's lists would not fit in 64 KB of LDS. Measured among 16-128 ranges
// and 128-512-column chunks: at 4096 x 11008 and 4096 x 14336, 56 ranges
// against 64 were 1% faster at 90% sparsity and as fast at 50% and at two
// tokens (48 and fewer lost there); at 8192 x 28672, 64 (48 and 80 slower).
void down_grid(int d_model, int d_ff, int bt, int *gc, int *gr, int *rows_per_group)
{
    *gc = (d_model + kColsPerLoad - 1) / kColsPerLoad;
    int r = *gc <= 8 ? 56 : 64;
    if (r > d_ff / 16)
        r = d_ff / 16;
    if (r < 1)
        r = 1;
    const int max_rows = (int)((65536 - down_lds_bytes(0, bt)) / (4 * (1 + bt))) & ~3;
    if ((d_ff + r - 1) / r > max_rows)
        r = (d_ff + max_rows - 1) / max_rows;
    *rows_per_group = ((d_ff + r - 1) / r + 3) & ~3;  // whole quads of neurons (16-byte loads)
    *gr = (d_ff + *rows_per_group - 1) / *rows_per_group;
}

// waves per block of the batch-4 predictor kernels: a block's ~11 active
// neurons (34% of 32 at 4 tokens) dealt to 8 waves instead of 4 leave each
// wave one or two row pairs to read instead of about three in a row (8B
// layer, low-rank: 38.2 -> 36.6 us at 4 tokens, 33.5 -> 32.5 at 3; ternary:
// 40.6 -> 38.2 and 36.6 -> 34.9). Up to d_model 4096: at 8192 the 8-wave
// kernels take 192 VGPRs, one block per CU.
constexpr int kPredWaves4 = 8;

template <int B, int NK, bool XREG, int LCPR>
static void coef_pred_lcpr(const CoefArgs &a, hipStream_t s)
{
    const int grid = (a.d_ff + kPredRows - 1) / kPredRows;
    const size_t lat_lds = LatentRegs<B, LCPR>::kRegs ? 0 : (size_t)B * a.d_rank * 4;
    // MFMA tiles pay off at 8 tokens; at 4 (a block's ~11 active neurons leave a
    // 16-row tile a third empty) the per-wave v_dot2 gather is faster (8B layer:
    // 38.2 against 41.5 us with the MFMA kernel)
    if constexpr (B >= 8) {
        // weight tiles, then max(latent, 4 x 2 x 16 x 16 partial sums)
        constexpr int STEPS = LatentRegs<B, LCPR>::kRegs ? kWtStepsWide : kWtStepsNarrow;
        const size_t lds = (size_t)kWavesPerBlock * WtShape<STEPS>::kWaveElems * 2 +
                           max(lat_lds, (size_t)kWavesPerBlock * 2 * 256 * 4);
        allow_lds(k_coef_pred_mfma<B, NK, LCPR>, lds);
        k_coef_pred_mfma<B, NK, LCPR><<<grid, kBlock, lds, s>>>(a);
    } else {
        const size_t lds = (XREG ? 0 : (size_t)B * NK * kColsPerLoad * 2) + lat_lds;
        constexpr int NWV = (B == 4 && !XREG && NK <= 8) ? kPredWaves4 : kWavesPerBlock;
        allow_lds(k_coef_pred<B, NK, XREG, LCPR, NWV>, lds);
        k_coef_pred<B, NK, XREG, LCPR, NWV><<<grid, NWV * kWave, lds, s>>>(a);
    }
}

// the predictor kernel is specialised on log2 of the B_t row length in 16-byte chunks
template <int B, int NK, bool XREG>
static hipError_t coef_pred_launch(const CoefArgs &a, hipStream_t s)
{
    switch (a.d_rank) {
    case 8: coef_pred_lcpr<B, NK, XREG, 0>(a, s); break;
    case 16: coef_pred_lcpr<B, NK, XREG, 1>(a, s); break;
    case 32: coef_pred_lcpr<B, NK, XREG, 2>(a, s); break;
    case 64: coef_pred_lcpr<B, NK, XREG, 3>(a, s); break;
    case 128: coef_pred_lcpr<B, NK, XREG, 4>(a, s); break;
    case 256: coef_pred_lcpr<B, NK, XREG, 5>(a, s); break;
    case 512: coef_pred_lcpr<B, NK, XREG, 6>(a, s); break;
    case 1024: coef_pred_lcpr<B, NK, XREG, 7>(a, s); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int B, int NK, bool XREG>
static hipError_t coef_tern_launch(const CoefArgs &a, hipStream_t s)
{
    const int grid = (a.d_ff + kPredRows - 1) / kPredRows;
    if constexpr (B >= 8) {  // MFMA gather, as for the low-rank predictor
        const size_t lds = tern_mfma_front_u32<B, NK>() * 4 + (size_t)kWavesPerBlock * 2 * 256 * 4;
        allow_lds(k_coef_tern_mfma<B, NK>, lds);
        k_coef_tern_mfma<B, NK><<<grid, kBlock, lds, s>>>(a);
    } else {
        const size_t lds = token_lds_bytes(B, NK);
        constexpr int NWV = (B == 4 && !XREG && NK <= 8) ? kPredWaves4 : kWavesPerBlock;
        allow_lds(k_coef_tern<B, NK, XREG, NWV>, lds);
        k_coef_tern<B, NK, XREG, NWV><<<grid, NWV * kWave, lds, s>>>(a);
    }
    return hipGetLastError();
}

template <int B, int NK>
static hipError_t coef_bn(int variant, const CoefArgs &a, hipStream_t s)
{
    constexpr bool XREG = tokens_in_regs(B, NK);
    // The one-row kernel keeps the tokens in registers for one token only: at
    // two they cost it 114 VGPRs (4 waves per SIMD), and the LDS copy measured
    // 8-10% faster at 2 tokens (7B and 70B shapes); the two-row kernel gained
    // nothing from it. At one token of d_model 8192 the registers win although
    // they leave 3 waves per SIMD (LDS copy: 4): 87.1 against 88.6 us per 70B
    // layer; at 4096 the two tie (22.1 us per 7B layer, 5 against 8 waves per
    // SIMD).
    constexpr bool XREG1 = B <= 1;
    const size_t lds = token_lds_bytes(B, NK);
    const size_t lds1 = XREG1 ? 0 : (size_t)B * NK * kColsPerLoad * 2;
    const int grid = (a.d_ff + kWavesPerBlock - 1) / kWavesPerBlock;
    switch (variant) {
    case kMono:
        allow_lds(k_coef_mono<B, NK, XREG1, false>, lds1);
        k_coef_mono<B, NK, XREG1, false><<<grid, kBlock, lds1, s>>>(a);
        break;
    case kCats:
        allow_lds(k_coef_mono<B, NK, XREG1, true>, lds1);
        k_coef_mono<B, NK, XREG1, true><<<grid, kBlock, lds1, s>>>(a);
        break;
    case kDualIdeal:
        allow_lds(k_coef_dual<B, NK, XREG, false>, lds);
        k_coef_dual<B, NK, XREG, false><<<grid, kBlock, lds, s>>>(a);
        break;
    case kDense:
        allow_lds(k_coef_dual<B, NK, XREG, true>, lds);
        k_coef_dual<B, NK, XREG, true><<<grid, kBlock, lds, s>>>(a);
        break;
    case kDualPred:
        return coef_pred_launch<B, NK, XREG>(a, s);
    case kDualTern:
        return coef_tern_launch<B, NK, XREG>(a, s);
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int B>
static hipError_t coef_b(int variant, const CoefArgs &a, hipStream_t s)
{
    switch (col_tile(a.d_model)) {
    case 1: return coef_bn<B, 1>(variant, a, s);
    case 2: return coef_bn<B, 2>(variant, a, s);
    case 4: return coef_bn<B, 4>(variant, a, s);
    case 8: return coef_bn<B, 8>(variant, a, s);
    default:
        // batch * d_model is capped at 32768 by the plan checks: no 8 x 8192 tile
        if constexpr (B * 16 <= 64)
            return coef_bn<B, 16>(variant, a, s);
        return hipErrorInvalidValue;
    }
}

hipError_t launch_coef(int variant, const CoefArgs &a, hipStream_t s)
{
    switch (batch_tile(a.nb)) {
    case 1: return coef_b<1>(variant, a, s);
    case 2: return coef_b<2>(variant, a, s);
    case 4: return coef_b<4>(variant, a, s);
    default: return coef_b<8>(variant, a, s);
    }
}

template <int B>
static hipError_t latent_b(const uint16_t *x, int nb, const uint16_t *At, int d_model, int d_rank,
                           float *lat, hipStream_t s)
{
    switch (col_tile(d_model)) {
    case 1: k_latent<B, 1><<<d_rank, kBlock, 0, s>>>(x, nb, At, d_model, d_rank, lat); break;
    case 2: k_latent<B, 2><<<d_rank, kBlock, 0, s>>>(x, nb, At, d_model, d_rank, lat); break;
    case 4: k_latent<B, 4><<<d_rank, kBlock, 0, s>>>(x, nb, At, d_model, d_rank, lat); break;
    case 8: k_latent<B, 8><<<d_rank, kBlock, 0, s>>>(x, nb, At, d_model, d_rank, lat); break;
    default: k_latent<B, 16><<<d_rank, kBlock, 0, s>>>(x, nb, At, d_model, d_rank, lat); break;
    }
    return hipGetLastError();
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

template <int B>
static hipError_t norm_b(const NormArgs &n, const uint16_t *At, int d_rank, float *lat,
                         hipStream_t s)
{
    const bool fused = At != nullptr;
#define CD_NORM_CASE(NK)                                                                  \
    if (fused)                                                                            \
        k_latent_norm<B, NK><<<d_rank, kBlock, 0, s>>>(n, At, d_rank, lat);               \
    else                                                                                  \
        k_norm<B, NK><<<1, kBlock, 0, s>>>(n);                                            \
    break;
    switch (col_tile(n.d_model)) {
    case 1: CD_NORM_CASE(1)
    case 2: CD_NORM_CASE(2)
    case 4: CD_NORM_CASE(4)
    case 8: CD_NORM_CASE(8)
    default:
        if constexpr (B * 16 <= 64) {  // batch * d_model <= 32768
            CD_NORM_CASE(16)
        }
        return hipErrorInvalidValue;
    }
#undef CD_NORM_CASE
    return hipGetLastError();
}

static hipError_t norm_dispatch(const NormArgs &n, const uint16_t *At, int d_rank, float *lat,
                                hipStream_t s)
{
    switch (batch_tile(n.nb)) {
    case 1: return norm_b<1>(n, At, d_rank, lat, s);
    case 2: return norm_b<2>(n, At, d_rank, lat, s);
    case 4: return norm_b<4>(n, At, d_rank, lat, s);
    default: return norm_b<8>(n, At, d_rank, lat, s);
    }
}

hipError_t launch_norm(const NormArgs &n, hipStream_t s)
{
    return norm_dispatch(n, nullptr, 0, nullptr, s);
}

hipError_t launch_latent_norm(const NormArgs &n, const uint16_t *At, int d_rank, float *lat,
                              hipStream_t s)
{
    return norm_dispatch(n, At, d_rank, lat, s);
}

// MFMA down kernel grid: 128-column chunks and 16 neuron ranges (measured best
// among 4-32 at 4096 x 14336, batches 4 and 8), raised until a range's lists
// fit in 64 KB of LDS
static void down_grid_mfma(int d_model, int d_ff, int bt, int *gc, int *gr, int *rows_per_group)
{
    int r = 16;
    if (r > d_ff / 16)
        r = d_ff / 16;
    if (r < 1)
        r = 1;
    for (;;) {
        const int rows = ((d_ff + r - 1) / r + 3) & ~3;
        if (rows <= kDownScanPasses * 4 * kBlock && down_mfma_lds_bytes(rows, bt) <= 65536)
            break;
        ++r;
    }
    *rows_per_group = ((d_ff + r - 1) / r + 3) & ~3;  // 16-byte aligned flag and s loads
    *gr = (d_ff + *rows_per_group - 1) / *rows_per_group;
    *gc = (d_model + 127) / 128;
}

static bool down_uses_mfma(int bt) { return bt >= kDownMfmaMinBatch; }

// the per-range partial sums of a deterministic call, added into y in range order
static hipError_t reduce_parts(const DownArgs &a, hipStream_t s)
{
    if (!a.part)
        return hipGetLastError();
    const int n = a.nb * a.d_model;
    k_reduce_parts<<<(n + kBlock - 1) / kBlock, kBlock, 0, s>>>(a.part, a.gr, n, a.y);
    return hipGetLastError();
}

size_t down_part_floats(int d_model, int d_ff, int bt)
{
    int gc = 0, gr = 0, rows = 0;
    if (down_uses_mfma(bt))
        down_grid_mfma(d_model, d_ff, bt, &gc, &gr, &rows);
    else
        down_grid(d_model, d_ff, bt, &gc, &gr, &rows);
    return (size_t)gr * bt * d_model;
}

hipError_t launch_down(const DownArgs &args, hipStream_t s)
{
    const int bt = batch_tile(args.nb);
    DownArgs a = args;
    if (down_uses_mfma(bt)) {
        down_grid_mfma(a.d_model, a.d_ff, bt, &a.gc, &a.gr, &a.rows_per_group);
        const size_t lds = down_mfma_lds_bytes(a.rows_per_group, bt);
        const int grid = a.gc * a.gr;
        if (bt == 4) {
            allow_lds(k_down_mfma<4>, lds);
            k_down_mfma<4><<<grid, kBlock, lds, s>>>(a);
        } else {
            allow_lds(k_down_mfma<8>, lds);
            k_down_mfma<8><<<grid, kBlock, lds, s>>>(a);
        }
        const hipError_t e = hipGetLastError();
        return e != hipSuccess ? e : reduce_parts(a, s);
    }
    down_grid(a.d_model, a.d_ff, bt, &a.gc, &a.gr, &a.rows_per_group);
    const size_t lds = down_lds_bytes(a.rows_per_group, bt);
    const int grid = a.gc * a.gr;
    if (bt == 1) {
        allow_lds(k_down<1>, lds);
        k_down<1><<<grid, kBlock, lds, s>>>(a);
    } else {
        allow_lds(k_down<2>, lds);
        k_down<2><<<grid, kBlock, lds, s>>>(a);
    }
    const hipError_t e = hipGetLastError();
    return e != hipSuccess ? e : reduce_parts(a, s);
}

template <int B, int NK>
static hipError_t gather_topk_bn(int variant, const CoefArgs &a, const double *q, hipStream_t s)
{
    constexpr bool XREG = B <= 2;
    if constexpr (XREG) {
        const int wgrid = (a.d_ff + kWavesPerBlock - 1) / kWavesPerBlock;
        switch (variant) {
        case kMono: k_gather_topk_w<B, NK, kMono><<<wgrid, kBlock, 0, s>>>(a, q); break;
        case kCats: k_gather_topk_w<B, NK, kCats><<<wgrid, kBlock, 0, s>>>(a, q); break;
        case kDualIdeal: k_gather_topk_w<B, NK, kDualIdeal><<<wgrid, kBlock, 0, s>>>(a, q); break;
        case kDualPred: k_gather_topk_w<B, NK, kDualPred><<<wgrid, kBlock, 0, s>>>(a, q); break;
        default: return hipErrorInvalidValue;
        }
    } else {
        // 8 waves per block up to d_model 4096, as in the predictor kernels: each
        // wave gathers one or two of a block's active neurons instead of about
        // three in a row (per-token M at 4 tokens 52.4 -> 48.7 us per 7B layer,
        // low-rank predictor at 8 tokens 74.5 -> 69.9 us per 8B layer)
        constexpr int GW = NK <= 8 ? 8 : kWavesPerBlock;
        const size_t lds = token_lds_bytes(B, NK);
        const int grid = (a.d_ff + kPredRows - 1) / kPredRows;
        switch (variant) {
        case kMono:
            allow_lds(k_gather_topk<B, NK, XREG, kMono, GW>, lds);
            k_gather_topk<B, NK, XREG, kMono, GW><<<grid, GW * kWave, lds, s>>>(a, q);
            break;
        case kCats:
            allow_lds(k_gather_topk<B, NK, XREG, kCats, GW>, lds);
            k_gather_topk<B, NK, XREG, kCats, GW><<<grid, GW * kWave, lds, s>>>(a, q);
            break;
        case kDualIdeal:
            k_gather_topk<B, NK, XREG, kDualIdeal><<<grid, kBlock, 0, s>>>(a, q);
            break;
        case kDualPred:
            allow_lds(k_gather_topk<B, NK, XREG, kDualPred, GW>, lds);
            k_gather_topk<B, NK, XREG, kDualPred, GW><<<grid, GW * kWave, lds, s>>>(a, q);
            break;
        default:
            return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

template <int B>
static hipError_t gather_topk_b(int variant, const CoefArgs &a, const double *q, hipStream_t s)
{
    switch (col_tile(a.d_model)) {
    case 1: return gather_topk_bn<B, 1>(variant, a, q, s);
    case 2: return gather_topk_bn<B, 2>(variant, a, q, s);
    case 4: return gather_topk_bn<B, 4>(variant, a, q, s);
    case 8: return gather_topk_bn<B, 8>(variant, a, q, s);
    default:
        if constexpr (B * 16 <= 64)
            return gather_topk_bn<B, 16>(variant, a, q, s);
        return hipErrorInvalidValue;
    }
}

// keys per thread of the select kernel for a row of n coefficients
static int topk_kpt(int n) { return n <= 16 * kTopkThreads ? 16 : 32; }

static void launch_topk_select(const float *coef, int ld, int n, int T, int use_abs, double k,
                               double *q, size_t lds, hipStream_t s, int *act = nullptr)
{
    if (topk_kpt(n) == 16) {
        allow_lds(k_topk_select<16>, lds);
        k_topk_select<16><<<T, kTopkThreads, lds, s>>>(coef, ld, n, use_abs, k, q, act);
    } else {
        allow_lds(k_topk_select<32>, lds);
        k_topk_select<32><<<T, kTopkThreads, lds, s>>>(coef, ld, n, use_abs, k, q, act);
    }
}

template <bool TWO>
static hipError_t topk_gather1_two(int cats, const CoefArgs &a, double k, double *q, int grid,
                                   hipStream_t s)
{
    const size_t lds = topk_select_lds_bytes();
    switch (col_tile(a.d_model)) {
    case 1:
        allow_lds(k_topk_gather1<1, TWO>, lds);
        k_topk_gather1<1, TWO><<<grid, kTopkThreads, lds, s>>>(a, cats, k, q);
        break;
    case 2:
        allow_lds(k_topk_gather1<2, TWO>, lds);
        k_topk_gather1<2, TWO><<<grid, kTopkThreads, lds, s>>>(a, cats, k, q);
        break;
    case 4:
        allow_lds(k_topk_gather1<4, TWO>, lds);
        k_topk_gather1<4, TWO><<<grid, kTopkThreads, lds, s>>>(a, cats, k, q);
        break;
    case 8:
        allow_lds(k_topk_gather1<8, TWO>, lds);
        k_topk_gather1<8, TWO><<<grid, kTopkThreads, lds, s>>>(a, cats, k, q);
        break;
    default:
        return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// whether a call runs select, flags and gather in one launch: one token, d_model
// <= 4096, d_ff within kFusedTopkGrid slices of kFusedTopkSlice neurons
static bool topk_fused(int variant, const CoefArgs &a)
{
    return a.nb == 1 && variant != kDualIdeal && col_tile(a.d_model) <= 8 &&
           a.d_ff <= kFusedTopkGrid * kFusedTopkSlice;
}

// slices of at least 16 neurons, at most kFusedTopkGrid of them
static hipError_t launch_topk_gather1(int variant, const CoefArgs &a, double k, double *q,
                                      hipStream_t s)
{
    if (!topk_fused(variant, a))
        return hipErrorInvalidValue;
    int grid = (a.d_ff + 15) / 16;
    grid = grid < kFusedTopkGrid ? grid : kFusedTopkGrid;
    if ((a.d_ff + grid - 1) / grid > kFusedTopkSlice)
        return hipErrorInvalidValue;
    const int cats = variant == kCats ? 1 : 0;
    return variant == kDualPred ? topk_gather1_two<true>(cats, a, k, q, grid, s)
                                : topk_gather1_two<false>(cats, a, k, q, grid, s);
}

bool topk_down_fused(const DownArgs &a)
{
    return a.nb == 1 && !a.part && col_tile(a.d_model) <= 8 &&
           a.d_ff <= kFusedTopkGrid * kFusedTopkSlice;
}

// 512-column chunks x neuron ranges, kFusedTopkGrid workgroups at most: at most
// 8 chunks (d_model <= 4096), so at least 32 ranges of at most 512 neurons
hipError_t launch_topk_down1(const DownArgs &args, const float *coef, int *act, double k,
                             double *q, hipStream_t s)
{
    if (!topk_down_fused(args))
        return hipErrorInvalidValue;
    DownArgs a = args;
    a.gc = (a.d_model + kColsPerLoad - 1) / kColsPerLoad;
    a.gr = kFusedTopkGrid / a.gc;
    a.rows_per_group = (a.d_ff + a.gr - 1) / a.gr;
    if (a.rows_per_group > kTopkThreads)
        return hipErrorInvalidValue;
    const size_t lds = topk_select_lds_bytes();  // holds the lists and the partial sums too
    static_assert((2 * kTopkThreads + (kTopkThreads / kWave) * kColsPerLoad) * 4 <=
                      ((size_t)kSelWords0 + kSelList + kWave) * 4,
                  "down lists and partial sums within the select's LDS");
    allow_lds(k_topk_down1, lds);
    k_topk_down1<<<a.gc * a.gr, kTopkThreads, lds, s>>>(a, coef, act, k, q);
    return hipGetLastError();
}

hipError_t launch_topk(int variant, const CoefArgs &a, double k, double *q, hipStream_t s)
{
    if (a.d_ff > kTopkThreads * kTopkPerThread)
        return hipErrorInvalidValue;
    if (variant == kDualTern)  // a signed predictor score and the W_gate + W_up gather
        variant = kDualPred;
    // ideal D: s is the dense coefficient, so the select sets the flags itself and
    // the down kernel reads s from a.coef (no gather kernel)
    const bool ideal = variant == kDualIdeal;
    if (topk_fused(variant, a))
        return launch_topk_gather1(variant, a, k, q, s);
    launch_topk_select(a.coef, a.d_ff, a.d_ff, a.nb, variant == kDualPred ? 0 : 1, k, q,
                       topk_select_lds_bytes(), s, ideal ? a.act : nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || ideal)
        return e;
    switch (batch_tile(a.nb)) {
    case 1: return gather_topk_b<1>(variant, a, q, s);
    case 2: return gather_topk_b<2>(variant, a, q, s);
    case 4: return gather_topk_b<4>(variant, a, q, s);
    default: return gather_topk_b<8>(variant, a, q, s);
    }
}

hipError_t launch_export(const int *act, const float *s_rows, int nb, int d_ff, int *idx_dst,
                         int *n_dst, float *s_dst, hipStream_t s)
{
    k_export<<<1, kExportThreads, 0, s>>>(act, s_rows, nb, d_ff, idx_dst, n_dst, s_dst);
    return hipGetLastError();
}

hipError_t launch_select(const float *coef, int ld, int n, int T, int use_abs, double k,
                         double *q_out, hipStream_t s)
{
    if (n <= kTopkThreads * kTopkPerThread) {  // keys fit in registers: the faster select
        launch_topk_select(coef, ld, n, T, use_abs, k, q_out, topk_select_lds_bytes(), s);
    } else {
        allow_lds(k_select_quantile, (size_t)n * 4);
        k_select_quantile<<<T, kSelThreads, (size_t)n * 4, s>>>(coef, ld, n, use_abs, k, q_out);
    }
    return hipGetLastError();
}

// Plain streaming read, a measurement aid: the bandwidth a kernel that reads
// n16 16-byte chunks can reach with the coefficient kernel's load pattern (one
// wave per 8 KB, all eight non-temporal 16-byte loads of a lane issued before
// any use) and no arithmetic but an xor per chunk. A lane stores its fold only
// if it equals a fixed value, which keeps the loads live without a store each.
__global__ __launch_bounds__(kBlock) void k_stream_read(const uint16_t *__restrict__ src,
                                                        size_t n16, uint32_t *sink)
{
    constexpr int kLoads = 8;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const size_t first = ((size_t)blockIdx.x * kWavesPerBlock + wave) * (kWave * kLoads);
    u32x4 w[kLoads];
#pragma unroll
    for (int k = 0; k < kLoads; ++k) {
        const size_t i = first + (size_t)k * kWave + lane;
        w[k] = load16_stream(or_zero(i < n16, src + i * 8));
    }
    uint32_t f = 0u;
#pragma unroll
    for (int k = 0; k < kLoads; ++k)
        f ^= w[k].x ^ w[k].y ^ w[k].z ^ w[k].w;
    if (f == 0x9e3779b9u)
        sink[0] = f;
}

hipError_t launch_stream_read(const void *src, size_t bytes, uint32_t *sink, hipStream_t s)
{
    const size_t n16 = bytes / 16;
    const size_t per_block = (size_t)kBlock * 8;  // 16-byte chunks per workgroup
    const size_t grid = (n16 + per_block - 1) / per_block;
    if (grid == 0 || grid > 0x7fffffffu)
        return hipErrorInvalidValue;
    k_stream_read<<<(unsigned)grid, kBlock, 0, s>>>(static_cast<const uint16_t *>(src), n16, sink);
    return hipGetLastError();
}

hipError_t launch_mean(const double *q, int T, float *out, hipStream_t s)
{
    k_mean<<<1, 64, 0, s>>>(q, T, out);
    return hipGetLastError();
}

} // namespace cdk
