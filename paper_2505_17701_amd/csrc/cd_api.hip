// C ABI of the COUNTDOWN sparse Gated-MLP FFN: plans, argument validation
// and launch sequencing. The arithmetic is in cd_kernels.hip.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/countdown.h"
#include "cd_internal.hpp"

namespace {

constexpr int kMaxDModel = 8192;
constexpr int kMaxBatch = 8;
constexpr int kMaxRank = 1024;
// Token columns of the widest tile a call launches: the batch rounded up to
// 1, 2, 4 or 8 tokens times d_model rounded up to 1, 2, 4, 8 or 16 chunks of
// 512 (batch tiles of 4 and 8 stage x in LDS).
constexpr int kMaxTileCols = 32768;

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_pow2(int v) { return v > 0 && (v & (v - 1)) == 0; }

}  // namespace

struct cd_plan {
    int d_model, d_ff, max_batch, d_rank;
    unsigned flags;
    int device;
    int last_batch;               // of the last FFN call (0 before the first)
    int *act;                     // [d_ff] neuron in IDX
    float *s;                     // [max_batch][d_ff] coefficients s of active neurons
    float *coef;                  // [max_batch][d_ff] dense coefficients (written by every
                                  // call with CD_PLAN_KEEP_COEF, by the per-token path always)
    double *q;                    // [max_batch] per-token thresholds of the last per-token call
    float *lat;                   // [max_batch][d_rank] predictor latent
    float *part;                  // per-range partial sums of y (CD_PLAN_DETERMINISTIC)
    unsigned phases;              // kernels launched per call (CD_PHASE_*)
    bool has_state;               // act / s hold a coefficient kernel's output
    bool s_in_coef;               // the last call's s is coef (ideal D, per-token thresholds)
};

namespace {

cd_status hip_status(hipError_t e) { return e == hipSuccess ? CD_OK : CD_EHIP; }

cd_status launched(hipError_t e) { return e == hipSuccess ? CD_OK : CD_EHIP; }

cd_status check_shape(int d_model, int d_ff, int max_batch, int d_rank)
{
    if (d_model < 8 || d_model % 8 || d_model > kMaxDModel)
        return d_model > kMaxDModel && d_model % 8 == 0 ? CD_EUNSUPPORTED : CD_EINVAL;
    if (d_ff < 8 || d_ff % 8)
        return CD_EINVAL;
    if (max_batch < 1)
        return CD_EINVAL;
    if (max_batch > kMaxBatch)
        return CD_EUNSUPPORTED;
    if (d_rank < 0)
        return CD_EINVAL;
    if (d_rank > 0 && (!is_pow2(d_rank) || d_rank < 8 || d_rank > kMaxRank))
        return CD_EUNSUPPORTED;
    if ((long long)cdk::batch_tile(max_batch) * cdk::col_tile(d_model) * 512 > kMaxTileCols)
        return CD_EUNSUPPORTED;
    return CD_OK;
}

cd_status check_args(int variant, int d_model, int d_ff, int max_batch, int d_rank, const void *x,
                     int B, const void *W_gate, const void *W_up, const void *W_down,
                     const void *A_t, const void *B_t, float thld, const void *y)
{
    cd_status st = check_shape(d_model, d_ff, max_batch, d_rank);
    if (st != CD_OK)
        return st;
    if (variant < CD_VARIANT_MONO || variant > CD_VARIANT_DUAL_TERN)
        return CD_EINVAL;
    if (B < 1 || B > max_batch)
        return CD_EINVAL;
    if (std::isnan(thld))
        return CD_EINVAL;
    const void *req[] = {x, W_gate, W_up, W_down, y};
    for (const void *p : req)
        if (!p || !aligned16(p))
            return CD_EINVAL;
    if (variant == CD_VARIANT_DUAL_PRED) {
        if (!A_t || !B_t || !aligned16(A_t) || !aligned16(B_t) || d_rank == 0)
            return CD_EINVAL;
    } else if (variant == CD_VARIANT_DUAL_TERN) {  // A_t: the packed ternary predictor
        if (!A_t || !aligned16(A_t) || B_t)
            return CD_EINVAL;
    } else if (A_t || B_t) {
        return CD_EINVAL;
    }
    return CD_OK;
}

// CD_VARIANT_* and cdk::Variant share their numbering
int kernel_variant(int variant) { return variant; }

// [a, a + na) and [b, b + nb) share a byte
bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

// A plan's workspace lives on the device current at its creation; a call made
// with another device current would hand that device foreign pointers.
cd_status plan_device_ok(const cd_plan *p)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return CD_EHIP;
    return dev == p->device ? CD_OK : CD_EINVAL;
}

// The outputs of a call (y, and the per-token thresholds q when given) share
// no memory with what it reads: the coefficient kernel zeroes y while other
// workgroups still read x and the weights. Null inputs are skipped.
bool outputs_disjoint(const cd_plan *p, int B, const void *x, const void *Wg, const void *Wu,
                      const void *Wd, const void *At, const void *Bt, const void *Tp,
                      const void *y, const void *q)
{
    const size_t xb = (size_t)B * p->d_model * sizeof(uint16_t);
    const size_t wb = (size_t)p->d_ff * p->d_model * sizeof(uint16_t);
    const size_t yb = (size_t)B * p->d_model * sizeof(float);
    const struct {
        const void *ptr;
        size_t n;
    } in[] = {{x, xb},
              {Wg, wb},
              {Wu, wb},
              {Wd, wb},
              {At, (size_t)p->d_rank * p->d_model * sizeof(uint16_t)},
              {Bt, (size_t)p->d_ff * p->d_rank * sizeof(uint16_t)},
              {Tp, (size_t)p->d_ff * cdk::tern_row_words(p->d_model) * sizeof(uint32_t)}};
    for (const auto &t : in) {
        if (!t.ptr)
            continue;
        if (overlaps(t.ptr, t.n, y, yb) || (q && overlaps(t.ptr, t.n, q, (size_t)B * sizeof(double))))
            return false;
    }
    return !(q && overlaps(q, (size_t)B * sizeof(double), y, yb));
}

cdk::CoefArgs coef_args(cd_plan *p, const uint16_t *x, int B, const uint16_t *Wg,
                        const uint16_t *Wu, const uint16_t *Bt, float thld, float *y,
                        const uint32_t *Tp = nullptr)
{
    cdk::CoefArgs a;
    a.x = x;
    a.nb = B;
    a.Wg = Wg;
    a.Wu = Wu;
    a.Bt = Bt;
    a.lat = p->lat;
    a.Tp = Tp;
    a.d_model = p->d_model;
    a.d_ff = p->d_ff;
    a.d_rank = p->d_rank;
    a.thld = thld;
    a.act = p->act;
    a.s = p->s;
    a.coef = (p->flags & CD_PLAN_KEEP_COEF) ? p->coef : nullptr;
    a.y = y;
    return a;
}

cdk::DownArgs down_args(cd_plan *p, int B, const uint16_t *Wd, float *y)
{
    cdk::DownArgs a;
    a.act = p->act;
    a.s = p->s_in_coef ? p->coef : p->s;
    a.nb = B;
    a.Wd = Wd;
    a.d_model = p->d_model;
    a.d_ff = p->d_ff;
    a.gc = a.gr = a.rows_per_group = 0;  // chosen per batch tile by launch_down
    a.y = y;
    a.part = p->part;
    return a;
}

// The per-neuron workspace no longer describes a finished coefficient kernel
// (a coefficient phase is starting, or a launch of it failed).
void forget_state(cd_plan *p)
{
    p->has_state = false;
    p->last_batch = 0;
    p->s_in_coef = false;
}

// The coefficient phase of a B-token call was enqueued: a down-only call of the
// same batch, and countdown_export_active, may read its workspace.
void keep_state(cd_plan *p, int B, bool s_in_coef)
{
    p->has_state = true;
    p->last_batch = B;
    p->s_in_coef = s_in_coef;
}

// A down-only call reads the flags and coefficients left by the plan's last
// coefficient kernel: there must be one, and it must have run on the same
// batch (its coefficients of later tokens were never written).
bool down_state_ok(const cd_plan *p, int B)
{
    return (p->phases & CD_PHASE_COEF) || (p->has_state && B == p->last_batch);
}

// Tp: the packed ternary predictor (CD_VARIANT_DUAL_TERN only)
cd_status run_ffn(cd_plan *p, int variant, const uint16_t *x, int B, const uint16_t *Wg,
                  const uint16_t *Wu, const uint16_t *Wd, const uint16_t *At, const uint16_t *Bt,
                  float thld, float *y, void *stream, const uint32_t *Tp = nullptr)
{
    if (!p)
        return CD_EINVAL;
    const bool tern = variant == CD_VARIANT_DUAL_TERN;
    if (tern && (At || Bt))
        return CD_EINVAL;
    cd_status st = check_args(variant, p->d_model, p->d_ff, p->max_batch, p->d_rank, x, B, Wg, Wu,
                              Wd, tern ? static_cast<const void *>(Tp) : At, Bt, thld, y);
    if (st != CD_OK)
        return st;
    if (!outputs_disjoint(p, B, x, Wg, Wu, Wd, At, Bt, Tp, y, nullptr))
        return CD_EINVAL;
    if ((st = plan_device_ok(p)) != CD_OK)
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (!down_state_ok(p, B))
        return CD_EINVAL;
    if (p->phases & CD_PHASE_COEF) {
        forget_state(p);
        if (variant == CD_VARIANT_DUAL_PRED) {
            st = launched(cdk::launch_latent(x, B, At, p->d_model, p->d_rank, p->lat, s));
            if (st != CD_OK)
                return st;
        }
        const cdk::CoefArgs ca = coef_args(p, x, B, Wg, Wu, Bt, thld, y, Tp);
        st = launched(cdk::launch_coef(kernel_variant(variant), ca, s));
        if (st != CD_OK)
            return st;
        keep_state(p, B, false);
    }
    if (p->phases & CD_PHASE_DOWN) {
        const cdk::DownArgs da = down_args(p, B, Wd, y);
        st = launched(cdk::launch_down(da, s));
    }
    return st;
}

cd_status run_ffn_residual(cd_plan *p, int variant, const float *h_in, const float *y_prev,
                           float *h_out, float eps, uint16_t *x_out, int B, const uint16_t *Wg,
                           const uint16_t *Wu, const uint16_t *Wd, const uint16_t *At,
                           const uint16_t *Bt, float thld, float *y, void *stream)
{
    if (!p || variant == CD_VARIANT_DUAL_TERN)
        return CD_EINVAL;
    cd_status st = check_args(variant, p->d_model, p->d_ff, p->max_batch, p->d_rank, x_out, B, Wg,
                              Wu, Wd, At, Bt, thld, y);
    if (st != CD_OK)
        return st;
    if (!h_in || !h_out || !aligned16(h_in) || !aligned16(h_out) ||
        (y_prev && !aligned16(y_prev)) || !(eps >= 0.0f) || std::isinf(eps))
        return CD_EINVAL;
    const size_t fb = (size_t)B * p->d_model * sizeof(float);
    const size_t xb = (size_t)B * p->d_model * sizeof(uint16_t);
    // h_in and y_prev are read by every workgroup of the first kernel while h_out and
    // x_out are written, and y is zeroed by the next: only y_prev and y may coincide
    if (overlaps(h_in, fb, h_out, fb) || overlaps(h_in, fb, x_out, xb) ||
        overlaps(h_out, fb, x_out, xb) || overlaps(h_out, fb, y, fb) ||
        overlaps(x_out, xb, y, fb) || overlaps(h_in, fb, y, fb) ||
        (y_prev && (overlaps(y_prev, fb, h_out, fb) || overlaps(y_prev, fb, x_out, xb))))
        return CD_EINVAL;
    if (!outputs_disjoint(p, B, nullptr, Wg, Wu, Wd, At, Bt, nullptr, y, nullptr))
        return CD_EINVAL;
    const void *weights[] = {Wg, Wu, Wd, At, Bt};
    const size_t wsz[] = {(size_t)p->d_ff * p->d_model * 2, (size_t)p->d_ff * p->d_model * 2,
                          (size_t)p->d_ff * p->d_model * 2, (size_t)p->d_rank * p->d_model * 2,
                          (size_t)p->d_ff * p->d_rank * 2};
    for (int i = 0; i < 5; ++i)
        if (weights[i] && (overlaps(weights[i], wsz[i], h_out, fb) ||
                           overlaps(weights[i], wsz[i], x_out, xb)))
            return CD_EINVAL;
    if ((st = plan_device_ok(p)) != CD_OK)
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (!down_state_ok(p, B))
        return CD_EINVAL;
    if (p->phases & CD_PHASE_COEF) {
        forget_state(p);
        cdk::NormArgs n;
        n.h_in = h_in;
        n.y_prev = y_prev;
        n.h_out = h_out;
        n.x_out = x_out;
        n.nb = B;
        n.d_model = p->d_model;
        n.eps = eps;
        if (variant == CD_VARIANT_DUAL_PRED)
            st = launched(cdk::launch_latent_norm(n, At, p->d_rank, p->lat, s));
        else
            st = launched(cdk::launch_norm(n, s));
        if (st != CD_OK)
            return st;
        const cdk::CoefArgs ca = coef_args(p, x_out, B, Wg, Wu, Bt, thld, y);
        st = launched(cdk::launch_coef(kernel_variant(variant), ca, s));
        if (st != CD_OK)
            return st;
        keep_state(p, B, false);
    }
    if (p->phases & CD_PHASE_DOWN) {
        const cdk::DownArgs da = down_args(p, B, Wd, y);
        st = launched(cdk::launch_down(da, s));
    }
    return st;
}

cd_status run_ffn_topk(cd_plan *p, int variant, const uint16_t *x, int B, const uint16_t *Wg,
                       const uint16_t *Wu, const uint16_t *Wd, const uint16_t *At,
                       const uint16_t *Bt, double k, double *thld_out, float *y, void *stream,
                       const uint32_t *Tp = nullptr)
{
    if (!p)
        return CD_EINVAL;
    if (variant != CD_VARIANT_MONO && variant != CD_VARIANT_DUAL_IDEAL &&
        variant != CD_VARIANT_DUAL_PRED && variant != CD_VARIANT_CATS &&
        variant != CD_VARIANT_DUAL_TERN)
        return CD_EINVAL;
    if (!(k >= 0.0 && k <= 1.0) || (thld_out && (reinterpret_cast<uintptr_t>(thld_out) & 7u)))
        return CD_EINVAL;
    const bool tern = variant == CD_VARIANT_DUAL_TERN;
    if (tern && (At || Bt))
        return CD_EINVAL;
    cd_status st = check_args(variant, p->d_model, p->d_ff, p->max_batch, p->d_rank, x, B, Wg, Wu,
                              Wd, tern ? static_cast<const void *>(Tp) : At, Bt, 0.0f, y);
    if (st != CD_OK)
        return st;
    if (p->d_ff > cdk::kTopkMaxDff)
        return CD_EUNSUPPORTED;
    if (!outputs_disjoint(p, B, x, Wg, Wu, Wd, At, Bt, Tp, y, thld_out))
        return CD_EINVAL;
    if ((st = plan_device_ok(p)) != CD_OK)
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (!down_state_ok(p, B))
        return CD_EINVAL;
    if (p->phases & CD_PHASE_COEF) {
        forget_state(p);
        if (variant == CD_VARIANT_DUAL_PRED) {
            st = launched(cdk::launch_latent(x, B, At, p->d_model, p->d_rank, p->lat, s));
            if (st != CD_OK)
                return st;
        }
        // dense coefficients of every neuron (threshold +inf: nothing is gathered yet)
        cdk::CoefArgs ca = coef_args(p, x, B, Wg, Wu, Bt, INFINITY, y, Tp);
        ca.coef = p->coef;
        st = launched(cdk::launch_coef(kernel_variant(variant), ca, s));
        if (st != CD_OK)
            return st;
        double *q = thld_out ? thld_out : p->q;
        if (variant == CD_VARIANT_DUAL_IDEAL && (p->phases & CD_PHASE_DOWN)) {
            // s is the coefficient itself: one token's select, flags and down
            // projection can run as one launch
            cdk::DownArgs da = down_args(p, B, Wd, y);
            da.s = p->coef;
            if (cdk::topk_down_fused(da)) {
                st = launched(cdk::launch_topk_down1(da, p->coef, p->act, k, q, s));
                if (st == CD_OK)
                    keep_state(p, B, true);
                return st;
            }
        }
        st = launched(cdk::launch_topk(kernel_variant(variant), ca, k, q, s));
        if (st != CD_OK)
            return st;
        keep_state(p, B, variant == CD_VARIANT_DUAL_IDEAL);
    }
    if (p->phases & CD_PHASE_DOWN) {
        const cdk::DownArgs da = down_args(p, B, Wd, y);
        st = launched(cdk::launch_down(da, s));
    }
    return st;
}

template <class T>
cd_status dalloc(T **ptr, size_t count)
{
    *ptr = nullptr;
    if (count == 0)
        return CD_OK;
    const hipError_t e = hipMalloc(reinterpret_cast<void **>(ptr), count * sizeof(T));
    if (e == hipSuccess)
        return CD_OK;
    *ptr = nullptr;
    return e == hipErrorOutOfMemory ? CD_ENOMEM : CD_EHIP;
}

void release(cd_plan *p)
{
    void *bufs[] = {p->act, p->s, p->coef, p->lat, p->q, p->part};
    for (void *b : bufs)
        if (b)
            (void)hipFree(b);
    delete p;
}

}  // namespace

extern "C" {

int countdown_abi_version(void) { return COUNTDOWN_ABI_VERSION; }

const char *countdown_status_string(cd_status st)
{
    switch (st) {
    case CD_OK: return "CD_OK: success";
    case CD_EINVAL: return "CD_EINVAL: invalid argument";
    case CD_EUNSUPPORTED: return "CD_EUNSUPPORTED: shape not supported by the kernels";
    case CD_EHIP: return "CD_EHIP: HIP runtime or launch failure";
    case CD_ENOMEM: return "CD_ENOMEM: device allocation failed";
    default: return "unknown countdown status";
    }
}

cd_status countdown_ffn_residual(cd_plan *plan, int variant, const float *h_in, const float *y_prev,
                                float *h_out, float eps, uint16_t *x_out, int B,
                                const uint16_t *W_gate, const uint16_t *W_up,
                                const uint16_t *W_down, const uint16_t *A_t, const uint16_t *B_t,
                                float thld, float *y, void *stream)
{
    if (variant == CD_VARIANT_DENSE)
        thld = -INFINITY;
    return run_ffn_residual(plan, variant, h_in, y_prev, h_out, eps, x_out, B, W_gate, W_up,
                            W_down, A_t, B_t, thld, y, stream);
}

cd_status countdown_ffn_cats(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, float thld, float *y,
                             void *stream)
{
    return run_ffn(plan, CD_VARIANT_CATS, x, B, W_gate, W_up, W_down, nullptr, nullptr, thld, y,
                   stream);
}

cd_status countdown_ffn_topk(cd_plan *plan, int variant, const uint16_t *x, int B,
                             const uint16_t *W_gate, const uint16_t *W_up, const uint16_t *W_down,
                             const uint16_t *A_t, const uint16_t *B_t, double k, double *thld_out,
                             float *y, void *stream)
{
    return run_ffn_topk(plan, variant, x, B, W_gate, W_up, W_down, A_t, B_t, k, thld_out, y,
                        stream);
}

cd_status countdown_check_shape(int d_model, int d_ff, int max_batch, int d_rank)
{
    return check_shape(d_model, d_ff, max_batch, d_rank);
}

cd_status countdown_check_args(int variant, int d_model, int d_ff, int max_batch, int d_rank,
                               const void *x, int B, const void *W_gate, const void *W_up,
                               const void *W_down, const void *A_t, const void *B_t, float thld,
                               const void *y)
{
    return check_args(variant, d_model, d_ff, max_batch, d_rank, x, B, W_gate, W_up, W_down, A_t,
                      B_t, thld, y);
}

cd_status countdown_plan_create(int d_model, int d_ff, int max_batch, int d_rank, unsigned flags,
                                cd_plan **out)
{
    if (!out)
        return CD_EINVAL;
    cd_status st = check_shape(d_model, d_ff, max_batch, d_rank);
    if (st != CD_OK)
        return st;
    if (flags & ~(CD_PLAN_KEEP_COEF | CD_PLAN_DETERMINISTIC))
        return CD_EINVAL;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return CD_EHIP;
    cd_plan *p = new (std::nothrow) cd_plan();
    if (!p)
        return CD_ENOMEM;
    p->d_model = d_model;
    p->d_ff = d_ff;
    p->max_batch = max_batch;
    p->d_rank = d_rank;
    p->flags = flags;
    p->device = dev;
    p->last_batch = 0;
    p->phases = CD_PHASE_ALL;
    p->has_state = false;
    p->s_in_coef = false;
    const size_t mb = (size_t)max_batch;
    st = dalloc(&p->act, (size_t)d_ff);
    if (st == CD_OK) st = dalloc(&p->s, mb * d_ff);
    if (st == CD_OK) st = dalloc(&p->coef, mb * d_ff);
    if (st == CD_OK) st = dalloc(&p->q, mb);
    if (st == CD_OK && d_rank > 0) st = dalloc(&p->lat, mb * d_rank);
    if (st == CD_OK && (flags & CD_PLAN_DETERMINISTIC)) {
        // the largest partial-sum array of any batch tile up to max_batch's
        size_t n = 0;
        for (int bt = 1; bt <= cdk::batch_tile(max_batch); bt *= 2) {
            const size_t f = cdk::down_part_floats(d_model, d_ff, bt);
            n = f > n ? f : n;
        }
        st = dalloc(&p->part, n);
    }
    if (st != CD_OK) {
        release(p);
        return st;
    }
    *out = p;
    return CD_OK;
}

cd_status countdown_plan_destroy(cd_plan *plan)
{
    if (!plan)
        return CD_OK;
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    const bool other = e == hipSuccess && cur != plan->device;
    if (other)
        e = hipSetDevice(plan->device);
    if (e == hipSuccess)
        e = hipDeviceSynchronize();
    release(plan);
    if (other)
        (void)hipSetDevice(cur);
    return hip_status(e);
}

cd_status countdown_ffn_mono(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, float thld, float *y,
                             void *stream)
{
    return run_ffn(plan, CD_VARIANT_MONO, x, B, W_gate, W_up, W_down, nullptr, nullptr, thld, y,
                   stream);
}

cd_status countdown_ffn_dual(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down, const uint16_t *A_t,
                             const uint16_t *B_t, float thld, float *y, void *stream)
{
    if (!plan)
        return CD_EINVAL;
    if ((A_t == nullptr) != (B_t == nullptr))
        return CD_EINVAL;
    const int variant = A_t ? CD_VARIANT_DUAL_PRED : CD_VARIANT_DUAL_IDEAL;
    return run_ffn(plan, variant, x, B, W_gate, W_up, W_down, A_t, B_t, thld, y, stream);
}

cd_status countdown_ffn_dense(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                              const uint16_t *W_up, const uint16_t *W_down, float *y, void *stream)
{
    return run_ffn(plan, CD_VARIANT_DENSE, x, B, W_gate, W_up, W_down, nullptr, nullptr,
                   -INFINITY, y, stream);
}

}  // extern "C"

namespace {

cd_status calibrate(cd_plan *p, int variant, const uint16_t *X, int T, const uint16_t *W_gate,
                    const uint16_t *W_up, const uint16_t *A_t, const uint16_t *B_t,
                    const uint32_t *Tp, double k, float *thld_out, double *q_out, void *stream)
{
    if (!p || !X || !aligned16(X) || T < 1 || !thld_out || !(k >= 0.0 && k <= 1.0))
        return CD_EINVAL;
    if (variant != CD_VARIANT_MONO && variant != CD_VARIANT_DUAL_IDEAL &&
        variant != CD_VARIANT_DUAL_PRED && variant != CD_VARIANT_CATS &&
        variant != CD_VARIANT_DUAL_TERN)
        return CD_EINVAL;
    const bool pred = variant == CD_VARIANT_DUAL_PRED;
    const bool tern = variant == CD_VARIANT_DUAL_TERN;
    if (tern) {
        if (!Tp || !aligned16(Tp))
            return CD_EINVAL;
    } else if (pred) {
        if (!A_t || !B_t || !aligned16(A_t) || !aligned16(B_t) || p->d_rank == 0)
            return CD_EINVAL;
    } else if (variant == CD_VARIANT_CATS) {
        if (!W_gate || !aligned16(W_gate))  // h = SiLU(x.W_gate) needs W_gate only
            return CD_EINVAL;
    } else if (!W_up || !aligned16(W_up) ||
               (variant == CD_VARIANT_DUAL_IDEAL && (!W_gate || !aligned16(W_gate)))) {
        return CD_EINVAL;
    }
    cd_status st = plan_device_ok(p);
    if (st != CD_OK)
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const int tb = p->max_batch;
    float *coef = nullptr, *ybuf = nullptr;
    double *q = nullptr;
    st = dalloc(&coef, (size_t)tb * p->d_ff);
    if (st == CD_OK) st = dalloc(&ybuf, (size_t)tb * p->d_model);
    if (st == CD_OK) st = dalloc(&q, (size_t)T);
    // The coefficient kernels run with thld = +inf (no neuron active) and
    // write the dense coefficient vectors of up to max_batch tokens at a time.
    const uint16_t *wg = W_gate ? W_gate : W_up;
    const uint16_t *wu = W_up ? W_up : W_gate;  // CATS calibration reads W_gate only
    for (int t0 = 0; st == CD_OK && t0 < T; t0 += tb) {
        const int nb = T - t0 < tb ? T - t0 : tb;
        const uint16_t *xb = X + (size_t)t0 * p->d_model;
        if (pred) {
            st = launched(cdk::launch_latent(xb, nb, A_t, p->d_model, p->d_rank, p->lat, s));
            if (st != CD_OK)
                break;
        }
        cdk::CoefArgs a = coef_args(p, xb, nb, wg, wu, B_t, INFINITY, ybuf, Tp);
        a.coef = coef;
        st = launched(cdk::launch_coef(variant, a, s));
        if (st != CD_OK)
            break;
        st = launched(cdk::launch_select(coef, p->d_ff, p->d_ff, nb, pred || tern ? 0 : 1, k,
                                         q + t0, s));
    }
    // the act / s workspace now describes a calibration batch, not an FFN call
    forget_state(p);
    if (st == CD_OK)
        st = hip_status(cdk::launch_mean(q, T, thld_out, s));
    if (st == CD_OK && q_out)
        st = hip_status(hipMemcpyAsync(q_out, q, sizeof(double) * T, hipMemcpyDeviceToDevice, s));
    const hipError_t se = hipStreamSynchronize(s);
    if (st == CD_OK && se != hipSuccess)
        st = CD_EHIP;
    if (coef) (void)hipFree(coef);
    if (ybuf) (void)hipFree(ybuf);
    if (q) (void)hipFree(q);
    return st;
}

}  // namespace

extern "C" {

cd_status countdown_calibrate(cd_plan *p, int variant, const uint16_t *X, int T,
                              const uint16_t *W_gate, const uint16_t *W_up, const uint16_t *A_t,
                              const uint16_t *B_t, double k, float *thld_out, double *q_out,
                              void *stream)
{
    if (variant == CD_VARIANT_DUAL_TERN)  // countdown_calibrate_tern takes the packed predictor
        return CD_EINVAL;
    return calibrate(p, variant, X, T, W_gate, W_up, A_t, B_t, nullptr, k, thld_out, q_out,
                     stream);
}

cd_status countdown_calibrate_tern(cd_plan *p, const uint16_t *X, int T,
                                   const uint32_t *theta_packed, double k, float *thld_out,
                                   double *q_out, void *stream)
{
    return calibrate(p, CD_VARIANT_DUAL_TERN, X, T, nullptr, nullptr, nullptr, nullptr,
                     theta_packed, k, thld_out, q_out, stream);
}

cd_status countdown_ffn_tern(cd_plan *plan, const uint16_t *x, int B, const uint16_t *W_gate,
                             const uint16_t *W_up, const uint16_t *W_down,
                             const uint32_t *theta_packed, float thld, float *y, void *stream)
{
    return run_ffn(plan, CD_VARIANT_DUAL_TERN, x, B, W_gate, W_up, W_down, nullptr, nullptr, thld,
                   y, stream, theta_packed);
}

cd_status countdown_ffn_tern_topk(cd_plan *plan, const uint16_t *x, int B,
                                  const uint16_t *W_gate, const uint16_t *W_up,
                                  const uint16_t *W_down, const uint32_t *theta_packed, double k,
                                  double *thld_out, float *y, void *stream)
{
    return run_ffn_topk(plan, CD_VARIANT_DUAL_TERN, x, B, W_gate, W_up, W_down, nullptr, nullptr,
                        k, thld_out, y, stream, theta_packed);
}

size_t countdown_ternary_words(int d_model, int d_ff)
{
    if (check_shape(d_model, d_ff, 1, 0) != CD_OK)
        return 0;
    return (size_t)d_ff * cdk::tern_row_words(d_model);
}

cd_status countdown_ternary_pack(const int8_t *theta_t, int d_model, int d_ff, uint32_t *packed)
{
    if (!theta_t || !packed || check_shape(d_model, d_ff, 1, 0) != CD_OK)
        return CD_EINVAL;
    const int row_words = cdk::tern_row_words(d_model);
    const int lane_words = row_words / 64;
    for (int i = 0; i < d_ff; ++i) {
        uint32_t *row = packed + (size_t)i * row_words;
        for (int w = 0; w < row_words; ++w)
            row[w] = 0u;
        const int8_t *t = theta_t + (size_t)i * d_model;
        for (int c = 0; c < d_model; ++c) {
            if (t[c] < -1 || t[c] > 1)
                return CD_EINVAL;
            if (t[c] == 0)
                continue;
            const uint32_t code = t[c] > 0 ? 1u : 2u;
            const int j = c / 512, l = (c % 512) / 8, e = c % 8;  // unit, lane, position
            const int m = e / 2;
            // A (even unit): bytes 1 / 3; B (odd unit): bytes 0 / 2; e odd: the upper byte
            const int byte = ((j & 1) ? 0 : 1) + ((e & 1) ? 2 : 0);
            row[l * lane_words + j / 2] |= code << (8 * byte + 2 * m);
        }
    }
    return CD_OK;
}

cd_status countdown_export_active(const cd_plan *p, int32_t *idx_dst, int32_t *n_dst,
                                  float *s_dst, float *coef_dst, void *stream)
{
    if (!p || (coef_dst && !(p->flags & CD_PLAN_KEEP_COEF)) || p->last_batch < 1)
        return CD_EINVAL;
    const cd_status st = plan_device_ok(p);
    if (st != CD_OK)
        return st;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    if (idx_dst || n_dst || s_dst)
        e = cdk::launch_export(p->act, p->s_in_coef ? p->coef : p->s, p->last_batch, p->d_ff,
                               idx_dst, n_dst, s_dst, s);
    if (coef_dst && e == hipSuccess)
        e = hipMemcpyAsync(coef_dst, p->coef, sizeof(float) * (size_t)p->last_batch * p->d_ff,
                           hipMemcpyDeviceToDevice, s);
    return hip_status(e);
}

cd_status countdown_stream_read(const void *src, size_t bytes, uint32_t *sink, void *stream)
{
    if (!src || !aligned16(src) || bytes == 0 || bytes % 16 || !sink ||
        (reinterpret_cast<uintptr_t>(sink) & 3u) ||
        bytes / 16 > (size_t)0x7fffffff * 256 * 8)  // the grid of 256-thread workgroups
        return CD_EINVAL;
    return hip_status(cdk::launch_stream_read(src, bytes, sink, reinterpret_cast<hipStream_t>(stream)));
}

cd_status countdown_plan_set_phases(cd_plan *p, unsigned phases)
{
    if (!p || phases == 0 || (phases & ~CD_PHASE_ALL))
        return CD_EINVAL;
    p->phases = phases;
    return CD_OK;
}

}  // extern "C"

// ------------------------------------------------- entry point without allocation
// countdown_ffn_mono_noalloc keeps the per-neuron workspace of a call (the
// active flags and the coefficients s of the active neurons) in this
// file-scope device array instead of a plan's hipMalloc'd buffers. Each device
// the library runs on holds its own copy until the process ends; its address
// on the current device comes from hipGetSymbolAddress on the first call made
// there (the name itself is a host-side stand-in, never passed to a kernel).
namespace {

constexpr int kNoallocMaxDff = 32768;
constexpr size_t kNoallocActBytes = (size_t)kNoallocMaxDff * sizeof(int);
constexpr size_t kNoallocBytes = kNoallocActBytes + (size_t)kMaxBatch * kNoallocMaxDff * sizeof(float);
constexpr int kNoallocMaxDevices = 64;

}  // namespace

static __device__ __align__(256) unsigned char scratch[kNoallocBytes];

namespace {

std::mutex g_scratch_mutex;
void *g_scratch_ptr[kNoallocMaxDevices];  // per device, set once

// Device address of the scratch array on the current device.
cd_status scratch_on_current_device(int *dev_out, void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess)
        return CD_EHIP;
    if (dev < 0 || dev >= kNoallocMaxDevices)
        return CD_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return CD_EHIP;
        g_scratch_ptr[dev] = p;
    }
    *dev_out = dev;
    *out = g_scratch_ptr[dev];
    return CD_OK;
}

}  // namespace

extern "C" cd_status countdown_ffn_mono_noalloc(const uint16_t *x, int B, const uint16_t *W_gate,
                                                const uint16_t *W_up, const uint16_t *W_down,
                                                int d_model, int d_ff, float thld, float *y,
                                                void *stream)
{
    // the shape and arguments first, on the host (run_ffn checks them again)
    cd_status st = check_args(CD_VARIANT_MONO, d_model, d_ff, B < 1 ? 1 : B, 0, x, B, W_gate,
                              W_up, W_down, nullptr, nullptr, thld, y);
    if (st != CD_OK)
        return st;
    if (d_ff > kNoallocMaxDff)
        return CD_EUNSUPPORTED;
    int dev = -1;
    void *ws = nullptr;
    if ((st = scratch_on_current_device(&dev, &ws)) != CD_OK)
        return st;
    // A plan on the stack whose workspace is the scratch array: act [d_ff], then
    // s [B][d_ff]. The coefficient kernel writes every act and zeroes y, and s is
    // read only where act is set, so nothing needs clearing between calls.
    cd_plan p{};
    p.d_model = d_model;
    p.d_ff = d_ff;
    p.max_batch = B;
    p.d_rank = 0;
    p.flags = 0;
    p.device = dev;
    p.act = static_cast<int *>(ws);
    p.s = reinterpret_cast<float *>(static_cast<unsigned char *>(ws) + kNoallocActBytes);
    p.phases = CD_PHASE_ALL;
    return run_ffn(&p, CD_VARIANT_MONO, x, B, W_gate, W_up, W_down, nullptr, nullptr, thld, y,
                   stream);
}
