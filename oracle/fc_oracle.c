/*
 * Oracle for the data-parallel gradient aggregation + SGD step of FireCaffe
 * (Iandola et al., "FireCaffe: near-linear acceleration of deep neural network
 * training on compute clusters").
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, scalar statement of
 * what the GPU path must compute.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load it.  It shares no source, header,
 * table or helper with the HIP library, and the HIP library never calls it.
 *
 * Build: gcc -O2 -ffp-contract=off (no -ffast-math, default x86-64 SSE
 * rounding: round-to-nearest-even, no flush-to-zero).  Every float operation
 * below is one IEEE-754 binary32 operation rounded once.
 *
 * What it computes, per segment j (one layer's weight or bias block) and
 * element i of that segment:
 *   x_k   = replica k's gradient value, widened to fp32  (Sec. 6
 *           "Implementing efficient data parallel training": each worker
 *           holds the sum of weight gradients over its share of the batch;
 *           16-bit gradient storage is the variant named in Sec. 8.2
 *           "Reducing communication among servers")
 *   s     = sum of x_0..x_{K-1} in binary reduction-tree order (Sec. 6.2
 *           "Reduction tree", Fig. 3b, Eq. 4: branching factor 2, depth
 *           log2(p)); the parameter-server variant adds the K vectors one
 *           after another at one node (Sec. 6.1 "Parameter server", Fig. 3a)
 *   ga    = s * (1/batch)   (Sec. 6: the aggregate equals what one GPU would
 *           sum over the whole batch)
 *   d     = ga + wd_j * w
 *   v'    = mu * v + lr_j * d
 *   w'    = w - v'          (batched SGD with momentum and weight decay,
 *           Sec. 3 "Preliminaries" and Sec. 7.1 item 2; the paper gives mu and
 *           wd but prints no update formula -- this is the Caffe solver
 *           convention it claims compatibility with, a reading)
 *   dst_k = w'  for every worker k  (Fig. 3 caption: the result travels back
 *           down the tree to every worker)
 *
 * Readings where the paper is silent:
 *   - tree shape for K not a power of two: pair neighbours level by level and
 *     carry an odd last node up unchanged (Sec. 6.2 only fixes the power-of-
 *     two case);
 *   - leaf k is replica k; operand order inside a pair is irrelevant because
 *     IEEE addition is commutative;
 *   - lr_j = lr * lr_mult_j and wd_j = wd * decay_mult_j, each one fp32
 *     rounding; c = 1.0f / (float)batch, one fp32 rounding.
 *
 * Learning-rate policies (Sec. 7.2: step -- divide by 10 at fixed points --
 * and the rate scaled with the batch; Sec. 7.3: polynomial decay with power
 * 0.5): rate = base_lr * (batch / base_batch) * factor(iter), evaluated in
 * double and rounded to float once.
 *
 * Pins (see tests): fp16 widening against numpy over all 65536 patterns; K=1
 * identity; all-ones sums to K; integer-valued inputs give the exact integer
 * sum in both orders; the pairwise-summation error bound against an exact
 * sum; a hand-worked example separating tree from linear order; an
 * independent numpy level-pairing; SGD closed forms and an fp64 evaluation.
 * The SGD convention and the averaging divisor are readings of the paper
 * (parity unpinned as to which convention the paper's authors ran).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
    uint64_t offset;   /* first element of the segment, in elements */
    uint64_t length;   /* number of elements */
    float lr_mult;     /* per-segment learning-rate multiplier */
    float decay_mult;  /* per-segment weight-decay multiplier */
} orc_segment;

enum { ORC_F32 = 0, ORC_F16 = 1 };
enum { ORC_TREE = 0, ORC_LINEAR = 1 };

/* IEEE-754 binary16 -> binary32, from the format's definition:
 *   exponent field 0      : (-1)^s * m * 2^-24            (zero / subnormal)
 *   exponent field 1..30  : (-1)^s * (1024 + m) * 2^(e-25)
 *   exponent field 31     : infinity (m = 0) or NaN (m != 0)
 * Every binary16 value is exactly representable in binary32. */
float orc_f16_to_f32(uint16_t h)
{
    int s = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int m = h & 0x3ff;
    float mag;
    if (e == 0)
        mag = ldexpf((float)m, -24);
    else if (e == 31)
        mag = (m == 0) ? INFINITY : NAN;
    else
        mag = ldexpf((float)(1024 + m), e - 25);
    return s ? -mag : mag;
}

static float leaf(const void* const* grads, int dtype, int k, uint64_t i)
{
    if (dtype == ORC_F16)
        return orc_f16_to_f32(((const uint16_t*)grads[k])[i]);
    return ((const float*)grads[k])[i];
}

/* Binary reduction tree over L[0..n-1] (Sec. 6.2, Fig. 3b): at each level neighbours
 * 2m and 2m+1 are added; an odd last entry moves up unchanged.  L is scratch
 * and is overwritten. */
static float tree_sum(float* L, int n)
{
    while (n > 1) {
        int pairs = n / 2;
        for (int m = 0; m < pairs; ++m)
            L[m] = L[2 * m] + L[2 * m + 1];
        if (n % 2 == 1) {
            L[pairs] = L[n - 1];
            n = pairs + 1;
        } else {
            n = pairs;
        }
    }
    return L[0];
}

/* Parameter-server order (Sec. 6.1, Fig. 3a): one node adds the workers' vectors one
 * after another. */
static float linear_sum(const float* L, int n)
{
    float s = L[0];
    for (int k = 1; k < n; ++k)
        s = s + L[k];
    return s;
}

static int check(const orc_segment* segs, int nseg, int K, int dtype, int order)
{
    if (nseg < 0 || (nseg > 0 && segs == NULL)) return -1;
    if (K < 1) return -1;
    if (dtype != ORC_F32 && dtype != ORC_F16) return -1;
    if (order != ORC_TREE && order != ORC_LINEAR) return -1;
    return 0;
}

/* out[i] = sum over k of widen(grads[k][i]), for every element i of every
 * segment; elements outside the segments are not touched. */
int orc_tree_reduce(const orc_segment* segs, int nseg, int K, int dtype, int order,
                    const void* const* grads, float* out)
{
    if (check(segs, nseg, K, dtype, order)) return -1;
    float* L = (float*)malloc(sizeof(float) * (size_t)K);
    if (!L) return -5;
    for (int j = 0; j < nseg; ++j) {
        for (uint64_t i = segs[j].offset; i < segs[j].offset + segs[j].length; ++i) {
            for (int k = 0; k < K; ++k)
                L[k] = leaf(grads, dtype, k, i);
            out[i] = (order == ORC_TREE) ? tree_sum(L, K) : linear_sum(L, K);
        }
    }
    free(L);
    return 0;
}

/* One momentum-SGD step with weight decay from the raw (unscaled) sum g. */
int orc_sgd_step(const orc_segment* segs, int nseg, float* w, float* v, const float* g,
                 float lr, float mu, float wd, int batch)
{
    if (nseg < 0 || (nseg > 0 && segs == NULL) || batch < 1) return -1;
    const float c = 1.0f / (float)batch;
    for (int j = 0; j < nseg; ++j) {
        const float lr_j = lr * segs[j].lr_mult;
        const float wd_j = wd * segs[j].decay_mult;
        for (uint64_t i = segs[j].offset; i < segs[j].offset + segs[j].length; ++i) {
            const float ga = g[i] * c;
            const float decay = wd_j * w[i];
            const float d = ga + decay;
            const float mom = mu * v[i];
            const float step = lr_j * d;
            const float vn = mom + step;
            const float wn = w[i] - vn;
            v[i] = vn;
            w[i] = wn;
        }
    }
    return 0;
}

/* dst[k][i] = src[i] for every worker k and every segment element i. */
int orc_broadcast(const orc_segment* segs, int nseg, int K, const float* src, float* const* dst)
{
    if (nseg < 0 || (nseg > 0 && segs == NULL) || K < 1) return -1;
    for (int k = 0; k < K; ++k)
        for (int j = 0; j < nseg; ++j)
            for (uint64_t i = segs[j].offset; i < segs[j].offset + segs[j].length; ++i)
                dst[k][i] = src[i];
    return 0;
}

/* Learning rate at iteration `iter` (kind 0 fixed, 1 step, 2 poly); returns
 * -1 for an invalid policy or iteration. */
int orc_lr_at(int kind, double base_lr, int base_batch, double gamma, int64_t stepsize, int64_t max_iter,
              double power, int64_t iter, int batch, float* lr)
{
    if (iter < 0 || batch < 1 || base_batch < 0 || !(base_lr >= 0.0)) return -1;
    double factor;
    if (kind == 0) {
        factor = 1.0;
    } else if (kind == 1) {
        if (stepsize < 1 || !(gamma > 0.0)) return -1;
        int64_t drops = iter / stepsize;              /* completed steps of the schedule */
        factor = pow(gamma, (double)drops);
    } else if (kind == 2) {
        if (max_iter < 1 || iter > max_iter || !(power >= 0.0)) return -1;
        double remaining = 1.0 - (double)iter / (double)max_iter;
        factor = pow(remaining, power);
    } else {
        return -1;
    }
    double scale = (base_batch > 0) ? (double)batch / (double)base_batch : 1.0;
    *lr = (float)(base_lr * scale * factor);
    return 0;
}

/* The whole step: reduce, then SGD on the sum, then optionally keep the raw
 * sum in out and send w' to every worker.  `scratch` holds n_total floats
 * (n_total = one past the last segment element) and receives the raw sum. */
int orc_step(const orc_segment* segs, int nseg, int K, int dtype, int order,
             const void* const* grads, float* w, float* v, float lr, float mu, float wd,
             int batch, float* scratch, float* out, float* const* bcast_dst)
{
    int rc = orc_tree_reduce(segs, nseg, K, dtype, order, grads, scratch);
    if (rc) return rc;
    rc = orc_sgd_step(segs, nseg, w, v, scratch, lr, mu, wd, batch);
    if (rc) return rc;
    if (out) {
        for (int j = 0; j < nseg; ++j)
            for (uint64_t i = segs[j].offset; i < segs[j].offset + segs[j].length; ++i)
                out[i] = scratch[i];
    }
    if (bcast_dst)
        rc = orc_broadcast(segs, nseg, K, w, bcast_dst);
    return rc;
}
