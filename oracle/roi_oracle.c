/*
 * roi_oracle.c -- plain CPU oracle for multi-level RoIAlign (and RoI max pooling,
 * deformable RoI pooling, non-maximum suppression).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that the GPU library can be
 * checked against something slow and obviously correct.  Only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it; the product path
 * never calls it, and it shares no source, header or helper with the HIP code.
 *
 * What it computes (MMDetection, arXiv 1906.07155):
 *   - §3.1 (model representation), RoIExtractor / SingleRoIExtractor: each RoI's
 *     features are pooled from the level of the FPN pyramid that matches the
 *     RoI's size, by a RoI pooling operator.
 *   - §2 (supported frameworks) cites Mask R-CNN for the RoIAlign operator used
 *     by the Faster/Mask R-CNN + FPN detectors; §1 says the bbox and mask
 *     operations run on GPUs; §3.2 (training pipeline) runs forward and backward
 *     every iteration, so the backward (the transpose) is needed too.
 *   - The same sections name RoIPool (Fast R-CNN's max pooling over quantized
 *     bins) as the other RoI pooling operator; oracle_roi_pool_fwd/bwd below
 *     follow its usual definition.
 *   - §2 also lists DCN (deformable RoI pooling) and DCNv2 (its modulated form):
 *     oracle_deform_roi_pool_fwd/bwd move every RoIAlign bin by a learned offset
 *     and scale it by a learned modulation; the definition is written above them.
 *   - §1 runs the bbox operations on the GPU and §2 lists Soft-NMS next to greedy
 *     NMS: oracle_nms (greedy) and oracle_nms_batched (per-category greedy or
 *     Soft-NMS with linear or Gaussian decay) select the proposals.
 *   The paper does not spell the operator out.  The definition below is the
 *   standard one (bilinear sampling on a regular grid inside each bin, averaged),
 *   and every convention the paper leaves open is fixed the same way as in the
 *   library's public header; the list of such readings lives with the design notes.
 *
 * Two geometry modes:
 *   MODE_MATH   (0): every coordinate and weight in double precision.  Used by
 *                    the invariant tests (closed forms, adjoint, brute force).
 *   MODE_PARITY (1): the sample geometry in IEEE binary32 with one rounding per
 *                    operation in the order written below (build with
 *                    -ffp-contract=off so no multiply-add is fused); products and
 *                    sums of feature values in double.  This is what the GPU is
 *                    compared against.
 *
 * Layout: every feature level is a dense double array [N][C][H][W]; RoIs are
 * float [K][5] = (batch_index, x1, y1, x2, y2) in input-image pixels; the output
 * is a dense double array [K][C][PH][PW].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define MODE_MATH 0
#define MODE_PARITY 1

/* Adaptive sampling grids (sampling_ratio == 0) are capped at this many samples
 * per bin side, matching the limit the GPU library documents for the same case. */
#define ADAPTIVE_GRID_CAP 64

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------- */
/* Level assignment (§3.1: the pyramid level matched to the RoI's size).      */
/* ------------------------------------------------------------------------- */

/* Threshold form of the FPN rule: the level is the number of thresholds
 * (finest_scale * 2^j)^2, j = 1 .. L-1, that the box area reaches.  Area and
 * thresholds are binary32 values, one rounding per operation.  With box_plus1 the
 * box is a range of whole pixels with both ends inside (the convention of the
 * pre-"aligned" detectors): each side is (x2 - x1) + 1, the difference rounded
 * first. */
void oracle_level_map(const float *rois, int64_t K, int32_t num_levels,
                      float finest_scale, int32_t box_plus1, int32_t *out)
{
    for (int64_t k = 0; k < K; ++k) {
        const float *r = rois + 5 * k;
        float w = r[3] - r[1];
        float h = r[4] - r[2];
        if (box_plus1) {
            w = w + 1.0f;
            h = h + 1.0f;
        }
        float area = w * h;
        int32_t lvl = 0;
        for (int32_t j = 1; j < num_levels; ++j) {
            float side = finest_scale * (float)(1 << j);
            float thr = side * side;
            if (area >= thr)
                lvl += 1;
        }
        out[k] = lvl;
    }
}

/* The logarithmic statement of the same rule, in double precision:
 * floor(log2(sqrt(w*h) / finest_scale)), clamped to [0, L-1].  Agrees with the
 * threshold form everywhere except within rounding distance of a threshold. */
void oracle_level_map_log2(const float *rois, int64_t K, int32_t num_levels,
                           double finest_scale, int32_t box_plus1, int32_t *out)
{
    for (int64_t k = 0; k < K; ++k) {
        const float *r = rois + 5 * k;
        double w = (double)r[3] - (double)r[1] + (box_plus1 ? 1.0 : 0.0);
        double h = (double)r[4] - (double)r[2] + (box_plus1 ? 1.0 : 0.0);
        double a = w * h;
        int32_t lvl = 0;
        if (a > 0.0) {
            double l = floor(log2(sqrt(a) / finest_scale));
            if (l > (double)(num_levels - 1))
                l = (double)(num_levels - 1);
            if (l > 0.0)
                lvl = (int32_t)l;
        }
        out[k] = lvl;
    }
}

/* ------------------------------------------------------------------------- */
/* One axis of the sampling grid.                                             */
/* ------------------------------------------------------------------------- */

typedef struct {
    int valid;      /* sample lies inside [-1, size] */
    int lo, hi;     /* the two neighbouring pixel indices after clamping */
    double w_lo;    /* weight of pixel lo (1 - frac) */
    double w_hi;    /* weight of pixel hi (frac) */
} axis_tap;

typedef struct {
    double start_d, bin_d;   /* MODE_MATH */
    float start_f, bin_f;    /* MODE_PARITY */
    int grid;                /* samples per bin along this axis */
    double len_d;            /* box length on the level (after the minimum size) */
    float len_f;
} axis_geom;

static int grid_from_bin(int sampling_ratio, double bin)
{
    if (sampling_ratio > 0)
        return sampling_ratio;
    if (!(bin > 0.0))
        return 0;
    double g = ceil(bin);
    if (g > (double)ADAPTIVE_GRID_CAP)
        g = (double)ADAPTIVE_GRID_CAP;
    return (int)g;
}

/* RoI extent along one axis -> start, bin size and grid.
 * start = c1*scale - off, end = c2*scale - off, length = end - start (at least 1
 * pixel when not aligned), bin = length / P. */
static axis_geom axis_setup(int mode, float c1, float c2, float scale, int aligned,
                            int P, int sampling_ratio)
{
    axis_geom g;
    memset(&g, 0, sizeof(g));
    if (mode == MODE_PARITY) {
        const float off = aligned ? 0.5f : 0.0f;
        float s = c1 * scale;
        s = s - off;
        float e = c2 * scale;
        e = e - off;
        float len = e - s;
        if (!aligned)
            len = fmaxf(len, 1.0f);
        float bin = len / (float)P;
        g.len_f = len;
        g.len_d = (double)len;
        g.start_f = s;
        g.bin_f = bin;
        g.start_d = (double)s;
        g.bin_d = (double)bin;
        g.grid = grid_from_bin(sampling_ratio, (double)bin);
    } else {
        const double off = aligned ? 0.5 : 0.0;
        double s = (double)c1 * (double)scale - off;
        double e = (double)c2 * (double)scale - off;
        double len = e - s;
        if (!aligned)
            len = fmax(len, 1.0);
        double bin = len / (double)P;
        g.len_d = len;
        g.start_d = s;
        g.bin_d = bin;
        g.grid = grid_from_bin(sampling_ratio, bin);
    }
    return g;
}

/* Sample i (0 <= i < grid) of bin p: coordinate start + p*bin + (i + 1/2)*bin/grid,
 * then the bilinear neighbours on a map of `size` pixels. */
static axis_tap axis_sample(int mode, const axis_geom *g, int p, int i, int size)
{
    axis_tap t;
    t.valid = 0;
    t.lo = t.hi = 0;
    t.w_lo = t.w_hi = 0.0;
    if (mode == MODE_PARITY) {
        float a = (float)p * g->bin_f;
        float b = g->start_f + a;
        float c = (float)i + 0.5f;
        float d = c * g->bin_f;
        float e = d / (float)g->grid;
        float v = b + e;
        if (v < -1.0f || v > (float)size)
            return t;
        v = fmaxf(v, 0.0f);
        int lo = (int)v;
        int hi;
        if (lo >= size - 1) {
            lo = size - 1;
            hi = size - 1;
            v = (float)lo;
        } else {
            hi = lo + 1;
        }
        float frac = v - (float)lo;
        float rest = 1.0f - frac;
        t.valid = 1;
        t.lo = lo;
        t.hi = hi;
        t.w_lo = (double)rest;
        t.w_hi = (double)frac;
    } else {
        double v = g->start_d + (double)p * g->bin_d +
                   ((double)i + 0.5) * g->bin_d / (double)g->grid;
        if (v < -1.0 || v > (double)size)
            return t;
        v = fmax(v, 0.0);
        int lo = (int)v;
        int hi;
        if (lo >= size - 1) {
            lo = size - 1;
            hi = size - 1;
            v = (double)lo;
        } else {
            hi = lo + 1;
        }
        double frac = v - (double)lo;
        t.valid = 1;
        t.lo = lo;
        t.hi = hi;
        t.w_lo = 1.0 - frac;
        t.w_hi = frac;
    }
    return t;
}

/* Batch index: column 0 of the RoI, truncated toward zero; -1 when it does not
 * name an image of the batch (such a RoI yields zeros and no gradient). */
static int roi_batch(float v, int64_t N)
{
    float t = truncf(v);
    if (!(t >= 0.0f) || !(t < (float)N))
        return -1;
    return (int)t;
}

/* ------------------------------------------------------------------------- */
/* Forward: out[k,c,ph,pw] = (1/count) * sum over samples and bilinear corners */
/* ------------------------------------------------------------------------- */

void oracle_roi_align_fwd(const double *const *feats, const int64_t *dims,
                          const float *scales, int32_t num_levels,
                          const float *rois, int64_t K, const int32_t *roi_levels,
                          int32_t PH, int32_t PW, int32_t sampling_ratio,
                          int32_t aligned, int32_t mode, double *out)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < K; ++k) {
        double *o = out + k * C * PH * PW;
        for (int64_t e = 0; e < C * PH * PW; ++e)
            o[e] = 0.0;
        const float *r = rois + 5 * k;
        int lvl = roi_levels ? roi_levels[k] : 0;
        if (lvl < 0 || lvl >= num_levels)
            continue;
        const int64_t N = dims[4 * lvl + 0];
        const int64_t H = dims[4 * lvl + 2];
        const int64_t W = dims[4 * lvl + 3];
        int b = roi_batch(r[0], N);
        if (b < 0)
            continue;
        axis_geom gx = axis_setup(mode, r[1], r[3], scales[lvl], aligned, PW, sampling_ratio);
        axis_geom gy = axis_setup(mode, r[2], r[4], scales[lvl], aligned, PH, sampling_ratio);
        int count = gy.grid * gx.grid;
        if (count < 1)
            count = 1;
        for (int64_t c = 0; c < C; ++c) {
            const double *F = feats[lvl] + ((int64_t)b * C + c) * H * W;
            for (int ph = 0; ph < PH; ++ph) {
                for (int pw = 0; pw < PW; ++pw) {
                    double sum = 0.0;
                    for (int iy = 0; iy < gy.grid; ++iy) {
                        axis_tap ty = axis_sample(mode, &gy, ph, iy, (int)H);
                        for (int ix = 0; ix < gx.grid; ++ix) {
                            axis_tap tx = axis_sample(mode, &gx, pw, ix, (int)W);
                            if (!ty.valid || !tx.valid)
                                continue;
                            sum += ty.w_lo * tx.w_lo * F[ty.lo * W + tx.lo];
                            sum += ty.w_lo * tx.w_hi * F[ty.lo * W + tx.hi];
                            sum += ty.w_hi * tx.w_lo * F[ty.hi * W + tx.lo];
                            sum += ty.w_hi * tx.w_hi * F[ty.hi * W + tx.hi];
                        }
                    }
                    o[(c * PH + ph) * PW + pw] = sum / (double)count;
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------- */
/* Backward: the transpose of the forward.  grad_feats[l][b,c,y,x] +=          */
/* grad_out[k,c,ph,pw] * weight / count for every sample and corner that the   */
/* forward reads.  Accumulates into grad_feats (the caller clears them).       */
/* Channels are independent, so the loop over channels is the parallel one and */
/* every channel plane is written by one thread in a fixed order.             */
/* ------------------------------------------------------------------------- */

void oracle_roi_align_bwd(const double *grad_out, double *const *grad_feats,
                          const int64_t *dims, const float *scales,
                          int32_t num_levels, const float *rois, int64_t K,
                          const int32_t *roi_levels, int32_t PH, int32_t PW,
                          int32_t sampling_ratio, int32_t aligned, int32_t mode)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        for (int64_t k = 0; k < K; ++k) {
            const float *r = rois + 5 * k;
            int lvl = roi_levels ? roi_levels[k] : 0;
            if (lvl < 0 || lvl >= num_levels)
                continue;
            const int64_t N = dims[4 * lvl + 0];
            const int64_t H = dims[4 * lvl + 2];
            const int64_t W = dims[4 * lvl + 3];
            int b = roi_batch(r[0], N);
            if (b < 0)
                continue;
            axis_geom gx = axis_setup(mode, r[1], r[3], scales[lvl], aligned, PW, sampling_ratio);
            axis_geom gy = axis_setup(mode, r[2], r[4], scales[lvl], aligned, PH, sampling_ratio);
            int count = gy.grid * gx.grid;
            if (count < 1)
                count = 1;
            double *G = grad_feats[lvl] + ((int64_t)b * C + c) * H * W;
            const double *g = grad_out + (k * C + c) * PH * PW;
            for (int ph = 0; ph < PH; ++ph) {
                for (int pw = 0; pw < PW; ++pw) {
                    double gv = g[ph * PW + pw] / (double)count;
                    for (int iy = 0; iy < gy.grid; ++iy) {
                        axis_tap ty = axis_sample(mode, &gy, ph, iy, (int)H);
                        for (int ix = 0; ix < gx.grid; ++ix) {
                            axis_tap tx = axis_sample(mode, &gx, pw, ix, (int)W);
                            if (!ty.valid || !tx.valid)
                                continue;
                            G[ty.lo * W + tx.lo] += gv * ty.w_lo * tx.w_lo;
                            G[ty.lo * W + tx.hi] += gv * ty.w_lo * tx.w_hi;
                            G[ty.hi * W + tx.lo] += gv * ty.w_hi * tx.w_lo;
                            G[ty.hi * W + tx.hi] += gv * ty.w_hi * tx.w_hi;
                        }
                    }
                }
            }
        }
    }
}

/* ------------------------------------------------------------------------- */
/* RoI max pooling -- the RoIPool of Fast R-CNN, the other RoI pooling        */
/* operator besides RoIAlign that the detectors of §2 / §3.1 use.              */
/*                                                                             */
/* Geometry, binary32, one rounding per operation in this order:               */
/*   start_x = roundf(x1 * scale), end_x = roundf(x2 * scale)  (halves away    */
/*   from zero); the box spans w = max(end_x - start_x + 1, 1) pixels (both    */
/*   ends inclusive); bin width bw = w / PW.  Bin column pw covers pixels      */
/*   [floor(pw * bw), ceil((pw + 1) * bw)) shifted by start_x and clipped to   */
/*   [0, W]; rows likewise.                                                     */
/* Output: the largest value in the bin; scanning rows top to bottom and each  */
/* row left to right, a value replaces the current one only if strictly larger */
/* (so the first maximum wins and a NaN is never chosen).  An empty bin gives  */
/* 0 and argmax -1; a non-empty bin that holds no comparable value gives       */
/* -FLT_MAX and argmax -1.  argmax = y * W + x of the chosen pixel.            */
/* Backward: every output gradient is added to its argmax pixel (none for -1). */
/* ------------------------------------------------------------------------- */

#define ORACLE_FLT_MAX 3.4028234663852886e38

typedef struct {
    int lo, hi;   /* [lo, hi) after clipping */
} pool_range;

static pool_range pool_bin(float c1, float c2, float scale, int P, int p, int size)
{
    float s = roundf(c1 * scale);
    float e = roundf(c2 * scale);
    float len = e - s;
    len = len + 1.0f;
    if (len < 1.0f)
        len = 1.0f;
    float bin = len / (float)P;
    float a = (float)p * bin;
    float b = (float)(p + 1) * bin;
    int lo = (int)floorf(a) + (int)s;
    int hi = (int)ceilf(b) + (int)s;
    pool_range r;
    r.lo = lo < 0 ? 0 : (lo > size ? size : lo);
    r.hi = hi < 0 ? 0 : (hi > size ? size : hi);
    return r;
}

void oracle_roi_pool_fwd(const double *const *feats, const int64_t *dims,
                         const float *scales, int32_t num_levels,
                         const float *rois, int64_t K, const int32_t *roi_levels,
                         int32_t PH, int32_t PW, double *out, int32_t *argmax)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < K; ++k) {
        double *o = out + k * C * PH * PW;
        int32_t *am = argmax + k * C * PH * PW;
        for (int64_t e = 0; e < C * PH * PW; ++e) {
            o[e] = 0.0;
            am[e] = -1;
        }
        const float *r = rois + 5 * k;
        int lvl = roi_levels ? roi_levels[k] : 0;
        if (lvl < 0 || lvl >= num_levels)
            continue;
        const int64_t N = dims[4 * lvl + 0];
        const int64_t H = dims[4 * lvl + 2];
        const int64_t W = dims[4 * lvl + 3];
        int b = roi_batch(r[0], N);
        if (b < 0)
            continue;
        for (int64_t c = 0; c < C; ++c) {
            const double *F = feats[lvl] + ((int64_t)b * C + c) * H * W;
            for (int ph = 0; ph < PH; ++ph) {
                pool_range ry = pool_bin(r[2], r[4], scales[lvl], PH, ph, (int)H);
                for (int pw = 0; pw < PW; ++pw) {
                    pool_range rx = pool_bin(r[1], r[3], scales[lvl], PW, pw, (int)W);
                    const int64_t e = (c * PH + ph) * PW + pw;
                    if (ry.hi <= ry.lo || rx.hi <= rx.lo)
                        continue;   /* empty bin: 0, -1 */
                    double best = -ORACLE_FLT_MAX;
                    int32_t where = -1;
                    for (int y = ry.lo; y < ry.hi; ++y)
                        for (int x = rx.lo; x < rx.hi; ++x)
                            if (F[y * W + x] > best) {
                                best = F[y * W + x];
                                where = (int32_t)(y * W + x);
                            }
                    o[e] = best;
                    am[e] = where;
                }
            }
        }
    }
}

void oracle_roi_pool_bwd(const double *grad_out, const int32_t *argmax,
                         double *const *grad_feats, const int64_t *dims,
                         int32_t num_levels, const float *rois, int64_t K,
                         const int32_t *roi_levels, int32_t PH, int32_t PW)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        for (int64_t k = 0; k < K; ++k) {
            int lvl = roi_levels ? roi_levels[k] : 0;
            if (lvl < 0 || lvl >= num_levels)
                continue;
            const int64_t N = dims[4 * lvl + 0];
            const int64_t H = dims[4 * lvl + 2];
            const int64_t W = dims[4 * lvl + 3];
            int b = roi_batch(rois[5 * k], N);
            if (b < 0)
                continue;
            double *G = grad_feats[lvl] + ((int64_t)b * C + c) * H * W;
            for (int e = 0; e < PH * PW; ++e) {
                const int64_t i = (k * C + c) * PH * PW + e;
                if (argmax[i] >= 0 && argmax[i] < H * W)
                    G[argmax[i]] += grad_out[i];
            }
        }
    }
}

/* ------------------------------------------------------------------------- */
/* Deformable RoI pooling -- DCN's deformable RoI pooling and its modulated    */
/* form from DCNv2, listed among the general modules of §2.  Each bin of the   */
/* RoIAlign grid above is moved by a learned offset, given normalized to the   */
/* box size: the shift of bin (ph, pw) is                                      */
/*   dx = (gamma * offset[k,0,ph,pw]) * len_x,  dy = (gamma * offset[k,1,ph,pw]) * len_y */
/* (len = the box length on the level, as in the RoIAlign setup), and it is   */
/* added to the bin start before the within-bin term:                          */
/*   x = ((x0 + pw*bw) + dx) + ((ix + 1/2)*bw) / gw                            */
/* (binary32, one rounding per operation, in parity mode).  Cut, clamp and     */
/* bilinear weights are RoIAlign's.  The modulated form multiplies the bin     */
/* average by mask[k,ph,pw]:  out = mask * (sum of weighted taps) / count.     */
/*                                                                             */
/* Gradients (the operator is piecewise bilinear in the shift):               */
/*   feature: grad_F += g * mask / count * corner weight (as RoIAlign's);      */
/*   offset x: sum over channels and valid samples of                          */
/*       g * mask / count * dV/dx * gamma * len_x,                             */
/*     dV/dx = hy*(F[yl,xh] - F[yl,xl]) + ly*(F[yh,xh] - F[yh,xl]) where the    */
/*     sample is not clamped along x (0 <= x and xl < W-1), else 0;           */
/*     offset y likewise with dV/dy = hx*(F[yh,xl] - F[yl,xl]) + lx*(F[yh,xh] - F[yl,xh]); */
/*   mask: sum over channels of g * (sum of weighted taps) / count.           */
/* ------------------------------------------------------------------------- */

typedef struct {
    axis_tap t;
    int slope;   /* 1 when the value is bilinear in this coordinate (not clamped) */
} deform_tap;

static deform_tap deform_sample(int mode, const axis_geom *g, float shift_f, double shift_d,
                                int p, int i, int size)
{
    deform_tap d;
    d.slope = 0;
    d.t.valid = 0;
    d.t.lo = d.t.hi = 0;
    d.t.w_lo = d.t.w_hi = 0.0;
    if (mode == MODE_PARITY) {
        float pos = (float)p * g->bin_f;
        float b = g->start_f + pos;
        float b2 = b + shift_f;
        float half = (float)i + 0.5f;
        float e0 = half * g->bin_f;
        float e = e0 / (float)g->grid;
        float v = b2 + e;
        if (!(v >= -1.0f) || v > (float)size)
            return d;
        d.slope = v >= 0.0f;
        v = fmaxf(v, 0.0f);
        int lo = (int)v;
        int hi;
        if (lo >= size - 1) {
            lo = size - 1;
            hi = size - 1;
            v = (float)lo;
            d.slope = 0;
        } else {
            hi = lo + 1;
        }
        float frac = v - (float)lo;
        float rest = 1.0f - frac;
        d.t.valid = 1;
        d.t.lo = lo;
        d.t.hi = hi;
        d.t.w_lo = (double)rest;
        d.t.w_hi = (double)frac;
    } else {
        const double within = (0.5 + (double)i) * g->bin_d / (double)g->grid;
        double v = g->start_d + (double)p * g->bin_d + shift_d + within;
        if (!(v >= -1.0) || v > (double)size)
            return d;
        d.slope = v >= 0.0;
        v = fmax(v, 0.0);
        int lo = (int)v;
        int hi;
        if (lo >= size - 1) {
            lo = size - 1;
            hi = size - 1;
            v = (double)lo;
            d.slope = 0;
        } else {
            hi = lo + 1;
        }
        double frac = v - (double)lo;
        d.t.valid = 1;
        d.t.lo = lo;
        d.t.hi = hi;
        d.t.w_lo = 1.0 - frac;
        d.t.w_hi = frac;
    }
    return d;
}

/* Shift of one bin along one axis, in both precisions. */
static void deform_shift(int mode, const axis_geom *g, float gamma, float off, float *sf,
                         double *sd)
{
    if (mode == MODE_PARITY) {
        float a = gamma * off;
        float b = a * g->len_f;
        *sf = b;
        *sd = (double)b;
    } else {
        *sf = 0.0f;
        *sd = (double)gamma * (double)off * g->len_d;
    }
}

typedef struct {
    int ok;              /* RoI names a valid level and image */
    int lvl, b;
    int64_t H, W;
    axis_geom gx, gy;
    int count;
} deform_roi;

static deform_roi deform_roi_setup(int mode, const int64_t *dims, const float *scales,
                                   int32_t num_levels, const float *r, const int32_t *roi_levels,
                                   int64_t k, int32_t PH, int32_t PW, int32_t sampling_ratio,
                                   int32_t aligned)
{
    deform_roi d;
    memset(&d, 0, sizeof(d));
    d.lvl = roi_levels ? roi_levels[k] : 0;
    if (d.lvl < 0 || d.lvl >= num_levels)
        return d;
    const int64_t N = dims[4 * d.lvl + 0];
    d.H = dims[4 * d.lvl + 2];
    d.W = dims[4 * d.lvl + 3];
    d.b = roi_batch(r[0], N);
    if (d.b < 0)
        return d;
    d.gx = axis_setup(mode, r[1], r[3], scales[d.lvl], aligned, PW, sampling_ratio);
    d.gy = axis_setup(mode, r[2], r[4], scales[d.lvl], aligned, PH, sampling_ratio);
    d.count = d.gy.grid * d.gx.grid;
    if (d.count < 1)
        d.count = 1;
    d.ok = 1;
    return d;
}

void oracle_deform_roi_pool_fwd(const double *const *feats, const int64_t *dims,
                                const float *scales, int32_t num_levels,
                                const float *rois, int64_t K, const int32_t *roi_levels,
                                int32_t PH, int32_t PW, int32_t sampling_ratio,
                                int32_t aligned, const float *offset, const float *mask,
                                float gamma, int32_t mode, double *out)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < K; ++k) {
        double *o = out + k * C * PH * PW;
        for (int64_t e = 0; e < C * PH * PW; ++e)
            o[e] = 0.0;
        deform_roi d = deform_roi_setup(mode, dims, scales, num_levels, rois + 5 * k,
                                        roi_levels, k, PH, PW, sampling_ratio, aligned);
        if (!d.ok)
            continue;
        for (int ph = 0; ph < PH; ++ph) {
            for (int pw = 0; pw < PW; ++pw) {
                const int64_t bin = (int64_t)ph * PW + pw;
                float sxf, syf;
                double sxd, syd;
                deform_shift(mode, &d.gx, gamma, offset[(k * 2 + 0) * PH * PW + bin], &sxf, &sxd);
                deform_shift(mode, &d.gy, gamma, offset[(k * 2 + 1) * PH * PW + bin], &syf, &syd);
                const double m = mask ? (double)mask[k * PH * PW + bin] : 1.0;
                for (int64_t c = 0; c < C; ++c) {
                    const double *F = feats[d.lvl] + ((int64_t)d.b * C + c) * d.H * d.W;
                    double sum = 0.0;
                    for (int iy = 0; iy < d.gy.grid; ++iy) {
                        deform_tap ty = deform_sample(mode, &d.gy, syf, syd, ph, iy, (int)d.H);
                        for (int ix = 0; ix < d.gx.grid; ++ix) {
                            deform_tap tx = deform_sample(mode, &d.gx, sxf, sxd, pw, ix, (int)d.W);
                            if (!ty.t.valid || !tx.t.valid)
                                continue;
                            sum += ty.t.w_lo * tx.t.w_lo * F[ty.t.lo * d.W + tx.t.lo];
                            sum += ty.t.w_lo * tx.t.w_hi * F[ty.t.lo * d.W + tx.t.hi];
                            sum += ty.t.w_hi * tx.t.w_lo * F[ty.t.hi * d.W + tx.t.lo];
                            sum += ty.t.w_hi * tx.t.w_hi * F[ty.t.hi * d.W + tx.t.hi];
                        }
                    }
                    o[c * PH * PW + bin] = m * (sum / (double)d.count);
                }
            }
        }
    }
}

/* Backward.  grad_feats (accumulated into; the caller clears them) in parallel over
 * channels; grad_offset [K][2][PH][PW] and grad_mask [K][PH][PW] (written) in
 * parallel over RoIs.  scale_offset / scale_mask (may be NULL) receive the same sums
 * taken over the absolute values of every term, the scale of their rounding error. */
void oracle_deform_roi_pool_bwd(const double *grad_out, const double *const *feats,
                                double *const *grad_feats, const int64_t *dims,
                                const float *scales, int32_t num_levels, const float *rois,
                                int64_t K, const int32_t *roi_levels, int32_t PH, int32_t PW,
                                int32_t sampling_ratio, int32_t aligned, const float *offset,
                                const float *mask, float gamma, int32_t mode,
                                double *grad_offset, double *grad_mask, double *scale_offset,
                                double *scale_mask)
{
    const int64_t C = dims[1];
#pragma omp parallel for schedule(static)
    for (int64_t c = 0; c < C; ++c) {
        for (int64_t k = 0; k < K; ++k) {
            deform_roi d = deform_roi_setup(mode, dims, scales, num_levels, rois + 5 * k,
                                            roi_levels, k, PH, PW, sampling_ratio, aligned);
            if (!d.ok)
                continue;
            double *G = grad_feats[d.lvl] + ((int64_t)d.b * C + c) * d.H * d.W;
            const double *g = grad_out + (k * C + c) * PH * PW;
            for (int ph = 0; ph < PH; ++ph) {
                for (int pw = 0; pw < PW; ++pw) {
                    const int64_t bin = (int64_t)ph * PW + pw;
                    float sxf, syf;
                    double sxd, syd;
                    deform_shift(mode, &d.gx, gamma, offset[(k * 2 + 0) * PH * PW + bin], &sxf, &sxd);
                    deform_shift(mode, &d.gy, gamma, offset[(k * 2 + 1) * PH * PW + bin], &syf, &syd);
                    const double m = mask ? (double)mask[k * PH * PW + bin] : 1.0;
                    const double gv = g[bin] * m / (double)d.count;
                    for (int iy = 0; iy < d.gy.grid; ++iy) {
                        deform_tap ty = deform_sample(mode, &d.gy, syf, syd, ph, iy, (int)d.H);
                        for (int ix = 0; ix < d.gx.grid; ++ix) {
                            deform_tap tx = deform_sample(mode, &d.gx, sxf, sxd, pw, ix, (int)d.W);
                            if (!ty.t.valid || !tx.t.valid)
                                continue;
                            G[ty.t.lo * d.W + tx.t.lo] += gv * ty.t.w_lo * tx.t.w_lo;
                            G[ty.t.lo * d.W + tx.t.hi] += gv * ty.t.w_lo * tx.t.w_hi;
                            G[ty.t.hi * d.W + tx.t.lo] += gv * ty.t.w_hi * tx.t.w_lo;
                            G[ty.t.hi * d.W + tx.t.hi] += gv * ty.t.w_hi * tx.t.w_hi;
                        }
                    }
                }
            }
        }
    }
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t k = 0; k < K; ++k) {
        for (int64_t e = 0; e < PH * PW; ++e) {
            grad_offset[(k * 2 + 0) * PH * PW + e] = 0.0;
            grad_offset[(k * 2 + 1) * PH * PW + e] = 0.0;
            if (grad_mask)
                grad_mask[k * PH * PW + e] = 0.0;
            if (scale_offset) {
                scale_offset[(k * 2 + 0) * PH * PW + e] = 0.0;
                scale_offset[(k * 2 + 1) * PH * PW + e] = 0.0;
            }
            if (scale_mask)
                scale_mask[k * PH * PW + e] = 0.0;
        }
        deform_roi d = deform_roi_setup(mode, dims, scales, num_levels, rois + 5 * k,
                                        roi_levels, k, PH, PW, sampling_ratio, aligned);
        if (!d.ok)
            continue;
        for (int ph = 0; ph < PH; ++ph) {
            for (int pw = 0; pw < PW; ++pw) {
                const int64_t bin = (int64_t)ph * PW + pw;
                float sxf, syf;
                double sxd, syd;
                deform_shift(mode, &d.gx, gamma, offset[(k * 2 + 0) * PH * PW + bin], &sxf, &sxd);
                deform_shift(mode, &d.gy, gamma, offset[(k * 2 + 1) * PH * PW + bin], &syf, &syd);
                const double m = mask ? (double)mask[k * PH * PW + bin] : 1.0;
                const double jx = (double)gamma * (mode == MODE_PARITY ? (double)d.gx.len_f : d.gx.len_d);
                const double jy = (double)gamma * (mode == MODE_PARITY ? (double)d.gy.len_f : d.gy.len_d);
                double ox = 0.0, oy = 0.0, om = 0.0, sx = 0.0, sy = 0.0, sm = 0.0;
                for (int64_t c = 0; c < C; ++c) {
                    const double *F = feats[d.lvl] + ((int64_t)d.b * C + c) * d.H * d.W;
                    const double gc = grad_out[(k * C + c) * PH * PW + bin];
                    double dvx = 0.0, dvy = 0.0, avx = 0.0, avy = 0.0, sum = 0.0, asum = 0.0;
                    for (int iy = 0; iy < d.gy.grid; ++iy) {
                        deform_tap ty = deform_sample(mode, &d.gy, syf, syd, ph, iy, (int)d.H);
                        for (int ix = 0; ix < d.gx.grid; ++ix) {
                            deform_tap tx = deform_sample(mode, &d.gx, sxf, sxd, pw, ix, (int)d.W);
                            if (!ty.t.valid || !tx.t.valid)
                                continue;
                            const double v11 = F[ty.t.lo * d.W + tx.t.lo];
                            const double v12 = F[ty.t.lo * d.W + tx.t.hi];
                            const double v21 = F[ty.t.hi * d.W + tx.t.lo];
                            const double v22 = F[ty.t.hi * d.W + tx.t.hi];
                            sum += ty.t.w_lo * tx.t.w_lo * v11 + ty.t.w_lo * tx.t.w_hi * v12 +
                                   ty.t.w_hi * tx.t.w_lo * v21 + ty.t.w_hi * tx.t.w_hi * v22;
                            asum += fabs(ty.t.w_lo * tx.t.w_lo * v11) + fabs(ty.t.w_lo * tx.t.w_hi * v12) +
                                    fabs(ty.t.w_hi * tx.t.w_lo * v21) + fabs(ty.t.w_hi * tx.t.w_hi * v22);
                            if (tx.slope) {
                                dvx += ty.t.w_lo * (v12 - v11) + ty.t.w_hi * (v22 - v21);
                                avx += fabs(ty.t.w_lo * (v12 - v11)) + fabs(ty.t.w_hi * (v22 - v21));
                            }
                            if (ty.slope) {
                                dvy += tx.t.w_lo * (v21 - v11) + tx.t.w_hi * (v22 - v12);
                                avy += fabs(tx.t.w_lo * (v21 - v11)) + fabs(tx.t.w_hi * (v22 - v12));
                            }
                        }
                    }
                    ox += gc * m / (double)d.count * dvx * jx;
                    oy += gc * m / (double)d.count * dvy * jy;
                    om += gc * sum / (double)d.count;
                    sx += fabs(gc * m / (double)d.count * jx) * avx;
                    sy += fabs(gc * m / (double)d.count * jy) * avy;
                    sm += fabs(gc) * asum / (double)d.count;
                }
                grad_offset[(k * 2 + 0) * PH * PW + bin] = ox;
                grad_offset[(k * 2 + 1) * PH * PW + bin] = oy;
                if (grad_mask)
                    grad_mask[k * PH * PW + bin] = om;
                if (scale_offset) {
                    scale_offset[(k * 2 + 0) * PH * PW + bin] = sx;
                    scale_offset[(k * 2 + 1) * PH * PW + bin] = sy;
                }
                if (scale_mask)
                    scale_mask[k * PH * PW + bin] = sm;
            }
        }
    }
}

/* ------------------------------------------------------------------------- */
/* Non-maximum suppression -- the step that turns scored proposals into the    */
/* RoIs above (the paper runs its bbox operations, NMS among them, on the GPU, */
/* §1).  Greedy: boxes are ranked by score, highest first (IEEE total order of */
/* the score bits, -0 below +0, NaN last; equal scores by index); in rank order */
/* a box is kept unless a kept box of the same category overlaps it with       */
/* IoU > threshold.  IoU is decided in binary32, one rounding per operation:   */
/*   iw = max(min(x2a, x2b) - max(x1a, x1b), 0), ih likewise, inter = iw * ih, */
/*   area = (x2 - x1) * (y2 - y1), uni = (area_a + area_b) - inter,            */
/*   iou = inter / uni;  suppress iff iou > threshold                          */
/* (a NaN IoU, e.g. two zero-area boxes, suppresses nothing).                 */
/* ------------------------------------------------------------------------- */

static uint32_t nms_rank_key(float s)
{
    uint32_t u;
    memcpy(&u, &s, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return 0xffffffffu;                    /* NaN: after every number */
    uint32_t asc = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ~asc;                               /* larger score, smaller key */
}

typedef struct {
    uint32_t key;
    int32_t idx;
} nms_item;

static int nms_item_cmp(const void *pa, const void *pb)
{
    const nms_item *a = (const nms_item *)pa, *b = (const nms_item *)pb;
    if (a->key != b->key)
        return a->key < b->key ? -1 : 1;
    return a->idx < b->idx ? -1 : (a->idx > b->idx ? 1 : 0);
}

float oracle_box_iou(const float *a, const float *b)
{
    float ix1 = fmaxf(a[0], b[0]);
    float iy1 = fmaxf(a[1], b[1]);
    float ix2 = fminf(a[2], b[2]);
    float iy2 = fminf(a[3], b[3]);
    float iw = ix2 - ix1;
    float ih = iy2 - iy1;
    iw = fmaxf(iw, 0.0f);
    ih = fmaxf(ih, 0.0f);
    float inter = iw * ih;
    float wa = a[2] - a[0];
    float ha = a[3] - a[1];
    float wb = b[2] - b[0];
    float hb = b[3] - b[1];
    float area_a = wa * ha;
    float area_b = wb * hb;
    float sum = area_a + area_b;
    float uni = sum - inter;
    return inter / uni;
}

/* Kept box indices in rank order (at most max_keep of them); returns their number. */
int32_t oracle_nms(const float *boxes, const float *scores, const int32_t *cats, int32_t N,
                   float threshold, int32_t max_keep, int32_t *keep_out)
{
    nms_item *it = (nms_item *)malloc(sizeof(nms_item) * (size_t)(N > 0 ? N : 1));
    char *removed = (char *)calloc((size_t)(N > 0 ? N : 1), 1);
    for (int32_t i = 0; i < N; ++i) {
        it[i].key = nms_rank_key(scores[i]);
        it[i].idx = i;
    }
    qsort(it, (size_t)N, sizeof(nms_item), nms_item_cmp);
    int32_t n = 0;
    for (int32_t r = 0; r < N && n < max_keep; ++r) {
        if (removed[r])
            continue;
        const int32_t i = it[r].idx;
        keep_out[n++] = i;
        for (int32_t q = r + 1; q < N; ++q) {
            const int32_t j = it[q].idx;
            if (removed[q] || (cats && cats[j] != cats[i]))
                continue;
            if (oracle_box_iou(boxes + 4 * (int64_t)i, boxes + 4 * (int64_t)j) > threshold)
                removed[q] = 1;
        }
    }
    free(it);
    free(removed);
    return n;
}

/* ------------------------------------------------------------------------- */
/* Batched proposal selection and Soft-NMS.  The paper lists Soft-NMS among     */
/* its general modules (§2) next to greedy NMS; a batch of images (or of        */
/* classes) is one call with one category per image (class).  Per category c:  */
/*   candidates: the boxes of category c whose score is >= score_threshold     */
/*   (a NaN score never is); ranked as in greedy NMS (total order of the score */
/*   bits, highest first, equal scores by index).                              */
/*   hard (method 0): greedy NMS over the candidates in rank order, a box      */
/*     removed when IoU > iou_threshold with a kept box;                       */
/*   soft (methods 1, 2), repeated while candidates remain and fewer than      */
/*     max_keep are kept: select the candidate with the largest current score  */
/*     (same total order; equal current scores by rank), output it with that   */
/*     score and remove it; every remaining candidate of the category is       */
/*     decayed, s = fl(s * w(iou)), iou = oracle_box_iou(selected, candidate): */
/*       linear (1):   w = fl(1 - iou) if iou > iou_threshold, else s is kept; */
/*       gaussian (2): w = soft_gauss_weight(iou, sigma);                      */
/*     a NaN iou leaves s unchanged; a candidate whose new score is below      */
/*     score_threshold is dropped.                                             */
/*   At most max_keep per category; the output of category c is its kept box   */
/*   indices in selection order (for hard: rank order) with their score at     */
/*   selection (hard: the input score), then -1 / 0 padding.                   */
/* ------------------------------------------------------------------------- */

/* The Gaussian decay exp(-iou^2 / sigma), rounded to binary32.  exp is evaluated */
/* in double by scaling and squaring (halve the argument until it is in [-1/2, 0], */
/* a degree-16 Taylor polynomial in Horner form, square back), one double rounding */
/* per operation in the written order, so that the CPU and the GPU library, each  */
/* implementing the same method, obtain the same binary32 weight (a score decides */
/* which box is selected next, so both must hold it in the same precision).       */
float oracle_soft_gauss_weight(float iou, float sigma)
{
    if (!(iou > 0.0f))
        return 1.0f;
    double x = -((double)iou * (double)iou) / (double)sigma;
    if (!(x >= -128.0))
        return 0.0f;   /* exp(x) < 2^-184 rounds to +0 (also an infinite IoU) */
    int k = 0;
    while (x < -0.5) {
        x = x * 0.5;
        ++k;
    }
    double e = 1.0;
    for (int n = 16; n >= 1; --n)
        e = 1.0 + (x * e) / (double)n;
    for (int i = 0; i < k; ++i)
        e = e * e;
    return (float)e;
}

/* keep_out / scores_out: [num_categories][max_keep]; num_keep_out: [num_categories]. */
void oracle_nms_batched(const float *boxes, const float *scores, const int32_t *cats,
                        int32_t N, int32_t num_categories, int32_t method,
                        float iou_threshold, float sigma, float score_threshold,
                        int32_t max_keep, int32_t *keep_out, float *scores_out,
                        int32_t *num_keep_out)
{
    nms_item *it = (nms_item *)malloc(sizeof(nms_item) * (size_t)(N > 0 ? N : 1));
    float *cur = (float *)malloc(sizeof(float) * (size_t)(N > 0 ? N : 1));
    char *alive = (char *)malloc((size_t)(N > 0 ? N : 1));
    for (int32_t c = 0; c < num_categories; ++c) {
        int32_t *ko = keep_out + (int64_t)c * max_keep;
        float *so = scores_out + (int64_t)c * max_keep;
        for (int32_t q = 0; q < max_keep; ++q) {
            ko[q] = -1;
            so[q] = 0.0f;
        }
        /* the candidates of category c, in rank order */
        int32_t n = 0;
        for (int32_t i = 0; i < N; ++i) {
            const int32_t ci = cats ? cats[i] : 0;
            if (ci != c || !(scores[i] >= score_threshold))
                continue;
            it[n].key = nms_rank_key(scores[i]);
            it[n].idx = i;
            ++n;
        }
        qsort(it, (size_t)n, sizeof(nms_item), nms_item_cmp);
        int32_t kept = 0;
        if (method == 0) {
            for (int32_t r = 0; r < n; ++r)
                alive[r] = 1;
            for (int32_t r = 0; r < n && kept < max_keep; ++r) {
                if (!alive[r])
                    continue;
                const int32_t i = it[r].idx;
                ko[kept] = i;
                so[kept] = scores[i];
                ++kept;
                for (int32_t q = r + 1; q < n; ++q) {
                    if (alive[q] && oracle_box_iou(boxes + 4 * (int64_t)i,
                                                   boxes + 4 * (int64_t)it[q].idx) > iou_threshold)
                        alive[q] = 0;
                }
            }
        } else {
            for (int32_t r = 0; r < n; ++r) {
                alive[r] = 1;
                cur[r] = scores[it[r].idx];
            }
            while (kept < max_keep) {
                /* the candidate with the largest current score; equal scores by rank */
                int32_t best = -1;
                for (int32_t r = 0; r < n; ++r) {
                    if (!alive[r])
                        continue;
                    if (best < 0 || nms_rank_key(cur[r]) < nms_rank_key(cur[best]))
                        best = r;
                }
                if (best < 0)
                    break;
                const int32_t m = it[best].idx;
                ko[kept] = m;
                so[kept] = cur[best];
                ++kept;
                alive[best] = 0;
                for (int32_t r = 0; r < n; ++r) {
                    if (!alive[r])
                        continue;
                    const float iou = oracle_box_iou(boxes + 4 * (int64_t)m,
                                                     boxes + 4 * (int64_t)it[r].idx);
                    if (iou != iou)
                        continue;                  /* NaN IoU: no decay */
                    if (method == 1) {
                        if (iou > iou_threshold) {
                            const float w = 1.0f - iou;
                            cur[r] = cur[r] * w;
                        }
                    } else {
                        cur[r] = cur[r] * oracle_soft_gauss_weight(iou, sigma);
                    }
                    if (cur[r] < score_threshold)
                        alive[r] = 0;
                }
            }
        }
        num_keep_out[c] = kept;
    }
    free(it);
    free(cur);
    free(alive);
}
