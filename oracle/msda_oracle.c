/*
 * Multi-scale deformable attention (MSDA): plain CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, obviously-correct definition that the
 * GPU library is checked against. Only the test-suite, the smoke check and the benchmark's
 * CPU-baseline leg load it; the product path never does. It shares no code, header, table
 * or helper with the GPU library.
 *
 * What is computed (paper, Sec. 3 "Co-design Analysis" and Sec. 4 "Implementation"):
 *   - each query q of batch n and head m samples L feature levels at P learned locations;
 *   - every sample is a bilinear interpolation over the 2x2 pixel neighbourhood around the
 *     location (Sec. 3, the paragraph on bilinear grid sampling);
 *   - the samples are weighted by the attention weights and summed over levels and points
 *     (Sec. 4, first paragraph: coordinates and weights, per-level bilinear sampling, then
 *     a weighted sum);
 *   - the backward pass produces the gradients w.r.t. the sampling locations and attention
 *     weights (element-wise work plus reductions over channels) and w.r.t. the value tensor
 *     (a scatter-add), Sec. 4.2.
 * The sampling convention is the grid-sample one the paper points to in Sec. 3 (Fig. 3,
 * the MMCV reference implementation): locations are normalized to [0,1] per level,
 * align_corners=False (pixel centre (h,w) sits at ((w+0.5)/W, (h+0.5)/H)), and reads
 * outside the map are zero.
 *
 * Readings where the paper is silent (each is listed with its reason in the design notes):
 *   - loc[...,0] is x (column, scaled by W), loc[...,1] is y (row, scaled by H);
 *   - in the default mode the image coordinates are formed in fp32 with one rounding,
 *     w_im = fmaf(x, W, -0.5f), h_im = fmaf(y, H, -0.5f), so that floor() decisions are
 *     reproducible bit for bit; everything after that is fp64. A second mode (coords_fp32 = 0)
 *     forms them in fp64 and exists for finite-difference tests;
 *   - a sample contributes only if -1 < h_im < H and -1 < w_im < W; each of its four corners
 *     contributes only if it lies on the map (zero padding);
 *   - at an integer h_im or w_im the derivative is the one of the cell [floor, floor+1].
 *
 * Layouts (row-major, all arrays float64, the caller converts exactly from fp32/fp16):
 *   value      [N, S, M, D]        S = sum_l H_l*W_l, pixel (h,w) of level l is row start_l + h*W_l + w
 *   shapes     [L, 2]  (H_l, W_l)   starts [L]
 *   loc        [N, Lq, M, L, P, 2]  normalized (x, y)
 *   attn       [N, Lq, M, L, P]
 *   out        [N, Lq, M, D]        (the same memory as [N, Lq, M*D])
 *   grad_out   [N, Lq, M, D]
 *   grad_value [N, S, M, D]         grad_loc [N, Lq, M, L, P, 2]   grad_attn [N, Lq, M, L, P]
 *
 * Threads: OpenMP over (n,q) for out / grad_loc / grad_attn and over (n,m) for grad_value.
 * Every output element is written by exactly one thread in a fixed order, so results do
 * not depend on the thread count.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <omp.h>

/* The four corners of one bilinear sample, in the order (h0,w0), (h0,w1), (h1,w0), (h1,w1). */
typedef struct {
    int in_range;     /* -1 < h_im < H and -1 < w_im < W                               */
    int64_t pix[4];   /* pixel index h*W + w within the level, or -1 if off the map     */
    double wt[4];     /* bilinear weights hh*hw, hh*lw, lh*hw, lh*lw                    */
    double lh, lw, hh, hw;
} corners_t;

/* Image coordinates, validity and the 2x2 neighbourhood of one normalized location. */
static void locate(double x, double y, int64_t H, int64_t W, int coords_fp32, corners_t* c)
{
    double w_im, h_im;
    if (coords_fp32) {
        w_im = (double)fmaf((float)x, (float)W, -0.5f);
        h_im = (double)fmaf((float)y, (float)H, -0.5f);
    } else {
        w_im = x * (double)W - 0.5;
        h_im = y * (double)H - 0.5;
    }
    memset(c, 0, sizeof(*c));
    for (int k = 0; k < 4; ++k) c->pix[k] = -1;
    c->in_range = (h_im > -1.0) && (w_im > -1.0) && (h_im < (double)H) && (w_im < (double)W);
    if (!c->in_range) return;

    double h0 = floor(h_im), w0 = floor(w_im);
    c->lh = h_im - h0;
    c->lw = w_im - w0;
    c->hh = 1.0 - c->lh;
    c->hw = 1.0 - c->lw;

    int64_t hs[4] = {(int64_t)h0, (int64_t)h0, (int64_t)h0 + 1, (int64_t)h0 + 1};
    int64_t ws[4] = {(int64_t)w0, (int64_t)w0 + 1, (int64_t)w0, (int64_t)w0 + 1};
    c->wt[0] = c->hh * c->hw;
    c->wt[1] = c->hh * c->lw;
    c->wt[2] = c->lh * c->hw;
    c->wt[3] = c->lh * c->lw;
    for (int k = 0; k < 4; ++k)
        if (hs[k] >= 0 && hs[k] < H && ws[k] >= 0 && ws[k] < W) c->pix[k] = hs[k] * W + ws[k];
}

static int set_threads(int threads)
{
    if (threads > 0) omp_set_num_threads(threads);
    int used = 1;
#pragma omp parallel
    {
#pragma omp single
        used = omp_get_num_threads();
    }
    return used;
}

/* Forward pass. Returns the number of threads used. */
int msda_oracle_forward(const double* value, const int64_t* shapes, const int64_t* starts,
                        const double* loc, const double* attn, double* out,
                        int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                        int64_t P, int coords_fp32, int threads)
{
    int used = set_threads(threads);
    (void)S;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t nq = 0; nq < N * Lq; ++nq) {
        int64_t n = nq / Lq;
        for (int64_t m = 0; m < M; ++m) {
            double* o = out + (nq * M + m) * D;
            for (int64_t d = 0; d < D; ++d) o[d] = 0.0;
            for (int64_t l = 0; l < L; ++l) {
                int64_t H = shapes[2 * l], W = shapes[2 * l + 1];
                for (int64_t p = 0; p < P; ++p) {
                    int64_t smp = ((nq * M + m) * L + l) * P + p;
                    double a = attn[smp];
                    corners_t c;
                    locate(loc[2 * smp], loc[2 * smp + 1], H, W, coords_fp32, &c);
                    if (!c.in_range) continue;
                    for (int k = 0; k < 4; ++k) {
                        if (c.pix[k] < 0) continue;
                        const double* v = value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;
                        for (int64_t d = 0; d < D; ++d) o[d] += a * c.wt[k] * v[d];
                    }
                }
            }
        }
    }
    return used;
}

/* Backward pass: grad_value (overwritten), grad_loc and grad_attn (overwritten).
 * Returns the number of threads used. */
int msda_oracle_backward(const double* value, const int64_t* shapes, const int64_t* starts,
                         const double* loc, const double* attn, const double* grad_out,
                         double* grad_value, double* grad_loc, double* grad_attn,
                         int64_t N, int64_t S, int64_t M, int64_t D, int64_t Lq, int64_t L,
                         int64_t P, int coords_fp32, int threads)
{
    int used = set_threads(threads);

    /* Part 1 (Sec. 4.2): gradients w.r.t. attention weights and sampling locations. */
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t nq = 0; nq < N * Lq; ++nq) {
        int64_t n = nq / Lq;
        for (int64_t m = 0; m < M; ++m) {
            const double* g = grad_out + (nq * M + m) * D;
            for (int64_t l = 0; l < L; ++l) {
                int64_t H = shapes[2 * l], W = shapes[2 * l + 1];
                for (int64_t p = 0; p < P; ++p) {
                    int64_t smp = ((nq * M + m) * L + l) * P + p;
                    double a = attn[smp];
                    corners_t c;
                    locate(loc[2 * smp], loc[2 * smp + 1], H, W, coords_fp32, &c);
                    grad_attn[smp] = 0.0;
                    grad_loc[2 * smp] = 0.0;
                    grad_loc[2 * smp + 1] = 0.0;
                    if (!c.in_range) continue;
                    const double* v[4];
                    for (int k = 0; k < 4; ++k)
                        v[k] = c.pix[k] < 0 ? 0
                                            : value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;
                    double ga = 0.0, gw = 0.0, gh = 0.0;
                    for (int64_t d = 0; d < D; ++d) {
                        double v00 = v[0] ? v[0][d] : 0.0, v01 = v[1] ? v[1][d] : 0.0;
                        double v10 = v[2] ? v[2][d] : 0.0, v11 = v[3] ? v[3][d] : 0.0;
                        double s = c.wt[0] * v00 + c.wt[1] * v01 + c.wt[2] * v10 + c.wt[3] * v11;
                        ga += g[d] * s;
                        /* d s / d w_im and d s / d h_im of the bilinear form */
                        gw += g[d] * (c.hh * (v01 - v00) + c.lh * (v11 - v10));
                        gh += g[d] * (c.hw * (v10 - v00) + c.lw * (v11 - v01));
                    }
                    grad_attn[smp] = ga;
                    /* chain rule through w_im = x*W - 1/2 and h_im = y*H - 1/2 */
                    grad_loc[2 * smp] = (double)W * a * gw;
                    grad_loc[2 * smp + 1] = (double)H * a * gh;
                }
            }
        }
    }

    /* Part 2 (Sec. 4.2): grad_value as a scatter-add. Each (n,m) slab is owned by one thread. */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t nm = 0; nm < N * M; ++nm) {
        int64_t n = nm / M, m = nm % M;
        for (int64_t s = 0; s < S; ++s)
            for (int64_t d = 0; d < D; ++d) grad_value[((n * S + s) * M + m) * D + d] = 0.0;
        for (int64_t q = 0; q < Lq; ++q) {
            const double* g = grad_out + ((n * Lq + q) * M + m) * D;
            for (int64_t l = 0; l < L; ++l) {
                int64_t H = shapes[2 * l], W = shapes[2 * l + 1];
                for (int64_t p = 0; p < P; ++p) {
                    int64_t smp = (((n * Lq + q) * M + m) * L + l) * P + p;
                    double a = attn[smp];
                    corners_t c;
                    locate(loc[2 * smp], loc[2 * smp + 1], H, W, coords_fp32, &c);
                    if (!c.in_range) continue;
                    for (int k = 0; k < 4; ++k) {
                        if (c.pix[k] < 0) continue;
                        double* gv = grad_value + ((n * S + starts[l] + c.pix[k]) * M + m) * D;
                        for (int64_t d = 0; d < D; ++d) gv[d] += a * c.wt[k] * g[d];
                    }
                }
            }
        }
    }
    return used;
}

/*
 * The step before the sampling (Sec. 4, first paragraph: the sampling coordinates and the
 * attention weights are computed first, then the per-level bilinear sampling runs). A deformable
 * attention layer predicts, for every sample, an offset in pixels of the sampled level and one
 * attention logit. The location is the query's reference point on that level plus the offset
 * divided by the level's size, and the weights of one (query, head) are a softmax over its L*P
 * logits:
 *   ref     [N, Lq, L, 2]       normalized (x, y) reference point per level
 *   offsets [N, Lq, M, L, P, 2] pixels: x along W_l, y along H_l
 *   logits  [N, Lq, M, L*P]
 *   loc     [N, Lq, M, L, P, 2] = ref + offsets / (W_l, H_l)
 *   attn    [N, Lq, M, L, P]    = softmax over the L*P logits of (n, q, m)
 * With coords_fp32 the location is evaluated in fp32, the division and then the addition each
 * rounded once, which is the arithmetic the GPU library uses, so both sample identical locations;
 * otherwise in fp64 (finite-difference tests). The softmax is fp64, shifted by the maximum logit.
 */
void msda_oracle_prologue(const double* ref, const double* offsets, const double* logits,
                          const int64_t* shapes, int64_t N, int64_t Lq, int64_t M, int64_t L, int64_t P,
                          int coords_fp32, double* loc, double* attn)
{
    const int64_t K = L * P;
#pragma omp parallel for schedule(static)
    for (int64_t nq = 0; nq < N * Lq; ++nq) {
        for (int64_t m = 0; m < M; ++m) {
            const double* z = logits + (nq * M + m) * K;
            double mx = z[0];
            for (int64_t k = 1; k < K; ++k) mx = z[k] > mx ? z[k] : mx;
            double sum = 0.0;
            for (int64_t k = 0; k < K; ++k) sum += exp(z[k] - mx);
            for (int64_t l = 0; l < L; ++l) {
                const double W = (double)shapes[2 * l + 1], H = (double)shapes[2 * l];
                const double rx = ref[(nq * L + l) * 2], ry = ref[(nq * L + l) * 2 + 1];
                for (int64_t p = 0; p < P; ++p) {
                    const int64_t k = l * P + p;
                    const int64_t smp = (nq * M + m) * K + k;
                    const double ox = offsets[2 * smp], oy = offsets[2 * smp + 1];
                    if (coords_fp32) {
                        const float fx = (float)ox / (float)W, fy = (float)oy / (float)H;
                        loc[2 * smp] = (double)((float)rx + fx);
                        loc[2 * smp + 1] = (double)((float)ry + fy);
                    } else {
                        loc[2 * smp] = rx + ox / W;
                        loc[2 * smp + 1] = ry + oy / H;
                    }
                    attn[smp] = exp(z[k] - mx) / sum;
                }
            }
        }
    }
}

/*
 * Gradients of the step above, from the sampling's grad_loc and grad_attn (chain rule):
 *   grad_offsets = grad_loc / (W_l, H_l)
 *   grad_logits  = attn * (grad_attn - sum_k attn_k grad_attn_k)   over the L*P samples of (n,q,m)
 *   grad_ref     = sum over heads and points of grad_loc           [N, Lq, L, 2]
 */
void msda_oracle_prologue_backward(const double* attn, const double* grad_loc, const double* grad_attn,
                                   const int64_t* shapes, int64_t N, int64_t Lq, int64_t M, int64_t L,
                                   int64_t P, double* grad_offsets, double* grad_logits, double* grad_ref)
{
    const int64_t K = L * P;
#pragma omp parallel for schedule(static)
    for (int64_t nq = 0; nq < N * Lq; ++nq) {
        for (int64_t l = 0; l < L; ++l) {
            grad_ref[(nq * L + l) * 2] = 0.0;
            grad_ref[(nq * L + l) * 2 + 1] = 0.0;
        }
        for (int64_t m = 0; m < M; ++m) {
            const int64_t s0 = (nq * M + m) * K;
            double dot = 0.0;
            for (int64_t k = 0; k < K; ++k) dot += attn[s0 + k] * grad_attn[s0 + k];
            for (int64_t l = 0; l < L; ++l) {
                const double W = (double)shapes[2 * l + 1], H = (double)shapes[2 * l];
                for (int64_t p = 0; p < P; ++p) {
                    const int64_t smp = s0 + l * P + p;
                    grad_offsets[2 * smp] = grad_loc[2 * smp] / W;
                    grad_offsets[2 * smp + 1] = grad_loc[2 * smp + 1] / H;
                    grad_logits[smp] = attn[smp] * (grad_attn[smp] - dot);
                    grad_ref[(nq * L + l) * 2] += grad_loc[2 * smp];
                    grad_ref[(nq * L + l) * 2 + 1] += grad_loc[2 * smp + 1];
                }
            }
        }
    }
}
