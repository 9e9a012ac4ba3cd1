/*
 * Oracle for 1xN pruning and the 1xN-pruned convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this file.  It is used by the tests, by the smoke check and by the
 * CPU-baseline leg of the benchmark, and nothing else.  It shares no code,
 * header, table or helper with the HIP library: it is written directly from
 * the paper (Lin et al., "1xN Pattern for Pruning Convolutional Neural
 * Networks", arXiv 2105.14713) in plain C with fp64 arithmetic, for a reader
 * to check against the paper by eye.  It is slow on purpose.
 *
 * Notation (Sec. 3.1): a layer's weight W has shape [n][m][h][w] (n output
 * channels, m input channels, kernel h x w).  Sec. 3.2 views W as the m x n
 * matrix Omega whose (k, j) element is the kernel W[j][k][:][:], and cuts
 * each row of Omega into n/N col-groups of N consecutive output kernels; the
 * mask T is m x (n/N).  Where n is not a multiple of N the last col-group is
 * ragged (G = ceil(n/N) groups; rows beyond n do not exist).
 *
 * Readings of points the paper leaves open (all fixed here, stated once):
 *   - l1 sums are taken in fp64, in the loop order written below.
 *   - Filter rearrangement sorts by decreasing filter l1 norm; equal norms
 *     keep ascending original index (a stable sort).
 *   - The number of pruned blocks is floor(p*K + 0.5) computed in double and
 *     clamped to [0, K]; t = K - pruned blocks are kept.
 *   - Equal block scores at the threshold: the lower row-major index
 *     k*G + g is kept first.
 *   - The BSR arrays are 0-based: P[0] = 0 and P[G] = t (the paper's
 *     1-based "fictitious" last entry t + 1).  Blocks inside a col-group are
 *     stacked in ascending input channel k.  D holds whole h x w kernels:
 *     D[t][N][h][w], rows beyond n are 0.
 *   - Eq. 8 is read with the col-group index j in the P subscripts and the
 *     block position z (not I_z) as the row of D.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Threads the parallel loops below use from now on (timing runs only). */
void oracle_set_num_threads(int k)
{
#ifdef _OPENMP
    if (k > 0) omp_set_num_threads(k);
#else
    (void)k;
#endif
}

/* ---------------------------------------------------------------------- */
/* Sec. 3.3, filter rearrangement (Fig. 2(a)).                             */
/* ---------------------------------------------------------------------- */

typedef struct {
    double key;
    int64_t idx;
} keyed;

/* Larger key first; equal keys by ascending index. */
static int by_key_desc_then_idx(const void* a, const void* b)
{
    const keyed* x = (const keyed*)a;
    const keyed* y = (const keyed*)b;
    if (x->key > y->key) return -1;
    if (x->key < y->key) return 1;
    if (x->idx < y->idx) return -1;
    if (x->idx > y->idx) return 1;
    return 0;
}

/*
 * The l1 norm of every filter W_j (one column of Omega):
 *     norm[j] = sum_k sum_q sum_r |W[j][k][q][r]|.
 */
void oracle_filter_norms(const double* w, int n, int m, int h, int wd, double* norm)
{
    for (int j = 0; j < n; j++) {
        double s = 0.0;
        for (int k = 0; k < m; k++)
            for (int q = 0; q < h; q++)
                for (int r = 0; r < wd; r++)
                    s += fabs(w[(((int64_t)j * m + k) * h + q) * wd + r]);
        norm[j] = s;
    }
}

/*
 * Rearranged filter order: perm[j'] is the original index of the filter that
 * takes position j' in Omega-tilde.  Filters are put in decreasing order of
 * their l1 norm.  Without rearrangement perm is the identity.
 */
void oracle_filter_perm(const double* w, int n, int m, int h, int wd, int rearrange, int32_t* perm)
{
    if (!rearrange) {
        for (int j = 0; j < n; j++) perm[j] = j;
        return;
    }
    double* norm = (double*)malloc(sizeof(double) * (size_t)n);
    keyed* order = (keyed*)malloc(sizeof(keyed) * (size_t)n);
    oracle_filter_norms(w, n, m, h, wd, norm);
    for (int j = 0; j < n; j++) {
        order[j].key = norm[j];
        order[j].idx = j;
    }
    qsort(order, (size_t)n, sizeof(keyed), by_key_desc_then_idx);
    for (int j = 0; j < n; j++) perm[j] = (int32_t)order[j].idx;
    free(order);
    free(norm);
}

/* W-tilde: filter j' of the rearranged layer is filter perm[j'] of W. */
void oracle_apply_perm(const double* w, int n, int m, int h, int wd, const int32_t* perm, double* wt)
{
    int64_t per_filter = (int64_t)m * h * wd;
    for (int j = 0; j < n; j++)
        memcpy(wt + (int64_t)j * per_filter, w + (int64_t)perm[j] * per_filter,
               sizeof(double) * (size_t)per_filter);
}

/* ---------------------------------------------------------------------- */
/* Sec. 3.2 / Eq. 4-5: block l1 scores of Omega-tilde.                     */
/* ---------------------------------------------------------------------- */

/*
 * Block (k, g) holds the N consecutive output kernels g*N .. g*N+N-1 of input
 * channel k.  Its score is the l1 norm of those kernels:
 *     S[k][g] = sum_{i<N, gN+i<n} sum_q sum_r |Wt[gN+i][k][q][r]|.
 * S is stored row-major by input channel k, G = ceil(n/N) columns.
 */
void oracle_block_scores(const double* wt, int n, int m, int h, int wd, int N, double* S)
{
    int G = (n + N - 1) / N;
    for (int k = 0; k < m; k++)
        for (int g = 0; g < G; g++) {
            double s = 0.0;
            for (int i = 0; i < N; i++) {
                int j = g * N + i;
                if (j >= n) break;
                for (int q = 0; q < h; q++)
                    for (int r = 0; r < wd; r++)
                        s += fabs(wt[(((int64_t)j * m + k) * h + q) * wd + r]);
            }
            S[(int64_t)k * G + g] = s;
        }
}

/* ---------------------------------------------------------------------- */
/* Eq. 1 and the solution of Eq. 5 (Sec. 3.3): per-layer top-(1-p) blocks. */
/* ---------------------------------------------------------------------- */

/* Number of blocks kept out of K at pruning rate p. */
int64_t oracle_kept_count(int64_t K, double p)
{
    double pruned = floor(p * (double)K + 0.5);
    if (pruned < 0.0) pruned = 0.0;
    if (pruned > (double)K) pruned = (double)K;
    return K - (int64_t)pruned;
}

/*
 * T[i] = 1 for the t blocks with the largest scores (ties: lower index i =
 * k*G + g first), 0 otherwise.  Returns t.  This maximises Eq. 5 under the
 * constraint ||T||_0 = t.
 */
int64_t oracle_select(const double* S, int64_t K, double p, uint8_t* T)
{
    int64_t t = oracle_kept_count(K, p);
    keyed* order = (keyed*)malloc(sizeof(keyed) * (size_t)(K > 0 ? K : 1));
    for (int64_t i = 0; i < K; i++) {
        order[i].key = S[i];
        order[i].idx = i;
    }
    qsort(order, (size_t)K, sizeof(keyed), by_key_desc_then_idx);
    memset(T, 0, (size_t)K);
    for (int64_t i = 0; i < t; i++) T[order[i].idx] = 1;
    free(order);
    return t;
}

/* ---------------------------------------------------------------------- */
/* Eq. 6: Omega-bar = Omega-tilde masked by T.                             */
/* ---------------------------------------------------------------------- */

void oracle_masked_weight(const double* wt, const uint8_t* T, int n, int m, int h, int wd, int N,
                          double* wbar)
{
    int G = (n + N - 1) / N;
    for (int j = 0; j < n; j++)
        for (int k = 0; k < m; k++) {
            int keep = T[(int64_t)k * G + j / N];
            for (int q = 0; q < h; q++)
                for (int r = 0; r < wd; r++) {
                    int64_t e = (((int64_t)j * m + k) * h + q) * wd + r;
                    wbar[e] = keep ? wt[e] : 0.0;
                }
        }
}

/* ---------------------------------------------------------------------- */
/* Sec. 3.4 (Fig. 3): BSR encoding of Omega-bar into (D, I, P).            */
/* ---------------------------------------------------------------------- */

/*
 * For every col-group g in order, the kept blocks of that col-group are
 * stacked (ascending input channel k); I records each block's row k and P
 * records where each col-group starts.  D[z] is the 1 x N block of kernels,
 * stored as [N][h][w].  Returns the number of blocks written.
 */
int64_t oracle_pack(const double* wt, const uint8_t* T, int n, int m, int h, int wd, int N,
                    int32_t* P, int32_t* I, double* D)
{
    int G = (n + N - 1) / N;
    int64_t blk = (int64_t)N * h * wd;
    int64_t z = 0;
    for (int g = 0; g < G; g++) {
        P[g] = (int32_t)z;
        for (int k = 0; k < m; k++) {
            if (!T[(int64_t)k * G + g]) continue;
            I[z] = k;
            for (int i = 0; i < N; i++) {
                int j = g * N + i;
                for (int q = 0; q < h; q++)
                    for (int r = 0; r < wd; r++) {
                        double v = 0.0;
                        if (j < n) v = wt[(((int64_t)j * m + k) * h + q) * wd + r];
                        D[z * blk + ((int64_t)i * h + q) * wd + r] = v;
                    }
            }
            z++;
        }
    }
    P[G] = (int32_t)z;
    return z;
}

/* ---------------------------------------------------------------------- */
/* Eq. 7: the convolution with the dense masked weight.                    */
/* ---------------------------------------------------------------------- */

/* One output element: Y[b][o][oh][ow] = sum_c sum_q sum_r X[..] * Wbar[o][c][q][r]. */
static double conv_one(const double* x, const double* wbar, int m, int H, int W, int h, int wd,
                       int sh, int sw, int ph, int pw, int b, int o, int oh, int ow)
{
    double acc = 0.0;
    for (int c = 0; c < m; c++)
        for (int q = 0; q < h; q++)
            for (int r = 0; r < wd; r++) {
                int ih = oh * sh - ph + q;
                int iw = ow * sw - pw + r;
                if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                acc += x[(((int64_t)b * m + c) * H + ih) * W + iw] *
                       wbar[(((int64_t)o * m + c) * h + q) * wd + r];
            }
    return acc;
}

/*
 * Direct convolution, NCHW input x[B][m][H][W], weight wbar[n][m][h][w],
 * output y[B][n][Ho][Wo] with Ho = (H + 2ph - h)/sh + 1 (likewise Wo).
 * The output channel index is the rearranged one.
 */
void oracle_conv2d(const double* x, const double* wbar, int B, int m, int H, int W, int n, int h,
                   int wd, int sh, int sw, int ph, int pw, double* y)
{
    int Ho = (H + 2 * ph - h) / sh + 1;
    int Wo = (W + 2 * pw - wd) / sw + 1;
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; b++)
        for (int o = 0; o < n; o++)
            for (int oh = 0; oh < Ho; oh++)
                for (int ow = 0; ow < Wo; ow++)
                    y[(((int64_t)b * n + o) * Ho + oh) * Wo + ow] =
                        conv_one(x, wbar, m, H, W, h, wd, sh, sw, ph, pw, b, o, oh, ow);
}

/* The same definition evaluated only at the listed flat output indices. */
void oracle_conv2d_at(const double* x, const double* wbar, int B, int m, int H, int W, int n, int h,
                      int wd, int sh, int sw, int ph, int pw, const int64_t* idx, int64_t count,
                      double* out)
{
    int Ho = (H + 2 * ph - h) / sh + 1;
    int Wo = (W + 2 * pw - wd) / sw + 1;
    (void)B;
#pragma omp parallel for schedule(dynamic, 64)
    for (int64_t s = 0; s < count; s++) {
        int64_t e = idx[s];
        int ow = (int)(e % Wo);
        int oh = (int)((e / Wo) % Ho);
        int o = (int)((e / ((int64_t)Wo * Ho)) % n);
        int b = (int)(e / ((int64_t)Wo * Ho * n));
        out[s] = conv_one(x, wbar, m, H, W, h, wd, sh, sw, ph, pw, b, o, oh, ow);
    }
}

/* ---------------------------------------------------------------------- */
/* The layer-to-layer step after the convolution (Sec. 4.1 networks).      */
/* ---------------------------------------------------------------------- */

/*
 * In place on y[B][n][hw]: y = act(scale[o] * y + bias[o]) for output channel
 * o, i.e. a batch norm folded for inference (or a bias) and then ReLU
 * (act = 1: max(y, 0)) or ReLU6 (act = 2: min(max(y, 0), 6)); act = 0 leaves
 * the affine value.  scale == NULL means 1, bias == NULL means 0.  Per Sec.
 * 3.3 a rearranged layer's channel o is original channel perm[o], so the
 * caller passes the parameters in the same order as the output channels.
 */
void oracle_epilogue(double* y, int B, int n, int64_t hw, const double* scale, const double* bias,
                     int act)
{
    for (int b = 0; b < B; b++)
        for (int o = 0; o < n; o++)
            for (int64_t i = 0; i < hw; i++) {
                double* v = &y[((int64_t)b * n + o) * hw + i];
                double u = *v;
                if (scale) u = u * scale[o];
                if (bias) u = u + bias[o];
                if (act >= 1 && u < 0.0) u = 0.0;
                if (act == 2 && u > 6.0) u = 6.0;
                *v = u;
            }
}

/* ---------------------------------------------------------------------- */
/* Backward of Eq. 7 for fine-tuning with the 1xN pattern fixed (Sec. 4.1). */
/* ---------------------------------------------------------------------- */

/*
 * Gradient with respect to the input: the adjoint of Eq. 7.  Every term
 * X[b][c][ih][iw] * Wbar[o][c][q][r] of output (b, o, oh, ow) sends
 * dY[b][o][oh][ow] * Wbar[o][c][q][r] back to X[b][c][ih][iw].
 * dy[B][n][Ho][Wo] in, dx[B][m][H][W] out.
 */
void oracle_conv2d_bwd_data(const double* dy, const double* wbar, int B, int m, int H, int W, int n,
                            int h, int wd, int sh, int sw, int ph, int pw, double* dx)
{
    int Ho = (H + 2 * ph - h) / sh + 1;
    int Wo = (W + 2 * pw - wd) / sw + 1;
    memset(dx, 0, sizeof(double) * (size_t)B * m * H * W);
#pragma omp parallel for schedule(static)
    for (int b = 0; b < B; b++)
        for (int o = 0; o < n; o++)
            for (int oh = 0; oh < Ho; oh++)
                for (int ow = 0; ow < Wo; ow++) {
                    double g = dy[(((int64_t)b * n + o) * Ho + oh) * Wo + ow];
                    for (int c = 0; c < m; c++)
                        for (int q = 0; q < h; q++)
                            for (int r = 0; r < wd; r++) {
                                int ih = oh * sh - ph + q;
                                int iw = ow * sw - pw + r;
                                if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                                dx[(((int64_t)b * m + c) * H + ih) * W + iw] +=
                                    g * wbar[(((int64_t)o * m + c) * h + q) * wd + r];
                            }
                }
}

/*
 * Gradient with respect to the weights, restricted to the kept 1xN blocks:
 * the weights of pruned blocks stay zero during fine-tuning, so their
 * gradient is not used and is returned as 0.
 *   dw[o][c][q][r] = T[c][o/N] * sum_{b,oh,ow} dY[b][o][oh][ow] * X[b][c][oh*sh-ph+q][ow*sw-pw+r]
 * x[B][m][H][W], dy[B][n][Ho][Wo], T[m][G] in; dw[n][m][h][w] out.
 */
void oracle_conv2d_bwd_weight(const double* x, const double* dy, const uint8_t* T, int B, int m, int H,
                              int W, int n, int h, int wd, int N, int sh, int sw, int ph, int pw,
                              double* dw)
{
    int Ho = (H + 2 * ph - h) / sh + 1;
    int Wo = (W + 2 * pw - wd) / sw + 1;
    int G = (n + N - 1) / N;
#pragma omp parallel for collapse(2) schedule(static)
    for (int o = 0; o < n; o++)
        for (int c = 0; c < m; c++)
            for (int q = 0; q < h; q++)
                for (int r = 0; r < wd; r++) {
                    double acc = 0.0;
                    if (T[(int64_t)c * G + o / N]) {
                        for (int b = 0; b < B; b++)
                            for (int oh = 0; oh < Ho; oh++)
                                for (int ow = 0; ow < Wo; ow++) {
                                    int ih = oh * sh - ph + q;
                                    int iw = ow * sw - pw + r;
                                    if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                                    acc += dy[(((int64_t)b * n + o) * Ho + oh) * Wo + ow] *
                                           x[(((int64_t)b * m + c) * H + ih) * W + iw];
                                }
                    }
                    dw[(((int64_t)o * m + c) * h + q) * wd + r] = acc;
                }
}

/* ---------------------------------------------------------------------- */
/* Eq. 8: block-wise decode over the BSR arrays.                           */
/* ---------------------------------------------------------------------- */

/*
 * For every output pixel and col-group g:
 *     Y[pixel][gN .. gN+N-1] = sum_{z = P[g]}^{P[g+1]-1} X[pixel, channel I[z]] . D[z]
 * where for an h x w kernel "X[pixel, channel c]" is the input patch of
 * channel c under the output pixel and "." is the patch-kernel inner
 * product.  Output rows beyond n are dropped.  Same shapes as oracle_conv2d.
 */
void oracle_decode(const double* x, const int32_t* P, const int32_t* I, const double* D, int B,
                   int m, int H, int W, int n, int h, int wd, int N, int sh, int sw, int ph, int pw,
                   double* y)
{
    int G = (n + N - 1) / N;
    int Ho = (H + 2 * ph - h) / sh + 1;
    int Wo = (W + 2 * pw - wd) / sw + 1;
    int64_t blk = (int64_t)N * h * wd;
    double* acc = (double*)malloc(sizeof(double) * (size_t)N);
    for (int b = 0; b < B; b++)
        for (int oh = 0; oh < Ho; oh++)
            for (int ow = 0; ow < Wo; ow++)
                for (int g = 0; g < G; g++) {
                    for (int i = 0; i < N; i++) acc[i] = 0.0;
                    for (int32_t z = P[g]; z < P[g + 1]; z++) {
                        int c = I[z];
                        for (int q = 0; q < h; q++)
                            for (int r = 0; r < wd; r++) {
                                int ih = oh * sh - ph + q;
                                int iw = ow * sw - pw + r;
                                if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                                double xv = x[(((int64_t)b * m + c) * H + ih) * W + iw];
                                for (int i = 0; i < N; i++)
                                    acc[i] += xv * D[z * blk + ((int64_t)i * h + q) * wd + r];
                            }
                    }
                    for (int i = 0; i < N; i++) {
                        int o = g * N + i;
                        if (o < n) y[(((int64_t)b * n + o) * Ho + oh) * Wo + ow] = acc[i];
                    }
                }
    free(acc);
}
