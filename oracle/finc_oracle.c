/*
 * finc_oracle.c -- plain, slow CPU reference of the FInC masked k x k
 * convolution layer, its FInC unit and the multi-scale sampling stack.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no source,
 * header, table or helper with the HIP library; the two meet only on the
 * seeded inputs drawn in Python.
 *
 * Everything is float64, nested loops, no blocking, no reordering.
 *
 * Layout: activations (B, C, H, W) row-major; weights (C_out, C_in, k, k)
 * row-major (OIHW).  Corners: 0 = TL, 1 = TR, 2 = BL, 3 = BR.
 *
 * Readings of the paper taken here (its text is garbled in places):
 *  - Convolution (Sec. 3, "Invertible Convolutions", conv equation) is a
 *    cross-correlation of the padded input with K; with the corner paddings of
 *    Sec. 4.1 (k-1 zero rows/cols on the two named sides) output pixel (i, j)
 *    reads input (i + a - oh, j + b - ow) for kernel position (a, b), where
 *    (oh, ow) = (k-1, k-1) TL, (k-1, 0) TR, (0, k-1) BL, (0, 0) BR.  Reads
 *    outside the image are zero.
 *  - The kernel position (oh, ow) multiplies the output pixel itself ("self
 *    tap").  At that position only c_in <= c_out is used (lower-triangular
 *    channel block); entries with c_in > c_out are ignored whatever they hold.
 *    All other positions are used in full.  The paper's own CInC masking fixes
 *    the self block to the identity (Sec. 1, proof of Theorem 1); that is the
 *    special case of unit diagonal and zero strictly-lower entries.
 *  - log|det| of one layer is H*W*sum_c log|K[c,c,oh,ow]|: the convolution
 *    matrix is triangular in the corner's pixel raster order with those
 *    diagonal entries (Sec. 3 "Algorithms for Computing Inverse ...", Fig. 1
 *    caption, Table 1 "Jacobian is 1" for unit diagonal).
 *  - The inverse here is the naive sequential substitution of Sec. 3
 *    ("Algorithms for Computing Inverse of Convolutions", the O(n^2 k^2) method
 *    of CInC / Emerging): pixels in the corner's raster order, channels in
 *    ascending order inside each pixel.  It deliberately does NOT follow the
 *    diagonal schedule of Algorithm 1.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ESINGULAR (-2)
#define ORC_ENOMEM (-5)

/* Padding offsets of the four corner variants (Sec. 4.1, corner padding
 * equations, read as k-1 zero rows/cols on the two named sides). */
static void corner_offsets(int corner, int k, int *oh, int *ow)
{
    *oh = (corner == 0 || corner == 1) ? k - 1 : 0; /* top padded    */
    *ow = (corner == 0 || corner == 2) ? k - 1 : 0; /* left padded   */
}

static int bad_shape(long B, int C, int H, int W, int k, int corner)
{
    return B < 0 || C < 1 || H < 1 || W < 1 || k < 1 || corner < 0 || corner > 3;
}

static double kw(const double *K, int C, int k, int co, int ci, int a, int b)
{
    return K[(((long)co * C + ci) * k + a) * k + b];
}

/* Weight as the layer uses it: the channel mask at the self tap. */
static double kmasked(const double *K, int C, int k, int oh, int ow,
                      int co, int ci, int a, int b)
{
    if (a == oh && b == ow && ci > co)
        return 0.0;
    return kw(K, C, k, co, ci, a, b);
}

/* Forward padded masked convolution, direct loop (Sec. 3 conv equation with
 * the Sec. 4.1 corner padding). */
int orc_forward(const double *x, double *y, const double *K, long B, int C,
                int H, int W, int k, int corner)
{
    if (bad_shape(B, C, H, W, k, corner) || !x || !y || !K)
        return ORC_EINVAL;
    int oh, ow;
    corner_offsets(corner, k, &oh, &ow);
    for (long n = 0; n < B; ++n) {
        const double *xn = x + n * (long)C * H * W;
        double *yn = y + n * (long)C * H * W;
        for (int co = 0; co < C; ++co)
            for (int i = 0; i < H; ++i)
                for (int j = 0; j < W; ++j) {
                    double s = 0.0;
                    for (int ci = 0; ci < C; ++ci)
                        for (int a = 0; a < k; ++a)
                            for (int b = 0; b < k; ++b) {
                                int ii = i + a - oh, jj = j + b - ow;
                                if (ii < 0 || ii >= H || jj < 0 || jj >= W)
                                    continue;
                                s += kmasked(K, C, k, oh, ow, co, ci, a, b) *
                                     xn[((long)ci * H + ii) * W + jj];
                            }
                    yn[((long)co * H + i) * W + j] = s;
                }
    }
    return ORC_OK;
}

/* log|det| of one layer's convolution matrix: triangular in the corner's
 * raster order, diagonal entry K[c,c,self] repeated at every pixel. */
int orc_logdet(const double *K, int C, int k, int corner, int H, int W,
               double *out)
{
    if (bad_shape(1, C, H, W, k, corner) || !K || !out)
        return ORC_EINVAL;
    int oh, ow;
    corner_offsets(corner, k, &oh, &ow);
    double s = 0.0;
    int singular = 0;
    for (int c = 0; c < C; ++c) {
        double d = kw(K, C, k, c, c, oh, ow);
        if (d == 0.0)
            singular = 1;
        s += log(fabs(d));
    }
    *out = (double)H * (double)W * s;
    return singular ? ORC_ESINGULAR : ORC_OK;
}

/* Inverse by sequential substitution in raster order (Sec. 3, "Algorithms
 * for Computing Inverse of Convolutions"): every pixel is solved after all
 * pixels it reads, then the channels of the pixel are solved against the
 * lower-triangular self block, c ascending. */
int orc_inverse(const double *y, double *x, const double *K, long B, int C,
                int H, int W, int k, int corner)
{
    if (bad_shape(B, C, H, W, k, corner) || !x || !y || !K)
        return ORC_EINVAL;
    int oh, ow;
    corner_offsets(corner, k, &oh, &ow);
    for (int c = 0; c < C; ++c)
        if (kw(K, C, k, c, c, oh, ow) == 0.0)
            return ORC_ESINGULAR;
    /* Raster order of the corner: rows top-down when the top is padded,
     * columns left-to-right when the left is padded. */
    int rows_down = (corner == 0 || corner == 1);
    int cols_right = (corner == 0 || corner == 2);
    for (long n = 0; n < B; ++n) {
        const double *yn = y + n * (long)C * H * W;
        double *xn = x + n * (long)C * H * W;
        for (int ri = 0; ri < H; ++ri) {
            int i = rows_down ? ri : H - 1 - ri;
            for (int rj = 0; rj < W; ++rj) {
                int j = cols_right ? rj : W - 1 - rj;
                for (int c = 0; c < C; ++c) {
                    double r = yn[((long)c * H + i) * W + j];
                    for (int a = 0; a < k; ++a)
                        for (int b = 0; b < k; ++b) {
                            int ii = i + a - oh, jj = j + b - ow;
                            if (ii < 0 || ii >= H || jj < 0 || jj >= W)
                                continue;
                            int self = (a == oh && b == ow);
                            int cmax = self ? c : C; /* self tap: ci < c only */
                            for (int ci = 0; ci < cmax; ++ci)
                                r -= kw(K, C, k, c, ci, a, b) *
                                     xn[((long)ci * H + ii) * W + jj];
                        }
                    xn[((long)c * H + i) * W + j] = r / kw(K, C, k, c, c, oh, ow);
                }
            }
        }
    }
    return ORC_OK;
}

/* ---- FInC unit: the four padded blocks TL, TR, BL, BR applied one after
 * the other, each with its own weights (K4 = 4 consecutive OIHW tensors). --- */

static const int UNIT_ORDER[4] = {0, 1, 2, 3};

int orc_unit_forward(const double *x, double *y, const double *K4, long B,
                     int C, int H, int W, int k)
{
    if (bad_shape(B, C, H, W, k, 0) || !x || !y || !K4)
        return ORC_EINVAL;
    long n = B * (long)C * H * W;
    long ksz = (long)C * C * k * k;
    double *t = (double *)malloc(sizeof(double) * (n > 0 ? n : 1));
    if (!t)
        return ORC_ENOMEM;
    memcpy(t, x, sizeof(double) * n);
    int rc = ORC_OK;
    for (int q = 0; q < 4 && rc == ORC_OK; ++q) {
        rc = orc_forward(t, y, K4 + q * ksz, B, C, H, W, k, UNIT_ORDER[q]);
        memcpy(t, y, sizeof(double) * n);
    }
    free(t);
    return rc;
}

int orc_unit_inverse(const double *y, double *x, const double *K4, long B,
                     int C, int H, int W, int k)
{
    if (bad_shape(B, C, H, W, k, 0) || !x || !y || !K4)
        return ORC_EINVAL;
    long n = B * (long)C * H * W;
    long ksz = (long)C * C * k * k;
    double *t = (double *)malloc(sizeof(double) * (n > 0 ? n : 1));
    if (!t)
        return ORC_ENOMEM;
    memcpy(t, y, sizeof(double) * n);
    int rc = ORC_OK;
    for (int q = 3; q >= 0 && rc == ORC_OK; --q) {
        rc = orc_inverse(t, x, K4 + q * ksz, B, C, H, W, k, UNIT_ORDER[q]);
        memcpy(t, x, sizeof(double) * n);
    }
    free(t);
    return rc;
}

int orc_unit_logdet(const double *K4, int C, int k, int H, int W, double *out)
{
    if (!out || !K4)
        return ORC_EINVAL;
    long ksz = (long)C * C * k * k;
    double s = 0.0;
    int rc = ORC_OK;
    for (int q = 0; q < 4; ++q) {
        double v;
        int r = orc_logdet(K4 + q * ksz, C, k, UNIT_ORDER[q], H, W, &v);
        if (r == ORC_EINVAL)
            return r;
        if (r != ORC_OK)
            rc = r;
        s += v;
    }
    *out = s;
    return rc;
}

/* ---- Channel-split FInC unit (Sec. 4.3, Fig. 2a, Alg. 2): the channels are
 * cut into four equal quarters; quarter g is one padded convolution block of
 * its own (C/4 channels, its own weights K_g, corner g: TL, TR, BL, BR), the
 * four side by side on the same pixels; the outputs are concatenated.  Each
 * quarter is inverted independently.  (Reading: the text names the fourth
 * quarter's padding TR again; the fourth corner, BR, is taken.)
 * Kq4 = 4 consecutive OIHW tensors of shape (C/4, C/4, k, k). ------------- */

typedef int (*orc_layer_fn)(const double *, double *, const double *, long, int, int,
                            int, int, int);

static int split_apply(const double *in, double *out, const double *Kq4, long B, int C,
                       int H, int W, int k, orc_layer_fn fn)
{
    if (bad_shape(B, C, H, W, k, 0) || C % 4 != 0 || !in || !out || !Kq4)
        return ORC_EINVAL;
    const int Cq = C / 4;
    const long part = (long)Cq * H * W;
    const long ksz = (long)Cq * Cq * k * k;
    double *a = (double *)malloc(sizeof(double) * (part > 0 ? part : 1));
    double *r = (double *)malloc(sizeof(double) * (part > 0 ? part : 1));
    if (!a || !r) {
        free(a);
        free(r);
        return ORC_ENOMEM;
    }
    int rc = ORC_OK;
    for (long b = 0; b < B && rc == ORC_OK; ++b) {
        for (int g = 0; g < 4 && rc == ORC_OK; ++g) {
            const long off = (b * C + (long)g * Cq) * H * W;
            memcpy(a, in + off, sizeof(double) * part);
            rc = fn(a, r, Kq4 + g * ksz, 1, Cq, H, W, k, g);
            memcpy(out + off, r, sizeof(double) * part);
        }
    }
    free(a);
    free(r);
    return rc;
}

int orc_split_forward(const double *x, double *y, const double *Kq4, long B, int C,
                      int H, int W, int k)
{
    return split_apply(x, y, Kq4, B, C, H, W, k, orc_forward);
}

int orc_split_inverse(const double *y, double *x, const double *Kq4, long B, int C,
                      int H, int W, int k)
{
    return split_apply(y, x, Kq4, B, C, H, W, k, orc_inverse);
}

int orc_split_logdet(const double *Kq4, int C, int k, int H, int W, double *out)
{
    if (!out || !Kq4 || C < 4 || C % 4 != 0)
        return ORC_EINVAL;
    const int Cq = C / 4;
    const long ksz = (long)Cq * Cq * k * k;
    double s = 0.0;
    int rc = ORC_OK;
    for (int g = 0; g < 4; ++g) {
        double v;
        int r = orc_logdet(Kq4 + g * ksz, Cq, k, g, H, W, &v);
        if (r == ORC_EINVAL)
            return r;
        if (r != ORC_OK)
            rc = r;
        s += v;
    }
    *out = s;
    return rc;
}

/* ---- Multi-scale glue (Sec. 4.4). ----------------------------------------
 * Actnorm: per-channel affine y = s * x + b (Glow's convention).
 * Squeeze: (C, H, W) -> (4C, H/2, W/2), out[4c + 2dy + dx][i][j] =
 *          in[c][2i + dy][2j + dx]; unsqueeze is its inverse.
 * Split:   the first half of the channels goes on, the second half is the
 *          latent; the inverse concatenates [h, z] on channels. */

void orc_actnorm_forward(const double *x, double *y, const double *s,
                         const double *b, long B, int C, int H, int W)
{
    for (long n = 0; n < B; ++n)
        for (int c = 0; c < C; ++c)
            for (long p = 0; p < (long)H * W; ++p) {
                long o = (n * C + c) * (long)H * W + p;
                y[o] = s[c] * x[o] + b[c];
            }
}

void orc_actnorm_inverse(const double *y, double *x, const double *s,
                         const double *b, long B, int C, int H, int W)
{
    for (long n = 0; n < B; ++n)
        for (int c = 0; c < C; ++c)
            for (long p = 0; p < (long)H * W; ++p) {
                long o = (n * C + c) * (long)H * W + p;
                x[o] = (y[o] - b[c]) / s[c];
            }
}

void orc_squeeze(const double *in, double *out, long B, int C, int H, int W)
{
    int H2 = H / 2, W2 = W / 2;
    for (long n = 0; n < B; ++n)
        for (int c = 0; c < C; ++c)
            for (int i = 0; i < H2; ++i)
                for (int j = 0; j < W2; ++j)
                    for (int dy = 0; dy < 2; ++dy)
                        for (int dx = 0; dx < 2; ++dx) {
                            int co = 4 * c + 2 * dy + dx;
                            out[((n * 4 * C + co) * H2 + i) * W2 + j] =
                                in[((n * C + c) * H + 2 * i + dy) * W + 2 * j + dx];
                        }
}

void orc_unsqueeze(const double *in, double *out, long B, int C4, int H2, int W2)
{
    int C = C4 / 4, H = 2 * H2, W = 2 * W2;
    for (long n = 0; n < B; ++n)
        for (int c = 0; c < C; ++c)
            for (int i = 0; i < H2; ++i)
                for (int j = 0; j < W2; ++j)
                    for (int dy = 0; dy < 2; ++dy)
                        for (int dx = 0; dx < 2; ++dx) {
                            int ci = 4 * c + 2 * dy + dx;
                            out[((n * C + c) * H + 2 * i + dy) * W + 2 * j + dx] =
                                in[((n * C4 + ci) * H2 + i) * W2 + j];
                        }
}

/* Stack parameter layout shared with the Python wrapper:
 *   K:     for level l = 0..L-1, unit u = 0..U-1, block q = 0..3:
 *          C_l*C_l*k*k doubles, C_l = C1 << l.
 *   scale, bias: for level l, unit u: C_l doubles.
 *   z[l]:  l < L-1: (B, C_l/2, H_l, W_l); z[L-1]: (B, C_{L-1}, H, W) top.
 *   x:     (B, C1, H1, W1). */
static long stack_koff(int l, int U, int C1, int k)
{
    long off = 0;
    for (int m = 0; m < l; ++m) {
        long C = (long)C1 << m;
        off += (long)U * 4 * C * C * k * k;
    }
    return off;
}

static long stack_soff(int l, int U, int C1)
{
    long off = 0;
    for (int m = 0; m < l; ++m)
        off += (long)U * ((long)C1 << m);
    return off;
}

/* Forward direction of the stack: per level U x [unit, actnorm], then (not at
 * the top) split and squeeze. */
int orc_stack_forward(const double *x, double *const *z, const double *K,
                      const double *scale, const double *bias, long B, int L,
                      int U, int C1, int H1, int W1, int k)
{
    if (L < 1 || U < 0 || B < 0 || C1 < 1 || H1 < 1 || W1 < 1 || k < 1 || !x || !z)
        return ORC_EINVAL;
    if (((H1 | W1) & ((1 << (L - 1)) - 1)) || (L > 1 && (C1 & 1)))
        return ORC_EINVAL;
    long maxn = B * (long)C1 * H1 * W1;
    double *h = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    double *t = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    if (!h || !t) {
        free(h);
        free(t);
        return ORC_ENOMEM;
    }
    memcpy(h, x, sizeof(double) * maxn);
    int rc = ORC_OK;
    for (int l = 0; l < L && rc == ORC_OK; ++l) {
        int C = C1 << l, H = H1 >> l, W = W1 >> l;
        long n = B * (long)C * H * W;
        long ksz = (long)C * C * k * k;
        const double *Kl = K + stack_koff(l, U, C1, k);
        const double *sl = scale + stack_soff(l, U, C1);
        const double *bl = bias + stack_soff(l, U, C1);
        for (int u = 0; u < U && rc == ORC_OK; ++u) {
            rc = orc_unit_forward(h, t, Kl + (long)u * 4 * ksz, B, C, H, W, k);
            orc_actnorm_forward(t, h, sl + (long)u * C, bl + (long)u * C, B, C, H, W);
        }
        if (rc != ORC_OK)
            break;
        if (l == L - 1) {
            memcpy(z[l], h, sizeof(double) * n);
            break;
        }
        int Ch = C / 2;
        long hw = (long)H * W;
        for (long b = 0; b < B; ++b) {
            memcpy(t + b * Ch * hw, h + b * C * hw, sizeof(double) * Ch * hw);
            memcpy(z[l] + b * Ch * hw, h + (b * C + Ch) * hw, sizeof(double) * Ch * hw);
        }
        orc_squeeze(t, h, B, Ch, H, W);
    }
    free(h);
    free(t);
    return rc;
}

/* Sampling direction: start from the top latent, per level U x [actnorm^-1,
 * unit^-1] with the units in reverse, then unsqueeze and concatenate the
 * level's latent behind it, down to (B, C1, H1, W1). */
int orc_stack_inverse(const double *const *z, double *x, const double *K,
                      const double *scale, const double *bias, long B, int L,
                      int U, int C1, int H1, int W1, int k)
{
    if (L < 1 || U < 0 || B < 0 || C1 < 1 || H1 < 1 || W1 < 1 || k < 1 || !x || !z)
        return ORC_EINVAL;
    if (((H1 | W1) & ((1 << (L - 1)) - 1)) || (L > 1 && (C1 & 1)))
        return ORC_EINVAL;
    long maxn = B * (long)C1 * H1 * W1;
    double *h = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    double *t = (double *)malloc(sizeof(double) * (maxn > 0 ? maxn : 1));
    if (!h || !t) {
        free(h);
        free(t);
        return ORC_ENOMEM;
    }
    int rc = ORC_OK;
    {
        int C = C1 << (L - 1), H = H1 >> (L - 1), W = W1 >> (L - 1);
        memcpy(h, z[L - 1], sizeof(double) * B * (long)C * H * W);
    }
    for (int l = L - 1; l >= 0 && rc == ORC_OK; --l) {
        int C = C1 << l, H = H1 >> l, W = W1 >> l;
        long ksz = (long)C * C * k * k;
        const double *Kl = K + stack_koff(l, U, C1, k);
        const double *sl = scale + stack_soff(l, U, C1);
        const double *bl = bias + stack_soff(l, U, C1);
        for (int u = U - 1; u >= 0 && rc == ORC_OK; --u) {
            orc_actnorm_inverse(h, t, sl + (long)u * C, bl + (long)u * C, B, C, H, W);
            rc = orc_unit_inverse(t, h, Kl + (long)u * 4 * ksz, B, C, H, W, k);
        }
        if (rc != ORC_OK || l == 0)
            break;
        /* h: (B, C, H, W) at level l -> unsqueeze to (B, C/4, 2H, 2W), then
         * concatenate the latent of level l-1 (B, C/4, 2H, 2W) behind it. */
        int Cq = C / 4, H2 = 2 * H, W2 = 2 * W;
        long hw = (long)H2 * W2;
        orc_unsqueeze(h, t, B, C, H, W);
        for (long b = 0; b < B; ++b) {
            memcpy(h + b * 2 * Cq * hw, t + b * Cq * hw, sizeof(double) * Cq * hw);
            memcpy(h + (b * 2 * Cq + Cq) * hw, z[l - 1] + b * Cq * hw,
                   sizeof(double) * Cq * hw);
        }
    }
    if (rc == ORC_OK)
        memcpy(x, h, sizeof(double) * maxn);
    free(h);
    free(t);
    return rc;
}

/* Backward of one layer, for training on the negative log-likelihood (Sec. 3
 * NLL equation; the appendix's training details).  Given x and dy = dL/dy for
 * y = layer(x):
 *   dx = J^T dy: every output gradient dy[co,i,j] is sent back along each tap
 *        to the input pixel that tap read, with the weight the layer used;
 *   dK[co,ci,a,b] = sum over images and output pixels of dy[co,i,j] times the
 *        input the tap read (zero outside the image); the masked entries (self
 *        tap, ci > co) get 0 -- the paper resets their gradients to zero after
 *        every training step -- and the self diagonal also gets
 *        gld * H * W / K[c,c,self], the gradient of gld * log|det|.
 * dx or dK may be NULL (not computed). */
int orc_backward(const double *x, const double *dy, const double *K, double *dx,
                 double *dK, double gld, long B, int C, int H, int W, int k,
                 int corner)
{
    if (bad_shape(B, C, H, W, k, corner) || !x || !dy || !K)
        return ORC_EINVAL;
    int oh, ow;
    corner_offsets(corner, k, &oh, &ow);
    const long plane = (long)H * W, img = (long)C * plane;
    if (dx) {
        for (long e = 0; e < B * img; ++e)
            dx[e] = 0.0;
        for (long n = 0; n < B; ++n)
            for (int co = 0; co < C; ++co)
                for (int i = 0; i < H; ++i)
                    for (int j = 0; j < W; ++j) {
                        const double g = dy[n * img + co * plane + (long)i * W + j];
                        for (int ci = 0; ci < C; ++ci)
                            for (int a = 0; a < k; ++a)
                                for (int b = 0; b < k; ++b) {
                                    int ii = i + a - oh, jj = j + b - ow;
                                    if (ii < 0 || ii >= H || jj < 0 || jj >= W)
                                        continue;
                                    dx[n * img + ci * plane + (long)ii * W + jj] +=
                                        kmasked(K, C, k, oh, ow, co, ci, a, b) * g;
                                }
                    }
    }
    if (dK) {
        for (int co = 0; co < C; ++co)
            for (int ci = 0; ci < C; ++ci)
                for (int a = 0; a < k; ++a)
                    for (int b = 0; b < k; ++b) {
                        double s = 0.0;
                        if (!(a == oh && b == ow && ci > co))
                            for (long n = 0; n < B; ++n)
                                for (int i = 0; i < H; ++i)
                                    for (int j = 0; j < W; ++j) {
                                        int ii = i + a - oh, jj = j + b - ow;
                                        if (ii < 0 || ii >= H || jj < 0 || jj >= W)
                                            continue;
                                        s += dy[n * img + co * plane + (long)i * W + j] *
                                             x[n * img + ci * plane + (long)ii * W + jj];
                                    }
                        if (a == oh && b == ow && ci == co)
                            s += gld * (double)H * (double)W / kw(K, C, k, co, co, a, b);
                        dK[(((long)co * C + ci) * k + a) * k + b] = s;
                    }
    }
    return ORC_OK;
}

/* Backward of the FInC unit (the four blocks TL, TR, BL, BR in sequence):
 * the inputs of the last three blocks, h1 = TL(x), h2 = TR(h1),
 * h3 = BL(h2), are recomputed by the forward; then the chain rule takes the
 * blocks in reverse, each block's orc_backward receiving the input gradient
 * of the block after it.  The unit's log|det| is the sum of its blocks', so
 * each block takes the same gld.  dx or dK4 may be NULL. */
int orc_unit_backward(const double *x, const double *dy, const double *K4, double *dx,
                      double *dK4, double gld, long B, int C, int H, int W, int k)
{
    if (bad_shape(B, C, H, W, k, 0) || !x || !dy || !K4)
        return ORC_EINVAL;
    const long n = B * (long)C * H * W, ksz = (long)C * C * k * k;
    const size_t bytes = sizeof(double) * (n > 0 ? n : 1);
    double *h[4] = {(double *)x, malloc(bytes), malloc(bytes), malloc(bytes)};
    double *g = malloc(bytes), *gn = malloc(bytes);
    int rc = (h[1] && h[2] && h[3] && g && gn) ? ORC_OK : ORC_ENOMEM;
    for (int q = 0; q < 3 && rc == ORC_OK; ++q)
        rc = orc_forward(h[q], h[q + 1], K4 + q * ksz, B, C, H, W, k, UNIT_ORDER[q]);
    if (rc == ORC_OK)
        memcpy(g, dy, sizeof(double) * n);
    for (int q = 3; q >= 0 && rc == ORC_OK; --q) {
        rc = orc_backward(h[q], g, K4 + q * ksz, gn, dK4 ? dK4 + q * ksz : NULL, gld, B, C, H,
                          W, k, UNIT_ORDER[q]);
        memcpy(g, gn, sizeof(double) * n);
    }
    if (rc == ORC_OK && dx)
        memcpy(dx, g, sizeof(double) * n);
    free(h[1]);
    free(h[2]);
    free(h[3]);
    free(g);
    free(gn);
    return rc;
}

/* Backward of the channel-split unit: quarter g (channels g C/4 .. (g+1) C/4
 * of every image) is one block with corner g and its own weights, so its
 * gradients come from orc_backward on that quarter alone, over the whole
 * batch; gld multiplies the unit's log|det| (the quarters' sum).  dx or
 * dKq4 may be NULL. */
int orc_split_backward(const double *x, const double *dy, const double *Kq4, double *dx,
                       double *dKq4, double gld, long B, int C, int H, int W, int k)
{
    if (bad_shape(B, C, H, W, k, 0) || C % 4 != 0 || !x || !dy || !Kq4)
        return ORC_EINVAL;
    const int Cq = C / 4;
    const long part = (long)Cq * H * W, ksz = (long)Cq * Cq * k * k;
    const size_t bytes = sizeof(double) * (B * part > 0 ? B * part : 1);
    double *xq = malloc(bytes), *gq = malloc(bytes), *dq = malloc(bytes);
    int rc = (xq && gq && dq) ? ORC_OK : ORC_ENOMEM;
    for (int g = 0; g < 4 && rc == ORC_OK; ++g) {
        for (long b = 0; b < B; ++b) {
            const long off = (b * C + (long)g * Cq) * H * W;
            memcpy(xq + b * part, x + off, sizeof(double) * part);
            memcpy(gq + b * part, dy + off, sizeof(double) * part);
        }
        rc = orc_backward(xq, gq, Kq4 + g * ksz, dq, dKq4 ? dKq4 + g * ksz : NULL, gld, B, Cq,
                          H, W, k, g);
        for (long b = 0; dx && rc == ORC_OK && b < B; ++b)
            memcpy(dx + (b * C + (long)g * Cq) * H * W, dq + b * part, sizeof(double) * part);
    }
    free(xq);
    free(gq);
    free(dq);
    return rc;
}

/* Backward of actnorm y = s x + b (per channel), whose log|det| is
 * H W sum_c log|s_c| per image:
 *   dx = s dy;  ds[c] = sum over images and pixels of dy x, plus
 *   gld H W / s[c];  db[c] = sum over images and pixels of dy.
 * dx, ds or db may be NULL. */
int orc_actnorm_backward(const double *x, const double *dy, const double *s, double *dx,
                         double *ds, double *db, double gld, long B, int C, int H, int W)
{
    if (B < 0 || C < 1 || H < 1 || W < 1 || !s || (B > 0 && (!x || !dy)))
        return ORC_EINVAL;
    const long plane = (long)H * W;
    for (int c = 0; c < C; ++c) {
        double sx = 0.0, sy = 0.0;
        for (long n = 0; n < B; ++n)
            for (long p = 0; p < plane; ++p) {
                const long o = (n * C + c) * plane + p;
                sx += dy[o] * x[o];
                sy += dy[o];
                if (dx)
                    dx[o] = s[c] * dy[o];
            }
        if (ds)
            ds[c] = sx + gld * (double)plane / s[c];
        if (db)
            db[c] = sy;
    }
    return ORC_OK;
}

/* Negative log-likelihood of each image (Sec. 3, the log-probability
 * equation, negated): the flow maps the image to latents whose values z
 * are standard normal, and the layers' log|det| (summed per image in
 * logdet) corrects the density, so
 *   nll[b] = sum over the image's latent values of (z^2 + log 2 pi) / 2
 *            - logdet[b],
 * and bits per dimension (Sec. 5, BPD equation) bpd[b] = nll[b] log2(e) / D
 * with D the image's values (the latents' total, n[0] + ... + n[L-1]).
 * z[l] holds B blocks of n[l] values, one per image.  bpd may be NULL. */
int orc_gauss_nll(const double *const *z, const long *n, int L, long B, const double *logdet,
                  double *nll, double *bpd)
{
    if (L < 1 || B < 0 || !z || !n || !logdet || !nll)
        return ORC_EINVAL;
    long D = 0;
    for (int l = 0; l < L; ++l) {
        if (n[l] < 1 || (B > 0 && !z[l]))
            return ORC_EINVAL;
        D += n[l];
    }
    const double log2pi = log(2.0 * 3.14159265358979323846);
    for (long b = 0; b < B; ++b) {
        double q = 0.0;
        for (int l = 0; l < L; ++l)
            for (long e = 0; e < n[l]; ++e) {
                const double v = z[l][b * n[l] + e];
                q += 0.5 * (v * v + log2pi);
            }
        nll[b] = q - logdet[b];
        if (bpd)
            bpd[b] = nll[b] / ((double)D * log(2.0));
    }
    return ORC_OK;
}

/* log|det| of the stack's forward direction, one image: every unit's (the
 * sum of its blocks') plus every actnorm's H W sum_c log|s_c|, at the
 * level's spatial size (the split and squeeze move values: no term). */
int orc_stack_logdet(const double *K, const double *scale, int L, int U, int C1, int H1, int W1,
                     int k, double *out)
{
    if (L < 1 || U < 0 || C1 < 1 || H1 < 1 || W1 < 1 || k < 1 || !K || !scale || !out)
        return ORC_EINVAL;
    double s = 0.0;
    int rc = ORC_OK;
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l, H = H1 >> l, W = W1 >> l;
        const long ksz = (long)C * C * k * k;
        const double *Kl = K + stack_koff(l, U, C1, k);
        const double *sl = scale + stack_soff(l, U, C1);
        for (int u = 0; u < U; ++u) {
            double v;
            const int r = orc_unit_logdet(Kl + (long)u * 4 * ksz, C, k, H, W, &v);
            if (r == ORC_EINVAL)
                return r;
            if (r != ORC_OK)
                rc = r;
            s += v;
            for (int c = 0; c < C; ++c)
                s += (double)H * W * log(fabs(sl[(long)u * C + c]));
        }
    }
    *out = s;
    return rc;
}

/* Backward of the stack's forward direction (orc_stack_forward) for the
 * gradients dz[l] of a loss with respect to its latents, plus gld times the
 * stack's log|det| of one image (orc_stack_logdet; -B for the log|det| part
 * of a batch's summed negative log-likelihood).
 * Every unit's input and every actnorm's input are recomputed by the forward;
 * then, level by level from the top: the level output's gradient is the
 * unsqueezed gradient of the next level's input (its first half, which went
 * on) beside dz[l] (its second half, the latent); the units run in reverse,
 * each actnorm's backward before its unit's.  Outputs: dx (the input's
 * gradient) and dK, dscale, dbias in the layouts of K, scale and bias; any
 * may be NULL. */
int orc_stack_backward(const double *x, const double *const *dz, const double *K,
                       const double *scale, const double *bias, double *dx, double *dK,
                       double *dscale, double *dbias, double gld, long B, int L, int U, int C1,
                       int H1, int W1, int k)
{
    if (L < 1 || U < 0 || B < 0 || C1 < 1 || H1 < 1 || W1 < 1 || k < 1 || !x || !dz || !K ||
        !scale || !bias)
        return ORC_EINVAL;
    if (((H1 | W1) & ((1 << (L - 1)) - 1)) || (L > 1 && (C1 & 1)))
        return ORC_EINVAL;
    const long n0 = B * (long)C1 * H1 * W1;
    const size_t bytes = sizeof(double) * (n0 > 0 ? n0 : 1);
    /* per level: the level's input, then per unit its input and its
     * actnorm's input (2 U + 1 activations of the level's size) */
    long total = 0;
    for (int l = 0; l < L; ++l)
        total += (2L * U + 1) * (n0 >> l);
    double *acts = malloc(sizeof(double) * (total > 0 ? total : 1));
    double *g = malloc(bytes), *gn = malloc(bytes), *gt = malloc(bytes);
    int rc = (acts && g && gn && gt) ? ORC_OK : ORC_ENOMEM;
    long off[8];
    /* forward, keeping the activations */
    long o = 0;
    for (int l = 0; l < L && rc == ORC_OK; ++l) {
        const int C = C1 << l, H = H1 >> l, W = W1 >> l;
        const long n = B * (long)C * H * W, ksz = (long)C * C * k * k;
        const double *Kl = K + stack_koff(l, U, C1, k);
        const double *sl = scale + stack_soff(l, U, C1), *bl = bias + stack_soff(l, U, C1);
        off[l] = o;
        double *in = acts + o;
        if (l == 0)
            memcpy(in, x, sizeof(double) * n);
        for (int u = 0; u < U && rc == ORC_OK; ++u) {
            /* h_u (the unit's input), t_u = unit(h_u), h_{u+1} = actnorm(t_u) */
            double *hu = in + (2L * u) * n, *tu = hu + n, *next = tu + n;
            rc = orc_unit_forward(hu, tu, Kl + (long)u * 4 * ksz, B, C, H, W, k);
            orc_actnorm_forward(tu, next, sl + (long)u * C, bl + (long)u * C, B, C, H, W);
        }
        o += (2L * U + 1) * n;
        if (l < L - 1 && rc == ORC_OK) {
            /* the level's output; its first half, squeezed, is the next input */
            const double *hout = in + (2L * U) * n;
            const int Ch = C / 2;
            const long hw = (long)H * W;
            for (long b = 0; b < B; ++b)
                memcpy(gn + b * Ch * hw, hout + b * C * hw, sizeof(double) * Ch * hw);
            orc_squeeze(gn, acts + o, B, Ch, H, W);
        }
    }
    /* backward, from the top level down */
    for (int l = L - 1; l >= 0 && rc == ORC_OK; --l) {
        const int C = C1 << l, H = H1 >> l, W = W1 >> l;
        const long n = B * (long)C * H * W, ksz = (long)C * C * k * k, hw = (long)H * W;
        const double *Kl = K + stack_koff(l, U, C1, k);
        const double *sl = scale + stack_soff(l, U, C1);
        double *in = acts + off[l];
        if (l == L - 1) {
            memcpy(g, dz[l], sizeof(double) * n);
        } else {
            /* g holds the next level's input gradient (2C channels at H/2) */
            const int Ch = C / 2;
            orc_unsqueeze(g, gn, B, 2 * C, H / 2, W / 2);
            for (long b = 0; b < B; ++b) {
                memcpy(g + b * C * hw, gn + b * Ch * hw, sizeof(double) * Ch * hw);
                memcpy(g + (b * C + Ch) * hw, dz[l] + b * Ch * hw, sizeof(double) * Ch * hw);
            }
        }
        for (int u = U - 1; u >= 0 && rc == ORC_OK; --u) {
            double *hu = in + (2L * u) * n, *tu = hu + n;
            const long so = stack_soff(l, U, C1) + (long)u * C;
            rc = orc_actnorm_backward(tu, g, sl + (long)u * C, gt, dscale ? dscale + so : NULL,
                                      dbias ? dbias + so : NULL, gld, B, C, H, W);
            if (rc == ORC_OK)
                rc = orc_unit_backward(hu, gt, Kl + (long)u * 4 * ksz, g,
                                       dK ? dK + stack_koff(l, U, C1, k) + (long)u * 4 * ksz
                                          : NULL,
                                       gld, B, C, H, W, k);
        }
    }
    if (rc == ORC_OK && dx)
        memcpy(dx, g, sizeof(double) * n0);
    free(acts);
    free(g);
    free(gn);
    free(gt);
    return rc;
}

/* ==========================================================================
 * The full FInC Flow (Sec. 4.4 "Architecture", Fig. 2b and 2c).
 *
 * A FInC Flow Step is, in the forward direction, a FInC unit (the
 * channel-split unit above, Sec. 4.3), an actnorm, an invertible 1x1
 * convolution and an affine coupling layer, in that order.  Readings taken
 * where the paper only names the layers (it follows Glow for all three):
 *  - 1x1 convolution: y = Wm x at every pixel, Wm a C x C matrix; its
 *    log|det| is H W log|det Wm|.
 *  - Coupling (RealNVP / Glow): x = [xa, xb] (channel halves); the network
 *    h = NN(xa) has C output channels, its first half the shift t, its
 *    second half the raw scale r; scale = sigmoid(r + 2);
 *    yb = (xb + t) * scale, ya = xa; log|det| = sum log scale (per image).
 *    NN is a 3x3 convolution, ReLU, a 1x1 convolution, ReLU, and a 3x3
 *    convolution whose output channel c is multiplied by exp(3 ls[c]) (the
 *    "modified" zero-initialised 3x3 convolution of Glow / Emerging); every
 *    convolution has a bias and zero "same" padding.
 *  - Multi-scale (Fig. 2c): per level, squeeze, K steps, then (below the
 *    top) split: the first half h1 goes on; the second half h2 becomes the
 *    latent z = (h2 - mean) * exp(-logsd) with (mean, logsd) = the halves of
 *    a prior network on h1, a 3x3 convolution with bias and exp(3 ls)
 *    output scale (Glow's split prior; its log|det| is -sum logsd).  The
 *    top level's output is the last latent.
 *
 * Parameter layout (doubles; C the level's channels, Ch = C/2, q = C/4,
 * hid the coupling network's width, k the unit kernel size):
 *   step:  Kq4 (4 q q k k) | an_s (C) | an_b (C) | Wm (C C) |
 *          W1 (hid Ch 3 3) | b1 (hid) | W2 (hid hid) | b2 (hid) |
 *          W3 (C hid 3 3) | b3 (C) | ls3 (C)
 *   prior: Wp (C Ch 3 3) | bp (C) | lsp (C)
 *   flow:  for level l = 0 .. L-1: K steps, then (l < L-1) the prior.
 * Convolution weights are OIHW.  Level l has C_l = 4 C0 2^l channels and
 * H0 / 2^(l+1) x W0 / 2^(l+1) pixels.
 * ========================================================================== */

/* y = Wm x at every pixel. */
int orc_conv1x1_forward(const double *x, double *y, const double *Wm, long B, int C, int H,
                        int W)
{
    if (B < 0 || C < 1 || H < 1 || W < 1 || !x || !y || !Wm)
        return ORC_EINVAL;
    const long plane = (long)H * W;
    for (long n = 0; n < B; ++n)
        for (int co = 0; co < C; ++co)
            for (long p = 0; p < plane; ++p) {
                double s = 0.0;
                for (int ci = 0; ci < C; ++ci)
                    s += Wm[(long)co * C + ci] * x[(n * C + ci) * plane + p];
                y[(n * C + co) * plane + p] = s;
            }
    return ORC_OK;
}

/* LU factorisation with partial pivoting of a C x C matrix (row-major, in
 * place); perm receives the row order.  Returns the log|det| and its sign in
 * *sign (0 if singular). */
static double lu_factor(double *A, int *perm, int C, int *sign)
{
    double ld = 0.0;
    int sg = 1;
    for (int i = 0; i < C; ++i)
        perm[i] = i;
    for (int c = 0; c < C; ++c) {
        int piv = c;
        for (int r = c + 1; r < C; ++r)
            if (fabs(A[(long)r * C + c]) > fabs(A[(long)piv * C + c]))
                piv = r;
        if (A[(long)piv * C + c] == 0.0) {
            *sign = 0;
            return -INFINITY;
        }
        if (piv != c) {
            for (int j = 0; j < C; ++j) {
                double t = A[(long)c * C + j];
                A[(long)c * C + j] = A[(long)piv * C + j];
                A[(long)piv * C + j] = t;
            }
            int t = perm[c];
            perm[c] = perm[piv];
            perm[piv] = t;
            sg = -sg;
        }
        double d = A[(long)c * C + c];
        if (d < 0)
            sg = -sg;
        ld += log(fabs(d));
        for (int r = c + 1; r < C; ++r) {
            double f = A[(long)r * C + c] / d;
            A[(long)r * C + c] = f;
            for (int j = c + 1; j < C; ++j)
                A[(long)r * C + j] -= f * A[(long)c * C + j];
        }
    }
    *sign = sg;
    return ld;
}

/* x = Wm^-1 y at every pixel, by LU with partial pivoting and substitution. */
int orc_conv1x1_inverse(const double *y, double *x, const double *Wm, long B, int C, int H,
                        int W)
{
    if (B < 0 || C < 1 || H < 1 || W < 1 || !x || !y || !Wm)
        return ORC_EINVAL;
    double *A = (double *)malloc(sizeof(double) * C * C);
    double *v = (double *)malloc(sizeof(double) * C);
    int *perm = (int *)malloc(sizeof(int) * C);
    if (!A || !v || !perm) {
        free(A);
        free(v);
        free(perm);
        return ORC_ENOMEM;
    }
    memcpy(A, Wm, sizeof(double) * C * C);
    int sign;
    lu_factor(A, perm, C, &sign);
    int rc = sign == 0 ? ORC_ESINGULAR : ORC_OK;
    const long plane = (long)H * W;
    for (long n = 0; n < B && rc == ORC_OK; ++n)
        for (long p = 0; p < plane; ++p) {
            for (int r = 0; r < C; ++r) { /* L v = P y */
                double s = y[(n * C + perm[r]) * plane + p];
                for (int j = 0; j < r; ++j)
                    s -= A[(long)r * C + j] * v[j];
                v[r] = s;
            }
            for (int r = C - 1; r >= 0; --r) { /* U x = v */
                double s = v[r];
                for (int j = r + 1; j < C; ++j)
                    s -= A[(long)r * C + j] * v[j];
                v[r] = s / A[(long)r * C + r];
            }
            for (int c = 0; c < C; ++c)
                x[(n * C + c) * plane + p] = v[c];
        }
    free(A);
    free(v);
    free(perm);
    return rc;
}

/* H W log|det Wm|. */
int orc_conv1x1_logdet(const double *Wm, int C, int H, int W, double *out)
{
    if (C < 1 || H < 1 || W < 1 || !Wm || !out)
        return ORC_EINVAL;
    double *A = (double *)malloc(sizeof(double) * C * C);
    int *perm = (int *)malloc(sizeof(int) * C);
    if (!A || !perm) {
        free(A);
        free(perm);
        return ORC_ENOMEM;
    }
    memcpy(A, Wm, sizeof(double) * C * C);
    int sign;
    double ld = lu_factor(A, perm, C, &sign);
    free(A);
    free(perm);
    *out = (double)H * (double)W * ld;
    return sign == 0 ? ORC_ESINGULAR : ORC_OK;
}

/* Same-padded r x r convolution (r odd), cross-correlation with zero padding
 * (r-1)/2 on every side, plus bias; then ReLU (relu != 0), then multiplied by
 * exp(3 ls[co]) (ls != NULL).  x (B, Ci, H, W), y (B, Co, H, W). */
static void conv_same(const double *x, double *y, const double *Wt, const double *bias,
                      const double *ls, long B, int Ci, int Co, int H, int W, int r, int relu)
{
    const long plane = (long)H * W;
    const int pad = (r - 1) / 2;
    for (long n = 0; n < B; ++n)
        for (int co = 0; co < Co; ++co)
            for (int i = 0; i < H; ++i)
                for (int j = 0; j < W; ++j) {
                    double s = bias[co];
                    for (int ci = 0; ci < Ci; ++ci)
                        for (int a = 0; a < r; ++a)
                            for (int b = 0; b < r; ++b) {
                                int ii = i + a - pad, jj = j + b - pad;
                                if (ii < 0 || ii >= H || jj < 0 || jj >= W)
                                    continue;
                                s += Wt[(((long)co * Ci + ci) * r + a) * r + b] *
                                     x[(n * Ci + ci) * plane + (long)ii * W + jj];
                            }
                    if (relu && s < 0.0)
                        s = 0.0;
                    if (ls)
                        s *= exp(3.0 * ls[co]);
                    y[(n * Co + co) * plane + (long)i * W + j] = s;
                }
}

static long coupling_params(int C, int hid)
{
    const long Ch = C / 2;
    return (long)hid * Ch * 9 + hid + (long)hid * hid + hid + (long)C * hid * 9 + 2L * C;
}

static long step_params(int C, int k, int hid)
{
    const long q = C / 4;
    return 4 * q * q * k * k + 2L * C + (long)C * C + coupling_params(C, hid);
}

static long prior_params(int C) { return (long)C * (C / 2) * 9 + 2L * C; }

/* The coupling network on xa (B, C/2, H, W) -> h (B, C, H, W); cp points at
 * W1 of the layout above. */
int orc_coupling_net(const double *xa, double *h, const double *cp, long B, int C, int H,
                     int W, int hid)
{
    if (B < 0 || C < 2 || (C & 1) || H < 1 || W < 1 || hid < 1 || !xa || !h || !cp)
        return ORC_EINVAL;
    const int Ch = C / 2;
    const long plane = (long)H * W;
    const double *W1 = cp, *b1 = W1 + (long)hid * Ch * 9, *W2 = b1 + hid, *b2 = W2 + (long)hid * hid;
    const double *W3 = b2 + hid, *b3 = W3 + (long)C * hid * 9, *ls3 = b3 + C;
    double *t1 = (double *)malloc(sizeof(double) * (B * hid * plane > 0 ? B * hid * plane : 1));
    double *t2 = (double *)malloc(sizeof(double) * (B * hid * plane > 0 ? B * hid * plane : 1));
    if (!t1 || !t2) {
        free(t1);
        free(t2);
        return ORC_ENOMEM;
    }
    conv_same(xa, t1, W1, b1, NULL, B, Ch, hid, H, W, 3, 1);
    conv_same(t1, t2, W2, b2, NULL, B, hid, hid, H, W, 1, 1);
    conv_same(t2, h, W3, b3, ls3, B, hid, C, H, W, 3, 0);
    free(t1);
    free(t2);
    return ORC_OK;
}

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* Affine coupling, forward: ya = xa, yb = (xb + t) sigmoid(r + 2); logdet[n]
 * += sum over the image of log sigmoid(r + 2) (logdet may be NULL). */
int orc_coupling_forward(const double *x, double *y, const double *cp, long B, int C, int H,
                         int W, int hid, double *logdet)
{
    if (B < 0 || C < 2 || (C & 1) || H < 1 || W < 1 || !x || !y || !cp)
        return ORC_EINVAL;
    const int Ch = C / 2;
    const long plane = (long)H * W, half = Ch * plane;
    double *xa = (double *)malloc(sizeof(double) * (B * half > 0 ? B * half : 1));
    double *h = (double *)malloc(sizeof(double) * (B * 2 * half > 0 ? B * 2 * half : 1));
    if (!xa || !h) {
        free(xa);
        free(h);
        return ORC_ENOMEM;
    }
    for (long n = 0; n < B; ++n)
        memcpy(xa + n * half, x + n * 2 * half, sizeof(double) * half);
    int rc = orc_coupling_net(xa, h, cp, B, C, H, W, hid);
    for (long n = 0; n < B && rc == ORC_OK; ++n) {
        double ld = 0.0;
        for (long e = 0; e < half; ++e) {
            double t = h[n * 2 * half + e], r = h[n * 2 * half + half + e];
            double s = sigmoid(r + 2.0);
            y[n * 2 * half + e] = x[n * 2 * half + e];
            y[n * 2 * half + half + e] = (x[n * 2 * half + half + e] + t) * s;
            ld += log(s);
        }
        if (logdet)
            logdet[n] += ld;
    }
    free(xa);
    free(h);
    return rc;
}

/* Affine coupling, inverse: xa = ya, xb = yb / sigmoid(r + 2) - t with
 * (t, r) = NN(ya). */
int orc_coupling_inverse(const double *y, double *x, const double *cp, long B, int C, int H,
                         int W, int hid)
{
    if (B < 0 || C < 2 || (C & 1) || H < 1 || W < 1 || !x || !y || !cp)
        return ORC_EINVAL;
    const int Ch = C / 2;
    const long plane = (long)H * W, half = Ch * plane;
    double *ya = (double *)malloc(sizeof(double) * (B * half > 0 ? B * half : 1));
    double *h = (double *)malloc(sizeof(double) * (B * 2 * half > 0 ? B * 2 * half : 1));
    if (!ya || !h) {
        free(ya);
        free(h);
        return ORC_ENOMEM;
    }
    for (long n = 0; n < B; ++n)
        memcpy(ya + n * half, y + n * 2 * half, sizeof(double) * half);
    int rc = orc_coupling_net(ya, h, cp, B, C, H, W, hid);
    for (long n = 0; n < B && rc == ORC_OK; ++n)
        for (long e = 0; e < half; ++e) {
            double t = h[n * 2 * half + e], r = h[n * 2 * half + half + e];
            x[n * 2 * half + e] = y[n * 2 * half + e];
            x[n * 2 * half + half + e] = y[n * 2 * half + half + e] / sigmoid(r + 2.0) - t;
        }
    free(ya);
    free(h);
    return rc;
}

/* One FInC Flow Step, forward: unit (channel-split), actnorm, 1x1, coupling.
 * logdet (B values, may be NULL) is incremented by the step's log|det| per
 * image. */
int orc_step_forward(const double *x, double *y, const double *sp, long B, int C, int H, int W,
                     int k, int hid, double *logdet)
{
    if (B < 0 || C < 4 || (C & 3) || H < 1 || W < 1 || k < 1 || !x || !y || !sp)
        return ORC_EINVAL;
    const int q = C / 4;
    const long n_el = B * (long)C * H * W;
    const double *Kq4 = sp, *s = Kq4 + 4L * q * q * k * k, *b = s + C, *Wm = b + C;
    const double *cp = Wm + (long)C * C;
    double *t1 = (double *)malloc(sizeof(double) * (n_el > 0 ? n_el : 1));
    double *t2 = (double *)malloc(sizeof(double) * (n_el > 0 ? n_el : 1));
    if (!t1 || !t2) {
        free(t1);
        free(t2);
        return ORC_ENOMEM;
    }
    int rc = orc_split_forward(x, t1, Kq4, B, C, H, W, k);
    if (rc == ORC_OK) {
        orc_actnorm_forward(t1, t2, s, b, B, C, H, W);
        rc = orc_conv1x1_forward(t2, t1, Wm, B, C, H, W);
    }
    if (rc == ORC_OK)
        rc = orc_coupling_forward(t1, y, cp, B, C, H, W, hid, logdet);
    if (rc == ORC_OK && logdet) {
        double lu, lw, la = 0.0;
        rc = orc_split_logdet(Kq4, C, k, H, W, &lu);
        if (rc == ORC_OK)
            rc = orc_conv1x1_logdet(Wm, C, H, W, &lw);
        for (int c = 0; c < C; ++c)
            la += log(fabs(s[c]));
        la *= (double)H * W;
        for (long n = 0; n < B && rc == ORC_OK; ++n)
            logdet[n] += lu + la + lw;
    }
    free(t1);
    free(t2);
    return rc;
}

/* One FInC Flow Step, inverse: coupling^-1, 1x1^-1, actnorm^-1, unit^-1. */
int orc_step_inverse(const double *y, double *x, const double *sp, long B, int C, int H, int W,
                     int k, int hid)
{
    if (B < 0 || C < 4 || (C & 3) || H < 1 || W < 1 || k < 1 || !x || !y || !sp)
        return ORC_EINVAL;
    const int q = C / 4;
    const long n_el = B * (long)C * H * W;
    const double *Kq4 = sp, *s = Kq4 + 4L * q * q * k * k, *b = s + C, *Wm = b + C;
    const double *cp = Wm + (long)C * C;
    double *t1 = (double *)malloc(sizeof(double) * (n_el > 0 ? n_el : 1));
    double *t2 = (double *)malloc(sizeof(double) * (n_el > 0 ? n_el : 1));
    if (!t1 || !t2) {
        free(t1);
        free(t2);
        return ORC_ENOMEM;
    }
    int rc = orc_coupling_inverse(y, t1, cp, B, C, H, W, hid);
    if (rc == ORC_OK)
        rc = orc_conv1x1_inverse(t1, t2, Wm, B, C, H, W);
    if (rc == ORC_OK) {
        orc_actnorm_inverse(t2, t1, s, b, B, C, H, W);
        rc = orc_split_inverse(t1, x, Kq4, B, C, H, W, k);
    }
    free(t1);
    free(t2);
    return rc;
}

/* Floats of a flow's parameters (layout above). */
long orc_flow_params(int L, int K, int C0, int k, int hid)
{
    long n = 0;
    for (int l = 0; l < L; ++l) {
        const int C = (4 * C0) << l;
        n += (long)K * step_params(C, k, hid);
        if (l < L - 1)
            n += prior_params(C);
    }
    return n;
}

/* Split prior of a level: (mean, logsd) = halves of a 3x3 convolution of h1
 * (B, C/2, H, W) with bias and exp(3 ls) output scale. */
static int prior_net(const double *h1, double *ms, const double *pp, long B, int C, int H, int W)
{
    const int Ch = C / 2;
    conv_same(h1, ms, pp, pp + (long)C * Ch * 9, pp + (long)C * Ch * 9 + C, B, Ch, C, H, W, 3,
              0);
    return ORC_OK;
}

/* Multi-scale flow, forward (density direction): x (B, C0, H0, W0) -> the
 * latents z[l] (l < L-1: (B, C_l/2, H_l, W_l); z[L-1]: (B, C_{L-1}, H_{L-1},
 * W_{L-1})) and logdet[n] (B values, overwritten): the sum of every step's
 * log|det| and of -sum logsd of every split. */
int orc_flow_forward(const double *x, double *const *z, const double *params, long B, int L,
                     int K, int C0, int H0, int W0, int k, int hid, double *logdet)
{
    if (B < 0 || L < 1 || K < 0 || C0 < 1 || k < 1 || hid < 1 || !x || !z || !params ||
        !logdet || (H0 % (2 << (L - 1))) || (W0 % (2 << (L - 1))))
        return ORC_EINVAL;
    const long tot = B * (long)C0 * H0 * W0;
    double *h = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    double *t = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    double *ms = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    if (!h || !t || !ms) {
        free(h);
        free(t);
        free(ms);
        return ORC_ENOMEM;
    }
    for (long n = 0; n < B; ++n)
        logdet[n] = 0.0;
    memcpy(h, x, sizeof(double) * tot);
    int C = C0, H = H0, W = W0, rc = ORC_OK;
    const double *p = params;
    for (int l = 0; l < L && rc == ORC_OK; ++l) {
        orc_squeeze(h, t, B, C, H, W);
        C *= 4;
        H /= 2;
        W /= 2;
        for (int s = 0; s < K && rc == ORC_OK; ++s) {
            rc = orc_step_forward(t, h, p, B, C, H, W, k, hid, logdet);
            memcpy(t, h, sizeof(double) * tot);
            p += step_params(C, k, hid);
        }
        if (rc != ORC_OK)
            break;
        const long plane = (long)H * W;
        if (l == L - 1) {
            memcpy(z[l], t, sizeof(double) * B * C * plane);
            break;
        }
        const int Ch = C / 2;
        for (long n = 0; n < B; ++n) /* h1 */
            memcpy(h + n * Ch * plane, t + n * C * plane, sizeof(double) * Ch * plane);
        prior_net(h, ms, p, B, C, H, W);
        for (long n = 0; n < B; ++n) {
            double ld = 0.0;
            for (long e = 0; e < Ch * plane; ++e) {
                double mean = ms[n * C * plane + e], logsd = ms[n * C * plane + Ch * plane + e];
                z[l][n * Ch * plane + e] = (t[n * C * plane + Ch * plane + e] - mean) * exp(-logsd);
                ld -= logsd;
            }
            logdet[n] += ld;
        }
        p += prior_params(C);
        C = Ch;
    }
    free(h);
    free(t);
    free(ms);
    return rc;
}

/* Multi-scale flow, sampling direction: from the latents to x. */
int orc_flow_sample(const double *const *z, double *x, const double *params, long B, int L,
                    int K, int C0, int H0, int W0, int k, int hid)
{
    if (B < 0 || L < 1 || K < 0 || C0 < 1 || k < 1 || hid < 1 || !x || !z || !params ||
        (H0 % (2 << (L - 1))) || (W0 % (2 << (L - 1))))
        return ORC_EINVAL;
    const long tot = B * (long)C0 * H0 * W0;
    double *h = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    double *t = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    double *ms = (double *)malloc(sizeof(double) * (tot > 0 ? tot : 1));
    const double **sp = (const double **)malloc(sizeof(double *) * (L * (K + 1) + 1));
    if (!h || !t || !ms || !sp) {
        free(h);
        free(t);
        free(ms);
        free(sp);
        return ORC_ENOMEM;
    }
    /* where each level's steps and prior start */
    const double *p = params;
    for (int l = 0; l < L; ++l) {
        const int C = (4 * C0) << l;
        for (int s = 0; s < K; ++s) {
            sp[l * (K + 1) + s] = p;
            p += step_params(C, k, hid);
        }
        sp[l * (K + 1) + K] = p;
        if (l < L - 1)
            p += prior_params(C);
    }
    int rc = ORC_OK;
    int C = (4 * C0) << (L - 1), H = H0 >> L, W = W0 >> L;
    memcpy(h, z[L - 1], sizeof(double) * B * C * H * W);
    for (int l = L - 1; l >= 0 && rc == ORC_OK; --l) {
        const long plane = (long)H * W;
        if (l < L - 1) {
            /* h holds h1 (B, C/2, H, W): the prior gives h2 = mean + exp(logsd) z */
            const int Ch = C / 2;
            prior_net(h, ms, sp[l * (K + 1) + K], B, C, H, W);
            for (long n = 0; n < B; ++n) {
                memcpy(t + n * C * plane, h + n * Ch * plane, sizeof(double) * Ch * plane);
                for (long e = 0; e < Ch * plane; ++e) {
                    double mean = ms[n * C * plane + e], logsd = ms[n * C * plane + Ch * plane + e];
                    t[n * C * plane + Ch * plane + e] = mean + exp(logsd) * z[l][n * Ch * plane + e];
                }
            }
            memcpy(h, t, sizeof(double) * B * C * plane);
        }
        for (int s = K - 1; s >= 0 && rc == ORC_OK; --s) {
            rc = orc_step_inverse(h, t, sp[l * (K + 1) + s], B, C, H, W, k, hid);
            memcpy(h, t, sizeof(double) * B * C * plane);
        }
        orc_unsqueeze(h, t, B, C, H, W);
        C /= 4;
        H *= 2;
        W *= 2;
        memcpy(h, t, sizeof(double) * B * C * H * W);
        /* the level below kept h (now the first half of its channels) */
        if (l > 0)
            C = C * 2; /* below: C_{l-1} = C_l / 2 channels, of which h is the half */
    }
    if (rc == ORC_OK)
        memcpy(x, h, sizeof(double) * tot);
    free(h);
    free(t);
    free(ms);
    free(sp);
    return rc;
}
