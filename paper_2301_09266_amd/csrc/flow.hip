// flow.hip -- the full FInC Flow on gfx950 (Sec. 4.4 "Architecture",
// Fig. 2b and 2c): the Step (channel-split FInC unit, actnorm, invertible
// 1x1 convolution, affine coupling) and the multi-scale flow with split
// priors, forward (density) and sampling directions, behind the C ABI of
// include/finc.h.
//
// Readings (the paper names these layers and follows Glow for them):
//  * 1x1 convolution: y = Wm x at every pixel; log|det| = H W log|det Wm|.
//  * Coupling: x = [xa, xb] (channel halves); h = NN(xa) has C channels, the
//    first half the shift t, the second the raw scale r; s = sigmoid(r + 2);
//    yb = (xb + t) s; log|det| = sum log s.  NN = 3x3 conv, ReLU, 1x1 conv,
//    ReLU, 3x3 conv times exp(3 ls) per output channel; every conv has a
//    bias and zero "same" padding.
//  * Multi-scale: per level squeeze, K Steps, then (below the top) split:
//    h1 goes on, z = (h2 - mean) exp(-logsd) with (mean, logsd) the halves
//    of a 3x3 conv (bias, exp(3 ls) scale) of h1; log|det| -sum logsd.
//
// Design:
//  * Every convolution of the coupling and prior networks, and the 1x1
//    convolution, is one kernel: an fp32 MFMA implicit GEMM
//    (v_mfma_f32_16x16x4_f32), D[c_out][pixel] = sum over k = (c_in, tap) of
//    W[c_out][k] x[k][pixel], with the K axis staged through LDS 64 values
//    at a time (weights and the gathered input window, both k-contiguous so
//    one 16-byte LDS read feeds four MFMAs), the next chunk's global loads
//    in flight during the current chunk's MFMAs, and bias, ReLU and the
//    output scale fused into the store.
//  * The 1x1 convolution and the actnorm next to it are one affine map per
//    pixel: prepared once per weight set in fp64 (Wm diag(s), Wm b forward;
//    diag(1/s) Wm^-1, -b/s inverse, by Gauss-Jordan elimination with partial
//    pivoting), applied by the same convolution kernel.
//  * The channel-split unit is the wavefront inverse of finc.hip (prepared
//    weights), the coupling's affine map and the split prior small
//    elementwise kernels; log|det| per image is summed in a fixed order
//    (one workgroup per image), so results are bitwise deterministic.
//  * All tensors are NCHW fp32; kernels take image strides, so channel
//    halves of a level tensor are read and written in place.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "conv_gemm.h"
#include "finc.h"

namespace {

// ---------------------------------------------------------------------------
// The 1x1 convolution with its actnorm, prepared in fp64 (one workgroup per
// weight set).  In the Step, u = s x + b (actnorm), v = Wm u, so
//   forward: v = (Wm diag(s)) x + Wm b,
//   inverse: x = (diag(1/s) Wm^-1) v - b / s,
// and the per-pixel log|det| is log|det Wm| + sum log|s|.  Wm = P^T L U by
// LU factorisation with partial pivoting (the largest magnitude in the
// column, the lowest row on ties); column j of Wm^-1 solves L U x = P e_j.
// Output, floats: Mi (C x C) | ci (C) | Mf (C x C) | cf (C), then one double:
// the per-pixel log|det| (-inf for a singular Wm).
// ---------------------------------------------------------------------------
constexpr int kLinThreads = 256;
constexpr int kLinMaxC = 64;

__device__ void lin_prepare(const float *Wm, const float *s, const float *b, int C, float *out,
                            double *ldout, double ld_extra) {
    __shared__ double A[kLinMaxC * kLinMaxC];
    __shared__ int perm[kLinMaxC];
    __shared__ int prow;
    __shared__ int singular;
    const int tid = threadIdx.x;
    for (int e = tid; e < C * C; e += kLinThreads)
        A[e] = (double)Wm[e];
    for (int r = tid; r < C; r += kLinThreads)
        perm[r] = r;
    if (tid == 0)
        singular = 0;
    __syncthreads();
    for (int c = 0; c < C; ++c) {
        if (tid < 64) {
            double best = -1.0;
            int br = C;
            for (int r = c + tid; r < C; r += 64) {
                const double v = fabs(A[r * C + c]);
                if (v > best) {
                    best = v;
                    br = r;
                }
            }
            for (int off = 32; off > 0; off >>= 1) {
                const double ov = __shfl_xor(best, off);
                const int orr = __shfl_xor(br, off);
                if (ov > best || (ov == best && orr < br)) {
                    best = ov;
                    br = orr;
                }
            }
            if (tid == 0) {
                prow = br;
                if (!(best > 0.0))
                    singular = 1;
            }
        }
        __syncthreads();
        const int pr = prow;
        if (pr != c) {
            for (int j = tid; j < C; j += kLinThreads) {
                const double t = A[c * C + j];
                A[c * C + j] = A[pr * C + j];
                A[pr * C + j] = t;
            }
            if (tid == 0) {
                const int t = perm[c];
                perm[c] = perm[pr];
                perm[pr] = t;
            }
        }
        __syncthreads();
        const double d = A[c * C + c];
        const int n = (C - 1 - c) * (C - 1 - c);
        for (int e = tid; e < n && d != 0.0; e += kLinThreads) {
            const int r = c + 1 + e / (C - 1 - c), j = c + 1 + e % (C - 1 - c);
            A[r * C + j] -= A[r * C + c] / d * A[c * C + j];
        }
        __syncthreads();
        for (int r = c + 1 + tid; r < C && d != 0.0; r += kLinThreads)
            A[r * C + c] /= d;
        __syncthreads();
    }
    // column j of Wm^-1 (thread j); the inverse map is diag(1/s) Wm^-1
    for (int j = tid; j < C && !singular; j += kLinThreads) {
        double v[kLinMaxC];
        for (int r = 0; r < C; ++r) {
            double acc = perm[r] == j ? 1.0 : 0.0;
            for (int m = 0; m < r; ++m)
                acc -= A[r * C + m] * v[m];
            v[r] = acc;
        }
        for (int r = C - 1; r >= 0; --r) {
            double acc = v[r];
            for (int m = r + 1; m < C; ++m)
                acc -= A[r * C + m] * v[m];
            v[r] = acc / A[r * C + r];
        }
        for (int r = 0; r < C; ++r)
            out[r * C + j] = (float)(v[r] / (s ? (double)s[r] : 1.0));
    }
    // forward map Wm diag(s), Wm b; inverse offset -b/s
    for (int e = tid; e < C * C; e += kLinThreads) {
        const int r = e / C, j = e - r * C;
        out[C * C + C + e] = (float)((double)Wm[e] * (s ? (double)s[j] : 1.0));
    }
    for (int r = tid; r < C; r += kLinThreads) {
        out[C * C + r] = b ? (float)(-(double)b[r] / (double)s[r]) : 0.0f;
        double acc = 0.0;
        for (int j = 0; j < C && b; ++j)
            acc += (double)Wm[r * C + j] * (double)b[j];
        out[2 * C * C + C + r] = (float)acc;
    }
    if (tid == 0) {
        double ld = ld_extra;
        for (int c = 0; c < C; ++c)
            ld += log(fabs(A[c * C + c])) + (s ? log(fabs((double)s[c])) : 0.0);
        *ldout = singular ? -INFINITY : ld;
    }
}

// One Step's weights per workgroup (the j-th at params + j pstride, prepared
// into prep + j qstride bytes).  With Kq4 (the Step's channel-split unit,
// quarters of q channels, kernel k) the per-pixel constant also holds the
// unit's log|det| per pixel, sum over quarters g and channels of
// log|Kq4[g][c][c][self tap of corner g]|.  Wm only (null s, b, Kq4): the
// plain 1x1 convolution.
__global__ __launch_bounds__(kLinThreads) void lin_prep_kernel(const float *params, long long pstride,
                                                               int off_wm, int off_s, int off_b,
                                                               int C, int q, int k, char *prep,
                                                               long long qstride, int off_out,
                                                               int off_ld, int with_actnorm) {
    const float *p = params + (long long)blockIdx.x * pstride;
    char *o = prep + (long long)blockIdx.x * qstride;
    double unit = 0.0;
    if (with_actnorm && threadIdx.x == 0) {
        for (int g = 0; g < 4; ++g) {
            const int sh = g < 2 ? k - 1 : 0, sw = (g == 0 || g == 2) ? k - 1 : 0;
            for (int c = 0; c < q; ++c)
                unit += log(fabs((double)p[(((long long)g * q + c) * q + c) * k * k + sh * k + sw]));
        }
    }
    lin_prepare(p + off_wm, with_actnorm ? p + off_s : nullptr, with_actnorm ? p + off_b : nullptr,
                C, reinterpret_cast<float *>(o + off_out), reinterpret_cast<double *>(o + off_ld),
                unit);
}

// ---------------------------------------------------------------------------
// Elementwise parts, one workgroup per image (fixed-order log|det| sums).
// Coupling (mode 0 forward, 1 inverse) on the second half v[b][Ch + c] of
// a level tensor, from h = NN(first half) with t = h[b][c], r = h[b][Ch + c]:
//   forward yb = (xb + t) s, logdet[b] += sum log s + HW * ldc (ldc: the
//   Step's per-pixel constant, or null); inverse xb = yb / s - t;
//   s = sigmoid(r + 2).
// Split prior (mode 2 sampling, 3 forward), with (mean, logsd) = (h[b][c],
// h[b][Ch + c]): sampling v[b][Ch + c] = mean + exp(logsd) z[b][c];
// forward z[b][c] = (v[b][Ch + c] - mean) exp(-logsd), logdet[b] -= sum logsd.
// ---------------------------------------------------------------------------
struct EltArgs {
    float *v;            // level tensor (second half of its channels)
    const float *vin;    // coupling inverse out of place: input level tensor, or null
    long long vins;      // its image stride
    const float *h;      // network output (B, 2 Ch, HW), packed
    float *z;            // latent (B, Ch, HW), packed (prior only)
    double *logdet;      // (B) or null
    const double *ldc;   // per-pixel constant log|det| of the Step, or null
    int mode, Ch, HW;
    long long vs;        // image stride of v
};

constexpr int kEltThreads = 256;

__global__ __launch_bounds__(kEltThreads) void elt_kernel(EltArgs a) {
    __shared__ double red[kEltThreads];
    const int b = blockIdx.x, tid = threadIdx.x;
    const int n = a.Ch * a.HW;
    float *vb = a.v + (long long)b * a.vs + n;
    const float *hb = a.h + (long long)b * 2 * n;
    float *zb = a.z ? a.z + (long long)b * n : nullptr;
    double acc = 0.0;
    for (int e = tid; e < n; e += kEltThreads) {
        const float t = hb[e], r = hb[n + e];
        if (a.mode == 0) {
            const float sg = 1.0f / (1.0f + expf(-(r + 2.0f)));
            vb[e] = (vb[e] + t) * sg;
            acc += (double)logf(sg);
        } else if (a.mode == 1) {
            const float sg = 1.0f / (1.0f + expf(-(r + 2.0f)));
            if (a.vin) {   // out of place: the first half is copied
                const float *ib = a.vin + (long long)b * a.vins;
                vb[e - n] = ib[e];
                vb[e] = ib[n + e] / sg - t;
            } else {
                vb[e] = vb[e] / sg - t;
            }
        } else if (a.mode == 2) {
            vb[e] = t + expf(r) * zb[e];
        } else {
            zb[e] = (vb[e] - t) * expf(-r);
            acc -= (double)r;
        }
    }
    if (!a.logdet)
        return;
    red[tid] = acc;
    __syncthreads();
    for (int s = kEltThreads / 2; s > 0; s >>= 1) {
        if (tid < s)
            red[tid] += red[tid + s];
        __syncthreads();
    }
    if (tid == 0)
        a.logdet[b] += red[0] + (a.ldc ? (double)a.HW * a.ldc[0] : 0.0);
}

// Squeeze (C, H, W) -> (4C, H/2, W/2), channel 4c + 2dy + dx <- (c, 2i+dy,
// 2j+dx) (dir 0), or its inverse (dir 1); image strides on both sides.
__global__ __launch_bounds__(256) void squeeze_kernel(const float *in, float *out, int B, int C,
                                                      int H, int W, long long is, long long os,
                                                      int dir) {
    const long long n = (long long)B * C * H * W;
    const int H2 = H / 2, W2 = W / 2, img = C * H * W;
    for (long long e = blockIdx.x * 256ll + threadIdx.x; e < n; e += (long long)gridDim.x * 256) {
        const int b = (int)(e / img), r = (int)(e - (long long)b * img);
        const int c = r / (H * W), p = r - c * H * W, i = p / W, j = p - i * W;
        const int sq = ((4 * c + 2 * (i & 1) + (j & 1)) * H2 + (i >> 1)) * W2 + (j >> 1);
        if (dir == 0)
            out[b * os + sq] = in[b * is + r];
        else
            out[b * os + r] = in[b * is + sq];
    }
}

}  // namespace

// ===========================================================================
// Host side
// ===========================================================================
namespace {

constexpr int kFlowMaxC = 64;      // channels of a Step (the 1x1 preparation's limit)
constexpr int kFlowMaxLevels = 6;

__global__ __launch_bounds__(256) void fill_kernel(double *p, int n, double v) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < n)
        p[i] = v;
}

__global__ __launch_bounds__(64) void scale_kernel(const double *src, double *dst, double f) {
    if (threadIdx.x == 0)
        dst[0] = f * src[0];
}

__global__ __launch_bounds__(256) void copy_kernel(const float *in, float *out, long long n) {
    for (long long e = blockIdx.x * 256ll + threadIdx.x; e < n; e += (long long)gridDim.x * 256)
        out[e] = in[e];
}

inline size_t up256(size_t n) { return (n + 255) & ~(size_t)255; }
inline bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}
int launched() { return hipGetLastError() == hipSuccess ? FINC_OK : FINC_EHIP; }

// The flow's convolutions: 3 x 3 "same" (coupling and prior networks) and
// 1 x 1 (the coupling's middle convolution, the 1x1 / actnorm map).
int launch_conv(const float *x, long long xs, float *y, long long ys, const float *Wt,
                const float *bias, const float *ls, int relu, int B, int Ci, int Co, int H, int W,
                int R, hipStream_t st, float *partial = nullptr) {
    if (R == 1)
        return launch_conv_r<1>(x, xs, y, ys, Wt, bias, ls, relu, B, Ci, Co, H, W, -1, -1, st,
                                partial);
    return launch_conv_r<3>(x, xs, y, ys, Wt, bias, ls, relu, B, Ci, Co, H, W, -1, -1, st,
                            partial);
}

// A 3 x 3 "same" convolution with few output channels (9 C >= 64) and a
// long K: the nine taps' 1 x 1 products as one GEMM with 9 C rows and no
// gather (Z = W_t x for every tap t, in Z (B, 9 C, H, W)), then their
// shifted sum with the bias and exp(3 ls) scale.  Z: 9 B C H W floats.
int launch_conv_taps(const float *x, long long xs, float *y, long long ys, const float *Wt,
                     const float *bias, const float *ls, int B, int Ci, int C, int H, int W,
                     hipStream_t st, float *Z) {
    if (B == 0)
        return FINC_OK;
    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.y = Z;
    a.Wt = Wt;
    a.B = B;
    a.Ci = Ci;
    a.Co = 9 * C;
    a.H = H;
    a.W = W;
    a.K = Ci;
    a.xs = xs;
    a.ys = (long long)9 * C * H * W;
    a.d_HW = make_div(H * W);
    a.d_W = make_div(W);
    a.trows = C;
    const long long Q = (long long)B * H * W;
    const dim3 grid(cdiv(Q, 64), cdiv(9 * C, 64));
    launch_wide<1>(a, grid, st);
    int rc = launched();
    if (rc != FINC_OK)
        return rc;
    const long long n = (long long)B * C * H * W;
    hipLaunchKernelGGL(shift_add_kernel, dim3((unsigned)(n / 256 + 1 < 8192 ? n / 256 + 1 : 8192)),
                       dim3(256), 0, st, Z, y, ys, bias, ls, B, C, H, W, make_div(H * W),
                       make_div(W), make_div(C));
    return launched();
}

// Offsets (floats) of one Step's parameters.
struct StepLayout {
    int C, q, Ch, k, hid;
    long long kq4, an_s, an_b, wm, w1, b1, w2, b2, w3, b3, ls3, total;
};
StepLayout step_layout(int C, int k, int hid) {
    StepLayout L;
    L.C = C;
    L.q = C / 4;
    L.Ch = C / 2;
    L.k = k;
    L.hid = hid;
    L.kq4 = 0;
    L.an_s = 4ll * L.q * L.q * k * k;
    L.an_b = L.an_s + C;
    L.wm = L.an_b + C;
    L.w1 = L.wm + (long long)C * C;
    L.b1 = L.w1 + (long long)hid * L.Ch * 9;
    L.w2 = L.b1 + hid;
    L.b2 = L.w2 + (long long)hid * hid;
    L.w3 = L.b2 + hid;
    L.b3 = L.w3 + (long long)C * hid * 9;
    L.ls3 = L.b3 + C;
    L.total = L.ls3 + C;
    return L;
}
long long prior_count(int C) { return (long long)C * (C / 2) * 9 + 2ll * C; }

// Prepared bytes of one Step: the channel-split unit's inverse weights, then
// the 1x1 / actnorm maps (floats) and the per-pixel log|det| (a double).
struct StepPrep {
    size_t unit, lin, ld, total;
};
StepPrep step_prep(int C, int k) {
    StepPrep p;
    p.unit = 0;
    p.lin = finc_workspace_bytes(C / 4, k, 4);
    p.ld = (p.lin + (2ull * C * C + 2ull * C) * sizeof(float) + 7) & ~(size_t)7;
    p.total = up256(p.ld + sizeof(double));
    return p;
}

bool valid_step(int C, int k, int hid) {
    return C >= 4 && C % 4 == 0 && C <= kFlowMaxC && k >= 1 && k <= FINC_MAX_K && hid >= 1 &&
           hid <= 4096;
}

int launch_elt(int mode, float *v, long long vs, const float *vin, long long vins, const float *h,
               float *z, double *logdet, const double *ldc, int B, int Ch, int HW,
               hipStream_t st) {
    if (B == 0)
        return FINC_OK;
    EltArgs a;
    memset(&a, 0, sizeof(a));
    a.v = v;
    a.vs = vs;
    a.vin = vin;
    a.vins = vins;
    a.h = h;
    a.z = z;
    a.logdet = logdet;
    a.ldc = ldc;
    a.mode = mode;
    a.Ch = Ch;
    a.HW = HW;
    hipLaunchKernelGGL(elt_kernel, dim3(B), dim3(kEltThreads), 0, st, a);
    return launched();
}

int launch_squeeze(const float *in, float *out, int B, int C, int H, int W, long long is,
                   long long os, int dir, hipStream_t st) {
    const long long n = (long long)B * C * H * W;
    if (n == 0)
        return FINC_OK;
    const int blocks = (int)(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096);
    hipLaunchKernelGGL(squeeze_kernel, dim3(blocks), dim3(256), 0, st, in, out, B, C, H, W, is, os,
                       dir);
    return launched();
}

// Scratch of a Step at (B, C, H, W): u (B C HW), hh (B C HW), t1, t2
// (B hid HW each), the partial sums of the coupling's last convolution
// (kMaxParts B C HW) or its nine taps' products (9 B C HW), floats, each
// 256-byte aligned.
struct StepScratch {
    float *u, *hh, *t1, *t2, *part;
};
size_t step_scratch_bytes(int B, int C, int H, int W, int hid) {
    const size_t hw = (size_t)H * W;
    const size_t parts = kMaxParts > 9 ? kMaxParts : 9;   // (K-split sums, or the taps' Z)
    return 2 * up256((size_t)B * C * hw * 4) + 2 * up256((size_t)B * hid * hw * 4) +
           up256(parts * B * C * hw * 4);
}
StepScratch carve(void *ws, int B, int C, int H, int W, int hid) {
    const size_t hw = (size_t)H * W;
    char *p = (char *)ws;
    StepScratch s;
    s.u = (float *)p;
    p += up256((size_t)B * C * hw * 4);
    s.hh = (float *)p;
    p += up256((size_t)B * C * hw * 4);
    s.t1 = (float *)p;
    p += up256((size_t)B * hid * hw * 4);
    s.t2 = (float *)p;
    p += up256((size_t)B * hid * hw * 4);
    s.part = (float *)p;
    return s;
}

// The coupling network on the first half of v (image stride vs) -> hh.
int coupling_net(const float *v, long long vs, const float *sp, const StepLayout &L,
                 const StepScratch &s, int B, int H, int W, hipStream_t st) {
    const long long hw = (long long)H * W;
    int rc = launch_conv(v, vs, s.t1, (long long)L.hid * hw, sp + L.w1, sp + L.b1, nullptr, 1, B,
                         L.Ch, L.hid, H, W, 3, st);
    if (rc == FINC_OK)
        rc = launch_conv(s.t1, (long long)L.hid * hw, s.t2, (long long)L.hid * hw, sp + L.w2,
                         sp + L.b2, nullptr, 1, B, L.hid, L.hid, H, W, 1, st);
    if (rc != FINC_OK)
        return rc;
    if (9 * L.C >= 64 && L.hid >= 64)
        return launch_conv_taps(s.t2, (long long)L.hid * hw, s.hh, (long long)L.C * hw,
                                sp + L.w3, sp + L.b3, sp + L.ls3, B, L.hid, L.C, H, W, st,
                                s.part);
    return launch_conv(s.t2, (long long)L.hid * hw, s.hh, (long long)L.C * hw, sp + L.w3,
                       sp + L.b3, sp + L.ls3, 0, B, L.hid, L.C, H, W, 3, st, s.part);
}

// Step forward in place on h (B, C, H, W; image stride C H W): unit, then
// the 1x1 map with its actnorm, then the coupling; logdet[b] += the Step's
// log|det| (logdet may be null).
int step_forward_dev(float *h, const float *x, double *logdet, const float *sp, const char *pp,
                     int B, int C, int H, int W, int k, int hid, const StepScratch &s,
                     hipStream_t st) {
    const StepLayout L = step_layout(C, k, hid);
    const StepPrep P = step_prep(C, k);
    const long long img = (long long)C * H * W;
    int rc = finc_split_forward(x, s.u, sp + L.kq4, nullptr, nullptr, B, C, H, W, k, st);
    const float *lin = (const float *)(pp + P.lin);
    if (rc == FINC_OK)
        rc = launch_conv(s.u, img, h, img, lin + C * C + C, lin + 2 * C * C + C, nullptr, 0, B, C,
                         C, H, W, 1, st);
    if (rc == FINC_OK)
        rc = coupling_net(h, img, sp, L, s, B, H, W, st);
    if (rc == FINC_OK)
        rc = launch_elt(0, h, img, nullptr, 0, s.hh, nullptr, logdet,
                        logdet ? (const double *)(pp + P.ld) : nullptr, B, L.Ch, H * W, st);
    return rc;
}

// Step inverse: y (read) -> x: coupling^-1 (out of place from y into x when
// they differ), the inverse 1x1 / actnorm map into u, the unit's wavefront
// inverse back into x.
int step_inverse_dev(const float *y, float *x, const float *sp, const char *pp, int B, int C,
                     int H, int W, int k, int hid, const StepScratch &s, hipStream_t st) {
    const StepLayout L = step_layout(C, k, hid);
    const StepPrep P = step_prep(C, k);
    const long long img = (long long)C * H * W;
    int rc = coupling_net(y, img, sp, L, s, B, H, W, st);
    if (rc == FINC_OK)
        rc = launch_elt(1, x, img, y == x ? nullptr : y, img, s.hh, nullptr, nullptr, nullptr, B,
                        L.Ch, H * W, st);
    const float *lin = (const float *)(pp + P.lin);
    if (rc == FINC_OK)
        rc = launch_conv(x, img, s.u, img, lin, lin + C * C, nullptr, 0, B, C, C, H, W, 1, st);
    if (rc == FINC_OK)
        rc = finc_split_inverse_prepared(s.u, x, pp + P.unit, B, C, H, W, k, st);
    return rc;
}

int step_prepare_dev(const float *sp, long long pstride, int n, int C, int k, int hid, char *pp,
                     hipStream_t st) {
    const StepLayout L = step_layout(C, k, hid);
    const StepPrep P = step_prep(C, k);
    static const int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
    for (int j = 0; j < n; ++j) {
        const int rc = finc_prepare(sp + j * pstride + L.kq4, 4, corners, L.q, k,
                                    pp + j * P.total + P.unit, st);
        if (rc != FINC_OK)
            return rc;
    }
    if (n == 0)
        return FINC_OK;
    hipLaunchKernelGGL(lin_prep_kernel, dim3(n), dim3(kLinThreads), 0, st, sp, pstride, (int)L.wm,
                       (int)L.an_s, (int)L.an_b, C, L.q, k, pp, (long long)P.total, (int)P.lin,
                       (int)P.ld, 1);
    return launched();
}

bool valid_flow(int B, int L, int K, int C0, int H0, int W0, int k, int hid) {
    if (B < 0 || L < 1 || L > kFlowMaxLevels || K < 0 || C0 < 1 || H0 < 1 || W0 < 1)
        return false;
    if ((H0 % (2 << (L - 1))) || (W0 % (2 << (L - 1))))
        return false;
    if ((long long)B * C0 * H0 * W0 >= (1ll << 31))
        return false;
    for (int l = 0; l < L; ++l)
        if (!valid_step((4 * C0) << l, k, hid))
            return false;
    return true;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

size_t finc_conv1x1_workspace_bytes(int C) {
    if (C < 1 || C > kFlowMaxC)
        return 0;
    return up256((2ull * C * C + 2ull * C) * sizeof(float)) + 256;
}

static int conv1x1_run(const float *in, float *out, const float *Wm, double *logdet, int B, int C,
                       int H, int W, void *workspace, int inverse, hipStream_t st) {
    if (B < 0 || C < 1 || C > kFlowMaxC || H < 1 || W < 1 || !in || !out || !Wm || !workspace ||
        ((uintptr_t)workspace & 255u) || (long long)B * C * H * W >= (1ll << 31))
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float), wsb = finc_conv1x1_workspace_bytes(C);
    if (overlap(in, bytes, out, bytes) || overlap(workspace, wsb, in, bytes) ||
        overlap(workspace, wsb, out, bytes) || overlap(workspace, wsb, Wm, (size_t)C * C * 4))
        return FINC_EINVAL;
    char *ws = (char *)workspace;
    const int off_ld = (int)up256((2ull * C * C + 2ull * C) * sizeof(float));
    hipLaunchKernelGGL(lin_prep_kernel, dim3(1), dim3(kLinThreads), 0, st, Wm, 0ll, 0, 0, 0, C, 1,
                       1, ws, 0ll, 0, off_ld, 0);
    int rc = launched();
    const float *lin = (const float *)ws;
    const long long img = (long long)C * H * W;
    if (rc == FINC_OK)
        rc = inverse ? launch_conv(in, img, out, img, lin, lin + C * C, nullptr, 0, B, C, C, H, W,
                                   1, st)
                     : launch_conv(in, img, out, img, lin + C * C + C, lin + 2 * C * C + C,
                                   nullptr, 0, B, C, C, H, W, 1, st);
    if (rc == FINC_OK && logdet) {   // H W log|det Wm| from the per-pixel value
        hipLaunchKernelGGL(scale_kernel, dim3(1), dim3(64), 0, st, (const double *)(ws + off_ld),
                           logdet, (double)H * W);
        rc = launched();
    }
    return rc;
}

int finc_conv1x1_forward(const float *x, float *y, const float *Wm, double *logdet, int B, int C,
                         int H, int W, void *workspace, hipStream_t stream) {
    return conv1x1_run(x, y, Wm, logdet, B, C, H, W, workspace, 0, stream);
}

int finc_conv1x1_inverse(const float *y, float *x, const float *Wm, int B, int C, int H, int W,
                         void *workspace, hipStream_t stream) {
    return conv1x1_run(y, x, Wm, nullptr, B, C, H, W, workspace, 1, stream);
}

size_t finc_step_param_count(int C, int k, int hid) {
    return valid_step(C, k, hid) ? (size_t)step_layout(C, k, hid).total : 0;
}

size_t finc_step_prepared_bytes(int C, int k) {
    return valid_step(C, k, 1) ? step_prep(C, k).total : 0;
}

size_t finc_step_workspace_bytes(int B, int C, int H, int W, int hid) {
    if (B < 0 || H < 1 || W < 1 || !valid_step(C, 1, hid))
        return 0;
    return step_scratch_bytes(B, C, H, W, hid);
}

int finc_step_prepare(const float *sp, int C, int k, int hid, void *prepared, hipStream_t stream) {
    if (!valid_step(C, k, hid) || !sp || !prepared || ((uintptr_t)prepared & 255u))
        return FINC_EINVAL;
    return step_prepare_dev(sp, 0, 1, C, k, hid, (char *)prepared, stream);
}

static bool step_args_ok(const float *in, const float *out, const float *sp, const void *prepared,
                         int B, int C, int H, int W, int k, int hid, const void *ws) {
    if (!valid_step(C, k, hid) || B < 0 || H < 1 || W < 1 || !in || !out || !sp || !prepared ||
        !ws || ((uintptr_t)prepared & 255u) || ((uintptr_t)ws & 255u) ||
        (long long)B * C * H * W >= (1ll << 31))
        return false;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t wsb = step_scratch_bytes(B, C, H, W, hid);
    const size_t pb = step_prep(C, k).total;
    const size_t sb = (size_t)step_layout(C, k, hid).total * sizeof(float);
    return !overlap(in, bytes, out, bytes) && !overlap(ws, wsb, in, bytes) &&
           !overlap(ws, wsb, out, bytes) && !overlap(ws, wsb, sp, sb) &&
           !overlap(ws, wsb, prepared, pb) && !overlap(out, bytes, sp, sb) &&
           !overlap(out, bytes, prepared, pb);
}

int finc_step_forward(const float *x, float *y, double *logdet, const float *sp,
                      const void *prepared, int B, int C, int H, int W, int k, int hid,
                      void *workspace, hipStream_t stream) {
    if (!step_args_ok(x, y, sp, prepared, B, C, H, W, k, hid, workspace))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    const StepScratch s = carve(workspace, B, C, H, W, hid);
    return step_forward_dev(y, x, logdet, sp, (const char *)prepared, B, C, H, W, k, hid, s, stream);
}

int finc_step_inverse(const float *y, float *x, const float *sp, const void *prepared, int B,
                      int C, int H, int W, int k, int hid, void *workspace, hipStream_t stream) {
    if (!step_args_ok(y, x, sp, prepared, B, C, H, W, k, hid, workspace))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    const StepScratch s = carve(workspace, B, C, H, W, hid);
    return step_inverse_dev(y, x, sp, (const char *)prepared, B, C, H, W, k, hid, s, stream);
}

size_t finc_flow_param_count(int L, int K, int C0, int k, int hid) {
    if (!valid_flow(1, L, K, C0, 2 << (L - 1), 2 << (L - 1), k, hid))
        return 0;
    long long n = 0;
    for (int l = 0; l < L; ++l) {
        const int C = (4 * C0) << l;
        n += (long long)K * step_layout(C, k, hid).total + (l < L - 1 ? prior_count(C) : 0);
    }
    return (size_t)n;
}

size_t finc_flow_prepared_bytes(int L, int K, int C0, int k) {
    if (!valid_flow(1, L, K, C0, 2 << (L - 1), 2 << (L - 1), k, 1))
        return 0;
    size_t n = 0;
    for (int l = 0; l < L; ++l)
        n += (size_t)K * step_prep((4 * C0) << l, k).total;
    return n;
}

// Workspace of a flow call: the level tensor, a second one for the
// squeezes, and a Step's scratch at level 0 (the largest).
size_t finc_flow_workspace_bytes(int B, int L, int C0, int H0, int W0, int hid) {
    if (!valid_flow(B, L, 0, C0, H0, W0, 1, hid))
        return 0;
    const size_t img = (size_t)B * C0 * H0 * W0 * sizeof(float);
    return 2 * up256(img) + step_scratch_bytes(B, 4 * C0, H0 / 2, W0 / 2, hid);
}

int finc_flow_prepare(const float *params, int L, int K, int C0, int k, int hid, void *prepared,
                      hipStream_t stream) {
    if (!valid_flow(1, L, K, C0, 2 << (L - 1), 2 << (L - 1), k, hid) || !params || !prepared ||
        ((uintptr_t)prepared & 255u))
        return FINC_EINVAL;
    const float *p = params;
    char *q = (char *)prepared;
    for (int l = 0; l < L; ++l) {
        const int C = (4 * C0) << l;
        const StepLayout S = step_layout(C, k, hid);
        const int rc = step_prepare_dev(p, S.total, K, C, k, hid, q, stream);
        if (rc != FINC_OK)
            return rc;
        p += (long long)K * S.total + (l < L - 1 ? prior_count(C) : 0);
        q += (size_t)K * step_prep(C, k).total;
    }
    return FINC_OK;
}

static bool flow_buffers_ok(const float *const *z, const float *x, const float *params,
                            const void *prepared, double *logdet, int B, int L, int K, int C0,
                            int H0, int W0, int k, int hid, const void *ws) {
    if (!valid_flow(B, L, K, C0, H0, W0, k, hid) || !z || !x || !params || !prepared || !ws ||
        ((uintptr_t)prepared & 255u) || ((uintptr_t)ws & 255u))
        return false;
    const size_t xb = (size_t)B * C0 * H0 * W0 * sizeof(float);
    const size_t wsb = finc_flow_workspace_bytes(B, L, C0, H0, W0, hid);
    const size_t pb = finc_flow_prepared_bytes(L, K, C0, k);
    const size_t parb = finc_flow_param_count(L, K, C0, k, hid) * sizeof(float);
    if (overlap(ws, wsb, x, xb) || overlap(ws, wsb, params, parb) || overlap(ws, wsb, prepared, pb))
        return false;
    if (logdet && (overlap(logdet, (size_t)B * 8, x, xb) || overlap(logdet, (size_t)B * 8, ws, wsb)))
        return false;
    for (int l = 0; l < L; ++l) {
        if (!z[l])
            return false;
        const int C = (4 * C0) << l, H = H0 >> (l + 1), W = W0 >> (l + 1);
        const size_t zb = (size_t)B * (l == L - 1 ? C : C / 2) * H * W * sizeof(float);
        if (overlap(z[l], zb, ws, wsb) || overlap(z[l], zb, x, xb) ||
            overlap(z[l], zb, params, parb) || overlap(z[l], zb, prepared, pb))
            return false;
    }
    return true;
}

int finc_flow_forward(const float *x, float *const *z, double *logdet, const float *params,
                      const void *prepared, int B, int L, int K, int C0, int H0, int W0, int k,
                      int hid, void *workspace, hipStream_t st) {
    if (!flow_buffers_ok((const float *const *)z, x, params, prepared, logdet, B, L, K, C0, H0, W0,
                         k, hid, workspace) ||
        !logdet)
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    const size_t img = up256((size_t)B * C0 * H0 * W0 * sizeof(float));
    float *hA = (float *)workspace, *hB = (float *)((char *)workspace + img);
    void *scratch = (char *)workspace + 2 * img;
    hipLaunchKernelGGL(fill_kernel, dim3(cdiv(B, 256)), dim3(256), 0, st, logdet, B, 0.0);
    int rc = launched();
    const float *p = params;
    const char *q = (const char *)prepared;
    const float *in = x;
    long long in_stride = (long long)C0 * H0 * W0;
    int Cin = C0, H = H0, W = W0;
    for (int l = 0; l < L && rc == FINC_OK; ++l) {
        const int C = 4 * Cin;
        H /= 2;
        W /= 2;
        const long long lev = (long long)C * H * W;
        rc = launch_squeeze(in, hA, B, Cin, 2 * H, 2 * W, in_stride, lev, 0, st);
        const StepLayout S = step_layout(C, k, hid);
        const StepScratch s = carve(scratch, B, C, H, W, hid);
        for (int j = 0; j < K && rc == FINC_OK; ++j) {
            rc = step_forward_dev(hA, hA, logdet, p, q, B, C, H, W, k, hid, s, st);
            p += S.total;
            q += step_prep(C, k).total;
        }
        if (rc != FINC_OK)
            break;
        if (l == L - 1) {
            const long long n = (long long)B * lev;
            hipLaunchKernelGGL(copy_kernel, dim3((unsigned)(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096)),
                               dim3(256), 0, st, hA, z[l], n);
            rc = launched();
            break;
        }
        // split prior on the first half, latent from the second
        rc = launch_conv(hA, lev, s.hh, lev, p, p + (long long)C * (C / 2) * 9,
                         p + (long long)C * (C / 2) * 9 + C, 0, B, C / 2, C, H, W, 3, st);
        if (rc == FINC_OK)
            rc = launch_elt(3, hA, lev, nullptr, 0, s.hh, z[l], logdet, nullptr, B, C / 2, H * W,
                            st);
        p += prior_count(C);
        // the next level squeezes the first half
        float *t = hA;
        hA = hB;
        hB = t;
        in = hB;
        in_stride = lev;
        Cin = C / 2;
    }
    return rc;
}

int finc_flow_sample(const float *const *z, float *x, const float *params, const void *prepared,
                     int B, int L, int K, int C0, int H0, int W0, int k, int hid, void *workspace,
                     hipStream_t st) {
    if (!flow_buffers_ok(z, x, params, prepared, nullptr, B, L, K, C0, H0, W0, k, hid, workspace))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    // where each level's Steps and prior start
    const float *lp[kFlowMaxLevels];
    const char *lq[kFlowMaxLevels];
    {
        const float *p = params;
        const char *q = (const char *)prepared;
        for (int l = 0; l < L; ++l) {
            const int C = (4 * C0) << l;
            lp[l] = p;
            lq[l] = q;
            p += (long long)K * step_layout(C, k, hid).total + (l < L - 1 ? prior_count(C) : 0);
            q += (size_t)K * step_prep(C, k).total;
        }
    }
    const size_t img = up256((size_t)B * C0 * H0 * W0 * sizeof(float));
    float *hA = (float *)workspace, *hB = (float *)((char *)workspace + img);
    void *scratch = (char *)workspace + 2 * img;
    int rc = FINC_OK;
    for (int l = L - 1; l >= 0 && rc == FINC_OK; --l) {
        const int C = (4 * C0) << l, H = H0 >> (l + 1), W = W0 >> (l + 1);
        const long long lev = (long long)C * H * W;
        const StepLayout S = step_layout(C, k, hid);
        const StepScratch s = carve(scratch, B, C, H, W, hid);
        const float *src = hA;
        if (l == L - 1) {
            src = z[l];   // the top latent, read by the first Step
        } else {
            // hA holds h1 in its first half: h2 = mean + exp(logsd) z_l
            const float *pp = lp[l] + (long long)K * S.total;
            rc = launch_conv(hA, lev, s.hh, lev, pp, pp + (long long)C * (C / 2) * 9,
                             pp + (long long)C * (C / 2) * 9 + C, 0, B, C / 2, C, H, W, 3, st);
            if (rc == FINC_OK)
                rc = launch_elt(2, hA, lev, nullptr, 0, s.hh, (float *)z[l], nullptr, nullptr, B,
                                C / 2, H * W, st);
        }
        for (int j = K - 1; j >= 0 && rc == FINC_OK; --j) {
            rc = step_inverse_dev(src, hA, lp[l] + (long long)j * S.total,
                                  lq[l] + (size_t)j * step_prep(C, k).total, B, C, H, W, k, hid, s,
                                  st);
            src = hA;
        }
        if (rc != FINC_OK)
            break;
        if (K == 0 && l == L - 1) {   // no Steps: the top latent itself
            const long long n = (long long)B * lev;
            hipLaunchKernelGGL(copy_kernel, dim3((unsigned)(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096)),
                               dim3(256), 0, st, z[l], hA, n);
            rc = launched();
        }
        // unsqueeze into the first half of the level below (or into x)
        if (rc == FINC_OK) {
            // (the level below has C / 2 channels at 2H x 2W: image stride 2 C H W)
            float *dst = l == 0 ? x : hB;
            rc = launch_squeeze(hA, dst, B, C / 4, 2 * H, 2 * W, lev,
                                l == 0 ? (long long)C0 * H0 * W0 : 2 * lev, 1, st);
            float *t = hA;
            hA = hB;
            hB = t;
        }
    }
    return rc;
}

}  // extern "C"
