// backward.hip -- backward of the masked k x k convolution layer on gfx950,
// for training on the negative log-likelihood (Sec. 3 NLL equation; the
// appendix's training details reset the masked weights' gradients to zero
// after every step), behind finc_backward of include/finc.h.
//
// y = layer(x) sends x[ci, i + a - oh, j + b - ow] to y[co, i, j] with weight
// K[co][ci][a][b] (zero at the masked self-tap entries ci > co), so for an
// output gradient dy:
//   dx[ci, s, t] = sum_{co, a, b} K[co][ci][a][b] dy[co, s - a + oh, t - b + ow]
//     -- a convolution of dy with the kernel transposed over channels and
//     flipped in space, run by the implicit-GEMM convolution of conv_gemm.h
//     reading K that way (tap a' = k-1-a reads row s + a' - (k-1-oh));
//   dK[co][ci][a][b] = sum over images and pixels of dy[co, i, j] times the
//     input the tap read (zero outside the image) -- a GEMM with
//     M = C_out, N = C_in k^2 and a reduction over the B H W positions, in
//     parts of the positions.
// The two are independent: one launch (backward_kernel) runs the tiles of
// both, and dk_reduce_kernel then adds dK's parts in order, sets the masked
// entries to 0 and adds the log|det| term gld H W / K[c][c][self] on the
// self diagonal.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "conv_gemm.h"
#include "finc.h"

namespace {

inline size_t up256b(size_t n) { return (n + 255) & ~(size_t)255; }
inline size_t imax_sz(size_t a, size_t b) { return a > b ? a : b; }
inline bool overlapb(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

// dK as a GEMM over positions.  Block: 16 c_out x 64 columns (column =
// ci k^2 + a k + b), 4 waves; every chunk of 64 positions (flattened over the
// batch) is staged in LDS -- dy[co][pos] and the gathered inputs
// x_tap[col][pos], both position-contiguous -- and wave w takes positions
// 16 w .. 16 w + 15 of it (lane group kq: 4 consecutive positions, one
// float4 per operand for four MFMAs).  The four waves' sums are added in
// order through LDS; part z covers chunks [z cpp, (z+1) cpp)
// and writes its sums to partial + z C (C k^2).
struct DkArgs {
    const float *x, *dy;
    float *partial;
    long long img;   // floats from one image to the next (x and dy)
    int B, C, H, W, k, oh, ow, N, cpp, nchunk;
    Div d_HW, d_W, d_kk, d_k;
};

constexpr int kDkLdsFloats = 80 * kSK;   // As (16 rows), Bs (64 rows); red reuses it

__device__ __forceinline__ void dk_tile(const DkArgs &a, int bx, int by, int bz, float *lds) {
    float *As = lds, *Bs = lds + 16 * kSK;
    float(*red)[16][65] = reinterpret_cast<float(*)[16][65]>(lds);
    const int tid = threadIdx.x, lane = tid & 63, kq = lane >> 4, li = lane & 15, wave = tid >> 6;
    const int col0 = bx * 64, co0 = by * 16;
    const int HW = a.H * a.W, P = a.B * HW, kk = a.k * a.k;
    const long long img = a.img;
    // staging roles: A: thread -> (co 16 x position quad 16); B: thread -> (col, 4 quads)
    const int aco = co0 + (tid >> 4), aq = tid & 15;
    const int bcol = col0 + (tid & 63), bq0 = tid >> 6;
    const bool colok = bcol < a.N;
    const int bci = colok ? divi(bcol, a.d_kk) : 0;
    const int bt = colok ? bcol - bci * kk : 0;
    const int ba = divi(bt, a.d_k), bb = bt - ba * a.k;
    float ra[4], rb[4][4];
    auto load_chunk = [&](int c) {
        const int p0 = c * 64;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int pos = p0 + 4 * aq + e;
            const bool ok = pos < P && aco < a.C;
            const int n = ok ? divi(pos, a.d_HW) : 0, p = ok ? pos - n * HW : 0;
            const float v = a.dy[ok ? n * img + (long long)aco * HW + p : 0];
            ra[e] = ok ? v : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int pos = p0 + 4 * (bq0 + 4 * u) + e;
                const bool pok = pos < P && colok;
                const int n = pok ? divi(pos, a.d_HW) : 0, p = pok ? pos - n * HW : 0;
                const int i = divi(p, a.d_W), j = p - i * a.W;
                const int ii = i + ba - a.oh, jj = j + bb - a.ow;
                const bool ok = pok && ii >= 0 && ii < a.H && jj >= 0 && jj < a.W;
                const float v = a.x[ok ? n * img + (long long)bci * HW + ii * a.W + jj : 0];
                rb[u][e] = ok ? v : 0.0f;
            }
        }
    };
    auto store_chunk = [&] {
        *reinterpret_cast<float4 *>(&As[(tid >> 4) * kSK + 4 * aq]) =
            make_float4(ra[0], ra[1], ra[2], ra[3]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
            *reinterpret_cast<float4 *>(&Bs[(tid & 63) * kSK + 4 * (bq0 + 4 * u)]) =
                make_float4(rb[u][0], rb[u][1], rb[u][2], rb[u][3]);
    };
    f32x4 acc[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
        acc[s] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const int c0 = bz * a.cpp, c1 = min(c0 + a.cpp, a.nchunk);
    if (c0 < c1) {
        load_chunk(c0);
        store_chunk();
    }
    __syncthreads();
    for (int c = c0; c < c1; ++c) {
        if (c + 1 < c1)
            load_chunk(c + 1);
        const float4 w4 = *reinterpret_cast<const float4 *>(&As[li * kSK + 16 * wave + 4 * kq]);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const float4 b4 =
                *reinterpret_cast<const float4 *>(&Bs[(16 * s + li) * kSK + 16 * wave + 4 * kq]);
            acc[s] = mfma4(w4.x, b4.x, acc[s]);
            acc[s] = mfma4(w4.y, b4.y, acc[s]);
            acc[s] = mfma4(w4.z, b4.z, acc[s]);
            acc[s] = mfma4(w4.w, b4.w, acc[s]);
        }
        if (c + 1 < c1) {
            __syncthreads();
            store_chunk();
            __syncthreads();
        }
    }
    // lane (kq, li) of wave w holds D[co 4 kq + rr][col 16 s + li]
    __syncthreads();   // every wave's last reads of As / Bs are done
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int rr = 0; rr < 4; ++rr)
            red[wave][4 * kq + rr][16 * s + li] = acc[s][rr];
    __syncthreads();
    float *pz = a.partial + (long long)bz * a.C * a.N;
    for (int e = tid; e < 16 * 64; e += 256) {
        const int r = e >> 6, cl = e & 63;
        const int co = co0 + r, col = col0 + cl;
        if (co < a.C && col < a.N)
            pz[(long long)co * a.N + col] =
                ((red[0][r][cl] + red[1][r][cl]) + red[2][r][cl]) + red[3][r][cl];
    }
}

// One launch for both gradients, which are independent of each other:
// blocks [0, ndx) are tiles of the input gradient's convolution (gx of them
// along the pixels), the others tiles of dK's GEMM (dgx along its columns,
// dgy along c_out, then the parts of the positions).
template <int R, int WCO, int NS>
__global__ __launch_bounds__(256) void backward_kernel(ConvArgs ca, int ndx, int gx, DkArgs da,
                                                       int dgx, int dgy) {
    constexpr int nc = conv_lds_floats<WCO, NS>();
    __shared__ __attribute__((aligned(16))) float lds[nc > kDkLdsFloats ? nc : kDkLdsFloats];
    int b = blockIdx.x;
    if (b < ndx) {
        conv_tile<R, WCO, NS>(ca, b % gx, b / gx, 0, lds);
        return;
    }
    b -= ndx;
    dk_tile(da, b % dgx, (b / dgx) % dgy, b / (dgx * dgy), lds);
}

// dK = the sum of the parts, in a fixed order: lane l of a group of 32
// threads adds parts l, l + 32, l + 64, ... in turn, then the 32 lane sums
// meet in a fixed butterfly; masked entries 0; gld H W / K[c][c][self] added
// on the self diagonal (in fp64).  8 outputs per block of 256 threads.
__global__ __launch_bounds__(256) void dk_reduce_kernel(const float *partial, int parts,
                                                        const float *K, float *dK, double gld,
                                                        int C, int k, int H, int W, int oh,
                                                        int ow) {
    const int N = C * k * k, n = C * N;
    const int e = blockIdx.x * 8 + (threadIdx.x >> 5), l = threadIdx.x & 31;
    const int ec = e < n ? e : n - 1;
    float v = 0.0f;
    for (int z = l; z < parts; z += 32)
        v += partial[(long long)z * n + ec];
#pragma unroll
    for (int off = 16; off > 0; off >>= 1)
        v += __shfl_xor(v, off, 32);
    if (l != 0 || e >= n)
        return;
    const int co = e / N, col = e - co * N, ci = col / (k * k), t = col - ci * k * k;
    const int a = t / k, b = t - a * k;
    const bool self = a == oh && b == ow;
    if (self && ci > co)
        v = 0.0f;   // masked: its gradient is reset to zero
    else if (self && ci == co)
        v = (float)((double)v + gld * (double)H * (double)W /
                                    (double)K[((co * C + co) * k + a) * k + b]);
    dK[e] = v;
}

// Parts of the position reduction: at least 2 chunks of 64 positions each,
// about 512 blocks over the chip (two per CU), and at most 16 M floats of
// partial sums.
int dk_parts(int B, int C, int H, int W, int k) {
    const long long nchunk = ((long long)B * H * W + 63) / 64;
    const long long tiles = (long long)((C * k * k + 63) / 64) * ((C + 15) / 16);
    long long parts = 512 / (tiles > 0 ? tiles : 1);
    if (parts > nchunk / 2)
        parts = nchunk / 2;
    const long long cap = (16ll << 20) / ((long long)C * C * k * k);
    if (parts > cap)
        parts = cap;
    return (int)(parts < 1 ? 1 : parts);
}

bool valid_bwd_shape(int B, int C, int H, int W, int k) {
    if (B < 0 || C < 1 || C > FINC_MAX_C || H < 1 || W < 1 || k < 1 || k > FINC_MAX_K)
        return false;
    return (long long)B * C * H * W < (1ll << 31);
}

template <int R, int WCO, int NS>
void launch_fused(const ConvArgs &ca, int ndx, int gx, const DkArgs &da, int dgx, int dgy, int ndk,
                  hipStream_t st) {
    hipLaunchKernelGGL((backward_kernel<R, WCO, NS>), dim3(ndx + ndk), dim3(256), 0, st, ca, ndx,
                       gx, da, dgx, dgy);
}

// The instance for kernel size R and the convolution's tile configuration:
// 64 c_out x 64 pixels at 64 channels, else 16 c_out x 32 pixels per wave
// (NS = 2) when that still gives 256 tiles, else 16 x 16 (NS = 1).
template <int R>
void launch_fused_r(const ConvArgs &ca, int cfg, int ndx, int gx, const DkArgs &da, int dgx,
                    int dgy, int ndk, hipStream_t st) {
    if (cfg == 2)
        launch_fused<R, 4, 4>(ca, ndx, gx, da, dgx, dgy, ndk, st);
    else if (cfg == 1)
        launch_fused<R, 1, 2>(ca, ndx, gx, da, dgx, dgy, ndk, st);
    else
        launch_fused<R, 1, 1>(ca, ndx, gx, da, dgx, dgy, ndk, st);
}

// Both gradients of one layer whose images lie img floats apart in x, dy and
// dx (C H W for a whole tensor, more for a channel slice of a wider one);
// partial: dk_parts(B, C, H, W, k) C^2 k^2 floats.  Arguments checked by
// the caller.
int launch_layer_backward(const float *x, const float *dy, const float *K, float *dx, float *dK,
                          double gld, int B, int C, int H, int W, int k, int corner,
                          long long img, float *partial, hipStream_t stream) {
    const int oh = (corner == FINC_TL || corner == FINC_TR) ? k - 1 : 0;
    const int ow = (corner == FINC_TL || corner == FINC_BL) ? k - 1 : 0;
    const int n = C * C * k * k;
    const long long Q = (long long)B * H * W;
    // the input gradient: the convolution of dy with K transposed and flipped
    ConvArgs ca;
    memset(&ca, 0, sizeof(ca));
    int cfg = 0, gx = 0, ndx = 0;
    if (dx && B > 0) {
        ca.x = dy;
        ca.y = dx;
        ca.Wt = K;
        ca.B = B;
        ca.Ci = C;
        ca.Co = C;
        ca.H = H;
        ca.W = W;
        ca.K = C * k * k;
        ca.ph = k - 1 - oh;
        ca.pw = k - 1 - ow;
        ca.xs = ca.ys = img;
        ca.d_HW = make_div(H * W);
        ca.d_W = make_div(W);
        ca.flip = 1;
        ca.fself = oh * k + ow;
        cfg = C >= 64 ? 2 : cdiv(Q, 128) >= 256 ? 1 : 0;
        const int bn = cfg == 2 ? 64 : cfg == 1 ? 128 : 64, bm = cfg == 2 ? 64 : 16;
        gx = cdiv(Q, bn);
        ndx = gx * cdiv(C, bm);
    }
    // dK's partial sums over parts of the positions
    DkArgs da;
    memset(&da, 0, sizeof(da));
    int parts = 0, dgx = 1, dgy = 1, ndk = 0;
    if (dK && B > 0) {
        parts = dk_parts(B, C, H, W, k);
        da.x = x;
        da.dy = dy;
        da.partial = partial;
        da.img = img;
        da.B = B;
        da.C = C;
        da.H = H;
        da.W = W;
        da.k = k;
        da.oh = oh;
        da.ow = ow;
        da.N = C * k * k;
        da.nchunk = cdiv(Q, 64);
        da.cpp = cdiv(da.nchunk, parts);
        parts = cdiv(da.nchunk, da.cpp);
        da.d_HW = make_div(H * W);
        da.d_W = make_div(W);
        da.d_kk = make_div(k * k);
        da.d_k = make_div(k);
        dgx = cdiv(da.N, 64);
        dgy = cdiv(C, 16);
        ndk = dgx * dgy * parts;
    }
    if (ndx + ndk > 0) {
        switch (k) {
        case 1: launch_fused_r<1>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        case 2: launch_fused_r<2>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        case 3: launch_fused_r<3>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        case 4: launch_fused_r<4>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        case 5: launch_fused_r<5>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        case 6: launch_fused_r<6>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        default: launch_fused_r<7>(ca, cfg, ndx, gx, da, dgx, dgy, ndk, stream); break;
        }
        const int rc = conv_launched();
        if (rc != FINC_OK)
            return rc;
    }
    if (!dK)
        return FINC_OK;
    hipLaunchKernelGGL(dk_reduce_kernel, dim3((n + 7) / 8), dim3(256), 0, stream, partial, parts,
                       K, dK, gld, C, k, H, W, oh, ow);
    return conv_launched();
}



// ---- actnorm backward -----------------------------------------------------
// y = s x + b per channel: dx = s dy; ds[c] = sum dy x + gld H W / s[c];
// db[c] = sum dy.  Block (c, part) covers images [part bpp, (part+1) bpp) of
// channel c: it writes dx there and its two sums (fp64, each thread's
// elements in order, then a fixed tree) to partial[(c parts + part) 2 + .];
// actnorm_reduce_kernel adds the parts in order.
constexpr int kAnThreads = 256;

__global__ __launch_bounds__(kAnThreads) void actnorm_bwd_kernel(const float *x, const float *dy,
                                                                 const float *s, float *dx,
                                                                 double *partial, int B, int C,
                                                                 int HW, int bpp, int parts) {
    __shared__ double red[2][kAnThreads];
    const int c = blockIdx.x, part = blockIdx.y, tid = threadIdx.x;
    const int b0 = part * bpp, b1 = min(b0 + bpp, B);
    const float sc = s[c];
    double sx = 0.0, sy = 0.0;
    for (int b = b0; b < b1; ++b) {
        const long long base = ((long long)b * C + c) * HW;
        for (int p = tid; p < HW; p += kAnThreads) {
            const float g = dy[base + p];
            sx += (double)g * (double)x[base + p];
            sy += (double)g;
            if (dx)
                dx[base + p] = sc * g;
        }
    }
    red[0][tid] = sx;
    red[1][tid] = sy;
    __syncthreads();
    for (int h = kAnThreads / 2; h > 0; h >>= 1) {
        if (tid < h) {
            red[0][tid] += red[0][tid + h];
            red[1][tid] += red[1][tid + h];
        }
        __syncthreads();
    }
    if (tid == 0) {
        partial[((long long)c * parts + part) * 2] = red[0][0];
        partial[((long long)c * parts + part) * 2 + 1] = red[1][0];
    }
}

__global__ __launch_bounds__(64) void actnorm_reduce_kernel(const double *partial, int parts,
                                                            const float *s, float *ds, float *db,
                                                            double gld, int C, int HW) {
    const int c = blockIdx.x * 64 + threadIdx.x;
    if (c >= C)
        return;
    double sx = 0.0, sy = 0.0;
    for (int z = 0; z < parts; ++z) {
        sx += partial[((long long)c * parts + z) * 2];
        sy += partial[((long long)c * parts + z) * 2 + 1];
    }
    if (ds)
        ds[c] = (float)(sx + gld * (double)HW / (double)s[c]);
    if (db)
        db[c] = (float)sy;
}

// Parts of the batch per channel: about 512 blocks over the chip, at least
// 16 K values per block.
int actnorm_parts(int B, int C, int HW) {
    long long parts = 512 / C;
    const long long per = (16384 + HW - 1) / HW;   // images per block at minimum
    if (parts > (B + per - 1) / per)
        parts = (B + per - 1) / per;
    return (int)(parts < 1 ? 1 : parts);
}

// ---- negative log-likelihood ----------------------------------------------
// One block per image: each latent's values in a fixed order (thread t takes
// t, t + 256, ...; fp64), a fixed tree over the threads, the latents in order.
constexpr int kNllMaxL = 16;
struct NllArgs {
    const float *z[kNllMaxL];
    long long n[kNllMaxL];
    int L;
    long long D;
    const double *logdet;
    double *nll, *bpd;
};

__global__ __launch_bounds__(256) void gauss_nll_kernel(NllArgs a) {
    __shared__ double red[256];
    const int b = blockIdx.x, tid = threadIdx.x;
    double total = 0.0;
    for (int l = 0; l < a.L; ++l) {
        const float *zb = a.z[l] + (long long)b * a.n[l];
        double q = 0.0;
        for (long long e = tid; e < a.n[l]; e += 256) {
            const double v = zb[e];
            q += v * v;
        }
        red[tid] = q;
        __syncthreads();
        for (int h = 128; h > 0; h >>= 1) {
            if (tid < h)
                red[tid] += red[tid + h];
            __syncthreads();
        }
        total += red[0];
        __syncthreads();
    }
    if (tid == 0) {
        const double log2pi = 1.8378770664093454836;   // log(2 pi)
        const double nll = 0.5 * (total + (double)a.D * log2pi) - a.logdet[b];
        a.nll[b] = nll;
        if (a.bpd)
            a.bpd[b] = nll / ((double)a.D * 0.69314718055994530942);   // / (D log 2)
    }
}


// ---- the multi-scale stack's training direction ----------------------------
// (B C H W < 2^31 values: int indices)

// y = s[c] x + b[c] (actnorm forward).
__global__ __launch_bounds__(256) void affine_kernel(const float *x, float *y, const float *s,
                                                     const float *b, int n, Div d_HW, Div d_C,
                                                     int C) {
    for (int e = blockIdx.x * 256 + threadIdx.x; e < n; e += gridDim.x * 256) {
        const int pl = divi(e, d_HW), c = pl - divi(pl, d_C) * C;
        y[e] = s[c] * x[e] + b[c];
    }
}

// Split and squeeze of a level's output h (B, C, H, W): channels [C/2, C)
// go to the latent z (B, C/2, H, W); channel c < C/2 at (2 i + dy, 2 j + dx)
// goes to channel 4 c + 2 dy + dx of the next level's input (B, 2C, H/2, W/2).
__global__ __launch_bounds__(256) void split_squeeze_kernel(const float *h, float *nxt, float *z,
                                                            int n, int C, int H, int W, Div d_HW,
                                                            Div d_C, Div d_W) {
    const int HW = H * W, Ch = C / 2;
    for (int e = blockIdx.x * 256 + threadIdx.x; e < n; e += gridDim.x * 256) {
        const int pl = divi(e, d_HW), p = e - pl * HW;
        const int b = divi(pl, d_C), c = pl - b * C;
        if (c >= Ch) {
            z[(b * Ch + c - Ch) * HW + p] = h[e];
        } else {
            const int i = divi(p, d_W), j = p - i * W;
            const int co = 4 * c + 2 * (i & 1) + (j & 1);
            nxt[((b * 2 * C + co) * (H / 2) + (i >> 1)) * (W / 2) + (j >> 1)] = h[e];
        }
    }
}

// Its adjoint: the gradient of a level's output, g (B, C, H, W), from the
// gradient of the next level's input gn (B, 2C, H/2, W/2) -- unsqueezed,
// first half -- and the latent's gradient dz (B, C/2, H, W), second half.
__global__ __launch_bounds__(256) void unsqueeze_concat_kernel(const float *gn, const float *dz,
                                                               float *g, int n, int C, int H,
                                                               int W, Div d_HW, Div d_C,
                                                               Div d_W) {
    const int HW = H * W, Ch = C / 2;
    for (int e = blockIdx.x * 256 + threadIdx.x; e < n; e += gridDim.x * 256) {
        const int pl = divi(e, d_HW), p = e - pl * HW;
        const int b = divi(pl, d_C), c = pl - b * C;
        if (c >= Ch) {
            g[e] = dz[(b * Ch + c - Ch) * HW + p];
        } else {
            const int i = divi(p, d_W), j = p - i * W;
            const int co = 4 * c + 2 * (i & 1) + (j & 1);
            g[e] = gn[((b * 2 * C + co) * (H / 2) + (i >> 1)) * (W / 2) + (j >> 1)];
        }
    }
}

// The stack's log|det| for one image -- every block's H W sum_c
// log|K[c][c][self]| and every actnorm's H W sum_c log|s_c| -- in fp64, each
// thread's terms in order and a fixed tree; written for every image.
__global__ __launch_bounds__(256) void stack_logdet_kernel(const float *K, const float *scale,
                                                           int L, int U, int C1, int H1, int W1,
                                                           int k, double *logdet, int B) {
    __shared__ double red[256];
    const int tid = threadIdx.x;
    double acc = 0.0;
    long long koff = 0, soff = 0;
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l;
        const double hw = (double)(H1 >> l) * (double)(W1 >> l);
        const long long ksz = (long long)C * C * k * k;
        // per unit: 4 C diagonal entries, then C scales
        for (int t = tid; t < U * 5 * C; t += 256) {
            const int u = t / (5 * C), r = t - u * 5 * C;
            if (r < 4 * C) {
                const int q = r / C, c = r - q * C;
                const int oh = (q == 0 || q == 1) ? k - 1 : 0, ow = (q == 0 || q == 2) ? k - 1 : 0;
                const float d = K[koff + (4ll * u + q) * ksz + ((long long)(c * C + c) * k + oh) * k + ow];
                acc += hw * log(fabs((double)d));
            } else {
                acc += hw * log(fabs((double)scale[soff + (long long)u * C + (r - 4 * C)]));
            }
        }
        koff += 4ll * U * ksz;
        soff += (long long)U * C;
    }
    red[tid] = acc;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (tid < h)
            red[tid] += red[tid + h];
        __syncthreads();
    }
    for (int b = tid; b < B; b += 256)
        logdet[b] = red[0];
}

int ew_blocks(long long n) { return (int)(n / 256 + 1 < 4096 ? n / 256 + 1 : 4096); }

struct StackShape {
    int B, L, U, C1, H1, W1, k;
    long long n0;   // values of a level-0 activation
    int C(int l) const { return C1 << l; }
    int H(int l) const { return H1 >> l; }
    int W(int l) const { return W1 >> l; }
    long long n(int l) const { return n0 >> l; }   // (C doubles, H W quarters)
    long long koff(int l) const {
        long long o = 0;
        for (int m = 0; m < l; ++m)
            o += 4ll * U * C(m) * C(m) * k * k;
        return o;
    }
    long long soff(int l) const {
        long long o = 0;
        for (int m = 0; m < l; ++m)
            o += (long long)U * C(m);
        return o;
    }
    long long kfloats() const { return koff(L); }
    long long sfloats() const { return soff(L); }
};

bool stack_shape_ok(const StackShape &s) {
    if (s.B < 0 || s.L < 1 || s.L > 8 || s.U < 0 || s.C1 < 1 || s.H1 < 1 || s.W1 < 1 || s.k < 1 ||
        s.k > FINC_MAX_K)
        return false;
    if (s.L > 1 && ((s.C1 & 1) || ((s.H1 | s.W1) & ((1 << (s.L - 1)) - 1))))
        return false;
    return (s.C1 << (s.L - 1)) <= FINC_MAX_C && s.n0 < (1ll << 31);
}

// Workspace of the stack's training calls: per level its 2 U + 1 activations
// (unit inputs, unit outputs, the level's output), three level-0 gradient
// buffers, and the unit and actnorm backward workspaces of the largest level.
struct StackWs {
    size_t acts, grads, unit_ws, an_ws, total;
};
StackWs stack_ws(const StackShape &s) {
    StackWs w;
    long long na = 0;
    for (int l = 0; l < s.L; ++l)
        na += (2ll * s.U + 1) * s.n(l);
    w.acts = up256b((size_t)na * sizeof(float));
    w.grads = 3 * up256b((size_t)s.n0 * sizeof(float));
    w.unit_ws = 0;
    w.an_ws = 0;
    for (int l = 0; l < s.L; ++l) {
        w.unit_ws = imax_sz(w.unit_ws, finc_unit_backward_workspace_bytes(s.B, s.C(l), s.H(l), s.W(l), s.k));
        w.an_ws = imax_sz(w.an_ws, finc_actnorm_backward_workspace_bytes(s.B, s.C(l), s.H(l), s.W(l)));
    }
    w.unit_ws = up256b(w.unit_ws);
    w.an_ws = up256b(w.an_ws);
    w.total = w.acts + w.grads + w.unit_ws + w.an_ws;
    return w;
}

// The forward direction, keeping every level's activations in acts (level l
// at acts + aoff[l]: h_0 = the level's input, t_0, h_1, t_1, ..., h_U = its
// output; t_u = unit(h_u), h_{u+1} = actnorm(t_u)); level 0's h_0 is x
// itself and the top level's h_U is written to its latent z[L-1] directly.
inline const float *stack_h(const float *x, const float *acts, const long long *aoff,
                            const StackShape &s, int l, int u) {
    return (l == 0 && u == 0) ? x : acts + aoff[l] + 2ll * u * s.n(l);
}

int stack_forward_keep(const float *x, float *const *z, const float *K, const float *scale,
                       const float *bias, const StackShape &s, float *acts, long long *aoff,
                       hipStream_t st) {
    long long o = 0;
    for (int l = 0; l < s.L; ++l) {
        const int C = s.C(l), H = s.H(l), W = s.W(l);
        const long long n = s.n(l), ksz = (long long)C * C * s.k * s.k;
        aoff[l] = o;
        o += (2ll * s.U + 1) * n;
        const bool top = l == s.L - 1;
        for (int u = 0; u < s.U; ++u) {
            const float *hu = stack_h(x, acts, aoff, s, l, u);
            float *tu = acts + aoff[l] + (2ll * u + 1) * n;
            float *nx = (top && u == s.U - 1) ? z[l] : tu + n;
            int rc = finc_unit_forward(hu, tu, K + s.koff(l) + 4ll * u * ksz, nullptr, nullptr,
                                       s.B, C, H, W, s.k, st);
            if (rc != FINC_OK)
                return rc;
            if (s.B > 0) {
                hipLaunchKernelGGL(affine_kernel, dim3(ew_blocks(n)), dim3(256), 0, st, tu, nx,
                                   scale + s.soff(l) + (long long)u * C,
                                   bias + s.soff(l) + (long long)u * C, (int)n, make_div(H * W),
                                   make_div(C), C);
                rc = conv_launched();
                if (rc != FINC_OK)
                    return rc;
            }
        }
        if (s.B == 0)
            continue;
        const float *hout = stack_h(x, acts, aoff, s, l, s.U);
        if (top) {
            if (s.U == 0 && hipMemcpyAsync(z[l], hout, (size_t)n * sizeof(float),
                                           hipMemcpyDeviceToDevice, st) != hipSuccess)
                return FINC_EHIP;
        } else {
            hipLaunchKernelGGL(split_squeeze_kernel, dim3(ew_blocks(n)), dim3(256), 0, st, hout,
                               acts + o, z[l], (int)n, C, H, W, make_div(H * W), make_div(C),
                               make_div(W));
            const int rc = conv_launched();
            if (rc != FINC_OK)
                return rc;
        }
    }
    return FINC_OK;
}

}  // namespace

extern "C" {

size_t finc_backward_workspace_bytes(int B, int C, int H, int W, int k) {
    if (!valid_bwd_shape(B, C, H, W, k))
        return 0;
    const int parts = dk_parts(B, C, H, W, k);
    return up256b((size_t)parts * C * C * k * k * sizeof(float));
}

int finc_backward(const float *x, const float *dy, const float *K, float *dx, float *dK,
                  double gld, int B, int C, int H, int W, int k, int corner, void *workspace,
                  hipStream_t stream) {
    if (!valid_bwd_shape(B, C, H, W, k) || corner < FINC_TL || corner > FINC_BR ||
        (B > 0 && (!x || !dy)) || !K || !workspace || ((uintptr_t)workspace & 255u))
        return FINC_EINVAL;
    const size_t act = (size_t)B * C * H * W * sizeof(float);
    const size_t wts = (size_t)C * C * k * k * sizeof(float);
    const size_t wsb = finc_backward_workspace_bytes(B, C, H, W, k);
    if (dx && (overlapb(dx, act, x, act) || overlapb(dx, act, dy, act) ||
               overlapb(dx, act, K, wts) || (dK && overlapb(dx, act, dK, wts)) ||
               overlapb(dx, act, workspace, wsb)))
        return FINC_EINVAL;
    if (dK && (overlapb(dK, wts, x, act) || overlapb(dK, wts, dy, act) ||
               overlapb(dK, wts, K, wts) || overlapb(dK, wts, workspace, wsb)))
        return FINC_EINVAL;
    if (overlapb(workspace, wsb, x, act) || overlapb(workspace, wsb, dy, act) ||
        overlapb(workspace, wsb, K, wts))
        return FINC_EINVAL;
    return launch_layer_backward(x, dy, K, dx, dK, gld, B, C, H, W, k, corner,
                                 (long long)C * H * W, (float *)workspace, stream);
}


// ---- backward of the FInC units ---------------------------------------------

size_t finc_unit_backward_workspace_bytes(int B, int C, int H, int W, int k) {
    if (!valid_bwd_shape(B, C, H, W, k))
        return 0;
    return 4 * up256b((size_t)B * C * H * W * sizeof(float)) +
           finc_backward_workspace_bytes(B, C, H, W, k);
}

int finc_unit_backward(const float *x, const float *dy, const float *K4, float *dx, float *dK4,
                       double gld, int B, int C, int H, int W, int k, void *workspace,
                       hipStream_t stream) {
    if (!valid_bwd_shape(B, C, H, W, k) || (B > 0 && (!x || !dy)) || !K4 || !workspace ||
        ((uintptr_t)workspace & 255u))
        return FINC_EINVAL;
    const size_t act = (size_t)B * C * H * W * sizeof(float);
    const size_t wts = 4 * (size_t)C * C * k * k * sizeof(float);
    const size_t wsb = finc_unit_backward_workspace_bytes(B, C, H, W, k);
    const void *ins[3] = {x, dy, K4};
    const size_t insz[3] = {act, act, wts};
    for (int i = 0; i < 3; ++i)
        if (overlapb(workspace, wsb, ins[i], insz[i]) || (dx && overlapb(dx, act, ins[i], insz[i])) ||
            (dK4 && overlapb(dK4, wts, ins[i], insz[i])))
            return FINC_EINVAL;
    if ((dx && (overlapb(dx, act, workspace, wsb) || (dK4 && overlapb(dx, act, dK4, wts)))) ||
        (dK4 && overlapb(dK4, wts, workspace, wsb)))
        return FINC_EINVAL;
    const size_t ksz = (size_t)C * C * k * k;
    char *w = (char *)workspace;
    const size_t slot = up256b(act);
    float *h[4] = {(float *)x, (float *)w, (float *)(w + slot), (float *)(w + 2 * slot)};
    float *g = (float *)(w + 3 * slot);
    float *partial = (float *)(w + 4 * slot);
    // the inputs of blocks TR, BL, BR, recomputed: h[q + 1] = block q (h[q])
    for (int q = 0; q < 3 && B > 0; ++q) {
        const int rc = finc_forward(h[q], h[q + 1], K4 + q * ksz, nullptr, nullptr, B, C, H, W,
                                    k, q, stream);
        if (rc != FINC_OK)
            return rc;
    }
    // blocks in reverse; the gradient alternates between g and the freed slots
    const float *gin = dy;
    float *gout[4] = {dx, g, h[3], g};   // block q writes its input gradient to gout[q]
    for (int q = 3; q >= 0; --q) {
        const int rc = launch_layer_backward(h[q], gin, K4 + q * ksz, gout[q],
                                             dK4 ? dK4 + q * ksz : nullptr, gld, B, C, H, W, k,
                                             q, (long long)C * H * W, partial, stream);
        if (rc != FINC_OK)
            return rc;
        gin = gout[q];
    }
    return FINC_OK;
}

size_t finc_split_backward_workspace_bytes(int B, int C, int H, int W, int k) {
    if (C % 4 != 0 || !valid_bwd_shape(B, C / 4, H, W, k))
        return 0;
    return finc_backward_workspace_bytes(B, C / 4, H, W, k);
}

int finc_split_backward(const float *x, const float *dy, const float *Kq4, float *dx,
                        float *dKq4, double gld, int B, int C, int H, int W, int k,
                        void *workspace, hipStream_t stream) {
    if (C % 4 != 0 || !valid_bwd_shape(B, C / 4, H, W, k) || (B > 0 && (!x || !dy)) || !Kq4 ||
        !workspace || ((uintptr_t)workspace & 255u))
        return FINC_EINVAL;
    const int q = C / 4;
    const size_t act = (size_t)B * C * H * W * sizeof(float);
    const size_t wts = 4 * (size_t)q * q * k * k * sizeof(float);
    const size_t wsb = finc_split_backward_workspace_bytes(B, C, H, W, k);
    const void *ins[3] = {x, dy, Kq4};
    const size_t insz[3] = {act, act, wts};
    for (int i = 0; i < 3; ++i)
        if (overlapb(workspace, wsb, ins[i], insz[i]) || (dx && overlapb(dx, act, ins[i], insz[i])) ||
            (dKq4 && overlapb(dKq4, wts, ins[i], insz[i])))
            return FINC_EINVAL;
    if ((dx && (overlapb(dx, act, workspace, wsb) || (dKq4 && overlapb(dx, act, dKq4, wts)))) ||
        (dKq4 && overlapb(dKq4, wts, workspace, wsb)))
        return FINC_EINVAL;
    const long long img = (long long)C * H * W, plane = (long long)q * H * W;
    const size_t ksz = (size_t)q * q * k * k;
    for (int g = 0; g < 4; ++g) {   // quarter g: corner g on channels [g q, (g+1) q)
        const int rc = launch_layer_backward(
            B > 0 ? x + g * plane : x, B > 0 ? dy + g * plane : dy, Kq4 + g * ksz,
            dx && B > 0 ? dx + g * plane : nullptr, dKq4 ? dKq4 + g * ksz : nullptr, gld, B, q,
            H, W, k, g, img, (float *)workspace, stream);
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

// ---- actnorm backward and the negative log-likelihood -----------------------

size_t finc_actnorm_backward_workspace_bytes(int B, int C, int H, int W) {
    if (B < 0 || C < 1 || H < 1 || W < 1 || (long long)B * C * H * W >= (1ll << 31))
        return 0;
    return up256b((size_t)2 * C * actnorm_parts(B, C, H * W) * sizeof(double));
}

int finc_actnorm_backward(const float *x, const float *dy, const float *s, float *dx, float *ds,
                          float *db, double gld, int B, int C, int H, int W, void *workspace,
                          hipStream_t stream) {
    const size_t wsb = finc_actnorm_backward_workspace_bytes(B, C, H, W);
    if (wsb == 0 || (B > 0 && (!x || !dy)) || !s || !workspace || ((uintptr_t)workspace & 255u))
        return FINC_EINVAL;
    const size_t act = (size_t)B * C * H * W * sizeof(float), vec = (size_t)C * sizeof(float);
    const void *ins[3] = {x, dy, s};
    const size_t insz[3] = {act, act, vec};
    void *outs[4] = {dx, ds, db, workspace};
    const size_t outsz[4] = {act, vec, vec, wsb};
    for (int o = 0; o < 4; ++o) {
        if (!outs[o])
            continue;
        for (int i = 0; i < 3; ++i)
            if (overlapb(outs[o], outsz[o], ins[i], insz[i]))
                return FINC_EINVAL;
        for (int o2 = o + 1; o2 < 4; ++o2)
            if (outs[o2] && overlapb(outs[o], outsz[o], outs[o2], outsz[o2]))
                return FINC_EINVAL;
    }
    const int HW = H * W, parts = actnorm_parts(B, C, HW);
    const int bpp = B > 0 ? cdiv(B, parts) : 0;
    double *partial = (double *)workspace;
    const int np = B > 0 ? cdiv(B, bpp) : 0;   // parts that hold images
    if (np > 0) {
        hipLaunchKernelGGL(actnorm_bwd_kernel, dim3(C, np), dim3(kAnThreads), 0, stream, x, dy, s,
                           dx, partial, B, C, HW, bpp, np);
        const int rc = conv_launched();
        if (rc != FINC_OK)
            return rc;
    }
    if (!ds && !db)
        return FINC_OK;
    hipLaunchKernelGGL(actnorm_reduce_kernel, dim3((C + 63) / 64), dim3(64), 0, stream, partial,
                       np, s, ds, db, gld, C, HW);
    return conv_launched();
}

int finc_gauss_nll(const float *const *z, const long long *n, int L, int B, const double *logdet,
                   double *nll, double *bpd, hipStream_t stream) {
    if (L < 1 || L > kNllMaxL || B < 0 || !z || !n || !logdet || !nll)
        return FINC_EINVAL;
    NllArgs a;
    memset(&a, 0, sizeof(a));
    a.L = L;
    for (int l = 0; l < L; ++l) {
        if (n[l] < 1 || (B > 0 && !z[l]))
            return FINC_EINVAL;
        a.z[l] = z[l];
        a.n[l] = n[l];
        a.D += n[l];
    }
    const size_t per = (size_t)B * sizeof(double);
    if (overlapb(nll, per, logdet, per) || (bpd && (overlapb(bpd, per, logdet, per) ||
                                                    overlapb(bpd, per, nll, per))))
        return FINC_EINVAL;
    for (int l = 0; l < L; ++l) {
        const size_t zb = (size_t)B * n[l] * sizeof(float);
        if (overlapb(nll, per, z[l], zb) || (bpd && overlapb(bpd, per, z[l], zb)))
            return FINC_EINVAL;
    }
    a.logdet = logdet;
    a.nll = nll;
    a.bpd = bpd;
    if (B == 0)
        return FINC_OK;
    hipLaunchKernelGGL(gauss_nll_kernel, dim3(B), dim3(256), 0, stream, a);
    return conv_launched();
}


// ---- the multi-scale stack's training direction ------------------------------

size_t finc_stack_train_workspace_bytes(int B, int L, int U, int C1, int H1, int W1, int k) {
    StackShape s{B, L, U, C1, H1, W1, k, (long long)B * C1 * H1 * W1};
    if (!stack_shape_ok(s))
        return 0;
    return stack_ws(s).total;
}

static bool stack_buffers_ok(const StackShape &s, const float *x, const float *const *z,
                             const float *K, const float *scale, const float *bias,
                             void *workspace, const void *const *outs, const size_t *outsz,
                             int nouts) {
    if ((s.B > 0 && !x) || !z || !K || !scale || !bias || !workspace ||
        ((uintptr_t)workspace & 255u))
        return false;
    const size_t wsb = stack_ws(s).total;
    const size_t xb = (size_t)s.n0 * sizeof(float);
    const void *ins[4] = {x, K, scale, bias};
    const size_t insz[4] = {xb, (size_t)s.kfloats() * sizeof(float),
                            (size_t)s.sfloats() * sizeof(float),
                            (size_t)s.sfloats() * sizeof(float)};
    for (int l = 0; l < s.L; ++l)
        if (s.B > 0 && !z[l])
            return false;
    for (int i = 0; i < 4; ++i)
        if (overlapb(workspace, wsb, ins[i], insz[i]))
            return false;
    for (int o = 0; o < nouts; ++o) {
        if (!outs[o])
            continue;
        if (overlapb(outs[o], outsz[o], workspace, wsb))
            return false;
        for (int i = 0; i < 4; ++i)
            if (overlapb(outs[o], outsz[o], ins[i], insz[i]))
                return false;
        for (int o2 = o + 1; o2 < nouts; ++o2)
            if (outs[o2] && overlapb(outs[o], outsz[o], outs[o2], outsz[o2]))
                return false;
    }
    return true;
}

int finc_stack_forward(const float *x, float *const *z, double *logdet, const float *K,
                       const float *scale, const float *bias, int B, int L, int U, int C1,
                       int H1, int W1, int k, void *workspace, hipStream_t stream) {
    StackShape s{B, L, U, C1, H1, W1, k, (long long)B * C1 * H1 * W1};
    if (!stack_shape_ok(s) || !z)
        return FINC_EINVAL;
    const void *outs[10];
    size_t outsz[10];
    int no = 0;
    for (int l = 0; l < L; ++l) {
        outs[no] = z[l];
        outsz[no++] = (size_t)(l == L - 1 ? s.n(l) : s.n(l) / 2) * sizeof(float);
    }
    outs[no] = logdet;
    outsz[no++] = (size_t)B * sizeof(double);
    if (!stack_buffers_ok(s, x, (const float *const *)z, K, scale, bias, workspace, outs, outsz,
                          no))
        return FINC_EINVAL;
    long long aoff[8];
    int rc = stack_forward_keep(x, z, K, scale, bias, s, (float *)workspace, aoff, stream);
    if (rc != FINC_OK || !logdet || B == 0)
        return rc;
    hipLaunchKernelGGL(stack_logdet_kernel, dim3(1), dim3(256), 0, stream, K, scale, L, U, C1,
                       H1, W1, k, logdet, B);
    return conv_launched();
}

int finc_stack_backward(const float *x, const float *const *dz, const float *K,
                        const float *scale, const float *bias, float *dx, float *dK,
                        float *dscale, float *dbias, double gld, int B, int L, int U, int C1,
                        int H1, int W1, int k, void *workspace, hipStream_t stream) {
    StackShape s{B, L, U, C1, H1, W1, k, (long long)B * C1 * H1 * W1};
    if (!stack_shape_ok(s) || !dz)
        return FINC_EINVAL;
    const void *outs[4] = {dx, dK, dscale, dbias};
    const size_t outsz[4] = {(size_t)s.n0 * sizeof(float), (size_t)s.kfloats() * sizeof(float),
                             (size_t)s.sfloats() * sizeof(float),
                             (size_t)s.sfloats() * sizeof(float)};
    if (!stack_buffers_ok(s, x, dz, K, scale, bias, workspace, outs, outsz, 4))
        return FINC_EINVAL;
    for (int l = 0; l < L; ++l) {   // the latents' gradients are inputs too
        const size_t zb = (size_t)(l == L - 1 ? s.n(l) : s.n(l) / 2) * sizeof(float);
        for (int o = 0; o < 4; ++o)
            if (outs[o] && overlapb(outs[o], outsz[o], dz[l], zb))
                return FINC_EINVAL;
        if (overlapb(workspace, stack_ws(s).total, dz[l], zb))
            return FINC_EINVAL;
    }
    const StackWs w = stack_ws(s);
    char *base = (char *)workspace;
    float *acts = (float *)base;
    float *gbuf[3];
    for (int i = 0; i < 3; ++i)
        gbuf[i] = (float *)(base + w.acts + i * up256b((size_t)s.n0 * sizeof(float)));
    void *unit_ws = base + w.acts + w.grads, *an_ws = base + w.acts + w.grads + w.unit_ws;
    // the forward again, keeping its activations (the latents it writes go to
    // a gradient buffer, unused until the forward is done)
    float *zscratch[8];
    for (int l = 0; l < L; ++l)
        zscratch[l] = gbuf[2];
    long long aoff[8];
    int rc = stack_forward_keep(x, zscratch, K, scale, bias, s, acts, aoff, stream);
    if (rc != FINC_OK)
        return rc;
    // gin: the gradient of the activation reached so far (the top latent's
    // gradient first); results alternate between two buffers, the input's
    // gradient goes to dx
    float *buf[2] = {gbuf[0], gbuf[2]}, *gt = gbuf[1];
    int cur = 0;
    const float *gin = dz[L - 1];
    for (int l = L - 1; l >= 0; --l) {
        const int C = s.C(l), H = s.H(l), W = s.W(l);
        const long long n = s.n(l), ksz = (long long)C * C * k * k;
        if (l < L - 1 && B > 0) {   // gin: the next level's input gradient
            float *o = buf[cur];
            cur ^= 1;
            hipLaunchKernelGGL(unsqueeze_concat_kernel, dim3(ew_blocks(n)), dim3(256), 0, stream,
                               gin, dz[l], o, (int)n, C, H, W, make_div(H * W), make_div(C),
                               make_div(W));
            rc = conv_launched();
            if (rc != FINC_OK)
                return rc;
            gin = o;
        }
        for (int u = U - 1; u >= 0; --u) {
            const float *hu = stack_h(x, acts, aoff, s, l, u);
            const float *tu = acts + aoff[l] + (2ll * u + 1) * n;
            const long long so = s.soff(l) + (long long)u * C;
            rc = finc_actnorm_backward(tu, gin, scale + so, gt, dscale ? dscale + so : nullptr,
                                       dbias ? dbias + so : nullptr, gld, B, C, H, W, an_ws,
                                       stream);
            if (rc != FINC_OK)
                return rc;
            const bool last = l == 0 && u == 0;
            float *o = last ? dx : buf[cur];
            if (!last)
                cur ^= 1;
            rc = finc_unit_backward(hu, gt, K + s.koff(l) + 4ll * u * ksz, o,
                                    dK ? dK + s.koff(l) + 4ll * u * ksz : nullptr, gld, B, C, H,
                                    W, k, unit_ws, stream);
            if (rc != FINC_OK)
                return rc;
            gin = o;
        }
    }
    // (no unit at level 0: the input's gradient is the level's)
    if (dx && U == 0 && B > 0 &&
        hipMemcpyAsync(dx, gin, (size_t)s.n0 * sizeof(float), hipMemcpyDeviceToDevice, stream) !=
            hipSuccess)
        return FINC_EHIP;
    return FINC_OK;
}

}  // extern "C"
