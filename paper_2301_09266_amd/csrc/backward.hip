// backward.hip -- backward of the masked k x k convolution layer on gfx950,
// for training on the negative log-likelihood (Sec. 2 NLL equation; the
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
    const long long img = (long long)a.C * HW;
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
    const int oh = (corner == FINC_TL || corner == FINC_TR) ? k - 1 : 0;
    const int ow = (corner == FINC_TL || corner == FINC_BL) ? k - 1 : 0;
    float *partial = (float *)workspace;
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
        ca.xs = ca.ys = (long long)C * H * W;
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

}  // extern "C"
