// conv_gemm.h -- an R x R convolution with per-axis offsets as an fp32 MFMA
// implicit GEMM on gfx950 (v_mfma_f32_16x16x4_f32), shared by the full flow
// (coupling and prior networks, the 1x1 convolution) and the backward of the
// masked layer (its input gradient, a convolution of the output gradient).
//
//   y[b][co][i][j] = act(bias[co] + sum_{ci,a,c} Wt[co][ci][a][c] *
//                        x[b][ci][i + a - ph][j + c - pw]) * oscale[co]
//
// zeros outside the image; act = ReLU or identity; oscale = exp(3 ls[co]) or
// 1; bias may be null (0).  Weights are OIHW, so W[co][k] with
// k = ci R^2 + a R + c is contiguous in k.  Pixels are flattened over the
// batch (q = b H W + p), so a block's tile may span images.
//
// Block: 256 threads, 4 waves arranged WCO (along c_out) x 4 / WCO (along
// pixels); each wave computes 16 c_out x 16 NS pixels (NS accumulators).
// K is staged 64 values at a time: A[co][k] (weights) and B[px][k] (the
// gathered input window, im2col on the fly), rows padded to 68 floats, the
// next chunk's global loads in flight during the current chunk's MFMAs.
// Within one 16-wide slice of k, lane group kq takes k = 4 kq .. 4 kq + 3 as
// the four MFMAs' k (one float4 LDS read each for A and B).  A long K may be
// split into parts (blockIdx.z) whose raw sums a second kernel adds in order.
// Every summation order is fixed: results are bitwise deterministic.
#ifndef FINC_CONV_GEMM_H
#define FINC_CONV_GEMM_H

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "finc.h"

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

inline int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }

// Division of a non-negative int by a divisor fixed on the host (multiply-
// high and shifts, Granlund and Montgomery's round-up method).
struct Div {
    unsigned m;
    int s1, s2;
};
inline Div make_div(int d) {
    int l = 0;
    while ((1ull << l) < (unsigned long long)d)
        ++l;
    Div f;
    f.m = (unsigned)((((1ull << l) - (unsigned long long)d) << 32) / (unsigned long long)d + 1);
    f.s1 = l < 1 ? l : 1;
    f.s2 = l > 1 ? l - 1 : 0;
    return f;
}
__device__ inline int divi(int x, const Div &f) {
    const unsigned t = __umulhi(f.m, (unsigned)x);
    return (int)((t + (((unsigned)x - t) >> f.s1)) >> f.s2);
}

struct ConvArgs {
    const float *x;
    float *y;
    const float *Wt;     // (Co, Ci, R, R)
    const float *bias;   // (Co) or null
    const float *ls;     // (Co) or null
    int relu;
    int B, Ci, Co, H, W, K;   // K = Ci R^2
    int ph, pw;               // input row / column offset: i + a - ph, j + c - pw
    long long xs, ys;         // floats from one image to the next
    Div d_HW, d_W;
    // split over K (blockIdx.z = part): part z sums chunks [z cps, (z+1) cps)
    // and writes its raw sums to partial + z Co Q (c_out-major)
    float *partial;
    int cps;
    // flip: Wt is a (Co, Co, R, R) kernel M read transposed over channels and
    // flipped in space, W[co][ci][a][c] = M[ci][co][R-1-a][R-1-c], with the
    // entries at M's tap fself zeroed where M's input channel exceeds its
    // output channel (co > ci here): the input gradient's weights of a
    // masked convolution with kernel M.
    int flip, fself;
    // trows (R = 1 launches; 0 = off): Wt is a 3 x 3 kernel M (trows, K, 3, 3)
    // read with the taps as rows, W[t trows + c][k] = M[c][k][t]: the GEMM
    // whose nine row blocks, shifted and added, give M's convolution
    int trows;
};

constexpr int kConvThreads = 256;
constexpr long long kWideSmallGrid = 256;   // blocks: one per compute unit
constexpr int kSK = 68;     // LDS row stride (floats) of 64-value k chunks

// k values staged at a time (KC): by default 32 for the 64 c_out x 64 px
// tile (half the LDS of 64, so twice the blocks a compute unit holds: 4-19%
// faster on the flow's 1 x 1 GEMMs when the grid covers the chip), 64 for
// the narrow tiles (a block's 16 weight rows are staged by 256 threads a
// quad each).  Grids of fewer blocks than compute units take 64: there the
// chunk loop's length, not occupancy, sets the time.
template <int WCO>
constexpr int conv_kc() {
    return WCO == 4 ? 32 : 64;
}

// LDS floats of one block of the <WCO, NS, KC> configuration (rows of KC + 4
// floats).
template <int WCO, int NS, int KC = conv_kc<WCO>()>
constexpr int conv_lds_floats() {
    return (16 * WCO + 16 * NS * (4 / WCO)) * (KC + 4);
}

// One output tile (bx along pixels, by along c_out, bz the part of K) with
// the block's LDS at lds (conv_lds_floats<WCO, NS, KC>() floats, 16-byte aligned).
template <int R, int WCO, int NS, int KC = conv_kc<WCO>()>
__device__ __forceinline__ void conv_tile(const ConvArgs &a, int bx, int by, int bz, float *lds) {
    constexpr int BM = 16 * WCO, BN = 16 * NS * (4 / WCO);
    constexpr int SK = KC + 4, KQ = KC / 4;   // row stride, quads per chunk row
    constexpr int TPP = kConvThreads / BN;   // threads per staged pixel
    constexpr int QPT = KQ / TPP;            // k quads per thread (B)
    constexpr int AQ = BM * KQ / kConvThreads;   // weight quads per thread
    static_assert(QPT >= 1 && AQ >= 1, "every thread stages whole quads");
    float *As = lds, *Bs = lds + BM * SK;
    const int tid = threadIdx.x, lane = tid & 63, kq = lane >> 4, li = lane & 15;
    const int wave = tid >> 6, wco = wave % WCO, wpx = wave / WCO;
    const int co0 = by * BM;
    const int n0 = bx * BN;
    const int HW = a.H * a.W, Q = a.B * HW;

    // this thread's staged pixel and its window's validity per tap
    const int spx = tid % BN, sk0 = tid / BN;   // pixel slot; first k quad
    const int q = n0 + spx;
    const bool qok = q < Q;
    const int qb = qok ? divi(q, a.d_HW) : 0, qp = qok ? q - qb * HW : 0;
    const int qi = divi(qp, a.d_W), qj = qp - qi * a.W;
    unsigned long long tapok = 0;
#pragma unroll
    for (int t = 0; t < R * R; ++t) {
        const int ii = qi + t / R - a.ph, jj = qj + t % R - a.pw;
        if (qok && ii >= 0 && ii < a.H && jj >= 0 && jj < a.W)
            tapok |= 1ull << t;
    }
    const float *xq = a.x + (long long)qb * a.xs + qp;

    float ra[AQ][4], rb[QPT][4];
    auto load_chunk = [&](int k0) {
#pragma unroll
        for (int u = 0; u < AQ; ++u) {
            const int idx = tid + u * kConvThreads;
            const int col = idx / KQ, kk = k0 + 4 * (idx % KQ);
            const int co = co0 + col;
            const float *w = a.Wt + (long long)(co < a.Co ? co : 0) * a.K;
            long long trow = 0;   // (trows) M's row c and tap t of row co
            int ttap = 0;
            if (a.trows) {
                const int cc = co < a.Co ? co : 0;
                ttap = cc / a.trows;
                trow = (long long)(cc - ttap * a.trows) * a.K;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bool ok = co < a.Co && kk + e < a.K;
                long long off = a.trows ? (trow + kk + e) * 9 + ttap : kk + e;
                if (a.flip) {   // M[ci][co][R^2 - 1 - t], t = a R + c
                    const int ci = (int)((unsigned)(kk + e) / (R * R));
                    const int t = R * R - 1 - (kk + e - ci * R * R);
                    off = ((long long)ci * a.Co + co) * (R * R) + t;
                    ok = ok && !(t == a.fself && co > ci);
                }
                const float v = (a.flip || a.trows ? a.Wt : w)[ok ? off : 0];
                ra[u][e] = ok ? v : 0.0f;
            }
        }
#pragma unroll
        for (int u = 0; u < QPT; ++u) {
            const int kk = k0 + 4 * (sk0 + u * TPP);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k = kk + e;
                const int ci = (int)((unsigned)k / (R * R));
                const int t = k - ci * R * R;
                const int ta = t / R, tb = t - ta * R;
                const bool ok = k < a.K && ((tapok >> t) & 1ull);
                const long long off = (long long)ci * HW + (ta - a.ph) * a.W + (tb - a.pw);
                const float v = xq[ok ? off : 0];
                rb[u][e] = ok ? v : 0.0f;
            }
        }
    };
    auto store_chunk = [&] {
#pragma unroll
        for (int u = 0; u < AQ; ++u) {
            const int idx = tid + u * kConvThreads;
            *reinterpret_cast<float4 *>(&As[(idx / KQ) * SK + 4 * (idx % KQ)]) =
                make_float4(ra[u][0], ra[u][1], ra[u][2], ra[u][3]);
        }
#pragma unroll
        for (int u = 0; u < QPT; ++u)
            *reinterpret_cast<float4 *>(&Bs[spx * SK + 4 * (sk0 + u * TPP)]) =
                make_float4(rb[u][0], rb[u][1], rb[u][2], rb[u][3]);
    };

    f32x4 acc[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s)
        acc[s] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const int nall = (a.K + KC - 1) / KC;
    const int cbeg = a.partial ? bz * a.cps : 0;
    const int nchunk = a.partial ? min(a.cps, nall - cbeg) : nall;
    load_chunk(cbeg * KC);
    store_chunk();
    __syncthreads();
    const float *arow = &As[(wco * 16 + li) * SK + 4 * kq];
    const float *brow = &Bs[(wpx * 16 * NS + li) * SK + 4 * kq];
    for (int c = 0; c < nchunk; ++c) {
        if (c + 1 < nchunk)
            load_chunk((cbeg + c + 1) * KC);   // in flight during the MFMAs
#pragma unroll
        for (int blk = 0; blk < KC / 16; ++blk) {
            const float4 w4 = *reinterpret_cast<const float4 *>(arow + 16 * blk);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                const float4 b4 = *reinterpret_cast<const float4 *>(brow + 16 * s * SK + 16 * blk);
                acc[s] = mfma4(w4.x, b4.x, acc[s]);
                acc[s] = mfma4(w4.y, b4.y, acc[s]);
                acc[s] = mfma4(w4.z, b4.z, acc[s]);
                acc[s] = mfma4(w4.w, b4.w, acc[s]);
            }
        }
        if (c + 1 < nchunk) {
            __syncthreads();
            store_chunk();
            __syncthreads();
        }
    }
    if (a.partial) {   // raw sums of this part of K
        float *pz = a.partial + (long long)bz * a.Co * Q;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int qo = n0 + wpx * 16 * NS + 16 * s + li;
#pragma unroll
            for (int rr = 0; rr < 4; ++rr) {
                const int co = co0 + wco * 16 + 4 * kq + rr;
                if (qo < Q && co < a.Co)
                    pz[(long long)co * Q + qo] = acc[s][rr];
            }
        }
        return;
    }
    // epilogue: lane (kq, li) holds c_out 4 kq + rr of pixel li of each slot
    float bv[4], sv[4];
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) {
        const int co = co0 + wco * 16 + 4 * kq + rr;
        const int cc = co < a.Co ? co : 0;
        bv[rr] = a.bias ? a.bias[cc] : 0.0f;
        sv[rr] = a.ls ? expf(3.0f * a.ls[cc]) : 1.0f;
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        const int qo = n0 + wpx * 16 * NS + 16 * s + li;
        if (qo >= Q)
            continue;
        const int b = divi(qo, a.d_HW), p = qo - b * HW;
        float *yq = a.y + (long long)b * a.ys + p;
#pragma unroll
        for (int rr = 0; rr < 4; ++rr) {
            const int co = co0 + wco * 16 + 4 * kq + rr;
            if (co < a.Co) {
                float v = acc[s][rr] + bv[rr];
                if (a.relu)
                    v = fmaxf(v, 0.0f);
                yq[(long long)co * HW] = v * sv[rr];
            }
        }
    }
}

template <int R, int WCO, int NS, int KC = conv_kc<WCO>()>
__global__ __launch_bounds__(kConvThreads) void conv_kernel(ConvArgs a) {
    __shared__ __attribute__((aligned(16))) float lds[conv_lds_floats<WCO, NS, KC>()];
    conv_tile<R, WCO, NS, KC>(a, blockIdx.x, blockIdx.y, blockIdx.z, lds);
}

// The 64 x 64 tile's launch, its chunk chosen by the grid's size.
template <int R>
void launch_wide(const ConvArgs &a, dim3 grid, hipStream_t st) {
    if ((long long)grid.x * grid.y * grid.z < kWideSmallGrid)
        hipLaunchKernelGGL((conv_kernel<R, 4, 4, 64>), grid, dim3(kConvThreads), 0, st, a);
    else
        hipLaunchKernelGGL((conv_kernel<R, 4, 4, 32>), grid, dim3(kConvThreads), 0, st, a);
}

// The parts of a K-split convolution added in order (part 0 first), then
// bias, ReLU and the output scale, as the unsplit kernel's epilogue does.
__global__ __launch_bounds__(256) void conv_reduce_kernel(ConvArgs a, int parts) {
    const int Q = a.B * a.H * a.W, HW = a.H * a.W;
    const long long n = (long long)a.Co * Q;
    for (long long e = blockIdx.x * 256ll + threadIdx.x; e < n; e += (long long)gridDim.x * 256) {
        const int co = (int)(e / Q), q = (int)(e - (long long)co * Q);
        float v = 0.0f;
        for (int z = 0; z < parts; ++z)
            v += a.partial[(long long)z * n + e];
        v += a.bias ? a.bias[co] : 0.0f;
        if (a.relu)
            v = fmaxf(v, 0.0f);
        if (a.ls)
            v *= expf(3.0f * a.ls[co]);
        const int b = divi(q, a.d_HW), p = q - b * HW;
        a.y[(long long)b * a.ys + (long long)co * HW + p] = v;
    }
}

int conv_launched() { return hipGetLastError() == hipSuccess ? FINC_OK : FINC_EHIP; }

// Parts a narrow convolution's K is split into (at most; their partial sums
// take kMaxParts Co B H W floats).
constexpr int kMaxParts = 8;

// Launch of one convolution with kernel size R (a compile-time instance).
// ph, pw < 0 mean "same" padding, (R - 1) / 2.  Narrow outputs (C_out < 64)
// with a long K are split into parts of at least 8 chunks, so that the grid
// covers the chip: the number of parts depends on K only (not on the batch)
// and the parts are added in order, so results stay deterministic and
// independent of B.  partial: kMaxParts Co B H W floats, or null (no split).
// The shifted sum of the nine row blocks of a tap-rows GEMM Z (B, 9 C, H, W):
// y[b][c][i][j] = (bias[c] + sum over taps t = 3 a + d, in order, of
// Z[b][t C + c][i + a - 1][j + d - 1], zero outside) * exp(3 ls[c]).
__global__ __launch_bounds__(256) void shift_add_kernel(const float *Z, float *y, long long ys,
                                                        const float *bias, const float *ls,
                                                        int B, int C, int H, int W, Div d_HW,
                                                        Div d_W, Div d_C) {
    const int HW = H * W, n = B * C * HW;
    for (int e = blockIdx.x * 256 + threadIdx.x; e < n; e += gridDim.x * 256) {
        const int pl = divi(e, d_HW), p = e - pl * HW;
        const int b = divi(pl, d_C), c = pl - b * C;
        const int i = divi(p, d_W), j = p - i * W;
        const float *zb = Z + (long long)b * 9 * C * HW;
        float v = 0.0f;
#pragma unroll
        for (int t = 0; t < 9; ++t) {
            const int ii = i + t / 3 - 1, jj = j + t % 3 - 1;
            if (ii >= 0 && ii < H && jj >= 0 && jj < W)
                v += zb[(long long)(t * C + c) * HW + ii * W + jj];
        }
        v += bias ? bias[c] : 0.0f;
        if (ls)
            v *= expf(3.0f * ls[c]);
        y[(long long)b * ys + (long long)c * HW + p] = v;
    }
}

template <int R>
int launch_conv_r(const float *x, long long xs, float *y, long long ys, const float *Wt,
                  const float *bias, const float *ls, int relu, int B, int Ci, int Co, int H, int W,
                  int ph, int pw, hipStream_t st, float *partial) {
    if (B == 0)
        return FINC_OK;
    ConvArgs a;
    memset(&a, 0, sizeof(a));
    a.x = x;
    a.y = y;
    a.Wt = Wt;
    a.bias = bias;
    a.ls = ls;
    a.relu = relu;
    a.B = B;
    a.Ci = Ci;
    a.Co = Co;
    a.H = H;
    a.W = W;
    a.K = Ci * R * R;
    a.ph = ph < 0 ? (R - 1) / 2 : ph;
    a.pw = pw < 0 ? (R - 1) / 2 : pw;
    a.xs = xs;
    a.ys = ys;
    a.d_HW = make_div(H * W);
    a.d_W = make_div(W);
    const long long Q = (long long)B * H * W;
    if (Co >= 64) {
        const dim3 grid(cdiv(Q, 64), cdiv(Co, 64));
        launch_wide<R>(a, grid, st);
        return conv_launched();
    }
    const int nchunk = cdiv(a.K, conv_kc<1>());
    int parts = 1;
    if (partial)
        while (parts < kMaxParts && nchunk >= 16 * parts)
            parts *= 2;
    a.cps = cdiv(nchunk, parts);
    parts = cdiv(nchunk, a.cps);
    a.partial = parts > 1 ? partial : nullptr;
    const dim3 grid(cdiv(Q, 128), cdiv(Co, 16), parts);
    hipLaunchKernelGGL((conv_kernel<R, 1, 2>), grid, dim3(kConvThreads), 0, st, a);
    if (parts > 1) {
        const int rc = conv_launched();
        if (rc != FINC_OK)
            return rc;
        const long long n = (long long)Co * Q;
        hipLaunchKernelGGL(conv_reduce_kernel, dim3((unsigned)(n / 256 + 1 < 8192 ? n / 256 + 1 : 8192)),
                           dim3(256), 0, st, a, parts);
    }
    return conv_launched();
}

}  // namespace

#endif  // FINC_CONV_GEMM_H
