// finc.hip -- HIP kernels for gfx950 and the C ABI of include/finc.h.
//
// Layer (Sec. 3 conv equation, Sec. 4.1 corner padding): output pixel (i, j)
// reads input (i + a - oh, j + b - ow) through kernel position (a, b), with
// (oh, ow) the self tap: TL (k-1, k-1), TR (k-1, 0), BL (0, k-1), BR (0, 0).
// Self tap: channels c_in <= c_out only.
//
// Design (one workgroup per image, whole image resident in LDS):
//  * Activations live in LDS pixel-major with the channel axis padded to a
//    multiple of 4 (CP), so the C values a pixel needs are one contiguous,
//    16-byte aligned run.  HBM traffic is one coalesced load and one
//    coalesced store per image per launch, whatever the number of layers
//    chained inside the launch (a whole FInC unit, or a whole stack level).
//  * Inverse (Algorithm 1): the H+W-1 anti-diagonals of the corner's frame are
//    processed in order with one workgroup barrier per diagonal (Theorems 1
//    and 2); all pixels of a diagonal and all their channels are computed at
//    once.  The C-step channel chain of the self block is removed up front:
//    weights are prepared as L^-1 and L^-1 K_s (L = lower-triangular self
//    block), so x_p = L^-1 y_p - sum_s (L^-1 K_s) x_src is a plain sum.
//  * The corner variants are address arithmetic: the diagonal index is taken
//    in the corner's flipped frame (the flips of Algorithm 2 never move data).
//  * Fixed summation order per output, no atomics: results are bitwise
//    deterministic and independent of the batch size.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "finc.h"

namespace {

constexpr int kWave = 64;
constexpr int kThreads = 256;   // 4 waves, one per SIMD of a CU
constexpr int kPrepThreads = 64;
constexpr int kMaxLayersPerPrep = 64;
constexpr int kMaxLevels = 8;

__host__ __device__ inline int round_up4(int c) { return (c + 3) & ~3; }

// Self tap (= padding offsets) of a corner.
__host__ __device__ inline void self_tap(int corner, int k, int &oh, int &ow) {
    oh = (corner == FINC_TL || corner == FINC_TR) ? k - 1 : 0;
    ow = (corner == FINC_TL || corner == FINC_BL) ? k - 1 : 0;
}

// Prepared weights of one layer: k*k blocks of CP x CP floats, block s =
// a*k + b, entry [c_in][c_out]; block s_self holds L^-1 (transposed), the
// others L^-1 K_s.  Padded rows/columns are zero.
__host__ __device__ inline size_t prep_layer_floats(int C, int k) {
    const size_t cp = (size_t)round_up4(C);
    const size_t f = (size_t)k * k * cp * cp;
    return (f + 63) & ~(size_t)63;   // 256-byte multiple
}

// ---------------------------------------------------------------------------
// Weight preparation: every column of L^-1 and of L^-1 K_s is one triangular
// solve L z = rhs (forward substitution in fp64), one solve per thread.
// ---------------------------------------------------------------------------
struct PrepArgs {
    const float *K;      // n layers, OIHW each
    float *out;          // n layers, prep_layer_floats each
    int C, k, n;
    unsigned char corner[kMaxLayersPerPrep];
};

__global__ __launch_bounds__(kPrepThreads) void prep_kernel(PrepArgs a) {
    extern __shared__ double psm[];
    const int C = a.C, k = a.k, kk = k * k, CP = round_up4(C);
    const int layer = blockIdx.y;
    const int tid = threadIdx.x;
    int sh, sw;
    self_tap(a.corner[layer], k, sh, sw);
    const float *K = a.K + (size_t)layer * C * C * kk;
    float *out = a.out + (size_t)layer * prep_layer_floats(C, k);
    double *L = psm;                 // C x C, row-major, upper part zero
    double *z = psm + C * C;         // column of this thread: z[m * 64 + tid]
    for (int idx = tid; idx < C * C; idx += kPrepThreads) {
        const int co = idx / C, m = idx - co * C;
        L[idx] = (m <= co) ? (double)K[((size_t)(co * C + m) * k + sh) * k + sw] : 0.0;
    }
    __syncthreads();
    const int r = blockIdx.x * kPrepThreads + tid;   // row (s, ci) of the output
    if (r >= kk * CP)
        return;
    const int s = r / CP, ci = r - s * CP;
    float *row = out + (size_t)r * CP;
    if (ci >= C) {
        for (int co = 0; co < CP; ++co)
            row[co] = 0.0f;
        return;
    }
    const int ka = s / k, kb = s - ka * k;
    const bool is_self = (ka == sh && kb == sw);
    for (int co = 0; co < C; ++co) {
        double t = is_self ? (co == ci ? 1.0 : 0.0)
                           : (double)K[((size_t)(co * C + ci) * k + ka) * k + kb];
        for (int m = 0; m < co; ++m)
            t -= L[co * C + m] * z[m * kPrepThreads + tid];
        z[co * kPrepThreads + tid] = t / L[co * C + co];
    }
    for (int co = 0; co < CP; ++co)
        row[co] = co < C ? (float)z[co * kPrepThreads + tid] : 0.0f;
}

// ---------------------------------------------------------------------------
// log|det|: H*W*sum over layers and channels of log|K[c,c,self]| (fp64,
// fixed-order tree sum).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kWave) void logdet_kernel(const float *K, int n, int corner0,
                                                       int C, int k, int H, int W,
                                                       double *out) {
    __shared__ double red[kWave];
    const int tid = threadIdx.x;
    double v = 0.0;
    for (int q = 0; q < n; ++q) {
        int sh, sw;
        self_tap(n == 1 ? corner0 : q, k, sh, sw);
        const float *Kq = K + (size_t)q * C * C * k * k;
        for (int c = tid; c < C; c += kWave)
            v += log(fabs((double)Kq[((size_t)(c * C + c) * k + sh) * k + sw]));
    }
    red[tid] = v;
    __syncthreads();
    for (int s = kWave / 2; s > 0; s >>= 1) {
        if (tid < s)
            red[tid] += red[tid + s];
        __syncthreads();
    }
    if (tid == 0)
        out[0] = (double)H * (double)W * red[0];
}

// ---------------------------------------------------------------------------
// Shared pieces of the LDS-resident kernels.
// ---------------------------------------------------------------------------
struct Geo {
    int C, CP, H, W, k;
};

// Lane mapping: a wave is cut into groups of CP lanes, one group per pixel,
// lane c of a group computes output channel c.  All lanes of a pixel sit in
// one wave.
struct LaneMap {
    int group, c, per_wave, stride;
    bool active;
};

__device__ inline LaneMap lane_map(int CP) {
    LaneMap m;
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    m.per_wave = kWave / CP;
    m.group = lane / CP;
    m.c = lane - m.group * CP;
    m.active = m.group < m.per_wave;
    m.stride = (blockDim.x / kWave) * m.per_wave;
    m.group += wave * m.per_wave;
    return m;
}

// Contiguous run of C (padded to CP) inputs times one weight column.  The
// run is split over four accumulators (c_in mod 4), joined pairwise: four
// independent FMA chains, and a rounding error that grows with C/4 instead of
// C (a single chain over a 48-channel unit loses ~1e-4 in a round trip).
__device__ inline float dot_run(const float *__restrict__ w, const float *__restrict__ v,
                                int CP) {
    float q0 = 0.0f, q1 = 0.0f, q2 = 0.0f, q3 = 0.0f;
    for (int ci = 0; ci < CP; ci += 4) {
        const float4 x = *reinterpret_cast<const float4 *>(v + ci);
        q0 = fmaf(w[(ci + 0) * CP], x.x, q0);
        q1 = fmaf(w[(ci + 1) * CP], x.y, q1);
        q2 = fmaf(w[(ci + 2) * CP], x.z, q2);
        q3 = fmaf(w[(ci + 3) * CP], x.w, q3);
    }
    return (q0 + q1) + (q2 + q3);
}

__device__ inline void load_nchw(float *dst, const float *__restrict__ src, const Geo &g) {
    const int HW = g.H * g.W;
    for (int idx = threadIdx.x; idx < g.C * HW; idx += blockDim.x) {
        const int c = idx / HW, p = idx - c * HW;
        dst[p * g.CP + c] = src[idx];
    }
}

__device__ inline void zero_pad_channels(float *buf, const Geo &g) {
    const int pad = g.CP - g.C;
    if (!pad)
        return;
    const int HW = g.H * g.W;
    for (int idx = threadIdx.x; idx < HW * pad; idx += blockDim.x) {
        const int p = idx / pad;
        buf[p * g.CP + g.C + (idx - p * pad)] = 0.0f;
    }
}

__device__ inline void store_nchw(float *__restrict__ dst, const float *src, const Geo &g) {
    const int HW = g.H * g.W;
    for (int idx = threadIdx.x; idx < g.C * HW; idx += blockDim.x) {
        const int c = idx / HW, p = idx - c * HW;
        dst[idx] = src[p * g.CP + c];
    }
}

__device__ inline void copy_floats(float *dst, const float *__restrict__ src, size_t n) {
    const float4 *s4 = reinterpret_cast<const float4 *>(src);
    float4 *d4 = reinterpret_cast<float4 *>(dst);
    for (size_t i = threadIdx.x; i < n / 4; i += blockDim.x)
        d4[i] = s4[i];
}

// ---------------------------------------------------------------------------
// Inverse of one layer inside LDS: Y (input, pixel-major) -> X.
// ---------------------------------------------------------------------------
__device__ void solve_layer(const float *Y, float *X, const float *wl, const Geo &g,
                            int corner) {
    const int C = g.C, CP = g.CP, H = g.H, W = g.W, k = g.k;
    int oh, ow;
    self_tap(corner, k, oh, ow);
    const bool flip_h = (corner == FINC_BL || corner == FINC_BR);
    const bool flip_w = (corner == FINC_TR || corner == FINC_BR);
    const int s_self = oh * k + ow;
    const LaneMap m = lane_map(CP);
    for (int d = 0; d < H + W - 1; ++d) {
        const int i_lo = d - (W - 1) > 0 ? d - (W - 1) : 0;
        const int i_hi = d < H - 1 ? d : H - 1;
        const int npix = i_hi - i_lo + 1;
        if (m.active) {
            for (int slot = m.group; slot < npix; slot += m.stride) {
                const int ip = i_lo + slot, jp = d - ip;
                const int i = flip_h ? H - 1 - ip : ip;
                const int j = flip_w ? W - 1 - jp : jp;
                const int p = i * W + j;
                const float acc = dot_run(wl + (size_t)s_self * CP * CP + m.c, Y + p * CP, CP);
                float sub = 0.0f;
                for (int a = 0; a < k; ++a) {
                    const int ii = i + a - oh;
                    if (ii < 0 || ii >= H)
                        continue;
                    for (int b = 0; b < k; ++b) {
                        const int jj = j + b - ow;
                        if (jj < 0 || jj >= W || (a == oh && b == ow))
                            continue;
                        sub += dot_run(wl + (size_t)(a * k + b) * CP * CP + m.c,
                                       X + (ii * W + jj) * CP, CP);
                    }
                }
                X[p * CP + m.c] = m.c < C ? acc - sub : 0.0f;
            }
        }
        __syncthreads();
    }
}

// One level of an inverse chain: an input tensor, U units of `lpu` layers,
// optional actnorm^-1 before each unit.
struct Level {
    const float *z;       // top level: (B, C, H, W) input; lower: latent (B, C/2, H, W)
    const float *prep;    // n_units * lpu prepared layers
    const float *scale;   // n_units * C, or null
    const float *bias;
    int C, H, W;
};

struct InvArgs {
    Level lv[kMaxLevels];
    float *out;           // (B, C_0, H_0, W_0)
    int L, k, n_units, lpu, corner0;
};

// Inverse of a whole chain with the image resident in LDS from the first
// load to the last store.  Level l's two activation buffers sit at
// [0, A_l) and [A_l, 2 A_l) (A_l = H_l W_l CP_l floats), its weights right
// after; when going down a level the unsqueezed result is written to
// [A_l, 2 A_l), which lies beyond everything the level above used
// (2 A_{l+1} <= A_l), so the transition needs no extra space.
__global__ __launch_bounds__(kThreads) void inverse_chain_kernel(InvArgs a) {
    extern __shared__ float sm[];
    const size_t b = blockIdx.x;
    const int k = a.k;
    float *Y = sm, *X = sm;
    Geo g = {0, 0, 0, 0, 0};
    for (int l = a.L - 1; l >= 0; --l) {
        const Level lv = a.lv[l];
        const Geo gp = g;   // geometry of the level above (valid when l < L-1)
        g.C = lv.C;
        g.CP = round_up4(lv.C);
        g.H = lv.H;
        g.W = lv.W;
        g.k = k;
        const int C = g.C, CP = g.CP, H = g.H, W = g.W, HW = H * W;
        float *lo = sm, *hi = sm + (size_t)HW * CP;
        if (l == a.L - 1) {
            load_nchw(hi, lv.z + b * (size_t)C * HW, g);
        } else {
            // concat(unsqueeze(h), z_l): channel c < C/2 of pixel (i, j) is
            // channel 4c + 2(i&1) + (j&1) of the level above at (i/2, j/2).
            const int Ch = C / 2;
            const float *lat = lv.z + b * (size_t)Ch * HW;
            for (int idx = threadIdx.x; idx < Ch * HW; idx += blockDim.x) {
                const int c = idx / HW, p = idx - c * HW;
                const int i = p / W, j = p - i * W;
                const int ci = 4 * c + 2 * (i & 1) + (j & 1);
                hi[p * CP + c] = Y[((i >> 1) * gp.W + (j >> 1)) * gp.CP + ci];
                hi[p * CP + Ch + c] = lat[idx];
            }
        }
        Y = hi;
        X = lo;
        // Padded channels of the input must read as zero (the prepared weights
        // are zero there, but 0 * junk may be NaN).  X needs nothing: every
        // pixel of it, padding included, is written before it is read.
        zero_pad_channels(Y, g);
        __syncthreads();
        float *wl = sm + 2 * (size_t)HW * CP;
        const size_t lstride = prep_layer_floats(C, k);
        const size_t wfloats = (size_t)k * k * CP * CP;
        for (int u = a.n_units - 1; u >= 0; --u) {
            if (lv.scale) {
                const float *s = lv.scale + (size_t)u * C;
                const float *bi = lv.bias + (size_t)u * C;
                for (int idx = threadIdx.x; idx < HW * C; idx += blockDim.x) {
                    const int p = idx / C, c = idx - p * C;
                    Y[p * CP + c] = (Y[p * CP + c] - bi[c]) / s[c];
                }
            }
            for (int q = a.lpu - 1; q >= 0; --q) {
                copy_floats(wl, lv.prep + (size_t)(u * a.lpu + q) * lstride, wfloats);
                __syncthreads();
                solve_layer(Y, X, wl, g, a.lpu == 1 ? a.corner0 : q);
                float *t = Y;
                Y = X;
                X = t;
            }
        }
    }
    store_nchw(a.out + b * (size_t)g.C * g.H * g.W, Y, g);
}

// ---------------------------------------------------------------------------
// Forward of n layers inside LDS (n = 1: one block; n = 4: a unit).
// ---------------------------------------------------------------------------
struct FwdArgs {
    const float *in;
    float *out;
    const float *K;   // n OIHW tensors
    Geo g;
    int n, corner0;
};

__global__ __launch_bounds__(kThreads) void forward_chain_kernel(FwdArgs a) {
    extern __shared__ float sm[];
    const Geo g = a.g;
    const int C = g.C, CP = g.CP, H = g.H, W = g.W, HW = H * W, k = g.k, kk = k * k;
    float *bufA = sm;
    float *bufB = sm + HW * CP;
    float *wl = sm + 2 * HW * CP;
    const size_t b = blockIdx.x;
    const size_t img = (size_t)C * HW;
    load_nchw(bufA, a.in + b * img, g);
    zero_pad_channels(bufA, g);
    zero_pad_channels(bufB, g);
    float *Xi = bufA, *Yo = bufB;
    const LaneMap m = lane_map(CP);
    for (int q = 0; q < a.n; ++q) {
        const int corner = a.n == 1 ? a.corner0 : q;
        int oh, ow;
        self_tap(corner, k, oh, ow);
        const float *K = a.K + (size_t)q * C * C * kk;
        // weights transposed to [s][c_in][c_out] with the channel mask applied
        for (int idx = threadIdx.x; idx < kk * CP * CP; idx += blockDim.x) {
            const int s = idx / (CP * CP), r = idx - s * CP * CP;
            const int ci = r / CP, co = r - ci * CP;
            const int ka = s / k, kb = s - ka * k;
            const bool keep = ci < C && co < C && !(ka == oh && kb == ow && ci > co);
            wl[idx] = keep ? K[((size_t)(co * C + ci) * k + ka) * k + kb] : 0.0f;
        }
        __syncthreads();
        if (m.active) {
            for (int p = m.group; p < HW; p += m.stride) {
                const int i = p / W, j = p - i * W;
                float acc = 0.0f;
                for (int ka = 0; ka < k; ++ka) {
                    const int ii = i + ka - oh;
                    if (ii < 0 || ii >= H)
                        continue;
                    for (int kb = 0; kb < k; ++kb) {
                        const int jj = j + kb - ow;
                        if (jj < 0 || jj >= W)
                            continue;
                        acc += dot_run(wl + (size_t)(ka * k + kb) * CP * CP + m.c,
                                       Xi + (ii * W + jj) * CP, CP);
                    }
                }
                Yo[p * CP + m.c] = m.c < C ? acc : 0.0f;
            }
        }
        __syncthreads();
        float *t = Xi;
        Xi = Yo;
        Yo = t;
    }
    store_nchw(a.out + b * img, Xi, g);
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
bool valid_shape(int B, int C, int H, int W, int k) {
    if (B < 0 || C < 1 || C > FINC_MAX_C || H < 1 || W < 1 || k < 1 || k > FINC_MAX_K)
        return false;
    const long long n = (long long)B * C * H * W;
    return n < (1LL << 31) && (long long)H * W < (1LL << 24);
}

bool valid_corner(int corner) { return corner >= FINC_TL && corner <= FINC_BR; }

bool overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

bool aligned256(const void *p) { return ((uintptr_t)p & 255u) == 0; }

size_t inverse_lds_bytes(const InvArgs &a) {
    size_t m = 0;
    for (int l = 0; l < a.L; ++l) {
        const size_t cp = (size_t)round_up4(a.lv[l].C);
        const size_t f = 2 * (size_t)a.lv[l].H * a.lv[l].W * cp + (size_t)a.k * a.k * cp * cp;
        m = f > m ? f : m;
    }
    return m * sizeof(float);
}

size_t chain_lds_bytes(int C, int H, int W, int k) {
    const size_t cp = (size_t)round_up4(C);
    return (2 * (size_t)H * W * cp + (size_t)k * k * cp * cp) * sizeof(float);
}

size_t prep_lds_bytes(int C) {
    return ((size_t)C * C + (size_t)kPrepThreads * C) * sizeof(double);
}

// Per-workgroup LDS limit of the current device (queried once per device).
int lds_limit(size_t *out) {
    static size_t cache[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return FINC_EHIP;
    if (dev < 64 && cache[dev]) {
        *out = cache[dev];
        return FINC_OK;
    }
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
        return FINC_EHIP;
    if (dev < 64)
        cache[dev] = (size_t)v;
    *out = (size_t)v;
    return FINC_OK;
}

int check_lds(size_t need) {
    size_t lim = 0;
    const int rc = lds_limit(&lim);
    if (rc != FINC_OK)
        return rc;
    return need <= lim ? FINC_OK : FINC_EUNSUPPORTED;
}

int launched() {
    return hipGetLastError() == hipSuccess ? FINC_OK : FINC_EHIP;
}

int launch_prep(const float *K, int n, const int *corners, int C, int k, float *out,
                hipStream_t stream) {
    const int CP = round_up4(C);
    const size_t lds = prep_lds_bytes(C);
    int rc = check_lds(lds);
    if (rc != FINC_OK)
        return rc;
    for (int first = 0; first < n; first += kMaxLayersPerPrep) {
        PrepArgs a;
        memset(&a, 0, sizeof(a));
        a.C = C;
        a.k = k;
        a.n = n - first < kMaxLayersPerPrep ? n - first : kMaxLayersPerPrep;
        a.K = K + (size_t)first * C * C * k * k;
        a.out = out + (size_t)first * prep_layer_floats(C, k);
        for (int q = 0; q < a.n; ++q)
            a.corner[q] = (unsigned char)corners[first + q];
        dim3 grid((k * k * CP + kPrepThreads - 1) / kPrepThreads, a.n);
        hipLaunchKernelGGL(prep_kernel, grid, dim3(kPrepThreads), lds, stream, a);
        rc = launched();
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

int launch_inverse_chain(const InvArgs &a, int B, hipStream_t stream) {
    if (B == 0)
        return FINC_OK;
    const size_t lds = inverse_lds_bytes(a);
    int rc = check_lds(lds);
    if (rc != FINC_OK)
        return rc;
    if (hipFuncSetAttribute((const void *)inverse_chain_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        (void)hipGetLastError();   // not needed on every runtime; the launch check decides
    hipLaunchKernelGGL(inverse_chain_kernel, dim3(B), dim3(kThreads), lds, stream, a);
    return launched();
}

int launch_forward_chain(const FwdArgs &a, int B, hipStream_t stream) {
    if (B == 0)
        return FINC_OK;
    const size_t lds = chain_lds_bytes(a.g.C, a.g.H, a.g.W, a.g.k);
    int rc = check_lds(lds);
    if (rc != FINC_OK)
        return rc;
    if (hipFuncSetAttribute((const void *)forward_chain_kernel,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        (void)hipGetLastError();   // not needed on every runtime; the launch check decides
    hipLaunchKernelGGL(forward_chain_kernel, dim3(B), dim3(kThreads), lds, stream, a);
    return launched();
}

Geo make_geo(int C, int H, int W, int k) {
    Geo g;
    g.C = C;
    g.CP = round_up4(C);
    g.H = H;
    g.W = W;
    g.k = k;
    return g;
}

// x/y overlap rule of the inverse: identical or disjoint.
bool inverse_alias_ok(const void *y, const void *x, size_t bytes) {
    return x == y || !overlap(x, bytes, y, bytes);
}

size_t stack_level_bytes(int l, int U, int C1, int k) {
    return (size_t)U * 4 * prep_layer_floats(C1 << l, k) * sizeof(float);
}

bool valid_stack(int B, int L, int U, int C1, int H1, int W1, int k) {
    if (L < 1 || L > kMaxLevels || U < 0 || B < 0 || C1 < 1 || H1 < 1 || W1 < 1)
        return false;
    if (L > 1 && (C1 & 1))
        return false;
    if (((H1 | W1) & ((1 << (L - 1)) - 1)) != 0)
        return false;
    if ((long long)C1 << (L - 1) > FINC_MAX_C)
        return false;
    return valid_shape(B, C1, H1, W1, k) && valid_shape(B, C1 << (L - 1), H1 >> (L - 1),
                                                        W1 >> (L - 1), k);
}

bool stack_call_ok(const float *const *z, const float *x, const float *scale,
                   const float *bias, int B, int L, int U, int C1, int H1, int W1, int k) {
    if (!valid_stack(B, L, U, C1, H1, W1, k) || !z || !x || !scale || !bias)
        return false;
    for (int l = 0; l < L; ++l)
        if (!z[l])
            return false;
    const size_t xbytes = (size_t)B * C1 * H1 * W1 * sizeof(float);
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l, H = H1 >> l, W = W1 >> l;
        const size_t zb = (size_t)B * (l == L - 1 ? C : C / 2) * H * W * sizeof(float);
        if (overlap(z[l], zb, x, xbytes))
            return false;
    }
    return true;
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

int finc_version(void) { return 100; }

const char *finc_strerror(int status) {
    switch (status) {
    case FINC_OK: return "success";
    case FINC_EINVAL: return "invalid argument";
    case FINC_ESINGULAR: return "singular layer (zero self-tap diagonal weight)";
    case FINC_EUNSUPPORTED: return "shape not supported (per-image working set exceeds LDS)";
    case FINC_EHIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

size_t finc_workspace_bytes(int C, int k, int n_layers) {
    if (C < 1 || C > FINC_MAX_C || k < 1 || k > FINC_MAX_K || n_layers < 0)
        return 0;
    return (size_t)n_layers * prep_layer_floats(C, k) * sizeof(float);
}

int finc_prepare(const float *K, int n_layers, const int *corners, int C, int k,
                 void *prepared, hipStream_t stream) {
    if (n_layers < 0 || C < 1 || C > FINC_MAX_C || k < 1 || k > FINC_MAX_K)
        return FINC_EINVAL;
    if (n_layers == 0)
        return FINC_OK;
    if (!K || !corners || !prepared || !aligned256(prepared))
        return FINC_EINVAL;
    for (int q = 0; q < n_layers; ++q)
        if (!valid_corner(corners[q]))
            return FINC_EINVAL;
    if (overlap(K, (size_t)n_layers * C * C * k * k * sizeof(float), prepared,
                finc_workspace_bytes(C, k, n_layers)))
        return FINC_EINVAL;
    return launch_prep(K, n_layers, corners, C, k, (float *)prepared, stream);
}

int finc_forward(const float *x, float *y, const float *K, int B, int C, int H, int W,
                 int k, int corner, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !valid_corner(corner) || !x || !y || !K)
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (overlap(x, bytes, y, bytes))
        return FINC_EINVAL;
    FwdArgs a;
    a.in = x;
    a.out = y;
    a.K = K;
    a.g = make_geo(C, H, W, k);
    a.n = 1;
    a.corner0 = corner;
    return launch_forward_chain(a, B, stream);
}

int finc_logdet(const float *K, int C, int k, int corner, int H, int W, double *out,
                hipStream_t stream) {
    if (!valid_shape(1, C, H, W, k) || !valid_corner(corner) || !K || !out)
        return FINC_EINVAL;
    hipLaunchKernelGGL(logdet_kernel, dim3(1), dim3(kWave), 0, stream, K, 1, corner, C, k, H,
                       W, out);
    return launched();
}

int finc_inverse_prepared(const float *y, float *x, const void *prepared, int B, int C,
                          int H, int W, int k, int corner, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !valid_corner(corner) || !x || !y || !prepared ||
        !aligned256(prepared))
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (!inverse_alias_ok(y, x, bytes) ||
        overlap(x, bytes, prepared, finc_workspace_bytes(C, k, 1)))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    a.lv[0] = Level{y, (const float *)prepared, nullptr, nullptr, C, H, W};
    a.out = x;
    a.L = 1;
    a.k = k;
    a.n_units = 1;
    a.lpu = 1;
    a.corner0 = corner;
    return launch_inverse_chain(a, B, stream);
}

int finc_inverse(const float *y, float *x, const float *K, int B, int C, int H, int W,
                 int k, int corner, void *workspace, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !valid_corner(corner) || !x || !y || !K ||
        !workspace || !aligned256(workspace))
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t wsb = finc_workspace_bytes(C, k, 1);
    if (!inverse_alias_ok(y, x, bytes) || overlap(workspace, wsb, x, bytes) ||
        overlap(workspace, wsb, y, bytes) ||
        overlap(workspace, wsb, K, (size_t)C * C * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    const int rc = finc_prepare(K, 1, &corner, C, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_inverse_prepared(y, x, workspace, B, C, H, W, k, corner, stream);
}

int finc_unit_forward(const float *x, float *y, const float *K4, int B, int C, int H,
                      int W, int k, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !x || !y || !K4)
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (overlap(x, bytes, y, bytes) && x != y)
        return FINC_EINVAL;
    FwdArgs a;
    a.in = x;
    a.out = y;
    a.K = K4;
    a.g = make_geo(C, H, W, k);
    a.n = 4;
    a.corner0 = FINC_TL;
    return launch_forward_chain(a, B, stream);
}

int finc_unit_logdet(const float *K4, int C, int k, int H, int W, double *out,
                     hipStream_t stream) {
    if (!valid_shape(1, C, H, W, k) || !K4 || !out)
        return FINC_EINVAL;
    hipLaunchKernelGGL(logdet_kernel, dim3(1), dim3(kWave), 0, stream, K4, 4, FINC_TL, C, k,
                       H, W, out);
    return launched();
}

int finc_unit_inverse_prepared(const float *y, float *x, const void *prepared4, int B,
                               int C, int H, int W, int k, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !x || !y || !prepared4 || !aligned256(prepared4))
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (!inverse_alias_ok(y, x, bytes) ||
        overlap(x, bytes, prepared4, finc_workspace_bytes(C, k, 4)))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    a.lv[0] = Level{y, (const float *)prepared4, nullptr, nullptr, C, H, W};
    a.out = x;
    a.L = 1;
    a.k = k;
    a.n_units = 1;
    a.lpu = 4;
    a.corner0 = FINC_TL;
    return launch_inverse_chain(a, B, stream);
}

int finc_unit_inverse(const float *y, float *x, const float *K4, int B, int C, int H,
                      int W, int k, void *workspace, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !x || !y || !K4 || !workspace ||
        !aligned256(workspace))
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t wsb = finc_workspace_bytes(C, k, 4);
    if (!inverse_alias_ok(y, x, bytes) || overlap(workspace, wsb, x, bytes) ||
        overlap(workspace, wsb, y, bytes) ||
        overlap(workspace, wsb, K4, (size_t)4 * C * C * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    static const int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
    const int rc = finc_prepare(K4, 4, corners, C, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_unit_inverse_prepared(y, x, workspace, B, C, H, W, k, stream);
}

size_t finc_stack_workspace_bytes(int L, int U, int C1, int k) {
    if (L < 1 || L > kMaxLevels || U < 0 || C1 < 1 || k < 1 || k > FINC_MAX_K ||
        ((long long)C1 << (L - 1)) > FINC_MAX_C)
        return 0;
    size_t total = 0;
    for (int l = 0; l < L; ++l)
        total += stack_level_bytes(l, U, C1, k);
    return total;
}

int finc_stack_prepare(const float *K, int L, int U, int C1, int k, void *prepared,
                       hipStream_t stream) {
    if (finc_stack_workspace_bytes(L, U, C1, k) == 0 && U != 0)
        return FINC_EINVAL;
    if (L < 1 || L > kMaxLevels || (L > 1 && (C1 & 1)) || !K || !prepared ||
        !aligned256(prepared))
        return FINC_EINVAL;
    size_t koff = 0, poff = 0;
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l;
        const int n = U * 4;
        int corners[kMaxLayersPerPrep];
        for (int done = 0; done < n; done += kMaxLayersPerPrep) {
            const int cnt = n - done < kMaxLayersPerPrep ? n - done : kMaxLayersPerPrep;
            for (int q = 0; q < cnt; ++q)
                corners[q] = (done + q) & 3;
            const int rc = launch_prep(K + koff + (size_t)done * C * C * k * k, cnt, corners,
                                       C, k,
                                       (float *)((char *)prepared + poff) +
                                           (size_t)done * prep_layer_floats(C, k),
                                       stream);
            if (rc != FINC_OK)
                return rc;
        }
        koff += (size_t)n * C * C * k * k;
        poff += stack_level_bytes(l, U, C1, k);
    }
    return FINC_OK;
}

int finc_stack_inverse_prepared(const float *const *z, float *x, const void *prepared,
                                const float *scale, const float *bias, int B, int L, int U,
                                int C1, int H1, int W1, int k, hipStream_t stream) {
    if (!prepared || !aligned256(prepared) ||
        !stack_call_ok(z, x, scale, bias, B, L, U, C1, H1, W1, k))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    size_t poff = 0, soff = 0;
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l;
        a.lv[l] = Level{z[l], (const float *)((const char *)prepared + poff), scale + soff,
                        bias + soff, C, H1 >> l, W1 >> l};
        poff += stack_level_bytes(l, U, C1, k);
        soff += (size_t)U * C;
    }
    a.out = x;
    a.L = L;
    a.k = k;
    a.n_units = U;
    a.lpu = 4;
    a.corner0 = FINC_TL;
    return launch_inverse_chain(a, B, stream);
}

int finc_stack_inverse(const float *const *z, float *x, const float *K, const float *scale,
                       const float *bias, int B, int L, int U, int C1, int H1, int W1, int k,
                       void *workspace, hipStream_t stream) {
    if (!K || !workspace || !aligned256(workspace) ||
        !stack_call_ok(z, x, scale, bias, B, L, U, C1, H1, W1, k))
        return FINC_EINVAL;
    const size_t wsb = finc_stack_workspace_bytes(L, U, C1, k);
    if (overlap(workspace, wsb, x, (size_t)B * C1 * H1 * W1 * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0)
        return FINC_OK;
    const int rc = finc_stack_prepare(K, L, U, C1, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_stack_inverse_prepared(z, x, workspace, scale, bias, B, L, U, C1, H1, W1, k,
                                       stream);
}

}  // extern "C"
