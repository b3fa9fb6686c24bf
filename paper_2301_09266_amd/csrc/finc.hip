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
#include <cstddef>
#include <mutex>
#include <type_traits>

#include <stdint.h>
#include <string.h>

#include "finc.h"

// The library is one translation unit, or several compiled in parallel:
// FINC_PART = g (0 <= g < kInverseGroups) holds only the inverse kernel
// instances of group g, FINC_PART = -2 everything else.  -1, the default,
// is the single unit with everything.
#ifndef FINC_PART
#define FINC_PART -1
#endif

namespace {

constexpr int kWave = 64;
constexpr int kPrepThreads = 64;
constexpr int kMaxLayersPerPrep = 64;
constexpr int kMaxLevels = 8;

__host__ __device__ inline int round_up4(int c) { return (c + 3) & ~3; }
__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ inline int imin(int a, int b) { return a < b ? a : b; }
__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }

// Division of a non-negative int by a divisor fixed on the host, as a
// multiply-high and two shifts (Granlund and Montgomery's round-up method:
// l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1; exact for every
// 32-bit dividend).
struct FastDiv {
    unsigned m;
    int s1, s2;
};
inline FastDiv make_fastdiv(int d) {
    int l = 0;
    while ((1ull << l) < (unsigned long long)d)
        ++l;
    FastDiv f;
    f.m = (unsigned)((((1ull << l) - (unsigned long long)d) << 32) / (unsigned long long)d + 1);
    f.s1 = l < 1 ? l : 1;
    f.s2 = l > 1 ? l - 1 : 0;
    return f;
}
__device__ inline int fdiv(int x, const FastDiv &f) {
    const unsigned t = __umulhi(f.m, (unsigned)x);
    return (int)((t + (((unsigned)x - t) >> f.s1)) >> f.s2);
}

// Pins a loaded value in a register at this point, so that the compiler
// cannot move the load into the branch that uses it: a group of loads whose
// results are pinned right after they are issued costs one memory latency,
// not one per load.
template <typename T>
__device__ inline void pin(T &x) {
    asm volatile("" : "+v"(x));
}

// Threads of the workgroup: the 16-bit group size at byte 12 of the implicit
// kernel arguments (code object v5), read with one scalar load.  Every launch
// here is a whole number of workgroups, so no remainder case is needed; the
// compiler's blockDim.x covers one with a 16-bit vector load, which would
// wait behind every vector load issued before it (the image loads that go
// out first thing).
typedef __attribute__((address_space(4))) const unsigned *KernargU32;
__device__ __forceinline__ int block_threads() {
    const KernargU32 gs = (KernargU32)(
        (__attribute__((address_space(4))) const char *)__builtin_amdgcn_implicitarg_ptr() + 12);
    return (int)(*gs & 0xffffu);
}

// Word 3 of a raw buffer descriptor (gfx9 family: 32-bit data format); with
// stride 0 a load past num_records bytes returns 0 and touches no memory.
constexpr int kBufferWord3 = 0x00020000;

// Taps in the frame of a corner: back-offset (dp, dq) in [0, k-1]^2 of the
// source pixel.  They are numbered by diagonal distance dp + dq = 1, 2, ...,
// 2(k-1) (dp ascending within a distance), the self tap (0, 0) last.
__host__ __device__ inline void tap_of(int t, int K, int &dp, int &dq) {
    dp = 0;
    dq = 0;
    int n = 0;
    for (int s = 1; s <= 2 * (K - 1); ++s) {
        const int lo = s - (K - 1) > 0 ? s - (K - 1) : 0, hi = s < K - 1 ? s : K - 1;
        const int cnt = hi - lo + 1;
        if (t < n + cnt) {
            dp = lo + (t - n);
            dq = s - dp;
            return;
        }
        n += cnt;
    }
}

// tap_of for a tap number that differs across the lanes of a wave: the same
// walk over the distances with a trip count that does not (K is uniform)
// and selects in place of the early return, so the wave does not branch.
__device__ inline void tap_of_lanes(int t, int K, int &dp, int &dq) {
    dp = 0;
    dq = 0;
    int n = 0;
    for (int s = 1; s <= 2 * (K - 1); ++s) {
        const int lo = s - (K - 1) > 0 ? s - (K - 1) : 0, hi = s < K - 1 ? s : K - 1;
        const int cnt = hi - lo + 1;
        const bool here = t >= n && t < n + cnt;
        dp = here ? lo + (t - n) : dp;
        dq = here ? s - (lo + (t - n)) : dq;
        n += cnt;
    }
}

// Number of the tap with back-offset (dp, dq) (the inverse of tap_of).
__host__ __device__ inline int tap_index(int dp, int dq, int K) {
    const int d = dp + dq;
    if (d == 0)
        return K * K - 1;
    int n = 0;
    for (int s = 1; s < d; ++s)
        n += imin(s, K - 1) - imax(0, s - (K - 1)) + 1;
    return n + dp - imax(0, d - (K - 1));
}

// Self tap (= padding offsets) of a corner.
__host__ __device__ inline void self_tap(int corner, int k, int &oh, int &ow) {
    oh = (corner == FINC_TL || corner == FINC_TR) ? k - 1 : 0;
    ow = (corner == FINC_TL || corner == FINC_BL) ? k - 1 : 0;
}

// Prepared weights of one layer, in the order the inverse's MFMA operands
// take them: quad u = t ncq + cq (tap t in the corner's frame, numbered by
// tap_of; input channels 4 cq .. 4 cq + 3), then output channel co, then the
// four input channels: W[u][co][e].  The self tap holds L^-1, the others
// -(L^-1 K_s) (negated: the inverse subtracts them).  Padded channels are
// zero, and a block of 64 zero floats follows (the load address of weight
// slots that do not exist).  ncq = CP / 4.
__host__ __device__ inline size_t prep_zero_offset(int C, int k) {
    const size_t cp = (size_t)round_up4(C);
    const size_t f = (size_t)k * k * cp * cp;
    return (f + 63) & ~(size_t)63;   // 256-byte multiple
}
__host__ __device__ inline size_t prep_layer_floats(int C, int k) {
    return prep_zero_offset(C, k) + 64;
}

// ---------------------------------------------------------------------------
// Weight preparation: every column of L^-1 and of L^-1 K_s is one
// lower-triangular solve L z = rhs in fp64, one solve per thread.
// Column-oriented, in blocks of 16 channels: the block's 16 unknowns are
// solved in registers (as soon as z_c is final it is eliminated from the rows
// below, so the dependent chain is one multiply and one FMA per channel),
// written out, and eliminated from the rows of later blocks, which wait in
// LDS.  L (strictly lower part, column-major, zero-padded) and the reciprocals
// of its diagonal are staged in LDS; all threads of a block read the same
// entries (broadcast).
// ---------------------------------------------------------------------------
struct PrepArgs {
    const float *K;      // n layers, OIHW each
    float *out;          // n layers, prep_layer_floats each
    int C, k, n;
    unsigned int corner_bits[kMaxLayersPerPrep / 16];   // 2 bits per layer
};

constexpr int kPrepBlk = 16;             // unknowns solved in registers at a time
constexpr int kPrepMax = 64;             // FINC_MAX_C rounded up to kPrepBlk

__host__ __device__ inline int prep_cb(int C) { return (C + kPrepBlk - 1) / kPrepBlk * kPrepBlk; }

// LDS (doubles) of prep_columns: L's strictly lower part (CB x CB, kept in
// fp32, the precision K holds it in), the reciprocals of its diagonal (CB),
// and the rows beyond the first register block of every thread's
// right-hand side.
__host__ __device__ inline int prep_lds_doubles(int C, int nth) {
    const int cb = prep_cb(C);
    return cb * cb / 2 + cb + (cb - kPrepBlk) * nth;
}

// One block's share of one layer's preparation: output rows (columns of the
// solves) col0 .. col0 + NTH - 1, row = (kernel position s, input channel
// ci).  zero_tail: this block also writes the layer's zero block.
template <int NTH>
__device__ __forceinline__ void prep_columns(const float *__restrict__ K, float *out, int C, int k,
                                             int corner, int col0, bool zero_tail, double *lds) {
    const int kk = k * k, CP = round_up4(C), CB = prep_cb(C), tid = threadIdx.x;
    // Lt[c CB + m] = L[m][c] for m > c, else 0 (fp32: converting to fp64 is
    // exact, and a column's multipliers are read 16 bytes at a time)
    float *Lt = reinterpret_cast<float *>(lds);
    double *rinv = lds + CB * CB / 2;  // 1 / L[c][c]; 1 beyond C
    double *zs = rinv + CB;            // zs[(m - 16) NTH + thread]: rows of later blocks
    int sh, sw;
    self_tap(corner, k, sh, sw);
    const int r = col0 + tid;
    const bool row_ok = r < kk * CP;
    const int s = r / CP, ci = r - s * CP;
    const int ka = s / k, kb = s - ka * k;
    const bool is_self = (ka == sh && kb == sw);
    const bool real = row_ok && ci < C;   // padding rows stay zero
    // K through a raw buffer (32-bit offsets): entries past its C^2 k^2
    // floats read 0, so no index is clamped.  Entries of L with a channel of
    // C or more are zeroed when stored; a right-hand side of a padding row is
    // zero through rhs_val.
    const int ckk = C * kk, ss = sh * k + sw;   // row stride of K's output channel; self tap
    const unsigned nrec = (unsigned)(C * ckk * 4);
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(K), (short)0, (int)nrec, kBufferWord3);
    auto kat = [&](int off) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rk, off, 0, 0));
    };
    auto Kself = [&](int m, int c) { return kat(((m * C + c) * kk + ss) * 4); };
    // Staging: every load of a round is issued before the round's stores, so
    // a round costs one memory latency; the first round holds the first 16
    // right-hand-side rows (kept in registers), U entries of L per thread and
    // the diagonal (all of it for C <= 16).
    constexpr int U = 8;
    const int rbase = real ? (ci * kk + ka * k + kb) * 4 : (int)nrec;   // rhs(m) at rbase + m ckk 4
    auto rhs = [&](int m) { return kat(rbase + m * ckk * 4); };
    auto rhs_val = [&](int m, float v) {
        return (m < C && real) ? (is_self ? (m == ci ? 1.0 : 0.0) : (double)v) : 0.0;
    };
    // entry idx = c CB + m of L's staging (column c, row m), stepped by NTH
    // from this thread's first one without a division per entry
    const int dc = NTH / CB, dm = NTH - dc * CB;
    int lc = tid / CB, lm = tid - lc * CB;
    auto lstep = [&](int &c, int &m) {
        c += dc;
        m += dm;
        if (m >= CB) {
            m -= CB;
            c += 1;
        }
    };
    auto put_l = [&](int c, int m, float v) {
        if (c < CB)
            Lt[c * CB + m] = (m > c && m < C) ? v : 0.0f;
    };
    double z[kPrepBlk];
    {
        float rv[kPrepBlk], lv[U];
        int cs[U], ms[U];
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            rv[u] = rhs(u);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            cs[u] = lc;
            ms[u] = lm;
            lv[u] = Kself(lm, lc);
            lstep(lc, lm);
        }
        float dv = Kself(tid, tid);
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            pin(rv[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            pin(lv[u]);
        pin(dv);
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            z[u] = rhs_val(u, rv[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            put_l(cs[u], ms[u], lv[u]);
        if (tid < CB)
            rinv[tid] = tid < C ? 1.0 / (double)dv : 1.0;
    }
    while (lc < CB) {
        float v[U];
        int cs[U], ms[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            cs[u] = lc;
            ms[u] = lm;
            v[u] = Kself(lm, lc);
            lstep(lc, lm);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            pin(v[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            put_l(cs[u], ms[u], v[u]);
    }
    for (int base = kPrepBlk; base < CB; base += kPrepBlk) {
        float v[kPrepBlk];
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            v[u] = rhs(base + u);
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            pin(v[u]);
#pragma unroll
        for (int u = 0; u < kPrepBlk; ++u)
            zs[(base + u - kPrepBlk) * NTH + tid] = rhs_val(base + u, v[u]);
    }
    __syncthreads();
    // kernel position (ka, kb) is back-offset (|ka - sh|, |kb - sw|) in the
    // corner's frame; this thread's column is element ci % 4 of quad
    // u = t ncq + ci / 4, for every output channel
    const double sg = is_self ? 1.0 : -1.0;
    const int t = tap_index(ka > sh ? ka - sh : sh - ka, kb > sw ? kb - sw : sw - kb, k);
    float *dst = out + ((size_t)(t * (CP / 4) + (ci >> 2)) * CP) * 4 + (ci & 3);
    for (int b0 = 0; b0 < CB; b0 += kPrepBlk) {
        if (b0 > 0) {
#pragma unroll
            for (int i = 0; i < kPrepBlk; ++i)
                z[i] = zs[(b0 + i - kPrepBlk) * NTH + tid];
        }
#pragma unroll
        for (int c = 0; c < kPrepBlk; ++c) {
            z[c] *= rinv[b0 + c];
            // column c's multipliers of rows b0 .. b0 + 15 (16-byte aligned:
            // CB and b0 are multiples of 16), read ahead of their use
            const float4 *lc = reinterpret_cast<const float4 *>(Lt + (b0 + c) * CB + b0);
            float lv[kPrepBlk];
#pragma unroll
            for (int q = c / 4; q < kPrepBlk / 4; ++q) {
                const float4 v = lc[q];
                lv[4 * q] = v.x;
                lv[4 * q + 1] = v.y;
                lv[4 * q + 2] = v.z;
                lv[4 * q + 3] = v.w;
            }
#pragma unroll
            for (int m = c + 1; m < kPrepBlk; ++m)
                z[m] -= (double)lv[m] * z[c];
        }
        if (row_ok) {
#pragma unroll
            for (int i = 0; i < kPrepBlk; ++i)
                if (b0 + i < CP)
                    dst[4 * (b0 + i)] = (float)(sg * z[i]);
        }
        for (int m = b0 + kPrepBlk; m < CB; ++m) {
            double acc = zs[(m - kPrepBlk) * NTH + tid];
#pragma unroll
            for (int c = 0; c < kPrepBlk; ++c)
                acc -= (double)Lt[(b0 + c) * CB + m] * z[c];
            zs[(m - kPrepBlk) * NTH + tid] = acc;
        }
    }
    if (zero_tail && tid < 16)
        reinterpret_cast<float4 *>(out + prep_zero_offset(C, k))[tid] =
            make_float4(0.0f, 0.0f, 0.0f, 0.0f);
}

#if FINC_PART < 0
__global__ __launch_bounds__(kPrepThreads) void prep_kernel(PrepArgs a) {
    __shared__ double lds[kPrepMax * kPrepMax + kPrepMax + (kPrepMax - kPrepBlk) * kPrepThreads];
    const int layer = blockIdx.y;
    const unsigned int cw = layer < 16   ? a.corner_bits[0]
                            : layer < 32 ? a.corner_bits[1]
                            : layer < 48 ? a.corner_bits[2]
                                         : a.corner_bits[3];
    prep_columns<kPrepThreads>(a.K + (size_t)layer * a.C * a.C * a.k * a.k,
                               a.out + (size_t)layer * prep_layer_floats(a.C, a.k), a.C, a.k,
                               (cw >> (2 * (layer & 15))) & 3, blockIdx.x * kPrepThreads,
                               blockIdx.x == 0, lds);
}
#endif

// ---------------------------------------------------------------------------
// log|det|: H*W*sum over layers and channels of log|K[c,c,self]| (fp64,
// fixed-order tree sum).
// ---------------------------------------------------------------------------
#if FINC_PART < 0
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
#endif

// ---------------------------------------------------------------------------
// Inverse (Algorithm 1) as an MFMA wavefront.
//
// One workgroup per image; the image stays in LDS for the whole chain of
// layers.  Per layer, with frames flipped so that every corner reads "up and
// to the left" (the flips of Algorithm 2 become address arithmetic):
//
//   x[p] = L^-1 y[p] - sum_{(dp,dq) != 0} (L^-1 K_(dp,dq)) x[p - (dp,dq)]
//
// where (dp, dq) in [0, k-1]^2 is the back-offset of a kernel position.  A
// pixel on anti-diagonal e reads diagonals e - (dp + dq); only the two taps
// with dp + dq = 1 read the diagonal solved in the previous step.  Every step
// is a small dense contraction per tile of 16 output channels x 16 frame rows
//     D[c_out][row] += A[c_out][k] * B[k][row]
// over k = (tap, input channel), issued as v_mfma_f32_16x16x4_f32: the
// prepared weights are the A operand, held in registers; the inputs are the B
// operand, gathered from LDS one 16-byte channel quad per lane.
//
// The k range is cut into "quads" (one tap, four input channels), four quads
// to a group (one group = four MFMAs).  Per tile one critical wave owns the
// two dp + dq = 1 taps and finishes diagonal e.  S helper waves own the rest,
// round-robin by group: "fresh" groups (dp + dq = 2, which read diagonal
// e - 1) and "stale" groups (dp + dq >= 3, and the L^-1 y term).  During step
// e a helper computes its share of diagonal e + 1 and leaves it as a partial
// tile in LDS.  One barrier per diagonal step (Theorems 1 and 2: H + W - 1
// steps).
//
// With a single channel tile the critical wave keeps its rows' previous
// pixels in its accumulator: its MFMA chain for diagonal e starts right after
// the barrier from registers (own row, and the row above by a DPP lane shift)
// while the partial tiles are read, which are added last.
//
// LDS per level: X, the solution, with a zero border of k-1 pixels on every
// side (the padded image of the paper's padding equation: out-of-image taps
// read zeros, so gathers never branch); Y, the layer input, unpadded; R, the
// partial tiles (two parities); Z, a zero block; T, a trash block for writes
// of rows that must not land.  All pixel-major with the channel axis padded
// to CP = 4 * ceil(C / 4).
// ---------------------------------------------------------------------------
typedef float f32x4 __attribute__((ext_vector_type(4)));



constexpr int kMaxWaves = 16;
constexpr size_t kLdsBytes = 160 * 1024;   // LDS of a gfx950 workgroup
constexpr int kMaxGroups = 8;                       // quad groups (x4 quads) per wave
// critical-wave forms an inverse instance is built with (low two bits of
// its MODE), and kOneLayer: a single level of a single layer without actnorm
// (the chain's loops and hand-overs compiled out)
constexpr int kCritGather = 0, kCritRegs = 1, kOneLayer = 4;
// kStream (with kOneLayer and kCritRegs): a single layer whose image does not
// fit in LDS.  Solution and input live in per-row rings of kRing frame
// columns; every kPhase diagonal steps the workgroup drains the solved
// columns to HBM, writes the input of the next kPhase diagonals (loaded a
// phase earlier into registers) and issues the loads of the phase after.
constexpr int kStream = 8;
// (with kStream) the banded stream form: the workgroup is one band of rows
// of an image, pipelined with the bands above and below through global
// progress counts (instances of their own: the counts and the border rows
// cost registers the plain stream form does not pay)
constexpr int kBanded = 16;
constexpr int kRing = 32, kPhase = 16;
constexpr int kStreamRegs = 8;   // prefetched input values per thread
// a single layer in LDS stores its rows as they complete when a row has at
// most kDrainRounds * 64 values (one value per lane and round)
constexpr int kDrainRounds = 8;

// Work split and LDS layout of one level (same for every layer of it).
struct Plan {
    int C, CP, H, W, K, P, WP;
    int MT, NT, T, S, S4, NW;   // row tiles, channel tiles, tiles, helpers per tile,
                                // partial-tile slots read per tile (S rounded up
                                // to 4), waves
    // partial tiles stored per tile: S4 (padded; slots from S on stay zero),
    // or S with one shared zero slot per parity (compact, when the padded
    // layout would not fit in LDS)
    int RS, compact;
    // stream: X holds frame rows -P .. H-1 and Y rows 0 .. H-1, each as a
    // ring of kRing frame columns (frame orientation, no border columns)
    int stream;
    int ncq, nq, nq_crit;       // quads per tap, quads of a tile, quads of the critical wave
    int fq0, fq1;               // fresh quads [fq0, fq1); stale quads [fq1, nq)
    int FG, SG;                 // fresh and stale groups of a tile's helpers
    int regcrit;                // 1: the critical taps are fed from registers (one channel tile)
    int offX, offY, offR, offZ, offT;  // LDS offsets (floats): solution, input, partial
                                       // tiles, zero block, trash block
    int lds_floats;
    int lstride;                // floats of one prepared layer
    int wave[kMaxWaves];        // per wave: role | mt << 2 | nt << 6 | h << 10 | groups << 14
    // divisions of the index arithmetic: CP / 4, W, H W / 4, H W, CP - C,
    // C, CP, W / 4, ncq (divisors below 1 are replaced by 1)
    FastDiv d_cp4, d_W, d_hw4, d_HW, d_pad, d_C, d_CP, d_w4, d_ncq, d_H;
};

// Quad groups of the busiest wave of a plan.
inline int plan_groups(const Plan &p) {
    const int crit = p.regcrit ? 2 : ceil_div(p.nq_crit, 4);
    return imax(crit, ceil_div(p.FG + p.SG, p.S));
}

// false if the shape needs more waves or registers than a workgroup has
// (stream: the ring layout; also false when a phase's input does not fit in
// the threads' prefetch registers)
inline bool make_plan(int C, int H, int W, int K, Plan &p, bool stream = false) {
    p.stream = stream ? 1 : 0;
    p.C = C;
    p.CP = round_up4(C);
    p.H = H;
    p.W = W;
    p.K = K;
    p.P = K - 1;
    p.WP = W + 2 * p.P;
    p.MT = ceil_div(H, 16);
    p.NT = ceil_div(p.CP, 16);
    p.T = p.MT * p.NT;
    p.ncq = p.CP / 4;
    p.nq = K * K * p.ncq;
    // With one channel tile the critical wave holds, in its accumulator, all
    // channels of its rows' previous pixels: the two dp + dq = 1 taps need no
    // gather.  Otherwise it gathers them (padded to whole quad groups).
    p.regcrit = (p.NT == 1 && K >= 2) ? 1 : 0;
    p.nq_crit = K < 2 ? 0 : (p.regcrit ? 2 * p.ncq : imin(p.nq, round_up4(2 * p.ncq)));
    // taps up to distance 2: the two of distance 1 and (k = 2) one or three
    // of distance 2
    const int taps2 = K < 2 ? 0 : (K == 2 ? 3 : 5);
    p.fq0 = p.nq_crit;
    p.fq1 = imax(p.nq_crit, imin(p.nq, taps2 * p.ncq));
    p.FG = ceil_div(p.fq1 - p.fq0, 4);
    p.SG = ceil_div(p.nq - p.fq1, 4);
    const int s_max = kMaxWaves / p.T - 1;
    if (s_max < 1)
        return false;
    // every fresh group on its own helper when possible, and about two
    // groups a helper
    p.S = imax(1, imin(s_max, imax(p.FG, ceil_div(p.FG + p.SG, 2))));
    if (plan_groups(p) > kMaxGroups)
        return false;
    const int nwork = p.T * (1 + p.S);   // critical and helper waves
    p.NW = nwork;
    p.S4 = round_up4(p.S);
    p.offX = 0;
    if (stream) {
        // one phase's input is prefetched, kStreamRegs values a thread:
        // idle waves join the workgroup for it when the working ones are
        // too few
        const int need = ceil_div(kPhase * H * C, kStreamRegs * kWave);
        if (!p.regcrit || need > kMaxWaves)
            return false;
        p.NW = imax(p.NW, need);
        p.offY = (H + p.P) * kRing * p.CP;
        p.offR = p.offY + H * kRing * p.CP;
    } else {
        p.offY = (H + 2 * p.P) * p.WP * p.CP;
        p.offR = p.offY + H * W * p.CP;
    }
    for (p.compact = 0; p.compact < 2; ++p.compact) {
        p.RS = p.compact ? p.S : p.S4;
        p.offZ = p.offR + 2 * (p.T * p.RS + p.compact) * 256;
        p.offT = p.offZ + 256;
        p.lds_floats = p.offT + 256;
        if ((size_t)p.lds_floats * sizeof(float) <= kLdsBytes || p.RS == p.S)
            break;
    }
    p.lstride = (int)prep_layer_floats(C, K);
    p.d_cp4 = make_fastdiv(p.CP / 4);
    p.d_W = make_fastdiv(W);
    p.d_hw4 = make_fastdiv(imax(H * W / 4, 1));
    p.d_HW = make_fastdiv(H * W);
    p.d_pad = make_fastdiv(imax(p.CP - C, 1));
    p.d_C = make_fastdiv(C);
    p.d_CP = make_fastdiv(p.CP);
    p.d_w4 = make_fastdiv(imax(W / 4, 1));
    p.d_ncq = make_fastdiv(p.ncq);
    p.d_H = make_fastdiv(H);
    // wave roles: critical waves of the tiles first, then S helpers per tile,
    // then idle waves; with the number of quad groups each one owns
    for (int w = 0; w < kMaxWaves; ++w) {
        int role = 2, tile = 0, h = 0, ng = 0;
        if (w < p.T) {
            role = 0;
            tile = w;
            ng = p.regcrit ? 2 : ceil_div(p.nq_crit, 4);
        } else if (w < nwork) {
            role = 1;
            tile = (w - p.T) / p.S;
            h = (w - p.T) - tile * p.S;
            ng = h < p.FG + p.SG ? ceil_div(p.FG + p.SG - h, p.S) : 0;
        }
        p.wave[w] = role | (tile % p.MT) << 2 | (tile / p.MT) << 6 | h << 10 | ng << 14;
    }
    return true;
}

__device__ inline f32x4 mfma4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// One level of an inverse chain: an input tensor, U units of `lpu` layers,
// optional actnorm^-1 before each unit.
struct Level {
    const float *z;       // top level: (B, C, H, W) input; lower: latent (B, C/2, H, W)
    const float *prep;    // n_units * lpu prepared layers
    const float *scale;   // n_units * C, or null
    const float *bias;
    Plan pl;
};

struct InvArgs {
    int L, n_units, lpu, corner0;
    // stamps (diagnostic, single-level calls only; null otherwise): lane 0 of
    // wave w of workgroup b writes stamps[(b * waves + w) * 4 + i], the
    // 100 MHz constant clock at i = 0 the wave's arguments loaded (and its
    // first image loads issued), 1 its set-up done (before the first step
    // barrier), 2 its last step done, 3 its part of the store issued.  (In the
    // first argument line, which the kernel's first round of loads brings.)
    long long *stamps;
    // split: the channel-split unit, its batch seen as (4B, C/4, H, W): the
    // workgroup of image b' = 4 b + g inverts quarter g with corner g and the
    // g-th prepared layer (one level of one layer)
    int split;
    // vec bit 0: the top level's input may be read 16 bytes at a time (H W a
    // multiple of 4, z 16-byte aligned); bit 1: the output may be written so
    // (the last level's W a multiple of 4, out 16-byte aligned)
    int vec;
    float *out;           // output of the last level: (B, C, H, W)
    int out_stride;       // floats from one image's output to the next (C H W when packed)
    // hin (chains that start below the top of a stack): the first level's
    // input is concat(unsqueeze(h), z), h being the level above's solution,
    // (2C, H/2, W/2) per image, hin_stride floats apart
    const float *hin;
    int hin_stride;
    // drain (a single layer held in LDS): 1 + the index of an idle wave that
    // stores each row of the solution as soon as its last pixel is solved, so
    // that the store after the last diagonal is one row; 0: none (the whole
    // image is stored after the last diagonal)
    int drain;
    Level lv[kMaxLevels]; // in the order they run
    // steps (diagnostic, single-level calls only; null otherwise): lane 0 of
    // wave w of workgroup b writes steps[b * waves + w] = the number of
    // diagonal steps (each ended by the step barrier) that wave ran
    int *steps;
    // banded stream form (0 bands otherwise): an image's frame rows cut into
    // bands of the plan's H rows, one workgroup each, img_H rows in all;
    // bflags = [timeout flag, ticket, diagonals drained per (image, band)],
    // zeroed before the launch
    int nbands, img_H;
    int *bflags;
};
static_assert(sizeof(InvArgs) <= 4096, "kernel arguments are limited to 4 KB");

// Spins of a band's wait for the band above before it gives up, sets the
// timeout flag and goes on (about a second; the wait is never that long
// when the band above runs)
constexpr int kBandSpin = 1 << 20;

// What one wave does at a level.  role 0: critical wave of `tile`; 1: helper
// h of `tile`; 2: idle (barriers only).
struct Role {
    int role, tile, mt, nt, h, ng;   // tile = nt * MT + mt; ng: quad groups the wave owns
};

__device__ inline int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// (diagnostic) stamp i of this wave of workgroup b, when asked for.  The
// clock is read only then: its scalar read would hold up the next wait for
// LDS operations.
__device__ inline void stamp(long long *stamps, size_t b, int i) {
    if (stamps) {
        // (wave-uniform address arithmetic: nothing the compiler moves ahead
        // of the test touches a vector register)
        const long long t = __builtin_amdgcn_s_memrealtime();
        const size_t slot = (b * (size_t)(block_threads() >> 6) + (size_t)wave_id()) * 4 + i;
        if ((threadIdx.x & 63) == 0)
            stamps[slot] = t;
    }
}

// This wave's role at level i (from the table the host filled in).
__device__ inline Role role_of(const InvArgs &a, int i) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int c = a.lv[i].pl.wave[wave];
    const int mt = (c >> 2) & 15, nt = (c >> 6) & 15;
    return Role{c & 3, nt * a.lv[i].pl.MT + mt, mt, nt, (c >> 10) & 15, (c >> 14) & 15};
}

// Quad that lane group kq of group g of a wave covers, or -1.  Critical wave
// (gathering form): quads 4 g + kq of [0, nq_crit).  Helper h: groups
// h, h + S, h + 2S, ... of the tile's fresh groups followed by its stale
// groups, so a helper's fresh groups come first.
__device__ inline int quad_of(const Plan &pl, const Role &r, int g, int kq) {
    if (r.role == 0) {
        const int u = 4 * g + kq;
        return u < pl.nq_crit ? u : -1;
    }
    if (r.role != 1)
        return -1;
    const int G = r.h + g * pl.S;
    if (G < pl.FG) {
        const int u = pl.fq0 + 4 * G + kq;
        return u < pl.fq1 ? u : -1;
    }
    const int u = pl.fq1 + 4 * (G - pl.FG) + kq;
    return G < pl.FG + pl.SG && u < pl.nq ? u : -1;
}

__device__ inline int corner_of(const InvArgs &a, int q) { return a.lpu == 1 ? a.corner0 : q; }

// Row order of the register-fed critical path's tiles (one channel tile of
// CP = 4 EQ channels, EQ = ncq): accumulator row 4 kq + e (lane group kq,
// register e) holds channel EQ kq + e for e < EQ, and rows with e >= EQ are
// empty.  The channels then fill registers 0 .. EQ-1 of every lane group,
// so a tap's contraction over the previous diagonal's channels, fed from
// those registers, takes EQ MFMAs instead of 4.  Returns the channel of row
// m, or -1.
__host__ __device__ inline int crit_row(int m, int eq) {
    return (m & 3) < eq ? eq * (m >> 2) + (m & 3) : -1;
}

// The A operands (prepared weights) of this lane's quads for one layer: lane
// (kq, li) holds, for group g and element e, the weight of input channel
// 4 (u % ncq) + e of quad u = quad_of(g, kq) into output channel 16 nt + li --
// one 16-byte load per group.  Nothing is computed on the loaded values, so
// the wait for them sinks to their first use (slots that do not exist read
// the zero block of the prepared layer).
template <int NG>
__device__ inline void load_weights(float (&w)[NG][4], const Plan &pl, const Role &r,
                                    const float *__restrict__ prep, bool perm) {
    const int lane = threadIdx.x & 63, kq = lane >> 4, li = lane & 15;
    // output channel of A row li: 16 nt + li, or (perm: the tile's critical
    // wave is register-fed) the row order of crit_row
    const int co = perm ? crit_row(li, pl.ncq) : r.nt * 16 + li;
    // raw buffer loads over the prepared layer: slots that do not exist read
    // past its end, which returns 0 (one 32-bit offset per load, no branch)
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(prep), (short)0, pl.lstride * 4, kBufferWord3);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
        const int u = quad_of(pl, r, g, kq);
        const bool valid = u >= 0 && co >= 0 && co < pl.C;
        // (four 32-bit loads: this compiler lowers the 128-bit raw buffer
        // load builtin to a 32-bit load)
        const int off = valid ? (u * pl.CP + co) * 16 : pl.lstride * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            w[g][e] = __builtin_bit_cast(float,
                                         __builtin_amdgcn_raw_buffer_load_b32(rs, off + 4 * e, 0, 0));
    }
}

// Weights of the register-fed critical path (one channel tile): group t is
// tap t of the quad order ((0,1), then (1,0)); lane (kq, li) holds, for
// element e < EQ = ncq, the weight of input channel EQ kq + e into output
// channel crit_row(li) (A operand; 0 where either does not exist).
template <int NG>
__device__ inline void load_crit_weights(float (&w)[NG][4], const Plan &pl,
                                         const float *__restrict__ prep) {
    const int lane = threadIdx.x & 63, kq = lane >> 4, li = lane & 15;
    const int eq = pl.ncq, o = crit_row(li, eq);
    // raw buffer loads over the prepared layer; weights that do not exist
    // read past its end, which returns 0
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(prep), (short)0, pl.lstride * 4, kBufferWord3);
#pragma unroll
    for (int t = 0; t < (NG < 2 ? NG : 2); ++t) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int c = eq * kq + e;
            const bool valid = o >= 0 && o < pl.C && e < eq && c < pl.C;
            const int at = (((t * pl.ncq + (c >> 2)) * pl.CP + o) << 2) + (c & 3);
            w[t][e] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rs, valid ? 4 * at : pl.lstride * 4,
                                                             0, 0));
        }
    }
}

// float4 copies / fills by all threads, four in flight per thread
__device__ inline void zero_floats(float *dst, int n) {   // n multiple of 4, dst 16B aligned
    float4 *d4 = reinterpret_cast<float4 *>(dst);
    const float4 z = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int i = threadIdx.x; i < n / 4; i += block_threads())
        d4[i] = z;
}

// X interior -> Y (both pixel-major, CP channels)
__device__ inline void copy_solution(float *sm, const Plan &pl) {
    const int n4 = pl.H * pl.W * pl.CP / 4, cp4 = pl.CP / 4;
    float4 *Y = reinterpret_cast<float4 *>(sm + pl.offY);
    const float4 *X = reinterpret_cast<const float4 *>(sm + pl.offX);
    for (int idx = threadIdx.x; idx < n4; idx += block_threads()) {
        const int p = fdiv(idx, pl.d_cp4), c4 = idx - p * cp4;
        const int i = fdiv(p, pl.d_W), j = p - i * pl.W;
        Y[idx] = X[((i + pl.P) * pl.WP + j + pl.P) * cp4 + c4];
    }
}

// Load the top level's input (B, C, H, W) -> Y, pixel-major, padded channels
// 0.  With vec4 (H W a multiple of 4 and src 16-byte aligned), a thread
// takes a block of four pixels by
// four channels (one channel quad): four 16-byte loads, one per channel,
// coalesced across the lanes, transposed in registers into four 16-byte LDS
// stores, one per pixel.  Otherwise it takes one pixel's channel quad (four
// scalar loads, one LDS store).  All of a thread's loads are in flight before
// the first store; `during` (work that does not touch Y) runs while the
// first round of loads is in flight.
// The first round of a thread's input loads (below), issued on their own:
// single-layer inverses issue them right after the kernel's arguments arrive,
// so that the set-up of the roles, weights and addresses runs under their
// latency.  Always the one-pixel form (slot u: channels 4 cq .. +3 of pixel
// p): each load lands in the register quad its 16-byte LDS store reads, so
// nothing between the issue and the store waits for the loads.  Raw buffer
// loads over the image's C H W floats: a 32-bit offset per load, and reads
// past the image (padding channels, threads without a slot) return 0.
struct InputRound {
    float s[4][4];
};
__device__ __forceinline__ void input_issue(const Plan &pl, const float *__restrict__ src,
                                            int tid, InputRound &q) {
    const int HW = pl.H * pl.W;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float *>(src), (short)0, pl.C * HW * 4, kBufferWord3);
    const int nthr = block_threads();
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int idx = tid + u * nthr;
        const int cq = fdiv(idx, pl.d_HW), p = idx - cq * HW;
        const int off = (4 * cq * HW + p) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            q.s[u][e] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(rs, off + e * HW * 4, 0, 0));
    }
}

// PRE: the first round was issued by input_issue into q (the one-pixel form
// then serves every round).
template <bool PRE, typename F>
__device__ __forceinline__ void load_input(float *sm, const Plan &pl,
                                           const float *__restrict__ src, bool vec4, F during,
                                           const InputRound &q) {
    const int HW = pl.H * pl.W, CP = pl.CP, C = pl.C, nq = CP / 4;
    float *Y = sm + pl.offY;
    auto pad0 = [&](float4 w, int cq) {   // padding channels are zero
        if (4 * cq + 3 >= C) {
            w.x = 4 * cq < C ? w.x : 0.0f;
            w.y = 4 * cq + 1 < C ? w.y : 0.0f;
            w.z = 4 * cq + 2 < C ? w.z : 0.0f;
            w.w = 0.0f;
        }
        return w;
    };
    if (vec4 && !PRE) {
        const int total = nq * (HW / 4);   // (pixel group, quad), quad fastest
        const float4 *s4 = reinterpret_cast<const float4 *>(src);
        constexpr int U = 2;
        // one round: the loads of slots u of base, `during` after the first,
        // then the transposed LDS stores
        auto round = [&](int base, auto first) {
            float4 v[U][4];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                const int pg = fdiv(idx, pl.d_cp4), cq = idx - pg * nq;
                const bool in = idx < total;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int c = 4 * cq + e;
                    v[u][e] = s4[in && c < C ? (size_t)c * (HW / 4) + pg : 0];
                }
            }
            if constexpr (decltype(first)::value)
                during();
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                if (idx < total) {
                    const int pg = fdiv(idx, pl.d_cp4), cq = idx - pg * nq;
                    *reinterpret_cast<float4 *>(Y + (size_t)(4 * pg + 0) * CP + 4 * cq) =
                        pad0(make_float4(v[u][0].x, v[u][1].x, v[u][2].x, v[u][3].x), cq);
                    *reinterpret_cast<float4 *>(Y + (size_t)(4 * pg + 1) * CP + 4 * cq) =
                        pad0(make_float4(v[u][0].y, v[u][1].y, v[u][2].y, v[u][3].y), cq);
                    *reinterpret_cast<float4 *>(Y + (size_t)(4 * pg + 2) * CP + 4 * cq) =
                        pad0(make_float4(v[u][0].z, v[u][1].z, v[u][2].z, v[u][3].z), cq);
                    *reinterpret_cast<float4 *>(Y + (size_t)(4 * pg + 3) * CP + 4 * cq) =
                        pad0(make_float4(v[u][0].w, v[u][1].w, v[u][2].w, v[u][3].w), cq);
                }
            }
        };
        int base = threadIdx.x;
        if (base < total) {
            round(base, std::true_type{});
            base += U * block_threads();
        } else {
            during();   // this thread had nothing to load
        }
        for (; base < total; base += U * block_threads())
            round(base, std::false_type{});
    } else {
        const int total = nq * HW;   // (quad, pixel), pixel fastest
        constexpr int U = 4;
        // one round: slots u of base (loads, or the prefetched first round),
        // `during` after the first, then the LDS stores
        auto round = [&](int base, auto pre, auto first) {
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                const int cq = fdiv(idx, pl.d_HW), p = idx - cq * HW;
                const bool in = idx < total;
                if constexpr (decltype(pre)::value) {
                    v[u] = make_float4(q.s[u][0], q.s[u][1], q.s[u][2], q.s[u][3]);
                } else {
                    float t[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int c = 4 * cq + e;
                        t[e] = src[in && c < C ? (size_t)c * HW + p : 0];
                    }
                    v[u] = make_float4(t[0], t[1], t[2], t[3]);
                }
            }
            if constexpr (decltype(first)::value)
                during();
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                if (idx < total) {
                    const int cq = fdiv(idx, pl.d_HW), p = idx - cq * HW;
                    *reinterpret_cast<float4 *>(Y + (size_t)p * CP + 4 * cq) = pad0(v[u], cq);
                }
            }
        };
        int base = threadIdx.x;
        if (PRE || base < total) {
            round(base, std::integral_constant<bool, PRE>{}, std::true_type{});
            base += U * block_threads();
        } else {
            during();   // this thread had nothing to load
        }
        for (; base < total; base += U * block_threads())
            round(base, std::false_type{}, std::false_type{});
    }
}

// Input of level l: the chain's input at the top; below, concat(unsqueeze(h),
// z_l) where h is the level above's solution, still in LDS: channel c < C/2
// of pixel (i, j) is channel 4c + 2(i&1) + (j&1) of h at (i/2, j/2).  Then
// the solution buffer (with its zero border) and the zero block are cleared.
// `work` (register-only set-up) runs while the top level's input is on its
// way.
template <bool HIN, bool PRE, typename F>
__device__ __forceinline__ void level_input(const Level &lv, bool top, const Plan &up, float *sm,
                                            size_t b, bool vec4, const float *hin,
                                            int hin_stride, F work, const InputRound &q) {
    const Plan &pl = lv.pl;
    const int C = pl.C, CP = pl.CP, W = pl.W, HW = pl.H * pl.W;
    float *Y = sm + pl.offY;
    auto clear = [&] {
        zero_floats(sm + pl.offX, pl.offY - pl.offX);
        zero_floats(sm + pl.offR, pl.offZ + 256 - pl.offR);   // (Z stays 0)
    };
    if (HIN && top && hin) {
        // the level above ran in a launch of its own: its solution comes from
        // HBM, unsqueezed (channel c < C/2 of pixel (i, j) is channel
        // 4c + 2(i&1) + (j&1) of h at (i/2, j/2)), the latent behind it.
        // All loads of a round in flight before its LDS stores.
        work();
        clear();
        const int Ch = C / 2, Wu = W / 2, HWu = (pl.H / 2) * Wu, total = CP * HW;
        const float *hb = hin + b * (size_t)hin_stride;
        const float *lat = lv.z + b * (size_t)Ch * HW;
        constexpr int U = 8;
        for (int base = threadIdx.x; base < total; base += U * block_threads()) {
            float v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = imin(base + u * block_threads(), total - 1);
                const int c = fdiv(idx, pl.d_HW), p = idx - c * HW;
                const int i = fdiv(p, pl.d_W), j = p - i * W;
                const float *src =
                    c < Ch ? hb + (size_t)(4 * c + 2 * (i & 1) + (j & 1)) * HWu + (i >> 1) * Wu +
                                 (j >> 1)
                           : lat + (size_t)imin(c - Ch, Ch - 1) * HW + p;
                v[u] = *src;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                pin(v[u]);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                if (idx < total) {
                    const int c = fdiv(idx, pl.d_HW), p = idx - c * HW;
                    Y[p * CP + c] = c < C ? v[u] : 0.0f;
                }
            }
        }
    } else if (top) {
        // the solution buffer and the partial tiles are cleared while the
        // image is on its way
        load_input<PRE>(sm, pl, lv.z + b * (size_t)C * HW, vec4, [&] {
            work();
            clear();
        }, q);
    } else {
        work();
        const int Ch = C / 2;
        const float *lat = lv.z + b * (size_t)Ch * HW;
        for (int idx = threadIdx.x; idx < CP * HW; idx += block_threads()) {
            const int c = fdiv(idx, pl.d_HW), p = idx - c * HW;
            const int i = fdiv(p, pl.d_W), j = p - i * W;
            float v = 0.0f;
            if (c < Ch) {
                const int ci = 4 * c + 2 * (i & 1) + (j & 1);
                v = sm[up.offX + (((i >> 1) + up.P) * up.WP + (j >> 1) + up.P) * up.CP + ci];
            } else if (c < C) {
                v = lat[(c - Ch) * HW + p];
            }
            Y[p * CP + c] = v;
        }
        __syncthreads();   // the level above's solution has been read
        clear();
    }
    __syncthreads();
}

// All layers of one level for one wave (NG quad groups).  Weights of the
// next layer are fetched into registers while the current one runs.  inq:
// the input's first round of loads, issued by the kernel (single-layer
// instances that hold the image in LDS; unused otherwise).
template <int NG, int MAXT, int MODE>
__device__ __attribute__((always_inline)) void level_waves(const InvArgs &a, const Level &lv,
                                                           bool top, const Plan &up,
                                                           const Plan &pl, const Role &r,
                                                           float *sm, size_t b,
                                                           const InputRound &inq) {
    constexpr int G = NG > 0 ? NG : 1;
    // weights of the next layer prefetched into registers when they fit (with
    // 16 waves a lane has 128 registers)
    constexpr bool kPrefetch = NG <= 4 && (MAXT <= 512 || NG <= 2);
    constexpr int GN = kPrefetch ? G : 1;
    // the register-fed critical wave owns the two dp + dq = 1 taps as groups
    // (MODE: kCritGather / kCritRegs -- the instance carries only the
    // critical loop its levels use)
    constexpr int CRIT = MODE & 3;
    constexpr bool kOne = (MODE & kOneLayer) != 0;
    constexpr bool kStr = (MODE & kStream) != 0;
    const bool regc = CRIT == kCritRegs && r.role == 0;
    const int ngw = r.ng;
    const int lane = threadIdx.x & 63, kq = lane >> 4, li = lane & 15;
    const int C = pl.C, CP = pl.CP, H = pl.H, W = pl.W, P = pl.P, WP = pl.WP;
    const int HW = H * W;
    const int mt = r.mt, nt = r.nt;
    const int E = H + W - 1;
    const int r0 = mt * 16, r1 = imin(mt * 16 + 15, H - 1);
    float *R = sm + pl.offR;
    const size_t lstride = pl.lstride;
    const int nlayers = kOne ? 1 : a.n_units * a.lpu;
    float w[G][4], wn[GN][4];
    // layer index n = 0 .. nlayers-1 runs unit u = U-1-n/lpu, block q = lpu-1-n%lpu
    const int quarter = blockIdx.x & 3;   // (split unit only)
    auto prep_of = [&](int n) {
        if (a.split)
            return lv.prep + (size_t)quarter * lstride;
        if (kOne)
            return lv.prep;
        const int u = a.n_units - 1 - n / a.lpu, q = a.lpu - 1 - n % a.lpu;
        return lv.prep + (size_t)(u * a.lpu + q) * lstride;
    };
    auto corner_at = [&](int n) {
        return a.split ? quarter : kOne ? a.corner0 : corner_of(a, a.lpu - 1 - n % a.lpu);
    };
    auto fetch = [&](auto &dst, int n) {
        if (regc)
            load_crit_weights(dst, pl, prep_of(n));
        else
            load_weights(dst, pl, r, prep_of(n), CRIT == kCritRegs && pl.regcrit);
    };
    // first layer's weights in flight while the level's input is loaded
    if (nlayers > 0) {
        if constexpr (kPrefetch)
            fetch(wn, 0);
        else
            fetch(w, 0);
    }
    // corner-free geometry of each group's quad: dp | dq << 4 | cq << 8, or
    // -1 where the quad does not exist (decoded while the input is on its way)
    int geo[G];
    auto decode = [&] {
        // lane l holds the back-offset of tap l (taps number at most 49); a
        // group's lanes fetch their taps' from those lanes (one cross-lane
        // read per group instead of one walk over the distances)
        int dpl, dql;
        tap_of_lanes(lane, pl.K, dpl, dql);
        const int tapv = dpl | dql << 4;
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            const int uq = quad_of(pl, r, g, kq), uc = uq < 0 ? 0 : uq;
            const int t = fdiv(uc, pl.d_ncq), cq = uc - t * pl.ncq;
            const int tv = __builtin_amdgcn_ds_bpermute(t << 2, tapv);
            geo[g] = uq < 0 ? -1 : tv | cq << 8;
        }
    };
    // --- stream form: input and output move between HBM and the rings in
    // phases of kPhase diagonals.  Element t of the phase starting at
    // diagonal d0: frame row i, channel c, diagonal d0 + t % kPhase
    // (consecutive threads take consecutive columns of one row).
    float ypre[kStreamRegs];
    const int nph = kPhase * H * C;
    // banded stream form: the workgroup's image and band come from a ticket
    // taken at its start (through the trash block, unused until the steps),
    // so a band only ever waits on a band that started before it
    constexpr bool banded = kStr && (MODE & kBanded) != 0;
    int bimg = (int)b, band = 0;
    if constexpr (banded) {
        int *tk = reinterpret_cast<int *>(sm + pl.offT);
        if (threadIdx.x == 0)
            tk[0] = __hip_atomic_fetch_add(a.bflags + 1, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        const int t = tk[0];
        __syncthreads();
        bimg = t / a.nbands;
        band = t - bimg * a.nbands;
    }
    const int imgH = banded ? a.img_H : H;   // rows of the whole image
    const int i0 = band * H;                 // the band's first frame row
    const int HWi = imgH * W;
    const float *zin = lv.z + (size_t)bimg * C * HWi;
    float *zout = a.out + (size_t)bimg * C * HWi;
    const int scorner = corner_at(0);
    const bool sfh = scorner == FINC_BL || scorner == FINC_BR;
    const bool sfw = scorner == FINC_TR || scorner == FINC_BR;
    auto selem = [&](int t, int d0, int &i, int &c, int &j) __attribute__((always_inline)) {
        const int rc = t >> 4;
        c = fdiv(rc, pl.d_H);
        i = rc - c * H;
        j = d0 + (t & (kPhase - 1)) - i;
    };
    // natural NCHW offset of frame pixel (i0 + i, j), channel c
    auto snat = [&](int c, int i, int j) __attribute__((always_inline)) {
        return c * HWi + (sfh ? imgH - 1 - (i0 + i) : i0 + i) * W + (sfw ? W - 1 - j : j);
    };
    // loads of the input of diagonals d0 .. d0 + kPhase - 1 into registers
    auto sissue = [&](int d0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kStreamRegs; ++u) {
            const int t = threadIdx.x + u * block_threads();
            int i, c, j;
            selem(t, d0, i, c, j);
            const bool ok = t < nph && (unsigned)j < (unsigned)W && (!banded || i0 + i < imgH);
            ypre[u] = zin[ok ? snat(c, i, j) : 0];
        }
    };
    // the loaded values into the input ring
    auto sput = [&](int d0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < kStreamRegs; ++u) {
            const int t = threadIdx.x + u * block_threads();
            int i, c, j;
            selem(t, d0, i, c, j);
            if (t < nph && (unsigned)j < (unsigned)W)
                sm[pl.offY + (i * kRing + (j & (kRing - 1))) * CP + c] = ypre[u];
        }
    };
    // solved diagonals d0 .. d1 to HBM
    auto sdrain = [&](int d0, int d1) __attribute__((always_inline)) {
        for (int t = threadIdx.x; t < nph; t += block_threads()) {
            int i, c, j;
            selem(t, d0, i, c, j);
            if (d0 + (t & (kPhase - 1)) <= d1 && (unsigned)j < (unsigned)W &&
                (!banded || i0 + i < imgH))
                zout[snat(c, i, j)] =
                    sm[pl.offX + ((i + P) * kRing + (j & (kRing - 1))) * CP + c];
        }
    };
    // (banded) thread 0 waits until the band above has drained `need`
    // diagonals (bounded: past kBandSpin tries the timeout flag is set and
    // the band goes on) and acquires what it drained -- one cache
    // invalidation for the workgroup, whose other waves wait at the barrier
    auto bwait = [&](int need) __attribute__((always_inline)) {
        if (threadIdx.x == 0) {
            const int *f = a.bflags + 2 + bimg * a.nbands + band - 1;
            for (int it = 0;
                 __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < need; ++it) {
                if (it >= kBandSpin) {
                    __hip_atomic_store(a.bflags, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(4);
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        }
        __syncthreads();
    };
    // (banded) frame rows i0 - P .. i0 - 1 -- the band above's last rows, as
    // it drained them -- at columns c0 .. c1 into the solution ring's border
    auto sborder = [&](int c0, int c1) __attribute__((always_inline)) {
        const int ncol = c1 - c0 + 1, nb = P * ncol * C;
        for (int t = threadIdx.x; t < nb; t += block_threads()) {
            const int jj = t % ncol, r2 = t / ncol, ii = r2 % P, c = r2 / P;
            const int j = c0 + jj, i = ii - P;
            sm[pl.offX + (ii * kRing + (j & (kRing - 1))) * CP + c] = zout[snat(c, i, j)];
        }
    };
    // (banded) the count of diagonals this band has drained, published by a
    // release store after the barrier (every wave's drain stores complete
    // before it)
    auto bpublish = [&](int ndiag) __attribute__((always_inline)) {
        __syncthreads();
        if (threadIdx.x == 0)
            __hip_atomic_store(a.bflags + 2 + bimg * a.nbands + band, ndiag, __ATOMIC_RELEASE,
                               __HIP_MEMORY_SCOPE_AGENT);
    };
    // end of diagonal step e: the barrier; in the stream form, at the end of
    // a phase, the exchange with HBM and one more barrier
    int nsteps = 0;   // diagonal steps this wave ran (the steps diagnostic)
    auto step_end = [&](int e) __attribute__((always_inline)) {
        ++nsteps;
        __syncthreads();
        if constexpr (kStr) {
            const bool pend = (e & (kPhase - 1)) == kPhase - 1;
            if (pend || e == E - 1) {
                if (pend)
                    sput(e + 2);   // input of diagonals e + 2 .. e + 1 + kPhase
                sdrain(e & ~(kPhase - 1), e);
                if (pend)
                    sissue(e + 2 + kPhase);
                if constexpr (banded) {
                    bpublish(e + 1);
                    // border columns of the next phase's diagonals: the band
                    // above's pixel (H - 1, c) is on its diagonal c + H - 1
                    if (band > 0 && pend && e + 2 < W) {
                        const int c1 = imin(e + 1 + kPhase, W - 1);
                        bwait(c1 + H);
                        sborder(e + 2, c1);
                    }
                }
                __syncthreads();
            }
        }
    };
    if constexpr (kStr) {
        // diagonals 0 .. kPhase of the input; the next phase's loads in flight
        sissue(1);
        decode();
        zero_floats(sm + pl.offX, pl.offT - pl.offX);   // rings, partial tiles, Z
        __syncthreads();
        if constexpr (banded) {
            if (band > 0) {   // border columns of diagonals 0 .. kPhase
                const int c1 = imin(kPhase, W - 1);
                bwait(c1 + H);
                sborder(0, c1);
            }
        }
        sput(1);
        if (threadIdx.x < C)
            sm[pl.offY + threadIdx.x] = zin[snat(threadIdx.x, 0, 0)];
        sissue(1 + kPhase);
        __syncthreads();
    } else {
        // (decode reads across lanes: every lane of the wave runs it here,
        // outside the input loader's per-thread branches)
        decode();
        level_input<!kOne, kOne>(lv, top, up, sm, b, (a.vec & 1) != 0, a.hin, a.hin_stride,
                                 [] {}, inq);
    }
    for (int n = 0; n < nlayers; ++n) {
        const int u = kOne ? 0 : a.n_units - 1 - n / a.lpu, q = kOne ? 0 : a.lpu - 1 - n % a.lpu;
        if (!kOne && n > 0) {   // previous layer's solution is this layer's input
            copy_solution(sm, pl);
            __syncthreads();
        }
        if (!kOne && q == a.lpu - 1 && lv.scale) {
            float *Y = sm + pl.offY;
            const float *s = lv.scale + (size_t)u * C;
            const float *bi = lv.bias + (size_t)u * C;
            for (int idx = threadIdx.x; idx < HW * C; idx += block_threads()) {
                const int p = fdiv(idx, pl.d_C), c = idx - p * C;
                Y[p * CP + c] = (Y[p * CP + c] - bi[c]) / s[c];
            }
            __syncthreads();
        }
        const int corner = corner_at(n);
        if constexpr (kPrefetch) {
#pragma unroll
            for (int g = 0; g < NG; ++g)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    w[g][e] = wn[g][e];
            if (n + 1 < nlayers)
                fetch(wn, n + 1);
        } else if (n > 0) {
            fetch(w, n);
        }

        // --- addresses: every gather and write address is an affine function
        // of the frame column of its row, which moves by one per diagonal.
        const bool fh = (corner == FINC_BL || corner == FINC_BR);
        const bool fw = (corner == FINC_TR || corner == FINC_BR);
        const int sh = fh ? -1 : 1, sw = fw ? -1 : 1;
        // gather row (frame) i = r0 + li, clamped into the image
        const int gi = mt * 16 + li;
        const int gic = imin(gi, H - 1);
        const int goi = fh ? H - 1 - gic : gic;
        const int bx0 = pl.offX + ((goi + P) * WP + P) * CP;
        const int by0 = pl.offY + goi * W * CP;
        // gather base of each group's quad (plus the column offset of the
        // step).  Quads that do not exist meet zero weights: they read the
        // layer input at the lane's own pixel (in bounds, finite).
        int gbase[G];
#pragma unroll
        for (int g = 0; g < NG; ++g) {
            const int dp = geo[g] & 15, dq = (geo[g] >> 4) & 15, cq4 = (geo[g] >> 8) << 2;
            if (geo[g] < 0)
                gbase[g] = by0;
            else if (dp == 0 && dq == 0)
                gbase[g] = by0 + cq4;
            else
                gbase[g] = bx0 + cq4 - (dp * sh * WP + dq * sw) * CP;
        }
        // Rows of the frame that have not started (frame column j < 0, or rows
        // below the image) gather zeros, so their partial tiles and carried
        // accumulators are exactly 0 and no masking is needed; finished rows
        // (j >= W) gather clamped garbage that only ever reaches finished rows.
        // Every gather, load and write is unconditional (no divergent branch on
        // the critical path); rows that must not be written go to a trash block.
        // Each role runs its own step loop (same barrier count), so the
        // critical loop carries nothing but its own work.
        const int zaddr = pl.offZ + 4 * lane, taddr = pl.offT + 4 * lane;
        const int dcol = fw ? -CP : CP;   // address step of one frame column
        const int fwo = fw ? (W - 1) * CP : 0;
        auto colx = [&](int j) {   // natural column of frame column j (clamped), times CP
            return fwo + __mul24(imin(imax(j, 0), W - 1), dcol);
        };
        // stream form: ring row base of each group's source and its column
        // back-offset (the self tap reads the input ring)
        int rbase[G], sdq[G];
        if constexpr (kStr) {
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                const int dp = geo[g] & 15, dq = (geo[g] >> 4) & 15, cq4 = (geo[g] >> 8) << 2;
                const bool self = geo[g] < 0 || (dp == 0 && dq == 0);
                rbase[g] = self ? pl.offY + gic * kRing * CP + (geo[g] < 0 ? 0 : cq4)
                                : pl.offX + (gic - dp + P) * kRing * CP + cq4;
                sdq[g] = self ? 0 : dq;
            }
        }
        // Gather addresses of every group at frame column j.
        auto addrs = [&](int (&ad)[G], int j) {
            const bool live = j >= 0 && gi < H;
            if constexpr (kStr) {
#pragma unroll
                for (int g = 0; g < NG; ++g)
                    ad[g] = live ? rbase[g] + __mul24((j - sdq[g]) & (kRing - 1), CP) : zaddr;
            } else {
                const int cx = colx(j);
#pragma unroll
                for (int g = 0; g < NG; ++g)
                    ad[g] = live ? gbase[g] + cx : zaddr;
            }
        };
        // The wave's B operands, one 16-byte load per group, all in flight
        // together.  `full`: the wave owns every group of the instance (no
        // per-group test); otherwise groups [0, ngw).
        auto load = [&](float4 (&av)[G], const int (&ad)[G], auto full) {
#pragma unroll
            for (int g = 0; g < NG; ++g)
                if (decltype(full)::value || g < ngw)
                    av[g] = *reinterpret_cast<const float4 *>(sm + ad[g]);
        };
        // D[output channel 4 kq + rr][row li] = sum over the wave's groups:
        // weights are the A operand (rows = output channels), gathered inputs
        // the B operand (columns = frame rows)
        auto mma = [&](const float4 (&av)[G], auto full) -> f32x4 {
            f32x4 c = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
            for (int g = 0; g < NG; ++g) {
                if (decltype(full)::value || g < ngw) {
                    c = mfma4(w[g][0], av[g].x, c);
                    c = mfma4(w[g][1], av[g].y, c);
                    c = mfma4(w[g][2], av[g].z, c);
                    c = mfma4(w[g][3], av[g].w, c);
                }
            }
            return c;
        };
        // Diagonals that meet the tile's rows; a role's other steps only keep
        // the barrier count (every role passes 1 + E barriers per layer).
        const int e_lo = r0, e_hi = imin(r1 + W - 1, E - 1);
        // the critical wave writes channels 16 nt + 4 kq .. +3 of its row's pixel
        const int wx0 = bx0 + nt * 16 + 4 * kq;
        const bool wch = nt * 16 + 4 * kq < CP && gi < H;
        // partial tiles: R[parity][T RS slots (+ one zero slot)][64 lanes][4].
        // The critical wave reads S4 slots, four at a time: padded, slot s of
        // its tile; compact, slots from S on are the zero slot of the parity.
        const int rstride = (pl.T * pl.RS + pl.compact) * 256;
        const int rown = (r.tile * pl.RS + (r.role == 1 ? r.h : 0)) * 256 + 4 * lane;
        const f32x4 *R0 = reinterpret_cast<const f32x4 *>(R + rown);
        const f32x4 *Rz = reinterpret_cast<const f32x4 *>(R + pl.T * pl.RS * 256 + 4 * lane);
        auto sbase = [&](int s, auto pad) {
            return decltype(pad)::value || s < pl.S ? R0 + s * 64 : Rz;
        };
        // slot s at parity offset po (in f32x4)
        auto slot = [&](int s, int po, auto pad) { return sbase(s, pad)[po]; };
        // the sum of a tile's partial tiles, in a fixed order
        auto partial_sum = [&](int po, auto pad) {
            f32x4 s0 = slot(0, po, pad) + slot(1, po, pad);
            const f32x4 s1 = slot(2, po, pad) + slot(3, po, pad);
            s0 += s1;
            for (int s4 = 4; s4 < pl.S4; s4 += 4) {
                f32x4 t0 = slot(s4, po, pad) + slot(s4 + 1, po, pad);
                const f32x4 t1 = slot(s4 + 2, po, pad) + slot(s4 + 3, po, pad);
                t0 += t1;
                s0 += t0;
            }
            return s0;
        };
        const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
        if (top && n == 0)
            stamp(a.stamps, b, 1);

        if (r.role == 1) {
            // helper: during step e, the partial tile of diagonal e + 1 (every
            // source is on diagonal e - 1 or earlier, or is y).  The next
            // step's gather addresses are formed while the tile's write lands.
            f32x4 *Rw = reinterpret_cast<f32x4 *>(R + rown);
            auto run = [&](auto full) {
                float4 av[G];
                int ad[G];
                if (e_lo == 0) {   // diagonal 0: all sources are zero but y
                    addrs(ad, -gi);
                    load(av, ad, full);
                    Rw[0] = mma(av, full);
                }
                // steps e whose diagonal e + 1 meets the tile
                const int lo = imax(e_lo - 1, 0), hi = e_hi - 1;
                addrs(ad, lo + 1 - gi);
                __syncthreads();
                int e = 0;
                for (; e < lo; ++e)
                    step_end(e);
                for (; e <= hi; ++e) {
                    load(av, ad, full);
                    Rw[((e + 1) & 1) * (rstride / 4)] = mma(av, full);
                    addrs(ad, e + 2 - gi);
                    step_end(e);
                }
                for (; e < E; ++e)
                    step_end(e);
            };
            if (ngw == NG)
                run(std::true_type{});
            else
                run(std::false_type{});
        } else if (CRIT == kCritRegs && r.role == 0) {
            // register-fed critical wave, its tile's rows in the order of
            // crit_row (EQ = ncq channels per lane group).  dprev: lane (kq,
            // li) holds channels EQ kq .. EQ kq + EQ-1 of row li's pixel of the
            // previous diagonal (0 for rows not started).  Its MFMA chain needs
            // nothing from LDS but, in a lower tile, lane li = 0's row above
            // (the last row of the tile above); the partial tiles are read
            // meanwhile and added last.  Each tap takes EQ MFMAs; the chain's
            // first kPre MFMAs (own row) depend on nothing but dprev: they are
            // issued before the barrier, while the write of the diagonal
            // becomes visible.
            auto crit = [&](auto pad, auto eqc) {
                constexpr int EQ = decltype(eqc)::value;
                constexpr int kPre = EQ < 4 ? EQ : 3;
                f32x4 dprev = zero, pre = zero;
                int j = e_lo - gi;   // frame column of row gi at the tile's first diagonal
                // write address of frame column j (the affine form; used only while
                // 0 <= j < W): channels EQ kq .. of the row's pixel
                int wcol = bx0 + EQ * kq + fwo + j * dcol;
                // lane li = 0 of a lower tile reads the tile above's last row
                // (solved in the previous step); other lanes read zeros
                const int ui = mt * 16 - 1;
                const int uoi = fh ? H - 1 - imax(ui, 0) : imax(ui, 0);
                int ju = e_lo - 16 * mt;   // frame column of row 16 mt (and of the row above it)
                int ucol = pl.offX + ((uoi + P) * WP + P) * CP + fwo + EQ * kq + ju * dcol;
                // (stream form: ring rows of the written row and of the row above)
                const int wxs = pl.offX + (gic + P) * kRing * CP + EQ * kq;
                // the first tile of a lower band: its row above is the band
                // above's last row, in the ring's border (else zeros)
                const bool upb = banded && band > 0 && mt == 0;
                const int uxs = pl.offX + ((upb ? -1 : imax(ui, 0)) + P) * kRing * CP + EQ * kq;
                const f32x4 *b1 = sbase(1, pad), *b2 = sbase(2, pad), *b3 = sbase(3, pad);
                __syncthreads();
                int e = 0;
                for (; e < e_lo; ++e)
                    step_end(e);
                for (; e <= e_hi; ++e) {
                    {
                        const int po = (e & 1) * (rstride / 4);
                        const int ucur = kStr ? uxs + __mul24(ju & (kRing - 1), CP) : ucol;
                        const int wcur = kStr ? wxs + __mul24(j & (kRing - 1), CP) : wcol;
                        float up[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                        if (mt > 0 || upb) {
                            const float *ua =
                                sm + ((li == 0 && (unsigned)ju < (unsigned)W) ? ucur : zaddr);
#pragma unroll
                            for (int e4 = 0; e4 < EQ; ++e4)
                                up[e4] = ua[e4];
                        }
                        // the first four partial tiles in flight during the MFMAs
                        const f32x4 q0 = R0[po], q1 = b1[po], q2 = b2[po], q3 = b3[po];
                        const bool ok = gi < H && (unsigned)j < (unsigned)W;
                        const int waddr = ok ? wcur : taddr;
                        __builtin_amdgcn_sched_barrier(0);
                        f32x4 p = pre;
                        // tap (0,1): own row, previous column; tap (1,0): row above,
                        // same column -- the neighbouring lane's previous result
                        // (row_shr:1 inside each row of 16 lanes; lane 0 takes `up`).
                        // Elements are copied to scalars first: this compiler
                        // bit-casts a vector element lvalue as element 0.
                        if constexpr (G >= 2) {   // (instances with G < 2 never get regc)
#pragma unroll
                            for (int e4 = kPre; e4 < EQ; ++e4)
                                p = mfma4(w[0][e4], dprev[e4], p);
#pragma unroll
                            for (int e4 = 0; e4 < EQ; ++e4) {
                                const float de = dprev[e4], ue = up[e4];
                                const float s1 = __int_as_float(__builtin_amdgcn_update_dpp(
                                    __float_as_int(ue), __float_as_int(de), 0x111, 0xf, 0xf, false));
                                p = mfma4(w[1][e4], s1, p);
                            }
                        }
                        __builtin_amdgcn_sched_barrier(0);
                        f32x4 rs = q0 + q1;
                        const f32x4 rt = q2 + q3;
                        rs += rt;
                        for (int s4 = 4; s4 < pl.S4; s4 += 4) {
                            f32x4 t0 = slot(s4, po, pad) + slot(s4 + 1, po, pad);
                            const f32x4 t1 = slot(s4 + 2, po, pad) + slot(s4 + 3, po, pad);
                            t0 += t1;
                            rs += t0;
                        }
                        const f32x4 x = rs + p;
                        if constexpr (EQ == 4) {
                            *reinterpret_cast<f32x4 *>(sm + waddr) = x;
                        } else {
#pragma unroll
                            for (int e4 = 0; e4 < EQ; ++e4)
                                sm[waddr + e4] = x[e4];
                        }
                        dprev = x;
                        __builtin_amdgcn_sched_barrier(0);
                        // next diagonal's own-row MFMAs, overlapping the write
                        pre = zero;
                        if constexpr (G >= 2) {
#pragma unroll
                            for (int e4 = 0; e4 < kPre; ++e4)
                                pre = mfma4(w[0][e4], dprev[e4], pre);
                        }
                    }
                    j += 1;
                    wcol += dcol;
                    ju += 1;
                    ucol += dcol;
                    step_end(e);
                }
                for (; e < E; ++e)
                    step_end(e);
            };
            auto crit_eq = [&](auto pad) {
                switch (pl.ncq) {
                    case 1: crit(pad, std::integral_constant<int, 1>{}); break;
                    case 2: crit(pad, std::integral_constant<int, 2>{}); break;
                    case 3: crit(pad, std::integral_constant<int, 3>{}); break;
                    default: crit(pad, std::integral_constant<int, 4>{}); break;
                }
            };
            if (pl.compact)
                crit_eq(std::false_type{});
            else
                crit_eq(std::true_type{});
        } else if (CRIT == kCritGather && r.role == 0) {
            // critical wave that gathers its dp + dq = 1 taps from LDS (several
            // channel tiles: the previous diagonal's channels sit in several
            // waves)
            auto run = [&](auto full, auto pad) {
                float4 av[G];
                int ad[G];
                addrs(ad, e_lo - gi);
                __syncthreads();
                int e = 0;
                for (; e < e_lo; ++e)
                    step_end(e);
                for (; e <= e_hi; ++e) {
                    const int j = e - gi;
                    load(av, ad, full);
                    const f32x4 rs = partial_sum((e & 1) * (rstride / 4), pad);
                    f32x4 x = mma(av, full);
                    x += rs;
                    const bool ok = wch && (unsigned)j < (unsigned)W;
                    *reinterpret_cast<f32x4 *>(sm + (ok ? wx0 + colx(j) : taddr)) = x;
                    addrs(ad, e + 1 - gi);
                    step_end(e);
                }
                for (; e < E; ++e)
                    step_end(e);
            };
            if (ngw == NG && !pl.compact)
                run(std::true_type{}, std::true_type{});
            else if (ngw == NG)
                run(std::true_type{}, std::false_type{});
            else if (!pl.compact)
                run(std::false_type{}, std::true_type{});
            else
                run(std::false_type{}, std::false_type{});
        } else if (kOne && !kStr && CRIT == kCritRegs && a.drain == wave_id() + 1) {
            // the drain wave: frame row fi is solved with diagonal fi + W - 1;
            // it goes out during the next step, the last one after the last
            // barrier.  Lane t of round u takes element t + 64 u of a row as
            // (channel, column); raw buffer stores over the image's output
            // drop the offsets past it (lanes beyond C W).
            const int nrounds = (C * W + kWave - 1) / kWave;   // <= kDrainRounds (host)
            const bool fh = corner == FINC_BL || corner == FINC_BR;
            const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
                a.out + b * (size_t)a.out_stride, (short)0, C * HW * 4, kBufferWord3);
            int lo[kDrainRounds], go[kDrainRounds];
#pragma unroll
            for (int u = 0; u < kDrainRounds; ++u) {
                const int t = lane + kWave * u;
                const int c = fdiv(t, pl.d_W), j = t - c * W;
                const bool ok = t < C * W;
                lo[u] = ok ? (j + P) * CP + c : 0;
                go[u] = ok ? (c * HW + j) * 4 : C * HW * 4;
            }
            // one row: R rounds of an LDS read, then R stores, the row's
            // offset in the stores' scalar offset
            auto drain_row = [&](int fi, auto rc) {
                constexpr int R = decltype(rc)::value;
                const int nr = fh ? H - 1 - fi : fi;
                const float *xr = sm + pl.offX + (nr + P) * WP * CP;
                float v[R];
#pragma unroll
                for (int u = 0; u < R; ++u)
                    v[u] = xr[lo[u]];
#pragma unroll
                for (int u = 0; u < R; ++u)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v[u]), ro,
                                                          go[u], nr * W * 4, 0);
            };
            auto drain_loop = [&](auto rc) {
                __syncthreads();
                for (int e = 0; e < E; ++e) {
                    step_end(e);
                    if (e >= W - 1)
                        drain_row(e - (W - 1), rc);
                }
            };
            switch (nrounds) {
                case 1: drain_loop(std::integral_constant<int, 1>{}); break;
                case 2: drain_loop(std::integral_constant<int, 2>{}); break;
                case 3: drain_loop(std::integral_constant<int, 3>{}); break;
                case 4: drain_loop(std::integral_constant<int, 4>{}); break;
                case 5: drain_loop(std::integral_constant<int, 5>{}); break;
                case 6: drain_loop(std::integral_constant<int, 6>{}); break;
                case 7: drain_loop(std::integral_constant<int, 7>{}); break;
                default: drain_loop(std::integral_constant<int, 8>{}); break;
            }
        } else {
            __syncthreads();
            for (int e = 0; e < E; ++e)
                step_end(e);
        }
    }
    if (a.steps && (threadIdx.x & 63) == 0)
        a.steps[b * (block_threads() >> 6) + (threadIdx.x >> 6)] = nsteps;
}

// A wave of a multi-level chain runs the level loop compiled for its own
// quad-group count at that level (G = the first count >= ng): a level whose
// waves own fewer groups than the chain's widest level then runs as it does
// on its own, without per-group tests and with the weight prefetch.  Every
// variant passes the same barriers, so the waves of one workgroup may run
// different ones.
template <int G, int NG, int MAXT, int MODE>
__device__ __attribute__((always_inline)) void level_waves_for(int ng, const InvArgs &a, const Level &lv, bool top,
                                const Plan &up, const Plan &pl, const Role &r, float *sm,
                                size_t b, const InputRound &inq) {
    if constexpr (G < NG) {
        if (ng <= G) {
            level_waves<G, MAXT, MODE>(a, lv, top, up, pl, r, sm, b, inq);
            return;
        }
        level_waves_for<G + 1, NG, MAXT, MODE>(ng, a, lv, top, up, pl, r, sm, b, inq);
    } else {
        level_waves<NG, MAXT, MODE>(a, lv, top, up, pl, r, sm, b, inq);
    }
}

// Inverse of a whole chain with the image in LDS from the first load to the
// last store.  Levels run in argument order (the top of a stack first);
// between levels the solution of the level above is unsqueezed and the
// level's latent appended behind it (channel split), straight from LDS into
// the next level's input.  The first level sits at a fixed argument offset,
// so its arguments arrive in the kernel's first round of scalar loads.
template <int NG, int MAXT, int MODE>
__global__ __launch_bounds__(MAXT) void inverse_chain_kernel(InvArgs a) {
    extern __shared__ float sm[];
    const size_t b = blockIdx.x;
    Level lv = a.lv[0];
    Plan above = lv.pl;   // plan of the level run before (unused at the first)
    // one round of scalar loads for everything the first level starts with:
    // one dword of every argument line up to the end of the first level, the
    // wave's role word and the workgroup size (a line of the implicit
    // arguments) -- later loads of these lines hit the scalar cache instead of
    // each costing a round trip to memory.  tid comes out of the same barrier,
    // so nothing that depends on it is scheduled (with a wait) before it.
    int tid = threadIdx.x;
    {
        const int *ai = reinterpret_cast<const int *>(&a);
        constexpr int kArgLines = (int)((offsetof(InvArgs, lv) + sizeof(Level) + 63) / 64);
        static_assert(kArgLines <= 8, "first level's arguments span at most 8 lines");
        auto line = [&](int l) { return ai[16 * (l < kArgLines ? l : kArgLines - 1)]; };
        const int l0 = line(0), l1 = line(1), l2 = line(2), l3 = line(3), l4 = line(4),
                  l5 = line(5), l6 = line(6), l7 = line(7), nthr = block_threads();
        const int rw =
            a.lv[0].pl.wave[__builtin_amdgcn_readfirstlane(threadIdx.x >> 6) & (kMaxWaves - 1)];
        asm volatile("" : "+v"(tid) : "s"(l0), "s"(l1), "s"(l2), "s"(l3), "s"(l4), "s"(l5),
                     "s"(l6), "s"(l7), "s"(nthr), "s"(rw));
    }
    constexpr bool kOne = (MODE & kOneLayer) != 0;
    // a single layer held in LDS reads its input straight from z: the first
    // round of those loads goes out now, ahead of the set-up
    InputRound inq;
    if constexpr (kOne && (MODE & kStream) == 0)
        input_issue(lv.pl, lv.z + b * (size_t)lv.pl.C * lv.pl.H * lv.pl.W, tid, inq);
    stamp(a.stamps, b, 0);
    for (int i = 0; i < (kOne ? 1 : a.L); ++i) {
        if (i > 0) {
            above = lv.pl;
            lv = a.lv[i];
        }
        const Plan &pl = lv.pl;
        const int CP = pl.CP, W = pl.W, HW = pl.H * pl.W;
        float *Y = sm + pl.offY;
        if constexpr (!kOne && MAXT == 1024) {   // (chains whose levels differ most)
            const Role r = role_of(a, i);
            level_waves_for<1, NG, MAXT, MODE>(r.ng, a, lv, i == 0, above, pl, r, sm, b, inq);
        } else {
            level_waves<NG, MAXT, MODE>(a, lv, i == 0, above, pl, role_of(a, i), sm, b, inq);
        }
        if (!kOne && a.n_units * a.lpu == 0) {   // no layers at this level: the input passes through
            for (int idx = threadIdx.x; idx < HW * CP; idx += block_threads()) {
                const int p = fdiv(idx, pl.d_CP), c = idx - p * CP;
                const int i = fdiv(p, pl.d_W), j = p - i * W;
                sm[pl.offX + ((i + pl.P) * pl.WP + j + pl.P) * CP + c] = Y[idx];
            }
            __syncthreads();
        }
    }
    stamp(a.stamps, b, 2);
    if ((MODE & kStream) != 0 || a.drain) {
        // (the solution went out phase by phase, or the drain wave stored
        // the rows as they were solved)
        stamp(a.stamps, b, 3);
        return;
    }
    const Plan &p0 = lv.pl;   // the last level run
    const int HW0 = p0.H * p0.W;
    float *dst = a.out + b * (size_t)a.out_stride;
    // With vec bit 1, a thread takes four pixels of a row by one
    // channel quad: four 16-byte LDS reads, one per pixel, transposed in
    // registers into four 16-byte stores, one per channel, coalesced across
    // the lanes.  Otherwise one pixel's quad: one LDS read, four scalar stores.
    const int nq0 = p0.CP / 4;
    auto xat = [&](int p, int cq) {
        const int i = fdiv(p, p0.d_W), j = p - i * p0.W;
        return *reinterpret_cast<const float4 *>(
            sm + p0.offX + ((i + p0.P) * p0.WP + j + p0.P) * p0.CP + 4 * cq);
    };
    if (a.vec & 2) {
        const int tot = nq0 * (HW0 / 4);   // (pixel group, quad), quad fastest
        float4 *d4 = reinterpret_cast<float4 *>(dst);
        constexpr int U = 2;
        for (int base = threadIdx.x; base < tot; base += U * block_threads()) {
            float4 v[U][4];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = imin(base + u * block_threads(), tot - 1);
                const int pg = fdiv(idx, p0.d_cp4), cq = idx - pg * nq0;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    v[u][i] = xat(4 * pg + i, cq);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                if (idx < tot) {
                    const int pg = fdiv(idx, p0.d_cp4), cq = idx - pg * nq0, c = 4 * cq;
                    float4 *d = d4 + (size_t)c * (HW0 / 4) + pg;
                    d[0] = make_float4(v[u][0].x, v[u][1].x, v[u][2].x, v[u][3].x);
                    if (c + 1 < p0.C)
                        d[HW0 / 4] = make_float4(v[u][0].y, v[u][1].y, v[u][2].y, v[u][3].y);
                    if (c + 2 < p0.C)
                        d[HW0 / 2] = make_float4(v[u][0].z, v[u][1].z, v[u][2].z, v[u][3].z);
                    if (c + 3 < p0.C)
                        d[3 * (HW0 / 4)] =
                            make_float4(v[u][0].w, v[u][1].w, v[u][2].w, v[u][3].w);
                }
            }
        }
    } else {
        constexpr int U = 4;
        const int tot = nq0 * HW0;   // (quad, pixel), pixel fastest
        for (int base = threadIdx.x; base < tot; base += U * block_threads()) {
            float4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = imin(base + u * block_threads(), tot - 1);
                const int cq = fdiv(idx, p0.d_HW), p = idx - cq * HW0;
                v[u] = xat(p, cq);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int idx = base + u * block_threads();
                if (idx < tot) {
                    const int cq = fdiv(idx, p0.d_HW), p = idx - cq * HW0, c = 4 * cq;
                    float *d = dst + (size_t)c * HW0 + p;
                    d[0] = v[u].x;
                    if (c + 1 < p0.C)
                        d[HW0] = v[u].y;
                    if (c + 2 < p0.C)
                        d[2 * HW0] = v[u].z;
                    if (c + 3 < p0.C)
                        d[3 * HW0] = v[u].w;
                }
            }
        }
    }
    stamp(a.stamps, b, 3);
}

// Inverse kernel instances, in groups of one workgroup size and one mode, by
// quad groups per wave (1..kMaxGroups).  The host picks one by address.
constexpr int kInverseGroups = 18;
constexpr int kModesPerSize = 6;
constexpr int kGroupThreads[kInverseGroups] = {256,  256,  256,  256,  256,  256,
                                               512,  512,  512,  512,  512,  512,
                                               1024, 1024, 1024, 1024, 1024, 1024};
constexpr int kGroupModes[kModesPerSize] = {kCritGather,
                                            kCritRegs,
                                            kCritGather | kOneLayer,
                                            kCritRegs | kOneLayer,
                                            kCritRegs | kOneLayer | kStream,
                                            kCritRegs | kOneLayer | kStream | kBanded};
constexpr int kGroupMode[kInverseGroups] = {
    kGroupModes[0], kGroupModes[1], kGroupModes[2], kGroupModes[3], kGroupModes[4], kGroupModes[5],
    kGroupModes[0], kGroupModes[1], kGroupModes[2], kGroupModes[3], kGroupModes[4], kGroupModes[5],
    kGroupModes[0], kGroupModes[1], kGroupModes[2], kGroupModes[3], kGroupModes[4], kGroupModes[5]};

template <int MAXT, int MODE>
const void *inverse_instance_of(int ng) {
    switch (ng) {
    case 1: return reinterpret_cast<const void *>(inverse_chain_kernel<1, MAXT, MODE>);
    case 2: return reinterpret_cast<const void *>(inverse_chain_kernel<2, MAXT, MODE>);
    case 3: return reinterpret_cast<const void *>(inverse_chain_kernel<3, MAXT, MODE>);
    case 4: return reinterpret_cast<const void *>(inverse_chain_kernel<4, MAXT, MODE>);
    case 5: return reinterpret_cast<const void *>(inverse_chain_kernel<5, MAXT, MODE>);
    case 6: return reinterpret_cast<const void *>(inverse_chain_kernel<6, MAXT, MODE>);
    case 7: return reinterpret_cast<const void *>(inverse_chain_kernel<7, MAXT, MODE>);
    default: return reinterpret_cast<const void *>(inverse_chain_kernel<8, MAXT, MODE>);
    }
}

}  // namespace

#define FINC_GROUPS(X) \
    X(0) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) \
        X(16) X(17)
#define FINC_CAT2(a, b) a##b
#define FINC_CAT(a, b) FINC_CAT2(a, b)

namespace finc_parts {
#define FINC_DECLARE(g) const void *inverse_group_##g(int ng);
FINC_GROUPS(FINC_DECLARE)
#if FINC_PART >= 0
const void *FINC_CAT(inverse_group_, FINC_PART)(int ng) {
    return inverse_instance_of<kGroupThreads[FINC_PART], kGroupMode[FINC_PART]>(ng);
}
#endif
}  // namespace finc_parts

#if FINC_PART < 0
namespace {

// ---------------------------------------------------------------------------
// Forward (Sec. 3 convolution with the Sec. 4.1 corner padding) as MFMA
// contractions: for a tile of 16 pixels and 16 output channels
//     D[c_out][pixel] = sum_{tap, c_in} K[c_out][c_in][tap] x[c_in][pixel + tap]
// over k = (tap, input-channel quad), the inputs gathered from a zero-bordered
// LDS copy of the image (out-of-image taps read the border) and the masked
// weights staged in LDS in the MFMA fragment layout.  A single layer splits
// each image into blocks of rows (with the k-1 halo rows) so that the grid
// covers the chip; a unit keeps the image in LDS across its four layers.
// ---------------------------------------------------------------------------
struct FwdPlan {
    int C, CP, H, W, K, P, WP;
    int NT, ncq, nq, NG;         // channel tiles, quads per tile (all taps), quad groups
                                 // (padded to a multiple of four)
    int NGr;                     // quad groups with weights, ceil(nq / 4)
    // padw 1: every quad group, padding ones included, has its fragments in
    // LDS (zeros for padding groups; the loop reads them like any other);
    // 0 (where those would not fit): padding groups read one shared zero
    // fragment, chosen per group.  NGw: fragments of a channel tile in LDS.
    int padw, NGw;
    int RB, nblk;                // rows per block, blocks per image
    int HB;                      // halo rows staged above and below a block
    int offI, offO, offW, offD;  // LDS floats: input rows (RB + 2P) x WP x CP, output
                                 // (chains only), weight fragments, quad offsets (ints)
    int lds_floats;
    int n, corner0;              // layers (1, or 4 for a unit: TL, TR, BL, BR)
    // divisions of the index arithmetic: staged plane of a full and of the
    // last row block, WP, NGw, ncq, K, NT, W, CP / 4
    FastDiv d_plane, d_plane_last, d_WP, d_NGw, d_ncq, d_K, d_NT, d_W, d_cp4;
};

struct FwdArgs {
    const float *in;
    float *out;
    const float *K;   // n OIHW tensors
    double *logdet;   // optional: H W sum over layers and channels of log|K[c,c,self]|
    float *prepared;  // optional: the layers' prepared weights, by the first blocks (ppl each)
    int nfwd, ppl;    // forward blocks; preparation blocks per layer
    // split: the channel-split unit, its batch seen as (4B, C/4, H, W): image
    // b' = 4 b + g is quarter g, with corner g and weights K + g C^2 k^2 (one
    // layer per block; four layers prepared)
    int split;
    FwdPlan fp;
};

constexpr int kFwdThreads = 256;
constexpr int kFwdMinBlocks = 256;   // a block per compute unit of the chip

template <bool PADW>
__global__ __launch_bounds__(kFwdThreads) void forward_kernel(FwdArgs a) {
    extern __shared__ float sm[];
    const FwdPlan &fp = a.fp;
    const int nprep = a.split ? 4 : fp.n;   // layers prepared
    const int npre = a.prepared ? nprep * a.ppl : 0;
    if ((int)blockIdx.x < npre) {
        // the weights for the inverse, prepared by the launch's first blocks
        // (dispatched first: their latency chain is the longest; the forward
        // blocks do not wait for them)
        const int pb = blockIdx.x, layer = pb / a.ppl, part = pb - layer * a.ppl;
        prep_columns<kFwdThreads>(a.K + (size_t)layer * fp.C * fp.C * fp.K * fp.K,
                                  a.prepared + (size_t)layer * prep_layer_floats(fp.C, fp.K),
                                  fp.C, fp.K, nprep == 1 ? fp.corner0 : layer, part * kFwdThreads,
                                  part == 0, reinterpret_cast<double *>(sm));
        return;
    }
    const int C = fp.C, CP = fp.CP, H = fp.H, W = fp.W, K = fp.K, P = fp.P, WP = fp.WP;
    if (a.logdet && (int)blockIdx.x == npre) {
        // log|det| on a block of its own (next after the preparation blocks,
        // so it is dispatched early and no forward block carries its fp64
        // logarithms): H W times the sum over the layers (or the four
        // quarters) and channels of log|K[c,c,self]|, straight from K; lane
        // l takes entries l, l + 64, ..., and the 64 lane sums meet in a
        // fixed butterfly
        if (threadIdx.x < 64) {
            const int lane = threadIdx.x, nl = a.split ? 4 : fp.n;
            double v = 0.0;
            for (int m = lane; m < nl * C; m += 64) {
                const int q = m / C, c = m - q * C;
                int oh, ow;
                self_tap(a.split ? q : (fp.n == 1 ? fp.corner0 : q), K, oh, ow);
                const float d = a.K[(((size_t)q * C + c) * C + c) * K * K + oh * K + ow];
                v += log(fabs((double)d));
            }
            for (int off = 32; off > 0; off >>= 1)
                v += __shfl_xor(v, off);
            if (lane == 0)
                a.logdet[0] = (double)H * (double)W * v;
        }
        return;
    }
    const int lane = threadIdx.x & 63, kq = lane >> 4, li = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nwaves = blockDim.x >> 6;
    const int bid = blockIdx.x - npre - (a.logdet ? 1 : 0);
    const int b = bid / fp.nblk, blk = bid - b * fp.nblk;
    const int corner0 = a.split ? (b & 3) : fp.corner0;   // this block's (first) corner
    const float *Kb = a.K + (a.split ? (size_t)(b & 3) * fp.C * fp.C * fp.K * fp.K : 0);
    const int i0 = blk * fp.RB, rb = imin(H, i0 + fp.RB) - i0, HB = fp.HB;
    float *X = sm + fp.offI;
    float4 *Wf = reinterpret_cast<float4 *>(sm + fp.offW);
    int *Dq = reinterpret_cast<int *>(sm + fp.offD);
    const size_t HW = (size_t)H * W;
    const float *xb = a.in + (size_t)b * C * HW;
    float *yb = a.out + (size_t)b * C * HW;
    // weight fragments: Wf[(nt NGw + g) 64 + lane].e = K[co][ci][tap] for
    // co = 16 nt + li, quad u = 4 g + kq (tap u / ncq, ci = 4 (u % ncq) + e),
    // the channel mask applied (self tap: ci <= co only).  A round is two
    // fragments a thread: eight raw buffer loads over the layer's C^2 k^2
    // floats at (co C + ci) k^2 + tap (entries that do not exist read past
    // the end, which returns 0), all in flight before the stores.
    const int nfrag = fp.NT * fp.NGw * 64;
    auto wload = [&](int q, int base, float(&v)[2][4]) {
        const int K2 = K * K;
        const unsigned nrec = (unsigned)(C * C * K2 * 4);
        const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<float *>(Kb + (size_t)q * C * C * K2), (short)0, (int)nrec, kBufferWord3);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = base + h * blockDim.x;
            const int f = idx >> 6, ln = idx & 63;
            const int nt = fdiv(f, fp.d_NGw), g = f - nt * fp.NGw;
            const int co = nt * 16 + (ln & 15), u = 4 * g + (ln >> 4);
            const int t = fdiv(u, fp.d_ncq), cq = u - t * fp.ncq;
            const bool ok = idx < nfrag && u < fp.nq && co < C;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int ci = 4 * cq + e;
                const int off = ok && ci < C ? ((co * C + ci) * K2 + t) * 4 : (int)nrec;
                v[h][e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rk, off, 0, 0));
            }
        }
    };
    // the self tap (number selft) keeps ci <= co only
    auto wstore = [&](float(&v)[2][4], int base, int selft) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = base + h * blockDim.x;
            const int f = idx >> 6, ln = idx & 63;
            const int nt = fdiv(f, fp.d_NGw), g = f - nt * fp.NGw;
            const int co = nt * 16 + (ln & 15), u = 4 * g + (ln >> 4);
            const int t = fdiv(u, fp.d_ncq), cq = u - t * fp.ncq;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                if (t == selft && 4 * cq + e > co)
                    v[h][e] = 0.0f;
            if (idx < nfrag)
                Wf[idx] = make_float4(v[h][0], v[h][1], v[h][2], v[h][3]);
        }
    };
    // the first layer's first round of weights goes out ahead of the input,
    // so that one memory latency covers both
    float wpre[2][4];
    wload(0, threadIdx.x, wpre);
    // zero-bordered input rows i0 - HB .. i0 + rb + HB - 1: every element of
    // the block is written once, with x where the taps of this launch read
    // the image and zero elsewhere (outside the image, padding channels, and
    // for a single layer the halo side its corner never reads).  Images
    // past 2^31 bytes: one element an item, loads unconditional from clamped
    // indices, eight in flight per thread.
    {
        int oh0, ow0;
        self_tap(corner0, K, oh0, ow0);
        const int up = fp.n == 1 ? oh0 : HB, down = fp.n == 1 ? P - oh0 : HB;
        const int lo = imax(0, i0 - up), hi = imin(H, i0 + rb + down);   // rows read
        const int nrow = rb + 2 * HB, plane = nrow * WP, total = CP * plane;
        const FastDiv dpl = blk == fp.nblk - 1 ? fp.d_plane_last : fp.d_plane;
        if ((long long)C * HW * 4 < (1LL << 31)) {
            // (pixel, channel quad) items, pixel fastest: four raw buffer
            // loads over the image's C H W floats each (32-bit offsets; reads
            // past the image, padding channels included, return 0; a pixel
            // outside the rows or columns read takes an offset past the
            // end), then one 16-byte LDS store
            const unsigned nrec = (unsigned)(C * HW * 4);
            const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<float *>(xb), (short)0, (int)nrec, kBufferWord3);
            const int nitem = plane * (CP / 4);
            constexpr int U = 2;
            for (int base = threadIdx.x; base < nitem; base += U * blockDim.x) {
                float v[U][4];
                int dst[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int idx = base + u * blockDim.x;
                    const int q = fdiv(idx, dpl), px = idx - q * plane;
                    const int pr = fdiv(px, fp.d_WP), pc = px - pr * WP;
                    const int i = i0 - HB + pr, j = pc - P;
                    const bool ok = idx < nitem && i >= lo && i < hi && j >= 0 && j < W;
                    const unsigned off = ok ? (unsigned)(4 * q * HW + i * W + j) * 4u : nrec;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[u][e] = __builtin_bit_cast(
                            float, __builtin_amdgcn_raw_buffer_load_b32(
                                       rs, (int)(ok ? off + (unsigned)(e * HW * 4) : nrec), 0, 0));
                    dst[u] = idx < nitem ? px * CP + 4 * q : -1;
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        pin(v[u][e]);
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (dst[u] >= 0)
                        *reinterpret_cast<float4 *>(X + dst[u]) =
                            make_float4(v[u][0], v[u][1], v[u][2], v[u][3]);
            }
        } else {
            constexpr int U = 8;
            for (int base = threadIdx.x; base < total; base += U * blockDim.x) {
                float v[U];
                bool inb[U];
                int dst[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int idx = base + u * blockDim.x;
                    const int c = fdiv(idx, dpl), rem = idx - c * plane;
                    const int pr = fdiv(rem, fp.d_WP), pc = rem - pr * WP;
                    const int i = i0 - HB + pr, j = pc - P;
                    inb[u] = idx < total && c < C && i >= lo && i < hi && j >= 0 && j < W;
                    v[u] = xb[inb[u] ? c * HW + (size_t)i * W + j : 0];
                    dst[u] = idx < total ? rem * CP + c : -1;
                }
#pragma unroll
                for (int u = 0; u < U; ++u)
                    pin(v[u]);
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (dst[u] >= 0)
                        X[dst[u]] = inb[u] ? v[u] : 0.0f;
            }
        }
    }
    for (int q = 0; q < fp.n; ++q) {
        const int corner = fp.n == 1 ? corner0 : q;
        int oh, ow;
        self_tap(corner, K, oh, ow);
        const int nfrag = fp.NT * fp.NGw * 64;
        int wb = threadIdx.x;
        if (q == 0) {   // (the first round went out before the input)
            wstore(wpre, wb, oh * K + ow);
            wb += 2 * blockDim.x;
            if (!PADW && threadIdx.x < 64)   // the padding groups' zero fragment
                Wf[nfrag + threadIdx.x] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        for (; wb < nfrag; wb += 2 * blockDim.x) {
            float v[2][4];
            wload(q, wb, v);
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    pin(v[h][e]);
            wstore(v, wb, oh * K + ow);
        }
        // gather offset of quad u relative to the output pixel's address (taps
        // reach up/left too: offsets are signed); padding quads, whose
        // weights are zero, read the output pixel's own input (offset 0)
        for (int u = threadIdx.x; u < fp.NG * 4; u += blockDim.x) {
            const int t = fdiv(u, fp.d_ncq), cq = u - t * fp.ncq;
            const int ka = fdiv(t, fp.d_K), kb = t - ka * K;
            Dq[u] = u < fp.nq ? ((ka - oh) * WP + (kb - ow)) * CP + 4 * cq : 0;
        }
        __syncthreads();
        const bool last = q == fp.n - 1;
        float *Yo = sm + fp.offO;
        // rows of this layer's output the block computes, rlo .. rhi - 1: its
        // own, and in a band of a unit also those its later layers read
        // (TL: k-1 above for TR; TL, TR: 2(k-1) below for BL and BR; BL:
        // k-1 below for BR), within the image
        int rlo = i0, rhi = i0 + rb;
        if (fp.n > 1 && fp.nblk > 1) {
            rlo = imax(0, i0 - (q == 0 ? P : 0));
            rhi = imin(H, i0 + rb + (q < 2 ? 2 * P : q == 2 ? P : 0));
        }
        const int npix = (rhi - rlo) * W, nitem = ceil_div(npix, 16) * fp.NT;
        const int xrow = rlo - i0 + HB;   // staged row of output row rlo
        for (int item = wave; item < nitem; item += nwaves) {
            const int tile = fdiv(item, fp.d_NT), nt = item - tile * fp.NT;
            const int p = tile * 16 + li;
            const bool valid = p < npix;
            const int pc = valid ? p : 0;
            const int il = fdiv(pc, fp.d_W), j = pc - il * W;
            const int base = ((il + xrow) * WP + j + P) * CP;
            // four accumulators over the quad groups (group g -> g mod 4), joined
            // pairwise: the rounding chain is a quarter as long as a single one
            f32x4 part[4];
#pragma unroll
            for (int v = 0; v < 4; ++v)
                part[v] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            // four groups at a time (NG is a multiple of four), without a
            // branch: their offset reads, then their 16-byte gathers and
            // weight reads, then their MFMAs
            const float4 *S4 = reinterpret_cast<const float4 *>(sm);   // regions are 16-byte aligned
            const int zf = fp.NT * fp.NGw;   // (!PADW) the zero fragment
            for (int g0 = 0; g0 < fp.NG; g0 += 4) {
                int d[4];
#pragma unroll
                for (int v = 0; v < 4; ++v)
                    d[v] = Dq[4 * (g0 + v) + kq];
                float4 xv[4], wv[4];
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    xv[v] = S4[(fp.offI + base + d[v]) >> 2];
                    const int f = PADW || g0 + v < fp.NGr ? nt * fp.NGw + g0 + v : zf;
                    wv[v] = Wf[f * 64 + lane];
                }
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    part[v] = mfma4(wv[v].x, xv[v].x, part[v]);
                    part[v] = mfma4(wv[v].y, xv[v].y, part[v]);
                    part[v] = mfma4(wv[v].z, xv[v].z, part[v]);
                    part[v] = mfma4(wv[v].w, xv[v].w, part[v]);
                }
            }
            const f32x4 acc = (part[0] + part[1]) + (part[2] + part[3]);
            const int co0 = nt * 16 + 4 * kq;
            if (last) {
                if (valid) {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (co0 + r < C)
                            yb[(co0 + r) * HW + (size_t)(rlo + il) * W + j] = acc[r];
                }
            } else if (valid && co0 < CP) {
                *reinterpret_cast<f32x4 *>(Yo + (size_t)p * CP + co0) = acc;
            }
        }
        if (!last) {   // this layer's output is the next one's input
            __syncthreads();
            for (int idx = threadIdx.x; idx < npix * CP / 4; idx += blockDim.x) {
                const int p = fdiv(idx, fp.d_cp4), c4 = idx - p * (CP / 4);
                const int il = fdiv(p, fp.d_W), j = p - il * W;
                reinterpret_cast<float4 *>(X)[((il + xrow) * WP + j + P) * (CP / 4) + c4] =
                    reinterpret_cast<const float4 *>(Yo)[idx];
            }
            __syncthreads();
        }
    }
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

// Plans of every level, LDS size and waves of an inverse chain launch.
// Returns FINC_EUNSUPPORTED when a level's work split or the level-to-level
// hand-over does not fit one workgroup.
int plan_inverse(InvArgs &a, size_t *lds_bytes, int *threads) {
    int lds = 0, nw = 1;
    for (int l = 0; l < a.L; ++l) {
        Plan &p = a.lv[l].pl;
        if (!make_plan(p.C, p.H, p.W, p.K, p))
            return FINC_EUNSUPPORTED;
        lds = imax(lds, p.lds_floats);
        nw = imax(nw, p.NW);
        // the unsqueeze reads the level above's solution (its image, not the
        // zero border) while writing this level's input: the two must not
        // overlap
        if (l > 0) {
            const Plan &u = a.lv[l - 1].pl;
            const int last = u.offX + ((u.H - 1 + u.P) * u.WP + u.W - 1 + u.P) * u.CP + u.CP - 1;
            if (last >= p.offY)
                return FINC_EUNSUPPORTED;
        }
    }
    *lds_bytes = (size_t)lds * sizeof(float);
    *threads = nw * kWave;
    return FINC_OK;
}

// Work split and LDS layout of a forward launch: n = 1 splits each image into
// blocks of rows (up to eight 16-pixel tiles a block, and a block per compute
// unit when the batch allows); a unit (n = 4) keeps whole images.
// whole: a unit keeps whole images (in place: an image must be read whole
// before any of it is written).
FwdPlan make_fwd_plan(int C, int H, int W, int K, int n, int corner0, int B, bool whole) {
    FwdPlan p;
    memset(&p, 0, sizeof(p));
    p.C = C;
    p.CP = round_up4(C);
    p.H = H;
    p.W = W;
    p.K = K;
    p.P = K - 1;
    p.WP = W + 2 * p.P;
    p.NT = ceil_div(p.CP, 16);
    p.ncq = p.CP / 4;
    p.nq = K * K * p.ncq;
    // quad groups, padded to a multiple of four (the MFMA loop takes four at
    // a time; padding groups have zero weights and read the pixel itself)
    p.NGr = ceil_div(p.nq, 4);
    p.NG = round_up4(p.NGr);
    p.padw = 1;
    p.n = n;
    p.corner0 = corner0;
    int rb_min;
    if (n == 1) {
        // row blocks of about 128 pixels (eight 16-pixel tiles, two a wave),
        // halved while the grid has fewer blocks than the chip has compute
        // units, but never below a full tile: every block stages all of the
        // layer's weights, so more and smaller blocks pay that again for less
        // work
        rb_min = imin(H, ceil_div(16, W));
        p.RB = imax(rb_min, imin(H, ceil_div(128, W)));
        while (p.RB > rb_min && (long long)B * ceil_div(H, p.RB) < kFwdMinBlocks)
            p.RB = imax(rb_min, p.RB / 2);
    } else {
        // a unit keeps whole images, or, with fewer of them than compute
        // units, bands of rows: TL and TR read k-1 rows up, BL and BR k-1
        // rows down, so a band stages 2(k-1) rows each side and each layer
        // also computes the rows of the halo its later layers read
        rb_min = imin(H, imax(ceil_div(16, W), 2 * p.P));
        p.RB = H;
        while (!whole && p.RB > rb_min && (long long)B * ceil_div(H, p.RB) < kFwdMinBlocks)
            p.RB = imax(rb_min, p.RB / 2);
    }
    // LDS layout for the rows of a block; blocks (bands, for a unit not
    // computed in place) are halved further while it does not fit
    auto layout = [&] {
        p.nblk = ceil_div(H, p.RB);
        p.HB = n > 1 && p.nblk > 1 ? 2 * p.P : p.P;
        p.offI = 0;
        p.offO = (p.RB + 2 * p.HB) * p.WP * p.CP;
        p.offW = p.offO + (n > 1 ? imin(H, p.RB + 3 * p.P) * W * p.CP : 0);
        p.NGw = p.padw ? p.NG : p.NGr;
        p.offD = p.offW + (p.NT * p.NGw + (p.padw ? 0 : 1)) * 256;   // (+ the zero fragment)
        p.lds_floats = p.offD + round_up4(4 * p.NG);
    };
    const int rb0 = p.RB;
    auto fit = [&] {
        p.RB = rb0;
        layout();
        while ((size_t)p.lds_floats * sizeof(float) > kLdsBytes && p.RB > rb_min &&
               !(n > 1 && whole)) {
            p.RB = imax(rb_min, p.RB / 2);
            layout();
        }
    };
    fit();
    if ((size_t)p.lds_floats * sizeof(float) > kLdsBytes && p.NG > p.NGr) {
        p.padw = 0;   // the padding groups' fragments do not fit: one zero fragment
        fit();
    }
    const int rb_last = H - (p.nblk - 1) * p.RB;
    p.d_plane = make_fastdiv((p.RB + 2 * p.HB) * p.WP);
    p.d_plane_last = make_fastdiv((rb_last + 2 * p.HB) * p.WP);
    p.d_WP = make_fastdiv(p.WP);
    p.d_NGw = make_fastdiv(p.NGw);
    p.d_ncq = make_fastdiv(p.ncq);
    p.d_K = make_fastdiv(K);
    p.d_NT = make_fastdiv(p.NT);
    p.d_W = make_fastdiv(W);
    p.d_cp4 = make_fastdiv(p.ncq);
    return p;
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
    for (int first = 0; first < n; first += kMaxLayersPerPrep) {
        PrepArgs a;
        memset(&a, 0, sizeof(a));
        a.C = C;
        a.k = k;
        a.n = n - first < kMaxLayersPerPrep ? n - first : kMaxLayersPerPrep;
        a.K = K + (size_t)first * C * C * k * k;
        a.out = out + (size_t)first * prep_layer_floats(C, k);
        for (int q = 0; q < a.n; ++q)
            a.corner_bits[q >> 4] |= (unsigned)(corners[first + q] & 3) << (2 * (q & 15));
        dim3 grid((k * k * CP + kPrepThreads - 1) / kPrepThreads, a.n);
        hipLaunchKernelGGL(prep_kernel, grid, dim3(kPrepThreads), 0, stream, a);
        const int rc = launched();
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

// The inverse kernel for a workgroup size (threads), a mode and quad groups
// per wave.
const void *inverse_instance(int threads, int mode, int ng) {
#if FINC_PART == -1
#define FINC_ENTRY(g) &inverse_instance_of<kGroupThreads[g], kGroupMode[g]>,
#else
#define FINC_ENTRY(g) &finc_parts::inverse_group_##g,
#endif
    static const void *(*const groups[kInverseGroups])(int) = {FINC_GROUPS(FINC_ENTRY)};
#undef FINC_ENTRY
    int m = -1;
    for (int i = 0; i < kModesPerSize; ++i)
        if (kGroupModes[i] == mode)
            m = i;
    if (m < 0)
        return nullptr;
    const int t = threads <= 256 ? 0 : threads <= 512 ? 1 : 2;
    return groups[kModesPerSize * t + m](ng);
}

// How an inverse chain is launched: the kernel instance (workgroup size,
// mode, quad groups per wave), its LDS, and whether the image is streamed
// (one stream-form launch per layer) because it does not fit in LDS.
struct InvChoice {
    int streamed;
    int threads, mode, ng;
    int compact;   // some level keeps compact partial tiles
    size_t lds;
    Plan sp;   // the stream form's plan (streamed only)
};

// The choice for a chain whose workgroups may use lds_lim bytes of LDS:
// FINC_EUNSUPPORTED when neither the LDS-resident chain nor (a single level of
// layers without actnorm) the stream form fits.  Host arithmetic only.
int choose_inverse(InvArgs &a, size_t lds_lim, InvChoice &c) {
    memset(&c, 0, sizeof(c));
    size_t lds = 0;
    int threads = 0;
    int rc = plan_inverse(a, &lds, &threads);
    if (rc == FINC_OK && lds > lds_lim)
        rc = FINC_EUNSUPPORTED;
    if (rc == FINC_EUNSUPPORTED && a.L == 1 && !a.lv[0].scale && !a.split) {
        const Level &l0 = a.lv[0];
        if (a.n_units * a.lpu < 1 || !make_plan(l0.pl.C, l0.pl.H, l0.pl.W, l0.pl.K, c.sp, true))
            return FINC_EUNSUPPORTED;
        c.lds = (size_t)c.sp.lds_floats * sizeof(float);
        if (c.lds > lds_lim)
            return FINC_EUNSUPPORTED;
        c.streamed = 1;
        c.threads = c.sp.NW * kWave;
        c.mode = kCritRegs | kOneLayer | kStream;
        c.ng = plan_groups(c.sp);
        c.compact = c.sp.compact;
        return FINC_OK;
    }
    if (rc != FINC_OK)
        return rc;
    int ng = 1, nreg = 0;
    for (int l = 0; l < a.L; ++l) {
        const Plan &p = a.lv[l].pl;
        ng = imax(ng, plan_groups(p));
        nreg += p.regcrit;
        c.compact |= p.compact;
    }
    // levels of one launch share the critical form: a stack whose levels
    // differ in it runs them in launches of their own
    if (nreg != 0 && nreg != a.L)
        return FINC_EUNSUPPORTED;
    int mode = nreg == a.L ? kCritRegs : kCritGather;
    if (a.L == 1 && a.n_units * a.lpu == 1 && !a.lv[0].scale)
        mode |= kOneLayer;   // (a single level has one critical form)
    c.threads = threads;
    c.mode = mode;
    c.ng = ng;
    c.lds = lds;
    // a single layer held in LDS with a register-fed critical path (one
    // channel tile): one more (idle) wave stores the rows of the solution as
    // they complete, on a SIMD that no critical wave uses (waves go to the
    // four SIMDs in turn; waves skipped for that are idle too); not for rows
    // of more than kDrainRounds values a lane.  (Chains of layers keep the
    // store after the last diagonal: their extra wave would wait at every
    // layer's barriers; the gathering critical forms keep their registers.)
    a.drain = 0;
    if ((mode & kOneLayer) != 0 && a.lv[0].pl.regcrit) {
        const Plan &p = a.lv[0].pl;
        int w = p.NW;
        while (p.T < 4 && w % 4 < p.T)
            ++w;
        if (p.C * p.W <= kDrainRounds * kWave && w < kMaxWaves) {
            a.drain = w + 1;
            c.threads = (w + 1) * kWave;
        }
    }
    return FINC_OK;
}

// A single level of layers without actnorm whose image does not fit in LDS:
// one stream-form launch per layer, in place on the output after the first
// (each workgroup reads a pixel's input before it writes the pixel).
int launch_streamed(const InvArgs &a, const InvChoice &ch, int B, hipStream_t stream) {
    const Level &l0 = a.lv[0];
    const Plan &p = ch.sp;
    const size_t lds = ch.lds;
    const int threads = ch.threads;
    int rc = FINC_OK;
    const void *k = inverse_instance(threads, ch.mode, ch.ng);
    if (!k)
        return FINC_EUNSUPPORTED;
    if (hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
        (void)hipGetLastError();
    for (int n = 0; n < a.n_units * a.lpu; ++n) {
        const int u = a.n_units - 1 - n / a.lpu, q = a.lpu - 1 - n % a.lpu;
        InvArgs s;
        memset(&s, 0, sizeof(s));
        s.L = s.n_units = s.lpu = 1;
        s.corner0 = a.lpu == 1 ? a.corner0 : q;
        s.out = a.out;
        s.lv[0].z = n == 0 ? l0.z : a.out;
        s.lv[0].prep = l0.prep + (size_t)(u * a.lpu + q) * p.lstride;
        s.lv[0].pl = p;
        s.steps = a.steps;   // (set for single layers only)
        s.stamps = a.stamps;
        void *args[] = {&s};
        (void)hipLaunchKernel(k, dim3(B), dim3(threads), args, lds, stream);
        rc = launched();
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

// ---- banded stream form: images whose level does not fit one workgroup --

__global__ void zero_ints_kernel(int *p, int n) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        p[i] = 0;
}

// The band height of a single layer of C channels on H x W images: the
// tallest multiple of 16 rows, at most 128 and at most the image's rows
// rounded up, whose stream-form plan fits a workgroup (registers for one
// phase's input, LDS); false if none does (C > 16 or k = 1).
bool banded_choice(int C, int H, int W, int k, size_t lds_lim, InvChoice &c, int &R, int &nb) {
    memset(&c, 0, sizeof(c));
    for (R = imin(128, ceil_div(H, 16) * 16); R >= 16; R -= 16) {
        if (!make_plan(C, R, W, k, c.sp, true))
            continue;
        c.lds = (size_t)c.sp.lds_floats * sizeof(float);
        if (c.lds > lds_lim)
            continue;
        c.streamed = 1;
        c.threads = c.sp.NW * kWave;
        c.mode = kCritRegs | kOneLayer | kStream | kBanded;
        c.ng = plan_groups(c.sp);
        c.compact = c.sp.compact;
        nb = ceil_div(H, R);
        return true;
    }
    return false;
}

inline size_t banded_flag_ints(int B, int nb) { return 2 + (size_t)B * nb; }

// n_layers layers (1: corner `corner`; 4: a unit, run BR, BL, TR, TL), each
// one launch of B * nb workgroups after the flags are cleared; the layers
// after the first work in place on x.
int launch_banded(const float *y, float *x, const float *prep, int n_layers, int corner, int B,
                  int C, int H, int W, int k, int *bflags, hipStream_t stream) {
    size_t lim = kLdsBytes;
    if (B > 0) {
        const int lrc = lds_limit(&lim);
        if (lrc != FINC_OK)
            return lrc;
    }
    InvChoice ch;
    int R = 0, nb = 0;
    if (!banded_choice(C, H, W, k, lim, ch, R, nb))
        return FINC_EUNSUPPORTED;
    if (B == 0)
        return FINC_OK;
    const void *kern = inverse_instance(ch.threads, ch.mode, ch.ng);
    if (!kern)
        return FINC_EUNSUPPORTED;
    if (hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)ch.lds) !=
        hipSuccess)
        (void)hipGetLastError();
    const int nflags = (int)banded_flag_ints(B, nb);
    for (int n = 0; n < n_layers; ++n) {
        const int q = n_layers - 1 - n;
        hipLaunchKernelGGL(zero_ints_kernel, dim3(imin(ceil_div(nflags, 256), 1024)), dim3(256), 0,
                           stream, bflags, nflags);
        int rc = launched();
        if (rc != FINC_OK)
            return rc;
        InvArgs s;
        memset(&s, 0, sizeof(s));
        s.L = s.n_units = s.lpu = 1;
        s.corner0 = n_layers == 1 ? corner : q;
        s.out = x;
        s.lv[0].z = n == 0 ? y : x;
        s.lv[0].prep = prep + (size_t)(n_layers == 1 ? 0 : q) * ch.sp.lstride;
        s.lv[0].pl = ch.sp;
        s.nbands = nb;
        s.img_H = H;
        s.bflags = bflags;
        void *args[] = {&s};
        (void)hipLaunchKernel(kern, dim3(B * nb), dim3(ch.threads), args, ch.lds, stream);
        rc = launched();
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

int launch_inverse_chain(InvArgs &a, int B, hipStream_t stream) {
    size_t lim = kLdsBytes;
    if (B > 0) {
        const int lrc = lds_limit(&lim);
        if (lrc != FINC_OK)
            return lrc;
    }
    InvChoice ch;
    const int rc = choose_inverse(a, lim, ch);
    if (rc != FINC_OK)
        return rc;
    if (B == 0)
        return FINC_OK;
    if (ch.streamed)
        return launch_streamed(a, ch, B, stream);   // the image does not fit in LDS
    const int threads = ch.threads, mode = ch.mode, ng = ch.ng;
    const size_t lds = ch.lds;
    {
        const Plan &top = a.lv[0].pl, &last = a.lv[a.L - 1].pl;
        if (a.out_stride == 0)
            a.out_stride = last.C * last.H * last.W;
        const bool in4 = (top.H * top.W) % 4 == 0 && ((uintptr_t)a.lv[0].z & 15u) == 0;
        const bool out4 =
            last.W % 4 == 0 && ((uintptr_t)a.out & 15u) == 0 && a.out_stride % 4 == 0;
        a.vec = (in4 ? 1 : 0) | (out4 ? 2 : 0);
    }
    const void *k = inverse_instance(threads, mode, ng);
    if (!k)
        return FINC_EUNSUPPORTED;
    if (hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
        (void)hipGetLastError();   // not needed on every runtime; the launch check decides
    void *args[] = {&a};
    (void)hipLaunchKernel(k, dim3(B), dim3(threads), args, lds, stream);
    return launched();
}

// true if the levels of a chain would each pick a different kernel instance
// than the chain as a whole (work split, quad groups or critical form)
bool levels_differ(const InvArgs &a) {
    Plan p0;
    for (int l = 0; l < a.L; ++l) {
        Plan p = a.lv[l].pl;
        if (!make_plan(p.C, p.H, p.W, p.K, p))
            return false;   // (the chain launch reports it)
        if (l == 0)
            p0 = p;
        else if (p.NW != p0.NW || plan_groups(p) != plan_groups(p0) || p.regcrit != p0.regcrit)
            return true;
    }
    return false;
}

// Channels up to which the forward launch also prepares the inverse's
// weights in its own blocks (their LDS is small); wider layers get a
// separate preparation launch.
constexpr int kFusedPrepMaxC = 16;

// split: the channel-split unit on (B, 4 C, H, W) seen as (4B, C, H, W), C
// here being the quarter's channels (n = 1).
int launch_forward(const float *x, float *y, const float *K, double *logdet, float *prepared,
                   int B, int C, int H, int W, int k, int n, int corner0, int split,
                   hipStream_t stream) {
    FwdArgs a;
    memset(&a, 0, sizeof(a));
    a.in = x;
    a.out = y;
    a.K = K;
    a.logdet = logdet;
    a.split = split;
    a.fp = make_fwd_plan(C, H, W, k, n, corner0, B, x == y);
    if (B == 0)
        return FINC_OK;
    const int nprep = split ? 4 : n;
    const bool fuse = prepared && C <= kFusedPrepMaxC;
    a.nfwd = B * a.fp.nblk;
    a.ppl = ceil_div(k * k * round_up4(C), kFwdThreads);
    a.prepared = fuse ? prepared : nullptr;
    size_t lds = (size_t)a.fp.lds_floats * sizeof(float);
    if (fuse)
        lds = lds > prep_lds_doubles(C, kFwdThreads) * sizeof(double)
                  ? lds
                  : prep_lds_doubles(C, kFwdThreads) * sizeof(double);
    int rc = check_lds(lds);
    if (rc != FINC_OK)
        return rc;
    const void *fk = a.fp.padw ? reinterpret_cast<const void *>(forward_kernel<true>)
                               : reinterpret_cast<const void *>(forward_kernel<false>);
    if (hipFuncSetAttribute(fk,
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        (void)hipGetLastError();   // not needed on every runtime; the launch check decides
    // preparation blocks, then the log|det| block, then the forward blocks
    const unsigned blocks = (unsigned)(a.nfwd + (fuse ? nprep * a.ppl : 0) + (logdet ? 1 : 0));
    void *args[] = {&a};
    (void)hipLaunchKernel(fk, dim3(blocks), dim3(kFwdThreads), args, lds, stream);
    rc = launched();
    if (rc != FINC_OK || !prepared || fuse)
        return rc;
    int corners[4] = {corner0, FINC_TR, FINC_BL, FINC_BR};
    if (nprep > 1)
        corners[0] = FINC_TL;
    return launch_prep(K, nprep, corners, C, k, prepared, stream);
}

Level level(const float *z, const void *prep, const float *scale, const float *bias, int C,
            int H, int W, int k) {
    Level v;
    memset(&v, 0, sizeof(v));
    v.z = z;
    v.prep = (const float *)prep;
    v.scale = scale;
    v.bias = bias;
    v.pl.C = C;
    v.pl.H = H;
    v.pl.W = W;
    v.pl.K = k;
    return v;
}

// x/y overlap rule of the inverse: identical or disjoint.
bool inverse_alias_ok(const void *y, const void *x, size_t bytes) {
    return x == y || !overlap(x, bytes, y, bytes);
}

size_t stack_level_bytes(int l, int U, int C1, int k) {
    return (size_t)U * 4 * prep_layer_floats(C1 << l, k) * sizeof(float);
}

// Channel-split unit: C a multiple of 4; seen as (4B, C/4, H, W).
bool valid_split(int B, int C, int H, int W, int k) {
    return C >= 4 && C % 4 == 0 && B >= 0 && B <= (1 << 28) &&
           valid_shape(4 * B, C / 4, H, W, k);
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

// Arguments of a stack call.  x (written) must be clear of every buffer the
// call reads: the latents, scale, bias, and K or the prepared weights (wb);
// a workspace the call writes (wb_written) must be clear of all of them too.
bool stack_call_ok(const float *const *z, const float *x, const float *scale,
                   const float *bias, int B, int L, int U, int C1, int H1, int W1, int k,
                   const float *K, const void *wb, bool wb_written) {
    if (!valid_stack(B, L, U, C1, H1, W1, k) || !z || !x || !scale || !bias || !wb)
        return false;
    for (int l = 0; l < L; ++l)
        if (!z[l])
            return false;
    size_t sb = 0, kb = 0;   // bytes of scale (= of bias), of K
    for (int l = 0; l < L; ++l) {
        sb += (size_t)U * (C1 << l) * sizeof(float);
        kb += (size_t)U * 4 * (C1 << l) * (C1 << l) * k * k * sizeof(float);
    }
    const size_t wbytes = finc_stack_workspace_bytes(L, U, C1, k);
    const size_t xbytes = (size_t)B * C1 * H1 * W1 * sizeof(float);
    auto clear = [&](const void *p, size_t n) {
        return !overlap(p, n, x, xbytes) && !(wb_written && overlap(p, n, wb, wbytes));
    };
    for (int l = 0; l < L; ++l) {
        const int C = C1 << l, H = H1 >> l, W = W1 >> l;
        const size_t zb = (size_t)B * (l == L - 1 ? C : C / 2) * H * W * sizeof(float);
        if (!clear(z[l], zb))
            return false;
    }
    if (!clear(scale, sb) || !clear(bias, sb) || (K && !clear(K, kb)))
        return false;
    return !overlap(wb, wbytes, x, xbytes);
}

// Prepared weights of finc_inverse_noalloc: one layer at the largest shape
// the library accepts (C = 64, k = 7: 803,072 bytes), in a device array of
// the library's own.  Each device holds its copy (at its own address) until
// the process ends.  In host code `scratch` names a host-side stand-in; the
// device address comes from hipGetSymbolAddress, once per device.
constexpr size_t kScratchBytes = 1u << 20;
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_ptr[kMaxDevices];

// Device address of this device's scratch array (looked up on the first call
// on the device, with that device current).
int scratch_of_device(void **out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return FINC_EHIP;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_ptr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
            return FINC_EHIP;
        scratch_ptr[dev] = p;
    }
    *out = scratch_ptr[dev];
    return FINC_OK;
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

int finc_forward_plan(int kind, int B, int C, int H, int W, int k, int in_place, int *info) {
    if (!info || (kind != FINC_PLAN_LAYER && kind != FINC_PLAN_UNIT && kind != FINC_PLAN_SPLIT))
        return FINC_EINVAL;
    if (kind == FINC_PLAN_SPLIT ? !valid_split(B, C, H, W, k) : !valid_shape(B, C, H, W, k))
        return FINC_EINVAL;
    const bool unit = kind == FINC_PLAN_UNIT;
    const FwdPlan fp = kind == FINC_PLAN_SPLIT
                           ? make_fwd_plan(C / 4, H, W, k, 1, FINC_TL, 4 * B, false)
                           : make_fwd_plan(C, H, W, k, unit ? 4 : 1, FINC_TL, B,
                                           unit && in_place);
    info[0] = fp.nblk;
    info[1] = fp.RB;
    info[2] = fp.lds_floats * (int)sizeof(float);
    return (size_t)info[2] <= kLdsBytes ? FINC_OK : FINC_EUNSUPPORTED;
}

static void put_choice(const InvChoice &c, int *dst) {
    dst[0] = c.threads;
    dst[1] = c.mode;
    dst[2] = c.ng;
    dst[3] = c.streamed;
    dst[4] = (int)c.lds;
    dst[5] = c.compact;
}

int finc_inverse_plan(int kind, int L, int U, int C, int H, int W, int k, int *info,
                      int max_launches) {
    if (!info || max_launches < 1)
        return FINC_EINVAL;
    static const float dummy[1] = {0.0f};   // stands for a non-null scale / bias
    InvArgs a;
    memset(&a, 0, sizeof(a));
    a.L = 1;
    a.n_units = 1;
    a.lpu = 1;
    if (kind == FINC_PLAN_LAYER) {
        if (!valid_shape(1, C, H, W, k))
            return FINC_EINVAL;
        a.lv[0] = level(dummy, nullptr, nullptr, nullptr, C, H, W, k);
    } else if (kind == FINC_PLAN_UNIT) {
        if (!valid_shape(1, C, H, W, k))
            return FINC_EINVAL;
        a.lv[0] = level(dummy, nullptr, nullptr, nullptr, C, H, W, k);
        a.lpu = 4;
    } else if (kind == FINC_PLAN_SPLIT) {
        if (!valid_split(1, C, H, W, k))
            return FINC_EINVAL;
        a.lv[0] = level(dummy, nullptr, nullptr, nullptr, C / 4, H, W, k);
        a.split = 1;
    } else if (kind == FINC_PLAN_STACK) {
        if (!valid_stack(1, L, U, C, H, W, k))
            return FINC_EINVAL;
        for (int l = 0; l < L; ++l)
            a.lv[L - 1 - l] = level(dummy, nullptr, dummy, dummy, C << l, H >> l, W >> l, k);
        a.L = L;
        a.n_units = U;
        a.lpu = 4;
        if (levels_differ(a)) {
            if (max_launches < L)
                return FINC_EINVAL;
            for (int i = 0; i < L; ++i) {
                InvArgs s;
                memset(&s, 0, sizeof(s));
                s.lv[0] = a.lv[i];
                s.L = 1;
                s.n_units = U;
                s.lpu = 4;
                s.hin = i > 0 ? dummy : nullptr;
                InvChoice c;
                const int rc = choose_inverse(s, kLdsBytes, c);
                if (rc != FINC_OK)
                    return rc;
                put_choice(c, info + 6 * i);
            }
            return L;
        }
    } else {
        return FINC_EINVAL;
    }
    InvChoice c;
    const int rc = choose_inverse(a, kLdsBytes, c);
    if (rc != FINC_OK)
        return rc;
    put_choice(c, info);
    return 1;
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

// The prepared-weights side output of a forward call: aligned, and clear of
// the activations and weights.
bool prepared_out_ok(const void *prepared, size_t pbytes, const void *x, const void *y,
                     size_t bytes, const void *K, size_t kbytes) {
    return aligned256(prepared) && !overlap(prepared, pbytes, x, bytes) &&
           !overlap(prepared, pbytes, y, bytes) && !overlap(prepared, pbytes, K, kbytes);
}

int finc_forward(const float *x, float *y, const float *K, double *logdet, void *prepared,
                 int B, int C, int H, int W, int k, int corner, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !valid_corner(corner) || !x || !y || !K)
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (overlap(x, bytes, y, bytes))
        return FINC_EINVAL;
    if (prepared && !prepared_out_ok(prepared, finc_workspace_bytes(C, k, 1), x, y, bytes, K,
                                     (size_t)C * C * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0) {   // nothing to run the forward on: the side outputs on their own
        int rc = FINC_OK;
        if (logdet)
            rc = finc_logdet(K, C, k, corner, H, W, logdet, stream);
        if (rc == FINC_OK && prepared)
            rc = finc_prepare(K, 1, &corner, C, k, prepared, stream);
        return rc;
    }
    return launch_forward(x, y, K, logdet, (float *)prepared, B, C, H, W, k, 1, corner, 0,
                          stream);
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
    a.lv[0] = level(y, prepared, nullptr, nullptr, C, H, W, k);
    a.out = x;
    a.L = 1;

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
    if (B == 0)   // nothing to launch; the shape is still checked
        return finc_inverse_prepared(y, x, workspace, 0, C, H, W, k, corner, stream);
    const int rc = finc_prepare(K, 1, &corner, C, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_inverse_prepared(y, x, workspace, B, C, H, W, k, corner, stream);
}

int finc_inverse_noalloc(const float *y, float *x, const float *K, int B, int C, int H, int W,
                         int k, int corner, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !valid_corner(corner) || !x || !y || !K)
        return FINC_EINVAL;
    if (finc_workspace_bytes(C, k, 1) > kScratchBytes)
        return FINC_EUNSUPPORTED;   // (no shape the library accepts gets here)
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (!inverse_alias_ok(y, x, bytes))
        return FINC_EINVAL;
    if (B == 0) {   // nothing to launch; the shape is still checked
        int info[6];
        const int n = finc_inverse_plan(FINC_PLAN_LAYER, 1, 1, C, H, W, k, info, 1);
        return n < 0 ? n : FINC_OK;
    }
    void *ws = nullptr;
    const int rc = scratch_of_device(&ws);
    if (rc != FINC_OK)
        return rc;
    return finc_inverse(y, x, K, B, C, H, W, k, corner, ws, stream);
}

int finc_unit_forward(const float *x, float *y, const float *K4, double *logdet,
                      void *prepared4, int B, int C, int H, int W, int k, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !x || !y || !K4)
        return FINC_EINVAL;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (overlap(x, bytes, y, bytes) && x != y)
        return FINC_EINVAL;
    if (prepared4 && !prepared_out_ok(prepared4, finc_workspace_bytes(C, k, 4), x, y, bytes, K4,
                                      (size_t)4 * C * C * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0) {
        int rc = FINC_OK;
        if (logdet)
            rc = finc_unit_logdet(K4, C, k, H, W, logdet, stream);
        if (rc == FINC_OK && prepared4) {
            const int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
            rc = finc_prepare(K4, 4, corners, C, k, prepared4, stream);
        }
        return rc;
    }
    return launch_forward(x, y, K4, logdet, (float *)prepared4, B, C, H, W, k, 4, FINC_TL, 0,
                          stream);
}

int finc_unit_logdet(const float *K4, int C, int k, int H, int W, double *out,
                     hipStream_t stream) {
    if (!valid_shape(1, C, H, W, k) || !K4 || !out)
        return FINC_EINVAL;
    hipLaunchKernelGGL(logdet_kernel, dim3(1), dim3(kWave), 0, stream, K4, 4, FINC_TL, C, k,
                       H, W, out);
    return launched();
}

int finc_split_logdet(const float *Kq4, int C, int k, int H, int W, double *out,
                      hipStream_t stream) {
    if (!valid_split(1, C, H, W, k))
        return FINC_EINVAL;
    return finc_unit_logdet(Kq4, C / 4, k, H, W, out, stream);   // same four corners
}

int finc_split_forward(const float *x, float *y, const float *Kq4, double *logdet,
                       void *prepared4, int B, int C, int H, int W, int k, hipStream_t stream) {
    if (!valid_split(B, C, H, W, k) || !x || !y || !Kq4)
        return FINC_EINVAL;
    const int Cq = C / 4;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (overlap(x, bytes, y, bytes))
        return FINC_EINVAL;
    if (prepared4 &&
        !prepared_out_ok(prepared4, finc_workspace_bytes(Cq, k, 4), x, y, bytes, Kq4,
                         (size_t)4 * Cq * Cq * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0) {
        int rc = FINC_OK;
        if (logdet)
            rc = finc_split_logdet(Kq4, C, k, H, W, logdet, stream);
        if (rc == FINC_OK && prepared4) {
            const int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
            rc = finc_prepare(Kq4, 4, corners, Cq, k, prepared4, stream);
        }
        return rc;
    }
    return launch_forward(x, y, Kq4, logdet, (float *)prepared4, 4 * B, Cq, H, W, k, 1, FINC_TL,
                          1, stream);
}

int finc_split_inverse_prepared(const float *y, float *x, const void *prepared4, int B, int C,
                                int H, int W, int k, hipStream_t stream) {
    if (!valid_split(B, C, H, W, k) || !x || !y || !prepared4 || !aligned256(prepared4))
        return FINC_EINVAL;
    const int Cq = C / 4;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    if (!inverse_alias_ok(y, x, bytes) ||
        overlap(x, bytes, prepared4, finc_workspace_bytes(Cq, k, 4)))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    a.lv[0] = level(y, prepared4, nullptr, nullptr, Cq, H, W, k);
    a.out = x;
    a.L = 1;
    a.n_units = 1;
    a.lpu = 1;
    a.corner0 = FINC_TL;
    a.split = 1;
    return launch_inverse_chain(a, 4 * B, stream);
}

// The diagnostics' shared path: the prepared inverse of a layer or of a
// channel-split unit with `per_wave` values of `elem` bytes written for every
// wave of every workgroup into buf (steps: ints; stamps: long longs).
static int inverse_diagnostic(int kind, const float *y, float *x, const void *prepared, int B,
                              int C, int H, int W, int k, int corner, void *buf, size_t elem,
                              int per_wave, int max_elems, hipStream_t stream) {
    if ((kind != FINC_PLAN_LAYER && kind != FINC_PLAN_SPLIT) || !buf || max_elems < 0 ||
        !valid_corner(corner))
        return FINC_EINVAL;
    const bool split = kind == FINC_PLAN_SPLIT;
    if (split ? !valid_split(B, C, H, W, k) : !valid_shape(B, C, H, W, k))
        return FINC_EINVAL;
    if (!x || !y || !prepared || !aligned256(prepared))
        return FINC_EINVAL;
    const int Cl = split ? C / 4 : C;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t pb = finc_workspace_bytes(Cl, k, split ? 4 : 1);
    int info[6];
    const int n = finc_inverse_plan(kind, 1, 1, C, H, W, k, info, 1);
    if (n < 0)
        return n;
    const long long count = (long long)(split ? 4 * B : B) * (info[0] / 64) * per_wave;
    if (count > max_elems)
        return FINC_EINVAL;
    const size_t bb = (size_t)count * elem;
    if (!inverse_alias_ok(y, x, bytes) || overlap(x, bytes, prepared, pb) ||
        overlap(buf, bb, x, bytes) || overlap(buf, bb, y, bytes) || overlap(buf, bb, prepared, pb))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    a.lv[0] = level(y, prepared, nullptr, nullptr, Cl, H, W, k);
    a.out = x;
    a.L = 1;
    a.n_units = 1;
    a.lpu = 1;
    a.corner0 = split ? FINC_TL : corner;
    a.split = split ? 1 : 0;
    if (elem == sizeof(int))
        a.steps = static_cast<int *>(buf);
    else
        a.stamps = static_cast<long long *>(buf);
    const int rc = launch_inverse_chain(a, split ? 4 * B : B, stream);
    return rc == FINC_OK ? (int)count : rc;
}

int finc_inverse_steps(int kind, const float *y, float *x, const void *prepared, int B, int C,
                       int H, int W, int k, int corner, int *steps, int max_steps,
                       hipStream_t stream) {
    return inverse_diagnostic(kind, y, x, prepared, B, C, H, W, k, corner, steps, sizeof(int), 1,
                              max_steps, stream);
}

int finc_inverse_timeline(int kind, const float *y, float *x, const void *prepared, int B,
                          int C, int H, int W, int k, int corner, long long *stamps,
                          int max_stamps, hipStream_t stream) {
    return inverse_diagnostic(kind, y, x, prepared, B, C, H, W, k, corner, stamps,
                              sizeof(long long), 4, max_stamps, stream);
}

int finc_banded_plan(int C, int H, int W, int k, int *info) {
    if (!info || !valid_shape(1, C, H, W, k))
        return FINC_EINVAL;
    InvChoice ch;
    int R = 0, nb = 0;
    if (!banded_choice(C, H, W, k, kLdsBytes, ch, R, nb))
        return FINC_EUNSUPPORTED;
    info[0] = ch.threads;
    info[1] = R;
    info[2] = nb;
    info[3] = (int)ch.lds;
    return FINC_OK;
}

size_t finc_banded_workspace_bytes(int B, int C, int H, int W, int k, int n_layers) {
    int info[4];
    if ((n_layers != 1 && n_layers != 4) || B < 0 || finc_banded_plan(C, H, W, k, info) != FINC_OK ||
        (long long)B * C * H * W >= (1ll << 31))
        return 0;
    const size_t prep = finc_workspace_bytes(C, k, n_layers);
    return prep + ((banded_flag_ints(B, info[2]) * sizeof(int) + 255) & ~(size_t)255);
}

static int banded_call(const float *y, float *x, const float *K, int n_layers, int corner, int B,
                       int C, int H, int W, int k, void *workspace, hipStream_t stream) {
    if (!valid_shape(B, C, H, W, k) || !x || !y || !K || !workspace || !aligned256(workspace))
        return FINC_EINVAL;
    int info[4];
    const int prc = finc_banded_plan(C, H, W, k, info);
    if (prc != FINC_OK)
        return prc;
    const size_t wsb = finc_banded_workspace_bytes(B, C, H, W, k, n_layers);
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t kb = (size_t)n_layers * C * C * k * k * sizeof(float);
    if (!inverse_alias_ok(y, x, bytes) || overlap(workspace, wsb, x, bytes) ||
        overlap(workspace, wsb, y, bytes) || overlap(workspace, wsb, K, kb))
        return FINC_EINVAL;
    int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
    if (n_layers == 1)
        corners[0] = corner;
    const int rc = finc_prepare(K, n_layers, corners, C, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    int *flags = reinterpret_cast<int *>(static_cast<char *>(workspace) +
                                         finc_workspace_bytes(C, k, n_layers));
    return launch_banded(y, x, static_cast<const float *>(workspace), n_layers, corner, B, C, H, W,
                         k, flags, stream);
}

int finc_inverse_banded(const float *y, float *x, const float *K, int B, int C, int H, int W,
                        int k, int corner, void *workspace, hipStream_t stream) {
    if (!valid_corner(corner))
        return FINC_EINVAL;
    return banded_call(y, x, K, 1, corner, B, C, H, W, k, workspace, stream);
}

int finc_unit_inverse_banded(const float *y, float *x, const float *K4, int B, int C, int H,
                             int W, int k, void *workspace, hipStream_t stream) {
    return banded_call(y, x, K4, 4, FINC_TL, B, C, H, W, k, workspace, stream);
}

int finc_split_inverse(const float *y, float *x, const float *Kq4, int B, int C, int H, int W,
                       int k, void *workspace, hipStream_t stream) {
    if (!valid_split(B, C, H, W, k) || !x || !y || !Kq4 || !workspace || !aligned256(workspace))
        return FINC_EINVAL;
    const int Cq = C / 4;
    const size_t bytes = (size_t)B * C * H * W * sizeof(float);
    const size_t wsb = finc_workspace_bytes(Cq, k, 4);
    if (!inverse_alias_ok(y, x, bytes) || overlap(workspace, wsb, x, bytes) ||
        overlap(workspace, wsb, y, bytes) ||
        overlap(workspace, wsb, Kq4, (size_t)4 * Cq * Cq * k * k * sizeof(float)))
        return FINC_EINVAL;
    if (B == 0)   // nothing to launch; the shape is still checked
        return finc_split_inverse_prepared(y, x, workspace, 0, C, H, W, k, stream);
    const int corners[4] = {FINC_TL, FINC_TR, FINC_BL, FINC_BR};
    const int rc = finc_prepare(Kq4, 4, corners, Cq, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_split_inverse_prepared(y, x, workspace, B, C, H, W, k, stream);
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
    a.lv[0] = level(y, prepared4, nullptr, nullptr, C, H, W, k);
    a.out = x;
    a.L = 1;

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
    if (B == 0)   // nothing to launch; the shape is still checked
        return finc_unit_inverse_prepared(y, x, workspace, 0, C, H, W, k, stream);
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
        !stack_call_ok(z, x, scale, bias, B, L, U, C1, H1, W1, k, nullptr, prepared, false))
        return FINC_EINVAL;
    InvArgs a;
    memset(&a, 0, sizeof(a));
    size_t poff = 0, soff = 0;
    for (int l = 0; l < L; ++l) {   // levels run top first
        const int C = C1 << l;
        a.lv[L - 1 - l] = level(z[l], (const char *)prepared + poff, scale + soff, bias + soff, C,
                                H1 >> l, W1 >> l, k);
        poff += stack_level_bytes(l, U, C1, k);
        soff += (size_t)U * C;
    }
    a.out = x;
    a.L = L;

    a.n_units = U;
    a.lpu = 4;
    a.corner0 = FINC_TL;
    if (!levels_differ(a))
        return launch_inverse_chain(a, B, stream);
    // Levels whose kernel instances differ (work split, quad groups or
    // critical form) run as launches of their own, each in its own instance:
    // one instance for all would be sized for the widest level and run the
    // others slower.  The hand-over goes through x, image by image: with
    // N = C1 H1 W1 floats per image, level l > 0 writes its solution to
    // [N / 2^l, N / 2^(l-1)) of its image's block and level 0 to all of it;
    // level l reads the level above's from [N / 2^(l+1), N / 2^l).  A level
    // reads only its own image's block and loads all of its input before its
    // first store, so no region is overwritten while another reads it.
    const int N = C1 * H1 * W1;
    for (int i = 0; i < L; ++i) {   // top first
        const int l = L - 1 - i;
        InvArgs s;
        memset(&s, 0, sizeof(s));
        s.lv[0] = a.lv[i];
        s.L = 1;
        s.n_units = U;
        s.lpu = 4;
        s.corner0 = FINC_TL;
        s.out = x + (l == 0 ? 0 : N >> l);
        s.out_stride = N;
        if (i > 0) {
            s.hin = x + (N >> (l + 1));
            s.hin_stride = N;
        }
        const int rc = launch_inverse_chain(s, B, stream);
        if (rc != FINC_OK)
            return rc;
    }
    return FINC_OK;
}

int finc_stack_inverse(const float *const *z, float *x, const float *K, const float *scale,
                       const float *bias, int B, int L, int U, int C1, int H1, int W1, int k,
                       void *workspace, hipStream_t stream) {
    if (!K || !workspace || !aligned256(workspace) ||
        !stack_call_ok(z, x, scale, bias, B, L, U, C1, H1, W1, k, K, workspace, true))
        return FINC_EINVAL;
    if (B == 0)   // nothing to launch; the shape is still checked
        return finc_stack_inverse_prepared(z, x, workspace, scale, bias, 0, L, U, C1, H1, W1, k,
                                           stream);
    const int rc = finc_stack_prepare(K, L, U, C1, k, workspace, stream);
    if (rc != FINC_OK)
        return rc;
    return finc_stack_inverse_prepared(z, x, workspace, scale, bias, B, L, U, C1, H1, W1, k,
                                       stream);
}

}  // extern "C"
#endif  // FINC_PART < 0
