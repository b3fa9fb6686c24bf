// Drives the host side of libfinc (argument checks, plan queries, workspace
// sizes) in a host-only build with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code: no call here reaches a
// kernel launch (every call either is host arithmetic only or is rejected
// before any HIP call), so the build needs no device code and no GPU.
// Test infrastructure: built and run by tests/test_sanitizers_cpu.py.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "finc.h"

static int failures = 0;
#define EXPECT(cond)                                                       \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

// Pointers that are never dereferenced: the calls below must reject them
// on the host.
static void *fake(unsigned long long a) { return (void *)(uintptr_t)a; }

static void plans() {
    const int HW[][2] = {{1, 1}, {1, 7}, {16, 16}, {13, 17}, {32, 32}, {64, 64}, {128, 128},
                         {129, 16}, {8, 200}};
    long long launches = 0;
    for (int kind = FINC_PLAN_LAYER; kind <= FINC_PLAN_SPLIT; ++kind)
        for (int C = 1; C <= 4 * FINC_MAX_C + 4; ++C)
            for (int k = 0; k <= FINC_MAX_K + 1; ++k)
                for (const auto &hw : HW) {
                    int *info = (int *)malloc(6 * sizeof(int));
                    const int r = finc_inverse_plan(kind, 1, 1, C, hw[0], hw[1], k, info, 1);
                    EXPECT(r == 1 || r == FINC_EINVAL || r == FINC_EUNSUPPORTED);
                    launches += r > 0 ? r : 0;
                    free(info);
                    int *fi = (int *)malloc(3 * sizeof(int));
                    for (int B : {0, 1, 64}) {
                        const int f = finc_forward_plan(kind, B, C, hw[0], hw[1], k, B == 1, fi);
                        EXPECT(f == FINC_OK || f == FINC_EINVAL || f == FINC_EUNSUPPORTED);
                    }
                    free(fi);
                }
    for (int L = 0; L <= 9; ++L)
        for (int C1 = 1; C1 <= 24; ++C1)
            for (int k = 1; k <= FINC_MAX_K; k += 2) {
                int *info = (int *)malloc(6 * sizeof(int) * (L > 0 ? L : 1));
                const int r = finc_inverse_plan(FINC_PLAN_STACK, L, 2, C1, 32, 32, k, info,
                                                L > 0 ? L : 1);
                EXPECT(r >= 1 || r == FINC_EINVAL || r == FINC_EUNSUPPORTED);
                EXPECT(r <= (L > 0 ? L : 1));
                free(info);
                if (L >= 2) {   // too small an info array is an error, not an overflow
                    int *one = (int *)malloc(6 * sizeof(int));
                    const int r1 = finc_inverse_plan(FINC_PLAN_STACK, L, 2, C1, 32, 32, k, one, 1);
                    EXPECT(r1 <= 1);
                    free(one);
                }
            }
    EXPECT(launches > 0);
    for (int C = 0; C <= 18; ++C)
        for (int k = 0; k <= FINC_MAX_K + 1; ++k)
            for (const auto &hw : HW) {
                int *bi = (int *)malloc(4 * sizeof(int));
                const int r = finc_banded_plan(C, hw[0] * 2, hw[1], k, bi);
                EXPECT(r == FINC_OK || r == FINC_EINVAL || r == FINC_EUNSUPPORTED);
                if (r == FINC_OK)
                    EXPECT(bi[1] % 16 == 0 && bi[1] <= 128 && bi[2] * bi[1] >= hw[0] * 2);
                free(bi);
                (void)finc_banded_workspace_bytes(5, C, hw[0] * 2, hw[1], k, 4);
            }
    EXPECT(finc_inverse_plan(FINC_PLAN_LAYER, 1, 1, 12, 16, 16, 3, nullptr, 1) == FINC_EINVAL);
    EXPECT(finc_inverse_plan(7, 1, 1, 12, 16, 16, 3, nullptr, 1) == FINC_EINVAL);
}

static void sizes() {
    for (int C = -1; C <= FINC_MAX_C + 2; ++C)
        for (int k = -1; k <= FINC_MAX_K + 1; ++k) {
            (void)finc_workspace_bytes(C, k, 1);
            (void)finc_workspace_bytes(C, k, 4);
            (void)finc_backward_workspace_bytes(64, C, 16, 16, k);
            (void)finc_unit_backward_workspace_bytes(3, C, 5, 7, k);
            (void)finc_split_backward_workspace_bytes(3, 4 * C, 5, 7, k);
            (void)finc_stack_workspace_bytes(3, 2, C, k);
            (void)finc_step_prepared_bytes(4 * C, k);
            (void)finc_step_param_count(4 * C, k, 16);
        }
    EXPECT(finc_backward_workspace_bytes(1 << 20, 64, 64, 64, 3) == 0);   // over 2^31 values
    EXPECT(finc_actnorm_backward_workspace_bytes(2, 0, 4, 4) == 0);
    (void)finc_flow_param_count(3, 28, 3, 3, 512);
    (void)finc_flow_prepared_bytes(3, 28, 3, 3);
    (void)finc_flow_workspace_bytes(100, 3, 3, 32, 32, 512);
    (void)finc_conv1x1_workspace_bytes(64);
    for (int s = -8; s <= 1; ++s)
        EXPECT(finc_strerror(s) != nullptr);
}

static void rejections() {
    const int B = 2, C = 12, H = 16, W = 16, k = 3;
    void *x = fake(0x100000), *y = fake(0x900000), *K = fake(0x1100000), *w = fake(0x40000000);
    float *xf = (float *)x, *yf = (float *)y;
    const float *Kf = (const float *)K;
    // overlapping output, misaligned or missing workspace, bad shapes, bad corners
    EXPECT(finc_forward(xf, xf + 8, Kf, nullptr, nullptr, B, C, H, W, k, 0, nullptr) ==
           FINC_EINVAL);
    EXPECT(finc_forward(xf, yf, Kf, nullptr, nullptr, B, C, H, W, k, 4, nullptr) == FINC_EINVAL);
    EXPECT(finc_forward(xf, yf, Kf, nullptr, nullptr, B, 0, H, W, k, 0, nullptr) == FINC_EINVAL);
    EXPECT(finc_inverse(yf, xf, Kf, B, C, H, W, k, 0, nullptr, nullptr) == FINC_EINVAL);
    EXPECT(finc_inverse(yf, xf, Kf, B, C, H, W, k, 0, fake(0x40000010), nullptr) == FINC_EINVAL);
    EXPECT(finc_inverse(yf, xf, Kf, B, C, H, W, 8, 0, w, nullptr) == FINC_EINVAL);
    EXPECT(finc_unit_inverse(yf, xf, Kf, B, C, H, W, k, nullptr, nullptr) == FINC_EINVAL);
    EXPECT(finc_split_forward(xf, yf, Kf, nullptr, nullptr, B, 6, H, W, k, nullptr) ==
           FINC_EINVAL);
    EXPECT(finc_backward(xf, yf, Kf, xf + 4, nullptr, 0.0, B, C, H, W, k, 0, w, nullptr) ==
           FINC_EINVAL);
    EXPECT(finc_unit_backward(xf, yf, Kf, nullptr, nullptr, 0.0, B, C, H, W, k, nullptr,
                              nullptr) == FINC_EINVAL);
    EXPECT(finc_split_backward(xf, yf, Kf, nullptr, nullptr, 0.0, B, 6, H, W, k, w, nullptr) ==
           FINC_EINVAL);
    float *s = (float *)fake(0x2000000);
    EXPECT(finc_actnorm_backward(xf, yf, s, nullptr, s, nullptr, 0.0, B, C, H, W, w, nullptr) ==
           FINC_EINVAL);
    const float *zs[3] = {xf, yf, Kf};
    const long long n[3] = {16, 8, 4};
    double *ld = (double *)fake(0x3000000);
    EXPECT(finc_gauss_nll(zs, n, 3, B, ld, ld, nullptr, nullptr) == FINC_EINVAL);
    EXPECT(finc_gauss_nll(zs, n, 0, B, ld, ld + 64, nullptr, nullptr) == FINC_EINVAL);
    // stack: z overlapping x, workspace overlapping a latent
    const float *z2[2] = {xf, xf + 16};
    EXPECT(finc_stack_inverse(z2, xf + 8, Kf, s, s, B, 2, 1, 2, 8, 8, 3, w, nullptr) ==
           FINC_EINVAL);
    EXPECT(finc_stack_inverse(z2, yf, Kf, s, s, B, 9, 1, 2, 8, 8, 3, w, nullptr) == FINC_EINVAL);
    EXPECT(finc_inverse_noalloc(yf, xf, Kf, B, C, H, W, 8, 0, nullptr) == FINC_EINVAL);
}

int main() {
    plans();
    sizes();
    rejections();
    if (failures)
        fprintf(stderr, "%d checks failed\n", failures);
    else
        printf("host sanitizer drive: all checks held\n");
    return failures ? 1 : 0;
}
