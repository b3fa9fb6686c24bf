/*
 * finc.h -- C ABI of the MI355X (gfx950) FInC Flow masked k x k convolution.
 *
 * The layer (Sec. 3 "Invertible Convolutions", Sec. 4.1 "Convolution
 * Design"): y = K * pad_corner(x), a cross-correlation of the input padded
 * with k-1 zero rows and columns on two sides (the "corner"), so output pixel
 * (i, j) reads input (i + a - oh, j + b - ow) for kernel position (a, b):
 *     TL (oh, ow) = (k-1, k-1)   TR (k-1, 0)   BL (0, k-1)   BR (0, 0).
 * Kernel position (oh, ow) multiplies the output pixel itself (the "self
 * tap"); there only channels c_in <= c_out are used (lower-triangular channel
 * block), every other position is used in full.  Entries with c_in > c_out at
 * the self tap are ignored whatever the buffer holds.  The convolution matrix
 * is then triangular in the corner's raster order with diagonal
 * K[c, c, oh, ow] (Fig. 1), so log|det| = H*W*sum_c log|K[c,c,oh,ow]| and the
 * inverse can be solved pixel diagonal by pixel diagonal (Algorithm 1,
 * Theorems 1 and 2).
 *
 * Conventions shared by every entry point:
 *  - Tensors are fp32, C-contiguous.  Activations (B, C, H, W); one layer's
 *    weights (C_out, C_in, k, k) ("OIHW").  Pointers marked "device" must be
 *    device memory of the current HIP device; the caller owns every buffer.
 *  - Calls are asynchronous on `stream` (0 = the null stream) and return after
 *    enqueueing.  Nothing is allocated, freed or synchronised by the library.
 *  - Return value: FINC_OK or a negative finc_status.  Arguments are checked
 *    before any HIP call: a bad argument returns FINC_EINVAL and enqueues
 *    nothing.  FINC_EUNSUPPORTED: the shape is valid but does not fit the
 *    kernels.  Inverse calls (also with B == 0): the per-image work split
 *    needs more waves or more weight registers per wave than one workgroup
 *    has, or its LDS layout exceeds 160 KB and the stream form (single layers
 *    of at most 16 channels) does not apply; finc_inverse_plan answers it for
 *    any shape.  Forward calls (B > 0): one block of rows with its halo does
 *    not fit in LDS (very wide rows); finc_forward_plan answers it.
 *    FINC_EHIP: a HIP runtime call failed (hipGetLastError after the launch).
 *    Device-side faults surface at the caller's next synchronisation.
 *  - A zero self-tap diagonal weight makes the layer singular: finc_logdet
 *    writes -inf and the inverse produces non-finite values (the weights are
 *    device-resident, so this is not detected on the host).
 *  - Results are bitwise deterministic and do not depend on B or on an
 *    image's position in the batch: each image is processed by one workgroup
 *    in a fixed summation order, without atomics.
 *  - Supported shapes: 1 <= C <= FINC_MAX_C, 1 <= k <= FINC_MAX_K, H, W >= 1,
 *    B >= 0 (B == 0 enqueues nothing), B*C*H*W < 2^31.
 */
#ifndef FINC_H
#define FINC_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FINC_MAX_C 64
#define FINC_MAX_K 7

/* Corner padding variants (Sec. 4.1, corner padding equations). */
enum { FINC_TL = 0, FINC_TR = 1, FINC_BL = 2, FINC_BR = 3 };

typedef enum {
    FINC_OK = 0,
    FINC_EINVAL = -1,
    FINC_ESINGULAR = -2,
    FINC_EUNSUPPORTED = -3,
    FINC_EHIP = -4
} finc_status;

/* Library version, major*10000 + minor*100 + patch. */
int finc_version(void);

/* Static text for a status code (never NULL). */
const char *finc_strerror(int status);

/* ---- Inverse kernel selection (host arithmetic only, no HIP call) --------
 * The inverse of Algorithm 1 runs as one of a fixed set of compiled kernel
 * instances, chosen on the host from the level shapes: workgroup size,
 * critical-path form ("mode") and weight quad groups held in registers per
 * wave.  finc_inverse_plan reports the instance(s) a call would launch, for
 * tests that must reach every instance and for capacity planning:
 *   kind FINC_PLAN_LAYER: finc_inverse(_prepared) on C x H x W, k;
 *   kind FINC_PLAN_UNIT:  finc_unit_inverse(_prepared);
 *   kind FINC_PLAN_SPLIT: finc_split_inverse(_prepared), C = the unit's
 *                         channels (a multiple of 4);
 *   kind FINC_PLAN_STACK: finc_stack_inverse(_prepared) with L levels of U
 *                         units, C = C1, H = H1, W = W1.
 * L and U are ignored except for FINC_PLAN_STACK.  For each distinct launch
 * (one; or L for a stack whose levels run in launches of their own) it writes
 * six ints to info: workgroup threads, mode bits (0 gathering critical wave,
 * 1 register-fed; +4 single layer; +8 stream form, one launch per layer),
 * quad groups per wave, 1 if streamed, LDS bytes, 1 if partial tiles are
 * kept in the compact layout (the padded one would not fit).  The LDS
 * budget is gfx950's 160 KB per workgroup.  Returns the number of launches
 * written, FINC_EINVAL for bad arguments (or max_launches too small), or
 * FINC_EUNSUPPORTED exactly when the corresponding call would return it. */
enum { FINC_PLAN_LAYER = 0, FINC_PLAN_UNIT = 1, FINC_PLAN_SPLIT = 2, FINC_PLAN_STACK = 3 };
int finc_inverse_plan(int kind, int L, int U, int C, int H, int W, int k, int *info,
                      int max_launches);

/* ---- Images whose level does not fit one workgroup (Sec. 5, Fig. 3's
 * large images) ---------------------------------------------------------------
 * The banded stream form: the image's rows (in the corner's frame) are cut
 * into bands of R rows, one workgroup each, every band running the column-
 * streaming diagonal wavefront of its own rows.  A band reads the k - 1 rows
 * above it -- the band above's solution -- from the output as that band
 * drains them, waiting on a per-band count of drained diagonals in the
 * workspace; the bands run pipelined, each about R + 16 diagonals behind the
 * one above (Thm. 2's H + W - 1 steps plus that lag per band).  A workgroup
 * takes its (image, band) from a ticket at its start, so it only ever waits
 * on a band that started before it.  Every wait is bounded: after about a
 * second the band sets the workspace's timeout flag (the int at byte offset
 * finc_workspace_bytes(C, k, n_layers)), goes on, and its image's result is
 * invalid.
 * finc_banded_plan: info[0] = workgroup threads, [1] = band rows R, [2] =
 *   bands per image, [3] = LDS bytes; FINC_EUNSUPPORTED when no band fits a
 *   workgroup (C > 16 or k = 1), FINC_EINVAL for a bad shape.
 * finc_banded_workspace_bytes: the prepared weights of n_layers (1 or 4)
 *   layers, then the flags; 0 for an unsupported shape.
 * finc_inverse_banded: as finc_inverse (one layer, corner `corner`);
 * finc_unit_inverse_banded: as finc_unit_inverse (four layers, one launch
 *   each, the later ones in place on x).  workspace: device, at least
 *   finc_banded_workspace_bytes(B, C, H, W, k, 1 or 4) bytes, 256-byte
 *   aligned, overwritten.  x == y is allowed; other overlaps FINC_EINVAL.
 *   Calls sharing one workspace must not overlap in time. */
int finc_banded_plan(int C, int H, int W, int k, int *info);
size_t finc_banded_workspace_bytes(int B, int C, int H, int W, int k, int n_layers);
int finc_inverse_banded(const float *y, float *x, const float *K, int B, int C, int H,
                        int W, int k, int corner, void *workspace, hipStream_t stream);
int finc_unit_inverse_banded(const float *y, float *x, const float *K4, int B, int C,
                             int H, int W, int k, void *workspace, hipStream_t stream);

/* Diagnostic of Theorem 2's step count: the inverse of finc_inverse_prepared
 * (kind FINC_PLAN_LAYER, one layer with corner `corner`) or of
 * finc_split_inverse_prepared (kind FINC_PLAN_SPLIT, corner ignored), which
 * also writes, for every wave w of the launch's workgroup b (b = image, or
 * 4 * image + quarter for the channel-split unit), steps[b * waves + w] = the
 * number of diagonal steps that wave ran, each ended by the workgroup's step
 * barrier (waves = the plan's threads / 64).  Every wave of every
 * workgroup runs H + W - 1 of them.  steps: device ints, at least that many
 * (max_steps; FINC_EINVAL if fewer), not overlapping x, y or prepared.
 * Returns the number of ints written, or an error as the inverse call would.
 * For tests and tools; the product calls do not count. */
int finc_inverse_steps(int kind, const float *y, float *x, const void *prepared, int B,
                       int C, int H, int W, int k, int corner, int *steps, int max_steps,
                       hipStream_t stream);

/* Diagnostic of where an inverse launch's time goes: the inverse of
 * finc_inverse_steps (same kinds, shapes and checks), which also writes, for
 * every wave w of workgroup b, stamps[(b * waves + w) * 4 + i] = the GPU's
 * 100 MHz constant clock (10 ns a tick) when that wave i = 0 had its
 * arguments, 1 had its set-up done (weights and the image in LDS; before its
 * first step barrier), 2 had run its last diagonal step, 3 had issued its
 * part of the solution's store (completion of the stores is not waited for).  stamps:
 * device long longs, at least 4 per wave (max_stamps; FINC_EINVAL if fewer),
 * not overlapping x, y or prepared.  Returns the number written, or an error
 * as the inverse call would.  For tests and tools; the product calls read no
 * clock. */
int finc_inverse_timeline(int kind, const float *y, float *x, const void *prepared, int B,
                          int C, int H, int W, int k, int corner, long long *stamps,
                          int max_stamps, hipStream_t stream);

/* The forward's work split (host arithmetic only): an image is cut into
 * blocks of rows, each staged in LDS with its halo rows and the layer's
 * weights; a unit keeps whole images, or bands of rows when the batch is
 * smaller than the GPU's compute units or an image does not fit (in place,
 * in_place != 0, a unit keeps whole images).  For finc_forward (kind
 * FINC_PLAN_LAYER), finc_unit_forward (FINC_PLAN_UNIT) and finc_split_forward
 * (FINC_PLAN_SPLIT, C = the unit's channels) on a batch of B images it writes
 * info[0] = blocks per image, info[1] = rows per block, info[2] = LDS bytes
 * per block, and returns FINC_OK, or FINC_EUNSUPPORTED when even the
 * smallest block does not fit in gfx950's 160 KB (the forward call then
 * returns it too), or FINC_EINVAL. */
int finc_forward_plan(int kind, int B, int C, int H, int W, int k, int in_place, int *info);

/* ---- Weight preparation (one-time per weight set) -----------------------
 * The inverse of one layer solves, per pixel, L x_p = y_p - sum_s K_s x_src
 * with L the self-tap channel block (lower triangular).  Preparation forms,
 * in fp64, L^-1 and L^-1 K_s for every other kernel position s, rounded to
 * fp32, so that every pixel of a diagonal step is a plain accumulation
 * (see Algorithm 1 and the channel mask of Sec. 4.1).
 *
 * finc_workspace_bytes: device bytes of prepared weights for n_layers layers
 *   of size (C, k); 0 for invalid arguments.
 * finc_prepare: K = n_layers consecutive OIHW tensors (device); corners =
 *   host array of n_layers corner ids; prepared = device buffer of at least
 *   finc_workspace_bytes(C, k, n_layers) bytes, 256-byte aligned, written by
 *   the call (its layout is private to the library). */
size_t finc_workspace_bytes(int C, int k, int n_layers);
int finc_prepare(const float *K, int n_layers, const int *corners, int C, int k,
                 void *prepared, hipStream_t stream);

/* ---- One padded masked convolution block (PCB) --------------------------
 * finc_forward: y = layer(x) (Sec. 3 conv equation with Sec. 4.1 padding).
 *   x, y: device (B, C, H, W); K: device OIHW.  x and y must not overlap.
 *   logdet: NULL, or device double that receives the layer's log|det| (as
 *   finc_logdet) from the same launch, as a flow layer's forward pass does.
 *   prepared: NULL, or device buffer of finc_workspace_bytes(C, k, 1) bytes,
 *   256-byte aligned, clear of x, y and K, that receives the weights as
 *   finc_prepare would write them (for finc_inverse_prepared) -- computed
 *   by extra workgroups of the same launch for C <= 16, by a second launch
 *   on the same stream otherwise.  B == 0 still fills both side outputs.
 * finc_logdet: out[0] (device double) = log|det| of the layer's H*W*C x
 *   H*W*C convolution matrix, the same for every image (Table 1 "Jacobian";
 *   -inf for a zero diagonal).
 * finc_inverse: x = layer^-1(y) by the diagonal wavefront of Algorithm 1:
 *   H + W - 1 dependent steps (Theorem 2), every pixel of a diagonal solved
 *   at once (Theorem 1).  workspace: device, >= finc_workspace_bytes(C, k, 1)
 *   bytes, 256-byte aligned, overwritten.  x == y (in place) is allowed; any
 *   other overlap is rejected.
 * finc_inverse_prepared: the same with weights already prepared by
 *   finc_prepare (one layer, same corner). */
int finc_forward(const float *x, float *y, const float *K, double *logdet,
                 void *prepared, int B, int C, int H, int W, int k, int corner,
                 hipStream_t stream);
int finc_logdet(const float *K, int C, int k, int corner, int H, int W,
                double *out, hipStream_t stream);
int finc_inverse(const float *y, float *x, const float *K, int B, int C, int H,
                 int W, int k, int corner, void *workspace, hipStream_t stream);
int finc_inverse_prepared(const float *y, float *x, const void *prepared, int B,
                          int C, int H, int W, int k, int corner,
                          hipStream_t stream);

/* ---- The inverse for callers that cannot allocate ------------------------
 * finc_inverse_noalloc: finc_inverse without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  The prepared
 * weights go to a 1 MiB device array of the library's own, one per device,
 * held until the process ends; the largest layer the library accepts
 * (C = 64, k = 7) needs 803,072 bytes of it, so every valid shape fits
 * (FINC_EUNSUPPORTED would report one that did not).  The call allocates and
 * frees nothing.  Its first call on a device looks up that device's array
 * address (a HIP runtime query).  Every call on one device shares that
 * device's array and rewrites all of it that the inverse reads: calls that
 * overlap on one device -- concurrently from several host threads, or on
 * several streams without ordering between them -- race and must not be
 * made.  Arguments, aliasing (x == y allowed) and results as finc_inverse:
 * bit for bit the same output. */
int finc_inverse_noalloc(const float *y, float *x, const float *K, int B, int C, int H,
                         int W, int k, int corner, hipStream_t stream);

/* ---- FInC unit: four PCBs TL, TR, BL, BR applied in sequence -----------
 * (Sec. 4.3 and Fig. 2a, read as four full-channel blocks one after the
 * other; the inverse runs BR^-1, BL^-1, TR^-1, TL^-1 in one launch, as
 * Algorithm 2 inverts a whole unit at once.)  K4: device, 4 consecutive OIHW
 * tensors in the order TL, TR, BL, BR.  Activations stay in on-chip memory
 * between the four blocks (a batch smaller than the GPU's compute units is
 * split into bands of rows, each band recomputing the rows its neighbours'
 * later blocks read).  finc_unit_forward allows x == y (then each image is
 * one band, read whole before it is written); the inverse's rules are as for
 * one block.
 * logdet (finc_unit_forward): NULL, or device double for the unit's log|det|;
 * prepared4: NULL, or device buffer of finc_workspace_bytes(C, k, 4) bytes
 * (rules as for finc_forward) for finc_unit_inverse_prepared.
 * finc_unit_logdet: sum of the four blocks' log|det|. */
int finc_unit_forward(const float *x, float *y, const float *K4, double *logdet,
                      void *prepared4, int B, int C, int H, int W, int k,
                      hipStream_t stream);
int finc_unit_logdet(const float *K4, int C, int k, int H, int W, double *out,
                     hipStream_t stream);
int finc_unit_inverse(const float *y, float *x, const float *K4, int B, int C,
                      int H, int W, int k, void *workspace, hipStream_t stream);
int finc_unit_inverse_prepared(const float *y, float *x, const void *prepared4,
                               int B, int C, int H, int W, int k,
                               hipStream_t stream);

/* ---- Channel-split FInC unit: four PCBs side by side --------------------
 * (Sec. 4.3, Fig. 2a, Algorithm 2: the channels are cut into four equal
 * quarters; quarter g is a PCB of its own with C/4 channels, its own masked
 * weights and corner g in the order TL, TR, BL, BR; the four act on the same
 * pixels in parallel and their outputs are concatenated.  The text names the
 * fourth quarter's padding TR a second time; BR is taken.)  Each quarter is
 * inverted independently, all four in one launch (a workgroup per image and
 * quarter, as Algorithm 2's grid of batch x 4).
 *   C: the unit's channels, a multiple of 4, C/4 <= FINC_MAX_C.
 *   Kq4: device, 4 consecutive OIHW tensors (C/4, C/4, k, k), quarter order.
 *   logdet (finc_split_forward): NULL, or device double for the unit's
 *     log|det| (the sum over the quarters); finc_split_logdet writes it alone.
 *   prepared4 / workspace: device buffer of finc_workspace_bytes(C/4, k, 4)
 *     bytes, 256-byte aligned: the quarters' prepared weights in quarter
 *     order (what finc_prepare(Kq4, 4, {TL, TR, BL, BR}, C/4, k, .) writes).
 * Aliasing and errors as for finc_forward / finc_inverse: the forward needs
 * x and y disjoint; the inverse allows x == y; FINC_EINVAL for C not a
 * multiple of 4 or any other bad argument. */
int finc_split_forward(const float *x, float *y, const float *Kq4, double *logdet,
                       void *prepared4, int B, int C, int H, int W, int k,
                       hipStream_t stream);
int finc_split_logdet(const float *Kq4, int C, int k, int H, int W, double *out,
                      hipStream_t stream);
int finc_split_inverse(const float *y, float *x, const float *Kq4, int B, int C,
                       int H, int W, int k, void *workspace, hipStream_t stream);
int finc_split_inverse_prepared(const float *y, float *x, const void *prepared4,
                                int B, int C, int H, int W, int k,
                                hipStream_t stream);

/* ---- Backward of one layer (training) -------------------------------------
 * The paper trains on the negative log-likelihood (Sec. 3, NLL equation) and
 * resets the masked weights' gradients to zero after every step (appendix,
 * training details).  For y = finc_forward(x, K, corner) and dy = dL/dy of a
 * loss L:
 *   dx: device (B, C, H, W), or NULL to skip: J^T dy, the gradient of L with
 *       respect to x;
 *   dK: device OIHW (C*C*k*k floats), or NULL to skip: the gradient of L
 *       with respect to K, summed over the batch, with the masked entries
 *       (self tap, c_in > c_out) set to 0, plus gld * H * W / K[c,c,self] on
 *       the self diagonal -- the gradient of gld * log|det| (gld = 0 for the
 *       convolution alone, -1 for the log|det| part of the NLL of one image).
 *   workspace: device, >= finc_backward_workspace_bytes(B, C, H, W, k) bytes,
 *       256-byte aligned, overwritten (the partial sums of dK over parts of
 *       the batch's pixels).
 * x, dy, K are read only; dx, dK and the workspace overwritten, overlapping
 * none of the inputs nor each other (else FINC_EINVAL).  With B = 0 only the
 * log|det| term remains in dK (x, dy may then be NULL).  Deterministic: no atomics, a fixed summation
 * order (dK depends on B through that order, as any sum over the batch). */
size_t finc_backward_workspace_bytes(int B, int C, int H, int W, int k);
int finc_backward(const float *x, const float *dy, const float *K, float *dx,
                  float *dK, double gld, int B, int C, int H, int W, int k,
                  int corner, void *workspace, hipStream_t stream);

/* Backward of the FInC units, by the chain rule over their blocks (same
 * gradient conventions as finc_backward; gld multiplies the unit's log|det|,
 * the sum of its four blocks', so each block takes the same gld).
 * finc_unit_backward: the unit of finc_unit_forward (blocks TL, TR, BL, BR
 *   in sequence, K4 = 4 OIHW tensors).  The inputs of blocks 2..4 are
 *   recomputed by the forward into the workspace, then the blocks run in
 *   reverse.  dK4: 4 C*C*k*k floats or NULL; dx may be NULL.  workspace:
 *   >= finc_unit_backward_workspace_bytes(B, C, H, W, k) bytes (four
 *   activations and dK's partial sums).  The forward's limits apply
 *   (FINC_EUNSUPPORTED where finc_forward_plan reports them).
 * finc_split_backward: the channel-split unit of finc_split_forward
 *   (Sec. 4.3): quarter g of the C channels is one block of C/4 channels
 *   with corner g; Kq4 / dKq4 = 4 (C/4, C/4, k, k) tensors.  workspace:
 *   >= finc_split_backward_workspace_bytes(B, C, H, W, k) bytes.
 * Aliasing and errors as for finc_backward. */
size_t finc_unit_backward_workspace_bytes(int B, int C, int H, int W, int k);
int finc_unit_backward(const float *x, const float *dy, const float *K4, float *dx,
                       float *dK4, double gld, int B, int C, int H, int W, int k,
                       void *workspace, hipStream_t stream);
size_t finc_split_backward_workspace_bytes(int B, int C, int H, int W, int k);
int finc_split_backward(const float *x, const float *dy, const float *Kq4, float *dx,
                        float *dKq4, double gld, int B, int C, int H, int W, int k,
                        void *workspace, hipStream_t stream);

/* Backward of actnorm y = s x + b (per channel c; log|det| H W sum_c
 * log|s_c| per image, Sec. 4.4): dx = s dy; ds[c] = sum over the batch's
 * pixels of dy x, plus gld H W / s[c]; db[c] = sum of dy.  x, dy, dx:
 * device (B, C, H, W); s, ds, db: device C floats; dx, ds or db may be
 * NULL.  workspace: >= finc_actnorm_backward_workspace_bytes(B, C, H, W)
 * bytes, 256-byte aligned (per-channel partial sums).  Sums in fp64, in a
 * fixed order.  Outputs overlapping any input or each other: FINC_EINVAL. */
size_t finc_actnorm_backward_workspace_bytes(int B, int C, int H, int W);
int finc_actnorm_backward(const float *x, const float *dy, const float *s, float *dx,
                          float *ds, float *db, double gld, int B, int C, int H, int W,
                          void *workspace, hipStream_t stream);

/* Training direction of the multi-scale stack (the stack of
 * finc_stack_inverse, its layout of K, scale and bias): the forward maps
 * images to latents -- per level U x [unit, actnorm], then below the top the
 * split (second half: the level's latent) and the squeeze of the first half
 * (Sec. 4.4, Fig. 2c) -- and its backward gives the gradients of a loss L
 * with respect to the input and every parameter, from the latents'
 * gradients dz[l] = dL/dz[l], plus gld times the gradient of the stack's
 * log|det| of one image (gld = -B for the log|det| part of a batch's summed
 * negative log-likelihood, whose latent gradients are dz = z).
 * finc_stack_forward: x device (B, C1, H1, W1); z host array of L device
 *   pointers shaped as for finc_stack_inverse (written); logdet: NULL or
 *   device doubles, B, each the stack's log|det| (every block's and every
 *   actnorm's; the same for every image).
 * finc_stack_backward: dz as z (read); dx (B, C1, H1, W1), dK, dscale, dbias
 *   in the layouts of x, K, scale and bias (written; any may be NULL, and
 *   the masked weights' gradients are 0).  The forward is run again inside
 *   the call to recompute the activations.
 * workspace: device, >= finc_stack_train_workspace_bytes(B, L, U, C1, H1, W1,
 *   k) bytes, 256-byte aligned, overwritten.  Requirements as for
 *   finc_stack_inverse, and the units' forward supported at every level
 *   (finc_forward_plan).  Outputs overlapping any input, the workspace or
 *   each other: FINC_EINVAL.  Deterministic (fixed summation orders). */
size_t finc_stack_train_workspace_bytes(int B, int L, int U, int C1, int H1, int W1, int k);
int finc_stack_forward(const float *x, float *const *z, double *logdet, const float *K,
                       const float *scale, const float *bias, int B, int L, int U, int C1,
                       int H1, int W1, int k, void *workspace, hipStream_t stream);
int finc_stack_backward(const float *x, const float *const *dz, const float *K,
                        const float *scale, const float *bias, float *dx, float *dK,
                        float *dscale, float *dbias, double gld, int B, int L, int U, int C1,
                        int H1, int W1, int k, void *workspace, hipStream_t stream);

/* Negative log-likelihood of each image under a standard normal latent
 * (Sec. 3, the log-probability equation negated) and its bits per dimension
 * (Sec. 5, BPD equation):
 *   nll[b] = sum over image b's latent values v of (v^2 + log 2 pi) / 2
 *            - logdet[b];   bpd[b] = nll[b] / (D log 2),
 * D = n[0] + ... + n[L-1] values per image.  z: host array of L device
 * pointers, z[l] holding B blocks of n[l] floats (one per image), 1 <= L
 * <= 16; logdet, nll, bpd: device doubles, B each (bpd may be NULL).  The
 * gradient of sum_b nll[b] with respect to z is z itself.  For data
 * quantised to 2^8 levels and scaled to [0, 1), add D log 256 to nll
 * before dividing (not done here: the equation has no such term).  Fixed
 * summation order (fp64). */
int finc_gauss_nll(const float *const *z, const long long *n, int L, int B,
                   const double *logdet, double *nll, double *bpd, hipStream_t stream);

/* ---- Multi-scale sampling stack (Sec. 4.4, Fig. 2c) ---------------------
 * L levels of U units; level l has C_l = C1 << l channels and spatial size
 * (H1 >> l, W1 >> l).  Forward direction (for the definition): per level
 * U x [unit, actnorm y = s*x + b], then, below the top, keep the first half
 * of the channels and squeeze (C, H, W) -> (4C, H/2, W/2) with channel
 * 4c + 2dy + dx <- (c, 2i+dy, 2j+dx); the second half is that level's latent.
 * finc_stack_inverse samples: starting from the top latent, per level
 * U x [actnorm^-1, unit^-1] with units in reverse, then unsqueeze and append
 * the level's latent as the second half of the channels.
 *   z: host array of L device pointers; z[l] for l < L-1 is (B, C_l/2, H_l,
 *      W_l), z[L-1] is (B, C_{L-1}, H_{L-1}, W_{L-1}).
 *   x: device (B, C1, H1, W1) output.  When the levels need different
 *      kernel instances they run as one launch each, and x also carries the
 *      hand-over between them (each image's block of x holds the upper
 *      levels' solutions until level 0 overwrites it): its contents are
 *      undefined until the call's work on `stream` has finished.
 *   K: device, for l, u, block q (TL, TR, BL, BR): C_l*C_l*k*k floats each.
 *   scale, bias: device, for l, u: C_l floats each (scale must be nonzero).
 *   workspace: device, >= finc_stack_workspace_bytes(L, U, C1, k) bytes,
 *   256-byte aligned, overwritten with prepared weights.
 * Requirements: C1 even when L > 1, H1 and W1 divisible by 2^(L-1),
 * C_{L-1} <= FINC_MAX_C, L <= 8, none of z, x overlap. */
size_t finc_stack_workspace_bytes(int L, int U, int C1, int k);
int finc_stack_inverse(const float *const *z, float *x, const float *K,
                       const float *scale, const float *bias, int B, int L,
                       int U, int C1, int H1, int W1, int k, void *workspace,
                       hipStream_t stream);
/* The same with weights already prepared into `prepared` by
 * finc_stack_prepare (which runs finc_prepare level by level). */
int finc_stack_prepare(const float *K, int L, int U, int C1, int k,
                       void *prepared, hipStream_t stream);
int finc_stack_inverse_prepared(const float *const *z, float *x,
                                const void *prepared, const float *scale,
                                const float *bias, int B, int L, int U, int C1,
                                int H1, int W1, int k, hipStream_t stream);

/* ---- The full FInC Flow (Sec. 4.4 "Architecture", Fig. 2b and 2c) ------
 * A Step is, forward: the channel-split FInC unit (as finc_split_forward),
 * actnorm u = s x + b, the invertible 1x1 convolution v = Wm u (Glow), and an
 * affine coupling: with v = [va, vb] (channel halves) and h = NN(va),
 * t = h[0 .. C/2), r = h[C/2 .. C), sc = sigmoid(r + 2): y = [va,
 * (vb + t) sc], log|det| += sum log sc.  NN is a 3x3 convolution (C/2 ->
 * hid), ReLU, a 1x1 convolution (hid -> hid), ReLU, and a 3x3 convolution
 * (hid -> C) times exp(3 ls[c]) per output channel; every convolution has a
 * bias and zero "same" padding.  (Readings: the paper names these layers
 * after Glow; the shift/scale halves, sigmoid(r + 2) and the exp(3 ls)
 * output scale are Glow's.)
 * Step parameters, one flat fp32 array (C = channels, q = C/4, Ch = C/2):
 *   Kq4 (4, q, q, k, k) | s (C) | b (C) | Wm (C, C) | W1 (hid, Ch, 3, 3) |
 *   b1 (hid) | W2 (hid, hid) | b2 (hid) | W3 (C, hid, 3, 3) | b3 (C) | ls3 (C)
 * The multi-scale flow of L levels, K Steps each, on (B, C0, H0, W0) images:
 * per level squeeze (as the stack), K Steps, then below the top a split
 * whose second half becomes the latent z_l = (h2 - mean) exp(-logsd), with
 * (mean, logsd) the halves of a 3x3 convolution of the first half (C/2 -> C,
 * bias, exp(3 ls) scale; Glow's split prior; log|det| -sum logsd); the top
 * level's output is the last latent.  Level l has C_l = 4 C0 2^l channels at
 * H0/2^(l+1) x W0/2^(l+1); z[l] is (B, C_l/2, ...) below the top and
 * (B, C_l, ...) at it.  Flow parameters: per level its K Steps, then (below
 * the top) the prior Wp (C_l, C_l/2, 3, 3) | bp (C_l) | lsp (C_l).
 * Requirements: every Step's C a multiple of 4, at most 64; its unit's
 * inverse supported (finc_inverse_plan, FINC_PLAN_SPLIT); H0, W0 divisible
 * by 2^L; L <= 6; hid <= 4096.
 * Prepared weights (finc_*_prepare, device, 256-byte aligned, private
 * layout): per Step the unit's inverse weights and, in fp64 then rounded,
 * the 1x1 convolution folded with the actnorm in both directions and the
 * Step's per-pixel constant log|det|.  The calls read params (device) for
 * the coupling and prior networks and prepared for the rest.
 * Workspace (device, 256-byte aligned, overwritten): scratch activations.
 * log|det| outputs are device doubles, one per image.  Aliasing: outputs
 * must not overlap inputs, params, prepared or the workspace (EINVAL).
 * Deterministic: fixed summation orders, no atomics. */
size_t finc_step_param_count(int C, int k, int hid);
size_t finc_step_prepared_bytes(int C, int k);
size_t finc_step_workspace_bytes(int B, int C, int H, int W, int hid);
int finc_step_prepare(const float *sp, int C, int k, int hid, void *prepared,
                      hipStream_t stream);
/* y = Step(x); logdet (B doubles, or NULL): += the Step's log|det|. */
int finc_step_forward(const float *x, float *y, double *logdet, const float *sp,
                      const void *prepared, int B, int C, int H, int W, int k, int hid,
                      void *workspace, hipStream_t stream);
/* x = Step^-1(y): coupling^-1, 1x1^-1 and actnorm^-1 (one prepared map),
 * then the unit's wavefront inverse (Algorithm 2). */
int finc_step_inverse(const float *y, float *x, const float *sp, const void *prepared, int B,
                      int C, int H, int W, int k, int hid, void *workspace,
                      hipStream_t stream);

size_t finc_flow_param_count(int L, int K, int C0, int k, int hid);
size_t finc_flow_prepared_bytes(int L, int K, int C0, int k);
size_t finc_flow_workspace_bytes(int B, int L, int C0, int H0, int W0, int hid);
int finc_flow_prepare(const float *params, int L, int K, int C0, int k, int hid,
                      void *prepared, hipStream_t stream);
/* Density direction: x (B, C0, H0, W0) -> latents z[0 .. L-1] (host array of
 * device pointers) and logdet (B doubles, overwritten). */
int finc_flow_forward(const float *x, float *const *z, double *logdet, const float *params,
                      const void *prepared, int B, int L, int K, int C0, int H0, int W0,
                      int k, int hid, void *workspace, hipStream_t stream);
/* Sampling direction: latents -> x. */
int finc_flow_sample(const float *const *z, float *x, const float *params,
                     const void *prepared, int B, int L, int K, int C0, int H0, int W0,
                     int k, int hid, void *workspace, hipStream_t stream);

/* The invertible 1x1 convolution alone (Sec. 4.4): y = Wm x at every pixel
 * (Wm (C, C), C <= 64); logdet (device double, or NULL) = H W log|det Wm|
 * (-inf if singular).  The inverse applies Wm^-1, formed in fp64 by LU with
 * partial pivoting.  workspace: finc_conv1x1_workspace_bytes(C), 256-byte
 * aligned. */
size_t finc_conv1x1_workspace_bytes(int C);
int finc_conv1x1_forward(const float *x, float *y, const float *Wm, double *logdet, int B,
                         int C, int H, int W, void *workspace, hipStream_t stream);
int finc_conv1x1_inverse(const float *y, float *x, const float *Wm, int B, int C, int H, int W,
                         void *workspace, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* FINC_H */
