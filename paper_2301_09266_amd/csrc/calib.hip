// calib.hip -- measurement kernels for the benchmark, built into a library
// of their own (libfinc_calib.so); the product library never uses them.
//
// barrier_chain_kernel: the cost of one synchronised step of a wavefront of
// dependent steps, with nothing else in it.  Every step, each thread writes
// one LDS value into the buffer of the step's parity, the workgroup passes a
// barrier, and each thread reads a value written by another wave -- the
// least one diagonal step of the inverse does (its solved pixels written,
// made visible, read by the next step's waves).  Two buffers by parity need
// one barrier per step, as in the inverse.
#include <hip/hip_runtime.h>

namespace {

__global__ __launch_bounds__(256) void barrier_chain_kernel(float *out, int steps) {
    __shared__ float v[2][256];
    const int t = threadIdx.x;
    float acc = (float)t;
    for (int s = 0; s < steps; ++s) {
        v[s & 1][t] = acc;
        __syncthreads();
        acc = acc * 0.5f + v[s & 1][(t + 64) & 255];
    }
    out[blockIdx.x * 256 + t] = acc;
}

}  // namespace

extern "C" {

// `blocks` workgroups of 256 threads run `steps` steps each; out holds
// blocks * 256 floats (the results, so that the loop is not removed).
int finc_calib_barrier_chain(float *out, int blocks, int steps, hipStream_t stream) {
    if (!out || blocks < 1 || steps < 0)
        return -1;
    hipLaunchKernelGGL(barrier_chain_kernel, dim3(blocks), dim3(256), 0, stream, out, steps);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
