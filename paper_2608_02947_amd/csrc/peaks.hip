// Microbenchmarks of the device limits the kernels are measured against: the dense
// bf16 MFMA rate, the v_exp_f32 rate, and the HBM read rate.  Built into their own
// library (libatf_peaks.so), outside the attention ABI of atf.h; bench.py --peaks
// times them with HIP events.  Every kernel here reads and writes only the buffers
// it is given, within the sizes it is given.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

// Back-to-back v_mfma_f32_32x32x16_bf16 on four independent accumulators per wave;
// one result per thread is stored so that nothing is optimised away.
__global__ __launch_bounds__(256) void mfma_loop(float* out, int iters, float seed) {
    bf16x8_t a, b;
    for (int i = 0; i < 8; ++i) {
        a[i] = (__bf16)(seed * float(threadIdx.x + i));
        b[i] = (__bf16)(seed * float(i + 1));
    }
    f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
    float r = 0.f;
    for (int i = 0; i < 16; ++i) r += c0[i] + c1[i] + c2[i] + c3[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = r;
}

// The same with v_mfma_f32_32x32x8_bf16 (half the depth, 16384 flops): what a K-step
// of 4 rotary pairs would cost against the 8-pair step above.
__global__ __launch_bounds__(256) void mfma8_loop(float* out, int iters, float seed) {
    typedef short s16x4_t __attribute__((ext_vector_type(4)));
    s16x4_t a, b;
    for (int i = 0; i < 4; ++i) {
        a[i] = short(threadIdx.x + i);
        b[i] = short(i + 1) + short(seed);
    }
    f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
    for (int it = 0; it < iters; ++it) {
        c0 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, b, c0, 0, 0, 0);
        c1 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, b, c1, 0, 0, 0);
        c2 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, b, c2, 0, 0, 0);
        c3 = __builtin_amdgcn_mfma_f32_32x32x8bf16_1k(a, b, c3, 0, 0, 0);
    }
    float r = 0.f;
    for (int i = 0; i < 16; ++i) r += c0[i] + c1[i] + c2[i] + c3[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = r;
}

// v_exp_f32 on 16 independent chains per thread (throughput, not latency, bound).
__global__ __launch_bounds__(256) void exp_loop(float* out, int iters, float seed) {
    float x[16];
    for (int i = 0; i < 16; ++i) x[i] = seed * float(threadIdx.x % 7 + i) - 1.0f;
    for (int it = 0; it < iters; ++it)
#pragma unroll
        for (int i = 0; i < 16; ++i) x[i] = __builtin_amdgcn_exp2f(x[i]) - 1.0f;
    float r = 0.f;
    for (int i = 0; i < 16; ++i) r += x[i];
    out[blockIdx.x * blockDim.x + threadIdx.x] = r;
}

// Streaming read of n16 16-byte words, grid-stride, four loads in flight per thread;
// one xor-sum per thread is stored.
__global__ __launch_bounds__(256) void read_loop(const u32x4_t* __restrict__ src, int64_t n16,
                                                 uint32_t* out) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    u32x4_t acc = {0u, 0u, 0u, 0u};
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4_t v0 = src[i], v1 = src[i + stride], v2 = src[i + 2 * stride],
                      v3 = src[i + 3 * stride];
        acc ^= v0 ^ v1 ^ v2 ^ v3;
    }
    for (; i < n16; i += stride) acc ^= src[i];
    out[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
}

}  // namespace

extern "C" {

// MFMA: `blocks` workgroups of 4 waves, each wave issuing 4 * iters MFMAs of 32768
// flops; out holds blocks * 256 floats.
int atf_probe_mfma_bf16(float* out, int blocks, int iters, void* stream) {
    if (out == nullptr || blocks < 1 || iters < 1) return -1;
    hipLaunchKernelGGL(mfma_loop, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), out,
                       iters, 0.001f);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

// MFMA 32x32x8 (16384 flops each), as atf_probe_mfma_bf16.
int atf_probe_mfma_bf16_k8(float* out, int blocks, int iters, void* stream) {
    if (out == nullptr || blocks < 1 || iters < 1) return -1;
    hipLaunchKernelGGL(mfma8_loop, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                       out, iters, 0.001f);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

// v_exp_f32: `blocks` x 256 threads, each 16 * iters exponentials; out blocks * 256 floats.
int atf_probe_exp2(float* out, int blocks, int iters, void* stream) {
    if (out == nullptr || blocks < 1 || iters < 1) return -1;
    hipLaunchKernelGGL(exp_loop, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), out,
                       iters, 0.001f);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

// HBM read: src holds bytes (a multiple of 16, 16-byte aligned); out blocks * 256 words.
int atf_probe_read(const void* src, int64_t bytes, uint32_t* out, int blocks, void* stream) {
    if (src == nullptr || out == nullptr || bytes < 16 || bytes % 16 != 0 || blocks < 1 ||
        reinterpret_cast<uintptr_t>(src) % 16 != 0)
        return -1;
    hipLaunchKernelGGL(read_loop, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4_t*>(src), bytes / 16, out);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
