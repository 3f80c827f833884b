// Measurement probes for the benchmark's second denominators on the GPU it
// runs on: the bandwidth of a plain device-to-device copy and the throughput
// of the int8 matrix instructions (dense 16x16x64 and 32x32x32, and the
// 4:2-sparse 16x16x128 the layer uses). Built as a library of its own
// (libsl_probe.so); not part of the layer or of its C ABI.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x16 __attribute__((ext_vector_type(16)));

// y[i] = x[i], 16 bytes a lane, four pieces in flight per lane, grid-stride
__global__ __launch_bounds__(256) void probe_copy_kernel(const i32x4 *__restrict__ x, i32x4 *__restrict__ y,
                                                         int64_t n)
{
    const int64_t step = (int64_t)gridDim.x * 256;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * step < n; i += 4 * step) {
        const i32x4 a = __builtin_nontemporal_load(x + i), b = __builtin_nontemporal_load(x + i + step);
        const i32x4 c = __builtin_nontemporal_load(x + i + 2 * step), d = __builtin_nontemporal_load(x + i + 3 * step);
        __builtin_nontemporal_store(a, y + i);
        __builtin_nontemporal_store(b, y + i + step);
        __builtin_nontemporal_store(c, y + i + 2 * step);
        __builtin_nontemporal_store(d, y + i + 3 * step);
    }
    for (; i < n; i += step) y[i] = x[i];
}

// iters rounds of 8 independent matrix instructions per wave; every thread
// writes one word of the results (so nothing is dropped), out has
// gridDim.x * 256 words. OP: 0 dense 16x16x64, 1 dense 32x32x32, 2 sparse
// 16x16x128.
template <int OP>
__global__ __launch_bounds__(256) void probe_mfma_kernel(int iters, int *out)
{
    const int lane = threadIdx.x & 63;
    const i32x4 a = {lane, 3, 5, 7};
    const i32x4 b = {1, lane, 2, 9};
    const i32x8 b8 = {lane, 1, 2, 3, 4, 5, 6, 7};
    int t = 0;
    if constexpr (OP == 1) {
        i32x16 acc[8];
        for (int i = 0; i < 8; ++i) acc[i] = i32x16{};
        for (int it = 0; it < iters; ++it)
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[i] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, acc[i], 0, 0, 0);
        for (int i = 0; i < 8; ++i) t ^= acc[i][0] ^ acc[i][15];
    } else {
        i32x4 acc[8];
        for (int i = 0; i < 8; ++i) acc[i] = i32x4{};
        for (int it = 0; it < iters; ++it)
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                if constexpr (OP == 0)
                    acc[i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[i], 0, 0, 0);
                else
                    acc[i] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(a, b8, acc[i], 0x44444444, 0, 0);
            }
        for (int i = 0; i < 8; ++i) t ^= acc[i][0] ^ acc[i][3];
    }
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = t;
}

extern "C" {

// Copies `bytes` (a multiple of 16) from x to y on `stream`; 0 on success.
int sl_probe_copy(const void *x, void *y, int64_t bytes, void *stream)
{
    if (bytes <= 0 || bytes % 16 || !x || !y) return -1;
    const int64_t n = bytes / 16;
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 256 * 8);
    hipLaunchKernelGGL(probe_copy_kernel, dim3((uint32_t)blocks), dim3(256), 0, (hipStream_t)stream,
                       (const i32x4 *)x, (i32x4 *)y, n);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// Runs `blocks` workgroups of 4 waves, each wave issuing 8 * iters
// instructions of kind op (0, 1, 2 as above); out holds blocks * 256 ints.
int sl_probe_mfma(int op, int blocks, int iters, int *out, void *stream)
{
    if (blocks <= 0 || iters <= 0 || !out || op < 0 || op > 2) return -1;
    hipStream_t s = (hipStream_t)stream;
    if (op == 0)
        hipLaunchKernelGGL(probe_mfma_kernel<0>, dim3(blocks), dim3(256), 0, s, iters, out);
    else if (op == 1)
        hipLaunchKernelGGL(probe_mfma_kernel<1>, dim3(blocks), dim3(256), 0, s, iters, out);
    else
        hipLaunchKernelGGL(probe_mfma_kernel<2>, dim3(blocks), dim3(256), 0, s, iters, out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

}  // extern "C"
