// Elementwise and reduction kernels of the plan search (Sec. 3.5, Alg. 1):
// the mean relative absolute error between two bf16 tensors, and the bf16
// residual add of the surrogate model's blocks.  Both are HBM-bound streams
// of 16-byte chunks.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "dfa_internal.h"

namespace dfa {

// Partial sums of the allocation-free MRAE entry point: one fp64 value per
// workgroup of the reduction, 8 KiB, one copy per device, held until the
// process ends.  In host code this name is only a stand-in for the symbol:
// kernels get the device address that scratch_partials() looks up.
static __device__ __align__(256) double scratch[MRAE_SCRATCH_PARTIALS];

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int MR_THREADS = 256;

__device__ __forceinline__ float bf16_lo(uint32_t x) { return __builtin_bit_cast(float, x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __builtin_bit_cast(float, x & 0xFFFF0000u); }

__device__ __forceinline__ float rel_err(float x, float y, float eps) {
    const float r = fabsf(x - y) / (fmaxf(fabsf(x), fabsf(y)) + eps);
    return fminf(r, 10.0f);   // r >= 0, so the lower clip at 0 is implicit
}

__device__ __forceinline__ uint32_t round_bf16(float f) {
    // round to nearest even (inputs are sums of finite bf16 values)
    const uint32_t u = __builtin_bit_cast(uint32_t, f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// Per-workgroup partial sums of the clipped relative errors, in fp64.  Each
// lane sums its grid-stride share of 16-byte chunks in fp32; the tail of
// fewer than 8 elements goes to the first lanes of workgroup 0.
__global__ void __launch_bounds__(MR_THREADS) mrae_partial_kernel(const u32x4* __restrict__ a, const u32x4* __restrict__ b,
                                                                  size_t n, float eps, double* __restrict__ partial) {
    const size_t n8 = n / 8;
    float acc = 0.f;
    for (size_t i = (size_t)blockIdx.x * MR_THREADS + threadIdx.x; i < n8; i += (size_t)gridDim.x * MR_THREADS) {
        const u32x4 va = a[i], vb = b[i];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            acc += rel_err(bf16_lo(va[k]), bf16_lo(vb[k]), eps);
            acc += rel_err(bf16_hi(va[k]), bf16_hi(vb[k]), eps);
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < n % 8) {
        const uint16_t* ah = (const uint16_t*)a;
        const uint16_t* bh = (const uint16_t*)b;
        const size_t j = n8 * 8 + threadIdx.x;
        acc += rel_err(__builtin_bit_cast(float, (uint32_t)ah[j] << 16), __builtin_bit_cast(float, (uint32_t)bh[j] << 16),
                       eps);
    }
    double v = acc;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    __shared__ double wsum[MR_THREADS / 64];
    if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
        for (int i = 0; i < MR_THREADS / 64; ++i) s += wsum[i];
        partial[blockIdx.x] = s;
    }
}

// Sum of the partials in a fixed order, divided by n.
__global__ void __launch_bounds__(MR_THREADS) mrae_final_kernel(const double* __restrict__ partial, int np, size_t n,
                                                                double* __restrict__ out) {
    __shared__ double s[MR_THREADS];
    double v = 0.0;
    for (int i = threadIdx.x; i < np; i += MR_THREADS) v += partial[i];
    s[threadIdx.x] = v;
    __syncthreads();
    for (int k = MR_THREADS / 2; k > 0; k >>= 1) {
        if (threadIdx.x < k) s[threadIdx.x] += s[threadIdx.x + k];
        __syncthreads();
    }
    if (threadIdx.x == 0) out[0] = n ? s[0] / (double)n : 0.0;
}

// out = bf16(a + b), elementwise; out may alias a or b.
__global__ void __launch_bounds__(256) add_bf16_kernel(const u32x4* a, const u32x4* b, u32x4* out, size_t n8) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (size_t)gridDim.x * 256) {
        const u32x4 va = a[i], vb = b[i];
        u32x4 r;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t lo = round_bf16(bf16_lo(va[k]) + bf16_lo(vb[k]));
            const uint32_t hi = round_bf16(bf16_hi(va[k]) + bf16_hi(vb[k]));
            r[k] = lo | (hi << 16);
        }
        out[i] = r;
    }
}

}  // namespace

size_t mrae_workgroups(size_t n, int max_partials) {
    const size_t n8 = n / 8;
    size_t blocks = (n8 + MR_THREADS - 1) / MR_THREADS;
    if (blocks < 1) blocks = 1;
    if (blocks > (size_t)max_partials) blocks = (size_t)max_partials;
    return blocks;
}

hipError_t launch_mrae(const void* a, const void* b, size_t n, float eps, double* partial, int max_partials,
                       double* out, hipStream_t stream) {
    const size_t blocks = mrae_workgroups(n, max_partials);
    hipLaunchKernelGGL(mrae_partial_kernel, dim3((unsigned)blocks), dim3(MR_THREADS), 0, stream, (const u32x4*)a,
                       (const u32x4*)b, n, eps, partial);
    hipLaunchKernelGGL(mrae_final_kernel, dim3(1), dim3(MR_THREADS), 0, stream, partial, (int)blocks, n, out);
    return hipGetLastError();
}

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
double* g_scratch_ptr[MAX_DEVICES];
}  // namespace

// Device address of `scratch` on the calling thread's current device, looked
// up once per device (with that device current) and kept.
hipError_t scratch_partials(double** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = (double*)p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_add_bf16(const void* a, const void* b, void* out, size_t n, hipStream_t stream) {
    const size_t n8 = n / 8;
    if (n8 == 0) return hipSuccess;
    size_t blocks = (n8 + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(add_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, (const u32x4*)a, (const u32x4*)b,
                       (u32x4*)out, n8);
    return hipGetLastError();
}

}  // namespace dfa
