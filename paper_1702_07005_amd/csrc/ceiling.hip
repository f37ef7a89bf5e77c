// ceiling.hip -- measurement aid for the benchmark (not part of the solver): the device-wide
// rates that bound an asynchronous coordinate-descent epoch on this GPU.
//   mode 0: scattered fp32 device-scope atomic adds (no return) into an array of L floats;
//   mode 1: scattered loads from the array and, independently, scattered atomic adds into it
//           (8 of each in flight per lane) -- the pattern of an epoch, where the atomics keep
//           invalidating the lines the gathers read;
//   mode 2: streaming copy of L floats (reads + writes);
//   mode 3: as mode 1 with entry i stored at float 16 i (one entry per 64 bytes).
// Returns operations per second (modes 0, 1, 3: atomic adds, i.e. gather-and-atomic pairs for
// 1 and 3; mode 2: bytes moved).
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint32_t mix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x7FEB352DU;
    x ^= x >> 15;
    x *= 0x846CA68BU;
    x ^= x >> 16;
    return x;
}

template <int MODE>
__global__ __launch_bounds__(256) void k_rate(float* __restrict__ a, uint32_t L, uint32_t per,
                                              float* __restrict__ sink) {
    constexpr uint32_t stride = MODE == 3 ? 16u : 1u;
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    float acc = 0.0f;
    for (uint32_t i = 0; i < per; i += 8) {
        float g[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const uint32_t h = mix32(t * per + i + r);
            if (MODE != 0) g[r] = a[(size_t)(mix32(h ^ 0x9E3779B9u) % L) * stride];
            __hip_atomic_fetch_add(a + (size_t)(h % L) * stride, 1.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (MODE != 0) {
#pragma unroll
            for (int r = 0; r < 8; ++r) acc += g[r];
        }
    }
    if (acc == 123456.0f) sink[0] = acc;  // keeps the loads
}

__global__ __launch_bounds__(256) void k_copy(const float4* __restrict__ in, float4* __restrict__ out, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) out[i] = in[i];
}

}  // namespace

extern "C" int scd_probe_rate(int mode, uint64_t L, void* stream, double* out) {
    if (!out || L < 1024 || L > (1ull << 31) || mode < 0 || mode > 3 || (mode == 3 && L > (1ull << 26))) return -1;
    hipStream_t s = (hipStream_t)stream;
    float* a = nullptr;
    float* b = nullptr;
    const size_t bytes = sizeof(float) * (size_t)L * (mode == 3 ? 16 : 1);
    if (hipMalloc(&a, bytes) != hipSuccess) return -3;
    if (hipMalloc(&b, mode == 2 ? bytes : 64) != hipSuccess) {  // copy target, or the loads' sink
        (void)hipFree(a);
        return -3;
    }
    int rc = 0;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    if (hipMemsetAsync(a, 0, bytes, s) != hipSuccess || hipEventCreate(&e0) != hipSuccess ||
        hipEventCreate(&e1) != hipSuccess)
        rc = -4;
    const uint32_t blocks = 256 * 32, per = 64;
    float best = 1e30f;
    for (int rep = 0; rep < 3 && rc == 0; ++rep) {
        (void)hipEventRecord(e0, s);
        if (mode == 0) hipLaunchKernelGGL(k_rate<0>, dim3(blocks), dim3(256), 0, s, a, (uint32_t)L, per, b);
        if (mode == 1) hipLaunchKernelGGL(k_rate<1>, dim3(blocks), dim3(256), 0, s, a, (uint32_t)L, per, b);
        if (mode == 3) hipLaunchKernelGGL(k_rate<3>, dim3(blocks), dim3(256), 0, s, a, (uint32_t)L, per, b);
        if (mode == 2)
            hipLaunchKernelGGL(k_copy, dim3(256 * 64), dim3(256), 0, s, reinterpret_cast<const float4*>(a),
                               reinterpret_cast<float4*>(b), bytes / 16);
        (void)hipEventRecord(e1, s);
        if (hipGetLastError() != hipSuccess || hipEventSynchronize(e1) != hipSuccess) {
            rc = -4;
            break;
        }
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, e0, e1);
        if (ms < best) best = ms;
    }
    if (rc == 0)
        *out = mode == 2 ? 2.0 * (double)(bytes / 16 * 16) / (best * 1e-3)
                         : (double)blocks * 256.0 * per / (best * 1e-3);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    (void)hipFree(a);
    if (b) (void)hipFree(b);
    return rc;
}
