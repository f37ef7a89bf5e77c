// ceiling.hip -- measurement aid for the benchmark (not part of the solver): the device-wide
// rates that bound an asynchronous coordinate-descent epoch on this GPU.
//   mode 0: scattered fp32 device-scope atomic adds (no return) into an array of L floats;
//   mode 1: scattered loads from the array and, independently, scattered atomic adds into it
//           (8 of each in flight per lane) -- the pattern of an epoch, where the atomics keep
//           invalidating the lines the gathers read;
//   mode 2: streaming copy of L floats (reads + writes);
//   mode 3: as mode 1 with entry i stored at float 16 i (one entry per 64 bytes);
//   modes 4-7: scattered atomic adds into a footprint touched by one XCD only: the array holds 8
//           regions of L entries, and each workgroup adds only into the region of the XCD it runs on
//           (read from the hardware XCC_ID register), fp32 at agent scope (4) and workgroup scope
//           (5), fp64 at agent scope (6) and workgroup scope (7).  If an XCD's L2 could resolve
//           atomics on lines no other XCD touches, these would run at L2 rates.
// Returns operations per second (modes 0, 1, 3-7: atomic adds, i.e. gather-and-atomic pairs for
// 1 and 3; mode 2: bytes moved).
//
// scd_probe_xcc_map: the XCD (hardware XCC_ID) each of `blocks` workgroups of a plain launch ran on.
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

// The XCD this wave runs on: bits [3:0] of the XCC_ID hardware register.
__device__ __forceinline__ uint32_t xcc_id() { return (uint32_t)__builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 15u; }

template <typename T, int SCOPE>
__global__ __launch_bounds__(256) void k_rate_xcd(T* __restrict__ a, uint32_t L, uint32_t per) {
    const uint32_t t = blockIdx.x * 256u + threadIdx.x;
    T* const region = a + (size_t)(xcc_id() & 7u) * L;
    for (uint32_t i = 0; i < per; i += 8) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const uint32_t h = mix32(t * per + i + r);
            __hip_atomic_fetch_add(region + h % L, (T)1, __ATOMIC_RELAXED, SCOPE);
        }
    }
}

__global__ __launch_bounds__(64) void k_xcc_map(uint32_t* __restrict__ out) {
    if (threadIdx.x == 0) out[blockIdx.x] = xcc_id();
}

__global__ __launch_bounds__(256) void k_copy(const float4* __restrict__ in, float4* __restrict__ out, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) out[i] = in[i];
}

}  // namespace

extern "C" int scd_probe_rate(int mode, uint64_t L, void* stream, double* out) {
    if (!out || L < 1024 || L > (1ull << 31) || mode < 0 || mode > 7 || (mode == 3 && L > (1ull << 26)) ||
        (mode >= 4 && L > (1ull << 26)))
        return -1;
    hipStream_t s = (hipStream_t)stream;
    float* a = nullptr;
    float* b = nullptr;
    // modes 4-7: 8 regions of L entries (fp32, or fp64 in modes 6-7)
    const size_t bytes = mode >= 4 ? (mode >= 6 ? sizeof(double) : sizeof(float)) * 8 * (size_t)L
                                   : sizeof(float) * (size_t)L * (mode == 3 ? 16 : 1);
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
        if (mode == 4)
            hipLaunchKernelGGL((k_rate_xcd<float, __HIP_MEMORY_SCOPE_AGENT>), dim3(blocks), dim3(256), 0, s, a,
                               (uint32_t)L, per);
        if (mode == 5)
            hipLaunchKernelGGL((k_rate_xcd<float, __HIP_MEMORY_SCOPE_WORKGROUP>), dim3(blocks), dim3(256), 0, s, a,
                               (uint32_t)L, per);
        if (mode == 6)
            hipLaunchKernelGGL((k_rate_xcd<double, __HIP_MEMORY_SCOPE_AGENT>), dim3(blocks), dim3(256), 0, s,
                               reinterpret_cast<double*>(a), (uint32_t)L, per);
        if (mode == 7)
            hipLaunchKernelGGL((k_rate_xcd<double, __HIP_MEMORY_SCOPE_WORKGROUP>), dim3(blocks), dim3(256), 0, s,
                               reinterpret_cast<double*>(a), (uint32_t)L, per);
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

extern "C" int scd_probe_xcc_map(uint32_t blocks, uint32_t* out_host) {
    if (!out_host || blocks < 1 || blocks > (1u << 20)) return -1;
    uint32_t* d = nullptr;
    if (hipMalloc(&d, sizeof(uint32_t) * blocks) != hipSuccess) return -3;
    hipLaunchKernelGGL(k_xcc_map, dim3(blocks), dim3(64), 0, nullptr, d);
    int rc = hipGetLastError() == hipSuccess &&
                     hipMemcpy(out_host, d, sizeof(uint32_t) * blocks, hipMemcpyDeviceToHost) == hipSuccess
                 ? 0
                 : -4;
    (void)hipFree(d);
    return rc;
}
