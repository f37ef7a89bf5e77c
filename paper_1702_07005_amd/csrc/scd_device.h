// scd_device.h -- device helpers shared by the epoch, hot-set and set-up kernels (gfx950, wave64):
// the per-epoch permutation, group reductions, shared-vector access, closed-form steps and segment
// loads.  Everything here is inline; each .hip file of the library includes it.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scd_kernels.h"

namespace scd {

// ----------------------------------------------------------------------------------------
// Permutation: 4-round balanced Feistel network on 2h bits + cycle-walking.
// ----------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t murmur_fmix32(uint32_t x) {
    x ^= x >> 16;
    x *= 0x85EBCA6BU;
    x ^= x >> 13;
    x *= 0xC2B2AE35U;
    x ^= x >> 16;
    return x;
}

__device__ __forceinline__ uint32_t feistel4(uint32_t x, const PermKeys& p) {
    uint32_t l = x >> p.h, r = x & p.mask, t;
    t = l ^ (murmur_fmix32(r ^ p.k[0]) & p.mask); l = r; r = t;
    t = l ^ (murmur_fmix32(r ^ p.k[1]) & p.mask); l = r; r = t;
    t = l ^ (murmur_fmix32(r ^ p.k[2]) & p.mask); l = r; r = t;
    t = l ^ (murmur_fmix32(r ^ p.k[3]) & p.mask); l = r; r = t;
    return (l << p.h) | r;
}

__device__ __forceinline__ uint32_t perm_at(uint32_t j, const PermKeys& p) {
    uint32_t x = feistel4(j, p);
    while (x >= p.n) x = feistel4(x, p);
    return x;
}

// ----------------------------------------------------------------------------------------
// Group reductions.  The butterfly makes every lane of the group hold the bitwise-identical
// sum (fp add is commutative), so all lanes take the same step without a broadcast.
// ----------------------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

template <int G>
__device__ __forceinline__ float group_sum(float x) {
    static_assert(G == 1 || G == 2 || G == 4 || G == 8 || G == 16 || G == 32 || G == 64, "group width");
    if constexpr (G >= 2) x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]  (lane ^ 1)
    if constexpr (G >= 4) x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]  (lane ^ 2)
    if constexpr (G >= 8) x += dpp_f<0x141>(x);  // row_half_mirror      (other quad of 8)
    if constexpr (G >= 16) x += dpp_f<0x140>(x); // row_mirror           (other half of 16)
    if constexpr (G >= 32) x += __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F));  // lane ^ 16
    if constexpr (G >= 64) {
        float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
        float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
        x = a + b;
    }
    return x;
}

template <int G>
__device__ __forceinline__ double group_sum_f64(double x) {
#pragma unroll
    for (int o = 1; o < G; o <<= 1) x += __shfl_xor(x, o, G);
    return x;
}

// ----------------------------------------------------------------------------------------
// Shared-vector access.
// ----------------------------------------------------------------------------------------
// The shared vector is stored as U = float, or double where fp32 accumulation would drift
// (very frequently updated entries); values enter the fp32 dot products as float.
template <bool FRESH, typename U>
__device__ __forceinline__ float ld_u(const U* p) {
    if constexpr (FRESH)
        return (float)__hip_atomic_load(const_cast<U*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
        return (float)*p;
}

__device__ __forceinline__ void atomic_add_u(float* p, float v) {
    __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void atomic_add_u(double* p, float v) {
    __hip_atomic_fetch_add(p, (double)v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ----------------------------------------------------------------------------------------
// Closed-form coordinate steps.  g = <a_m, u>, s = |a_m|^2, m_old = model[m], ylab = the
// coordinate's constant (cy_m = <y, a_m> for the ridge primal, the label for the duals).
// Returns the new model value; *coef is the factor of val in the scatter u += coef * a_m.
// ----------------------------------------------------------------------------------------
template <int FORM>
__device__ __forceinline__ float coord_step(float g, float s, float m_old, float ylab, const StepConsts& k,
                                            float* coef) {
    if constexpr (FORM == FORM_RIDGE_PRIMAL) {
        // eq. (update_primal): d = (<y - w, a_m> - lambda N beta_m) / (|a_m|^2 + lambda N);
        // w moves by d a_m.
        float d = ((ylab - g) - k.lamN * m_old) / (s + k.lamN);
        *coef = d;
        return m_old + d;
    } else if constexpr (FORM == FORM_SVM_DUAL) {
        // exact maximisation of the hinge dual along alpha_i, projected on [0, 1].
        float a = 1.0f;
        if (s > 0.0f) a = fminf(fmaxf(m_old + k.lamN * (1.0f - ylab * g) / s, 0.0f), 1.0f);
        *coef = (a - m_old) * ylab * k.inv_lamN;
        return a;
    } else {
        // eq. (update_dual): d = (lambda y_n - <wbar, abar_n> - lambda N alpha_n) / (lambda N + |abar_n|^2).
        float d = (k.lam * ylab - g - k.lamN * m_old) / (k.lamN + s);
        *coef = d;
        return m_old + d;
    }
}

// ----------------------------------------------------------------------------------------
// Per-coordinate metadata and register-cached segment slices.
// ----------------------------------------------------------------------------------------
struct CoordMeta {
    int64_t s0, s1;
    uint32_t m;
    float m_old, sn, ylab;
};

__device__ __forceinline__ CoordMeta load_meta_of(const EpochArgs& a, uint32_t m) {
    CoordMeta c;
    c.m = m;
    c.s0 = a.ptr[c.m];
    c.s1 = a.ptr[c.m + 1];
    c.m_old = a.model[c.m];
    c.sn = a.norms[c.m];
    c.ylab = a.y[c.m];
    return c;
}

__device__ __forceinline__ CoordMeta load_meta(const EpochArgs& a, uint32_t j) {
    return load_meta_of(a, perm_at(j, a.perm));
}

// Register slice r of a segment: element s0 + lane + r*G.  Lanes past the end read element 0
// (always present: the library never hands the kernels an empty idx/val) with weight 0, so the
// hot path needs no branches and the compiler can count outstanding loads exactly.
template <int G, int R>
__device__ __forceinline__ void load_seg(const EpochArgs& a, const CoordMeta& c, int lane, int (&ci)[R],
                                         float (&cv)[R]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t k = c.s0 + lane + (int64_t)r * G;
        const bool in = k < c.s1;
        const int64_t kk = in ? k : 0;
        ci[r] = a.idx[kk];
        const float v = a.val[kk];
        cv[r] = in ? v : 0.0f;
    }
}


// As load_seg, but lanes past the end keep entry 0's value: the pipelined kernel masks them
// through out-of-range shared-vector offsets (the gather returns 0, the atomic is dropped), so
// no select has to wait for the loaded value next to the load.
template <int G, int R>
__device__ __forceinline__ void load_seg_raw(const EpochArgs& a, const CoordMeta& c, int lane, int (&ci)[R],
                                             float (&cv)[R]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t k = c.s0 + lane + (int64_t)r * G;
        const int64_t kk = k < c.s1 ? k : 0;
        ci[r] = a.idx[kk];
        cv[r] = a.val[kk];
    }
}

// ----------------------------------------------------------------------------------------
// Shared-vector access of the pipelined kernel.  The shared vector is addressed as a raw
// buffer: the hardware range check returns 0 for a load at an offset outside [0, bytes) and
// drops an fp32 atomic there.  A lane past its segment's end, or a whole coordinate whose
// step is zero, thus issues the same instructions as the others with no memory traffic, and
// each iteration of k_epoch_pipe issues a fixed number of vector memory operations: the
// compiler can wait for one load without also waiting for atomics issued after it (the
// completion counter is in order).  There is no fp64 buffer atomic builtin, so an fp64
// shared vector is updated with unconditional global atomics whose inactive lanes add 0 to a
// slot of their own in a scratch array (`sink`) instead.  (A FLAT atomic aimed at LDS would
// avoid that traffic, but a pending FLAT operation makes the compiler wait for everything.)
// ----------------------------------------------------------------------------------------
template <typename U>
struct SharedBuf {
    __amdgpu_buffer_rsrc_t r;
    uint32_t oob;  // first out-of-range byte offset
    U* base;
    U* sink;       // fp64 only: this lane's scratch slot
    uint32_t shift;  // log2 of the bytes between consecutive entries
};

template <typename U>
__device__ __forceinline__ SharedBuf<U> shared_buf(void* u, uint32_t bytes, U* sink, uint32_t shift) {
    // word 3 = 0x00020000: 32-bit data format, the gfx9-family raw-buffer setting.
    return {__builtin_amdgcn_make_buffer_rsrc(u, (short)0, (int)bytes, 0x00020000), bytes, static_cast<U*>(u), sink,
            shift};
}

template <bool FRESH, typename U>
__device__ __forceinline__ float buf_load(const SharedBuf<U>& b, uint32_t i, bool in) {
    // cache policy 16 = sc1: device-scope load, as __hip_atomic_load at agent scope emits.
    constexpr int pol = FRESH ? 16 : 0;
    const uint32_t off = in ? i << b.shift : b.oob;
    if constexpr (sizeof(U) == 4) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b.r, (int)off, 0, pol));
    } else {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(b.r, (int)off, 0, pol);
        return (float)__builtin_bit_cast(double, v);
    }
}

template <typename U>
__device__ __forceinline__ void buf_atomic_add(const SharedBuf<U>& b, uint32_t i, bool in, float v) {
    if constexpr (sizeof(U) == 4) {
        (void)__builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(v, b.r, (int)(in ? i << b.shift : b.oob), 0, 0);
    } else {
        U* p = in ? reinterpret_cast<U*>(reinterpret_cast<char*>(b.base) + ((size_t)i << b.shift)) : b.sink;
        __hip_atomic_fetch_add(p, in ? (double)v : 0.0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// A segment longer than the register slices, streamed in blocks of G * kLongBlock entries:
// each lane loads kLongBlock indices and values, then issues kLongBlock gathers (or atomics),
// so a block costs one or two memory round trips instead of one per entry.  Segments that
// cover most of the shared vector otherwise stay between their gather and their scatter for
// milliseconds, long enough to overlap others they couple strongly with.  Lanes past the end
// re-read entry s0 and are masked by an out-of-range shared-vector offset.
constexpr int kLongBlock = 16;

template <int G, bool FRESH, typename U>
__device__ __forceinline__ float long_dot(const EpochArgs& a, const SharedBuf<U>& ub, int lane, int64_t s0,
                                          int64_t s1) {
    float acc = 0.0f;
    for (int64_t b = s0; b < s1; b += (int64_t)G * kLongBlock) {
        int ix[kLongBlock];
        float vx[kLongBlock];
        bool in[kLongBlock];
#pragma unroll
        for (int r = 0; r < kLongBlock; ++r) {
            const int64_t k = b + lane + (int64_t)r * G;
            in[r] = k < s1;
            const int64_t kk = in[r] ? k : s0;
            ix[r] = a.idx[kk];
            vx[r] = a.val[kk];
        }
        float gv[kLongBlock];
#pragma unroll
        for (int r = 0; r < kLongBlock; ++r) gv[r] = buf_load<FRESH>(ub, (uint32_t)ix[r], in[r]);
#pragma unroll
        for (int r = 0; r < kLongBlock; ++r) acc = fmaf(vx[r], gv[r], acc);
    }
    return acc;
}

template <int G, typename U>
__device__ __forceinline__ void long_scatter(const EpochArgs& a, const SharedBuf<U>& ub, int lane, int64_t s0,
                                             int64_t s1, float coef) {
    for (int64_t b = s0; b < s1; b += (int64_t)G * kLongBlock) {
        int ix[kLongBlock];
        float vx[kLongBlock];
        bool in[kLongBlock];
#pragma unroll
        for (int r = 0; r < kLongBlock; ++r) {
            const int64_t k = b + lane + (int64_t)r * G;
            in[r] = k < s1;
            const int64_t kk = in[r] ? k : s0;
            ix[r] = a.idx[kk];
            vx[r] = a.val[kk];
        }
#pragma unroll
        for (int r = 0; r < kLongBlock; ++r) buf_atomic_add(ub, (uint32_t)ix[r], in[r], coef * vx[r]);
    }
}

// Workgroups for a grid-stride pass over n elements (256 threads, at most 8192 workgroups).
inline unsigned grid_for(int64_t n) {
    int64_t b = (n + 255) / 256;
    if (b > 8192) b = 8192;
    if (b < 1) b = 1;
    return (unsigned)b;
}

}  // namespace scd
