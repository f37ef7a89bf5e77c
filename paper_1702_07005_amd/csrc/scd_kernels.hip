// scd_kernels.hip -- HIP kernels for gfx950 (CDNA4, wave64) of asynchronous stochastic
// coordinate descent/ascent (arXiv 1702.07005, Sec. III-C "TPA-SCD", Alg. 2).
//
// Every coordinate c owns one segment [ptr[c], ptr[c+1]) of (idx, val): a column of A for
// the ridge primal (CSC), a row for the duals (CSR).  One epoch = one persistent launch in
// which groups of lanes take permutation positions j = g, g + P, g + 2P, ... (P groups in
// flight: the "window"), and for the coordinate m = pi(j):
//   1. gather  g = <a_m, u>   over the segment (u = the shared vector, see below),
//   2. reduce the lane partials inside the group (DPP / swizzle, LDS across waves),
//   3. step    closed form of the formulation -> model[m], scatter coefficient,
//   4. scatter u[idx] += coef * val  with device-scope fp32 atomics (no return).
//
// Shared vector kept on the device, per formulation:
//   ridge primal : w = A beta.  The step needs <y - w, a_m> (eq. update_primal); it is taken
//                  as cy_m - <w, a_m> with cy_m = <y, a_m> computed once at set-up, so each
//                  stored entry costs one gather (w) instead of two (y and w).
//   SVM dual     : w = sum_i alpha_i y_i x_i / (lambda N).
//   ridge dual   : wbar = A^T alpha (eq. update_dual).
// `y` in the epoch arguments is the per-coordinate constant: cy for the ridge primal, the
// label for the duals.
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

__global__ void k_perm_fill(PermKeys p, int32_t* __restrict__ out) {
    uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j < p.n) out[j] = (int32_t)perm_at(j, p);
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
// Epoch kernel, sub-wave / wave groups: G lanes per coordinate, 256-thread workgroups,
// persistent over permutation positions j = g, g + P, ...  The first R*G elements of a
// segment stay in registers between the gather and the scatter (A is read once); longer
// segments stream their tail twice; TAIL = false is the instantiation for matrices whose
// segments all fit the register slices (no tail code, exact load counting).
//
// Software pipeline: loads and no-return atomics share one in-order completion counter per
// wave, so waiting for a load also waits for every atomic issued before it.  Each group
// therefore issues the NEXT coordinate's metadata and segment loads before the CURRENT
// coordinate's atomics; consuming them later never waits on the scatter.  Issue order per
// iteration: gathers(k), meta(k+1), [reduce + step k], segment(k+1), atomics(k).
// ----------------------------------------------------------------------------------------
template <int FORM, int G, int R, bool FRESH, bool TAIL, typename U>
__global__ __launch_bounds__(256) void k_epoch_group(EpochArgs a) {
    U* const uu = static_cast<U*>(a.u);
    const int lane = threadIdx.x & (G - 1);
    const uint32_t gid = (blockIdx.x * 256u + threadIdx.x) / G;
    if (gid >= a.n_groups || gid >= a.perm.n) return;
    uint32_t j = gid;
    CoordMeta cur = load_meta(a, j);
    int ci[R];
    float cv[R];
    load_seg<G, R>(a, cur, lane, ci, cv);
    for (;;) {
        float gv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) gv[r] = ld_u<FRESH>(uu + ci[r]);
        const uint32_t jn = j + a.n_groups;
        const bool more = jn < a.perm.n;
        const CoordMeta nxt = load_meta(a, more ? jn : j);
        float acc = 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r) acc = fmaf(cv[r], gv[r], acc);
        const int64_t len = cur.s1 - cur.s0;
        if constexpr (TAIL) {
            for (int64_t k = cur.s0 + lane + (int64_t)R * G; k < cur.s1; k += G)
                acc = fmaf(a.val[k], ld_u<FRESH>(uu + a.idx[k]), acc);
        }
        const float g = group_sum<G>(acc);
        float coef;
        const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
        if (lane == 0) a.model[cur.m] = m_new;
        int ni[R];
        float nv[R];
        load_seg<G, R>(a, nxt, lane, ni, nv);
        if (coef != 0.0f) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if ((int64_t)(lane + r * G) < len) atomic_add_u(uu + ci[r], coef * cv[r]);
            if constexpr (TAIL) {
                for (int64_t k = cur.s0 + lane + (int64_t)R * G; k < cur.s1; k += G)
                    atomic_add_u(uu + a.idx[k], coef * a.val[k]);
            }
        }
        if (!more) break;
        j = jn;
        cur = nxt;
        for (int r = 0; r < R; ++r) {  // register renaming; scalarised by the compiler
            ci[r] = ni[r];
            cv[r] = nv[r];
        }
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
};

template <typename U>
__device__ __forceinline__ SharedBuf<U> shared_buf(void* u, uint32_t bytes, U* sink) {
    // word 3 = 0x00020000: 32-bit data format, the gfx9-family raw-buffer setting.
    return {__builtin_amdgcn_make_buffer_rsrc(u, (short)0, (int)bytes, 0x00020000), bytes, static_cast<U*>(u), sink};
}

template <bool FRESH, typename U>
__device__ __forceinline__ float buf_load(const SharedBuf<U>& b, uint32_t i, bool in) {
    // cache policy 16 = sc1: device-scope load, as __hip_atomic_load at agent scope emits.
    constexpr int pol = FRESH ? 16 : 0;
    const uint32_t off = in ? i * (uint32_t)sizeof(U) : b.oob;
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
        (void)__builtin_amdgcn_raw_ptr_buffer_atomic_fadd_f32(v, b.r, (int)(in ? i * 4u : b.oob), 0, 0);
    } else {
        U* p = in ? b.base + i : b.sink;
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

// One coordinate of k_epoch_pipe.  On entry `ci/cv` hold the current coordinate's segment
// and `nxt` the next one's metadata (both loaded one step earlier).  Issue order:
//   gathers(cur), segment(nxt) -> ni/nv, metadata two positions ahead -> nn,
//   [wait for the gathers] reduce + step + model store, atomics(cur).
// The loads consumed by the next step are all issued before this step's atomics.  Without
// `drain`, the next gathers follow the atomics at once: one gather round trip per coordinate,
// but a group then has two coordinates in flight (the previous one's scatter may not have
// landed).  With `drain` (the window binds) the group waits for its atomics first: two round
// trips per coordinate, against three for the plain kernels, whose segment and metadata
// loads are not prefetched.
template <int G>
__device__ __forceinline__ float pipe_reduce(float acc, float (*part)[G > 64 ? G / 64 : 1], int& buf) {
    if constexpr (G <= 64) {
        return group_sum<G>(acc);
    } else {
        constexpr int NW = G / 64;
        acc = group_sum<64>(acc);
        if ((threadIdx.x & 63) == 0) part[buf][threadIdx.x >> 6] = acc;
        __syncthreads();
        float g = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) g += part[buf][w];
        buf ^= 1;
        return g;
    }
}

// A segment longer than the register slices (rare; skewed lengths): stream it twice, gather
// then scatter, in blocks (long_dot, long_scatter) with ordinary waits.  It ends by issuing the same operations, in the same
// order, as the end of the pipelined step (next segment, metadata two ahead, then 1 + R
// operations standing in for the model store and the atomics), so that the compiler's wait
// counts after the step stay exact on both paths.
template <int FORM, int G, int R, bool FRESH, typename U>
__device__ __forceinline__ void pipe_long(const EpochArgs& a, const SharedBuf<U>& ub, int lane, uint32_t j,
                                       const CoordMeta& cur, const CoordMeta& nxt, int (&ni)[R], float (&nv)[R],
                                       CoordMeta& nn, float (*part)[G > 64 ? G / 64 : 1], int& buf) {
    const float g = pipe_reduce<G>(long_dot<G, FRESH>(a, ub, lane, cur.s0, cur.s1), part, buf);
    float coef;
    const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
    a.model[cur.m] = m_new;
    if (coef != 0.0f) long_scatter<G>(a, ub, lane, cur.s0, cur.s1, coef);
    const uint64_t P = a.n_groups, n = a.perm.n;
    load_seg_raw<G, R>(a, nxt, lane, ni, nv);
    const uint64_t j2 = (uint64_t)j + 2 * P;
    nn = load_meta_of(a, perm_at(j2 < n ? (uint32_t)j2 : j, a.perm));
#pragma unroll
    for (int r = 0; r <= R; ++r) buf_atomic_add(ub, 0u, false, 0.0f);
}

template <int FORM, int G, int R, bool FRESH, typename U>
__device__ __forceinline__ bool pipe_step(const EpochArgs& a, const SharedBuf<U>& ub, int lane, uint32_t j,
                                          const CoordMeta& cur, const int (&ci)[R], const float (&cv)[R],
                                          const CoordMeta& nxt, int (&ni)[R], float (&nv)[R], CoordMeta& nn,
                                          float (*part)[G > 64 ? G / 64 : 1], int& buf) {
    // When the window binds, the previous coordinate's atomics (the wave's latest operations) must
    // land before this coordinate gathers, so that a group never has two coordinates in flight.
    if (a.drain) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    const int64_t len = cur.s1 - cur.s0;
    if (len > (int64_t)G * R) {
        pipe_long<FORM, G, R, FRESH, U>(a, ub, lane, j, cur, nxt, ni, nv, nn, part, buf);
        return (uint64_t)j + a.n_groups < a.perm.n;
    }
    float gv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) gv[r] = buf_load<FRESH>(ub, (uint32_t)ci[r], (int64_t)(lane + r * G) < len);
    // The scheduler may not move work across these points: the gathers go out first, and the
    // prefetches are issued before the wait for the gathers (it would otherwise sink them
    // below the dot product and put their round trip on the critical path).
    __builtin_amdgcn_sched_barrier(0);
    const uint64_t P = a.n_groups, n = a.perm.n;
    const bool more = (uint64_t)j + P < n;
    load_seg_raw<G, R>(a, nxt, lane, ni, nv);
    const uint64_t j2 = (uint64_t)j + 2 * P;
    const uint32_t m2 = perm_at(j2 < n ? (uint32_t)j2 : j, a.perm);
    nn = load_meta_of(a, m2);
    __builtin_amdgcn_sched_barrier(0);
    float acc = 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) acc = fmaf(cv[r], gv[r], acc);
    const float g = pipe_reduce<G>(acc, part, buf);
    float coef;
    const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
    a.model[cur.m] = m_new;  // every lane of the group stores the same value: no branch
    const bool moves = coef != 0.0f;
#pragma unroll
    for (int r = 0; r < R; ++r) buf_atomic_add(ub, (uint32_t)ci[r], moves && (int64_t)(lane + r * G) < len, coef * cv[r]);
    return more;
}

// ----------------------------------------------------------------------------------------
// Epoch kernel, software-pipelined two coordinates deep, shared vector addressed as a raw
// buffer.  G lanes per coordinate (4..64 in 256-thread workgroups, or G = 256: one
// workgroup per coordinate, wave sums combined through LDS).  Segments of up to G*R entries
// stay in registers; longer ones take pipe_long.  The loop body is unrolled twice so that the register
// arrays of consecutive coordinates alternate instead of being copied (a copy would have to
// wait for the loads that fill it).
// ----------------------------------------------------------------------------------------
template <int FORM, int G, int R, bool FRESH, typename U>
__global__ __launch_bounds__(256) void k_epoch_pipe(EpochArgs a) {
    __shared__ float part[2][G > 64 ? G / 64 : 1];
    const int lane = threadIdx.x & (G - 1);
    const uint32_t gid = (blockIdx.x * 256u + threadIdx.x) / G;
    if (gid >= a.n_groups || gid >= a.perm.n) return;  // G = 256: the whole workgroup leaves
    const SharedBuf<U> ub =
        shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x);
    const uint32_t P = a.n_groups;
    uint32_t j = gid;
    int buf = 0;
    CoordMeta cA = load_meta(a, j);
    int ciA[R], ciB[R];
    float cvA[R], cvB[R];
    load_seg_raw<G, R>(a, cA, lane, ciA, cvA);
    CoordMeta cB = load_meta(a, (uint64_t)j + P < a.perm.n ? j + P : j);
    // Inactive operations standing in for the model store and the atomics that follow the
    // metadata loads inside the loop: both ways into the loop then have the same operations
    // outstanding, and the compiler's wait counts need not assume the shorter one.
#pragma unroll
    for (int r = 0; r <= R; ++r) buf_atomic_add(ub, 0u, false, 0.0f);
    for (;;) {
        CoordMeta cA2, cB2;
        if (!pipe_step<FORM, G, R, FRESH>(a, ub, lane, j, cA, ciA, cvA, cB, ciB, cvB, cA2, part, buf)) break;
        j += P;
        if (!pipe_step<FORM, G, R, FRESH>(a, ub, lane, j, cB, ciB, cvB, cA2, ciA, cvA, cB2, part, buf)) break;
        j += P;
        cA = cA2;
        cB = cB2;
    }
}

// ----------------------------------------------------------------------------------------
// Epoch kernel with a position queue: one workgroup per coordinate, draining, and positions
// claimed in permutation order from a counter (queue[0]) instead of taken at a fixed stride.
// With a fixed stride, a workgroup that draws long segments falls behind the others; on
// skewed lengths the processing order then drifts by thousands of positions from the
// permutation, and the iterates follow a different sequence than the sequential algorithm
// on the same permutation (by as much as a different permutation would).  With the queue a
// coordinate starts within a few windows of its position.
//
// A claim takes `chunk` consecutive positions (one atomic add of `chunk`): one counter
// serves about 8e7 returning atomics per second, so wide windows claim several positions at
// a time.  Chunk c of a workgroup covers its steps [c*chunk, (c+1)*chunk); it is claimed in
// step c*chunk - kQueueLead with one returning atomic issued with the prefetch loads.  Every
// step issues that atomic through a raw buffer whose range holds only queue[0]: lane 0 at
// offset 0 when the step claims, every other lane (and lane 0 in other steps) out of range,
// which makes no access.  There is no branch, so the compiler's count of the operations issued
// after the gathers stays exact.  The claim lands by the next step's drain; lane 0 writes it to
// an LDS ring before that step's reduction barrier, and every wave reads it after the barrier,
// when it loads the metadata of the chunk's first coordinate two steps ahead.  No wait or
// barrier is added.  Each workgroup counts itself out in queue[1]; the last one resets both
// words for the next launch.
// ----------------------------------------------------------------------------------------
constexpr int kQueueRing = 4;  // chunk bases held in LDS (chunk number mod 4)
constexpr int kQueueLead = 4;  // steps between a claim and the first step of its chunk

// Position of step `k` of this workgroup (>= n once the queue is exhausted).
__device__ __forceinline__ uint32_t queue_pos(const uint32_t* ring, uint32_t k, uint32_t chunk) {
    return ring[(k / chunk) % kQueueRing] + k % chunk;
}

// One coordinate of k_epoch_queue (step k of this workgroup).  `cur` and its segment `ci/cv`,
// and `nxt`'s metadata were loaded one step earlier.  Loads `nxt`'s segment into `ni/nv` and
// the metadata of the coordinate two steps ahead into `nn`; returns that coordinate's position
// (>= n when the queue is exhausted; `nn` then describes a valid stand-in coordinate).
template <int FORM, int R, bool FRESH, typename U>
__device__ __forceinline__ uint32_t queue_step(const EpochArgs& a, const SharedBuf<U>& ub,
                                               const __amdgpu_buffer_rsrc_t& qr, int lane, uint32_t k,
                                               const CoordMeta& cur, const int (&ci)[R], const float (&cv)[R],
                                               const CoordMeta& nxt, int (&ni)[R], float (&nv)[R], CoordMeta& nn,
                                               uint32_t* ring, uint32_t& claim, float (*part)[4], int& buf) {
    constexpr int G = 256;
    const uint32_t K = a.chunk;
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this workgroup's atomics and its last claim have landed
    // The previous step claimed chunk (k - 1 + kQueueLead) / K if it began one.
    if (lane == 0 && k > 0 && (k - 1 + kQueueLead) % K == 0) ring[((k - 1 + kQueueLead) / K) % kQueueRing] = claim;
    const uint32_t n = a.perm.n;
    const uint32_t p2 = queue_pos(ring, k + 2, K);  // its chunk was published before the previous barrier
    const uint32_t m2 = p2 < n ? perm_at(p2, a.perm) : cur.m;
    const int qoff = lane == 0 && (k + kQueueLead) % K == 0 ? 0 : 4;
    const int64_t len = cur.s1 - cur.s0;
    if (len > (int64_t)G * R) {
        // Longer than the register slices: stream the segment twice (gather, then scatter).
        const float g = pipe_reduce<G>(long_dot<G, FRESH>(a, ub, lane, cur.s0, cur.s1), part, buf);
        float coef;
        const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
        a.model[cur.m] = m_new;
        if (coef != 0.0f) long_scatter<G>(a, ub, lane, cur.s0, cur.s1, coef);
        load_seg_raw<G, R>(a, nxt, lane, ni, nv);
        nn = load_meta_of(a, m2);
        claim = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)K, qr, qoff, 0, 0);
    } else {
        float gv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) gv[r] = buf_load<FRESH>(ub, (uint32_t)ci[r], (int64_t)(lane + r * G) < len);
        __builtin_amdgcn_sched_barrier(0);
        load_seg_raw<G, R>(a, nxt, lane, ni, nv);
        nn = load_meta_of(a, m2);
        claim = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)K, qr, qoff, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        float acc = 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r) acc = fmaf(cv[r], gv[r], acc);
        const float g = pipe_reduce<G>(acc, part, buf);
        float coef;
        const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
        a.model[cur.m] = m_new;  // every lane stores the same value
        const bool moves = coef != 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r)
            buf_atomic_add(ub, (uint32_t)ci[r], moves && (int64_t)(lane + r * G) < len, coef * cv[r]);
    }
    return p2;
}

template <int FORM, int R, bool FRESH, typename U>
__global__ __launch_bounds__(256) void k_epoch_queue(EpochArgs a) {
    constexpr int G = 256;
    __shared__ float part[2][G / 64];
    __shared__ uint32_t ring[kQueueRing];
    const int lane = threadIdx.x;
    const uint32_t n = a.perm.n;
    const uint32_t K = a.chunk;
    // word 3 = 0x00020000: 32-bit data format, the gfx9-family raw-buffer setting.
    const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(a.queue, (short)0, 4, 0x00020000);
    // The chunks that cover steps [0, kQueueLead): the steps' own claims start with the next one.
    const uint32_t first = (kQueueLead + K - 1) / K;  // 1..kQueueLead
    uint32_t c[kQueueLead];
#pragma unroll
    for (int i = 0; i < kQueueLead; ++i)
        c[i] = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)K, qr, lane == 0 && (uint32_t)i < first ? 0 : 4,
                                                                         0, 0);
    if (lane == 0) {
        // Claims of one lane on one address are performed in order; sort anyway.
#pragma unroll
        for (int i = 1; i < kQueueLead; ++i)
#pragma unroll
            for (int t = kQueueLead - 1; t >= i; --t)
                if ((uint32_t)t < first && c[t] < c[t - 1]) {
                    const uint32_t x = c[t];
                    c[t] = c[t - 1];
                    c[t - 1] = x;
                }
#pragma unroll
        for (int i = 0; i < kQueueLead; ++i)
            if ((uint32_t)i < first) ring[i % kQueueRing] = c[i];
    }
    __syncthreads();
    uint32_t pA = queue_pos(ring, 0, K), pB = queue_pos(ring, 1, K);
    if (pA < n) {
        const SharedBuf<U> ub =
            shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x);
        int buf = 0;
        uint32_t claim = 0, k = 0;
        CoordMeta cA = load_meta_of(a, perm_at(pA, a.perm));
        int ciA[R], ciB[R];
        float cvA[R], cvB[R];
        load_seg_raw<G, R>(a, cA, lane, ciA, cvA);
        CoordMeta cB = load_meta_of(a, pB < n ? perm_at(pB, a.perm) : cA.m);
        for (;;) {
            CoordMeta cA2, cB2;
            const uint32_t pA2 = queue_step<FORM, R, FRESH>(a, ub, qr, lane, k++, cA, ciA, cvA, cB, ciB, cvB, cA2,
                                                            ring, claim, part, buf);
            if (pB >= n) break;
            const uint32_t pB2 = queue_step<FORM, R, FRESH>(a, ub, qr, lane, k++, cB, ciB, cvB, cA2, ciA, cvA, cB2,
                                                            ring, claim, part, buf);
            if (pA2 >= n) break;
            cA = cA2;
            cB = cB2;
            pB = pB2;
        }
    }
    if (lane == 0) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // every claim of this workgroup has been performed
        const uint32_t done = __hip_atomic_fetch_add(a.queue + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (done == gridDim.x - 1) {  // the others have finished claiming: reset for the next launch
            __hip_atomic_store(a.queue, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(a.queue + 1, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// ----------------------------------------------------------------------------------------
// Epoch kernel for skewed segment lengths: a 256-thread workgroup takes a batch of NG = 256/G
// consecutive permutation positions per round, one per group.  Segments up to `long_len`
// entries are processed by their group as in k_epoch_group; longer ones are handed to the
// whole workgroup (LDS combine), one after the other, so that a long segment's gather-to-
// scatter interval stays as short as a short segment's.  One barrier per batch (vote) plus
// one per long segment.
// ----------------------------------------------------------------------------------------
// `ng` (<= NG) groups of each workgroup take positions, so that gridDim.x * ng coordinates
// are in flight at most.
template <int FORM, int G, int R, bool FRESH, typename U>
__global__ __launch_bounds__(256) void k_epoch_mixed(EpochArgs a, uint32_t long_len, uint32_t ng) {
    U* const uu = static_cast<U*>(a.u);
    constexpr int NG = 256 / G, NW = 4;
    __shared__ uint32_t longs[2][NG];
    __shared__ float part[2][NW];
    const int tid = threadIdx.x, lane = tid & (G - 1), grp = tid / G, wave = tid >> 6;
    const uint32_t n_batches = (a.perm.n + ng - 1) / ng;
    int lb = 0, pb = 0;
    for (uint32_t b = blockIdx.x; b < n_batches; b += gridDim.x) {
        const uint32_t j = b * ng + grp;
        uint32_t my_long = 0xFFFFFFFFu;
        if ((uint32_t)grp < ng && j < a.perm.n) {
            const uint32_t m = perm_at(j, a.perm);
            const int64_t s0 = a.ptr[m], s1 = a.ptr[m + 1];
            if (s1 - s0 > (int64_t)long_len) {
                my_long = m;
            } else {
                const float m_old = a.model[m];
                const float sn = a.norms[m];
                const float ylab = a.y[m];
                int ci[R];
                float cv[R];
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const int64_t k = s0 + lane + (int64_t)r * G;
                    if (k < s1) { ci[r] = a.idx[k]; cv[r] = a.val[k]; }
                    else { ci[r] = -1; cv[r] = 0.0f; }
                }
                float acc = 0.0f;
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (ci[r] >= 0) acc = fmaf(cv[r], ld_u<FRESH>(uu + ci[r]), acc);
                for (int64_t k = s0 + lane + (int64_t)R * G; k < s1; k += G)
                    acc = fmaf(a.val[k], ld_u<FRESH>(uu + a.idx[k]), acc);
                const float g = group_sum<G>(acc);
                float coef;
                const float m_new = coord_step<FORM>(g, sn, m_old, ylab, a.k, &coef);
                if (lane == 0) a.model[m] = m_new;
                if (coef != 0.0f) {
#pragma unroll
                    for (int r = 0; r < R; ++r)
                        if (ci[r] >= 0) atomic_add_u(uu + ci[r], coef * cv[r]);
                    for (int64_t k = s0 + lane + (int64_t)R * G; k < s1; k += G)
                        atomic_add_u(uu + a.idx[k], coef * a.val[k]);
                }
            }
        }
        if (lane == 0) longs[lb][grp] = my_long;
        const int any_long = __syncthreads_or(my_long != 0xFFFFFFFFu);
        if (any_long) {
            for (int q = 0; q < NG; ++q) {
                const uint32_t m = longs[lb][q];
                if (m == 0xFFFFFFFFu) continue;
                const int64_t s0 = a.ptr[m], s1 = a.ptr[m + 1];
                const float m_old = a.model[m];
                const float sn = a.norms[m];
                const float ylab = a.y[m];
                float acc = 0.0f;
                for (int64_t k = s0 + tid; k < s1; k += 256) acc = fmaf(a.val[k], ld_u<FRESH>(uu + a.idx[k]), acc);
                acc = group_sum<64>(acc);
                if ((tid & 63) == 0) part[pb][wave] = acc;
                __syncthreads();
                const float g = part[pb][0] + part[pb][1] + part[pb][2] + part[pb][3];
                float coef;
                const float m_new = coord_step<FORM>(g, sn, m_old, ylab, a.k, &coef);
                if (tid == 0) a.model[m] = m_new;
                if (coef != 0.0f)
                    for (int64_t k = s0 + tid; k < s1; k += 256) atomic_add_u(uu + a.idx[k], coef * a.val[k]);
                pb ^= 1;
            }
        }
        lb ^= 1;
    }
}

// ----------------------------------------------------------------------------------------
// Epoch kernel, one workgroup of BS threads per coordinate (long segments): wave sums by
// DPP, then the BS/64 wave sums through a double-buffered LDS array (one barrier per
// coordinate).  ORDERED adds a device-scope fence and a barrier after the scatter so that
// with a single workgroup the next coordinate sees every update (sequential Alg. 1).
// ----------------------------------------------------------------------------------------
template <int FORM, int BS, int R, bool FRESH, bool ORDERED, typename U>
__global__ __launch_bounds__(BS) void k_epoch_block(EpochArgs a) {
    U* const uu = static_cast<U*>(a.u);
    constexpr int NW = BS / 64;
    __shared__ float part[2][NW];
    const int tid = threadIdx.x, wave = tid >> 6;
    int buf = 0;
    if (blockIdx.x >= a.n_groups) return;
    for (uint32_t j = blockIdx.x; j < a.perm.n; j += a.n_groups) {
        const uint32_t m = perm_at(j, a.perm);
        const int64_t s0 = a.ptr[m], s1 = a.ptr[m + 1];
        const float m_old = a.model[m];
        const float sn = a.norms[m];
        const float ylab = a.y[m];
        int ci[R];
        float cv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int64_t k = s0 + tid + (int64_t)r * BS;
            if (k < s1) { ci[r] = a.idx[k]; cv[r] = a.val[k]; }
            else { ci[r] = -1; cv[r] = 0.0f; }
        }
        float acc = 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (ci[r] >= 0) acc = fmaf(cv[r], ld_u<FRESH>(uu + ci[r]), acc);
        for (int64_t k = s0 + tid + (int64_t)R * BS; k < s1; k += BS)
            acc = fmaf(a.val[k], ld_u<FRESH>(uu + a.idx[k]), acc);
        acc = group_sum<64>(acc);
        if ((tid & 63) == 0) part[buf][wave] = acc;
        __syncthreads();
        float g = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) g += part[buf][w];
        float coef;
        const float m_new = coord_step<FORM>(g, sn, m_old, ylab, a.k, &coef);
        if (tid == 0) a.model[m] = m_new;
        if (coef != 0.0f) {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (ci[r] >= 0) atomic_add_u(uu + ci[r], coef * cv[r]);
            for (int64_t k = s0 + tid + (int64_t)R * BS; k < s1; k += BS)
                atomic_add_u(uu + a.idx[k], coef * a.val[k]);
        }
        if constexpr (ORDERED) {
            __threadfence();
            __syncthreads();
        }
        buf ^= 1;
    }
}

// ----------------------------------------------------------------------------------------
// Ordered epoch (window 1) with the whole shared vector resident in LDS: one workgroup of
// 1024 threads walks the permutation in order; gathers and scatters hit LDS only
// (ds_add_f32), two barriers per coordinate.  The shared vector is loaded at the start and
// written back at the end of the epoch.
// ----------------------------------------------------------------------------------------
template <int FORM, typename U>
__global__ __launch_bounds__(1024) void k_epoch_ordered_lds(EpochArgs a, uint32_t L) {
    constexpr int BS = 1024, NW = BS / 64;
    extern __shared__ __align__(16) unsigned char lds_bytes[];
    U* const uu = static_cast<U*>(a.u);
    U* su = reinterpret_cast<U*>(lds_bytes);                           // L entries
    float* part = reinterpret_cast<float*>(su + ((L + 63) & ~63u));    // 2 * NW floats
    const int tid = threadIdx.x, wave = tid >> 6;
    for (uint32_t i = tid; i < L; i += BS) su[i] = uu[i];
    __syncthreads();
    int buf = 0;
    for (uint32_t j = 0; j < a.perm.n; ++j) {
        const uint32_t m = perm_at(j, a.perm);
        const int64_t s0 = a.ptr[m], s1 = a.ptr[m + 1];
        const float m_old = a.model[m];
        const float sn = a.norms[m];
        const float ylab = a.y[m];
        float acc = 0.0f;
        for (int64_t k = s0 + tid; k < s1; k += BS) acc = fmaf(a.val[k], (float)su[a.idx[k]], acc);
        acc = group_sum<64>(acc);
        if ((tid & 63) == 0) part[buf * NW + wave] = acc;
        __syncthreads();
        float g = 0.0f;
#pragma unroll
        for (int w = 0; w < NW; ++w) g += part[buf * NW + w];
        float coef;
        const float m_new = coord_step<FORM>(g, sn, m_old, ylab, a.k, &coef);
        if (tid == 0) a.model[m] = m_new;
        if (coef != 0.0f)
            for (int64_t k = s0 + tid; k < s1; k += BS) atomicAdd(su + a.idx[k], (U)(coef * a.val[k]));
        __syncthreads();
        buf ^= 1;
    }
    for (uint32_t i = tid; i < L; i += BS) uu[i] = su[i];
}

// ----------------------------------------------------------------------------------------
// Frozen gather-dot: out[c] = <a_c, u> with the epoch kernel's arithmetic (fp32 FMA per
// lane, group butterfly), for every coordinate in index order.
// ----------------------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(256) void k_gather_dots(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                                                     const float* __restrict__ val, const float* __restrict__ u,
                                                     uint32_t C, float* __restrict__ out) {
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < C; c += ngroups) {
        const int64_t s0 = ptr[c], s1 = ptr[c + 1];
        float acc = 0.0f;
        for (int64_t k = s0 + lane; k < s1; k += G) acc = fmaf(val[k], u[idx[k]], acc);
        acc = group_sum<G>(acc);
        if (lane == 0) out[c] = acc;
    }
}

// ----------------------------------------------------------------------------------------
// Set-up: squared segment norms and, when y is given (ridge primal), cy_c = <y, a_c>
// (fp64 accumulation, fp32 results); input validation.
// ----------------------------------------------------------------------------------------
template <int G>
__global__ __launch_bounds__(256) void k_norms(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                                               const float* __restrict__ val, const float* __restrict__ y,
                                               uint32_t C, float* __restrict__ out, float* __restrict__ cy,
                                               double* __restrict__ cyd) {
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < C; c += ngroups) {
        double acc = 0.0, dy = 0.0;
        for (int64_t k = ptr[c] + lane; k < ptr[c + 1]; k += G) {
            acc += (double)val[k] * (double)val[k];
            if (y) dy += (double)val[k] * (double)y[idx[k]];
        }
        acc = group_sum_f64<G>(acc);
        if (y) dy = group_sum_f64<G>(dy);
        if (lane == 0) {
            out[c] = (float)acc;
            if (y) {
                cy[c] = (float)dy;
                cyd[c] = dy;
            }
        }
    }
}

// flags bits: 1 ptr not monotone / wrong ends, 2 index out of range, 4 non-finite value,
// 8 non-finite label, 16 label not +-1.
// flags[1] (as unsigned long long) receives the longest segment.
__global__ void k_validate_ptr(const int64_t* __restrict__ ptr, uint32_t S, int64_t nnz, int* flags) {
    uint32_t c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c == 0 && (ptr[0] != 0 || ptr[S] != nnz)) atomicOr(flags, 1);
    if (c < S) {
        const int64_t len = ptr[c + 1] - ptr[c];
        if (len < 0) atomicOr(flags, 1);
        else atomicMax(reinterpret_cast<unsigned long long*>(flags) + 1, (unsigned long long)len);
    }
}

__global__ void k_validate_entries(const int32_t* __restrict__ idx, const float* __restrict__ val, int64_t nnz,
                                   int64_t bound, int* flags) {
    int f = 0;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < nnz; k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t i = idx[k];
        if (i < 0 || (int64_t)i >= bound) f |= 2;
        if (!isfinite(val[k])) f |= 4;
    }
    if (f) atomicOr(flags, f);
}

__global__ void k_validate_labels(const float* __restrict__ y, int64_t n, int pm1, int* flags) {
    int f = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const float v = y[i];
        if (!isfinite(v)) f |= 8;
        else if (pm1 && v != 1.0f && v != -1.0f) f |= 16;
    }
    if (f) atomicOr(flags, f);
}

// ----------------------------------------------------------------------------------------
// Objective / duality-gap reductions (fp64).  Every workgroup sums, over the coordinates it owns,
// the fp64 dot d_c and up to three terms, and over its slice of the shared vector two more, and
// stores its five partial sums; one workgroup then adds the partials in workgroup order
// (deterministic; no cross-workgroup fences inside the pass).
//   ridge primal (u = w, r = y - w, d = <a_c, r> = <a_c, y> - <a_c, w>):
//                                  S0 += d^2,  S1 += beta^2          | V0 += r^2, V1 += r*y
//   svm dual     (u = w):          S0 += max(0, 1 - y d), S1 += alpha | V0 += w^2
//   ridge dual   (u = wbar):       S0 += (d/lambda - y)^2, S1 += alpha^2, S2 += alpha*y | V0 += wbar^2
// ----------------------------------------------------------------------------------------
template <int NS>
__device__ __forceinline__ void block_reduce_store(double (&v)[NS], double* out) {
    __shared__ double red[NS][256 / 64];
    const int tid = threadIdx.x;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        double x = v[s];
        x = group_sum_f64<64>(x);
        if ((tid & 63) == 0) red[s][tid >> 6] = x;
    }
    __syncthreads();
    if (tid == 0) {
#pragma unroll
        for (int s = 0; s < NS; ++s) out[s] = red[s][0] + red[s][1] + red[s][2] + red[s][3];
    }
}

template <int FORM, int G, typename U>
__global__ __launch_bounds__(256) void k_objective(ObjArgs o, double* __restrict__ partials) {
    constexpr int NS = 5;
    const U* __restrict__ u = static_cast<const U*>(o.u);
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    double t[NS] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < o.C; c += ngroups) {
        double d = 0.0;
        for (int64_t k = o.ptr[c] + lane; k < o.ptr[c + 1]; k += G) d += (double)o.val[k] * (double)u[o.idx[k]];
        d = group_sum_f64<G>(d);
        if (lane == 0) {
            const double mo = o.model[c];
            if constexpr (FORM == FORM_RIDGE_PRIMAL) {
                const double r = o.cyd[c] - d;
                t[0] += r * r;
                t[1] += mo * mo;
            } else if constexpr (FORM == FORM_SVM_DUAL) {
                const double l = 1.0 - (double)o.y[c] * d;
                t[0] += l > 0.0 ? l : 0.0;
                t[1] += mo;
            } else {
                const double e = d / o.lam - (double)o.y[c];
                t[0] += e * e;
                t[1] += mo * mo;
                t[2] += mo * (double)o.y[c];
            }
        }
    }
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < o.L; i += (int64_t)gridDim.x * 256) {
        if constexpr (FORM == FORM_RIDGE_PRIMAL) {
            const double r = (double)o.yv[i] - (double)u[i];
            t[3] += r * r;
            t[4] += r * (double)o.yv[i];
        } else {
            const double x = (double)u[i];
            t[3] += x * x;
        }
    }
    block_reduce_store<NS>(t, partials + (size_t)blockIdx.x * NS);
}

// ----------------------------------------------------------------------------------------
// Coupling probe (set-up only).  With a~_c = sigma_c a_c / sqrt(|a_c|^2 + mu) (sigma_c = the
// label for the SVM, 1 otherwise; mu = lambda N for the ridge steps, 0 for the SVM step),
// G = A~^T A~ holds the step-normalised couplings between coordinates.  A probe with
// Rademacher signs z_c scatters T = A~ z; the gather pass forms (A~^T T)_c - G_cc z_c, the
// off-diagonal part of (G z)_c, whose square has expectation kappa_c = sum_{j != c} G_cj^2
// (Hutchinson), accumulated per coordinate in K.  z = 1 (probe 0) gives the coherent sum
// |A~ 1|^2 instead (vector pass).
// ----------------------------------------------------------------------------------------
__device__ __forceinline__ float probe_sign(uint32_t c, uint32_t probe) {
    if (probe == 0) return 1.0f;
    return (murmur_fmix32(c ^ (probe * 0x9E3779B9u)) & 1u) ? 1.0f : -1.0f;
}

template <int G>
__global__ __launch_bounds__(256) void k_probe_scatter(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                                                       const float* __restrict__ val, const float* __restrict__ norms,
                                                       const float* __restrict__ sign, uint32_t C, float mu,
                                                       uint32_t probe, float* __restrict__ T) {
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < C; c += ngroups) {
        const float sc = norms[c];
        if (!(sc > 0.0f)) continue;
        const float coef = probe_sign(c, probe) * (sign ? sign[c] : 1.0f) * rsqrtf(sc + mu);
        for (int64_t k = ptr[c] + lane; k < ptr[c + 1]; k += G) atomic_add_u(T + idx[k], coef * val[k]);
    }
}

template <int G>
__global__ __launch_bounds__(256) void k_probe_gather(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                                                      const float* __restrict__ val, const float* __restrict__ norms,
                                                      const float* __restrict__ sign, const float* __restrict__ T,
                                                      uint32_t C, float mu, uint32_t probe, float* __restrict__ K,
                                                      double* __restrict__ partials) {
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    double t[4] = {0.0, 0.0, 0.0, 0.0};  // |G z|^2, sum G_cc^2, sum G_cc, non-empty coordinates
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < C; c += ngroups) {
        const float sc = norms[c];
        if (!(sc > 0.0f)) continue;
        double d = 0.0;
        for (int64_t k = ptr[c] + lane; k < ptr[c + 1]; k += G) d += (double)val[k] * (double)T[idx[k]];
        d = group_sum_f64<G>(d);
        if (lane == 0) {
            const double scale = (sign ? (double)sign[c] : 1.0) / sqrt((double)sc + (double)mu);
            const double diag = (double)sc / ((double)sc + (double)mu);
            // Off-diagonal part of (G z)_c: its square has expectation sum_{j != c} G_cj^2.
            const double g = d * scale - diag * (double)probe_sign(c, probe);
            t[0] += g * g;
            t[1] += diag * diag;
            t[2] += diag;
            t[3] += 1.0;
            if (K) K[c] += (float)(g * g);  // summed over probes
        }
    }
    block_reduce_store<4>(t, partials + (size_t)blockIdx.x * 4);
}

// Largest per-coordinate off-diagonal row mass kappa_c = sum_{j != c} G_cj^2, from the probe
// sums K[c] over `probes` Rademacher probes.  Non-negative floats order like their bit patterns.
__global__ __launch_bounds__(256) void k_kappa_max(const float* __restrict__ K, const float* __restrict__ norms,
                                                   uint32_t C, float inv_probes, unsigned* __restrict__ out) {
    float best = 0.0f;
    for (uint32_t c = blockIdx.x * 256u + threadIdx.x; c < C; c += gridDim.x * 256u) {
        const float sc = norms[c];
        if (!(sc > 0.0f)) continue;
        best = fmaxf(best, K[c] * inv_probes);
    }
    for (int o = 32; o > 0; o >>= 1) best = fmaxf(best, __shfl_xor(best, o, 64));
    if ((threadIdx.x & 63) == 0 && best > 0.0f) atomicMax(out, __float_as_uint(best));
}

__global__ __launch_bounds__(256) void k_sumsq(const float* __restrict__ T, int64_t L, double* __restrict__ partials) {
    double t[1] = {0.0};
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < L; i += (int64_t)gridDim.x * 256) {
        const double x = T[i];
        t[0] += x * x;
    }
    block_reduce_store<1>(t, partials + blockIdx.x);
}

// Sum `nparts` rows of `width` doubles in index order (one workgroup; deterministic).
// Sums `width` (at most kSumWidthMax) columns of `partials` [nparts][width] in one workgroup, in an
// order fixed by nparts alone (so the result does not depend on timing): thread t adds rows t,
// t + 256, ... in turn, each wave combines its lanes by an xor butterfly, and thread 0 adds the
// four wave sums in wave order.
constexpr int kSumWidthMax = 8;

__global__ __launch_bounds__(256) void k_sum_partials(const double* __restrict__ partials, int nparts, int width,
                                                      double* __restrict__ out) {
    __shared__ double sh[4][kSumWidthMax];
    double x[kSumWidthMax];
#pragma unroll
    for (int w = 0; w < kSumWidthMax; ++w) x[w] = 0.0;
    for (int p = threadIdx.x; p < nparts; p += 256) {
#pragma unroll
        for (int w = 0; w < kSumWidthMax; ++w)
            if (w < width) x[w] += partials[(size_t)p * width + w];
    }
#pragma unroll
    for (int w = 0; w < kSumWidthMax; ++w)
        for (int o = 32; o > 0; o >>= 1) x[w] += __shfl_xor(x[w], o, 64);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
        for (int w = 0; w < kSumWidthMax; ++w) sh[wave][w] = x[w];
    }
    __syncthreads();
    if (threadIdx.x == 0)
        for (int w = 0; w < width; ++w) out[w] = ((sh[0][w] + sh[1][w]) + sh[2][w]) + sh[3][w];
}

// ----------------------------------------------------------------------------------------
// Host-side launchers.
// ----------------------------------------------------------------------------------------
template <int FORM, int G, bool FRESH, typename U>
static hipError_t launch_group(const EpochArgs& a, int blocks, bool tail, hipStream_t s) {
    constexpr int R = slice_depth(G);
    if (tail)
        hipLaunchKernelGGL((k_epoch_group<FORM, G, R, FRESH, true, U>), dim3(blocks), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((k_epoch_group<FORM, G, R, FRESH, false, U>), dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int FORM, int G, bool FRESH, typename U>
static hipError_t launch_pipe(const EpochArgs& a, int blocks, hipStream_t s) {
    constexpr int R = G == 256 ? 16 : slice_depth(G);
    hipLaunchKernelGGL((k_epoch_pipe<FORM, G, R, FRESH, U>), dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int FORM, bool FRESH, typename U>
static hipError_t launch_queue(const EpochArgs& a, int blocks, hipStream_t s) {
    hipLaunchKernelGGL((k_epoch_queue<FORM, kQueueSlices, FRESH, U>), dim3(blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

template <int FORM, int G, bool FRESH, typename U>
static hipError_t launch_mixed(const EpochArgs& a, int blocks, uint32_t long_len, hipStream_t s) {
    constexpr int R = slice_depth(G);
    const uint32_t ng = (a.n_groups + blocks - 1) / blocks;  // <= 256 / G by construction of the plan
    hipLaunchKernelGGL((k_epoch_mixed<FORM, G, R, FRESH, U>), dim3(blocks), dim3(256), 0, s, a, long_len, ng);
    return hipGetLastError();
}

template <int FORM, bool FRESH, typename U>
static hipError_t launch_pipe_by_width(const EpochArgs& a, const LaunchPlan& lp, hipStream_t s) {
    switch (lp.group) {
        case 4: return launch_pipe<FORM, 4, FRESH, U>(a, lp.blocks, s);
        case 8: return launch_pipe<FORM, 8, FRESH, U>(a, lp.blocks, s);
        case 16: return launch_pipe<FORM, 16, FRESH, U>(a, lp.blocks, s);
        case 32: return launch_pipe<FORM, 32, FRESH, U>(a, lp.blocks, s);
        case 64: return launch_pipe<FORM, 64, FRESH, U>(a, lp.blocks, s);
        case 256: return launch_pipe<FORM, 256, FRESH, U>(a, lp.blocks, s);
        default: return hipErrorInvalidValue;
    }
}

template <int FORM, bool FRESH, typename U>
static hipError_t launch_by_width(const EpochArgs& a, const LaunchPlan& lp, hipStream_t s) {
    const bool mixed = lp.kind == PLAN_MIXED;
    switch (lp.group) {
#define SCD_CASE(GW)                                                                           \
    case GW:                                                                                   \
        return mixed ? launch_mixed<FORM, GW, FRESH, U>(a, lp.blocks, lp.long_len, s)          \
                     : launch_group<FORM, GW, FRESH, U>(a, lp.blocks, lp.tail, s);
        SCD_CASE(4)
        SCD_CASE(8)
        SCD_CASE(16)
        SCD_CASE(32)
        SCD_CASE(64)
#undef SCD_CASE
        default: return hipErrorInvalidValue;
    }
}

template <int FORM, typename U>
static hipError_t launch_epoch_typed(const EpochArgs& a, const LaunchPlan& lp, hipStream_t s) {
    if (lp.kind == PLAN_ORDERED_LDS) {
        hipLaunchKernelGGL((k_epoch_ordered_lds<FORM, U>), dim3(1), dim3(1024), lp.lds_bytes, s, a, lp.L);
        return hipGetLastError();
    }
    if (lp.kind == PLAN_PIPE)
        return lp.fresh ? launch_pipe_by_width<FORM, true, U>(a, lp, s) : launch_pipe_by_width<FORM, false, U>(a, lp, s);
    if (lp.kind == PLAN_QUEUE)
        return lp.fresh ? launch_queue<FORM, true, U>(a, lp.blocks, s) : launch_queue<FORM, false, U>(a, lp.blocks, s);
    if (lp.kind == PLAN_BLOCK) {
        if (lp.ordered)
            hipLaunchKernelGGL((k_epoch_block<FORM, 256, 16, true, true, U>), dim3(lp.blocks), dim3(256), 0, s, a);
        else if (lp.fresh)
            hipLaunchKernelGGL((k_epoch_block<FORM, 256, 16, true, false, U>), dim3(lp.blocks), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((k_epoch_block<FORM, 256, 16, false, false, U>), dim3(lp.blocks), dim3(256), 0, s, a);
        return hipGetLastError();
    }
    return lp.fresh ? launch_by_width<FORM, true, U>(a, lp, s) : launch_by_width<FORM, false, U>(a, lp, s);
}

template <int FORM>
static hipError_t launch_epoch_form(const EpochArgs& a, const LaunchPlan& lp, hipStream_t s) {
    return lp.wide ? launch_epoch_typed<FORM, double>(a, lp, s) : launch_epoch_typed<FORM, float>(a, lp, s);
}

hipError_t launch_epoch(int form, const EpochArgs& a, const LaunchPlan& lp, hipStream_t s) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: return launch_epoch_form<FORM_RIDGE_PRIMAL>(a, lp, s);
        case FORM_SVM_DUAL: return launch_epoch_form<FORM_SVM_DUAL>(a, lp, s);
        case FORM_RIDGE_DUAL: return launch_epoch_form<FORM_RIDGE_DUAL>(a, lp, s);
        default: return hipErrorInvalidValue;
    }
}

template <int FORM>
static hipError_t prepare_form(bool wide, size_t lds_bytes) {
    const void* f = wide ? reinterpret_cast<const void*>(&k_epoch_ordered_lds<FORM, double>)
                         : reinterpret_cast<const void*>(&k_epoch_ordered_lds<FORM, float>);
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t ordered_lds_prepare(int form, bool wide, size_t lds_bytes) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: return prepare_form<FORM_RIDGE_PRIMAL>(wide, lds_bytes);
        case FORM_SVM_DUAL: return prepare_form<FORM_SVM_DUAL>(wide, lds_bytes);
        case FORM_RIDGE_DUAL: return prepare_form<FORM_RIDGE_DUAL>(wide, lds_bytes);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_perm_fill(const PermKeys& p, int32_t* out, hipStream_t s) {
    const uint32_t blocks = (p.n + 255) / 256;
    hipLaunchKernelGGL(k_perm_fill, dim3(blocks), dim3(256), 0, s, p, out);
    return hipGetLastError();
}

hipError_t launch_gather_dots(const int64_t* ptr, const int32_t* idx, const float* val, const float* u, uint32_t C,
                              int G, int blocks, float* out, hipStream_t s) {
    switch (G) {
        case 4: hipLaunchKernelGGL(k_gather_dots<4>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, u, C, out); break;
        case 8: hipLaunchKernelGGL(k_gather_dots<8>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, u, C, out); break;
        case 16: hipLaunchKernelGGL(k_gather_dots<16>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, u, C, out); break;
        case 32: hipLaunchKernelGGL(k_gather_dots<32>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, u, C, out); break;
        default: hipLaunchKernelGGL(k_gather_dots<64>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, u, C, out); break;
    }
    return hipGetLastError();
}

hipError_t launch_norms(const int64_t* ptr, const int32_t* idx, const float* val, const float* y, uint32_t C, int G,
                        int blocks, float* out, float* cy, double* cyd, hipStream_t s) {
    switch (G) {
        case 4: hipLaunchKernelGGL(k_norms<4>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, y, C, out, cy, cyd); break;
        case 8: hipLaunchKernelGGL(k_norms<8>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, y, C, out, cy, cyd); break;
        case 16: hipLaunchKernelGGL(k_norms<16>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, y, C, out, cy, cyd); break;
        case 32: hipLaunchKernelGGL(k_norms<32>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, y, C, out, cy, cyd); break;
        default: hipLaunchKernelGGL(k_norms<64>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, y, C, out, cy, cyd); break;
    }
    return hipGetLastError();
}

hipError_t launch_validate(const int64_t* ptr, uint32_t S, const int32_t* idx, const float* val, int64_t nnz,
                           int64_t bound, const float* y, int64_t ny, int pm1, int* flags, hipStream_t s) {
    hipLaunchKernelGGL(k_validate_ptr, dim3((S + 256) / 256), dim3(256), 0, s, ptr, S, nnz, flags);
    if (nnz > 0) {
        int64_t b = (nnz + 255) / 256;
        if (b > 8192) b = 8192;
        hipLaunchKernelGGL(k_validate_entries, dim3((unsigned)b), dim3(256), 0, s, idx, val, nnz, bound, flags);
    }
    int64_t b = (ny + 255) / 256;
    if (b > 4096) b = 4096;
    if (b < 1) b = 1;
    hipLaunchKernelGGL(k_validate_labels, dim3((unsigned)b), dim3(256), 0, s, y, ny, pm1, flags);
    return hipGetLastError();
}

template <int FORM, typename U>
static void objective_typed(const ObjArgs& o, int G, int blocks, double* partials, hipStream_t s) {
    switch (G) {
#define SCD_OBJ(GW)                                                                                         \
    case GW:                                                                                                \
        hipLaunchKernelGGL((k_objective<FORM, GW, U>), dim3(blocks), dim3(256), 0, s, o, partials);         \
        break;
        SCD_OBJ(4)
        SCD_OBJ(8)
        SCD_OBJ(16)
        SCD_OBJ(32)
        default: SCD_OBJ(64)
#undef SCD_OBJ
    }
}

template <int FORM>
static void objective_form(const ObjArgs& o, int G, int blocks, double* partials, hipStream_t s) {
    if (o.wide)
        objective_typed<FORM, double>(o, G, blocks, partials, s);
    else
        objective_typed<FORM, float>(o, G, blocks, partials, s);
}

// sums[0..2] = coordinate sums, sums[3..4] = vector sums.
hipError_t launch_objective(int form, const ObjArgs& o, int G, int blocks, double* partials, double* sums,
                            hipStream_t s) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: objective_form<FORM_RIDGE_PRIMAL>(o, G, blocks, partials, s); break;
        case FORM_SVM_DUAL: objective_form<FORM_SVM_DUAL>(o, G, blocks, partials, s); break;
        case FORM_RIDGE_DUAL: objective_form<FORM_RIDGE_DUAL>(o, G, blocks, partials, s); break;
        default: return hipErrorInvalidValue;
    }
    hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(256), 0, s, partials, blocks, 5, sums);
    return hipGetLastError();
}

// out[0] = |G z|^2 (probe > 0) or |A~ 1|^2 (probe 0), out[1] = sum G_cc^2, out[2] = sum G_cc,
// out[3] = non-empty coordinates.
hipError_t launch_probe(const int64_t* ptr, const int32_t* idx, const float* val, const float* norms,
                        const float* sign, uint32_t C, int64_t L, float mu, uint32_t probe, int G, int blocks,
                        float* T, float* K, double* partials, double* out, hipStream_t s) {
    hipError_t e = hipMemsetAsync(T, 0, sizeof(float) * (size_t)L, s);
    if (e != hipSuccess) return e;
#define SCD_PROBE(GW)                                                                                          \
    hipLaunchKernelGGL(k_probe_scatter<GW>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, norms, sign, C, mu, \
                       probe, T);                                                                              \
    hipLaunchKernelGGL(k_probe_gather<GW>, dim3(blocks), dim3(256), 0, s, ptr, idx, val, norms, sign, T, C,   \
                       mu, probe, probe ? K : nullptr, partials)
    switch (G) {
        case 4: SCD_PROBE(4); break;
        case 8: SCD_PROBE(8); break;
        case 16: SCD_PROBE(16); break;
        case 32: SCD_PROBE(32); break;
        default: SCD_PROBE(64); break;
    }
#undef SCD_PROBE
    hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(256), 0, s, partials, blocks, 4, out);
    if (probe == 0) {
        hipLaunchKernelGGL(k_sumsq, dim3(blocks), dim3(256), 0, s, T, L, partials);
        hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(256), 0, s, partials, blocks, 1, out);
    }
    return hipGetLastError();
}

hipError_t launch_kappa_max(const float* K, const float* norms, uint32_t C, int probes, int blocks, unsigned* out,
                            hipStream_t s) {
    hipLaunchKernelGGL(k_kappa_max, dim3(blocks), dim3(256), 0, s, K, norms, C, 1.0f / (float)probes, out);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------------------
// Storage-width conversions of the shared vector and the per-entry update count.
// ----------------------------------------------------------------------------------------
template <typename A, typename B>
__global__ __launch_bounds__(256) void k_convert(const A* __restrict__ in, int64_t n, B* __restrict__ out) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) out[i] = (B)in[i];
}

// hits[i] = number of stored entries with index i (one atomic per entry); max into out[0].
__global__ __launch_bounds__(256) void k_count_hits(const int32_t* __restrict__ idx, int64_t nnz,
                                                    unsigned* __restrict__ hits) {
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < nnz; k += (int64_t)gridDim.x * 256)
        atomicAdd(hits + idx[k], 1u);
}

__global__ __launch_bounds__(256) void k_max_u32(const unsigned* __restrict__ v, int64_t n, unsigned* __restrict__ out) {
    unsigned best = 0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) best = max(best, v[i]);
    for (int o = 32; o > 0; o >>= 1) best = max(best, (unsigned)__shfl_xor((int)best, o, 64));
    if ((threadIdx.x & 63) == 0 && best) atomicMax(out, best);
}

static unsigned grid_for(int64_t n) {
    int64_t b = (n + 255) / 256;
    if (b > 8192) b = 8192;
    if (b < 1) b = 1;
    return (unsigned)b;
}

hipError_t launch_convert_f32_to_f64(const float* in, int64_t n, double* out, hipStream_t s) {
    hipLaunchKernelGGL((k_convert<float, double>), dim3(grid_for(n)), dim3(256), 0, s, in, n, out);
    return hipGetLastError();
}

hipError_t launch_convert_f64_to_f32(const double* in, int64_t n, float* out, hipStream_t s) {
    hipLaunchKernelGGL((k_convert<double, float>), dim3(grid_for(n)), dim3(256), 0, s, in, n, out);
    return hipGetLastError();
}

hipError_t launch_max_hits(const int32_t* idx, int64_t nnz, int64_t L, unsigned* hits, unsigned* out, hipStream_t s) {
    if (nnz > 0) hipLaunchKernelGGL(k_count_hits, dim3(grid_for(nnz)), dim3(256), 0, s, idx, nnz, hits);
    hipLaunchKernelGGL(k_max_u32, dim3(grid_for(L)), dim3(256), 0, s, hits, L, out);
    return hipGetLastError();
}


// ----------------------------------------------------------------------------------------
// Hot-set epoch: one workgroup for a window of at most kHotMaxWindow coordinates in flight.
//
// With so few coordinates in flight an epoch is bound by latency: each coordinate waits one
// round trip for its gathers, and on skewed data most gathers hit the few entries that every
// coordinate updates, whose lines the atomics keep invalidating.  Here the n_hot most-updated
// entries of the shared vector live in LDS for the whole epoch (loaded at the start, written
// back at the end), so their gathers and atomic adds stay inside the CU and are seen at once
// by the other in-flight coordinates, which all run in the same workgroup.
//
// Wave 0 (the consumer) runs the W in-flight coordinates, 8 lanes each, and reads nothing but
// LDS.  Waves 1..kHotProducers fill per-producer LDS buffers with the next batches of B
// permutation positions: each coordinate's metadata and, per stored entry, its value and
// either its hot slot or (cold entry) its index and current shared-vector value.  Each wave
// has its own completion counter, so the producers' load latency never stalls the consumer.
// Cold values are therefore read up to a few batches before their coordinate runs; cold
// entries are by construction rarely updated, so such a read seldom misses an update.
// Producer and consumer hand buffers over through LDS sequence numbers; every wait is bounded
// (spin_limit sleeps), after which the wave sets *err and all waves leave.
// ----------------------------------------------------------------------------------------
size_t hot_lds_bytes(uint32_t hot_bytes, uint32_t B, uint32_t Smax) {
    return (size_t)hot_bytes + 64 + (size_t)kHotProducers * (5u * B + 3u * B * Smax) * sizeof(uint32_t);
}

__device__ __forceinline__ bool hot_wait(uint32_t* flag, uint32_t want, uint32_t* abort_flag, uint32_t limit,
                                         int* err) {
    uint32_t spins = 0;
    for (;;) {
        if (__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) == want) return true;
        if (__hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) return false;
        if (++spins > limit) {
            __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// One step's worth of a batch buffer for a consumer lane: coordinate metadata and the lane's SL
// entries (key, value, cold value).
template <int SL>
struct HotStep {
    uint32_t m, len;
    float m_old, sn, ylab;
    int32_t kk[SL];
    float vv[SL], xv[SL];
};

template <int SL>
__device__ __forceinline__ void hot_load_step(HotStep<SL>& t, const uint32_t* mb, const int32_t* key, const float* val,
                                              const float* cold, uint32_t B, uint32_t c, uint32_t e0, bool act) {
    t.m = mb[c];
    t.len = act ? mb[B + c] : 0u;
    t.m_old = __uint_as_float(mb[2u * B + c]);
    t.sn = __uint_as_float(mb[3u * B + c]);
    t.ylab = __uint_as_float(mb[4u * B + c]);
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        t.kk[r] = key[e0 + 8 * r];
        t.vv[r] = val[e0 + 8 * r];
        t.xv[r] = cold[e0 + 8 * r];
    }
}

// The consumer for coordinates of at most 8 * SL entries.  Per step: read the hot values the
// current keys point at, read the next step's metadata and entries (always, the last step
// re-reads its own, so that the number of LDS operations is fixed and the wait for the hot values
// never covers the prefetch), then reduce, step and scatter.  Hot entries are updated in LDS; the
// new model value and each cold entry's update go back into the batch buffer, and the producer
// that owns it issues the global stores and atomics before refilling it, so this wave never
// waits on global memory.
template <int FORM, typename U, int SL>
__device__ __forceinline__ void hot_consumer(const HotArgs& h, U* hot, uint32_t* ready, uint32_t* freed,
                                             uint32_t* abort_flag, uint32_t* bufs, uint32_t nb, int lane) {
    const EpochArgs& a = h.e;
    const uint32_t B = h.B, Smax = h.Smax, W = h.W, buf_words = 5u * B + 3u * B * Smax, S = B / W;
    const uint32_t g = (uint32_t)lane >> 3, sub = (uint32_t)lane & 7u;
    const bool act = g < W;
    for (uint32_t b = 0; b < nb; ++b) {
        const uint32_t p = b % kHotProducers, n = b / kHotProducers;
        if (!hot_wait(ready + p, n + 1, abort_flag, h.spin_limit, h.err)) return;
        uint32_t* const mb = bufs + p * buf_words;
        const int32_t* key = reinterpret_cast<const int32_t*>(mb + 5u * B);
        const float* val = reinterpret_cast<const float*>(key + B * Smax);
        float* const coldw = const_cast<float*>(val + B * Smax);
        HotStep<SL> cur;
        uint32_t c = act ? g : 0u;
        hot_load_step<SL>(cur, mb, key, val, coldw, B, c, c * Smax + sub, act);
        for (uint32_t st = 0; st < S; ++st) {
            const uint32_t e0 = c * Smax + sub;
            U hv[SL];
#pragma unroll
            for (int r = 0; r < SL; ++r) hv[r] = hot[cur.kk[r] >= 0 ? cur.kk[r] : 0];
            __builtin_amdgcn_sched_barrier(0);
            const uint32_t cn = st + 1 < S ? (st + 1) * W + (act ? g : 0u) : c;
            HotStep<SL> nxt;
            hot_load_step<SL>(nxt, mb, key, val, coldw, B, cn, cn * Smax + sub, act);
            __builtin_amdgcn_sched_barrier(0);
            float acc = 0.0f;
#pragma unroll
            for (int r = 0; r < SL; ++r) {
                const uint32_t msk = cur.kk[r] >= 0 ? 0xFFFFFFFFu : 0u;
                const float x = __uint_as_float((__float_as_uint((float)hv[r]) & msk) | (__float_as_uint(cur.xv[r]) & ~msk));
                if (sub + 8u * r < cur.len) acc = fmaf(cur.vv[r], x, acc);
            }
            const float gsum = group_sum<8>(acc);
            float coef;
            const float m_new = coord_step<FORM>(gsum, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
            if (act && cur.m != 0xFFFFFFFFu) {
                if (sub == 0) mb[2u * B + c] = __float_as_uint(m_new);
#pragma unroll
                for (int r = 0; r < SL; ++r) {
                    if (sub + 8u * r < cur.len) {
                        const float d = coef * cur.vv[r];
                        coldw[e0 + 8 * r] = d;  // read back only for cold entries
                        if (cur.kk[r] >= 0 && coef != 0.0f) atomicAdd(&hot[cur.kk[r]], (U)d);
                    }
                }
            }
            cur = nxt;
            c = cn;
        }
        __hip_atomic_store(freed + p, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

// Writes out a consumed batch buffer: new model values, and the updates of cold entries as
// device-scope atomics (fire and forget).
template <typename U>
__device__ __forceinline__ void hot_flush(const EpochArgs& a, const uint32_t* mb, const int32_t* key, const float* valb,
                                          const float* coldb, uint32_t B, uint32_t NB, int lane) {
    U* const uu = static_cast<U*>(a.u);
    if ((uint32_t)lane < B) {
        const uint32_t m = mb[lane];
        if (m != 0xFFFFFFFFu) a.model[m] = __uint_as_float(mb[2u * B + lane]);
    }
    for (uint32_t e = (uint32_t)lane; e < NB; e += 64) {
        const int32_t kk = key[e];
        const float d = coldb[e];
        if (kk < 0 && valb[e] != 0.0f && d != 0.0f) atomic_add_u(uu + ~kk, d);
    }
}

template <typename U>
__device__ __forceinline__ void hot_producer(const HotArgs& h, uint32_t* ready, uint32_t* freed, uint32_t* abort_flag,
                                             uint32_t* bufs, uint32_t nb, int q, int lane) {
    const EpochArgs& a = h.e;
    const U* const uu = static_cast<const U*>(a.u);
    const uint32_t B = h.B, Smax = h.Smax, C = a.perm.n, buf_words = 5u * B + 3u * B * Smax, NB = B * Smax;
    uint32_t* const mb = bufs + q * buf_words;
    int32_t* const key = reinterpret_cast<int32_t*>(mb + 5u * B);
    float* const valb = reinterpret_cast<float*>(key + NB);
    float* const coldb = valb + NB;
    constexpr int NE = kHotEntriesPerLane;
    // Buffer slot e = t * 64 + lane holds entry e % Smax of coordinate e / Smax of the batch; the
    // mapping is the same for every batch.
    const uint32_t c0 = (uint32_t)lane / Smax, k0 = (uint32_t)lane - c0 * Smax;
    const uint32_t dc = 64u / Smax, dk = 64u - dc * Smax;
    for (uint32_t b = (uint32_t)q; b < nb + kHotProducers; b += kHotProducers) {
        const uint32_t n = b / kHotProducers;
        if (n > 0 || b < nb) {  // the buffer's previous batch (if any) must have been consumed
            if (!hot_wait(freed + q, n, abort_flag, h.spin_limit, h.err)) return;
        }
        if (n > 0) hot_flush<U>(a, mb, key, valb, coldb, B, NB, lane);
        if (b >= nb) break;
        // Metadata: lane c < B holds coordinate c of the batch.
        const uint32_t j = b * B + (uint32_t)lane;
        const bool live = (uint32_t)lane < B && j < C;
        const uint32_t m = live ? perm_at(j, a.perm) : 0xFFFFFFFFu;
        const uint32_t mm = live ? m : 0u;  // loads below always hit a valid coordinate
        const int64_t s0 = a.ptr[mm], s1 = a.ptr[mm + 1];
        const float m_old = a.model[mm], sn = a.norms[mm], ylab = a.y[mm];
        const uint32_t len = live ? (uint32_t)(s1 - s0) : 0u;
        if ((uint32_t)lane < B) {
            mb[lane] = m;
            mb[B + lane] = len;
            mb[2u * B + lane] = __float_as_uint(m_old);
            mb[3u * B + lane] = __float_as_uint(sn);
            mb[4u * B + lane] = __float_as_uint(ylab);
        }
        // Entries, two stages of unconditional loads (entry 0 stands in for unused slots): index,
        // value and hot slot, then the current value of the shared vector.
        int32_t ix[NE];
        float vv[NE];
        uint32_t sl[NE];
        bool in[NE];
        uint32_t c = c0, k = k0;
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const uint32_t cc = c < B ? c : 0u;
            const int64_t sc = __shfl(s0, (int)cc);
            const uint32_t lc = (uint32_t)__shfl((int)len, (int)cc);
            in[t] = c < B && k < lc;
            const int64_t kk = in[t] ? sc + k : 0;
            ix[t] = a.idx[kk];
            vv[t] = a.val[kk];
            sl[t] = h.slot_entry[kk];
            c += dc;
            k += dk;
            if (k >= Smax) {
                k -= Smax;
                ++c;
            }
        }
        float cv[NE];
#pragma unroll
        for (int t = 0; t < NE; ++t) cv[t] = (float)uu[ix[t]];
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const uint32_t e = (uint32_t)t * 64u + (uint32_t)lane;
            if (e < NB) {
                key[e] = !in[t] ? 0 : (sl[t] != kHotCold ? (int32_t)sl[t] : ~ix[t]);
                valb[e] = in[t] ? vv[t] : 0.0f;
                coldb[e] = cv[t];
            }
        }
        __hip_atomic_store(ready + q, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

template <int FORM, typename U>
__global__ __launch_bounds__(64 * (1 + kHotProducers)) void k_epoch_hot(HotArgs h) {
    extern __shared__ __align__(16) unsigned char hot_lds[];
    const EpochArgs& a = h.e;
    U* const hot = reinterpret_cast<U*>(hot_lds);
    uint32_t* const ready = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes);
    uint32_t* const freed = ready + kHotProducers;
    uint32_t* const abort_flag = freed + kHotProducers;
    uint32_t* const bufs = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes + 64);
    U* const uu = static_cast<U*>(a.u);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (uint32_t i = tid; i < h.n_hot; i += blockDim.x) hot[i] = uu[h.hot_ids[i]];
    if (tid < 2 * kHotProducers + 1) ready[tid] = 0u;  // ready, freed and abort are contiguous
    __syncthreads();
    const uint32_t nb = (a.perm.n + h.B - 1) / h.B;
    if (wave == 0) {
        switch (h.Smax / 8) {  // entries per consumer lane
            case 1: hot_consumer<FORM, U, 1>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 2: hot_consumer<FORM, U, 2>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 3: hot_consumer<FORM, U, 3>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 4: hot_consumer<FORM, U, 4>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 5: hot_consumer<FORM, U, 5>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 6: hot_consumer<FORM, U, 6>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            case 7: hot_consumer<FORM, U, 7>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
            default: hot_consumer<FORM, U, 8>(h, hot, ready, freed, abort_flag, bufs, nb, lane); break;
        }
    } else
        hot_producer<U>(h, ready, freed, abort_flag, bufs, nb, wave - 1, lane);
    __syncthreads();
    for (uint32_t i = tid; i < h.n_hot; i += blockDim.x) uu[h.hot_ids[i]] = hot[i];
}

template <int FORM>
static hipError_t hot_prepare_form(bool wide, size_t lds_bytes) {
    const void* f = wide ? reinterpret_cast<const void*>(&k_epoch_hot<FORM, double>)
                         : reinterpret_cast<const void*>(&k_epoch_hot<FORM, float>);
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t hot_prepare(int form, bool wide, size_t lds_bytes) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: return hot_prepare_form<FORM_RIDGE_PRIMAL>(wide, lds_bytes);
        case FORM_SVM_DUAL: return hot_prepare_form<FORM_SVM_DUAL>(wide, lds_bytes);
        case FORM_RIDGE_DUAL: return hot_prepare_form<FORM_RIDGE_DUAL>(wide, lds_bytes);
        default: return hipErrorInvalidValue;
    }
}

template <int FORM>
static hipError_t launch_hot_form(bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s) {
    const dim3 block(64 * (1 + kHotProducers));
    if (wide)
        hipLaunchKernelGGL((k_epoch_hot<FORM, double>), dim3(1), block, lds_bytes, s, h);
    else
        hipLaunchKernelGGL((k_epoch_hot<FORM, float>), dim3(1), block, lds_bytes, s, h);
    return hipGetLastError();
}

hipError_t launch_epoch_hot(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: return launch_hot_form<FORM_RIDGE_PRIMAL>(wide, h, lds_bytes, s);
        case FORM_SVM_DUAL: return launch_hot_form<FORM_SVM_DUAL>(wide, h, lds_bytes, s);
        case FORM_RIDGE_DUAL: return launch_hot_form<FORM_RIDGE_DUAL>(wide, h, lds_bytes, s);
        default: return hipErrorInvalidValue;
    }
}

// ----------------------------------------------------------------------------------------
// Hot-set selection (set-up): the entries whose hit count (stored entries pointing at them,
// i.e. atomic adds per epoch) is at least T.  Slots are assigned in index order, so the set
// and its layout are a deterministic function of the matrix and T.
// ----------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_hot_count_ge(const unsigned* __restrict__ hits, int64_t L, unsigned T,
                                                      unsigned long long* __restrict__ out2) {
    unsigned long long cnt = 0, sum = 0;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < L; i += (int64_t)gridDim.x * 256) {
        const unsigned v = hits[i];
        if (v >= T) {
            ++cnt;
            sum += v;
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        cnt += __shfl_xor(cnt, o, 64);
        sum += __shfl_xor(sum, o, 64);
    }
    if ((threadIdx.x & 63) == 0 && (cnt || sum)) {
        atomicAdd(out2, cnt);
        atomicAdd(out2 + 1, sum);
    }
}

// Workgroup b covers indices [b * kHotAssignBlock, (b + 1) * kHotAssignBlock); thread t takes 4
// consecutive ones.
__global__ __launch_bounds__(256) void k_hot_block_count(const unsigned* __restrict__ hits, int64_t L, unsigned T,
                                                         unsigned* __restrict__ block_counts) {
    __shared__ unsigned red[4];
    const int64_t base = (int64_t)blockIdx.x * kHotAssignBlock + 4 * threadIdx.x;
    unsigned c = 0;
    for (int r = 0; r < 4; ++r) c += (base + r < L && hits[base + r] >= T) ? 1u : 0u;
    for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o, 64);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) block_counts[blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

__global__ __launch_bounds__(256) void k_hot_assign(const unsigned* __restrict__ hits, int64_t L, unsigned T,
                                                    const unsigned* __restrict__ block_base,
                                                    uint16_t* __restrict__ slot_of, int32_t* __restrict__ hot_ids) {
    __shared__ unsigned scan[256];
    const int64_t base = (int64_t)blockIdx.x * kHotAssignBlock + 4 * threadIdx.x;
    bool f[4];
    unsigned c = 0;
    for (int r = 0; r < 4; ++r) {
        f[r] = base + r < L && hits[base + r] >= T;
        c += f[r] ? 1u : 0u;
    }
    scan[threadIdx.x] = c;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {  // inclusive Hillis-Steele scan
        const unsigned add = threadIdx.x >= (unsigned)o ? scan[threadIdx.x - o] : 0u;
        __syncthreads();
        scan[threadIdx.x] += add;
        __syncthreads();
    }
    unsigned slot = block_base[blockIdx.x] + scan[threadIdx.x] - c;
    for (int r = 0; r < 4; ++r) {
        if (base + r >= L) break;
        if (f[r]) {
            slot_of[base + r] = (uint16_t)slot;
            hot_ids[slot] = (int32_t)(base + r);
            ++slot;
        } else {
            slot_of[base + r] = kHotCold;
        }
    }
}

hipError_t launch_count_hits(const int32_t* idx, int64_t nnz, unsigned* hits, hipStream_t s) {
    if (nnz > 0) hipLaunchKernelGGL(k_count_hits, dim3(grid_for(nnz)), dim3(256), 0, s, idx, nnz, hits);
    return hipGetLastError();
}

hipError_t launch_hot_count_ge(const unsigned* hits, int64_t L, unsigned T, unsigned long long* out2, hipStream_t s) {
    hipLaunchKernelGGL(k_hot_count_ge, dim3(grid_for(L)), dim3(256), 0, s, hits, L, T, out2);
    return hipGetLastError();
}

hipError_t launch_hot_block_count(const unsigned* hits, int64_t L, unsigned T, unsigned* block_counts, hipStream_t s) {
    const int64_t nb = (L + kHotAssignBlock - 1) / kHotAssignBlock;
    hipLaunchKernelGGL(k_hot_block_count, dim3((unsigned)nb), dim3(256), 0, s, hits, L, T, block_counts);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void k_hot_entry_slots(const int32_t* __restrict__ idx, int64_t nnz,
                                                         const uint16_t* __restrict__ slot_of,
                                                         uint16_t* __restrict__ slot_entry) {
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < nnz; k += (int64_t)gridDim.x * 256)
        slot_entry[k] = slot_of[idx[k]];
}

hipError_t launch_hot_entry_slots(const int32_t* idx, int64_t nnz, const uint16_t* slot_of, uint16_t* slot_entry,
                                  hipStream_t s) {
    const int64_t want = (nnz + 255) / 256;
    const unsigned blocks = (unsigned)(want < 1 ? 1 : want > 65536 ? 65536 : want);
    hipLaunchKernelGGL(k_hot_entry_slots, dim3(blocks), dim3(256), 0, s, idx, nnz, slot_of, slot_entry);
    return hipGetLastError();
}

hipError_t launch_hot_assign(const unsigned* hits, int64_t L, unsigned T, const unsigned* block_base, uint16_t* slot_of,
                             int32_t* hot_ids, hipStream_t s) {
    const int64_t nb = (L + kHotAssignBlock - 1) / kHotAssignBlock;
    hipLaunchKernelGGL(k_hot_assign, dim3((unsigned)nb), dim3(256), 0, s, hits, L, T, block_base, slot_of, hot_ids);
    return hipGetLastError();
}

}  // namespace scd
