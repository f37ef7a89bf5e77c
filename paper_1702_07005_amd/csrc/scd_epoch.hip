// scd_epoch.hip -- epoch kernels for gfx950 (CDNA4, wave64) of asynchronous stochastic
// coordinate descent/ascent (arXiv 1702.07005, Sec. III-C "TPA-SCD", Alg. 2).
//
// Every coordinate c owns one segment [ptr[c], ptr[c+1]) of (idx, val): a column of A for
// the ridge primal (CSC), a row for the duals (CSR).  One epoch = one persistent launch in
// which groups of lanes take permutation positions, at a fixed stride j = g, g + P, g + 2P, ...
// or in order from a queue (P groups in flight: the "window"), and for the coordinate m = pi(j):
//   1. gather  g = <a_m, u>   over the segment (u = the shared vector, see below),
//   2. reduce the lane partials inside the group (DPP / swizzle, LDS across waves),
//   3. step    closed form of the formulation -> model[m], scatter coefficient,
//   4. scatter u[idx] += coef * val  with device-scope atomics (no return; fp32, or fp64 where
//      one entry takes many adds per epoch).
//
// Shared vector kept on the device, per formulation:
//   ridge primal : w = A beta.  The step needs <y - w, a_m> (eq. update_primal); it is taken
//                  as cy_m - <w, a_m> with cy_m = <y, a_m> computed once at set-up, so each
//                  stored entry costs one gather (w) instead of two (y and w).
//   SVM dual     : w = sum_i alpha_i y_i x_i / (lambda N).
//   ridge dual   : wbar = A^T alpha (eq. update_dual).
// `y` in the epoch arguments is the per-coordinate constant: cy for the ridge primal, the
// label for the duals.
#include "scd_device.h"

namespace scd {

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
        // With a binding window the previous coordinate's atomics land first (the group lives in
        // one wave, whose completion counter covers them all).
        if (a.drain) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
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
    // A wave's wait covers only its own atomics: with G = 256 the group spans four waves, and a
    // barrier after the wait holds every wave's gathers until all four have landed theirs.
    if (a.drain) {
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        if constexpr (G > 64) __builtin_amdgcn_s_barrier();
    }
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
        shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x, a.u_shift);
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
    // vmcnt(0): this wave's atomics and its last claim have landed; the barrier extends that to the
    // atomics of all four waves before any of them gathers the next coordinate.
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __builtin_amdgcn_s_barrier();
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
            shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x,
                          a.u_shift);
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
        if constexpr (!ORDERED) {
            // With a binding window every wave's atomics of the previous coordinate land before any
            // wave gathers this one, so a workgroup holds one coordinate between gather and scatter.
            if (a.drain) {
                __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
                __builtin_amdgcn_s_barrier();
            }
        }
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

}  // namespace scd
