// scd_team.hip -- team epoch kernel: long segments with few coordinates in flight.
//
// Alg. 2 gives each coordinate one thread block.  With long segments and a binding window (tens of
// coordinates in flight), that leaves most CUs idle, and each coordinate's thousands of scattered
// gathers and atomics go through one CU's address unit and its outstanding-miss capacity: on the
// text-SVM workload (3,700 entries per row, 32 rows in flight) one row takes about 14 us in one
// workgroup.  Here a team of K workgroups (on K CUs) processes each in-flight coordinate, member k
// on the entries whose shared-vector index lies in the k-th of K index ranges:
//
//   1. gather: member k reads the shared-vector entries of its part of the segment;
//   2. reduce: the workgroup sums its lanes' products (DPP within each wave, LDS across waves);
//   3. exchange: wave 0 publishes the partial sum in a 64-bit slot (fp32 bits + step tag) and
//      polls the team's K slots until all carry this step's tag; every member adds the K partials
//      in the same order, so all compute the same inner product and the same step (eq.
//      update_primal, the SVM dual step, or eq. update_dual);
//   4. scatter: member k adds coef * a_m into its own index range, then waits for those atomics
//      before it gathers the team's next coordinate (each wave waits for its own, and a barrier
//      joins the four waves, so the wait covers every atomic of the member).
//
// Because a member's gathers and atomics touch only its own index range, its own wait in step 4
// is enough: when any member gathers coordinate c + 1, every update of coordinate c to the entries
// it reads has landed.  A team thus holds one coordinate between gather and scatter, as a
// draining group of the pipelined kernel does, and n_groups teams keep the window.
//
// Slots: team t, step tag g, member k at slots[(t * 2 + g % 2) * kTeamMax + k].  Tags grow by one
// per step (and across launches, from the host's counter), so a slot that has not been rewritten
// for this step carries an older tag.  A member overwrites the slot of step g at step g + 2, after
// it has seen every member's partial of step g + 1, which each member publishes only after it has
// read all partials of step g: no member still waits on the value being overwritten.  Each slot is
// one location written and read with 64-bit device-scope atomics, so no ordering between
// locations is needed.  Every wait is bounded (spin_limit sleeps); a member that gives up sets
// *err and leaves, and the others give up in turn.  The grid fits the CUs (one workgroup per CU at
// most), so every member is resident while the others wait for it.
#include <algorithm>

#include "scd_device.h"
#include "scd_kernels.h"

namespace scd {
namespace {

// Member k's part of coordinate m, as loaded: the segment start and the part's offsets stay
// separate until the step that uses them (after its full wait), so that no addition has to wait
// for loads issued as prefetches.
struct TeamMeta {
    int64_t base;
    uint32_t o0, o1, m;
    float m_old, sn, ylab;
};

__device__ __forceinline__ TeamMeta team_meta(const TeamArgs& t, uint32_t m, uint32_t k) {
    TeamMeta c;
    c.m = m;
    c.base = t.e.ptr[m];
    const uint32_t* o = t.off + (size_t)m * (t.K + 1) + k;
    c.o0 = o[0];
    c.o1 = o[1];
    c.m_old = t.e.model[m];
    c.sn = t.e.norms[m];
    c.ylab = t.e.y[m];
    return c;
}

__device__ __forceinline__ CoordMeta team_part(const TeamMeta& t) {
    CoordMeta c;
    c.m = t.m;
    c.s0 = t.base + t.o0;
    c.s1 = t.base + t.o1;
    c.m_old = t.m_old;
    c.sn = t.sn;
    c.ylab = t.ylab;
    return c;
}

__device__ __forceinline__ uint64_t team_pack(float p, uint32_t tag) {
    return ((uint64_t)tag << 32) | (uint64_t)__builtin_bit_cast(uint32_t, p);
}

// Scatter of one register slice.  Every step begins with a full wait, so no wait count depends on
// the number of operations issued here: inactive lanes simply issue nothing.
template <typename U>
__device__ __forceinline__ void team_atomic(const SharedBuf<U>& b, uint32_t i, bool in, float v) {
    if constexpr (sizeof(U) == 4)
        buf_atomic_add(b, i, in, v);  // out-of-range offset: dropped
    else if (in)
        atomic_add_u(reinterpret_cast<U*>(reinterpret_cast<char*>(b.base) + ((size_t)i << b.shift)), v);
}

// One coordinate of the team (its position j, step tag `tag`).  `cur` and its part `ci/cv` and
// `nxt`'s metadata were loaded one step earlier; loads `nxt`'s part into `ni/nv` and the
// metadata of the coordinate two steps ahead into `nn`.  Returns false after the team's last
// coordinate or when a wait gave up.
template <int FORM, int R, bool FRESH, typename U>
__device__ __forceinline__ bool team_step(const TeamArgs& t, const SharedBuf<U>& ub, uint32_t k, uint32_t team,
                                          int lane, uint32_t j, uint32_t tag, const TeamMeta& tcur,
                                          const int (&ci)[R], const float (&cv)[R], const TeamMeta& tnxt,
                                          int (&ni)[R], float (&nv)[R], TeamMeta& nn, float (*part)[4],
                                          float* gsum, int* gok) {
    const EpochArgs& a = t.e;
    // This member's atomics of the previous coordinate land before it gathers again: each wave
    // waits for its own, and the barrier holds all four waves until every one has.
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    const CoordMeta cur = team_part(tcur), nxt = team_part(tnxt);
    const int64_t len = cur.s1 - cur.s0;
    const uint64_t P = a.n_groups, n = a.perm.n;
    const bool more = (uint64_t)j + P < n;
    const uint64_t j2 = (uint64_t)j + 2 * P;
    const uint32_t m2 = perm_at(j2 < n ? (uint32_t)j2 : j, a.perm);
    const bool lng = len > (int64_t)256 * R;
    // The gathers go out first (a long part is streamed and summed here instead); the next part
    // and the metadata two ahead are prefetched on both paths by the same code, issued before the
    // wait for the gathers.
    float acc = 0.0f, gv[R];
    if (lng) {
        acc = long_dot<256, FRESH>(a, ub, lane, cur.s0, cur.s1);
    } else {
#pragma unroll
        for (int r = 0; r < R; ++r) gv[r] = buf_load<FRESH>(ub, (uint32_t)ci[r], (int64_t)(lane + r * 256) < len);
    }
    __builtin_amdgcn_sched_barrier(0);
    load_seg_raw<256, R>(a, nxt, lane, ni, nv);
    nn = team_meta(t, m2, k);
    __builtin_amdgcn_sched_barrier(0);
    if (!lng) {
#pragma unroll
        for (int r = 0; r < R; ++r) acc = fmaf(cv[r], gv[r], acc);
    }
    const int wave = lane >> 6, par = (int)(tag & 1u);
    acc = group_sum<64>(acc);
    if ((lane & 63) == 0) part[par][wave] = acc;
    __syncthreads();
    if (wave == 0) {
        const float p = (part[par][0] + part[par][1]) + (part[par][2] + part[par][3]);
        uint64_t* slot = t.slots + ((size_t)team * 2 + (size_t)par) * kTeamMax;
        if (lane == 0) __hip_atomic_store(slot + k, team_pack(p, tag), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int q = lane & (kTeamMax - 1);
        const bool mine = (uint32_t)lane < t.K;
        uint32_t pv = 0;
        int ok = 1;
        for (uint32_t spins = 0;; ++spins) {
            const uint64_t v = mine ? __hip_atomic_load(slot + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                    : team_pack(0.0f, tag);
            if (__all((uint32_t)(v >> 32) == tag)) {
                pv = (uint32_t)v;
                break;
            }
            if (spins >= t.spin_limit) {
                ok = 0;
                if (lane == 0) __hip_atomic_fetch_or(t.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        // The K partials in member order: every member forms the same sum.
        float g = 0.0f;
#pragma unroll
        for (int w = 0; w < kTeamMax; ++w)
            if ((uint32_t)w < t.K) g += __builtin_bit_cast(float, __builtin_amdgcn_readlane((int)pv, w));
        if (lane == 0) {
            gsum[par] = g;
            gok[par] = ok;
        }
    }
    __syncthreads();
    if (!gok[par]) return false;
    const float g = gsum[par];
    float coef;
    const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
    a.model[cur.m] = m_new;  // every lane of every member stores the same value
    if (coef != 0.0f) {
        if (lng) {
            long_scatter<256>(a, ub, lane, cur.s0, cur.s1, coef);
        } else {
#pragma unroll
            for (int r = 0; r < R; ++r) team_atomic(ub, (uint32_t)ci[r], (int64_t)(lane + r * 256) < len, coef * cv[r]);
        }
    }
    return more;
}

template <int FORM, int R, bool FRESH, typename U>
__global__ __launch_bounds__(256) void k_epoch_team(TeamArgs t) {
    __shared__ float part[2][4];
    __shared__ float gsum[2];
    __shared__ int gok[2];
    const EpochArgs& a = t.e;
    // XCD-aware placement.  Workgroups are dispatched to the kTeamXcds XCDs in turn (workgroup b to XCD
    // b mod kTeamXcds).  Member k of team t is placed on XCD (t + k) mod kTeamXcds, so the owners of
    // each index range (member k of every team) are spread over all XCDs whatever K is.  In the plain
    // order (workgroup t K + k), K = 8 put every owner of range k on XCD k; the scatter into each
    // range then went through one XCD, and an epoch took 40% longer than at K = 7 or 9.  Workgroup b
    // takes the (b / kTeamXcds)-th pair, in team-major order, among the pairs placed on its XCD;
    // workgroups beyond them leave.
    uint32_t team = 0xFFFFFFFFu, k = 0;
    {
        const uint32_t x = blockIdx.x % kTeamXcds, want = blockIdx.x / kTeamXcds;
        uint32_t seen = 0;
        for (uint32_t tt = 0; tt < a.n_groups && team == 0xFFFFFFFFu; ++tt)
            for (uint32_t kk = 0; kk < t.K; ++kk)
                if ((tt + kk) % kTeamXcds == x) {
                    if (seen == want) {
                        team = tt;
                        k = kk;
                        break;
                    }
                    ++seen;
                }
    }
    if (team == 0xFFFFFFFFu || team >= a.perm.n) return;  // the whole workgroup leaves
    const int lane = threadIdx.x;
    const SharedBuf<U> ub =
        shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x, a.u_shift);
    const uint32_t P = a.n_groups;
    uint32_t j = team, tag = t.tag0;
    TeamMeta cA = team_meta(t, perm_at(j, a.perm), k);
    int ciA[R], ciB[R];
    float cvA[R], cvB[R];
    load_seg_raw<256, R>(a, team_part(cA), lane, ciA, cvA);
    TeamMeta cB = team_meta(t, perm_at((uint64_t)j + P < a.perm.n ? j + P : j, a.perm), k);
    for (;;) {
        TeamMeta cA2, cB2;
        if (!team_step<FORM, R, FRESH, U>(t, ub, k, team, lane, j, tag, cA, ciA, cvA, cB, ciB, cvB, cA2, part, gsum,
                                          gok))
            break;
        j += P;
        ++tag;
        if (!team_step<FORM, R, FRESH, U>(t, ub, k, team, lane, j, tag, cB, ciB, cvB, cA2, ciA, cvA, cB2, part, gsum,
                                          gok))
            break;
        j += P;
        ++tag;
        cA = cA2;
        cB = cB2;
    }
}

// Groups the entries of each segment by index range, keeping their order within a range: one wave
// per segment, two passes (count, then place) over 64-entry chunks, with one ballot per range and
// chunk.  off[m(K+1)+q] = entries of segment m in ranges below q.
__global__ __launch_bounds__(256) void k_team_partition(const int64_t* __restrict__ ptr, const int32_t* __restrict__ idx,
                                                        const float* __restrict__ val, uint32_t C,
                                                        const uint32_t* __restrict__ bound, int K,
                                                        int32_t* __restrict__ oidx, float* __restrict__ oval,
                                                        uint32_t* __restrict__ off) {
    __shared__ uint32_t sb[kTeamMax + 1];
    if (threadIdx.x <= (unsigned)K) sb[threadIdx.x] = bound[threadIdx.x];
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
    for (uint32_t m = blockIdx.x * 4u + (threadIdx.x >> 6); m < C; m += gridDim.x * 4u) {
        const int64_t s0 = ptr[m], s1 = ptr[m + 1];
        uint32_t pos[kTeamMax];
#pragma unroll
        for (int q = 0; q < kTeamMax; ++q) pos[q] = 0;
        for (int64_t b = s0; b < s1; b += 64) {
            const int64_t e = b + lane;
            const bool in = e < s1;
            const uint32_t i = in ? (uint32_t)idx[e] : 0u;
            int r = 0;
            for (int q = 1; q < K; ++q) r += i >= sb[q] ? 1 : 0;
#pragma unroll
            for (int q = 0; q < kTeamMax; ++q)
                if (q < K) pos[q] += (uint32_t)__popcll(__ballot(in && r == q));
        }
        // Exclusive prefix: pos[q] becomes the first offset of range q.
        uint32_t run = 0;
#pragma unroll
        for (int q = 0; q < kTeamMax; ++q) {
            if (q < K) {
                const uint32_t c = pos[q];
                pos[q] = run;
                if (lane == q) off[(size_t)m * (K + 1) + q] = run;
                run += c;
            }
        }
        if (lane == 0) off[(size_t)m * (K + 1) + K] = run;
        for (int64_t b = s0; b < s1; b += 64) {
            const int64_t e = b + lane;
            const bool in = e < s1;
            const uint32_t i = in ? (uint32_t)idx[e] : 0u;
            const float v = in ? val[e] : 0.0f;
            int r = 0;
            for (int q = 1; q < K; ++q) r += i >= sb[q] ? 1 : 0;
#pragma unroll
            for (int q = 0; q < kTeamMax; ++q) {
                if (q < K) {
                    const uint64_t mask = __ballot(in && r == q);
                    if (in && r == q) {
                        const int64_t d = s0 + pos[q] + __popcll(mask & below);
                        oidx[d] = (int32_t)i;
                        oval[d] = v;
                    }
                    pos[q] += (uint32_t)__popcll(mask);
                }
            }
        }
    }
}

// An ordinary launch.  The members wait for one another, so the whole grid must be resident at
// once: the plan keeps it within the CUs (one 256-thread workgroup per CU at most), and the launch
// is refused unless the occupancy query confirms that every CU holds at least one workgroup of
// this kernel.  Work enqueued earlier on the same stream has finished when the grid starts; a
// kernel of another stream or process that holds CUs can delay members, and the bounded waits then
// report an error instead of hanging.  (A cooperative launch would give the same guarantee, but
// it runs on a separate device queue of the runtime; the only processes whose profiler runs ended
// in a fault inside the exit handlers, after the profiler's own finalisation, were those that had
// made such launches.)
template <int FORM, bool FRESH, typename U>
hipError_t launch_team_typed(const TeamArgs& t, int blocks, int cus, hipStream_t s) {
    const void* f = reinterpret_cast<const void*>(&k_epoch_team<FORM, kTeamSlices, FRESH, U>);
    int per_cu = 0;
    const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, 256, 0);
    if (e != hipSuccess) return e;
    if (per_cu < 1 || blocks > per_cu * cus) return hipErrorCooperativeLaunchTooLarge;
    hipLaunchKernelGGL((k_epoch_team<FORM, kTeamSlices, FRESH, U>), dim3(blocks), dim3(256), 0, s, t);
    return hipGetLastError();
}

template <int FORM>
hipError_t launch_team_form(bool wide, bool fresh, const TeamArgs& t, int blocks, int cus, hipStream_t s) {
    if (wide)
        return fresh ? launch_team_typed<FORM, true, double>(t, blocks, cus, s)
                     : launch_team_typed<FORM, false, double>(t, blocks, cus, s);
    return fresh ? launch_team_typed<FORM, true, float>(t, blocks, cus, s)
                 : launch_team_typed<FORM, false, float>(t, blocks, cus, s);
}

}  // namespace

hipError_t launch_epoch_team(int form, bool wide, bool fresh, const TeamArgs& t, int blocks, int cus, hipStream_t s) {
    switch (form) {
        case FORM_RIDGE_PRIMAL: return launch_team_form<FORM_RIDGE_PRIMAL>(wide, fresh, t, blocks, cus, s);
        case FORM_SVM_DUAL: return launch_team_form<FORM_SVM_DUAL>(wide, fresh, t, blocks, cus, s);
        case FORM_RIDGE_DUAL: return launch_team_form<FORM_RIDGE_DUAL>(wide, fresh, t, blocks, cus, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_team_partition(const int64_t* ptr, const int32_t* idx, const float* val, uint32_t C,
                                 const uint32_t* bound, int K, int32_t* out_idx, float* out_val, uint32_t* off,
                                 hipStream_t s) {
    if (K < 1 || K > kTeamMax) return hipErrorInvalidValue;
    if (C == 0) return hipSuccess;
    const unsigned blocks = (unsigned)std::min<uint64_t>(8192, ((uint64_t)C + 3) / 4);
    hipLaunchKernelGGL(k_team_partition, dim3(blocks), dim3(256), 0, s, ptr, idx, val, C, bound, K, out_idx, out_val,
                       off);
    return hipGetLastError();
}

}  // namespace scd
