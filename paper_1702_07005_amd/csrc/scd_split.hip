// scd_split.hip -- split epoch kernel: the queued kernel over work units, with long segments split
// into parts that many workgroups (on many CUs) gather and scatter at once.
//
// Alg. 2 gives each coordinate one thread block.  On skewed lengths (text columns: the densest
// cover every row) one workgroup streams a long segment for milliseconds, and while it is between
// its gather and its scatter thousands of other coordinates start, among them other dense columns
// it couples strongly with.  The processing order and the window then no longer bound the
// staleness the step sees.  Here a segment of len > part entries is cut into k = ceil(len / part)
// parts, and the epoch's work is a sequence of units in permutation order:
//
//   FULL    (len <= part)  gather, reduce, step (eq. update_primal, the SVM dual step, or eq.
//                          update_dual), model store, scatter: one unit of the queued kernel;
//   GATHER  part i of k    gather part i, reduce, publish the partial inner product in a 64-bit slot
//                          (fp32 bits | launch tag << 32) at partials[unit index];
//   SCATTER part i of k    wait until the k GATHER slots of the coordinate carry this launch's tag,
//                          sum them in a fixed order (the same in every part, so every part takes the
//                          bitwise-same step), store the model (part 0) and scatter part i.
//
// A coordinate's k GATHER units are followed at once by its k SCATTER units, so the workgroups that
// claim them next process the parts side by side: the segment is between its first gather and its
// last scatter for about two unit steps instead of len / part of them.  Units are claimed from the
// position queue in chunks, as in the queued kernel (one returning atomic per chunk, issued with
// the prefetches); a workgroup processes its claimed units in order.
//
// Progress: a GATHER or FULL unit never waits on another workgroup.  A SCATTER unit waits only on
// GATHER units with smaller indices.  The smallest unfinished unit is therefore always the current
// unit of the workgroup that claimed it (its earlier units are finished), and if it is a SCATTER
// unit, the GATHER units it waits on are finished: it finishes.  This holds however many units a
// workgroup holds and however many workgroups are resident.  Every wait is still bounded (spin_limit
// sleeps); a unit that gives up sets *err and skips its scatter, and the other waits then give up too.
//
// Pre-pass (each epoch, stream-ordered before the epoch kernel): the units of permutation position j
// depend on len(pi(j)) only, so a count pass (tiles of kSplitPrepTile positions), one exclusive scan
// of the tile counts, and a write pass that recomputes the counts, scans them inside the tile and
// writes the records.  A record carries the coordinate's metadata (segment range, norm, model value
// at the start of the epoch, constant), so the epoch kernel reads one 32-byte record per unit instead
// of five scattered words.
#include "scd_device.h"
#include "scd_kernels.h"

namespace scd {
namespace {

constexpr int kSplitRing = 4;  // chunk bases held in LDS (chunk number mod 4)
constexpr int kSplitLead = 4;  // steps between a claim and the first step of its chunk
constexpr int kPrepPer = kSplitPrepTile / 256;  // positions per thread of the pre-pass

__device__ __forceinline__ uint32_t split_kind(uint32_t info) { return info >> 30; }
__device__ __forceinline__ uint32_t split_parts(uint32_t info) { return (info >> 15) & 0x7FFFu; }
__device__ __forceinline__ uint32_t split_index(uint32_t info) { return info & 0x7FFFu; }

__device__ __forceinline__ uint32_t units_at(const int64_t* ptr, const PermKeys& p, uint32_t j, uint32_t part) {
    const uint32_t m = perm_at(j, p);
    return split_units_of(ptr[m + 1] - ptr[m], part);
}

// Sum of v over the 256 threads of the workgroup (every thread gets it).
__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* sh) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = v;
    __syncthreads();
    const uint32_t t = sh[0] + sh[1] + sh[2] + sh[3];
    __syncthreads();
    return t;
}

__global__ __launch_bounds__(256) void k_split_total(const int64_t* __restrict__ ptr, uint32_t C, uint32_t part,
                                                     unsigned long long* out) {
    __shared__ uint32_t sh[4];
    uint32_t t = 0;
    for (uint32_t m = blockIdx.x * 256u + threadIdx.x; m < C; m += gridDim.x * 256u)
        t += split_units_of(ptr[m + 1] - ptr[m], part);
    t = block_sum_u32(t, sh);
    if (threadIdx.x == 0) atomicAdd(out, (unsigned long long)t);
}

// Units of each tile of kSplitPrepTile permutation positions.
__global__ __launch_bounds__(256) void k_split_count(const int64_t* __restrict__ ptr, PermKeys p, uint32_t part,
                                                     uint32_t* __restrict__ tile_units) {
    __shared__ uint32_t sh[4];
    const uint64_t j0 = (uint64_t)blockIdx.x * kSplitPrepTile + (uint64_t)threadIdx.x * kPrepPer;
    uint32_t t = 0;
#pragma unroll
    for (int i = 0; i < kPrepPer; ++i)
        if (j0 + i < p.n) t += units_at(ptr, p, (uint32_t)(j0 + i), part);
    t = block_sum_u32(t, sh);
    if (threadIdx.x == 0) tile_units[blockIdx.x] = t;
}

// Exclusive scan of the tile counts in place (one workgroup of 1024 threads).
__global__ __launch_bounds__(1024) void k_split_scan(uint32_t* __restrict__ tile_units, uint32_t n_tiles) {
    __shared__ uint32_t sh[1024];
    const uint32_t per = (n_tiles + 1023u) / 1024u;
    const uint32_t b0 = min(n_tiles, threadIdx.x * per), b1 = min(n_tiles, b0 + per);
    uint32_t s = 0;
    for (uint32_t b = b0; b < b1; ++b) s += tile_units[b];
    sh[threadIdx.x] = s;
    __syncthreads();
    for (uint32_t o = 1; o < 1024u; o <<= 1) {
        const uint32_t v = threadIdx.x >= o ? sh[threadIdx.x - o] : 0u;
        __syncthreads();
        sh[threadIdx.x] += v;
        __syncthreads();
    }
    uint32_t run = sh[threadIdx.x] - s;
    for (uint32_t b = b0; b < b1; ++b) {
        const uint32_t x = tile_units[b];
        tile_units[b] = run;
        run += x;
    }
}

// Writes the unit records of each tile, at the tile's offset.  Thread t takes positions t, t + 256,
// ... of the tile, so that consecutive lanes write consecutive records (most positions are one
// unit); the offsets follow position order: slice i (positions i * 256 + t) after slices < i.
__global__ __launch_bounds__(256) void k_split_write(EpochArgs a, uint32_t part,
                                                     const uint32_t* __restrict__ tile_base,
                                                     SplitUnit* __restrict__ units) {
    __shared__ uint32_t wsum[4];
    const PermKeys& p = a.perm;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const uint64_t j0 = (uint64_t)blockIdx.x * kSplitPrepTile;
    uint32_t base = tile_base[blockIdx.x];
    for (int i = 0; i < kPrepPer; ++i) {
        const uint64_t j = j0 + (uint64_t)i * 256 + t;
        const bool in = j < p.n;
        const uint32_t m = in ? perm_at((uint32_t)j, p) : 0u;
        const int64_t s0 = in ? a.ptr[m] : 0, len = in ? a.ptr[m + 1] - s0 : 0;
        const uint32_t cnt = in ? split_units_of(len, part) : 0u;
        // Exclusive prefix of cnt over the slice's 256 threads: inside the wave, then across waves.
        uint32_t incl = cnt;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t v = __shfl_up(incl, o, 64);
            if (lane >= o) incl += v;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        uint32_t before = 0;
        for (int w = 0; w < wave; ++w) before += wsum[w];
        const uint32_t total = wsum[0] + wsum[1] + wsum[2] + wsum[3];
        __syncthreads();
        const uint32_t at = base + before + incl - cnt;
        base += total;
        if (!in) continue;
        SplitUnit r;
        r.m = m;
        r.m_old = a.model[m];
        r.sn = a.norms[m];
        r.ylab = a.y[m];
        if (cnt == 1u) {
            r.s0 = s0;
            r.len = (uint32_t)len;
            r.info = (uint32_t)SPLIT_FULL << 30;
            units[at] = r;
        } else {
            const uint32_t k = cnt / 2u;
            for (uint32_t q = 0; q < k; ++q) {
                r.s0 = s0 + (int64_t)q * part;
                const int64_t rest = len - (int64_t)q * part;
                r.len = (uint32_t)(rest < (int64_t)part ? rest : (int64_t)part);
                r.info = ((uint32_t)SPLIT_GATHER << 30) | (k << 15) | q;
                units[at + q] = r;
                r.info = ((uint32_t)SPLIT_SCATTER << 30) | (k << 15) | q;
                units[at + k + q] = r;
            }
        }
    }
}

__device__ __forceinline__ uint32_t split_pos(const uint32_t* ring, uint32_t k, uint32_t chunk) {
    return ring[(k / chunk) % kSplitRing] + k % chunk;
}

// Register slices of a unit's range: element s0 + lane + r * 256.  Slices past the end for the whole
// wave are not loaded (and not used); in a slice that the end cuts, lanes past it read entry 0
// (always present: the library never hands the kernels an empty idx/val) and are masked by an
// out-of-range shared-vector offset (gathers return 0, atomics are dropped).
template <int R>
__device__ __forceinline__ void load_unit_seg(const EpochArgs& a, const SplitUnit& c, int lane, int (&ci)[R],
                                              float (&cv)[R]) {
    const int64_t wb = lane & ~63;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (wb + r * 256 >= (int64_t)c.len) continue;  // no entry of this wave in slice r
        const int64_t k = lane + (int64_t)r * 256;
        const int64_t kk = k < (int64_t)c.len ? c.s0 + k : 0;
        ci[r] = a.idx[kk];
        cv[r] = a.val[kk];
    }
}

// Sum over the workgroup's 256 lanes: DPP within each wave, then the four wave sums through LDS in
// wave order (double-buffered, so that one barrier per reduction suffices).
__device__ __forceinline__ float pipe_reduce_256(float acc, float (*part)[4], int& buf) {
    acc = group_sum<64>(acc);
    if ((threadIdx.x & 63) == 0) part[buf][threadIdx.x >> 6] = acc;
    __syncthreads();
    const float g = (part[buf][0] + part[buf][1]) + (part[buf][2] + part[buf][3]);
    buf ^= 1;
    return g;
}

template <typename U>
__device__ __forceinline__ void split_atomic(const SharedBuf<U>& b, uint32_t i, bool in, float v) {
    if constexpr (sizeof(U) == 4)
        buf_atomic_add(b, i, in, v);  // out-of-range offset: dropped
    else if (in)
        atomic_add_u(reinterpret_cast<U*>(reinterpret_cast<char*>(b.base) + ((size_t)i << b.shift)), v);
}

// One unit (step k of this workgroup; `at` = its unit index).  `cur` and its range `ci/cv`, and
// `nxt`'s record, were loaded one step earlier.  Loads `nxt`'s range into `ni/nv` and the record of
// the unit two steps ahead into `nn`; returns that unit's index (>= n_units when the queue is
// exhausted; `nn` then holds unit 0 as a stand-in that is never processed).
template <int FORM, int R, bool FRESH, typename U>
__device__ __forceinline__ uint32_t split_step(const SplitArgs& sa, const SharedBuf<U>& ub,
                                               const __amdgpu_buffer_rsrc_t& qr, int lane, uint32_t k,
                                               const SplitUnit& cur, uint32_t at, const int (&ci)[R],
                                               const float (&cv)[R], const SplitUnit& nxt, int (&ni)[R],
                                               float (&nv)[R], SplitUnit& nn, uint32_t* ring, uint32_t& claim,
                                               float (*part)[4], int& buf, float* gsum, int* gok) {
    const EpochArgs& a = sa.e;
    const uint32_t K = a.chunk;
    // vmcnt(0): this wave's atomics and its last claim have landed; the barrier extends that to the
    // atomics of all four waves before any of them gathers the next unit.
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __builtin_amdgcn_s_barrier();
    // The previous step claimed chunk (k - 1 + kSplitLead) / K if it began one.
    if (lane == 0 && k > 0 && (k - 1 + kSplitLead) % K == 0) ring[((k - 1 + kSplitLead) / K) % kSplitRing] = claim;
    const uint32_t n = sa.n_units;
    const uint32_t p2 = split_pos(ring, k + 2, K);  // its chunk was published before the previous barrier
    const int qoff = lane == 0 && (k + kSplitLead) % K == 0 ? 0 : 4;
    const uint32_t kind = split_kind(cur.info);
    const int64_t len = cur.len;
    const bool gathers = kind != SPLIT_SCATTER;
    // A slice that holds none of the unit's entries for this wave (most units are short) issues
    // nothing: the branch is uniform over the wave.
    const int64_t wb = lane & ~63;
    float gv[R];
#pragma unroll
    for (int r = 0; r < R; ++r)
        if (gathers && wb + r * 256 < len) gv[r] = buf_load<FRESH>(ub, (uint32_t)ci[r], (int64_t)(lane + r * 256) < len);
    __builtin_amdgcn_sched_barrier(0);
    load_unit_seg<R>(a, nxt, lane, ni, nv);
    nn = sa.units[p2 < n ? p2 : 0u];
    claim = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)K, qr, qoff, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (kind == SPLIT_SCATTER) {
        const uint32_t parts = split_parts(cur.info), idx = split_index(cur.info);
        if (lane < 64) {
            // Wave 0 waits for the coordinate's parts (GATHER units at - idx - parts + q) and sums them:
            // lane l holds parts l, l + 64, l + 128, l + 192, added in that order, then the butterfly.
            const uint64_t* slot = sa.partials + (at - idx - parts);
            uint32_t pv[4] = {0u, 0u, 0u, 0u};
            int ok = 1;
            for (uint32_t spins = 0;; ++spins) {
                bool have = true;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t q = (uint32_t)lane + 64u * t;
                    if (q < parts) {
                        const uint64_t v =
                            __hip_atomic_load(const_cast<uint64_t*>(slot + q), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        pv[t] = (uint32_t)v;
                        have = have && (uint32_t)(v >> 32) == sa.tag;
                    }
                }
                if (__all(have)) break;
                // Once any wait has given up, the others give up at their next check (every 256
                // sleeps, and before the first), so a failure costs one limit, not one per unit.
                const bool failed = (spins & 255u) == 0 &&
                                    __hip_atomic_load(sa.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
                if (spins >= sa.spin_limit || failed) {
                    ok = 0;
                    if (lane == 0) __hip_atomic_fetch_or(sa.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            float s = 0.0f;
#pragma unroll
            for (int t = 0; t < 4; ++t)
                if ((uint32_t)lane + 64u * t < parts) s += __builtin_bit_cast(float, pv[t]);
            s = group_sum<64>(s);
            if (lane == 0) {
                gsum[0] = s;
                gok[0] = ok;
            }
        }
        __syncthreads();
        if (gok[0]) {
            float coef;
            const float m_new = coord_step<FORM>(gsum[0], cur.sn, cur.m_old, cur.ylab, a.k, &coef);
            if (idx == 0) a.model[cur.m] = m_new;
            if (coef != 0.0f) {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (wb + r * 256 < len) split_atomic(ub, (uint32_t)ci[r], (int64_t)(lane + r * 256) < len, coef * cv[r]);
            }
        }
    } else {
        float acc = 0.0f;
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (wb + r * 256 < len) acc = fmaf(cv[r], gv[r], acc);
        const float g = pipe_reduce_256(acc, part, buf);
        if (kind == SPLIT_FULL) {
            float coef;
            const float m_new = coord_step<FORM>(g, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
            a.model[cur.m] = m_new;  // every lane stores the same value
            if (coef != 0.0f) {
#pragma unroll
                for (int r = 0; r < R; ++r)
                    if (wb + r * 256 < len) split_atomic(ub, (uint32_t)ci[r], (int64_t)(lane + r * 256) < len, coef * cv[r]);
            }
        } else if (lane == 0) {
            const uint64_t v = ((uint64_t)sa.tag << 32) | (uint64_t)__builtin_bit_cast(uint32_t, g);
            __hip_atomic_store(sa.partials + at, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    return p2;
}

template <int FORM, int R, bool FRESH, typename U>
__device__ __forceinline__ void epoch_split(const SplitArgs& sa) {
    __shared__ float part[2][4];
    __shared__ uint32_t ring[kSplitRing];
    __shared__ float gsum[1];
    __shared__ int gok[1];
    const EpochArgs& a = sa.e;
    const int lane = threadIdx.x;
    const uint32_t n = sa.n_units;
    const uint32_t K = a.chunk;
    // word 3 = 0x00020000: 32-bit data format, the gfx9-family raw-buffer setting.
    const __amdgpu_buffer_rsrc_t qr = __builtin_amdgcn_make_buffer_rsrc(a.queue, (short)0, 4, 0x00020000);
    // The chunks that cover steps [0, kSplitLead): the steps' own claims start with the next one.
    const uint32_t first = (kSplitLead + K - 1) / K;  // 1..kSplitLead
    uint32_t c[kSplitLead];
#pragma unroll
    for (int i = 0; i < kSplitLead; ++i)
        c[i] = (uint32_t)__builtin_amdgcn_raw_ptr_buffer_atomic_add_i32((int)K, qr, lane == 0 && (uint32_t)i < first ? 0 : 4,
                                                                         0, 0);
    if (lane == 0) {
        // Claims of one lane on one address are performed in order; sort anyway.
#pragma unroll
        for (int i = 1; i < kSplitLead; ++i)
#pragma unroll
            for (int t = kSplitLead - 1; t >= i; --t)
                if ((uint32_t)t < first && c[t] < c[t - 1]) {
                    const uint32_t x = c[t];
                    c[t] = c[t - 1];
                    c[t - 1] = x;
                }
#pragma unroll
        for (int i = 0; i < kSplitLead; ++i)
            if ((uint32_t)i < first) ring[i % kSplitRing] = c[i];
    }
    __syncthreads();
    uint32_t pA = split_pos(ring, 0, K), pB = split_pos(ring, 1, K);
    if (pA < n) {
        const SharedBuf<U> ub =
            shared_buf<U>(a.u, a.u_bytes, reinterpret_cast<U*>(a.sink) + (size_t)blockIdx.x * 256 + threadIdx.x,
                          a.u_shift);
        int buf = 0;
        uint32_t claim = 0, k = 0;
        SplitUnit cA = sa.units[pA];
        int ciA[R], ciB[R];
        float cvA[R], cvB[R];
        load_unit_seg<R>(a, cA, lane, ciA, cvA);
        SplitUnit cB = sa.units[pB < n ? pB : 0u];
        for (;;) {
            SplitUnit cA2, cB2;
            const uint32_t pA2 = split_step<FORM, R, FRESH>(sa, ub, qr, lane, k++, cA, pA, ciA, cvA, cB, ciB, cvB, cA2,
                                                            ring, claim, part, buf, gsum, gok);
            if (pB >= n) break;
            const uint32_t pB2 = split_step<FORM, R, FRESH>(sa, ub, qr, lane, k++, cB, pB, ciB, cvB, cA2, ciA, cvA, cB2,
                                                            ring, claim, part, buf, gsum, gok);
            if (pA2 >= n) break;
            cA = cA2;
            cB = cB2;
            pA = pA2;
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

// fp32 shared vector: at most 168 registers, so that three workgroups fit a CU (the window's
// workgroups are resident at once up to 768).  The fp64 variant needs more and keeps two.
template <int FORM, int R, bool FRESH>
__global__ __launch_bounds__(256, 3) void k_epoch_split(SplitArgs sa) {
    epoch_split<FORM, R, FRESH, float>(sa);
}

template <int FORM, int R, bool FRESH>
__global__ __launch_bounds__(256) void k_epoch_split_f64(SplitArgs sa) {
    epoch_split<FORM, R, FRESH, double>(sa);
}

template <int FORM, bool FRESH, typename U>
hipError_t launch_split_typed(const SplitArgs& sa, int blocks, hipStream_t s) {
    if constexpr (sizeof(U) == 4)
        hipLaunchKernelGGL((k_epoch_split<FORM, kQueueSlices, FRESH>), dim3(blocks), dim3(256), 0, s, sa);
    else
        hipLaunchKernelGGL((k_epoch_split_f64<FORM, kQueueSlices, FRESH>), dim3(blocks), dim3(256), 0, s, sa);
    return hipGetLastError();
}

template <int FORM>
hipError_t launch_split_form(bool wide, bool fresh, const SplitArgs& sa, int blocks, hipStream_t s) {
    if (wide)
        return fresh ? launch_split_typed<FORM, true, double>(sa, blocks, s)
                     : launch_split_typed<FORM, false, double>(sa, blocks, s);
    return fresh ? launch_split_typed<FORM, true, float>(sa, blocks, s)
                 : launch_split_typed<FORM, false, float>(sa, blocks, s);
}

}  // namespace

hipError_t launch_split_total(const int64_t* ptr, uint32_t C, uint32_t part, unsigned long long* out, hipStream_t s) {
    if (hipError_t e = launch_fill_zero(reinterpret_cast<uint64_t*>(out), 1u, s); e != hipSuccess) return e;
    hipLaunchKernelGGL(k_split_total, dim3(grid_for(C)), dim3(256), 0, s, ptr, C, part, out);
    return hipGetLastError();
}

hipError_t launch_epoch_split(int form, bool wide, bool fresh, const SplitArgs& sa, uint32_t part,
                              uint32_t* tile_units, SplitUnit* units, int blocks, hipStream_t s) {
    const uint32_t C = sa.e.perm.n;
    const uint32_t tiles = (uint32_t)(((uint64_t)C + kSplitPrepTile - 1) / kSplitPrepTile);
    hipLaunchKernelGGL(k_split_count, dim3(tiles), dim3(256), 0, s, sa.e.ptr, sa.e.perm, part, tile_units);
    hipLaunchKernelGGL(k_split_scan, dim3(1), dim3(1024), 0, s, tile_units, tiles);
    hipLaunchKernelGGL(k_split_write, dim3(tiles), dim3(256), 0, s, sa.e, part, tile_units, units);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    switch (form) {
        case FORM_RIDGE_PRIMAL: return launch_split_form<FORM_RIDGE_PRIMAL>(wide, fresh, sa, blocks, s);
        case FORM_SVM_DUAL: return launch_split_form<FORM_SVM_DUAL>(wide, fresh, sa, blocks, s);
        case FORM_RIDGE_DUAL: return launch_split_form<FORM_RIDGE_DUAL>(wide, fresh, sa, blocks, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace scd
