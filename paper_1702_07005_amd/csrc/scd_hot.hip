// scd_hot.hip -- the hot-set epoch kernel for gfx950 (windows of at most 8 coordinates: the
// most-updated shared-vector entries in LDS, one consumer wave, producer waves) and the set-up
// that chooses the hot set and each stored entry's slot.
#include "scd_device.h"

namespace scd {

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
    return (size_t)hot_bytes + kHotFlagBytes + kHotScratchBytes +
           (size_t)kHotProducers * (5u * B + 3u * B * Smax) * sizeof(uint32_t);
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

// One step of the consumer: W coordinates, 8 lanes each.  Reads the hot values the keys of `cur`
// point at, then the metadata and entries of the next step into `nxt` (the last step of a batch
// re-reads its own), then reduces, steps and scatters.  The plain LDS writes are issued by every
// lane (an inactive group writes into its own slots of `scr`), so only the hot-entry atomics sit
// behind a branch: a coordinate whose step is zero (in the SVM dual, most of them once their alpha
// sits at a bound) issues none.
template <int FORM, typename U, int SL>
__device__ __forceinline__ void hot_step(const EpochArgs& a, U* hot, uint32_t* mb, const int32_t* key,
                                         const float* val, float* coldw, float* scr, uint32_t B,
                                         uint32_t Smax, uint32_t cn, bool act, uint32_t sub, int lane,
                                         const HotStep<SL>& cur, uint32_t c, HotStep<SL>& nxt) {
    U hv[SL];
#pragma unroll
    for (int r = 0; r < SL; ++r) hv[r] = hot[cur.kk[r] >= 0 ? cur.kk[r] : 0];
    __builtin_amdgcn_sched_barrier(0);
    hot_load_step<SL>(nxt, mb, key, val, coldw, B, cn, cn * Smax + sub, act);
    __builtin_amdgcn_sched_barrier(0);
    float acc = 0.0f;
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        // Padding entries have value 0; a cold entry's value came with it.
        const float x = cur.kk[r] >= 0 ? (float)hv[r] : cur.xv[r];
        acc = fmaf(cur.vv[r], x, acc);
    }
    const float gsum = group_sum<8>(acc);
    float coef;
    const float m_new = coord_step<FORM>(gsum, cur.sn, cur.m_old, cur.ylab, a.k, &coef);
    // The model value and the updates go into this coordinate's batch slots (an empty position at
    // the end of the epoch has m = EMPTY and zero values, which the flush skips).
    const uint32_t e0 = c * Smax + sub;
    uint32_t* const mw = act ? mb + 2u * B + c : reinterpret_cast<uint32_t*>(scr + lane);
    *mw = __float_as_uint(m_new);
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        const float d = coef * cur.vv[r];
        float* const cw = act ? coldw + e0 + 8 * r : scr + lane;
        *cw = d;  // read back only for cold entries
        if (act && cur.kk[r] >= 0 && sub + 8u * r < cur.len && coef != 0.0f) atomicAdd(hot + cur.kk[r], (U)d);
    }
}

// The consumer for coordinates of at most 8 * SL entries: the steps of each batch, unrolled twice
// so that the two step records alternate instead of being copied (a copy would wait for the
// prefetch).  Hot entries are updated in LDS; the new model value and each cold entry's update go
// back into the batch buffer, and the producer that owns it issues the global stores and atomics
// before refilling it, so this wave never waits on global memory.
template <int FORM, typename U, int SL>
__device__ __forceinline__ void hot_consumer(const HotArgs& h, U* hot, uint32_t* ready, uint32_t* freed,
                                             uint32_t* abort_flag, uint32_t* bufs, float* scr, uint32_t nb,
                                             int lane) {
    const EpochArgs& a = h.e;
    const uint32_t B = h.B, Smax = h.Smax, W = h.W, buf_words = 5u * B + 3u * B * Smax, S = B / W;
    const uint32_t g = (uint32_t)lane >> 3, sub = (uint32_t)lane & 7u;
    const bool act = g < W;
    const uint32_t g0 = act ? g : 0u;  // inactive lanes read coordinate 0 of each step and write nothing
    for (uint32_t b = 0; b < nb; ++b) {
        const uint32_t p = b % kHotProducers, n = b / kHotProducers;
        if (!hot_wait(ready + p, n + 1, abort_flag, h.spin_limit, h.err)) return;
        uint32_t* const mb = bufs + p * buf_words;
        const int32_t* key = reinterpret_cast<const int32_t*>(mb + 5u * B);
        const float* val = reinterpret_cast<const float*>(key + B * Smax);
        float* const coldw = const_cast<float*>(val + B * Smax);
        HotStep<SL> sa, sb;
        hot_load_step<SL>(sa, mb, key, val, coldw, B, g0, g0 * Smax + sub, act);
        uint32_t st = 0;
        for (; st + 1 < S; st += 2) {
            const uint32_t c0 = st * W + g0, c1 = c0 + W;
            const uint32_t c2 = st + 2 < S ? c1 + W : c1;
            hot_step<FORM, U, SL>(a, hot, mb, key, val, coldw, scr, B, Smax, c1, act, sub, lane, sa, c0, sb);
            hot_step<FORM, U, SL>(a, hot, mb, key, val, coldw, scr, B, Smax, c2, act, sub, lane, sb, c1, sa);
        }
        if (st < S) {
            const uint32_t c0 = st * W + g0;
            hot_step<FORM, U, SL>(a, hot, mb, key, val, coldw, scr, B, Smax, c0, act, sub, lane, sa, c0, sb);
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
    float* const scr = reinterpret_cast<float*>(hot_lds + h.hot_bytes + kHotFlagBytes);  // 64 floats
    uint32_t* const bufs = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes + kHotFlagBytes + kHotScratchBytes);
    static_assert((2 * kHotProducers + 1) * sizeof(uint32_t) <= kHotFlagBytes, "handover words exceed their area");
    U* const uu = static_cast<U*>(a.u);
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    for (uint32_t i = tid; i < h.n_hot; i += blockDim.x) hot[i] = uu[h.hot_ids[i]];
    if (tid < 2 * kHotProducers + 1) ready[tid] = 0u;  // ready, freed and abort are contiguous
    __syncthreads();
    const uint32_t nb = (a.perm.n + h.B - 1) / h.B;
    if (wave == 0) {
        switch (h.Smax / 8) {  // entries per consumer lane
            case 1: hot_consumer<FORM, U, 1>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 2: hot_consumer<FORM, U, 2>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 3: hot_consumer<FORM, U, 3>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 4: hot_consumer<FORM, U, 4>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 5: hot_consumer<FORM, U, 5>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 6: hot_consumer<FORM, U, 6>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            case 7: hot_consumer<FORM, U, 7>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
            default: hot_consumer<FORM, U, 8>(h, hot, ready, freed, abort_flag, bufs, scr, nb, lane); break;
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
