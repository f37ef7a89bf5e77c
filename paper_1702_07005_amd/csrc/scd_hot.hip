// scd_hot.hip -- the hot-set epoch kernel for gfx950 (windows of at most 16 coordinates: the
// most-updated shared-vector entries in LDS, one or two consumer waves, producer waves) and the
// set-up that chooses the hot set and each stored entry's slot.
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
// Waves 0..NC-1 (the consumers, NC = 1 to 4) run the in-flight coordinates, 8 lanes each and at
// most kHotMaxGroups per wave, and read nothing but LDS; batch b goes to consumer b mod NC, and
// each consumer steps through its batches independently of the others (their hot-entry updates
// meet in LDS atomics).  The other NP = kHotWaves - NC waves (producers) fill per-producer LDS
// buffers with the next batches of permutation positions: each coordinate's metadata and, per
// stored entry, its value and either its hot slot or (cold entry) its index and current
// shared-vector value.  Each wave has its own completion counter, so the producers' load latency
// never stalls a consumer.
//
// Adaptive window.  Only coordinates whose step is nonzero change the shared vector, so only they
// make the reads of the others stale.  When the window is automatic, each epoch counts the
// coordinates that moved and sets the next epoch's window so that the expected number of moving
// coordinates in flight stays at what the coupling rule allows: W = 1 + (w_rule - 1) / f, f the
// fraction that moved (in the hinge SVM dual most coordinates sit at a bound of the box and do not
// move).  The first epoch after the state or the options changed opens with a launch over its
// first 1/kHotOpening of the positions at w_rule and runs the rest at the window that opening gives;
// the window lives in device memory, so the epochs of one call need no synchronisation with the host.
// The producers read cold values up to a few batches before their coordinate runs; cold entries are
// by construction rarely updated, so such a read seldom misses an update.
// Producer and consumer hand buffers over through LDS sequence numbers; every wait is bounded
// (spin_limit sleeps), after which the wave sets *err and all waves leave.
// ----------------------------------------------------------------------------------------
size_t hot_lds_bytes(uint32_t hot_bytes, uint32_t cap, uint32_t Smax) {
    return (size_t)hot_bytes + kHotFlagBytes + kHotScratchBytes +
           (size_t)kHotMaxProducers * hot_buf_words(cap, Smax) * sizeof(uint32_t);
}

size_t staged_lds_bytes(uint32_t hot_bytes, uint32_t cap, uint32_t Smax) {
    const size_t stager = (size_t)kHotWaves * hot_buf_words(cap, Smax) * sizeof(uint32_t) + 16;
    const size_t hot = hot_lds_bytes(hot_bytes, cap, Smax);
    return hot > stager ? hot : stager;
}

// A value that is the same in every lane of the wave (a wave's index, a word that every lane read
// from one address), marked so: the compiler then keeps it in a scalar register and branches on it
// with scalar branches instead of execution masks.
__device__ __forceinline__ uint32_t wave_uniform(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

__device__ __forceinline__ bool hot_wait(uint32_t* flag, uint32_t want, uint32_t* abort_flag, uint32_t limit,
                                         int* err) {
    uint32_t spins = 0;
    for (;;) {
        if (wave_uniform(__hip_atomic_load(flag, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP)) == want) return true;
        if (wave_uniform(__hip_atomic_load(abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP))) return false;
        if (++spins > limit) {
            __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// One batch buffer in LDS (room for cap coordinates of Smax entry slots each; 32-bit words, 16-byte
// aligned).  The layout depends on cap only, so batches of different sizes share it.
struct HotBuf {
    float4* rec;    // [B]: model value, step scale, label or <y, a_m>, cold part of the gathered dot;
                    // the consumer then overwrites .z and .w with the new model value and the
                    // scatter coefficient
    int2* kv;       // [B * Smax]: key and value bits of each entry slot.  A hot entry's key is its
                    // slot in the hot array; a cold or padding slot has value 0 and the key of the
                    // zero cell of the consumer lane that takes it (hot array slot n_hot + lane).
    uint32_t* mid;  // [B]: coordinate index, or kHotEmpty for positions past the end of the epoch
};

__device__ __forceinline__ HotBuf hot_buf(uint32_t* base, uint32_t cap, uint32_t Smax) {
    HotBuf b;
    b.rec = reinterpret_cast<float4*>(base);
    b.kv = reinterpret_cast<int2*>(base + 4u * cap);
    b.mid = base + 4u * cap + 2u * cap * Smax;
    return b;
}

constexpr uint32_t kHotEmpty = 0xFFFFFFFFu;

// The closed-form steps of coord_step with each coordinate's divisor folded into a scale that the
// producer computes (so the consumer's step has no division):
//   ridge primal  sc = 1 / (|a_m|^2 + lambda N)      d = (<y, a_m> - g - lambda N beta_m) sc
//   SVM dual      sc = lambda N / |x_i|^2, -1 if 0    alpha_i <- clip(alpha_i + sc (1 - y_i g), 0, 1)
//   ridge dual    sc = 1 / (lambda N + |abar_n|^2)   d = (lambda y_n - g - lambda N alpha_n) sc
template <int FORM>
__device__ __forceinline__ float hot_step_scale(float s, const StepConsts& k) {
    if constexpr (FORM == FORM_SVM_DUAL)
        return s > 0.0f ? k.lamN / s : -1.0f;
    else
        return 1.0f / (s + k.lamN);
}

template <int FORM>
__device__ __forceinline__ float hot_coord_step(float g, float m_old, float sc, float ylab, const StepConsts& k,
                                                float* coef) {
    if constexpr (FORM == FORM_RIDGE_PRIMAL) {
        const float d = ((ylab - g) - k.lamN * m_old) * sc;
        *coef = d;
        return m_old + d;
    } else if constexpr (FORM == FORM_SVM_DUAL) {
        // An empty row (sc < 0): the dual is linear in alpha_i with positive slope, so alpha_i = 1.
        const float a = sc < 0.0f ? 1.0f : fminf(fmaxf(m_old + sc * (1.0f - ylab * g), 0.0f), 1.0f);
        *coef = (a - m_old) * ylab * k.inv_lamN;
        return a;
    } else {
        const float d = (k.lam * ylab - g - k.lamN * m_old) * sc;
        *coef = d;
        return m_old + d;
    }
}

// One step's worth of a batch buffer for a consumer lane: the coordinate's record and the lane's SL
// entry slots (key, value).
template <int SL>
struct HotStep {
    float4 r;
    int32_t kk[SL];
    float vv[SL];
};

template <int SL>
__device__ __forceinline__ void hot_load_step(HotStep<SL>& t, const HotBuf& hb, uint32_t c, uint32_t e0) {
    t.r = hb.rec[c];
#pragma unroll
    for (int r = 0; r < SL; ++r) {
        const int2 p = hb.kv[e0 + 8 * r];
        t.kk[r] = p.x;
        t.vv[r] = __int_as_float(p.y);
    }
}

// One step of the consumer: W coordinates, 8 lanes each.  Reads the hot values the keys of `cur`
// point at, then the record and entries of the next step into `nxt` (the last step of a batch
// re-reads its own), then reduces (hot part plus the producer's cold part), steps and scatters.
// The new model value and the scatter coefficient go back into the coordinate's record (one write,
// issued by every lane; an inactive group writes into its own cells of `scr`); the producer forms
// the cold entries' updates from the coefficient when it writes the batch out.  The LDS atomics sit
// behind one branch per step, taken by the groups whose step is nonzero (in the SVM dual, once their
// alpha sits at a bound, most coordinates do not move).  A cold or padding slot reads its lane's
// zero cell and adds coef * 0 to it, so no slot needs a select.
template <int FORM, typename U, int SL>
__device__ __forceinline__ void hot_step(const StepConsts& k, U* hot, const HotBuf& hb, float* scr, uint32_t Smax,
                                         uint32_t cn, bool act, uint32_t sub, int lane, const HotStep<SL>& cur,
                                         uint32_t c, HotStep<SL>& nxt) {
    U hv[SL];
#pragma unroll
    for (int r = 0; r < SL; ++r) hv[r] = hot[cur.kk[r]];
    __builtin_amdgcn_sched_barrier(0);
    hot_load_step<SL>(nxt, hb, cn, __umul24(cn, Smax) + sub);
    __builtin_amdgcn_sched_barrier(0);
    float acc = 0.0f;
#pragma unroll
    for (int r = 0; r < SL; ++r) acc = fmaf(cur.vv[r], (float)hv[r], acc);
    const float gsum = group_sum<8>(acc) + cur.r.w;
    float coef;
    const float m_new = hot_coord_step<FORM>(gsum, cur.r.x, cur.r.y, cur.r.z, k, &coef);
    if (!act) coef = 0.0f;
    // (An empty position at the end of the epoch has kHotEmpty as its index, which the flush skips.)
    *reinterpret_cast<float2*>(act ? &hb.rec[c].z : scr + 2 * lane) = make_float2(m_new, coef);
    if (coef != 0.0f) {
#pragma unroll
        for (int r = 0; r < SL; ++r) atomicAdd(hot + cur.kk[r], (U)(coef * cur.vv[r]));
    }
}

// Consumer `ci` for coordinates of at most 8 * SL entries: the steps of each of its batches, unrolled
// twice so that the two step records alternate instead of being copied (a copy would wait for the
// prefetch).  Hot entries are updated in LDS; the new model value and the coefficient go back into
// the batch buffer, and the producer that owns it issues the global stores and atomics before
// refilling it, so this wave never waits on global memory.
template <int FORM, typename U, int SL>
__device__ __forceinline__ void hot_consumer(const HotArgs& h, const HotSched& sc, uint32_t ci, U* hot,
                                             uint32_t* ready, uint32_t* freed, uint32_t* abort_flag, uint32_t* bufs,
                                             float* scr, int lane) {
    const StepConsts k = h.e.k;
    // The instance for rows of Smax entries has SL = Smax / 8 (the host picks it so): Smax is a
    // compile-time constant, so the slot range tests fold and the slot offsets need no 32-bit multiply.
    constexpr uint32_t Smax = 8u * SL;
    const uint32_t W = hot_groups(sc, ci), B = hot_batch(sc, ci), bw = hot_buf_words(h.cap, Smax);
    const uint32_t S = B / W;
    const uint32_t g = (uint32_t)lane >> 3, sub = (uint32_t)lane & 7u;
    const bool act = g < W;
    const uint32_t g0 = act ? g : 0u;  // inactive lanes read coordinate 0 of each step and write nothing
    float* const my_scr = scr + ci * 128u;
    // The consumers set the epoch's pace; each shares its SIMD with two or three producer waves, so it
    // takes the highest issue priority (2% of the full click epoch).
    __builtin_amdgcn_s_setprio(3);
    for (uint32_t b = ci; b < sc.nb; b += sc.NC) {
        const uint32_t p = b % sc.NP, n = b / sc.NP;
        if (!hot_wait(ready + p, n + 1, abort_flag, h.spin_limit, h.err)) return;
        const HotBuf hb = hot_buf(bufs + p * bw, h.cap, Smax);
        HotStep<SL> sa, sb;
        hot_load_step<SL>(sa, hb, g0, g0 * Smax + sub);
        uint32_t st = 0;
        for (; st + 1 < S; st += 2) {
            const uint32_t c0 = st * W + g0, c1 = c0 + W;
            const uint32_t c2 = st + 2 < S ? c1 + W : c1;
            hot_step<FORM, U, SL>(k, hot, hb, my_scr, Smax, c1, act, sub, lane, sa, c0, sb);
            hot_step<FORM, U, SL>(k, hot, hb, my_scr, Smax, c2, act, sub, lane, sb, c1, sa);
        }
        if (st < S) {
            const uint32_t c0 = st * W + g0;
            hot_step<FORM, U, SL>(k, hot, hb, my_scr, Smax, c0, act, sub, lane, sa, c0, sb);
        }
        __hip_atomic_store(freed + p, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

// The same consumer with 16 lanes per coordinate, for consumers of at most 4 coordinates per step
// (the adaptive plans with three or four consumers): 4 coordinates fill the wave, each lane holds
// SL2 = ceil(Smax / 16) entry slots (slot sub + 16 r of its coordinate), so a step issues fewer LDS
// gathers and atomics per lane and sums over 16 lanes.  The batch image is the one the 8-lane
// consumer reads; a lane's slots past Smax read its own zero cell (hot array slot n_hot + lane).
// Only the first lane of a coordinate writes its record back (the others write into `scr`).
template <int SL2>
__device__ __forceinline__ void hot_load_step16(HotStep<SL2>& t, const HotBuf& hb, uint32_t c, uint32_t Smax,
                                                uint32_t sub, int32_t zkey) {
    t.r = hb.rec[c];
#pragma unroll
    for (int r = 0; r < SL2; ++r) {
        const uint32_t k = sub + 16u * (uint32_t)r;
        const bool in = k < Smax;
        const int2 p = hb.kv[__umul24(c, Smax) + (in ? k : 0u)];
        t.kk[r] = in ? p.x : zkey;
        t.vv[r] = in ? __int_as_float(p.y) : 0.0f;
    }
}

template <int FORM, typename U, int SL2>
__device__ __forceinline__ void hot_step16(const StepConsts& k, U* hot, const HotBuf& hb, float* scr, uint32_t Smax,
                                           uint32_t cn, bool act, uint32_t sub, int lane, int32_t zkey,
                                           const HotStep<SL2>& cur, uint32_t c, HotStep<SL2>& nxt) {
    U hv[SL2];
#pragma unroll
    for (int r = 0; r < SL2; ++r) hv[r] = hot[cur.kk[r]];
    __builtin_amdgcn_sched_barrier(0);
    hot_load_step16<SL2>(nxt, hb, cn, Smax, sub, zkey);
    __builtin_amdgcn_sched_barrier(0);
    float acc = 0.0f;
#pragma unroll
    for (int r = 0; r < SL2; ++r) acc = fmaf(cur.vv[r], (float)hv[r], acc);
    const float gsum = group_sum<16>(acc) + cur.r.w;
    float coef;
    const float m_new = hot_coord_step<FORM>(gsum, cur.r.x, cur.r.y, cur.r.z, k, &coef);
    if (!act) coef = 0.0f;
    *reinterpret_cast<float2*>(act && sub == 0 ? &hb.rec[c].z : scr + 2 * lane) = make_float2(m_new, coef);
    if (coef != 0.0f) {
#pragma unroll
        for (int r = 0; r < SL2; ++r) atomicAdd(hot + cur.kk[r], (U)(coef * cur.vv[r]));
    }
}

template <int FORM, typename U, int SL2, int SL>
__device__ __forceinline__ void hot_consumer16(const HotArgs& h, const HotSched& sc, uint32_t ci, U* hot,
                                               uint32_t* ready, uint32_t* freed, uint32_t* abort_flag, uint32_t* bufs,
                                               float* scr, int lane) {
    const StepConsts k = h.e.k;
    constexpr uint32_t Smax = 8u * SL;  // as in hot_consumer
    const uint32_t W = hot_groups(sc, ci), B = hot_batch(sc, ci), bw = hot_buf_words(h.cap, Smax);
    const uint32_t S = B / W;
    const uint32_t g = (uint32_t)lane >> 4, sub = (uint32_t)lane & 15u;
    const bool act = g < W;
    const uint32_t g0 = act ? g : 0u;  // inactive lanes read coordinate 0 of each step and write nothing
    const int32_t zkey = (int32_t)(h.n_hot + (uint32_t)lane);
    float* const my_scr = scr + ci * 128u;
    __builtin_amdgcn_s_setprio(3);  // as in hot_consumer
    for (uint32_t b = ci; b < sc.nb; b += sc.NC) {
        const uint32_t p = b % sc.NP, n = b / sc.NP;
        if (!hot_wait(ready + p, n + 1, abort_flag, h.spin_limit, h.err)) return;
        const HotBuf hb = hot_buf(bufs + p * bw, h.cap, Smax);
        HotStep<SL2> sa, sb;
        hot_load_step16<SL2>(sa, hb, g0, Smax, sub, zkey);
        uint32_t st = 0;
        for (; st + 1 < S; st += 2) {
            const uint32_t c0 = st * W + g0, c1 = c0 + W;
            const uint32_t c2 = st + 2 < S ? c1 + W : c1;
            hot_step16<FORM, U, SL2>(k, hot, hb, my_scr, Smax, c1, act, sub, lane, zkey, sa, c0, sb);
            hot_step16<FORM, U, SL2>(k, hot, hb, my_scr, Smax, c2, act, sub, lane, zkey, sb, c1, sa);
        }
        if (st < S) {
            const uint32_t c0 = st * W + g0;
            hot_step16<FORM, U, SL2>(k, hot, hb, my_scr, Smax, c0, act, sub, lane, zkey, sa, c0, sb);
        }
        __hip_atomic_store(freed + p, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
}

// A producer's view of one batch: lane c < B loads coordinate c's metadata.  The coordinate index
// is computed first (arithmetic only) and the loads are issued later, so that they can be issued
// behind the previous batch's entry loads.
struct HotMeta {
    uint32_t m;  // coordinate, or kHotEmpty
    int64_t s0, s1;
    float m_old, sn, ylab;
};

__device__ __forceinline__ uint32_t hot_coord(const HotArgs& h, const HotSched& sc, uint32_t b, int lane) {
    if (b >= sc.nb || (uint32_t)lane >= hot_batch_size(sc, b)) return kHotEmpty;
    const uint32_t k = hot_batch_start(sc, b) + (uint32_t)lane;  // position within this launch's range
    return k < h.pos_n ? perm_at(h.pos0 + k, h.e.perm) : kHotEmpty;
}

__device__ __forceinline__ void hot_meta_load(const EpochArgs& a, HotMeta& t) {
    const uint32_t mm = t.m != kHotEmpty ? t.m : 0u;  // the loads always hit a valid coordinate
    t.s0 = a.ptr[mm];
    t.s1 = a.ptr[mm + 1];
    t.m_old = a.model[mm];
    t.sn = a.norms[mm];
    t.ylab = a.y[mm];
}

// Raw-buffer load of a shared-vector entry, kept in its storage type; a lane with `in` false
// reads at an out-of-range offset (0, no memory traffic).  Branch-free, so the compiler's count of
// the memory operations behind an earlier load stays exact.
template <typename U>
__device__ __forceinline__ U hot_load_u(const SharedBuf<U>& b, uint32_t i, bool in) {
    const uint32_t off = in ? i << b.shift : b.oob;
    if constexpr (sizeof(U) == 4)
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(b.r, (int)off, 0, 0));
    else
        return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(b.r, (int)off, 0, 0));
}

// Producer wave q fills buffer q with batches q, q + NP, ...  (NP is a multiple of NC, so the batches
// of one buffer all go to the same consumer and have the same size.)  Slot e = t * 64 + lane of a
// batch holds entry e % Smax of coordinate e / Smax; since Smax is a multiple of 8, each aligned
// group of 8 lanes holds entries of one coordinate.  Per slot the producer loads the entry's key
// (hot slot or index, precomputed for every stored entry) and value, and a cold entry's
// shared-vector value; it writes the key and value of hot entries, and adds each coordinate's cold
// part of the dot (value times shared-vector value over its cold entries) into its record.  It is software-pipelined: the metadata of its next batch
// is loaded while this batch's entries are in flight, and the consumed batch it replaces is read out
// of LDS before the new one is written in and written out to global memory (new model values,
// device-scope atomics for the cold entries' updates) after, so that no wait for this batch's loads
// also waits for those stores and atomics.  The cold entries' indices and values stay in registers
// until that write-out.
// Adds to *moved_total the coordinates of its batches whose step was nonzero.
template <int FORM, typename U>
__device__ __forceinline__ void hot_producer(const HotArgs& h, const HotSched& sc, uint32_t* ready, uint32_t* freed,
                                             uint32_t* abort_flag, uint32_t* bufs, uint32_t* moved_total, int q,
                                             int lane) {
    const EpochArgs& a = h.e;
    U* const uu = static_cast<U*>(a.u);
    const SharedBuf<U> ub = shared_buf<U>(a.u, a.u_bytes, nullptr, a.u_shift);
    const uint32_t Smax = h.Smax, nb = sc.nb, NP = sc.NP;
    // Every batch of this buffer goes to consumer q mod NC and has that consumer's size.
    const uint32_t B = hot_batch(sc, hot_consumer_of(sc, (uint32_t)q)), NB = B * Smax;
    const HotBuf hb = hot_buf(bufs + q * hot_buf_words(h.cap, Smax), h.cap, Smax);
    constexpr int NE = kHotEntriesPerLane;
    const uint32_t c0 = (uint32_t)lane / Smax, k0 = (uint32_t)lane - c0 * Smax;
    const uint32_t dc = 64u / Smax, dk = 64u - dc * Smax;
    HotMeta md;
    md.m = hot_coord(h, sc, (uint32_t)q, lane);
    uint32_t moved = 0;  // this lane's coordinates whose step was nonzero
    hot_meta_load(a, md);
    int32_t fl_ix[NE];  // the buffer's current batch: cold entries' indices and values (0: none)
    float fl_v[NE];
#pragma unroll
    for (int t = 0; t < NE; ++t) {
        fl_ix[t] = 0;
        fl_v[t] = 0.0f;
    }
    for (uint32_t b = (uint32_t)q; b < nb + NP; b += NP) {
        const uint32_t n = b / NP;
        int32_t ky[NE];  // entry key: -1 - hot slot, or the shared-vector index of a cold entry
        float vv[NE];
        bool in[NE];
        float part[NE];  // cold part of the dot, summed over each aligned group of 8 lanes
        HotMeta nx;
        nx.m = hot_coord(h, sc, b + NP, lane);
        if (b < nb) {
            // Entries (entry 0 stands in for unused slots): key and value.
            const uint32_t len = md.m != kHotEmpty ? (uint32_t)(md.s1 - md.s0) : 0u;
            uint32_t c = c0, k = k0;
#pragma unroll
            for (int t = 0; t < NE; ++t) {
                const uint32_t cc = c < B ? c : 0u;
                const int64_t sc = __shfl(md.s0, (int)cc);
                const uint32_t lc = (uint32_t)__shfl((int)len, (int)cc);
                in[t] = c < B && k < lc;
                const int64_t kk = in[t] ? sc + k : 0;
                ky[t] = h.entry_key[kk];
                vv[t] = a.val[kk];
                c += dc;
                k += dk;
                if (k >= Smax) {
                    k -= Smax;
                    ++c;
                }
            }
            hot_meta_load(a, nx);
            // Only cold entries need their shared-vector value.  Their products are summed per
            // coordinate here, before the wait for the buffer (the loaded values are needed nowhere
            // else, and holding them would take two registers each for an fp64 shared vector).
            U cv[NE];
#pragma unroll
            for (int t = 0; t < NE; ++t) cv[t] = hot_load_u<U>(ub, (uint32_t)ky[t], in[t] && ky[t] >= 0);
#pragma unroll
            for (int t = 0; t < NE; ++t) part[t] = group_sum<8>(vv[t] * (float)cv[t]);
        }
        // The buffer's previous batch (if any) must have been consumed.
        if (n > 0 || b < nb) {
            if (!hot_wait(freed + q, n, abort_flag, h.spin_limit, h.err)) break;
        }
        // Read out the consumed batch: new model values, and each cold entry's update (the
        // coordinate's coefficient times the entry's value, the product the consumer formed for
        // its hot entries).
        uint32_t old_m = kHotEmpty;
        float old_model = 0.0f;
        float old_d[NE];
        if (n > 0) {
            if ((uint32_t)lane < B) {
                old_m = hb.mid[lane];
                const float2 zw = *reinterpret_cast<const float2*>(&hb.rec[lane].z);
                old_model = zw.x;
                moved += (old_m != kHotEmpty && zw.y != 0.0f) ? 1u : 0u;
            }
            uint32_t c = c0, k = k0;
#pragma unroll
            for (int t = 0; t < NE; ++t) {
                old_d[t] = c < B ? hb.rec[c].w * fl_v[t] : 0.0f;
                c += dc;
                k += dk;
                if (k >= Smax) {
                    k -= Smax;
                    ++c;
                }
            }
        }
        int32_t old_ix[NE];
#pragma unroll
        for (int t = 0; t < NE; ++t) old_ix[t] = fl_ix[t];
        if (b < nb) {
            if ((uint32_t)lane < B) {
                hb.mid[lane] = md.m;
                hb.rec[lane] = make_float4(md.m_old, hot_step_scale<FORM>(md.sn, a.k), md.ylab, 0.0f);
            }
            uint32_t c = c0, k = k0;
#pragma unroll
            for (int t = 0; t < NE; ++t) {
                const uint32_t e = (uint32_t)t * 64u + (uint32_t)lane;
                const bool hot = in[t] && ky[t] < 0;
                const bool cold = in[t] && ky[t] >= 0;
                if (e < NB) {
                    // The consumer lane of this slot is (c mod W) * 8 + k mod 8; the W coordinates
                    // of one step are consecutive, so c mod 8 tells them apart just as well.
                    const uint32_t zlane = ((c & 7u) << 3) | (k & 7u);
                    hb.kv[e] = make_int2(hot ? -1 - ky[t] : (int32_t)(h.n_hot + zlane),
                                         __float_as_int(hot ? vv[t] : 0.0f));
                    // Added into the coordinate's record (rec.w starts at 0, written above by this wave).
                    if ((lane & 7) == 0 && part[t] != 0.0f) atomicAdd(&hb.rec[c].w, part[t]);
                }
                fl_ix[t] = ky[t];
                fl_v[t] = cold ? vv[t] : 0.0f;
                c += dc;
                k += dk;
                if (k >= Smax) {
                    k -= Smax;
                    ++c;
                }
            }
            __hip_atomic_store(ready + q, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
        if (n > 0) {
            // Fire and forget.
            if (old_m != kHotEmpty) a.model[old_m] = old_model;
#pragma unroll
            for (int t = 0; t < NE; ++t)
                if (old_d[t] != 0.0f) atomic_add_u(uu + old_ix[t], old_d[t]);
        }
        if (b >= nb) break;
        md = nx;
    }
    for (int o = 32; o > 0; o >>= 1) moved += __shfl_xor(moved, o, 64);
    if (lane == 0) atomicAdd(moved_total, moved);
}

// SL: entries per consumer lane (Smax / 8), a template parameter so that each instance holds one
// consumer variant.
template <int FORM, typename U, int SL>
__global__ __launch_bounds__(64 * kHotWaves) void k_epoch_hot(HotArgs h) {
    extern __shared__ __align__(16) unsigned char hot_lds[];
    const EpochArgs& a = h.e;
    U* const hot = reinterpret_cast<U*>(hot_lds);
    uint32_t* const ready = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes);
    uint32_t* const freed = ready + kHotMaxProducers;
    uint32_t* const abort_flag = freed + kHotMaxProducers;
    uint32_t* const moved = abort_flag + 1;
    // Scratch: write targets of inactive consumer lanes (128 floats per consumer).  The hot array ends
    // with kHotZeroCells zero cells (one per consumer lane) that cold and padding slots point at.
    float* const scr = reinterpret_cast<float*>(hot_lds + h.hot_bytes + kHotFlagBytes);
    uint32_t* const bufs = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes + kHotFlagBytes + kHotScratchBytes);
    static_assert((2 * kHotMaxProducers + 2) * sizeof(uint32_t) <= kHotFlagBytes, "handover words exceed their area");
    static_assert((kHotWaves - 3) % 3 == 0 && (kHotWaves - 4) % 4 == 0 && (kHotWaves - 2) % 2 == 0,
                  "a buffer's batches must share a consumer");
    U* const uu = static_cast<U*>(a.u);
    const int tid = threadIdx.x, wave = (int)wave_uniform((uint32_t)tid >> 6), lane = tid & 63;
    // This launch's window: fixed, or set by the previous launch of the adaptive plan (and then run by
    // as many consumers as keep two coordinates each per step, up to four).
    uint32_t W = h.W, NC = h.NC;
    if (h.adapt_in) {
        const uint32_t v = __hip_atomic_load(h.adapt_in, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v >= 2 && v <= (uint32_t)kHotMaxWindow) W = v;
    }
    if (h.adapt_out) NC = hot_adaptive_consumers(W);
    const HotSched sc = hot_sched(W, NC, h.cap, h.pos_n);
    for (uint32_t i = tid; i < h.n_hot + kHotZeroCells; i += blockDim.x) hot[i] = i < h.n_hot ? uu[h.hot_ids[i]] : U(0);
    if (tid < 2 * kHotMaxProducers + 2) ready[tid] = 0u;  // ready, freed, abort and moved are contiguous
    __syncthreads();
    if ((uint32_t)wave < sc.NC) {
        if (sc.w_hi <= 4)
            hot_consumer16<FORM, U, (SL + 1) / 2, SL>(h, sc, (uint32_t)wave, hot, ready, freed, abort_flag, bufs, scr, lane);
        else
            hot_consumer<FORM, U, SL>(h, sc, (uint32_t)wave, hot, ready, freed, abort_flag, bufs, scr, lane);
    } else {
        hot_producer<FORM, U>(h, sc, ready, freed, abort_flag, bufs, moved, wave - (int)sc.NC, lane);
    }
    __syncthreads();
    for (uint32_t i = tid; i < h.n_hot; i += blockDim.x) uu[h.hot_ids[i]] = hot[i];
    // Next launch's window: (W - 1) f kappa <= budget with a fraction f of this launch's coordinates
    // moving, i.e. W = 1 + (w_rule - 1) / f, at most what the consumers hold.  A launch that gave up
    // keeps the window.
    if (h.adapt_out && tid == 0 && *abort_flag == 0u) {
        const uint64_t mv = *moved, wmax = kHotMaxWindow;
        uint64_t w = mv ? 1 + (uint64_t)(h.w_rule - 1) * h.pos_n / mv : wmax;
        w = w < h.w_rule ? h.w_rule : w > wmax ? wmax : w;
        __hip_atomic_store(h.adapt_out, (uint32_t)w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// ----------------------------------------------------------------------------------------
// Staged hot-set epoch (large matrices).  At full size the single workgroup's producer waves bound
// the epoch: each batch costs a producer wave about 1,400 instructions (slot layout, metadata,
// 64-bit entry addresses) and three dependent memory round trips, and one CU holds only twelve such
// waves (their registers).  Here that work runs on other CUs of workgroup 0's XCD:
//
//   stager waves (workgroups kHotXcds, 2 kHotXcds, ...): claim the next batch from a counter, wait
//     until its ring record is free, read the coordinates' metadata and entry keys and values,
//     gather the cold entries' shared-vector values, assemble the batch's LDS image in their own LDS
//     (records with each coordinate's cold part of the dot, hot keys and values, zero-cell keys for
//     cold slots) and copy it into the record; then wait until those stores have completed and
//     publish the record's tag (batch + 1).  A batch runs at most kHotRing + NP batches after its
//     stager read the cold values; cold entries are by construction rarely updated (an earlier
//     version gathered them in the loader, about NP batches ahead, at the same per-epoch gap
//     ratios and 6% more epoch time).
//   loader waves (workgroup 0, in place of the producers): once the consumer has finished the
//     buffer's previous batch, publish its results (each coordinate's new model value and scatter
//     coefficient) in a result ring; then take the record of the next batch (read ahead when its
//     tag was already set), copy it into the buffer, free the record and hand the buffer over.
//   The stager of a batch waits for its results and writes the model values and the cold entries'
//     updates out, so the hot-set workgroup never waits behind a device-scope atomic.
//
// A record is published by its stager's stores, a wait until they have completed, and the tag
// store; the loader polls the tag (system scope) and then, before it loads the record, drops every
// clean line the XCD's caches may hold (an agent-scope acquire: L1 and L2 invalidate).  Without
// that acquire (sc0 loads only, which the compiler's model treats as coherent between the CUs of
// one XCD) the loader now and then took some rows of a record stale: about one corrupted batch in
// 5-10 epochs of the full click workload, each row's model value stored while its update never
// reached the shared vector.  An L1 invalidate alone did not prevent it (3 of 3 runs corrupted);
// the acquire did (132 epochs without one, over the variants tried), at about 5% of the epoch
// time.  A full agent-scope release on the stager side (an L2 write-back per batch) doubled the
// epoch.  Each stager workgroup also acquires once when it starts, before it reads the metadata
// (the model values the previous epoch stored).  The stagers run on workgroup 0's XCD (hardware
// XCC_ID; the others leave), so the ring stays in one L2.  The flags are zeroed before every
// launch; every wait is bounded.
// ----------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t hot_xcc_id() {
    return (uint32_t)__builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20) & 15u;
}

// Ring, flags and results as raw buffers (byte offsets), shared by the CUs of one XCD: stores with sc0,
// polls volatile (system scope, re-read each time), record loads after an agent-scope acquire.
typedef int xcd_v2 __attribute__((ext_vector_type(2)));
typedef int xcd_v4 __attribute__((ext_vector_type(4)));
constexpr int kXcdLoad = 1;                    // sc0
constexpr int kXcdPoll = 1 | (int)(1u << 31);  // sc0, volatile
constexpr int kXcdStore = 1;                   // sc0

__device__ __forceinline__ __amdgpu_buffer_rsrc_t xcd_rsrc(const void* p, uint32_t bytes) {
    // word 3 = 0x00020000: 32-bit data format, the gfx9-family raw-buffer setting.
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ bool flag_wait(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t want, uint32_t limit,
                                          int* err) {
    for (uint32_t spins = 0;; ++spins) {
        if (wave_uniform((uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, kXcdPoll)) == want) return true;
        if (spins >= limit) {
            __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

__device__ __forceinline__ void flag_set(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t v) {
    __builtin_amdgcn_raw_buffer_store_b32((int)v, r, (int)off, 0, kXcdStore);
}

template <int FORM, typename U>
__device__ void staged_stager(const HotArgs& h, const HotSched& sc, uint32_t* lds) {
    const EpochArgs& a = h.e;
    const int lane = threadIdx.x & 63, wave = (int)wave_uniform(threadIdx.x >> 6);
    {
        uint32_t* const same_xcd_word = lds + (uint32_t)kHotWaves * hot_buf_words(h.cap, h.Smax);
        uint32_t& same_xcd = *same_xcd_word;
        if (threadIdx.x == 0) {
            uint32_t ok = 0;
            for (uint32_t spins = 0; spins < h.spin_limit; ++spins) {
                if (__hip_atomic_load(h.prog, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == h.tag) {
                    ok = __hip_atomic_load(h.prog + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == hot_xcc_id();
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
            same_xcd = ok;
        }
        __syncthreads();
        if (!same_xcd) return;
    }
    // Metadata written by the previous launch (model values) is read below: drop clean cached lines.
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    const SharedBuf<U> ub = shared_buf<U>(a.u, a.u_bytes, nullptr, a.u_shift);
    const uint32_t Smax = h.Smax, cap = h.cap, IW = hot_buf_words(cap, Smax), RW = staged_rec_words(cap, Smax);
    const HotBuf hb = hot_buf(lds + (uint32_t)wave * IW, cap, Smax);
    const __amdgpu_buffer_rsrc_t fr = xcd_rsrc(h.flags, kHotFlagWords * 4u);
    const __amdgpu_buffer_rsrc_t rr = xcd_rsrc(h.results, kHotResultWords * 8u);
    uint32_t* const claim = h.flags + 3 * kHotRing;
    U* const uu = static_cast<U*>(a.u);
    constexpr int NE = kStagedEntriesPerLane;
    const uint32_t c0 = (uint32_t)lane / Smax, k0 = (uint32_t)lane - c0 * Smax;
    const uint32_t dc = 64u / Smax, dk = 64u - dc * Smax;
    for (;;) {
        uint32_t b = 0;
        if (lane == 0) b = __hip_atomic_fetch_add(claim, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        b = wave_uniform(b);  // lane 0's claim
        if (b >= sc.nb) break;
        const uint32_t s = b % kHotRing;
        // The record's previous batch (b - kHotRing) must have been loaded.
        if (b >= kHotRing && !flag_wait(fr, (kHotRing + s) * 4u, b - kHotRing + 1u, h.spin_limit, h.err)) break;
        const uint32_t B = hot_batch_size(sc, b), NB = B * Smax;
        HotMeta md;
        md.m = hot_coord(h, sc, b, lane);
        hot_meta_load(a, md);
        const uint32_t len = md.m != kHotEmpty ? (uint32_t)(md.s1 - md.s0) : 0u;
        int32_t ky[NE];
        float vv[NE];
        bool in[NE];
        uint32_t c = c0, k = k0;
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const uint32_t cc = c < B ? c : 0u;
            const int64_t s0 = __shfl(md.s0, (int)cc);
            const uint32_t lc = (uint32_t)__shfl((int)len, (int)cc);
            in[t] = c < B && k < lc;
            const int64_t kk = in[t] ? s0 + k : 0;
            ky[t] = h.entry_key[kk];
            vv[t] = a.val[kk];
            c += dc;
            k += dk;
            if (k >= Smax) {
                k -= Smax;
                ++c;
            }
        }
        // The cold entries' shared-vector values, read now: a batch runs at most kHotRing + NP batches
        // after it is staged, and cold entries are by construction rarely updated.
        U cv[NE];
#pragma unroll
        for (int t = 0; t < NE; ++t) cv[t] = hot_load_u<U>(ub, (uint32_t)ky[t], in[t] && ky[t] >= 0);
        // The LDS image, as a producer writes it; each record's cold part of the dot is added below.
        if ((uint32_t)lane < B) {
            hb.mid[lane] = md.m;
            hb.rec[lane] = make_float4(md.m_old, hot_step_scale<FORM>(md.sn, a.k), md.ylab, 0.0f);
        }
        c = c0;
        k = k0;
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const uint32_t e = (uint32_t)t * 64u + (uint32_t)lane;
            const bool hot = in[t] && ky[t] < 0;
            if (e < NB) {
                const uint32_t zlane = ((c & 7u) << 3) | (k & 7u);
                hb.kv[e] = make_int2(hot ? -1 - ky[t] : (int32_t)(h.n_hot + zlane), __float_as_int(hot ? vv[t] : 0.0f));
            }
            c += dc;
            k += dk;
            if (k >= Smax) {
                k -= Smax;
                ++c;
            }
        }
        // Cold part: each aligned group of 8 slots belongs to one coordinate (Smax is a multiple of 8).
        c = c0;
        k = k0;
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const uint32_t e = (uint32_t)t * 64u + (uint32_t)lane;
            const bool cold = in[t] && ky[t] >= 0;
            const float part = group_sum<8>(cold ? vv[t] * (float)cv[t] : 0.0f);
            if (e < NB && (lane & 7) == 0 && part != 0.0f) atomicAdd(&hb.rec[c].w, part);
            c += dc;
            k += dk;
            if (k >= Smax) {
                k -= Smax;
                ++c;
            }
        }
        // Copy the image into the record (the wave's LDS operations complete in order).
        uint32_t* const rec = h.ring + (size_t)s * RW;
        const uint4* src = reinterpret_cast<const uint4*>(hb.rec);
        uint4* dst = reinterpret_cast<uint4*>(rec);
        for (uint32_t i = (uint32_t)lane; i < IW / 4u; i += 64u) dst[i] = src[i];
        // Publish only after every store of the record has completed.
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        if (lane == 0) flag_set(fr, s * 4u, b + 1u);
        // Wait for the batch's results (lane c: coordinate c's model value and coefficient, tagged b + 1),
        // then write the model values and the cold entries' updates out.
        const uint32_t roff = (s * 64u + (uint32_t)lane) * 16u;
        float model_new = 0.0f, coef = 0.0f;
        bool got = false;
        for (uint32_t spins = 0;; ++spins) {
            if ((uint32_t)lane < B && !got) {
                const xcd_v4 w = __builtin_amdgcn_raw_buffer_load_b128(rr, (int)roff, 0, kXcdPoll);
                if ((uint32_t)w[1] == b + 1u && (uint32_t)w[3] == b + 1u) {
                    got = true;
                    model_new = __int_as_float(w[0]);
                    coef = __int_as_float(w[2]);
                }
            }
            if (__all(got || (uint32_t)lane >= B)) break;
            if (spins >= h.spin_limit) {
                if (lane == 0) __hip_atomic_fetch_or(h.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        // The results are read: the record's result slot may take batch b + R.
        if (lane == 0) flag_set(fr, (2 * kHotRing + s) * 4u, b + 1u);
        if ((uint32_t)lane < B && md.m != kHotEmpty) a.model[md.m] = model_new;
        c = c0;
        k = k0;
#pragma unroll
        for (int t = 0; t < NE; ++t) {
            const float cf = __shfl(coef, (int)(c < B ? c : 0u));
            const float d = in[t] && ky[t] >= 0 ? cf * vv[t] : 0.0f;
            if (d != 0.0f) atomic_add_u(uu + ky[t], d);
            c += dc;
            k += dk;
            if (k >= Smax) {
                k -= Smax;
                ++c;
            }
        }
    }
}

constexpr uint32_t kStagedImageVecs = (hot_buf_words(64, kStagedEntriesPerLane) / 4 + 63) / 64;  // uint4 per lane, at most

// A loader's loads of one ring record (at byte offset rbase): the LDS image of its batch.  ioff holds
// the lane's offsets within a record (computed once per launch; lanes past the record carry an
// out-of-range offset, so they read 0 and touch no memory), and the record's base goes in the scalar
// offset.  An agent-scope acquire comes first, so that no line cached from the slot's previous batch
// is read; the caller has seen the record's tag.  The loads are only issued here.
template <int IV>
__device__ __forceinline__ void staged_record_load(__amdgpu_buffer_rsrc_t gr, uint32_t rbase, const uint32_t (&ioff)[IV],
                                                   xcd_v4 (&img)[IV]) {
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
    for (int v = 0; v < IV; ++v) img[v] = __builtin_amdgcn_raw_buffer_load_b128(gr, (int)ioff[v], (int)rbase, kXcdLoad);
}

// Loader wave q of workgroup 0 (buffer q, batches q, q + NP, ...).  Per batch: once the consumer has
// finished the buffer's previous batch, publish that batch's results (model value and coefficient of
// each coordinate, as 64-bit words tagged with the batch) for its stager; then take the new batch's
// record (usually loaded ahead, see below; else wait for its tag and load it now), write it into the
// buffer, free the record and hand the buffer to the consumer.  The stager has already added each
// coordinate's cold part of the dot, so the loader gathers nothing, and it issues no atomic on the
// shared vector.
template <int FORM, typename U>
__device__ __forceinline__ void staged_loader(const HotArgs& h, const HotSched& sc, uint32_t* ready, uint32_t* freed,
                                              uint32_t* abort_flag, uint32_t* bufs, uint32_t* moved_total, int q,
                                              int lane) {
    const uint32_t Smax = h.Smax, nb = sc.nb, NP = sc.NP, cap = h.cap;
    const uint32_t IW = hot_buf_words(cap, Smax), RW = staged_rec_words(cap, Smax);
    const uint32_t B = hot_batch(sc, hot_consumer_of(sc, (uint32_t)q));
    const HotBuf hb = hot_buf(bufs + q * IW, cap, Smax);
    const __amdgpu_buffer_rsrc_t fr = xcd_rsrc(h.flags, kHotFlagWords * 4u);
    const __amdgpu_buffer_rsrc_t rr = xcd_rsrc(h.results, kHotResultWords * 8u);
    const __amdgpu_buffer_rsrc_t gr = xcd_rsrc(h.ring, kHotRing * RW * 4u);
    constexpr int IV = (int)kStagedImageVecs;
    uint32_t moved = 0;
    // Flag words are read ahead so that their round trips overlap the consumer's steps: when batch b
    // has been handed over, the loader reads whether the result slot of the batch it hands over next
    // is free, and the record tag of its batch after next.  If the tag of its next batch (read one
    // batch earlier) is already set, it also issues that batch's record loads into registers then.
    // A flag word that was read ahead and not yet set is read again when needed.  A flag, once set,
    // stays set for the launch.  The words read ahead stay in vector registers until the consumer has
    // released the buffer (`*_v`), so that the wait for their loads, which also waits for the record
    // loads and result stores issued before them, falls after that release and not before it.
    uint32_t tag_seen = 0, tag_ahead = 0, res_seen = 0;
    uint32_t tag_seen_v = 0, tag_ahead_v = 0, res_seen_v = 0;
    bool pre = false;  // img holds batch b's record, loaded ahead
    xcd_v4 img[IV];
    // Offsets within a record; out-of-range ones stay out of range once the record's base (below
    // 2^20) is added.
    uint32_t ioff[IV];
#pragma unroll
    for (int v = 0; v < IV; ++v) {
        const uint32_t i = (uint32_t)lane + 64u * (uint32_t)v;
        ioff[v] = i < IW / 4u ? 16u * i : 0x7FF00000u;
    }
    if ((uint32_t)q + NP < nb)
        tag_ahead_v = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
            fr, (int)((((uint32_t)q + NP) % kHotRing) * 4u), 0, kXcdPoll);
    for (uint32_t b = (uint32_t)q; b < nb + NP; b += NP) {
        const uint32_t n = b / NP;
        if (n > 0 || b < nb) {
            if (!hot_wait(freed + q, n, abort_flag, h.spin_limit, h.err)) break;
        }
        tag_seen = wave_uniform(tag_seen_v);
        tag_ahead = wave_uniform(tag_ahead_v);
        res_seen = wave_uniform(res_seen_v);
        // Results of the buffer's previous batch, for the stager that assembled it: read out of the
        // buffer now, stored to the result ring after the buffer has been handed over again (so that
        // no wait for the stores' completion sits between the consumer's release and the hand-over).
        const uint32_t c = b - NP, cs = c % kHotRing;
        xcd_v2 w0 = {0, 0}, w1 = {0, 0};
        if (n > 0) {
            if (c >= kHotRing && res_seen != c - kHotRing + 1u &&
                !flag_wait(fr, (2 * kHotRing + cs) * 4u, c - kHotRing + 1u, h.spin_limit, h.err)) {
                __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                break;
            }
            if ((uint32_t)lane < B) {
                const uint32_t m = hb.mid[lane];
                const float2 zw = *reinterpret_cast<const float2*>(&hb.rec[lane].z);
                moved += (m != kHotEmpty && zw.y != 0.0f) ? 1u : 0u;
                // Each 8-byte half (value, tag) is written and read whole, so a reader that sees the tag
                // sees its value.
                w0 = xcd_v2{__float_as_int(zw.x), (int)(c + 1u)};
                w1 = xcd_v2{__float_as_int(zw.y), (int)(c + 1u)};
            }
        }
        // The result stores.  A loader never waits for a record's tag while it holds results it could
        // publish: the stager it waits for may itself be waiting for those results.
        bool published = n == 0;
        auto publish = [&]() {
            if ((uint32_t)lane < B) {
                const uint32_t roff = (cs * 64u + (uint32_t)lane) * 16u;
                __builtin_amdgcn_raw_buffer_store_b64(w0, rr, (int)roff, 0, kXcdStore);
                __builtin_amdgcn_raw_buffer_store_b64(w1, rr, (int)roff + 8, 0, kXcdStore);
            }
            published = true;
        };
        const uint32_t s = b % kHotRing, b2 = b + NP, b3 = b2 + NP;
        if (b < nb) {
            if (!pre) {
                if (tag_seen != b + 1u) {
                    if (!published) publish();
                    if (!flag_wait(fr, s * 4u, b + 1u, h.spin_limit, h.err)) {
                        __hip_atomic_store(abort_flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                        break;
                    }
                }
                staged_record_load<IV>(gr, s * RW * 4u, ioff, img);
            }
            // Wait for the record's loads (so its slot may be freed below), write it into the buffer
            // and hand the buffer over.
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
            __atomic_signal_fence(__ATOMIC_SEQ_CST);
            xcd_v4* const dst = reinterpret_cast<xcd_v4*>(hb.rec);
#pragma unroll
            for (int v = 0; v < IV; ++v) {
                const uint32_t i = (uint32_t)lane + 64u * (uint32_t)v;
                if (64u * (uint32_t)(v + 1) <= IW / 4u || i < IW / 4u) dst[i] = img[v];  // the first test is uniform
            }
            __hip_atomic_store(ready + q, n + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
            // The loads of the next batch's record go out here, while no other load or store of this
            // wave is in flight (the acquire before them waits for all of them).
            pre = b2 < nb && tag_ahead == b2 + 1u;
            if (pre) staged_record_load<IV>(gr, (b2 % kHotRing) * RW * 4u, ioff, img);
        }
        if (!published) publish();
        if (b >= nb) break;
        // Free this batch's record for batch b + R, and read the flag words ahead.
        if (lane == 0) flag_set(fr, (kHotRing + s) * 4u, b + 1u);
        tag_seen_v = b2 < nb && !pre ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
                                           fr, (int)((b2 % kHotRing) * 4u), 0, kXcdPoll)
                                     : 0u;
        tag_ahead_v = b3 < nb ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
                                    fr, (int)((b3 % kHotRing) * 4u), 0, kXcdPoll)
                              : 0u;
        res_seen_v = b >= kHotRing ? (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(
                                         fr, (int)((2 * kHotRing + s) * 4u), 0, kXcdPoll)
                                   : 0u;
    }
    for (int o = 32; o > 0; o >>= 1) moved += __shfl_xor(moved, o, 64);
    if (lane == 0) atomicAdd(moved_total, moved);
}

template <int FORM, typename U, int SL>
__global__ __launch_bounds__(64 * kHotWaves) void k_epoch_staged(HotArgs h) {
    extern __shared__ __align__(16) unsigned char hot_lds[];
    const EpochArgs& a = h.e;
    uint32_t W = h.W, NC = h.NC;
    if (h.adapt_in) {
        const uint32_t v = __hip_atomic_load(h.adapt_in, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (v >= 2 && v <= (uint32_t)kHotMaxWindow) W = v;
    }
    if (h.adapt_out) NC = hot_adaptive_consumers(W);
    const HotSched sc = hot_sched(W, NC, h.cap, h.pos_n);
    if (blockIdx.x > 0) {
        if (blockIdx.x % kHotXcds == 0 && blockIdx.x / kHotXcds <= h.stagers)
            staged_stager<FORM, U>(h, sc, reinterpret_cast<uint32_t*>(hot_lds));
        return;
    }
    U* const hot = reinterpret_cast<U*>(hot_lds);
    uint32_t* const ready = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes);
    uint32_t* const freed = ready + kHotMaxProducers;
    uint32_t* const abort_flag = freed + kHotMaxProducers;
    uint32_t* const moved = abort_flag + 1;
    float* const scr = reinterpret_cast<float*>(hot_lds + h.hot_bytes + kHotFlagBytes);
    uint32_t* const bufs = reinterpret_cast<uint32_t*>(hot_lds + h.hot_bytes + kHotFlagBytes + kHotScratchBytes);
    U* const uu = static_cast<U*>(a.u);
    const int tid = threadIdx.x, wave = (int)wave_uniform((uint32_t)tid >> 6), lane = tid & 63;
    if (tid == 0) {
        // Workgroup 0's XCD and this launch, for the stagers.
        __hip_atomic_store(h.prog + 1, hot_xcc_id(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_s_waitcnt(0x0F70);
        __hip_atomic_store(h.prog, h.tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (uint32_t i = tid; i < h.n_hot + kHotZeroCells; i += blockDim.x) hot[i] = i < h.n_hot ? uu[h.hot_ids[i]] : U(0);
    if (tid < 2 * kHotMaxProducers + 2) ready[tid] = 0u;
    __syncthreads();
    if ((uint32_t)wave < sc.NC) {
        if (sc.w_hi <= 4)
            hot_consumer16<FORM, U, (SL + 1) / 2, SL>(h, sc, (uint32_t)wave, hot, ready, freed, abort_flag, bufs, scr, lane);
        else
            hot_consumer<FORM, U, SL>(h, sc, (uint32_t)wave, hot, ready, freed, abort_flag, bufs, scr, lane);
    } else
        staged_loader<FORM, U>(h, sc, ready, freed, abort_flag, bufs, moved, wave - (int)sc.NC, lane);
    __syncthreads();
    for (uint32_t i = tid; i < h.n_hot; i += blockDim.x) uu[h.hot_ids[i]] = hot[i];
    if (h.adapt_out && tid == 0 && *abort_flag == 0u) {
        const uint64_t mv = *moved, wmax = kHotMaxWindow;
        uint64_t w = mv ? 1 + (uint64_t)(h.w_rule - 1) * h.pos_n / mv : wmax;
        w = w < h.w_rule ? h.w_rule : w > wmax ? wmax : w;
        __hip_atomic_store(h.adapt_out, (uint32_t)w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The kernel instance for a formulation, storage type and row width (Smax / 8 entries per consumer lane).
template <int FORM, typename U>
static const void* hot_kernel_sl(uint32_t sl) {
    switch (sl) {
        case 1: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 1>);
        case 2: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 2>);
        case 3: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 3>);
        case 4: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 4>);
        case 5: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 5>);
        case 6: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 6>);
        case 7: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 7>);
        case 8: return reinterpret_cast<const void*>(&k_epoch_hot<FORM, U, 8>);
        default: return nullptr;
    }
}

static const void* hot_kernel(int form, bool wide, uint32_t Smax) {
    if (Smax % 8 != 0) return nullptr;  // the consumers take Smax = 8 * SL
    const uint32_t sl = Smax / 8;
    switch (form) {
        case FORM_RIDGE_PRIMAL:
            return wide ? hot_kernel_sl<FORM_RIDGE_PRIMAL, double>(sl) : hot_kernel_sl<FORM_RIDGE_PRIMAL, float>(sl);
        case FORM_SVM_DUAL:
            return wide ? hot_kernel_sl<FORM_SVM_DUAL, double>(sl) : hot_kernel_sl<FORM_SVM_DUAL, float>(sl);
        case FORM_RIDGE_DUAL:
            return wide ? hot_kernel_sl<FORM_RIDGE_DUAL, double>(sl) : hot_kernel_sl<FORM_RIDGE_DUAL, float>(sl);
        default: return nullptr;
    }
}

hipError_t hot_prepare(int form, bool wide, uint32_t Smax, size_t lds_bytes) {
    const void* f = hot_kernel(form, wide, Smax);
    if (!f) return hipErrorInvalidValue;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

template <int FORM, typename U>
static const void* staged_kernel_sl(uint32_t sl) {
    switch (sl) {
        case 1: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 1>);
        case 2: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 2>);
        case 3: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 3>);
        case 4: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 4>);
        case 5: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 5>);
        case 6: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 6>);
        case 7: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 7>);
        case 8: return reinterpret_cast<const void*>(&k_epoch_staged<FORM, U, 8>);
        default: return nullptr;
    }
}

static const void* staged_kernel(int form, bool wide, uint32_t Smax) {
    if (Smax % 8 != 0) return nullptr;  // as in hot_kernel
    const uint32_t sl = Smax / 8;
    switch (form) {
        case FORM_RIDGE_PRIMAL:
            return wide ? staged_kernel_sl<FORM_RIDGE_PRIMAL, double>(sl) : staged_kernel_sl<FORM_RIDGE_PRIMAL, float>(sl);
        case FORM_SVM_DUAL:
            return wide ? staged_kernel_sl<FORM_SVM_DUAL, double>(sl) : staged_kernel_sl<FORM_SVM_DUAL, float>(sl);
        case FORM_RIDGE_DUAL:
            return wide ? staged_kernel_sl<FORM_RIDGE_DUAL, double>(sl) : staged_kernel_sl<FORM_RIDGE_DUAL, float>(sl);
        default: return nullptr;
    }
}

hipError_t staged_prepare(int form, bool wide, uint32_t Smax, size_t lds_bytes) {
    const void* f = staged_kernel(form, wide, Smax);
    if (!f) return hipErrorInvalidValue;
    return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t launch_epoch_staged(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s) {
    const void* f = staged_kernel(form, wide, h.Smax);
    if (!f || !h.ring || !h.flags || !h.results || !h.prog || h.stagers < 1 || h.cap > 64) return hipErrorInvalidValue;
    // A stager keeps one batch image per wave in the dynamic LDS every workgroup of the launch receives.
    if (staged_lds_bytes(h.hot_bytes, h.cap, h.Smax) > lds_bytes) return hipErrorInvalidValue;
    hipError_t e = launch_fill_zero(reinterpret_cast<uint64_t*>(h.flags), kHotFlagWords / 2, s);
    if (e == hipSuccess) e = launch_fill_zero(h.results, kHotResultWords, s);
    if (e != hipSuccess) return e;
    HotArgs arg = h;
    void* args[] = {&arg};
    return hipLaunchKernel(f, dim3(1 + kHotXcds * h.stagers), dim3(64 * kHotWaves), args, lds_bytes, s);
}

hipError_t launch_epoch_hot(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s) {
    const void* f = hot_kernel(form, wide, h.Smax);
    if (!f) return hipErrorInvalidValue;
    HotArgs arg = h;
    void* args[] = {&arg};
    return hipLaunchKernel(f, dim3(1), dim3(64 * kHotWaves), args, lds_bytes, s);
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

// Each stored entry's key for the producers: -1 - slot for an entry whose shared-vector index is hot,
// else the index (so a producer reads one array instead of idx and a slot array).
__global__ __launch_bounds__(256) void k_hot_entry_keys(const int32_t* __restrict__ idx, int64_t nnz,
                                                        const uint16_t* __restrict__ slot_of,
                                                        int32_t* __restrict__ entry_key) {
    for (int64_t k = (int64_t)blockIdx.x * 256 + threadIdx.x; k < nnz; k += (int64_t)gridDim.x * 256) {
        const int32_t i = idx[k];
        const uint16_t sl = slot_of[i];
        entry_key[k] = sl != kHotCold ? -1 - (int32_t)sl : i;
    }
}

hipError_t launch_hot_entry_keys(const int32_t* idx, int64_t nnz, const uint16_t* slot_of, int32_t* entry_key,
                                 hipStream_t s) {
    const int64_t want = (nnz + 255) / 256;
    const unsigned blocks = (unsigned)(want < 1 ? 1 : want > 65536 ? 65536 : want);
    hipLaunchKernelGGL(k_hot_entry_keys, dim3(blocks), dim3(256), 0, s, idx, nnz, slot_of, entry_key);
    return hipGetLastError();
}

hipError_t launch_hot_assign(const unsigned* hits, int64_t L, unsigned T, const unsigned* block_base, uint16_t* slot_of,
                             int32_t* hot_ids, hipStream_t s) {
    const int64_t nb = (L + kHotAssignBlock - 1) / kHotAssignBlock;
    hipLaunchKernelGGL(k_hot_assign, dim3((unsigned)nb), dim3(256), 0, s, hits, L, T, block_base, slot_of, hot_ids);
    return hipGetLastError();
}

}  // namespace scd
