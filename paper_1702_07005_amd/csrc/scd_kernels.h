// scd_kernels.h -- argument structures and launchers shared by the C ABI and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scd {

enum { FORM_RIDGE_PRIMAL = 0, FORM_SVM_DUAL = 1, FORM_RIDGE_DUAL = 2 };

// Register-slice depth of the G-lane epoch kernels: each lane keeps up to slice_depth(G)
// entries of its coordinate's segment between the gather and the scatter.
constexpr int slice_depth(int G) { return G <= 4 ? 4 : G <= 8 ? 6 : G == 16 ? 10 : G == 32 ? 5 : 4; }

// Keys of one epoch's permutation of [0, n): 4 Feistel round keys on 2h bits.
struct PermKeys {
    uint32_t k[4];
    uint32_t h;
    uint32_t mask;
    uint32_t n;
    uint32_t pad_;
};

// Constants of the closed-form steps (lambda is the paper's normalised lambda).
struct StepConsts {
    float lamN;      // lambda * N
    float inv_lamN;  // 1 / (lambda * N)
    float lam;       // lambda
    float pad_;
};

struct EpochArgs {
    const int64_t* ptr;
    const int32_t* idx;
    const float* val;
    const float* y;      // per-coordinate constant: <y, a_c> (ridge primal) or the label (duals)
    float* model;        // [C]
    void* u;             // shared vector [L], float or double (LaunchPlan::wide)
    const float* norms;  // [C]
    StepConsts k;
    PermKeys perm;       // perm.n = C
    uint32_t n_groups;   // persistent groups (coordinates in flight at most)
    uint32_t u_bytes;    // byte size of the shared vector when below 2^31 (raw-buffer range), else 0
    uint32_t u_shift;    // log2 of the bytes from one shared-vector entry to the next in u: the
                         // entry size (2 or 3), or kSpreadShift when u is the spread copy
    double* sink;        // pipelined kernel, fp64 shared vector: 256 slots per workgroup that
                         // inactive lanes add 0 to
    uint32_t drain;      // wait for the group's own atomics before its next gathers (window binds)
    uint32_t chunk;      // queued kernel: consecutive positions per claim (1..kQueueChunkMax)
    uint32_t* queue;     // queued kernel: [0] next permutation position, [1] workgroups finished (both 0
                         // between launches)
};

constexpr uint32_t kQueueChunkMax = 64;
// Spread copy of a small shared vector for the pipelined and queued kernels: one entry per 64
// bytes, so that concurrent gathers and atomics of different entries never share a segment.
constexpr uint32_t kSpreadShift = 6;
constexpr int kQueueSlices = 16;  // register slices per lane of the queued kernel (256 x 16 entries held)

enum {
    PLAN_GROUP = 0,
    PLAN_BLOCK = 1,
    PLAN_ORDERED_LDS = 2,
    PLAN_MIXED = 3,
    PLAN_PIPE = 4,
    PLAN_HOT = 5,
    PLAN_QUEUE = 6,
    PLAN_TEAM = 7,
    PLAN_HOT_STAGED = 8,  // PLAN_HOT with stager workgroups assembling the batches (large matrices)
    PLAN_SPLIT = 9        // PLAN_QUEUE over work units: long segments split into parts (many CUs each)
};

struct LaunchPlan {
    int kind;        // PLAN_*
    int group;       // lanes per coordinate (PLAN_GROUP, PLAN_MIXED, PLAN_PIPE: 4..64 or 256)
    int blocks;      // workgroups launched
    int fresh;       // device-scope gathers
    int ordered;     // PLAN_BLOCK with a single workgroup, fenced between coordinates
    uint32_t L;      // shared-vector length (PLAN_ORDERED_LDS)
    uint32_t long_len;  // PLAN_MIXED: segments longer than this go to the whole workgroup
    int tail;           // PLAN_GROUP: some segment is longer than the register slices
    int drain;          // PLAN_PIPE, PLAN_GROUP, PLAN_BLOCK: the window binds, so each group lets its scatter
                        // land before it gathers again
    int chunk;          // PLAN_QUEUE, PLAN_SPLIT: consecutive positions (units) per claim
    uint32_t part;      // PLAN_SPLIT: entries per part of a long segment (multiple of 64, <= kSplitMaxPart)
    int wide;           // shared vector stored as double
    int unbound;        // PLAN_PIPE: the window does not bind (every coordinate may be in flight)
    int team;           // PLAN_TEAM: workgroups per in-flight coordinate (K)
    size_t lds_bytes;
};

struct ObjArgs {
    const int64_t* ptr;
    const int32_t* idx;
    const float* val;
    const void* u;       // shared vector as maintained (float, or double when `wide`)
    int wide;
    const float* model;
    const float* y;      // per-coordinate labels (duals)
    const float* yv;     // per-shared-entry labels (ridge primal: y over rows)
    const double* cyd;   // ridge primal: <y, a_c> in fp64
    uint32_t C;
    int64_t L;
    double lam;
};

// Hot-set epoch (one workgroup of kHotWaves waves): the n_hot most-updated shared-vector entries live
// in LDS for the epoch; one to four consumer waves run the in-flight coordinates from LDS only (each
// up to kHotMaxGroups of them, 8 lanes each), and the other waves stream the next batches (segment,
// hot slot or cold value) into LDS buffers, one buffer per producer.  kHotWaves - NC is a multiple
// of NC for every consumer count NC used (11, 10, 9, 8 for NC = 1..4), so the batches of one buffer
// all go to one consumer.
constexpr int kHotWaves = 12;
constexpr int kHotMaxConsumers = 4;
constexpr int kHotMaxProducers = kHotWaves - 1;  // with one consumer
constexpr int kHotEntriesPerLane = 10;  // producer lanes x this >= batch entries (64 x 10 = 640)
// Stager lanes x this >= a staged batch's entries (64 x 15 = 960).  Staged batches are larger, so
// that the hot workgroup's per-batch hand-over (a loader's turn, the consumer's wait and first
// read) is spread over more consumer steps; the hot set that fits beside such buffers is smaller.
constexpr int kStagedEntriesPerLane = 15;
constexpr int kHotFlagBytes = 128;      // LDS words: ready[producer], freed[producer], abort, moved count
constexpr int kHotScratchBytes = kHotMaxConsumers * 64 * 8;  // write targets of inactive consumer lanes
constexpr int kHotZeroCells = 64;         // hot-array cells after the hot set, one per consumer lane
constexpr int kHotMaxGroups = 8;          // coordinates per consumer step (groups of 8 lanes)
constexpr int kHotMaxWindow = 2 * kHotMaxGroups;  // coordinates in flight at most
// The first adaptive epoch runs its first 1/kHotOpening of the positions at the coupling rule's window.
constexpr uint32_t kHotOpening = 16;
constexpr int kHotMaxSegment = 64;

constexpr uint16_t kHotCold = 0xFFFF;    // slot_of value of an entry that is not hot

// 32-bit words of one batch buffer (B coordinates, Smax entry slots each): a 4-word record per
// coordinate, key and value per slot, coordinate index; rounded up to 16 bytes so that every buffer
// and its records stay aligned.
__host__ __device__ constexpr uint32_t hot_buf_words(uint32_t B, uint32_t Smax) {
    return (5u * B + 2u * B * Smax + 3u) & ~3u;
}
// Coordinates per batch for rows of Smax entry slots, with `per_lane` entries per producer lane.
__host__ __device__ constexpr uint32_t hot_batch_cap(uint32_t Smax, uint32_t per_lane) {
    return 64u * per_lane / Smax < 64u ? 64u * per_lane / Smax : 64u;
}

// Staged variant of the hot-set epoch: stager workgroups (on the XCD of workgroup 0: workgroups
// kHotXcds, 2 kHotXcds, ...) claim batches, read their metadata and entries, gather the cold entries'
// shared-vector values, and write each batch's LDS image (with every coordinate's cold part of the
// dot) into a ring of kHotRing records in device memory; workgroup 0's loader waves copy records
// into LDS and hand the results back; the stagers write them out.
constexpr int kHotXcds = 8;
constexpr int kHotStagers = 16;
constexpr uint32_t kHotRing = 32;
// 32-bit words of one ring record: the LDS image of a batch buffer.
__host__ __device__ constexpr uint32_t staged_rec_words(uint32_t cap, uint32_t Smax) {
    return hot_buf_words(cap, Smax);
}
// Words of the ring's flags: tag[R] (batch + 1 staged), slot_free[R] (batch + 1 loaded), res_free[R]
// (batch + 1 whose results its stager has read), the claim counter, padded; zeroed before every launch.
constexpr uint32_t kHotFlagWords = 3 * kHotRing + 64;
// 64-bit words of the result ring: per record, 2 words (model value, coefficient; each with the batch
// + 1 in its high half) per coordinate of the batch; zeroed before every launch.
constexpr uint32_t kHotResultWords = kHotRing * 64 * 2;

struct HotArgs {
    EpochArgs e;
    const int32_t* entry_key;    // [nnz]: per stored entry, -1 - the LDS slot of its shared-vector
                                 // index when that entry is hot, else the index itself
    const int32_t* hot_ids;   // [n_hot]: shared-vector index of each slot
    uint32_t n_hot;
    uint32_t W;               // coordinates in flight (2..kHotMaxWindow) unless `adapt_in` sets them
    uint32_t NC;              // consumer waves (1, or 2 when W may exceed kHotMaxGroups)
    uint32_t cap;             // coordinates a batch buffer holds; a consumer with w groups takes
                              // batches of cap / w * w coordinates
    uint32_t Smax;            // entries per coordinate reserved in a batch buffer (multiple of 8)
    uint32_t hot_bytes;       // LDS bytes of the hot array and its zero cells (16-byte aligned)
    uint32_t spin_limit;      // bounded waits: after this many sleeps a wave gives up and sets *err
    uint32_t w_rule;          // adaptive window: coordinates in flight the coupling rule allows
                              // when every coordinate moves
    uint32_t pos0, pos_n;     // permutation positions [pos0, pos0 + pos_n) of the epoch that this
                              // launch runs: the whole epoch, or one of its segments
    // Staged variant only (null otherwise):
    uint32_t* ring;            // [kHotRing][staged_rec_words(cap, Smax)]
    uint32_t* flags;           // [kHotFlagWords], zero at launch
    uint64_t* results;         // [kHotResultWords], zero at launch
    uint32_t* prog;            // [4]: launch tag and XCD of workgroup 0, for the stagers
    uint32_t tag;              // this launch's tag (nonzero, new for every staged launch of the handle)
    uint32_t stagers;          // stager workgroups
    const uint32_t* adapt_in;  // adaptive window (null: W): coordinates in flight for this launch,
                               // written by the previous one
    uint32_t* adapt_out;       // adaptive window (null: none): receives the next launch's window, set
                               // from the coordinates whose step was nonzero in this one
    int* err;
};

// Coordinates per batch and consumer steps of a hot-set epoch with W coordinates in flight on NC
// consumer waves: consumer c runs w_c coordinates per step, the first n_hi consumers w_hi =
// ceil(W / NC) and the rest w_lo = floor(W / NC), so that the shares sum to W; batch b goes to
// consumer b mod NC and holds S w_c coordinates, S = cap / w_hi steps for every consumer.  Equal step
// counts keep the consumers in step with one another (the batches go round them in turn), so the
// epoch runs W coordinates per step time.  Scalar fields only: the kernels select between them,
// which keeps the struct in registers.
struct HotSched {
    uint32_t NC, NP;   // consumer and producer waves
    uint32_t W;        // coordinates in flight
    uint32_t w_hi, w_lo, n_hi;
    uint32_t S;        // steps per batch
    uint32_t nb;       // batches in the launch
};

__host__ __device__ inline uint32_t hot_groups(const HotSched& s, uint32_t c) { return c < s.n_hi ? s.w_hi : s.w_lo; }
__host__ __device__ inline uint32_t hot_batch(const HotSched& s, uint32_t c) { return s.S * hot_groups(s, c); }
__host__ __device__ inline uint32_t hot_consumer_of(const HotSched& s, uint32_t b) { return b % s.NC; }

__host__ __device__ inline HotSched hot_sched(uint32_t W, uint32_t NC, uint32_t cap, uint32_t n) {
    HotSched s{};
    s.NC = NC;
    s.NP = (uint32_t)kHotWaves - NC;
    s.W = W;
    s.w_lo = W / NC;
    s.n_hi = W - s.w_lo * NC;
    s.w_hi = s.w_lo + (s.n_hi ? 1u : 0u);
    s.S = cap / s.w_hi;
    const uint32_t round = s.S * W, q = n / round;  // a round: one batch for each consumer
    uint32_t rem = n - q * round, nb = q * NC;
    for (uint32_t c = 0; c < NC && rem > 0; ++c) {
        const uint32_t B = hot_batch(s, c);
        rem = rem > B ? rem - B : 0u;
        ++nb;
    }
    s.nb = nb;
    return s;
}

// First permutation position of batch b (within the launch's range), and its size.
__host__ __device__ inline uint32_t hot_batch_start(const HotSched& s, uint32_t b) {
    const uint32_t r = b % s.NC;
    return (b / s.NC) * s.S * s.W + s.S * (r * s.w_lo + (r < s.n_hi ? r : s.n_hi));
}
__host__ __device__ inline uint32_t hot_batch_size(const HotSched& s, uint32_t b) {
    return hot_batch(s, hot_consumer_of(s, b));
}

// The consumer waves for an adaptive window of W: as many as keep at least two coordinates per
// consumer step, up to kHotMaxConsumers.  A step takes about the same time whatever it holds (about
// 600 cycles for 3 to 4 coordinates at full click size, its two LDS round trips and dependent
// instructions dominating; 730 for 8), so the epoch's rate is the window over the step time, and
// more, narrower consumers shorten the step: full-size click epochs at 16 in flight took 0.83 s on
// four consumers of 4 and 0.95 s on two of 8.
__host__ __device__ inline uint32_t hot_adaptive_consumers(uint32_t W) {
    const uint32_t n = W / 2;
    return n < 1 ? 1u : n > (uint32_t)kHotMaxConsumers ? (uint32_t)kHotMaxConsumers : n;
}

size_t hot_lds_bytes(uint32_t hot_bytes, uint32_t B, uint32_t Smax);
// Dynamic LDS of a staged launch: every workgroup gets the same size, and a stager keeps one batch
// image per wave, which exceeds the hot workgroup's need when the hot set is small.
size_t staged_lds_bytes(uint32_t hot_bytes, uint32_t cap, uint32_t Smax);
hipError_t hot_prepare(int form, bool wide, uint32_t Smax, size_t lds_bytes);
hipError_t launch_epoch_hot(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s);
// The staged variant (h.ring, h.flags, h.prog set): zeroes the flags, then launches 1 + kHotXcds *
// h.stagers workgroups.
hipError_t launch_epoch_staged(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s);
hipError_t staged_prepare(int form, bool wide, uint32_t Smax, size_t lds_bytes);
hipError_t launch_hot_count_ge(const unsigned* hits, int64_t L, unsigned T, unsigned long long* out2, hipStream_t s);
hipError_t launch_hot_block_count(const unsigned* hits, int64_t L, unsigned T, unsigned* block_counts, hipStream_t s);
hipError_t launch_hot_assign(const unsigned* hits, int64_t L, unsigned T, const unsigned* block_base, uint16_t* slot_of,
                             int32_t* hot_ids, hipStream_t s);
constexpr int kHotAssignBlock = 1024;  // shared-vector indices per workgroup in the slot assignment

// Team epoch: each of the n_groups in-flight coordinates is processed by a team of K workgroups
// (K <= kTeamMax), member k on the entries of the coordinate's segment whose shared-vector index
// lies in the k-th of K index ranges.  `e.idx`/`e.val` are the segment entries grouped by range
// (k_team_partition); member k's part of coordinate m is [ptr[m] + off[m(K+1)+k],
// ptr[m] + off[m(K+1)+k+1]).  The members exchange their partial dot products through 64-bit slots
// (fp32 bits, 32-bit step tag): slots[(team * 2 + tag % 2) * kTeamMax + k].
constexpr int kTeamMax = 16;
constexpr uint32_t kTeamXcds = 8;  // XCDs of the MI355X, to which workgroups are dispatched in turn
// Workgroups of a team launch: kTeamXcds times the most (team, member) pairs placed on one XCD, with
// member k of team t on XCD (t + k) mod kTeamXcds.
inline int team_grid(int64_t teams, int64_t K) {
    int64_t cnt[kTeamXcds] = {0};
    for (int64_t t = 0; t < teams; ++t)
        for (int64_t k = 0; k < K; ++k) ++cnt[(t + k) % kTeamXcds];
    int64_t mx = 0;
    for (uint32_t x = 0; x < kTeamXcds; ++x) mx = cnt[x] > mx ? cnt[x] : mx;
    return (int)(mx * kTeamXcds);
}
constexpr int kTeamSlices = 4;  // register slices per lane (256 x 4 entries of a member's part held)

struct TeamArgs {
    EpochArgs e;
    const uint32_t* off;   // [C * (K + 1)]
    uint64_t* slots;       // [n_groups * 2 * kTeamMax]
    uint32_t K;
    uint32_t tag0;         // tag of the first step of this launch (tags grow by one per step)
    uint32_t spin_limit;   // bounded waits: after this many sleeps a member gives up and sets *err
    int* err;
};

// `cus`: compute units of the device; the launch is refused unless the whole grid is resident at once.
hipError_t launch_epoch_team(int form, bool wide, bool fresh, const TeamArgs& t, int blocks, int cus, hipStream_t s);
// Groups each segment's entries by index range: bound[0] = 0 < bound[1] <= ... <= bound[K] = L.
hipError_t launch_team_partition(const int64_t* ptr, const int32_t* idx, const float* val, uint32_t C,
                                 const uint32_t* bound, int K, int32_t* out_idx, float* out_val, uint32_t* off,
                                 hipStream_t s);

// Split epoch: the queued kernel over work units instead of permutation positions.  Before each
// epoch a pre-pass lays the units out in permutation order: a segment of at most `part` entries is
// one FULL unit; a longer one, of k = ceil(len / part) parts, is k GATHER units (part i's partial
// inner product) followed by k SCATTER units (each waits for the coordinate's k partials, sums them
// in a fixed order, takes the step and scatters part i).  The workgroups claim units in order from
// the queue, so a long segment's parts are gathered, and then scattered, by many CUs at once.
constexpr uint32_t kSplitMaxPart = 256 * kQueueSlices;  // a part fits the register slices
constexpr uint32_t kSplitMaxParts = 256;                // parts per segment (4 per lane of the polling wave)
constexpr uint32_t kSplitPrepTile = 2048;               // positions per workgroup of the pre-pass
enum { SPLIT_FULL = 0, SPLIT_GATHER = 1, SPLIT_SCATTER = 2 };

// One work unit, 32 bytes.  info = kind << 30 | parts << 15 | part index (parts, index < 2^15).
// m_old is the model value at the start of the epoch: each coordinate is visited once per epoch and
// only its own step writes it.
struct SplitUnit {
    int64_t s0;    // first entry of the unit's range
    uint32_t len;  // entries in the range
    uint32_t m;    // coordinate
    float m_old, sn, ylab;
    uint32_t info;
};
static_assert(sizeof(SplitUnit) == 32, "SplitUnit is 32 bytes");

__host__ __device__ inline uint32_t split_units_of(int64_t len, uint32_t part) {
    return len <= (int64_t)part ? 1u : 2u * (uint32_t)((len + part - 1) / part);
}

struct SplitArgs {
    EpochArgs e;           // e.perm: the epoch's permutation; e.queue, e.chunk as for the queued kernel
    const SplitUnit* units;
    uint64_t* partials;    // [n_units]: GATHER unit u writes (fp32 bits | tag << 32) at partials[u]
    uint32_t n_units;
    uint32_t tag;          // this launch's tag (never 0; the host counts launches)
    uint32_t spin_limit;   // bounded waits: after this many sleeps a SCATTER unit gives up and sets *err
    int* err;
};

// Units of all coordinates for part length `part` (independent of the permutation): out[0] (u64).
hipError_t launch_split_total(const int64_t* ptr, uint32_t C, uint32_t part, unsigned long long* out, hipStream_t s);
// Pre-pass and epoch.  `block_units` holds ceil(C / kSplitPrepTile) words of scratch; `units` holds
// n_units records.
hipError_t launch_epoch_split(int form, bool wide, bool fresh, const SplitArgs& sa, uint32_t part,
                              uint32_t* block_units, SplitUnit* units, int blocks, hipStream_t s);

hipError_t launch_epoch(int form, const EpochArgs& a, const LaunchPlan& lp, hipStream_t s);
hipError_t ordered_lds_prepare(int form, bool wide, size_t lds_bytes);
hipError_t launch_convert_f32_to_f64(const float* in, int64_t n, double* out, hipStream_t s);
hipError_t launch_convert_f64_to_f32(const double* in, int64_t n, float* out, hipStream_t s);
hipError_t launch_max_hits(const int32_t* idx, int64_t nnz, int64_t L, unsigned* hits, unsigned* out, hipStream_t s);
hipError_t launch_count_hits(const int32_t* idx, int64_t nnz, unsigned* hits, hipStream_t s);
hipError_t launch_hot_entry_keys(const int32_t* idx, int64_t nnz, const uint16_t* slot_of, int32_t* entry_key,
                                  hipStream_t s);
hipError_t launch_perm_fill(const PermKeys& p, int32_t* out, hipStream_t s);
// Copies the packed shared vector into its spread copy (entry i at byte i << kSpreadShift), or back.
hipError_t launch_spread(void* packed, void* spread, int64_t L, bool wide, bool to_spread, hipStream_t s);
hipError_t launch_gather_dots(const int64_t* ptr, const int32_t* idx, const float* val, const float* u, uint32_t C,
                              int G, int blocks, float* out, hipStream_t s);
hipError_t launch_norms(const int64_t* ptr, const int32_t* idx, const float* val, const float* y, uint32_t C, int G,
                        int blocks, float* out, float* cy, double* cyd, hipStream_t s);
hipError_t launch_validate(const int64_t* ptr, uint32_t S, const int32_t* idx, const float* val, int64_t nnz,
                           int64_t bound, const float* y, int64_t ny, int pm1, int* flags, hipStream_t s);
hipError_t launch_probe(const int64_t* ptr, const int32_t* idx, const float* val, const float* norms,
                        const float* sign, uint32_t C, int64_t L, float mu, uint32_t probe, int G, int blocks,
                        float* T, float* K, double* partials, double* out, hipStream_t s);
hipError_t launch_kappa_max(const float* K, const float* norms, uint32_t C, int probes, int blocks, unsigned* out,
                            hipStream_t s);
// One objective evaluation: k_objective (partials[blocks][5]) and k_sum_partials (sums[0..4]).  With
// o.cyd null the ridge primal gathers y beside the shared vector.
hipError_t launch_objective(int form, const ObjArgs& o, int G, int blocks, double* partials, double* sums,
                            hipStream_t s);
hipError_t launch_fill_zero(uint64_t* p, uint32_t n_words, hipStream_t s);
// Sets the calling thread's message returned by scd_last_error.
void set_last_error(const char* msg);

// Workgroups of the objective's pass, and its lanes per coordinate for segments of `mean` entries on
// average (the epoch kernels' group width, at most one wave).
constexpr int kObjBlocksMax = 2048;
inline int objective_group(double mean) {
    const int widths[5] = {4, 8, 16, 32, 64};
    for (int G : widths)
        if (mean <= (double)(G * slice_depth(G))) return G;
    return 64;
}
inline int objective_blocks(int64_t C, int G) {
    int64_t b = (C * G + 255) / 256;
    if (b > kObjBlocksMax) b = kObjBlocksMax;
    if (b < 1) b = 1;
    return (int)b;
}

// Primal and dual objectives from the five sums of one evaluation (fp64 on the host):
//   ridge primal: t0 = sum_m <a_m, r>^2, t1 = |beta|^2, t3 = |r|^2, t4 = <r, y>   (r = y - A beta)
//   SVM dual:     t0 = sum hinge, t1 = sum alpha, t3 = |w|^2
//   ridge dual:   t0 = |A wbar / lambda - y|^2, t1 = |alpha|^2, t2 = <alpha, y>, t3 = |wbar|^2
inline void objectives_from_sums(int form, double N, double lam, const double* t, double* P, double* D) {
    if (form == FORM_RIDGE_PRIMAL) {
        *P = t[3] / (2.0 * N) + 0.5 * lam * t[1];
        *D = -t[3] / (2.0 * N) - t[0] / (2.0 * lam * N * N) + t[4] / N;
    } else if (form == FORM_SVM_DUAL) {
        *P = t[0] / N + 0.5 * lam * t[3];
        *D = t[1] / N - 0.5 * lam * t[3];
    } else {
        *P = t[0] / (2.0 * N) + 0.5 * t[3] / lam;
        *D = -0.5 * N * t[1] - t[3] / (2.0 * lam) + t[2];
    }
}

}  // namespace scd
