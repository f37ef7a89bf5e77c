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
    uint32_t drain;      // pipelined kernel: wait for the group's own atomics before its next gathers
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
    PLAN_TEAM = 7
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
    int drain;          // PLAN_PIPE: the window binds, so each group lets its scatter land before it gathers again
    int chunk;          // PLAN_QUEUE: consecutive permutation positions per claim
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

// Hot-set epoch (one workgroup): the n_hot most-updated shared-vector entries live in LDS for the
// epoch; one consumer wave runs the W in-flight coordinates from LDS only, kHotProducers waves stream
// the next batches (segment, hot slot or cold value) into LDS buffers.
constexpr int kHotProducers = 11;
constexpr int kHotEntriesPerLane = 10;  // producer lanes x this >= batch entries (64 x 10 = 640)
constexpr int kHotFlagBytes = 128;      // LDS handover words: ready[producer], freed[producer], abort
constexpr int kHotScratchBytes = 64 * 8;  // write targets of the consumer's inactive lanes (8 bytes each)
constexpr int kHotZeroCells = 64;         // hot-array cells after the hot set, one per consumer lane
constexpr int kHotMaxWindow = 8;         // consumer wave: W groups of 8 lanes
constexpr int kHotMaxSegment = 64;
constexpr uint16_t kHotCold = 0xFFFF;    // slot_of value of an entry that is not hot

// 32-bit words of one batch buffer (B coordinates, Smax entry slots each): a 4-word record per
// coordinate, key and value per slot, coordinate index; rounded up to 16 bytes so that every buffer
// and its records stay aligned.
__host__ __device__ constexpr uint32_t hot_buf_words(uint32_t B, uint32_t Smax) {
    return (5u * B + 2u * B * Smax + 3u) & ~3u;
}

struct HotArgs {
    EpochArgs e;
    const int32_t* entry_key;    // [nnz]: per stored entry, -1 - the LDS slot of its shared-vector
                                 // index when that entry is hot, else the index itself
    const int32_t* hot_ids;   // [n_hot]: shared-vector index of each slot
    uint32_t n_hot;
    uint32_t W;               // coordinates in flight (<= kHotMaxWindow)
    uint32_t B;               // coordinates per batch (multiple of W)
    uint32_t Smax;            // entries per coordinate reserved in a batch buffer (multiple of 8)
    uint32_t hot_bytes;       // LDS bytes of the hot array and its zero cells (16-byte aligned)
    uint32_t spin_limit;      // bounded waits: after this many sleeps a wave gives up and sets *err
    int* err;
};

size_t hot_lds_bytes(uint32_t hot_bytes, uint32_t B, uint32_t Smax);
hipError_t hot_prepare(int form, bool wide, size_t lds_bytes);
hipError_t launch_epoch_hot(int form, bool wide, const HotArgs& h, size_t lds_bytes, hipStream_t s);
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

hipError_t launch_epoch_team(int form, bool wide, bool fresh, const TeamArgs& t, int blocks, hipStream_t s);
// Groups each segment's entries by index range: bound[0] = 0 < bound[1] <= ... <= bound[K] = L.
hipError_t launch_team_partition(const int64_t* ptr, const int32_t* idx, const float* val, uint32_t C,
                                 const uint32_t* bound, int K, int32_t* out_idx, float* out_val, uint32_t* off,
                                 hipStream_t s);

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
hipError_t launch_objective(int form, const ObjArgs& o, int G, int blocks, double* partials, double* sums,
                            hipStream_t s);

}  // namespace scd
