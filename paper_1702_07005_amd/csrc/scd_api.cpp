// scd_api.cpp -- the C ABI of include/scd.h: handle lifecycle, validation, launch planning,
// objectives and state.  All compute runs in the HIP kernels of scd_epoch.hip, scd_hot.hip and
// scd_setup.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "scd.h"
#include "scd_kernels.h"

using namespace scd;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define HIP_TRY(expr)                                                                            \
    do {                                                                                         \
        hipError_t e_ = (expr);                                                                  \
        if (e_ != hipSuccess)                                                                    \
            return fail(e_ == hipErrorOutOfMemory ? SCD_ERR_OOM : SCD_ERR_HIP, "%s: %s (%s:%d)", \
                        #expr, hipGetErrorString(e_), __FILE__, __LINE__);                       \
    } while (0)

// SplitMix64 (Steele, Lea, Flood 2014): output n (n >= 1) of the generator started at state s.
uint64_t splitmix64(uint64_t s, uint64_t n) {
    uint64_t z = s + 0x9E3779B97F4A7C15ULL * n;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

PermKeys make_perm(uint64_t seed, uint64_t epoch, uint32_t n) {
    PermKeys p{};
    const uint64_t base = splitmix64(seed, epoch + 1);
    for (int r = 0; r < 4; ++r) p.k[r] = (uint32_t)splitmix64(base, (uint64_t)r + 1);
    uint32_t h = 1;
    while (h < 16 && ((uint64_t)1 << (2 * h)) < (uint64_t)n) ++h;
    p.h = h;
    p.mask = (1u << h) - 1u;
    p.n = n;
    return p;
}


constexpr int kBlockThreads = 256;
constexpr int kBlocksPerCU = 8;
constexpr int kGapSlots = 4;
// Window rule: (window - 1) x (worst coordinate's mean squared coupling) <= budget.  The SVM's
// box projection tolerates stale reads far better than the unconstrained ridge steps.
constexpr double kCouplingBudgetSvm = 0.15;
constexpr double kCouplingBudgetRidge = 0.015;
constexpr int kProbes = 8;                // Hutchinson probes of the coupling estimate
// An entry of the shared vector receiving K atomic adds per epoch drifts by about
// sqrt(K) * 2^-24 of its magnitude in fp32; above this many it is kept in fp64 (drift < 1e-5).
constexpr uint32_t kWideHits = 28000;
// The pipelined kernel addresses the shared vector as a raw buffer (byte offsets below 2^31).
constexpr int64_t kPipeMaxBytes = (int64_t(1) << 31) - 8;
// Largest spread copy of the shared vector (64 bytes per entry: up to 4 M entries).
constexpr int64_t kSpreadMaxBytes = int64_t(256) << 20;
// Hot-set kernel: hot entries kept in LDS (sized for an fp64 shared vector next to the largest
// batch buffers), minimum share of stored entries they must cover, and the bound on its waits
// (sleeps of about 64 cycles each: about half a second).
constexpr double kHotMinCover = 0.1;
constexpr uint32_t kHotSpinLimit = 1u << 24;
// Team kernel, automatic choice: segments of at least this many entries on average, and a shared
// vector larger than one XCD's L2 (its gathers miss L2, so a coordinate's time in one workgroup is
// set by that CU's outstanding misses).  Measured at 16-20 coordinates in flight: rows of 1,500
// entries on an 8 MB shared vector, 5.9 ms per epoch in one workgroup each, 3.6 ms in teams of 8;
// the 2,000 x 200 dense ridge (8 KB), 47 us against 82 us; rows of 370 entries, 1.02 ms against
// 1.16 ms.
constexpr double kTeamMinMean = 1024.0;
// ... and segments of about equal length: teams walk positions at a fixed stride, so on skewed
// lengths those that draw long segments fall behind and the processing order drifts from the
// permutation (the queued kernel's case).
constexpr double kTeamMaxSkew = 4.0;  // longest segment at most this many times the mean
constexpr int64_t kTeamMinSharedBytes = int64_t(4) << 20;
// Staged hot-set epochs, automatic choice: matrices whose entries (8 bytes each) exceed the
// 256 MB Infinity Cache, so that the producers' loads go to HBM, and a GPU with CUs for the stagers.
constexpr int64_t kStagedMinBytes = int64_t(256) << 20;

}  // namespace

void scd::set_last_error(const char* msg) { g_err = msg; }

struct scd_solver {
    int form = 0;
    int64_t n_rows = 0, n_cols = 0, nnz = 0, C = 0, L = 0;
    const int64_t* ptr = nullptr;
    const int32_t* idx = nullptr;
    const float* val = nullptr;
    const float* y = nullptr;
    double lambda = 0.0;
    float* model = nullptr;
    void* u = nullptr;  // shared vector: float, or double when `wide`
    int wide = 0;
    uint32_t max_hits = 0;  // most stored entries sharing one shared-vector index
    float* norms = nullptr;
    float* cy = nullptr;  // ridge primal: <y, a_c> per coordinate
    double* cyd = nullptr;  // the same in fp64 (objective evaluation)
    void* dummy = nullptr;  // one zero entry standing in for idx/val of an all-empty matrix
    int* flags = nullptr;
    double* partials = nullptr;
    double* sums = nullptr;
    double* host_sums = nullptr;  // pinned
    // Asynchronous duality-gap slots: pinned sums and a completion event per slot.
    double* slot_sums = nullptr;  // pinned, kGapSlots x 5
    hipEvent_t slot_event[4] = {nullptr, nullptr, nullptr, nullptr};
    int slot_pending[4] = {0, 0, 0, 0};
    int64_t epoch = 0;
    int device = 0;
    int cus = 0;
    size_t max_lds = 0;
    int64_t max_seg = 0;
    double coupling = 0.0, coherence = 0.0;
    int64_t auto_window = 0;
    // options
    int64_t window = 0;
    int64_t group = 0;
    int64_t fresh = 0;
    int64_t pipeline = 1;
    int64_t queue_chunk = 0;  // option: positions per queue claim, 0 = by window
    int64_t spread = 1;       // option: run an unbound pipelined plan on the spread copy
    void* us = nullptr;       // spread copy of the shared vector (entry i at byte i << kSpreadShift),
                              // allocated at create when it takes at most kSpreadMaxBytes
    double* sink = nullptr;  // pipelined kernel, fp64 shared vector: slots inactive lanes add 0 to
    uint32_t* queue = nullptr;  // queued kernel: next position, workgroups finished (zero between launches)
    // Hot-set kernel (windows of at most kHotMaxWindow): built on first need.
    int64_t hot = 1;              // option
    int hot_built = 0;
    int32_t* entry_key = nullptr;    // [nnz]: per stored entry, -1 - its hot slot, or its index when not hot
    int32_t* hot_ids = nullptr;   // [n_hot]
    uint32_t n_hot = 0;
    double hot_cover = 0.0;       // fraction of stored entries that point at a hot entry
    int* hot_err = nullptr;       // device flag set by a timed-out wait in the hot-set kernel
    int64_t adapt = 1;            // option: automatic window of the hot-set kernel follows the moving fraction
    uint32_t* hot_adapt = nullptr;  // [2]: the hot-set kernel's window for the next epoch (device)
    int adapt_fresh = 1;          // the next hot-set epoch starts from the rule's window (state or options changed)
    // Staged hot-set epochs (stager workgroups assemble the batches): ring and flags, allocated with the
    // hot-set tables.
    int64_t staged = 1;           // option: 0 never, 1 automatic (large matrices), 2 whenever the hot set runs
    uint32_t* ring = nullptr;     // [kHotRing][staged_rec_words(cap, Smax)]
    uint32_t* ring_flags = nullptr;  // [kHotFlagWords]
    uint64_t* ring_results = nullptr;  // [kHotResultWords]
    uint32_t* ring_prog = nullptr;   // [4]
    uint32_t ring_tag = 1;        // tag of the next staged launch (never 0)
    int64_t hot_wait_limit = 0;   // option (test hook): sleeps per wait before giving up, 0 = kHotSpinLimit
    int* err_host = nullptr;      // pinned copies of hot_err: one per gap slot + one for reduce_state
    // Team kernel (long segments, few coordinates in flight): tables built on first need for K.
    int64_t team = 1;             // option: 0 never, 1 automatic, 2..kTeamMax members forced
    int team_k = 0;               // K of the built tables (0 = none)
    int32_t* team_idx = nullptr;  // [nnz]: segment entries grouped by index range
    float* team_val = nullptr;    // [nnz]
    uint32_t* team_off = nullptr;  // [C * (K + 1)]
    uint32_t* team_bound = nullptr;  // [K + 1]
    uint64_t* team_slots = nullptr;  // [cus * 2 * kTeamMax] partial-sum slots (tag 0 at allocation)
    uint32_t team_tag = 1;        // tag of the next team step
    // Split kernel (long segments cut into parts, many CUs each): unit tables built on first need for
    // a part length.
    int64_t split = 1;            // option: 0 never, 1 automatic, 2 wherever the queued kernel could run
    int64_t split_part = 0;       // option: entries per part, 0 = kSplitMaxPart
    uint32_t split_built = 0;     // part length of the tables (0 = none)
    uint32_t split_n = 0;         // units per epoch at that part length
    SplitUnit* split_units = nullptr;  // [split_n] records, rewritten by each epoch's pre-pass
    uint64_t* split_partials = nullptr;  // [split_n] tagged partial sums (tag 0 at allocation)
    uint32_t* split_tiles = nullptr;  // [ceil(C / kSplitPrepTile)] pre-pass scratch
    uint32_t split_tag = 1;       // tag of the next split launch (never 0)
};

namespace {

int auto_group(const scd_solver* h) {
    const double mean = h->C > 0 ? (double)h->nnz / (double)h->C : 0.0;
    const int widths[5] = {4, 8, 16, 32, 64};
    for (int G : widths)
        if (mean <= (double)(G * slice_depth(G))) return G;
    return kBlockThreads;  // one workgroup per coordinate
}

int64_t shared_bytes(const scd_solver* h) { return h->L * (int64_t)(h->wide ? sizeof(double) : sizeof(float)); }

// Batch geometry of the hot-set kernel for window W (the first epoch's when adaptive).
struct HotGeom {
    uint32_t W, NC, cap, Smax, hot_bytes;
    bool adaptive;
    size_t lds;
};

// The hot-set kernel's window adapts to the fraction of coordinates that move when the window is
// automatic (the coupling rule assumes that every coordinate in flight moves).
bool hot_adaptive(const scd_solver* h) { return h->window == 0 && h->adapt != 0; }

bool hot_geometry(const scd_solver* h, int64_t W, HotGeom* g) {
    if (W < 2 || W > kHotMaxWindow || h->max_seg > kHotMaxSegment || h->C < 1) return false;
    g->W = (uint32_t)W;
    g->adaptive = hot_adaptive(h);
    // A second consumer wave when the window may exceed what one consumer holds.
    g->NC = (g->adaptive || W > kHotMaxGroups) ? 2u : 1u;
    g->Smax = (uint32_t)std::max<int64_t>(8, (h->max_seg + 7) / 8 * 8);
    g->cap = hot_batch_cap(g->Smax, kHotEntriesPerLane);  // the staged plan's is larger (staged_cap)
    if (g->cap < (uint32_t)kHotMaxGroups) return false;
    g->hot_bytes = (uint32_t)(((size_t)(h->n_hot + kHotZeroCells) * (h->wide ? sizeof(double) : sizeof(float)) + 15) /
                              16 * 16);
    g->lds = hot_lds_bytes(g->hot_bytes, g->cap, g->Smax);
    return true;
}

// Largest hot set that fits LDS next to the largest batch buffers (64 x kStagedEntriesPerLane slots, the
// staged plan's, which exceed the single-workgroup plan's) as
// fp64 entries, so that it stays valid at both widths of the shared vector.
uint32_t hot_capacity(const scd_solver* h) {
    const size_t worst = hot_lds_bytes(0, 64, kStagedEntriesPerLane);
    if (h->max_lds <= worst + 16) return 0;
    const size_t cells = (h->max_lds - worst - 16) / sizeof(double);
    if (cells <= (size_t)kHotZeroCells) return 0;
    return (uint32_t)std::min<size_t>(cells - kHotZeroCells, kHotCold - 1);
}

// Without draining, a pipelined group can have two coordinates in flight (its previous scatter
// may not have landed when it gathers again).  Drain when that would exceed the window; a window
// of at least C does not bind.
int pipe_drain(const scd_solver* h, int64_t window, int64_t groups) {
    return window > 0 && window < h->C && 2 * groups > window ? 1 : 0;
}

// The coupling budget was set with the plain kernels, whose coordinates spend part of each step
// outside the gather-to-scatter interval.  A draining pipelined group keeps its coordinate in that
// interval for nearly the whole step, so at the same window more coordinates are really between
// gather and scatter.  With the automatic window such plans keep 4/5 of it in flight: at full
// text-SVM size (41 -> 32) the worst per-epoch gap ratio to the sequential algorithm over 24 runs
// fell from 2.06 to 1.81.
int64_t pipe_groups(const scd_solver* h, int64_t window, int64_t groups) {
    if (h->window != 0 || !pipe_drain(h, window, groups)) return groups;
    return std::max<int64_t>(1, groups * 4 / 5);
}

// The staged variant: option 2, or option 1 with a matrix beyond the Infinity Cache; it needs its ring and
// enough CUs for the stagers (all on the XCD of the hot-set workgroup).
bool staged_plan(const scd_solver* h) {
    if (h->staged == 0 || !h->ring || h->cus < 1 + kHotXcds * kHotStagers) return false;
    return h->staged == 2 || h->nnz * 8 > kStagedMinBytes;
}

// The staged plan's batches: kStagedEntriesPerLane slots per stager lane.  False if its LDS (the hot
// workgroup's buffers, or the stagers' images) would not fit; the hot set is sized so that it does.
bool staged_geometry(const scd_solver* h, HotGeom* g) {
    const uint32_t cap = hot_batch_cap(g->Smax, kStagedEntriesPerLane);
    if (cap < (uint32_t)kHotMaxGroups || staged_lds_bytes(g->hot_bytes, cap, g->Smax) > h->max_lds) return false;
    g->cap = cap;
    g->lds = hot_lds_bytes(g->hot_bytes, cap, g->Smax);
    return true;
}

bool hot_plan(const scd_solver* h, int64_t window, HotGeom* g) {
    // Its producers read cold values through a raw buffer over the shared vector (below 2 GiB).
    return h->hot && h->group == 0 && h->hot_built && h->n_hot > 0 && h->hot_cover >= kHotMinCover &&
           shared_bytes(h) <= kPipeMaxBytes && hot_geometry(h, window, g) && g->lds <= h->max_lds;
}

// Segment lengths too skewed for the team kernel's fixed-stride walk.
bool skewed_for_teams(const scd_solver* h) {
    return h->C > 0 && (double)h->max_seg > kTeamMaxSkew * ((double)h->nnz / (double)h->C);
}

// Members per in-flight coordinate of the team kernel for the current options, and the number of
// teams (0 = the team kernel does not apply).  Teams hold one coordinate each between gather and
// scatter, as draining pipelined groups do, and take the same share of the window.
int team_members(const scd_solver* h, int64_t* teams) {
    const int64_t window = h->window ? h->window : h->auto_window;
    if (h->team == 0 || !h->pipeline || h->group != 0 || shared_bytes(h) > kPipeMaxBytes || window < 2 ||
        window >= h->C || h->max_seg >= (int64_t(1) << 32) || h->cus < 2)
        return 0;
    int64_t groups = pipe_groups(h, window, std::min<int64_t>(window, (int64_t)h->cus));
    // A team's coordinate stays between its gather and its scatter for a larger part of each step
    // than a pipelined group's (the exchange of partial sums sits in that interval): on the
    // text-SVM twin (3,500 x 166,000) the worst per-epoch gap ratio to the sequential algorithm
    // at a team window of 6 matched the pipelined kernel's at about 8.  With the automatic window
    // teams therefore take 7/8 of the pipelined share (full-size text SVM: 32 -> 28 rows in
    // flight; worst ratio 1.49 over 24 runs of 8 epochs, against 1.80 at 32).
    if (h->window == 0) groups = std::max<int64_t>(1, groups * 7 / 8);
    int64_t K;
    if (skewed_for_teams(h)) return 0;
    if (h->team >= 2) {
        K = h->team;
    } else {
        const double mean = (double)h->nnz / (double)h->C;
        if (mean < kTeamMinMean || shared_bytes(h) < kTeamMinSharedBytes) return 0;
        K = std::min<int64_t>(kTeamMax, h->cus / groups);
    }
    // A member's part beyond the register slices is streamed twice and stays between gather and
    // scatter for several block round trips: as in the queued kernel, the automatic window is
    // then halved (a 1,500 x 166,000 case with 1,500-entry parts reached 2.07x the sequential
    // gap at the undivided share).
    if (h->window == 0 && K >= 2 && (h->max_seg + K - 1) / K > (int64_t)kBlockThreads * kTeamSlices) {
        groups = std::max<int64_t>(1, groups / 2);
        if (h->team < 2) K = std::min<int64_t>(kTeamMax, h->cus / groups);
    }
    if (K < 2 || groups * K > h->cus) return 0;
    *teams = groups;
    return (int)K;
}

uint32_t split_part_len(const scd_solver* h) { return h->split_part ? (uint32_t)h->split_part : kSplitMaxPart; }

// The split kernel's limits: at most kSplitMaxParts parts per segment, fewer than 2^32 units per epoch
// (a bound that does not depend on the permutation: each position yields one unit, or two per part).
bool split_fits(const scd_solver* h, uint32_t part) {
    if (h->split == 0 || h->max_seg > (int64_t)part * kSplitMaxParts) return false;
    const double bound = (double)h->C + 2.0 * ((double)h->nnz / part + (double)h->C);
    return bound < 4.0e9;
}

int plan_epoch(const scd_solver* h, LaunchPlan* lp, uint32_t* n_groups) {
    memset(lp, 0, sizeof *lp);
    lp->fresh = (int)h->fresh;
    const int G = h->group ? (int)h->group : auto_group(h);
    const int64_t window = h->window ? h->window : h->auto_window;
    lp->wide = h->wide;
    const int64_t cap_blocks = (int64_t)h->cus * kBlocksPerCU;
    // The pipelined, queued and split kernels address the shared vector as a raw buffer.
    const bool pipe_ok = h->pipeline && shared_bytes(h) <= kPipeMaxBytes;
    if (h->split == 2 && pipe_ok && h->group == 0 && split_fits(h, split_part_len(h))) {
        // Forced (a test hook): the split kernel with `window` workgroups, also for window 1, where its
        // single workgroup takes the units in order.
        int64_t groups = std::min<int64_t>(window > 0 ? window : cap_blocks, std::min<int64_t>(cap_blocks, h->C));
        groups = std::max<int64_t>(groups, 1);
        lp->kind = PLAN_SPLIT;
        lp->part = split_part_len(h);
        lp->drain = 1;
        lp->chunk = (int)(h->queue_chunk ? h->queue_chunk
                                         : std::min<int64_t>(kQueueChunkMax, std::max<int64_t>(1, groups / 64)));
        lp->group = kBlockThreads;
        lp->blocks = (int)groups;
        *n_groups = (uint32_t)groups;
        return SCD_OK;
    }
    if (window == 1) {
        const size_t need = (size_t)((h->L + 63) & ~int64_t(63)) * (h->wide ? sizeof(double) : sizeof(float)) +
                            2 * 16 * sizeof(float);
        if (need <= h->max_lds) {
            lp->kind = PLAN_ORDERED_LDS;
            lp->L = (uint32_t)h->L;
            lp->lds_bytes = need;
            lp->blocks = 1;
            *n_groups = 1;
            return SCD_OK;
        }
        lp->kind = PLAN_BLOCK;
        lp->ordered = 1;
        lp->fresh = 1;
        lp->blocks = 1;
        *n_groups = 1;
        return SCD_OK;
    }
    // The team kernel first: chosen automatically only for long segments (which the hot-set kernel
    // never takes), and an explicit "team" option is taken as given.
    int64_t teams = 0;
    const int K = team_members(h, &teams);
    if (K && h->team_k == K) {
        lp->kind = PLAN_TEAM;
        lp->team = K;
        lp->group = kBlockThreads;
        lp->drain = 1;
        lp->blocks = team_grid(teams, K);
        *n_groups = (uint32_t)teams;
        return SCD_OK;
    }
    HotGeom hg;
    if (hot_plan(h, window, &hg)) {
        const bool staged = staged_plan(h) && staged_geometry(h, &hg);
        lp->kind = staged ? PLAN_HOT_STAGED : PLAN_HOT;
        lp->group = 8;
        lp->blocks = 1;
        lp->lds_bytes = staged ? staged_lds_bytes(hg.hot_bytes, hg.cap, hg.Smax) : hg.lds;  // hg: staged_geometry's
        // Coordinates in flight at most: what the consumers hold when the window adapts.
        *n_groups = hg.adaptive ? (uint32_t)kHotMaxWindow : hg.W;
        return SCD_OK;
    }
    if (G == kBlockThreads) {
        int64_t groups = cap_blocks;
        if (window > 0 && window < groups) groups = window;
        if (groups > h->C) groups = h->C;
        if (groups < 1) groups = 1;
        if (pipe_ok) groups = pipe_groups(h, window, groups);
        lp->kind = pipe_ok ? PLAN_PIPE : PLAN_BLOCK;
        lp->drain = pipe_drain(h, window, groups);
        lp->unbound = window >= h->C;
        lp->group = kBlockThreads;
        lp->blocks = (int)groups;
        *n_groups = (uint32_t)groups;
        return SCD_OK;
    }
    const int64_t per_block = kBlockThreads / G;
    int64_t groups = cap_blocks * per_block;
    if (window > 0 && window < groups) groups = window;
    if (groups > h->C) groups = h->C;
    if (groups < 1) groups = 1;
    // Segments longer than twice the group's register cache would keep their gather-to-scatter
    // interval open far longer than the others.
    const int64_t long_len = 2 * (int64_t)G * slice_depth(G);
    const bool skewed = h->max_seg > long_len;
    if (pipe_ok && skewed && h->group == 0 && groups <= cap_blocks) {
        // Few coordinates in flight and skewed lengths: each in-flight coordinate gets a workgroup
        // of its own, so a long segment is streamed by 256 lanes without holding up others, and
        // the workgroups take positions from a queue, so that those that draw long segments do
        // not fall behind the permutation order.  The plain kernel for this case serialises long
        // segments inside a workgroup instead.
        // A segment beyond the register slices is streamed in blocks and stays between its
        // gather and its scatter for several block round trips, not one: such coordinates (the
        // densest columns, which couple most strongly with each other) overlap more of the
        // others.  With every column fitting the slices the default window kept the per-epoch gap
        // within 1.06x of the sequential algorithm's (30 runs, text-ridge 3,500 x 166,000); at
        // full size (columns of up to 350,000 entries) the same rule went past 2x in 5 runs of 12,
        // half of it in none.
        const uint32_t part = split_part_len(h);
        const bool split = h->split == 1 && split_fits(h, part) && h->max_seg > (int64_t)part;
        if (!split && h->window == 0 && h->max_seg > (int64_t)kBlockThreads * kQueueSlices)
            groups = std::max<int64_t>(1, groups / 2);
        // The split kernel cuts such segments into parts that many workgroups gather and scatter side
        // by side, so a dense column is in flight for about two unit steps: the window is kept.
        lp->kind = split ? PLAN_SPLIT : PLAN_QUEUE;
        lp->part = part;
        lp->drain = 1;
        // One counter serves about 8e7 claims per second; a workgroup claims about once per
        // 2-4 us, so every 64 workgroups share one claim per step.
        lp->chunk = (int)(h->queue_chunk ? h->queue_chunk
                                         : std::min<int64_t>(kQueueChunkMax, std::max<int64_t>(1, groups / 64)));
        lp->group = kBlockThreads;
        lp->blocks = (int)groups;
        *n_groups = (uint32_t)groups;
        return SCD_OK;
    }
    lp->kind = skewed ? PLAN_MIXED : PLAN_GROUP;
    lp->long_len = (uint32_t)long_len;
    lp->tail = h->max_seg > (int64_t)G * slice_depth(G);
    if (lp->kind == PLAN_GROUP) lp->drain = pipe_drain(h, window, groups);
    if (!skewed && pipe_ok) {
        groups = pipe_groups(h, window, groups);
        lp->kind = PLAN_PIPE;  // segments beyond the slices take its long path
        lp->drain = pipe_drain(h, window, groups);
        lp->unbound = window >= h->C;
    }
    lp->group = G;
    lp->blocks = (int)((groups + per_block - 1) / per_block);
    if (lp->kind == PLAN_MIXED) {
        // Each workgroup takes ceil(groups / blocks) positions per batch.
        const int64_t ng = (groups + lp->blocks - 1) / lp->blocks;
        groups = ng * lp->blocks;
    }
    *n_groups = (uint32_t)groups;
    return SCD_OK;
}

// Number of entries with at least T hits, and the sum of their hits (synchronises).
int hot_count(scd_solver* h, const unsigned* hits, unsigned T, unsigned long long* dev2, hipStream_t s,
              unsigned long long* count, unsigned long long* sum) {
    unsigned long long host2[2] = {0, 0};
    HIP_TRY(hipMemsetAsync(dev2, 0, 2 * sizeof(unsigned long long), s));
    HIP_TRY(launch_hot_count_ge(hits, h->L, T, dev2, s));
    HIP_TRY(hipMemcpyAsync(host2, dev2, sizeof host2, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    *count = host2[0];
    *sum = host2[1];
    return SCD_OK;
}

// Hot set of the hot-set kernel: the entries with at least T stored entries pointing at them (T
// the smallest threshold that keeps the set within LDS capacity), slots in index order, so the
// set is a deterministic function of the matrix.  Built once, on first need; synchronises.
int build_hot_tables(scd_solver* h, hipStream_t s) {
    if (h->hot_built) return SCD_OK;
    h->hot_built = 1;  // a set that cannot help (n_hot = 0) is not retried
    const uint32_t cap = hot_capacity(h);
    if (cap == 0 || h->nnz == 0 || h->max_seg > kHotMaxSegment || h->max_hits == 0) return SCD_OK;
    unsigned* hits = nullptr;
    unsigned long long* dev2 = nullptr;
    unsigned* blocks = nullptr;
    uint16_t* slot_of = nullptr;  // [L]: slot of each shared-vector entry, kHotCold when not hot
    bool skip = false;
    const int64_t nblk = (h->L + kHotAssignBlock - 1) / kHotAssignBlock;
    int rc = SCD_OK;
    auto hip = [&](hipError_t e, const char* what) {
        if (rc == SCD_OK && e != hipSuccess)
            rc = fail(e == hipErrorOutOfMemory ? SCD_ERR_OOM : SCD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
        return rc == SCD_OK;
    };
    hip(hipMalloc(&hits, sizeof(unsigned) * (size_t)h->L), "hipMalloc(hits)");
    hip(hipMalloc(&dev2, 2 * sizeof(unsigned long long)), "hipMalloc(counts)");
    hip(hipMalloc(&blocks, sizeof(unsigned) * (size_t)nblk), "hipMalloc(block counts)");
    if (rc == SCD_OK) {
        hip(hipMemsetAsync(hits, 0, sizeof(unsigned) * (size_t)h->L, s), "zero hits");
        hip(launch_count_hits(h->idx, h->nnz, hits, s), "count hits");
    }
    // Smallest T in [1, max_hits + 1] with count(hits >= T) <= cap (count at max_hits + 1 is 0).
    unsigned lo = 1, hi = h->max_hits + 1;
    unsigned long long cnt = 0, sum = 0;
    while (rc == SCD_OK && lo < hi) {
        const unsigned mid = lo + (hi - lo) / 2;
        if (int r = hot_count(h, hits, mid, dev2, s, &cnt, &sum)) rc = r;
        else if (cnt <= cap) hi = mid;
        else lo = mid + 1;
    }
    if (rc == SCD_OK && (rc = hot_count(h, hits, lo, dev2, s, &cnt, &sum)) == SCD_OK && cnt > 0) {
        std::vector<unsigned> base((size_t)nblk);
        hip(launch_hot_block_count(hits, h->L, lo, blocks, s), "hot block counts");
        hip(hipMemcpyAsync(base.data(), blocks, sizeof(unsigned) * (size_t)nblk, hipMemcpyDeviceToHost, s),
            "copy block counts");
        hip(hipStreamSynchronize(s), "synchronize");
        unsigned run = 0;
        for (auto& b : base) {
            const unsigned c = b;
            b = run;
            run += c;
        }
        hip(hipMemcpyAsync(blocks, base.data(), sizeof(unsigned) * (size_t)nblk, hipMemcpyHostToDevice, s),
            "copy block bases");
        hip(hipMalloc(&slot_of, sizeof(uint16_t) * (size_t)h->L), "hipMalloc(slot_of)");
        hip(hipMalloc(&h->hot_ids, sizeof(int32_t) * (size_t)cnt), "hipMalloc(hot_ids)");
        hip(launch_hot_assign(hits, h->L, lo, blocks, slot_of, h->hot_ids, s), "hot slots");
        // Each stored entry's key (-1 - hot slot, or its index), which the producers read in place of
        // idx (4 bytes per entry).  Without the memory for it the hot-set kernel is not used.
        if (rc == SCD_OK) {
            const hipError_t e = hipMalloc(&h->entry_key, sizeof(int32_t) * (size_t)h->nnz);
            if (e == hipErrorOutOfMemory) {
                (void)hipGetLastError();
                h->entry_key = nullptr;
                skip = true;
            } else {
                hip(e, "hipMalloc(entry_key)");
            }
        }
        if (rc == SCD_OK && !skip) hip(launch_hot_entry_keys(h->idx, h->nnz, slot_of, h->entry_key, s), "entry keys");
        hip(hipStreamSynchronize(s), "synchronize");
        if (rc == SCD_OK && !skip) {
            h->n_hot = (uint32_t)cnt;
            h->hot_cover = (double)sum / (double)h->nnz;
            // The staged variant's ring (a few hundred KB); without it only the single-workgroup kernel runs.
            const uint32_t Smax = (uint32_t)std::max<int64_t>(8, (h->max_seg + 7) / 8 * 8);
            const uint32_t cap = hot_batch_cap(Smax, kStagedEntriesPerLane);
            const size_t ring_bytes = sizeof(uint32_t) * (size_t)kHotRing * staged_rec_words(cap, Smax);
            if (hipMalloc(&h->ring, ring_bytes) != hipSuccess ||
                hipMalloc(&h->ring_flags, sizeof(uint32_t) * kHotFlagWords) != hipSuccess ||
                hipMalloc(&h->ring_results, sizeof(uint64_t) * kHotResultWords) != hipSuccess ||
                hipMalloc(&h->ring_prog, 4 * sizeof(uint32_t)) != hipSuccess) {
                (void)hipGetLastError();
                (void)hipFree(h->ring);
                (void)hipFree(h->ring_flags);
                (void)hipFree(h->ring_results);
                (void)hipFree(h->ring_prog);
                h->ring = nullptr;
                h->ring_flags = nullptr;
                h->ring_results = nullptr;
                h->ring_prog = nullptr;
            } else {
                hip(hipMemsetAsync(h->ring_prog, 0, 4 * sizeof(uint32_t), s), "zero ring_prog");
            }
        }
    }
    (void)hipFree(hits);
    (void)hipFree(dev2);
    (void)hipFree(blocks);
    (void)hipFree(slot_of);
    if (rc != SCD_OK || skip) {
        (void)hipFree(h->entry_key);
        (void)hipFree(h->hot_ids);
        h->entry_key = nullptr;
        h->hot_ids = nullptr;
        h->n_hot = 0;
    }
    return rc;
}

// Builds the hot set when the current options would use the hot-set kernel.
int hot_if_needed(scd_solver* h, hipStream_t s) {
    const int64_t window = h->window ? h->window : h->auto_window;
    HotGeom g;
    if (!h->hot || h->group != 0 || h->hot_built || !hot_geometry(h, window, &g)) return SCD_OK;
    return build_hot_tables(h, s);
}

void free_team_tables(scd_solver* h) {
    (void)hipFree(h->team_idx);
    (void)hipFree(h->team_val);
    (void)hipFree(h->team_off);
    (void)hipFree(h->team_bound);
    h->team_idx = nullptr;
    h->team_val = nullptr;
    h->team_off = nullptr;
    h->team_bound = nullptr;
    h->team_k = 0;
}

// Tables of the team kernel for K members: index-range bounds with about nnz/K stored entries per
// range, and a copy of the segments with each segment's entries grouped by range.  Built once per
// K, on first need (synchronises).  Without memory for the copy the team kernel is not used.
int build_team_tables(scd_solver* h, int K, hipStream_t s) {
    if (h->team_k == K) return SCD_OK;
    free_team_tables(h);
    size_t free_b = 0, total_b = 0;
    HIP_TRY(hipMemGetInfo(&free_b, &total_b));
    const size_t nnz1 = (size_t)std::max<int64_t>(h->nnz, 1);
    const size_t need = nnz1 * 8 + (size_t)h->C * (K + 1) * 4 + sizeof(unsigned) * (size_t)h->L;
    if (need + (size_t(1) << 30) > free_b) return SCD_OK;
    if (!h->team_slots) {
        const size_t sb = sizeof(uint64_t) * 2 * kTeamMax * (size_t)h->cus;
        HIP_TRY(hipMalloc(&h->team_slots, sb));
        HIP_TRY(hipMemsetAsync(h->team_slots, 0, sb, s));
    }
    unsigned* hits = nullptr;
    // Without memory for the tables the other kernels run instead: an allocation that fails here
    // (after the check above, e.g. by fragmentation) is not an error of the calling function.
    const bool got = hipMalloc(&hits, sizeof(unsigned) * (size_t)h->L) == hipSuccess &&
                     hipMalloc(&h->team_idx, sizeof(int32_t) * nnz1) == hipSuccess &&
                     hipMalloc(&h->team_val, sizeof(float) * nnz1) == hipSuccess &&
                     hipMalloc(&h->team_off, sizeof(uint32_t) * (size_t)h->C * (K + 1)) == hipSuccess &&
                     hipMalloc(&h->team_bound, sizeof(uint32_t) * (K + 1)) == hipSuccess;
    if (!got) {
        (void)hipGetLastError();  // clear the allocation failure
        (void)hipFree(hits);
        free_team_tables(h);
        return SCD_OK;
    }
    int rc = SCD_OK;
    auto hip = [&](hipError_t e, const char* what) {
        if (rc == SCD_OK && e != hipSuccess) rc = fail(SCD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    };
    std::vector<unsigned> hh;
    if (rc == SCD_OK) {
        hip(hipMemsetAsync(hits, 0, sizeof(unsigned) * (size_t)h->L, s), "zero team hits");
        if (h->nnz > 0) hip(launch_count_hits(h->idx, h->nnz, hits, s), "count hits");
        hh.resize((size_t)h->L);
        hip(hipMemcpyAsync(hh.data(), hits, sizeof(unsigned) * (size_t)h->L, hipMemcpyDeviceToHost, s), "copy hits");
        hip(hipStreamSynchronize(s), "synchronize");
    }
    if (rc == SCD_OK) {
        // bound[q] = the first index whose preceding entries number at least q * nnz / K.
        std::vector<uint32_t> bound((size_t)K + 1, (uint32_t)h->L);
        bound[0] = 0;
        const double total = (double)h->nnz;
        double cum = 0.0;
        int q = 1;
        for (int64_t i = 0; i < h->L && q < K; ++i) {
            while (q < K && cum * K >= q * total) bound[(size_t)q++] = (uint32_t)i;
            cum += hh[(size_t)i];
        }
        hip(hipMemcpyAsync(h->team_bound, bound.data(), sizeof(uint32_t) * (K + 1), hipMemcpyHostToDevice, s),
            "copy team bounds");
        hip(launch_team_partition(h->ptr, h->idx, h->val, (uint32_t)h->C, h->team_bound, K, h->team_idx, h->team_val,
                                  h->team_off, s),
            "team partition");
        hip(hipStreamSynchronize(s), "synchronize");
    }
    (void)hipFree(hits);
    if (rc != SCD_OK) {
        free_team_tables(h);
        return rc;
    }
    h->team_k = K;
    return SCD_OK;
}

// Builds the team tables when the current options would use the team kernel.
int team_if_needed(scd_solver* h, hipStream_t s) {
    int64_t teams = 0;
    const int K = team_members(h, &teams);
    if (!K || h->team_k == K) return SCD_OK;
    return build_team_tables(h, K, s);
}

void free_split_tables(scd_solver* h) {
    (void)hipFree(h->split_units);
    (void)hipFree(h->split_partials);
    (void)hipFree(h->split_tiles);
    h->split_units = nullptr;
    h->split_partials = nullptr;
    h->split_tiles = nullptr;
    h->split_built = 0;
    h->split_n = 0;
}

// Unit tables of the split kernel for part length `part`: the number of units per epoch (the same
// for every permutation), the records the pre-pass rewrites each epoch, the tagged partial sums and
// the pre-pass's tile counts.  Built once per part length (synchronises).
int build_split_tables(scd_solver* h, uint32_t part, hipStream_t s) {
    if (h->split_built == part) return SCD_OK;
    free_split_tables(h);
    unsigned long long* total = nullptr;
    unsigned long long n = 0;
    HIP_TRY(hipMalloc(&total, sizeof *total));
    hipError_t e = launch_split_total(h->ptr, (uint32_t)h->C, part, total, s);
    if (e == hipSuccess) e = hipMemcpyAsync(&n, total, sizeof n, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(total);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "split unit count: %s", hipGetErrorString(e));
    if (n == 0 || n >= 0xFFFFFFFFull) return fail(SCD_ERR_UNSUPPORTED, "split kernel: %llu units per epoch", n);
    const size_t tiles = (size_t)((h->C + kSplitPrepTile - 1) / kSplitPrepTile);
    e = hipMalloc(&h->split_units, sizeof(SplitUnit) * (size_t)n);
    if (e == hipSuccess) e = hipMalloc(&h->split_partials, sizeof(uint64_t) * (size_t)n);
    if (e == hipSuccess) e = hipMalloc(&h->split_tiles, sizeof(uint32_t) * std::max<size_t>(tiles, 1));
    if (e == hipSuccess) e = hipMemsetAsync(h->split_partials, 0, sizeof(uint64_t) * (size_t)n, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        free_split_tables(h);
        return fail(SCD_ERR_HIP, "split tables (%llu units): %s", n, hipGetErrorString(e));
    }
    h->split_built = part;
    h->split_n = (uint32_t)n;
    h->split_tag = 1;
    return SCD_OK;
}

// Builds the split tables when the current options would use the split kernel.
int split_if_needed(scd_solver* h, hipStream_t s) {
    LaunchPlan lp;
    uint32_t n_groups = 1;
    if (plan_epoch(h, &lp, &n_groups) != SCD_OK || lp.kind != PLAN_SPLIT) return SCD_OK;
    return build_split_tables(h, lp.part, s);
}

int check_hot_err(int v) {
    if (v)
        return fail(SCD_ERR_HIP,
                    "epoch kernel: a bounded wait (between the hot-set kernel's waves, the team kernel's members or "
                    "the split kernel's parts) timed out; the state is invalid");
    return SCD_OK;
}

int obj_group(const scd_solver* h) {
    const int G = h->group ? (int)h->group : auto_group(h);
    return G > 64 ? 64 : G;
}

int obj_blocks(const scd_solver* h, int G) { return objective_blocks(h->C, G); }

int check_handle(scd_handle_t h) {
    if (!h) return fail(SCD_ERR_INVALID, "null handle");
    return SCD_OK;
}

int set_device(const scd_solver* h) {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != h->device) HIP_TRY(hipSetDevice(h->device));
    return SCD_OK;
}

void release(scd_solver* h) {
    if (!h) return;
    (void)hipFree(h->model);
    (void)hipFree(h->u);
    (void)hipFree(h->norms);
    (void)hipFree(h->cy);
    (void)hipFree(h->cyd);
    (void)hipFree(h->dummy);
    (void)hipFree(h->flags);
    (void)hipFree(h->partials);
    (void)hipFree(h->sums);
    (void)hipFree(h->sink);
    (void)hipFree(h->us);
    (void)hipFree(h->queue);
    (void)hipFree(h->hot_adapt);
    (void)hipFree(h->ring);
    (void)hipFree(h->ring_flags);
    (void)hipFree(h->ring_results);
    (void)hipFree(h->ring_prog);
    (void)hipFree(h->entry_key);
    (void)hipFree(h->hot_ids);
    (void)hipFree(h->hot_err);
    free_team_tables(h);
    free_split_tables(h);
    (void)hipFree(h->team_slots);
    (void)hipHostFree(h->err_host);
    if (h->host_sums) (void)hipHostFree(h->host_sums);
    if (h->slot_sums) (void)hipHostFree(h->slot_sums);
    for (hipEvent_t& e : h->slot_event)
        if (e) (void)hipEventDestroy(e);
    delete h;
}

// Enqueue the five reduction sums of the current state and their copy into host[0..4].
int enqueue_sums(scd_solver* h, hipStream_t s, double* host) {
    ObjArgs o{};
    o.ptr = h->ptr;
    o.idx = h->idx;
    o.val = h->val;
    o.u = h->u;
    o.wide = h->wide;
    o.model = h->model;
    o.y = h->form == FORM_RIDGE_PRIMAL ? nullptr : h->y;
    o.yv = h->form == FORM_RIDGE_PRIMAL ? h->y : nullptr;
    o.cyd = h->cyd;
    o.C = (uint32_t)h->C;
    o.L = h->L;
    o.lam = h->lambda;
    const int G = obj_group(h);
    const int blocks = obj_blocks(h, G);
    HIP_TRY(launch_objective(h->form, o, G, blocks, h->partials, h->sums, s));
    HIP_TRY(hipMemcpyAsync(host, h->sums, 5 * sizeof(double), hipMemcpyDeviceToHost, s));
    return SCD_OK;
}

// The same, waiting for the result in h->host_sums.
int reduce_state(scd_solver* h, hipStream_t s) {
    if (int r = enqueue_sums(h, s, h->host_sums)) return r;
    HIP_TRY(hipMemcpyAsync(h->err_host + kGapSlots, h->hot_err, sizeof(int), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return check_hot_err(h->err_host[kGapSlots]);
}

void objectives_from_sums(const scd_solver* h, const double* t, double* P, double* D) {
    scd::objectives_from_sums(h->form, (double)h->n_rows, h->lambda, t, P, D);
}

}  // namespace

extern "C" {

const char* scd_last_error(void) { return g_err.c_str(); }

int scd_create(const scd_matrix_t* A, const float* y, double lambda, int32_t formulation, void* stream,
               scd_handle_t* out) {
    g_err.clear();
    if (!out) return fail(SCD_ERR_INVALID, "out is null");
    *out = nullptr;
    if (!A) return fail(SCD_ERR_INVALID, "matrix is null");
    if (formulation < SCD_RIDGE_PRIMAL || formulation > SCD_RIDGE_DUAL)
        return fail(SCD_ERR_INVALID, "unknown formulation %d", (int)formulation);
    const int want = formulation == SCD_RIDGE_PRIMAL ? SCD_CSC : SCD_CSR;
    if (A->layout != want)
        return fail(SCD_ERR_INVALID, "formulation %d needs layout %s", (int)formulation,
                    want == SCD_CSC ? "CSC (columns = coordinates)" : "CSR (rows = coordinates)");
    if (A->n_rows < 1 || A->n_cols < 1 || A->nnz < 0)
        return fail(SCD_ERR_INVALID, "bad sizes n_rows=%lld n_cols=%lld nnz=%lld", (long long)A->n_rows,
                    (long long)A->n_cols, (long long)A->nnz);
    if (A->n_rows > 2147483647LL || A->n_cols > 2147483647LL)
        return fail(SCD_ERR_INVALID, "dimensions must be below 2^31");
    if (!A->ptr || (A->nnz > 0 && (!A->idx || !A->val)) || !y)
        return fail(SCD_ERR_INVALID, "null device pointer");
    if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail(SCD_ERR_INVALID, "lambda must be finite and > 0");

    scd_solver* h = new (std::nothrow) scd_solver;
    if (!h) return fail(SCD_ERR_OOM, "host allocation failed");
    h->form = formulation;
    h->n_rows = A->n_rows;
    h->n_cols = A->n_cols;
    h->nnz = A->nnz;
    h->C = formulation == SCD_RIDGE_PRIMAL ? A->n_cols : A->n_rows;
    h->L = formulation == SCD_RIDGE_PRIMAL ? A->n_rows : A->n_cols;
    h->ptr = A->ptr;
    h->idx = A->idx;
    h->val = A->val;
    h->y = y;
    h->lambda = lambda;
    hipStream_t s = (hipStream_t)stream;

    int rc = SCD_OK;
    auto step = [&](int r) { if (rc == SCD_OK) rc = r; return rc == SCD_OK; };
    auto hip = [&](hipError_t e, const char* what) {
        if (rc != SCD_OK) return false;
        if (e != hipSuccess) rc = fail(e == hipErrorOutOfMemory ? SCD_ERR_OOM : SCD_ERR_HIP, "%s: %s", what,
                                       hipGetErrorString(e));
        return rc == SCD_OK;
    };
    hip(hipGetDevice(&h->device), "hipGetDevice");
    if (rc == SCD_OK) {
        hipDeviceProp_t prop;
        if (hip(hipGetDeviceProperties(&prop, h->device), "hipGetDeviceProperties")) {
            h->cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 1;
            h->max_lds = prop.sharedMemPerBlock;
            int v = 0;
            if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device) == hipSuccess &&
                (size_t)v > h->max_lds)
                h->max_lds = (size_t)v;
        }
    }
    hip(hipMalloc(&h->model, sizeof(float) * (size_t)h->C), "hipMalloc(model)");
    hip(hipMalloc(&h->u, sizeof(float) * (size_t)h->L), "hipMalloc(shared)");
    hip(hipMalloc(&h->norms, sizeof(float) * (size_t)h->C), "hipMalloc(norms)");
    if (formulation == SCD_RIDGE_PRIMAL) {
        hip(hipMalloc(&h->cy, sizeof(float) * (size_t)h->C), "hipMalloc(cy)");
        hip(hipMalloc(&h->cyd, sizeof(double) * (size_t)h->C), "hipMalloc(cyd)");
    }

    hip(hipMalloc(&h->flags, 2 * sizeof(int64_t)), "hipMalloc(flags)");
    if (h->nnz == 0) {
        // The epoch kernels read element 0 of idx/val unconditionally (weight 0 when unused).
        hip(hipMalloc(&h->dummy, 8), "hipMalloc(dummy)");
        hip(hipMemsetAsync(h->dummy, 0, 8, s), "zero dummy");
        h->idx = static_cast<const int32_t*>(h->dummy);
        h->val = static_cast<const float*>(h->dummy);
    }
    hip(hipMalloc(&h->partials, sizeof(double) * (size_t)kObjBlocksMax * 5), "hipMalloc(partials)");
    hip(hipMalloc(&h->sums, sizeof(double) * 8), "hipMalloc(sums)");
    hip(hipMalloc(&h->hot_err, sizeof(int)), "hipMalloc(hot_err)");
    hip(hipMemsetAsync(h->hot_err, 0, sizeof(int), s), "zero hot_err");
    hip(hipHostMalloc(&h->err_host, sizeof(int) * (kGapSlots + 1), hipHostMallocDefault), "hipHostMalloc(err)");
    if (rc == SCD_OK) memset(h->err_host, 0, sizeof(int) * (kGapSlots + 1));
    if (rc == SCD_OK) {
        const size_t sink_bytes = sizeof(double) * 256 * (size_t)h->cus * kBlocksPerCU;
        hip(hipMalloc(&h->sink, sink_bytes), "hipMalloc(sink)");
        hip(hipMemsetAsync(h->sink, 0, sink_bytes, s), "zero sink");
        hip(hipMalloc(&h->queue, 2 * sizeof(uint32_t)), "hipMalloc(queue)");
        hip(hipMalloc(&h->hot_adapt, 2 * sizeof(uint32_t)), "hipMalloc(hot_adapt)");
        hip(hipMemsetAsync(h->hot_adapt, 0, 2 * sizeof(uint32_t), s), "zero hot_adapt");
        if ((h->L << kSpreadShift) <= kSpreadMaxBytes) hip(hipMalloc(&h->us, (size_t)h->L << kSpreadShift), "hipMalloc(spread)");
        hip(hipMemsetAsync(h->queue, 0, 2 * sizeof(uint32_t), s), "zero queue");
    }
    hip(hipHostMalloc(&h->host_sums, sizeof(double) * 8, hipHostMallocDefault), "hipHostMalloc");
    hip(hipHostMalloc(&h->slot_sums, sizeof(double) * 5 * kGapSlots, hipHostMallocDefault), "hipHostMalloc(slots)");
    for (int i = 0; i < kGapSlots; ++i)
        hip(hipEventCreateWithFlags(&h->slot_event[i], hipEventDisableTiming), "hipEventCreate");

    // Validation pass over ptr, idx, val and y.
    int64_t fl[2] = {0, 0};  // validation bits, longest segment
    hip(hipMemsetAsync(h->flags, 0, 2 * sizeof(int64_t), s), "hipMemsetAsync(flags)");
    hip(launch_validate(h->ptr, (uint32_t)h->C, h->idx, h->val, h->nnz, h->L, h->y, h->n_rows,
                        formulation == SCD_SVM_DUAL, h->flags, s),
        "validate");
    hip(hipMemcpyAsync(fl, h->flags, 2 * sizeof(int64_t), hipMemcpyDeviceToHost, s), "copy flags");
    hip(hipStreamSynchronize(s), "synchronize");
    const int flags = (int)(fl[0] & 0xFFFFFFFF);
    h->max_seg = fl[1];
    if (rc == SCD_OK && flags) {
        if (flags & 1) step(fail(SCD_ERR_INVALID, "ptr must start at 0, end at nnz and be non-decreasing"));
        else if (flags & 2) step(fail(SCD_ERR_INVALID, "an index is outside [0, %lld)", (long long)h->L));
        else if (flags & 16) step(fail(SCD_ERR_INVALID, "SVM labels must be -1 or +1"));
        else step(fail(SCD_ERR_NUMERIC, "non-finite matrix value or label"));
    }
    if (rc == SCD_OK) {
        // Largest number of updates one shared-vector entry receives per epoch (h->u as counters).
        unsigned* hits = static_cast<unsigned*>(h->u);
        hip(hipMemsetAsync(hits, 0, sizeof(unsigned) * (size_t)h->L, s), "zero hits");
        hip(hipMemsetAsync(h->flags, 0, sizeof(unsigned), s), "zero max hits");
        hip(launch_max_hits(h->idx, h->nnz, h->L, hits, reinterpret_cast<unsigned*>(h->flags), s), "count hits");
        hip(hipMemcpyAsync(&h->max_hits, h->flags, sizeof(unsigned), hipMemcpyDeviceToHost, s), "copy hits");
        hip(hipStreamSynchronize(s), "synchronize");
        if (rc == SCD_OK && h->max_hits > kWideHits) {
            h->wide = 1;
            (void)hipFree(h->u);
            h->u = nullptr;
            hip(hipMalloc(&h->u, sizeof(double) * (size_t)h->L), "hipMalloc(shared, fp64)");
        }
    }
    if (rc == SCD_OK) {
        const int G = obj_group(h);
        hip(launch_norms(h->ptr, h->idx, h->val, formulation == SCD_RIDGE_PRIMAL ? h->y : nullptr, (uint32_t)h->C,
                         G, obj_blocks(h, G), h->norms, h->cy, h->cyd, s),
            "norms");
        // Coupling of the coordinates (sets the default window), using h->u as the probe vector.
        const float mu = formulation == SCD_SVM_DUAL ? 0.0f : (float)(lambda * (double)h->n_rows);
        const float* sign = formulation == SCD_SVM_DUAL ? h->y : nullptr;
        // Probe 0 (all-ones): sum of G's entries, sum of its diagonal, non-empty coordinates.
        // Probes 1..kProbes (Rademacher): per-coordinate squared off-diagonal row mass into K = h->model.
        double coh2 = 0.0, diag1 = 0.0, cn = 0.0;
        hip(hipMemsetAsync(h->model, 0, sizeof(float) * (size_t)h->C, s), "zero probe sums");  // K[c]
        for (uint32_t probe = 0; probe <= (uint32_t)kProbes && rc == SCD_OK; ++probe) {
            hip(launch_probe(h->ptr, h->idx, h->val, h->norms, sign, (uint32_t)h->C, h->L, mu, probe, G,
                             obj_blocks(h, G), static_cast<float*>(h->u), h->model, h->partials, h->sums, s),
                "coupling probe");
            hip(hipMemcpyAsync(h->host_sums, h->sums, 4 * sizeof(double), hipMemcpyDeviceToHost, s), "copy probe");
            hip(hipStreamSynchronize(s), "synchronize");
            if (rc != SCD_OK) break;
            if (probe == 0) {
                coh2 = h->host_sums[0];
                diag1 = h->host_sums[2];
                cn = h->host_sums[3];
            }
        }
        unsigned kmax_bits = 0;
        hip(hipMemsetAsync(h->flags, 0, sizeof(unsigned), s), "zero kappa");
        hip(launch_kappa_max(h->model, h->norms, (uint32_t)h->C, kProbes, obj_blocks(h, G),
                             reinterpret_cast<unsigned*>(h->flags), s),
            "kappa max");
        hip(hipMemcpyAsync(&kmax_bits, h->flags, sizeof(unsigned), hipMemcpyDeviceToHost, s), "copy kappa");
        hip(hipStreamSynchronize(s), "synchronize");
        if (rc == SCD_OK) {
            float kmax = 0.0f;
            memcpy(&kmax, &kmax_bits, sizeof kmax);
            const double pairs = cn * (cn - 1.0);
            h->coherence = pairs > 0.0 ? (coh2 - diag1) / pairs : 0.0;
            // Worst coordinate's mean squared coupling to one other coordinate.
            h->coupling = cn > 1.0 ? (double)kmax / (cn - 1.0) : 0.0;
            const double budget = formulation == SCD_SVM_DUAL ? kCouplingBudgetSvm : kCouplingBudgetRidge;
            int64_t w = INT64_MAX;
            if (h->coupling > 0.0) w = 1 + (int64_t)std::min(9.0e18, std::floor(budget / h->coupling));
            if (h->coupling > 1e-6) w = std::min<int64_t>(w, std::max<int64_t>(1, h->C / 16));
            h->auto_window = std::max<int64_t>(1, std::min<int64_t>(w, h->C));
        }
        if (rc == SCD_OK) step(hot_if_needed(h, s));
        if (rc == SCD_OK) step(team_if_needed(h, s));
        if (rc == SCD_OK) step(split_if_needed(h, s));
        hip(hipMemsetAsync(h->model, 0, sizeof(float) * (size_t)h->C, s), "zero model");
        hip(hipMemsetAsync(h->u, 0, (h->wide ? sizeof(double) : sizeof(float)) * (size_t)h->L, s), "zero shared");
        hip(hipStreamSynchronize(s), "synchronize");
    }
    if (rc != SCD_OK) {
        release(h);
        return rc;
    }
    *out = h;
    return SCD_OK;
}

int scd_destroy(scd_handle_t h) {
    if (!h) return SCD_OK;
    const int dev = h->device;
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != dev) (void)hipSetDevice(dev);
    hipError_t e = hipDeviceSynchronize();
    release(h);
    if (cur >= 0 && cur != dev) (void)hipSetDevice(cur);
    if (e != hipSuccess) return fail(SCD_ERR_HIP, "hipDeviceSynchronize: %s", hipGetErrorString(e));
    return SCD_OK;
}

int scd_epochs(scd_handle_t h, uint64_t seed, int32_t n_epochs, void* stream) {
    if (int r = check_handle(h)) return r;
    if (n_epochs < 0) return fail(SCD_ERR_INVALID, "n_epochs must be >= 0");
    if (int r = set_device(h)) return r;
    LaunchPlan lp;
    uint32_t n_groups = 1;
    if (int r = plan_epoch(h, &lp, &n_groups)) return r;
    if (lp.kind == PLAN_ORDERED_LDS) HIP_TRY(ordered_lds_prepare(h->form, lp.wide != 0, lp.lds_bytes));
    if (lp.kind == PLAN_SPLIT)
        if (int r = build_split_tables(h, lp.part, (hipStream_t)stream)) return r;
    HotGeom hg{};
    if (lp.kind == PLAN_HOT || lp.kind == PLAN_HOT_STAGED) {
        hot_plan(h, h->window ? h->window : h->auto_window, &hg);
        if (lp.kind == PLAN_HOT_STAGED) staged_geometry(h, &hg);  // held when the plan was made
        hg.lds = lp.lds_bytes;  // the staged launch's workgroups all get the larger of the two needs
        if (lp.kind == PLAN_HOT)
            HIP_TRY(hot_prepare(h->form, h->wide != 0, hg.Smax, hg.lds));
        else
            HIP_TRY(staged_prepare(h->form, h->wide != 0, hg.Smax, hg.lds));
    }
    EpochArgs a{};
    a.ptr = h->ptr;
    a.idx = h->idx;
    a.val = h->val;
    a.y = h->form == FORM_RIDGE_PRIMAL ? h->cy : h->y;
    a.model = h->model;
    a.u = h->u;
    a.norms = h->norms;
    const double lamN = h->lambda * (double)h->n_rows;
    a.k.lamN = (float)lamN;
    a.k.inv_lamN = (float)(1.0 / lamN);
    a.k.lam = (float)h->lambda;
    a.n_groups = n_groups;
    a.u_bytes = shared_bytes(h) <= kPipeMaxBytes ? (uint32_t)shared_bytes(h) : 0u;
    a.u_shift = h->wide ? 3u : 2u;
    // With every coordinate in flight (the window does not bind) the pipelined kernel runs on the
    // spread copy when there is one: packed, the gathers of entries whose 64-byte segment other
    // coordinates' atomics are updating wait behind those atomics (measured: gather-and-atomic
    // pairs on 100,000 packed fp32 entries at 9.5 G/s, spread one per 64 bytes at 20 G/s, the rate
    // of the atomics alone).  With a binding window the epoch is bound by the latency of the
    // coordinates in flight instead, and a coordinate that gathers many neighbouring entries (a
    // dense column) would touch one segment per entry instead of one per 16.
    const bool spread = h->us && h->spread && lp.kind == PLAN_PIPE && lp.unbound && n_epochs > 0;
    if (spread) {
        a.u = h->us;
        a.u_bytes = (uint32_t)(h->L << kSpreadShift);
        a.u_shift = kSpreadShift;
    }
    a.sink = h->sink;
    a.drain = (uint32_t)lp.drain;
    a.queue = h->queue;
    a.chunk = (uint32_t)std::max(1, lp.chunk);
    hipStream_t s = (hipStream_t)stream;
    if (spread) HIP_TRY(launch_spread(h->u, h->us, h->L, h->wide != 0, true, s));
    for (int32_t e = 0; e < n_epochs; ++e) {
        a.perm = make_perm(seed, (uint64_t)h->epoch, (uint32_t)h->C);
        if (lp.kind == PLAN_TEAM) {
            TeamArgs ta{};
            ta.e = a;
            ta.e.idx = h->team_idx;
            ta.e.val = h->team_val;
            ta.e.drain = 1;
            ta.off = h->team_off;
            ta.slots = h->team_slots;
            ta.K = (uint32_t)lp.team;
            ta.tag0 = h->team_tag;
            ta.spin_limit = h->hot_wait_limit > 0 ? (uint32_t)h->hot_wait_limit : kHotSpinLimit;
            ta.err = h->hot_err;
            HIP_TRY(launch_epoch_team(h->form, h->wide != 0, lp.fresh != 0, ta, lp.blocks, h->cus, s));
            // Steps of the busiest team, plus one: the next launch's tags are all new.
            h->team_tag += (uint32_t)((h->C + n_groups - 1) / n_groups + 1);
        } else if (lp.kind == PLAN_SPLIT) {
            SplitArgs sa{};
            sa.e = a;
            sa.units = h->split_units;
            sa.partials = h->split_partials;
            sa.n_units = h->split_n;
            sa.tag = h->split_tag;
            sa.spin_limit = h->hot_wait_limit > 0 ? (uint32_t)h->hot_wait_limit : kHotSpinLimit;
            sa.err = h->hot_err;
            HIP_TRY(launch_epoch_split(h->form, h->wide != 0, lp.fresh != 0, sa, lp.part, h->split_tiles, h->split_units,
                                       lp.blocks, s));
            h->split_tag = h->split_tag == 0xFFFFFFFFu ? 1u : h->split_tag + 1u;
        } else if (lp.kind == PLAN_HOT || lp.kind == PLAN_HOT_STAGED) {
            HotArgs ha{};
            ha.e = a;
            ha.entry_key = h->entry_key;
            ha.hot_ids = h->hot_ids;
            ha.n_hot = h->n_hot;
            ha.W = hg.W;
            ha.NC = hg.NC;
            ha.cap = hg.cap;
            ha.Smax = hg.Smax;
            ha.hot_bytes = hg.hot_bytes;
            ha.w_rule = hg.W;
            ha.adapt_out = hg.adaptive ? h->hot_adapt : nullptr;
            ha.spin_limit = h->hot_wait_limit > 0 ? (uint32_t)h->hot_wait_limit : kHotSpinLimit;
            ha.err = h->hot_err;
            // The first epoch after the state or the options changed has no moving fraction to go by:
            // its opening segment (1/kHotOpening of the positions) runs at the rule's window, and the
            // rest at the window that the rule gives from that segment's moving fraction.  Every
            // later epoch is one launch at the window its predecessor left.
            const uint32_t C = (uint32_t)h->C;
            const bool opening = hg.adaptive && h->adapt_fresh && C >= 2 * kHotOpening;
            const uint32_t n_open = opening ? (C + kHotOpening - 1) / kHotOpening : C;
            for (int part = 0; part < (opening ? 2 : 1); ++part) {
                ha.pos0 = part ? n_open : 0u;
                ha.pos_n = part ? C - n_open : n_open;
                ha.adapt_in = hg.adaptive && !h->adapt_fresh ? h->hot_adapt : nullptr;
                h->adapt_fresh = 0;
                if (lp.kind == PLAN_HOT_STAGED) {
                    ha.ring = h->ring;
                    ha.flags = h->ring_flags;
                    ha.results = h->ring_results;
                    ha.prog = h->ring_prog;
                    ha.tag = h->ring_tag;
                    ha.stagers = kHotStagers;
                    h->ring_tag = h->ring_tag == 0xFFFFFFFFu ? 1u : h->ring_tag + 1u;
                    HIP_TRY(launch_epoch_staged(h->form, h->wide != 0, ha, hg.lds, s));
                } else {
                    HIP_TRY(launch_epoch_hot(h->form, h->wide != 0, ha, hg.lds, s));
                }
            }
        } else {
            HIP_TRY(launch_epoch(h->form, a, lp, s));
        }
        ++h->epoch;
    }
    if (spread) HIP_TRY(launch_spread(h->u, h->us, h->L, h->wide != 0, false, s));
    return SCD_OK;
}

int scd_objective(scd_handle_t h, void* stream, double* primal, double* dual) {
    if (int r = check_handle(h)) return r;
    if (int r = set_device(h)) return r;
    if (int r = reduce_state(h, (hipStream_t)stream)) return r;
    double P, D;
    objectives_from_sums(h, h->host_sums, &P, &D);
    if (!std::isfinite(P) || !std::isfinite(D)) return fail(SCD_ERR_NUMERIC, "non-finite objective (P=%g, D=%g)", P, D);
    if (primal) *primal = P;
    if (dual) *dual = D;
    return SCD_OK;
}

int scd_duality_gap(scd_handle_t h, void* stream, double* gap) {
    if (!gap) return fail(SCD_ERR_INVALID, "gap is null");
    double P = 0, D = 0;
    if (int r = scd_objective(h, stream, &P, &D)) return r;
    *gap = h->form == FORM_SVM_DUAL ? P - D : std::fabs(P - D);
    return SCD_OK;
}

int scd_duality_gap_async(scd_handle_t h, void* stream, int32_t slot) {
    if (int r = check_handle(h)) return r;
    if (slot < 0 || slot >= kGapSlots) return fail(SCD_ERR_INVALID, "slot must be in [0, %d)", kGapSlots);
    if (h->slot_pending[slot]) return fail(SCD_ERR_INVALID, "slot %d already holds an unread evaluation", slot);
    if (int r = set_device(h)) return r;
    hipStream_t s = (hipStream_t)stream;
    if (int r = enqueue_sums(h, s, h->slot_sums + 5 * slot)) return r;
    HIP_TRY(hipMemcpyAsync(h->err_host + slot, h->hot_err, sizeof(int), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipEventRecord(h->slot_event[slot], s));
    h->slot_pending[slot] = 1;
    return SCD_OK;
}

int scd_duality_gap_wait(scd_handle_t h, int32_t slot, double* gap, double* primal, double* dual) {
    if (int r = check_handle(h)) return r;
    if (slot < 0 || slot >= kGapSlots) return fail(SCD_ERR_INVALID, "slot must be in [0, %d)", kGapSlots);
    if (!h->slot_pending[slot]) return fail(SCD_ERR_INVALID, "slot %d holds no evaluation", slot);
    h->slot_pending[slot] = 0;
    HIP_TRY(hipEventSynchronize(h->slot_event[slot]));
    if (int r = check_hot_err(h->err_host[slot])) return r;
    double P, D;
    objectives_from_sums(h, h->slot_sums + 5 * slot, &P, &D);
    if (!std::isfinite(P) || !std::isfinite(D)) return fail(SCD_ERR_NUMERIC, "non-finite objective (P=%g, D=%g)", P, D);
    if (gap) *gap = h->form == FORM_SVM_DUAL ? P - D : std::fabs(P - D);
    if (primal) *primal = P;
    if (dual) *dual = D;
    return SCD_OK;
}

int scd_get_state(scd_handle_t h, float* model, float* shared, int64_t* epoch, void* stream) {
    if (int r = check_handle(h)) return r;
    if (int r = set_device(h)) return r;
    hipStream_t s = (hipStream_t)stream;
    if (model) HIP_TRY(hipMemcpyAsync(model, h->model, sizeof(float) * (size_t)h->C, hipMemcpyDeviceToDevice, s));
    if (shared) {
        if (h->wide)
            HIP_TRY(launch_convert_f64_to_f32(static_cast<const double*>(h->u), h->L, shared, s));
        else
            HIP_TRY(hipMemcpyAsync(shared, h->u, sizeof(float) * (size_t)h->L, hipMemcpyDeviceToDevice, s));
    }
    if (epoch) *epoch = h->epoch;
    return SCD_OK;
}

int scd_set_state(scd_handle_t h, const float* model, const float* shared, int64_t epoch, void* stream) {
    if (int r = check_handle(h)) return r;
    if (epoch < 0) return fail(SCD_ERR_INVALID, "epoch must be >= 0");
    if (int r = set_device(h)) return r;
    hipStream_t s = (hipStream_t)stream;
    HIP_TRY(hipMemsetAsync(h->hot_err, 0, sizeof(int), s));  // a written state replaces an invalid one
    h->adapt_fresh = 1;  // the moving fraction of the previous epochs says nothing about this state
    if (model) HIP_TRY(hipMemcpyAsync(h->model, model, sizeof(float) * (size_t)h->C, hipMemcpyDeviceToDevice, s));
    if (shared) {
        if (h->wide)
            HIP_TRY(launch_convert_f32_to_f64(shared, h->L, static_cast<double*>(h->u), s));
        else
            HIP_TRY(hipMemcpyAsync(h->u, shared, sizeof(float) * (size_t)h->L, hipMemcpyDeviceToDevice, s));
    }
    h->epoch = epoch;
    return SCD_OK;
}

int scd_set_option(scd_handle_t h, const char* key, int64_t value) {
    if (int r = check_handle(h)) return r;
    if (!key) return fail(SCD_ERR_INVALID, "key is null");
    h->adapt_fresh = 1;  // the next hot-set epoch starts again from the rule's window
    if (!strcmp(key, "staged")) {
        if (value < 0 || value > 2) return fail(SCD_ERR_INVALID, "staged must be 0, 1 or 2");
        h->staged = value;
    } else if (!strcmp(key, "adapt")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "adapt must be 0 or 1");
        h->adapt = value;
        if (int r = set_device(h)) return r;
        if (int r = hot_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "window")) {
        if (value < 0 || value > 2147483647LL) return fail(SCD_ERR_INVALID, "window must be in [0, 2^31)");
        h->window = value;
        if (int r = set_device(h)) return r;
        if (int r = hot_if_needed(h, nullptr)) return r;
        if (int r = team_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "hot")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "hot must be 0 or 1");
        h->hot = value;
        if (int r = set_device(h)) return r;
        if (int r = hot_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "group")) {
        if (!(value == 0 || value == 4 || value == 8 || value == 16 || value == 32 || value == 64 ||
              value == kBlockThreads))
            return fail(SCD_ERR_INVALID, "group must be 0, 4, 8, 16, 32, 64 or 256");
        h->group = value;
        if (int r = set_device(h)) return r;
        if (int r = hot_if_needed(h, nullptr)) return r;
        if (int r = team_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "team")) {
        if (value < 0 || value > kTeamMax) return fail(SCD_ERR_INVALID, "team must be in [0, %d]", kTeamMax);
        // Teams walk positions at a fixed stride; on skewed segment lengths those that draw long
        // segments fall behind and the processing order drifts from the permutation (a forced team
        // of 4 on the skewed text-ridge columns reached 2.28x the sequential per-epoch gap).
        if (value >= 2 && skewed_for_teams(h))
            return fail(SCD_ERR_UNSUPPORTED,
                        "team %lld: the longest segment (%lld entries) exceeds %.0f times the mean; skewed lengths "
                        "take the queued kernel",
                        (long long)value, (long long)h->max_seg, kTeamMaxSkew);
        h->team = value;
        if (int r = set_device(h)) return r;
        if (int r = team_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "fresh_reads")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "fresh_reads must be 0 or 1");
        h->fresh = value;
    } else if (!strcmp(key, "hot_wait_limit")) {
        if (value < 0 || value > (int64_t)0xFFFFFFFF) return fail(SCD_ERR_INVALID, "hot_wait_limit must be in [0, 2^32)");
        h->hot_wait_limit = value;
    } else if (!strcmp(key, "pipeline")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "pipeline must be 0 or 1");
        h->pipeline = value;
        if (int r = set_device(h)) return r;
        if (int r = team_if_needed(h, nullptr)) return r;
    } else if (!strcmp(key, "spread")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "spread must be 0 or 1");
        h->spread = value;
    } else if (!strcmp(key, "queue_chunk")) {
        if (value < 0 || value > (int64_t)kQueueChunkMax) return fail(SCD_ERR_INVALID, "queue_chunk must be in [0, 64]");
        h->queue_chunk = value;
    } else if (!strcmp(key, "split")) {
        if (value < 0 || value > 2) return fail(SCD_ERR_INVALID, "split must be 0, 1 or 2");
        h->split = value;
    } else if (!strcmp(key, "split_part")) {
        if (value != 0 && (value < 64 || value > (int64_t)kSplitMaxPart || value % 64 != 0))
            return fail(SCD_ERR_INVALID, "split_part must be 0 or a multiple of 64 in [64, %u]", kSplitMaxPart);
        h->split_part = value;
    } else if (!strcmp(key, "shared_fp64")) {
        if (value != 0 && value != 1) return fail(SCD_ERR_INVALID, "shared_fp64 must be 0 or 1");
        if (value == h->wide) return SCD_OK;
        if (int r = set_device(h)) return r;
        // Re-store the shared vector at the other width (synchronises the device).
        void* nu = nullptr;
        HIP_TRY(hipMalloc(&nu, (value ? sizeof(double) : sizeof(float)) * (size_t)h->L));
        hipError_t e = value ? launch_convert_f32_to_f64(static_cast<const float*>(h->u), h->L,
                                                         static_cast<double*>(nu), nullptr)
                             : launch_convert_f64_to_f32(static_cast<const double*>(h->u), h->L,
                                                         static_cast<float*>(nu), nullptr);
        if (e == hipSuccess) e = hipDeviceSynchronize();
        if (e != hipSuccess) {
            (void)hipFree(nu);
            return fail(SCD_ERR_HIP, "shared_fp64 conversion: %s", hipGetErrorString(e));
        }
        (void)hipFree(h->u);
        h->u = nu;
        h->wide = (int)value;
        if (int r = team_if_needed(h, nullptr)) return r;
    } else {
        return fail(SCD_ERR_UNSUPPORTED, "unknown option '%s'", key);
    }
    if (int r = set_device(h)) return r;
    return split_if_needed(h, nullptr);
}

int scd_get_option(scd_handle_t h, const char* key, int64_t* value) {
    if (int r = check_handle(h)) return r;
    if (!key || !value) return fail(SCD_ERR_INVALID, "null argument");
    if (!strcmp(key, "window")) *value = h->window;
    else if (!strcmp(key, "group")) *value = h->group;
    else if (!strcmp(key, "fresh_reads")) *value = h->fresh;
    else if (!strcmp(key, "pipeline")) *value = h->pipeline;
    else if (!strcmp(key, "spread")) *value = h->spread;
    else if (!strcmp(key, "queue_chunk")) *value = h->queue_chunk;
    else if (!strcmp(key, "split")) *value = h->split;
    else if (!strcmp(key, "split_part")) *value = h->split_part;
    else if (!strcmp(key, "hot")) *value = h->hot;
    else if (!strcmp(key, "hot_wait_limit")) *value = h->hot_wait_limit;
    else if (!strcmp(key, "team")) *value = h->team;
    else if (!strcmp(key, "shared_fp64")) *value = h->wide;
    else if (!strcmp(key, "adapt")) *value = h->adapt;
    else if (!strcmp(key, "staged")) *value = h->staged;
    else if (!strcmp(key, "next_window")) {
        // Coordinates in flight the next epoch will use (read-only; synchronises the device).
        LaunchPlan lp;
        uint32_t n_groups = 1;
        plan_epoch(h, &lp, &n_groups);
        HotGeom hg{};
        const int64_t window = h->window ? h->window : h->auto_window;
        if ((lp.kind == PLAN_HOT || lp.kind == PLAN_HOT_STAGED) && hot_plan(h, window, &hg) && hg.adaptive) {
            uint32_t v = 0;
            if (!h->adapt_fresh) {
                if (int r = set_device(h)) return r;
                HIP_TRY(hipDeviceSynchronize());
                HIP_TRY(hipMemcpy(&v, h->hot_adapt, sizeof v, hipMemcpyDeviceToHost));
            }
            *value = v ? (int64_t)v : window;
        } else {
            scd_info_t info;
            scd_get_info(h, &info);
            *value = info.window;
        }
    }
    else return fail(SCD_ERR_UNSUPPORTED, "unknown option '%s'", key);
    return SCD_OK;
}

int scd_get_info(scd_handle_t h, scd_info_t* info) {
    if (int r = check_handle(h)) return r;
    if (!info) return fail(SCD_ERR_INVALID, "info is null");
    LaunchPlan lp;
    uint32_t n_groups = 1;
    plan_epoch(h, &lp, &n_groups);
    info->formulation = h->form;
    info->group_lanes = (lp.kind == PLAN_GROUP || lp.kind == PLAN_MIXED || lp.kind == PLAN_PIPE || lp.kind == PLAN_HOT ||
                         lp.kind == PLAN_HOT_STAGED || lp.kind == PLAN_QUEUE || lp.kind == PLAN_SPLIT)
                            ? lp.group
                        : lp.kind == PLAN_TEAM                 ? kBlockThreads * lp.team
                        : lp.kind == PLAN_BLOCK && !lp.ordered ? kBlockThreads
                                                               : 1024;
    info->kernel = lp.kind;
    info->hot_entries = (int32_t)h->n_hot;
    HotGeom hg{};
    info->adaptive_window = (lp.kind == PLAN_HOT || lp.kind == PLAN_HOT_STAGED) &&
                            hot_plan(h, h->window ? h->window : h->auto_window, &hg) && hg.adaptive;
    info->reserved = 0;
    info->long_len = lp.kind == PLAN_MIXED ? lp.long_len : lp.kind == PLAN_SPLIT ? lp.part : 0;
    info->shared_fp64 = h->wide;
    info->max_hits = h->max_hits;
    info->n_coords = h->C;
    info->shared_len = h->L;
    info->nnz = h->nnz;
    info->epoch = h->epoch;
    info->max_segment = h->max_seg;
    // Coordinates in flight at most: a group that does not drain holds two (its previous scatter may
    // not have landed when it gathers again).
    const bool two = (lp.kind == PLAN_PIPE || lp.kind == PLAN_GROUP || (lp.kind == PLAN_BLOCK && !lp.ordered)) &&
                     !lp.drain;
    info->window = two ? std::min<int64_t>(2 * (int64_t)n_groups, h->C) : n_groups;
    info->lambda = h->lambda;
    info->coupling = h->coupling;
    info->coherence = h->coherence;
    info->auto_window = h->auto_window;
    return SCD_OK;
}

int scd_gather_dots(scd_handle_t h, const float* u, float* out, void* stream) {
    if (int r = check_handle(h)) return r;
    if (!u || !out) return fail(SCD_ERR_INVALID, "null device pointer");
    if (int r = set_device(h)) return r;
    const int G = obj_group(h);
    HIP_TRY(launch_gather_dots(h->ptr, h->idx, h->val, u, (uint32_t)h->C, G, obj_blocks(h, G), out,
                               (hipStream_t)stream));
    return SCD_OK;
}

int scd_norms(scd_handle_t h, float* out, void* stream) {
    if (int r = check_handle(h)) return r;
    if (!out) return fail(SCD_ERR_INVALID, "null device pointer");
    if (int r = set_device(h)) return r;
    HIP_TRY(hipMemcpyAsync(out, h->norms, sizeof(float) * (size_t)h->C, hipMemcpyDeviceToDevice, (hipStream_t)stream));
    return SCD_OK;
}

int scd_permutation(uint64_t seed, int64_t epoch, int64_t n, int32_t* out, void* stream) {
    if (n < 1 || n > 2147483647LL) return fail(SCD_ERR_INVALID, "n must be in [1, 2^31)");
    if (epoch < 0) return fail(SCD_ERR_INVALID, "epoch must be >= 0");
    if (!out) return fail(SCD_ERR_INVALID, "null device pointer");
    HIP_TRY(launch_perm_fill(make_perm(seed, (uint64_t)epoch, (uint32_t)n), out, (hipStream_t)stream));
    return SCD_OK;
}

}  // extern "C"
