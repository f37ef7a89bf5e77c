/*
 * scd.h -- C ABI of libscd: asynchronous stochastic coordinate descent/ascent (SCD) for
 * generalized linear models on one AMD Instinct MI355X (gfx950).
 *
 * Method: Parnell, Duenner, Atasu, Sifalakis, Pozidis, "Large-Scale Stochastic Learning
 * using GPUs" (arXiv 1702.07005).  One epoch visits every coordinate once, in a fresh
 * random permutation (Sec. III-A, Alg. 1); many coordinates are processed concurrently,
 * each by a group of GPU lanes that splits the coordinate's sparse inner product, reduces
 * it, applies the closed-form coordinate step and scatters the shared-vector update with
 * device atomics (Sec. III-C, Alg. 2, "TPA-SCD").
 *
 * Problem statement (Sec. II): A in R^{N x M} (N examples, M features), labels y in R^N,
 * regularisation lambda > 0 -- the paper's lambda of eq. (primal_obj), i.e. the objectives
 * carry the 1/N normalisation and the closed-form ridge minimiser is
 * (A^T A + N lambda I)^{-1} A^T y.
 *
 * Formulations:
 *   SCD_RIDGE_PRIMAL  coordinates = features; A given by columns (CSC); model beta in R^M;
 *                     shared vector w = A beta in R^N.  Step: eq. (update_primal).
 *   SCD_SVM_DUAL      coordinates = examples; A given by rows (CSR); y in {-1, +1};
 *                     model alpha in [0,1]^N; shared vector w = sum_i alpha_i y_i x_i/(lambda N)
 *                     in R^M.  Hinge-loss SVM, P(w) = (1/N) sum max(0, 1 - y_i x_i.w)
 *                     + lambda/2 |w|^2, D(alpha) = (1/N) sum alpha_i - lambda/2 |w|^2; step
 *                     alpha_i <- clip(alpha_i + lambda N (1 - y_i x_i.w)/|x_i|^2, 0, 1)
 *                     (alpha_i <- 1 for an empty row).
 *   SCD_RIDGE_DUAL    coordinates = examples; A given by rows (CSR); model alpha in R^N;
 *                     shared vector wbar = A^T alpha in R^M.  Step: eq. (update_dual).
 *
 * Conventions shared by every call:
 *   - Status: every call returns SCD_OK (0) or a negative scd_status_t and never aborts or
 *     throws across the ABI; scd_last_error() gives a message for the calling thread.
 *   - Memory: pointers named *_dev are device pointers on the handle's GPU; all others are
 *     host pointers.  Arrays are dense and contiguous.
 *   - Ownership: the handle BORROWS A (ptr/idx/val) and y: they must stay allocated and
 *     unmodified until scd_destroy.  The handle owns its model, shared vector, norms and
 *     scratch and frees them in scd_destroy.
 *   - Streams: `stream` is a hipStream_t (NULL = the null stream).  Calls that only
 *     enqueue work return immediately; calls that return values to the host synchronise
 *     the stream.  A handle is not thread-safe; separate handles on separate streams are.
 *     The work of one handle must be ordered: enqueue it on one stream, or order the streams
 *     with events.  Its epochs share scratch (the queued kernel's position counter, the gap
 *     evaluation slots), so two epochs of one handle running at once process coordinates twice.
 *   - Faults inside kernels surface as SCD_ERR_HIP at the next synchronising call.
 */
#ifndef SCD_H
#define SCD_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct scd_solver *scd_handle_t;

typedef enum {
    SCD_RIDGE_PRIMAL = 0,
    SCD_SVM_DUAL = 1,
    SCD_RIDGE_DUAL = 2
} scd_formulation_t;

typedef enum {
    SCD_CSC = 0, /* segments are columns: ptr has n_cols+1 entries, idx are row indices   */
    SCD_CSR = 1  /* segments are rows:    ptr has n_rows+1 entries, idx are column indices */
} scd_layout_t;

typedef enum {
    SCD_OK = 0,
    SCD_ERR_INVALID = -1,     /* bad argument, inconsistent matrix, wrong layout for the formulation */
    SCD_ERR_UNSUPPORTED = -2, /* valid request this build does not implement (e.g. unknown option)   */
    SCD_ERR_OOM = -3,         /* device or pinned-host allocation failed                              */
    SCD_ERR_HIP = -4,         /* a HIP runtime call failed (includes earlier kernel faults)           */
    SCD_ERR_NUMERIC = -5      /* non-finite input values or a non-finite objective                    */
} scd_status_t;

/* A sparse matrix in compressed form, stored on the device.
 *   ptr: int64[S+1], S = n_cols (CSC) or n_rows (CSR); ptr[0] = 0, non-decreasing, ptr[S] = nnz.
 *   idx: int32[nnz], 0-based, in [0, n_rows) for CSC and [0, n_cols) for CSR.
 *   val: float32[nnz], finite.
 * Duplicate indices inside one segment are allowed (they act as a sum). */
typedef struct {
    int64_t n_rows;
    int64_t n_cols;
    int64_t nnz;
    int32_t layout; /* scd_layout_t */
    int32_t reserved;
    const int64_t *ptr;
    const int32_t *idx;
    const float *val;
} scd_matrix_t;

/* Read-only facts about a handle. */
typedef struct {
    int32_t formulation;  /* scd_formulation_t                                        */
    int32_t group_lanes;  /* lanes per coordinate of the epoch kernel (1024 = ordered; the team
                             kernel: 256 x its members)                                */
    int64_t n_coords;     /* C: M for SCD_RIDGE_PRIMAL, N for the duals                */
    int64_t shared_len;   /* length of the shared vector: N (ridge primal) or M         */
    int64_t nnz;
    int64_t epoch;        /* global epoch counter (epochs run so far)                  */
    int64_t max_segment;  /* longest coordinate segment                                */
    int64_t window;       /* coordinates in flight at most (whose updates other
                             coordinates may not see yet); with an adaptive window (see
                             adaptive_window) the most the epoch kernel can hold          */
    double lambda;
    double coupling;      /* largest over coordinates c of sum_{j != c} G_cj^2 / (C - 1), G the
                             step-normalised Gram matrix of the coordinates (estimated at
                             create with Rademacher probes)                             */
    double coherence;     /* mean off-diagonal entry of G (signed sum)                  */
    int64_t auto_window;  /* window chosen from `coupling` when the option is 0         */
    int64_t long_len;     /* kernel 3: segments longer than this are processed by a
                             whole workgroup inside the group kernel; kernel 9: the part
                             length (entries); 0 otherwise                              */
    int32_t shared_fp64;  /* 1 if the shared vector is stored in fp64                   */
    uint32_t max_hits;    /* most stored entries sharing one shared-vector index, i.e.
                             the most atomic adds one entry receives per epoch          */
    int32_t kernel;       /* epoch kernel the next scd_epochs launches: 0 lane groups,
                             1 one workgroup per coordinate, 2 ordered with the shared
                             vector in LDS, 3 lane groups with long segments handed to the
                             workgroup, 4 software-pipelined, 5 hot set in LDS (one
                             workgroup, at most 16 coordinates in flight), 6 one workgroup
                             per coordinate taking positions from a queue (skewed
                             segment lengths), 7 a team of workgroups per coordinate,
                             each on its own range of shared-vector indices (long
                             segments, few coordinates in flight), 8 hot set in LDS with
                             stager workgroups assembling the batches (option "staged"),
                             9 as 6 over work units, long segments split into parts
                             that many workgroups process side by side (option "split") */
    int32_t hot_entries;  /* shared-vector entries the hot-set kernel keeps in LDS
                             (0 until it is first needed)                               */
    int32_t adaptive_window; /* 1 if the epoch kernel sets each epoch's window from the
                             coordinates that moved in the previous one (option "adapt"):
                             the first epoch opens at auto_window                       */
    int32_t reserved;
} scd_info_t;

/* Create a solver for min P / max D of the chosen formulation (Sec. II; Sec. III-C).
 *   A:       device matrix; layout must be SCD_CSC for SCD_RIDGE_PRIMAL and SCD_CSR otherwise.
 *   y_dev:   float32[n_rows] labels (device); for SCD_SVM_DUAL every label is -1 or +1.
 *   lambda:  the paper's normalised lambda (> 0, finite).
 *   stream:  hipStream_t used for the set-up work; the call synchronises it.
 * Validates A and y on the device (one pass), computes |a_c|^2 for every coordinate and sets
 * model = 0, shared vector = 0 (Alg. 1/2 initialisation), epoch = 0.
 * Errors: SCD_ERR_INVALID (null/negative sizes, wrong layout, ptr not monotone, index out of
 * range, labels not +-1 for the SVM, lambda <= 0), SCD_ERR_NUMERIC (non-finite values or labels),
 * SCD_ERR_OOM, SCD_ERR_HIP.  On error *out is set to NULL. */
int scd_create(const scd_matrix_t *A, const float *y_dev, double lambda, int32_t formulation,
               void *stream, scd_handle_t *out);

/* Free everything the handle owns (not A or y).  NULL-safe.  Synchronises the device. */
int scd_destroy(scd_handle_t h);

/* Run n_epochs >= 0 epochs (Alg. 1 epochs executed as in Alg. 2): epoch t (global counter,
 * continued across calls) visits the coordinates in the order pi_{seed,t} of
 * scd_permutation; each visit is the exact coordinate step of the formulation against the
 * shared vector as it stands, followed by an atomic scatter of the change into the shared
 * vector.  Up to `window` coordinates are in flight at once (option "window"); window = 1
 * reproduces the sequential order of Alg. 1 exactly.  Enqueues only. */
int scd_epochs(scd_handle_t h, uint64_t seed, int32_t n_epochs, void *stream);

/* Primal and dual objective of the current state, in fp64 (synchronises):
 *   SCD_RIDGE_PRIMAL: P(beta) of eq. (primal_obj) and D((y - w)/N) of eq. (dual_obj), with the
 *                     maintained shared vector w standing in for A beta (Sec. II-C).
 *   SCD_RIDGE_DUAL:   P(wbar/lambda) and D(alpha) (Sec. II-C), wbar = maintained A^T alpha.
 *   SCD_SVM_DUAL:     P(w) and D(alpha) of the hinge SVM, w = maintained shared vector.
 * Either output pointer may be NULL. */
int scd_objective(scd_handle_t h, void *stream, double *primal, double *dual);

/* Duality gap |P - D| of the current state (Sec. II-C: G_P for the ridge primal, G_D for the
 * ridge dual; P - D >= 0 for the SVM).  Synchronises. */
int scd_duality_gap(scd_handle_t h, void *stream, double *gap);

/* Asynchronous duality gap, for training loops that check convergence without stalling the GPU:
 * scd_duality_gap_async enqueues the evaluation of the current state (as scd_duality_gap) on
 * `stream` into one of 4 slots (0..3) and returns at once; scd_duality_gap_wait blocks until that
 * evaluation is done and returns the gap (and, if not NULL, P and D).  A slot must be waited on
 * before it is reused (SCD_ERR_INVALID otherwise).  Evaluations share the handle's reduction
 * scratch, so all of them must be enqueued on the same stream as the epochs. */
int scd_duality_gap_async(scd_handle_t h, void *stream, int32_t slot);
int scd_duality_gap_wait(scd_handle_t h, int32_t slot, double *gap, double *primal, double *dual);

/* Copy the state out (device buffers, may be NULL to skip), exactly as the solver holds it:
 *   model_dev:  float32[n_coords]   (beta, or alpha)
 *   shared_dev: float32[shared_len] (w = A beta, or w(alpha), or wbar = A^T alpha)
 *   epoch:      host int64 (may be NULL).  Enqueues only, so it reports no error of the
 *   epochs before it: a hot-set, team or split epoch whose waits timed out (see "hot_wait_limit") leaves a
 *   partial state that this call copies as is; the next synchronising call returns the error.
 *   A state copied out and written back with scd_set_state resumes bit-exactly when the shared
 *   vector is stored in fp32 (option "shared_fp64" = 0); an fp64 shared vector is exchanged
 *   rounded to fp32. */
int scd_get_state(scd_handle_t h, float *model_dev, float *shared_dev, int64_t *epoch, void *stream);

/* Overwrite the state (resume from a checkpoint).  model_dev/shared_dev in the layout of
 * scd_get_state (NULL leaves that part unchanged); epoch >= 0 sets the global epoch counter.
 * The caller is responsible for the shared vector matching the model (the invariant
 * w = A beta of Sec. II-A, wbar = A^T alpha of Sec. II-B).  Enqueues only. */
int scd_set_state(scd_handle_t h, const float *model_dev, const float *shared_dev, int64_t epoch,
                  void *stream);

/* Tuning and test options (host-side, take effect at the next scd_epochs):
 *   "window"      coordinates in flight at most; 1 = ordered (Alg. 1's sequence exactly);
 *                 0 (default) = chosen at create from the measured coupling of the coordinates:
 *                 W = 1 + b / coupling (b = 0.15 for the SVM dual, 0.015 for the ridge forms), at
 *                 most C/16 when the coupling exceeds 1e-6, at most what the GPU holds.  Concurrent coordinates read each other's stale shared-vector
 *                 entries; strongly coupled problems need a small window to keep the per-epoch
 *                 convergence of the sequential algorithm.
 *   "group"       lanes per coordinate: 0 = by segment length (default), 4, 8, 16, 32, 64, or
 *                 256 (one workgroup per coordinate).
 *   "fresh_reads" 1 = gather the shared vector with device-scope loads (bypass non-coherent
 *                 caches), 0 = plain loads.
 *   "pipeline"    1 (default) = use the software-pipelined epoch kernel where it applies
 *                 (shared vector below 2 GiB; with skewed segment lengths only when each
 *                 in-flight coordinate can have a workgroup of its own, then with workgroups
 *                 taking positions from a queue), 0 = the plain kernels.
 *   "spread"      1 (default) = when the shared vector has at most 4 M entries and the window
 *                 does not bind (every coordinate may be in flight), the pipelined kernel runs on a
 *                 copy that holds one entry per 64 bytes (scd_epochs copies it out before its
 *                 epochs and back after them, on the same stream), so that the gathers of one
 *                 coordinate do not wait behind other coordinates' atomics on neighbouring
 *                 entries; 0 = it runs on the packed vector.
 *   "queue_chunk" consecutive permutation positions each workgroup of the queued kernel claims
 *                 at a time: 0 (default) = 1 per 64 coordinates in flight (at least 1), else
 *                 1..64.  Larger chunks lower the claim rate on the queue's counter and let
 *                 coordinates start further from their permutation positions.
 *   "split"       1 (default) = where the queued kernel (6) would run and some segment is longer than
 *                 "split_part" entries, run kernel 9 instead: before each epoch a pre-pass (three
 *                 kernels on the same stream) lays out the epoch's work units in permutation order,
 *                 one per segment of at most split_part entries, and for a longer one of k parts, k
 *                 gather units (partial inner products, published in device memory) followed by k
 *                 scatter units (each waits for the k partials, takes the step and scatters its
 *                 part).  Workgroups claim units in order, so a long segment is gathered and
 *                 scattered by many CUs at once, and the window is not halved for long segments.
 *                 The unit tables (40 bytes per unit, about one unit per coordinate) are made when
 *                 this first applies for a part length: at create, on any scd_set_option, or at the
 *                 first such epoch (synchronising).  Segments of more than 256 parts, or more than
 *                 4e9 units, take kernel 6.  0 = never; 2 = a test hook: kernel 9 whenever "group" is 0,
 *                 "pipeline" is 1 and the shared vector takes less than 2 GB, with as many workgroups
 *                 as the window (window 1: one workgroup, which takes the units in order).
 *   "split_part"  entries per part of kernel 9: 0 (default) = 4,096 (what a workgroup's register
 *                 slices hold), else a multiple of 64 in [64, 4096].
 *   "hot"         1 (default) = with at most 16 coordinates in flight, segments of at most 64
 *                 entries and "group" 0, run the epoch in one workgroup that keeps the most-updated
 *                 shared-vector entries in LDS (their gathers and adds never leave the CU) and
 *                 reads the others ahead of their coordinates; 0 = never.  The hot set is chosen
 *                 (a pass over the matrix, synchronising) when this first applies: at create, or
 *                 when "window" or "hot" is set.
 *   "team"        1 (default) = with a binding window, segments of at least 1,024 entries on
 *                 average and none longer than 4 times that, a shared vector of at least 4 MB and
 *                 "group" 0, process each in-flight
 *                 coordinate with a team of K workgroups (K = CUs / coordinates in flight, at
 *                 most 16), member k on the entries whose shared-vector index lies in the k-th of
 *                 K ranges of about equal entry count; the members exchange their partial inner
 *                 products through device memory.  It needs a copy of A with each segment's
 *                 entries grouped by range (8 bytes per stored entry, made when this first
 *                 applies: at create, or when "window", "team", "group", "pipeline" or
 *                 "shared_fp64" is set; synchronising; skipped when device memory is short).
 *                 0 = never; 2..16 = K members whenever the window binds and (coordinates in
 *                 flight) x K is at most the number of CUs.  With the automatic window, teams take
 *                 7/8 of the window's share that the other draining kernels take.
 *   "staged"      1 (default) = when the hot-set kernel runs the epoch and the matrix's entries take more
 *                 than 256 MB (beyond the GPU's Infinity Cache), the batches it runs are assembled by
 *                 stager workgroups on the hot-set workgroup's XCD (coordinate metadata, entry keys and
 *                 values, and the cold entries' shared-vector values) and passed through a ring of 32
 *                 records in device memory, so that the one workgroup only copies records and runs
 *                 the steps; 2 =
 *                 whenever the hot-set kernel runs; 0 = never.  The stagers need the GPU's CUs beside
 *                 the hot-set workgroup: a kernel of another stream that holds them delays the epoch,
 *                 and its bounded waits then report SCD_ERR_HIP.
 *   "adapt"       1 (default) = when the window is automatic and the hot-set kernel runs the epoch,
 *                 each epoch's window follows the fraction f of coordinates whose step was nonzero
 *                 in the previous epoch: W = 1 + (auto_window - 1) / f, at most 16, run by
 *                 min(4, W / 2) consumer waves whose shares differ by at most one.  A coordinate
 *                 whose step is zero (in the hinge SVM dual, one whose alpha stays at a bound of
 *                 the box) changes nothing that others read, so the coupling rule's budget holds
 *                 for the coordinates in flight that move.  The window is kept in device memory,
 *                 so it needs no synchronisation.  The first epoch after scd_create, scd_set_state
 *                 or scd_set_option is two launches: its first ceil(C / 16) positions at
 *                 auto_window, the rest at the window that the fraction moving among those gives
 *                 (one launch at auto_window when C < 32).  0 = auto_window in every epoch.
 *   "hot_wait_limit"  test hook: sleeps (about 64 cycles each) one wait between the waves of the
 *                 hot-set kernel, between the members of a team, or of a scatter unit of kernel 9
 *                 for its segment's partials, may take before giving up;
 *                 the next synchronising call then returns SCD_ERR_HIP and the state stays invalid
 *                 until scd_set_state.  0 (default) = 2^24.
 *   "shared_fp64" 1 = store the shared vector in fp64 (fp64 atomic adds), 0 = fp32.  Chosen at
 *                 create: fp64 when some entry receives more than 28,000 atomic adds per epoch,
 *                 where fp32 accumulation would drift by more than about 1e-5 of its magnitude.
 *                 The state calls exchange fp32 copies either way.
 * Errors: SCD_ERR_UNSUPPORTED for an unknown key, SCD_ERR_INVALID for a bad value. */
int scd_set_option(scd_handle_t h, const char *key, int64_t value);
/* Reads an option's value, or the read-only key "next_window": the coordinates the next epoch will
 * keep in flight at most (with an adaptive window, the value the last epoch left in device memory;
 * this read synchronises the device). */
int scd_get_option(scd_handle_t h, const char *key, int64_t *value);

int scd_get_info(scd_handle_t h, scd_info_t *info);

/* out_dev[c] = sum over coordinate c's segment of val * u_dev[idx]  (float32, c < n_coords):
 * the sparse gather-dot of the epoch kernel (the inner product of eq. update_primal /
 * update_dual) against a frozen vector u_dev[shared_len].  Enqueues only. */
int scd_gather_dots(scd_handle_t h, const float *u_dev, float *out_dev, void *stream);

/* out_dev[c] = |a_c|^2 (float32[n_coords]): the squared segment norms used by every step. */
int scd_norms(scd_handle_t h, float *out_dev, void *stream);

/* The visiting order of epoch `epoch`: out_dev[j] = pi_{seed,epoch}(j), j < n (int32[n]),
 * 1 <= n < 2^31.  pi is a 4-round balanced Feistel network on 2h bits (h >= 1 smallest with
 * 2^(2h) >= n), round function fmix32(R xor k_r) mod 2^h (MurmurHash3 finaliser), round keys
 * k_r = low 32 bits of SplitMix64 output r+1 from state b, b = SplitMix64 output epoch+1 from
 * state seed, values outside [0, n) re-encrypted until inside (cycle-walking).  The paper only
 * asks for a fresh random permutation per epoch (Alg. 1, Alg. 2).  Enqueues only. */
int scd_permutation(uint64_t seed, int64_t epoch, int64_t n, int32_t *out_dev, void *stream);

/* Allocation-free objectives of a given state, for callers that cannot allocate device memory (code
 * in tight serving or evaluation loops, harnesses that forbid hipMalloc): the same P and D as
 * scd_objective, for the state (model_dev, shared_dev) of formulation `formulation` on (A, y_dev,
 * lambda), without a handle.
 *   A, y_dev, lambda, formulation: as for scd_create (A and y are read, not kept).
 *   model_dev:  float32[C] (C = n_cols for SCD_RIDGE_PRIMAL, n_rows otherwise), device.
 *   shared_dev: float32[L] (L = n_rows for SCD_RIDGE_PRIMAL, n_cols otherwise), device: the shared
 *               vector standing in for A beta, w(alpha) or A^T alpha (Sec. II-C).
 *   primal, dual: host outputs (either may be NULL).
 * The call validates A and y on the device as scd_create does (same errors), runs the objective
 * pass and synchronises the stream.  It calls no allocating routine: its scratch (validation flags,
 * up to 2,048 x 5 fp64 partial sums, 5 sums; 82,048 bytes) is a fixed device array of the library,
 * one copy per GPU, held from the first call on that GPU until the process ends, so no input size
 * can exceed it (sizes are limited as for scd_create: dimensions below 2^31).  Calls on one GPU
 * share that array: calls that overlap in time on one GPU (two host threads, or two streams without
 * ordering) race and must be serialised by the caller.  Errors: SCD_ERR_INVALID, SCD_ERR_NUMERIC,
 * SCD_ERR_HIP (as scd_create), SCD_ERR_UNSUPPORTED for a device index above 63. */
int scd_objective_static(const scd_matrix_t *A, const float *y_dev, double lambda, int32_t formulation,
                         const float *model_dev, const float *shared_dev, void *stream, double *primal,
                         double *dual);

/* Message describing the last error on the calling thread ("" if none). */
const char *scd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SCD_H */
