// scd_setup.hip -- set-up and evaluation kernels for gfx950: the permutation array, the frozen
// gather-dot, squared norms (and <y, a_c>), input validation, the objective / duality-gap
// reductions, the coupling probe, precision conversions and per-entry hit counts.
#include "scd_device.h"

namespace scd {

__global__ void k_perm_fill(PermKeys p, int32_t* __restrict__ out) {
    uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j < p.n) out[j] = (int32_t)perm_at(j, p);
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

constexpr int kObjSlices = 8;  // entries per lane per block of the objective's gather-dot

// DIRECT (ridge primal only): <a_c, y - w> is gathered from y and w in fp64 instead of taken as
// <y, a_c> (o.cyd, computed at set-up) minus <a_c, w>; for callers that hold no set-up data.
template <int FORM, int G, typename U, bool DIRECT>
__global__ __launch_bounds__(256) void k_objective(ObjArgs o, double* __restrict__ partials) {
    constexpr int NS = 5;
    const U* __restrict__ u = static_cast<const U*>(o.u);
    const int lane = threadIdx.x & (G - 1);
    const uint32_t ngroups = gridDim.x * (256u / G);
    double t[NS] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (uint32_t c = (blockIdx.x * 256u + threadIdx.x) / G; c < o.C; c += ngroups) {
        // Blocks of G * kObjSlices entries: all index and value loads of a block, then all its
        // gathers, so that a block costs two memory round trips instead of two per entry.  Lanes
        // past the end re-read entry s0 with weight 0.
        const int64_t s0 = o.ptr[c], s1 = o.ptr[c + 1];
        double d = 0.0;
        for (int64_t b = s0; b < s1; b += (int64_t)G * kObjSlices) {
            int ix[kObjSlices];
            float vx[kObjSlices];
#pragma unroll
            for (int r = 0; r < kObjSlices; ++r) {
                const int64_t k = b + lane + (int64_t)r * G;
                const bool in = k < s1;
                const int64_t kk = in ? k : s0;
                ix[r] = o.idx[kk];
                const float v = o.val[kk];
                vx[r] = in ? v : 0.0f;
            }
            U g[kObjSlices];
#pragma unroll
            for (int r = 0; r < kObjSlices; ++r) g[r] = u[ix[r]];
            if constexpr (DIRECT) {
                float yy[kObjSlices];
#pragma unroll
                for (int r = 0; r < kObjSlices; ++r) yy[r] = o.yv[ix[r]];
#pragma unroll
                for (int r = 0; r < kObjSlices; ++r) d += (double)vx[r] * ((double)yy[r] - (double)g[r]);
            } else {
#pragma unroll
                for (int r = 0; r < kObjSlices; ++r) d += (double)vx[r] * (double)g[r];
            }
        }
        d = group_sum_f64<G>(d);
        if (lane == 0) {
            const double mo = o.model[c];
            if constexpr (FORM == FORM_RIDGE_PRIMAL) {
                const double r = DIRECT ? d : o.cyd[c] - d;
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

// Packed shared vector <-> its spread copy (entry i at byte offset i << kSpreadShift of the copy; the
// bytes between entries are never read).
template <typename U>
__global__ __launch_bounds__(256) void k_spread(U* __restrict__ packed, U* __restrict__ spread, int64_t L,
                                                bool to_spread) {
    constexpr uint32_t step = (1u << kSpreadShift) / sizeof(U);
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < L; i += (int64_t)gridDim.x * 256) {
        if (to_spread)
            spread[i * step] = packed[i];
        else
            packed[i] = spread[i * step];
    }
}

hipError_t launch_spread(void* packed, void* spread, int64_t L, bool wide, bool to_spread, hipStream_t s) {
    if (wide)
        hipLaunchKernelGGL(k_spread<double>, dim3(grid_for(L)), dim3(256), 0, s, static_cast<double*>(packed),
                           static_cast<double*>(spread), L, to_spread);
    else
        hipLaunchKernelGGL(k_spread<float>, dim3(grid_for(L)), dim3(256), 0, s, static_cast<float*>(packed),
                           static_cast<float*>(spread), L, to_spread);
    return hipGetLastError();
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

template <int FORM, typename U, bool DIRECT>
static void objective_typed(const ObjArgs& o, int G, int blocks, double* partials, hipStream_t s) {
    switch (G) {
#define SCD_OBJ(GW)                                                                                         \
    case GW:                                                                                                \
        hipLaunchKernelGGL((k_objective<FORM, GW, U, DIRECT>), dim3(blocks), dim3(256), 0, s, o, partials); \
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
    // The ridge primal without <y, a_c> from set-up gathers y beside w.
    if constexpr (FORM == FORM_RIDGE_PRIMAL) {
        if (!o.cyd) {
            if (o.wide)
                objective_typed<FORM, double, true>(o, G, blocks, partials, s);
            else
                objective_typed<FORM, float, true>(o, G, blocks, partials, s);
            return;
        }
    }
    if (o.wide)
        objective_typed<FORM, double, false>(o, G, blocks, partials, s);
    else
        objective_typed<FORM, float, false>(o, G, blocks, partials, s);
}

__global__ __launch_bounds__(256) void k_fill_zero(uint64_t* __restrict__ p, uint32_t n) {
    for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < n; i += gridDim.x * 256u) p[i] = 0ull;
}

hipError_t launch_fill_zero(uint64_t* p, uint32_t n_words, hipStream_t s) {
    if (n_words == 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill_zero, dim3((n_words + 255) / 256 > 64 ? 64 : (n_words + 255) / 256), dim3(256), 0, s, p,
                       n_words);
    return hipGetLastError();
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


hipError_t launch_count_hits(const int32_t* idx, int64_t nnz, unsigned* hits, hipStream_t s) {
    if (nnz > 0) hipLaunchKernelGGL(k_count_hits, dim3(grid_for(nnz)), dim3(256), 0, s, idx, nnz, hits);
    return hipGetLastError();
}

}  // namespace scd
