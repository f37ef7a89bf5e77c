// scd_static.hip -- scd_objective_static: the objectives of a given state without a handle and
// without any allocation, for callers that cannot allocate device memory.
//
// The evaluation is the one scd_objective runs (Sec. II-C: P, D and the duality gap of the state),
// preceded by the validation pass of scd_create (the caller's matrix has not been checked by a
// handle).  Its scratch -- the validation flags, one row of fp64 partial sums per workgroup of the
// objective pass and the five reduced sums -- lives in the file-scope device array `scratch`, of a
// fixed size that does not depend on the input (the objective pass uses at most kObjBlocksMax
// workgroups).  Each GPU holds its own copy of the array from the first call on it until the process
// ends; host code reaches it only through the address hipGetSymbolAddress returns on that device.
#include <hip/hip_runtime.h>

#include <cmath>
#include <mutex>
#include <string>

#include "scd.h"
#include "scd_kernels.h"

namespace scd {
namespace {

// Layout of the scratch array, in 8-byte words: validation flags (2 words: flag bits, longest
// segment), then kObjBlocksMax x 5 partial sums, then the 5 reduced sums.
constexpr uint32_t kFlagWords = 2;
constexpr uint32_t kPartialWords = (uint32_t)kObjBlocksMax * 5;
constexpr uint32_t kSumWords = 8;
constexpr uint32_t kScratchWords = kFlagWords + kPartialWords + kSumWords;  // 82,048 bytes

__device__ __align__(256) uint64_t scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device, once looked up

// Records the message that scd_last_error returns on this thread.
int fail_static(int code, const char* msg, hipError_t e = hipSuccess) {
    std::string m = msg;
    if (e != hipSuccess) {
        m += ": ";
        m += hipGetErrorString(e);
    }
    set_last_error(m.c_str());
    return code;
}

// The device address of `scratch` on the current device (looked up once per device).
int scratch_on_current_device(uint64_t** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_static(SCD_ERR_HIP, "hipGetDevice", e);
    if (dev < 0 || dev >= kMaxDevices) return fail_static(SCD_ERR_UNSUPPORTED, "device index beyond 63");
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return fail_static(SCD_ERR_HIP, "hipGetSymbolAddress(scratch)", e);
        g_scratch[dev] = p;
    }
    *out = static_cast<uint64_t*>(g_scratch[dev]);
    return SCD_OK;
}

}  // namespace
}  // namespace scd

using namespace scd;

extern "C" int scd_objective_static(const scd_matrix_t* A, const float* y, double lambda, int32_t formulation,
                                    const float* model, const float* shared, void* stream, double* primal,
                                    double* dual) {
    set_last_error("");
    if (!A || !y || !model || !shared) return fail_static(SCD_ERR_INVALID, "null argument");
    if (formulation < SCD_RIDGE_PRIMAL || formulation > SCD_RIDGE_DUAL)
        return fail_static(SCD_ERR_INVALID, "unknown formulation");
    const int want = formulation == SCD_RIDGE_PRIMAL ? SCD_CSC : SCD_CSR;
    if (A->layout != want) return fail_static(SCD_ERR_INVALID, "layout does not match the formulation");
    if (A->n_rows < 1 || A->n_cols < 1 || A->nnz < 0 || A->n_rows > 2147483647LL || A->n_cols > 2147483647LL)
        return fail_static(SCD_ERR_INVALID, "sizes must be in [1, 2^31) (nnz >= 0)");
    if (!A->ptr || (A->nnz > 0 && (!A->idx || !A->val))) return fail_static(SCD_ERR_INVALID, "null device pointer");
    if (!(lambda > 0.0) || !std::isfinite(lambda)) return fail_static(SCD_ERR_INVALID, "lambda must be finite and > 0");
    const int64_t C = formulation == SCD_RIDGE_PRIMAL ? A->n_cols : A->n_rows;
    const int64_t L = formulation == SCD_RIDGE_PRIMAL ? A->n_rows : A->n_cols;
    hipStream_t s = (hipStream_t)stream;
    uint64_t* scr = nullptr;
    if (int r = scratch_on_current_device(&scr)) return r;
    uint64_t* const flags = scr;
    double* const partials = reinterpret_cast<double*>(scr + kFlagWords);
    double* const sums = reinterpret_cast<double*>(scr + kFlagWords + kPartialWords);

    // Validation (the pass of scd_create): indices in range, ptr monotone, finite values and labels.
    hipError_t e = launch_fill_zero(flags, kFlagWords, s);
    if (e == hipSuccess)
        e = launch_validate(A->ptr, (uint32_t)C, A->idx, A->val, A->nnz, L, y, A->n_rows,
                            formulation == SCD_SVM_DUAL, reinterpret_cast<int*>(flags), s);
    int64_t fl[2] = {0, 0};
    if (e == hipSuccess) e = hipMemcpyAsync(fl, flags, sizeof fl, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail_static(SCD_ERR_HIP, "validation pass", e);
    const int bits = (int)(fl[0] & 0xFFFFFFFF);
    if (bits & 1) return fail_static(SCD_ERR_INVALID, "ptr must start at 0, end at nnz and be non-decreasing");
    if (bits & 2) return fail_static(SCD_ERR_INVALID, "an index is outside the shared vector");
    if (bits & 16) return fail_static(SCD_ERR_INVALID, "SVM labels must be -1 or +1");
    if (bits) return fail_static(SCD_ERR_NUMERIC, "non-finite matrix value or label");

    ObjArgs o{};
    o.ptr = A->ptr;
    o.idx = A->idx;
    o.val = A->val;
    o.u = shared;
    o.wide = 0;
    o.model = model;
    o.y = formulation == SCD_RIDGE_PRIMAL ? nullptr : y;
    o.yv = formulation == SCD_RIDGE_PRIMAL ? y : nullptr;
    o.cyd = nullptr;  // the ridge primal gathers y beside the shared vector
    o.C = (uint32_t)C;
    o.L = L;
    o.lam = lambda;
    const int G = objective_group(C > 0 ? (double)A->nnz / (double)C : 0.0);
    const int blocks = objective_blocks(C, G);
    double t[5] = {0, 0, 0, 0, 0};
    e = launch_objective(formulation, o, G, blocks, partials, sums, s);
    if (e == hipSuccess) e = hipMemcpyAsync(t, sums, sizeof t, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return fail_static(SCD_ERR_HIP, "objective pass", e);
    double P = 0.0, D = 0.0;
    objectives_from_sums(formulation, (double)A->n_rows, lambda, t, &P, &D);
    if (!std::isfinite(P) || !std::isfinite(D)) return fail_static(SCD_ERR_NUMERIC, "non-finite objective");
    if (primal) *primal = P;
    if (dual) *dual = D;
    return SCD_OK;
}
