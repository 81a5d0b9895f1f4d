// The C ABI of libiabn (include/iabn.h): argument validation on the host
// before any launch, the choice between the channel-resident and the
// streaming kernels, and the entry points themselves.

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <cmath>
#include <mutex>

#include "launch.h"

#define IABN_VERSION 10100

namespace iabn_impl {
namespace {

thread_local char g_last_error[256] = "";

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_last_error[0] = '\0';
    return IABN_OK;
}

constexpr int64_t kMaxChannelElems = (int64_t(1) << 31) - 1;
constexpr int64_t kMaxChannels = int64_t(1) << 20;
constexpr int64_t kMaxTotalElems = int64_t(1) << 46;
constexpr int64_t kTargetBlocks = 512;     // 2 blocks of 4 waves per CU on 256 CUs (measured best)
// The inference forward keeps no partial sums, so it chooses its slices
// freely: with fewer than kEvalManyBlocksBelow channels it cuts them for
// about kEvalTargetBlocks blocks (each thread moves a few accesses, and the
// chip holds many more waves): (8, 64, 256x256) fp16 25.2 us against 28.3,
// (32, 64, 112x112) 19.5 against 21.1, (8, 128, 128x128) 13.6 against 15.9;
// from 256 channels up the training passes' slicing is faster ((32, 256,
// 56x56) fp16 19.8 us against 21.5), and so it is for the checkpointing's
// recomputation on every shape measured.
constexpr int64_t kEvalTargetBlocks = 8192;
constexpr int64_t kEvalManyBlocksBelow = 256;

int64_t eval_target_blocks(int64_t C) {
    return C < kEvalManyBlocksBelow ? kEvalTargetBlocks : kTargetBlocks;
}
constexpr int64_t kMinSliceElems = 4096;   // at least 16 elements per thread
constexpr int64_t kMaxSlices = 1024;
constexpr int64_t kSliceAlign = 8;         // slices start on a 16-byte access of any dtype
constexpr int64_t kLineBytes = 128;        // L2 cache line

int elem_bytes(int dtype) { return dtype == IABN_F32 ? 4 : 2; }

bool valid_dtype(int dtype) { return dtype == IABN_F32 || dtype == IABN_F16 || dtype == IABN_BF16; }

// Slices per channel and slice length in elements; depends on the shape only.
struct Split {
    int64_t P;
    int64_t L;
};

Split split_channel(int64_t m, int64_t C, int64_t target_blocks = kTargetBlocks) {
    int64_t P = (target_blocks + C - 1) / C;
    const int64_t pmax_len = (m + kMinSliceElems - 1) / kMinSliceElems;
    if (P > pmax_len) P = pmax_len;
    if (P > kMaxSlices) P = kMaxSlices;
    if (P < 1) P = 1;
    int64_t L = (m + P - 1) / P;
    L = (L + kSliceAlign - 1) / kSliceAlign * kSliceAlign;
    P = (m + L - 1) / L;
    return {P, L};
}

// Validates the shape; `train` also needs N*HW >= 2.
int check_shape(int64_t N, int64_t C, int64_t HW, bool train) {
    if (N < 0 || C < 0 || HW < 0)
        return fail(IABN_ERR_SHAPE, "negative size N=%lld C=%lld HW=%lld", (long long)N,
                    (long long)C, (long long)HW);
    if (C > kMaxChannels) return fail(IABN_ERR_SHAPE, "C=%lld exceeds 2^20", (long long)C);
    if (N != 0 && HW > kMaxChannelElems / N)
        return fail(IABN_ERR_SHAPE, "N*HW exceeds 2^31-1");
    if (C != 0 && N * HW > kMaxTotalElems / C)
        return fail(IABN_ERR_SHAPE, "N*C*HW exceeds 2^46");
    if (train && C > 0 && N * HW < 2)
        return fail(IABN_ERR_SHAPE, "training needs N*HW >= 2 values per channel, got %lld",
                    (long long)(N * HW));
    return IABN_OK;
}

size_t workspace_bytes_for(int64_t N, int64_t C, int64_t HW) {
    if (C == 0 || N * HW == 0) return 0;
    const Split sp = split_channel(N * HW, C);
    return static_cast<size_t>(C) * static_cast<size_t>(sp.P) * kWaves * sizeof(Partial);
}

// The access geometry for `vec` elements per access.
Geom make_geom(int64_t N, int64_t C, int64_t HW, int dtype, int vec,
               int64_t target_blocks = kTargetBlocks) {
    const int64_t m = N * HW;
    const Split sp = split_channel(m, C, target_blocks);
    Geom g;
    g.C = static_cast<uint32_t>(C);
    g.P = static_cast<uint32_t>(sp.P);
    g.vrow = static_cast<uint32_t>(HW / vec);
    g.vchan = static_cast<uint32_t>(m / vec);
    g.lv = static_cast<uint32_t>(sp.L / vec);
    g.vec = static_cast<uint32_t>(vec);
    g.row_div = iabn_divmagic_make(g.vrow);
    g.nstride = static_cast<uint64_t>(C) * g.vrow;
    g.m = static_cast<double>(m);
    g.inv_m = 1.0 / g.m;
    g.xcd_order = (HW * elem_bytes(dtype)) % kLineBytes != 0 ? 1u : 0u;
    g.xcd_q = static_cast<uint32_t>(C / kXcds);
    g.xcd_r = static_cast<uint32_t>(C % kXcds);
    return g;
}

bool aligned_to(const void* p, uintptr_t bytes) {
    return p == nullptr || (reinterpret_cast<uintptr_t>(p) & (bytes - 1)) == 0;
}

// Elements per access: the widest of 16, 8, 4 (and 2 for 2-byte types)
// bytes that divides a row and to which every given tensor is aligned (an
// access never crosses a row; slices start on multiples of 8 elements, so
// every width divides them).  Null pointers are ignored.
int access_vec(int64_t HW, int dtype, const void* a, const void* b, const void* c) {
    const int eb = elem_bytes(dtype);
    for (int bytes = 16; bytes > eb; bytes /= 2) {
        const int v = bytes / eb;
        if (HW % v == 0 && aligned_to(a, bytes) && aligned_to(b, bytes) && aligned_to(c, bytes))
            return v;
    }
    return 1;
}

int check_workspace(int64_t N, int64_t C, int64_t HW, const void* ws, size_t bytes) {
    const size_t need = workspace_bytes_for(N, C, HW);
    if (need == 0) return IABN_OK;
    if (ws == nullptr) return fail(IABN_ERR_NULL, "workspace is NULL (%zu bytes needed)", need);
    if (bytes < need)
        return fail(IABN_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
    if ((reinterpret_cast<uintptr_t>(ws) & 15u) != 0)
        return fail(IABN_ERR_WORKSPACE, "workspace is not 16-byte aligned");
    return IABN_OK;
}

int check_params(float eps, float slope) {
    if (!(eps > 0.f) || !std::isfinite(eps)) return fail(IABN_ERR_PARAM, "eps must be finite and > 0");
    if (!(slope > 0.f) || !std::isfinite(slope))
        return fail(IABN_ERR_PARAM, "slope must be finite and > 0 (the activation must be invertible)");
    return IABN_OK;
}

int launched(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(IABN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

int validate_common(int dtype, int64_t N, int64_t C, int64_t HW, bool train) {
    if (!valid_dtype(dtype)) return fail(IABN_ERR_DTYPE, "unknown dtype %d", dtype);
    return check_shape(N, C, HW, train);
}

bool empty(int64_t N, int64_t C, int64_t HW) { return C == 0 || N * HW == 0; }

const char* fwd_name(int fm) {
    return fm == kFwdOut ? "standard forward" : fm == kFwdCkpt ? "checkpointing forward" : "forward";
}

// Training forward of the three arms (fm: kFwdInPlace, kFwdOut, kFwdCkpt).
// x is the input (kFwdInPlace: z on return; kFwdCkpt: xhat on return); out
// receives z for kFwdOut and kFwdCkpt.  Everything is validated before the
// first launch, so an error changes nothing.
// ws_if_streaming: the workspace is checked only where the streaming
// kernels run (the channel-resident ones use none); otherwise it must hold
// iabn_workspace_size bytes whichever kernels run.
int forward_train_impl(int fm, void* x, void* out, int dtype, const float* gamma,
                       const float* beta, float* running_mean, float* running_var,
                       float* save_mean, float* save_var, float eps, float momentum, float slope,
                       int64_t N, int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                       void* stream, bool ws_if_streaming = false) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!x || !gamma || !beta || !running_mean || !running_var || !save_mean || !save_var ||
        (fm != kFwdInPlace && !out))
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if (!(momentum >= 0.f && momentum <= 1.f))
        return fail(IABN_ERR_PARAM, "momentum must lie in [0, 1]");
    const int vec = access_vec(HW, dtype, x, fm == kFwdInPlace ? nullptr : out, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const FwdParams prm = {gamma,    beta, running_mean, running_var, save_mean, save_var,
                           fm == kFwdInPlace ? nullptr : out, eps, momentum, slope};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    FusedPlan fp;
    const bool fused = plan_fused(C, g, elem_bytes(dtype), false, fm == kFwdInPlace, &fp);
    if ((!fused || !ws_if_streaming) &&
        (rc = check_workspace(N, C, HW, workspace, workspace_bytes)))
        return rc;
    if (fused) {
        if (!launch_fwd_fused(dtype, fm, x, g, fp, prm, st))
            return fail(IABN_ERR_HIP, "no %s kernel built for T=%d R=%d", fwd_name(fm), fp.T, fp.R);
        return launched(fwd_name(fm));
    }
    Partial* part = static_cast<Partial*>(workspace);
    launch_fwd_stats(dtype, vec, static_cast<const void*>(x), g, part, st);
    if ((rc = launched("fwd_stats"))) return rc;
    launch_fwd_apply(dtype, vec, x, g, static_cast<const Partial*>(part), prm, true, fm, st);
    return launched(fwd_name(fm));
}

const char* bwd_name(int bm, bool ii) {
    return bm == kBwdFromXZ     ? "standard backward"
           : bm == kBwdFromXhat ? "checkpointing backward"
           : ii                 ? "backward (formulation II)"
                                : "backward";
}

// Backward of every formulation (bm, ii: see BwdSign).  u is z, x or xhat;
// zs is the stored z for kBwdFromXZ; dz_dx holds dz on entry, dx on return.
int backward_impl(int bm, bool ii, const void* u, const void* zs, void* dz_dx, int dtype,
                  const float* gamma, const float* beta, const float* save_mean,
                  const float* save_var, float* dgamma, float* dbeta, float eps, float slope,
                  int64_t N, int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                  void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!u || !dz_dx || !gamma || !beta || !save_var || !dgamma || !dbeta ||
        (bm == kBwdFromXZ && (!zs || !save_mean)))
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const int vec = access_vec(HW, dtype, u, dz_dx, bm == kBwdFromXZ ? zs : nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, save_mean, save_var, dgamma, dbeta, eps, slope, ii ? 1 : 0};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    FusedPlan fp;
    if (plan_fused(C, g, elem_bytes(dtype), true, bm == kBwdFromZ, &fp)) {
        if (!launch_bwd_fused(dtype, bm, u, zs, dz_dx, g, fp, prm, st))
            return fail(IABN_ERR_HIP, "no %s kernel built for T=%d R=%d", bwd_name(bm, ii), fp.T, fp.R);
        return launched(bwd_name(bm, ii));
    }
    Partial* part = static_cast<Partial*>(workspace);
    launch_bwd_reduce(dtype, vec, u, zs, static_cast<const void*>(dz_dx), g, prm, bm, part, st);
    if ((rc = launched("bwd_reduce"))) return rc;
    launch_bwd_apply(dtype, vec, u, zs, dz_dx, g, static_cast<const Partial*>(part), prm, bm, st);
    return launched(bwd_name(bm, ii));
}

// ---------------------------------------------------------------- static scratch

// The scratch of iabn_forward_train_noalloc: the streaming kernels' partial
// results, in a file-scope device array instead of a caller's workspace.
// Each device holds its own copy (zero-initialised when the library's code
// object is loaded on it) until the process ends.  Its size bounds the
// partials of one call: C * P slices * 4 waves * 32 bytes, at most 765
// slices (C = 255, P = 3) where the forward takes the streaming kernels,
// about 96 KiB.  Nothing in it needs to start at zero: every partial a call
// reads was written by the same call.
constexpr size_t kScratchBytes = size_t(128) << 10;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// The device address of `scratch` on each device (null until first use),
// taken with that device current; host code uses these, never `scratch`.
constexpr int kMaxDevices = 64;
void* g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mutex;

int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(IABN_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(IABN_ERR_HIP, "device %d: the scratch table holds %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return fail(IABN_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_addr[dev] = p;
    }
    *out = g_scratch_addr[dev];
    return IABN_OK;
}

}  // namespace
}  // namespace iabn_impl

using namespace iabn_impl;

// ---------------------------------------------------------------- C ABI

extern "C" {

int iabn_version(void) { return IABN_VERSION; }

const char* iabn_status_string(int status) {
    switch (status) {
        case IABN_OK: return "IABN_OK";
        case IABN_ERR_NULL: return "IABN_ERR_NULL: a required pointer is NULL";
        case IABN_ERR_SHAPE: return "IABN_ERR_SHAPE: invalid tensor shape";
        case IABN_ERR_PARAM: return "IABN_ERR_PARAM: eps, momentum or slope out of range";
        case IABN_ERR_DTYPE: return "IABN_ERR_DTYPE: unknown storage type";
        case IABN_ERR_WORKSPACE: return "IABN_ERR_WORKSPACE: workspace too small or misaligned";
        case IABN_ERR_HIP: return "IABN_ERR_HIP: the HIP runtime rejected a launch";
        default: return "unknown iabn status";
    }
}

const char* iabn_last_error(void) { return g_last_error; }

size_t iabn_workspace_size(int64_t N, int64_t C, int64_t HW, int dtype) {
    if (!valid_dtype(dtype)) return 0;
    if (check_shape(N, C, HW, false) != IABN_OK) return 0;
    return workspace_bytes_for(N, C, HW);
}

int iabn_plan(int op, int dtype, int64_t N, int64_t C, int64_t HW, iabn_plan_t* plan) {
    if (plan == nullptr) return fail(IABN_ERR_NULL, "plan is NULL");
    if (op < IABN_OP_FORWARD_TRAIN || op > IABN_OP_CKPT_RECOMPUTE)
        return fail(IABN_ERR_PARAM, "unknown op %d", op);
    const bool train = op != IABN_OP_FORWARD_EVAL && op != IABN_OP_CKPT_RECOMPUTE;
    int rc = validate_common(dtype, N, C, HW, train);
    if (rc) return rc;
    memset(plan, 0, sizeof *plan);
    if (empty(N, C, HW)) return ok();
    // The same choices as the entry points make, on aligned tensors.
    const int vec = access_vec(HW, dtype, nullptr, nullptr, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec,
                             op == IABN_OP_FORWARD_EVAL ? eval_target_blocks(C) : kTargetBlocks);
    const int eb = elem_bytes(dtype);
    const bool backward =
        op == IABN_OP_BACKWARD || op == IABN_OP_STD_BACKWARD || op == IABN_OP_CKPT_BACKWARD;
    const bool narrow_ok = op == IABN_OP_FORWARD_TRAIN || op == IABN_OP_BACKWARD;
    plan->access_bytes = vec * eb;
    plan->xcd_order = static_cast<int>(g.xcd_order);
    FusedPlan fp;
    if (train && plan_fused(C, g, eb, backward, narrow_ok, &fp)) {
        const int64_t past = static_cast<int64_t>(g.vchan) - static_cast<int64_t>(fp.T) * fp.R;
        const int64_t past_per_thread = past > 0 ? (past + fp.T - 1) / fp.T : 0;
        const int64_t lds = fused_lds_accesses(fp.T, backward, op == IABN_OP_STD_BACKWARD);
        plan->channel_resident = 1;
        plan->threads = fp.T * fp.cpb;
        plan->reg_accesses = fp.R;
        plan->lds_accesses = static_cast<int>(past_per_thread < lds ? past_per_thread : lds);
        plan->strips = fused_strips(g, fp, vec * eb == 16) ? 1 : 0;
        plan->blocks = C / fp.cpb;
        plan->channels_per_block = fp.cpb;
    } else {
        plan->threads = kThreads;
        plan->blocks = C * static_cast<int64_t>(g.P);
    }
    return ok();
}

int iabn_forward_stats(const void* x, int dtype, int64_t N, int64_t C, int64_t HW,
                       void* workspace, size_t workspace_bytes, void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (x == nullptr) return fail(IABN_ERR_NULL, "x is NULL");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const int vec = access_vec(HW, dtype, x, nullptr, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    launch_fwd_stats(dtype, vec, x, g, static_cast<Partial*>(workspace),
                     static_cast<hipStream_t>(stream));
    return launched("fwd_stats");
}

int iabn_forward_apply(void* x_z, int dtype, const float* gamma, const float* beta,
                       float* running_mean, float* running_var, float* save_mean,
                       float* save_var, float eps, float momentum, float slope, int64_t N,
                       int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                       void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!x_z || !gamma || !beta || !running_mean || !running_var || !save_mean || !save_var)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if (!(momentum >= 0.f && momentum <= 1.f))
        return fail(IABN_ERR_PARAM, "momentum must lie in [0, 1]");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const int vec = access_vec(HW, dtype, x_z, nullptr, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const FwdParams prm = {gamma, beta, running_mean, running_var, save_mean, save_var,
                           nullptr, eps, momentum, slope};
    launch_fwd_apply(dtype, vec, x_z, g, static_cast<const Partial*>(workspace), prm, true,
                     kFwdInPlace, static_cast<hipStream_t>(stream));
    return launched("fwd_apply");
}

int iabn_forward_train(void* x_z, int dtype, const float* gamma, const float* beta,
                       float* running_mean, float* running_var, float* save_mean,
                       float* save_var, float eps, float momentum, float slope, int64_t N,
                       int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                       void* stream) {
    return forward_train_impl(kFwdInPlace, x_z, nullptr, dtype, gamma, beta, running_mean,
                              running_var, save_mean, save_var, eps, momentum, slope, N, C, HW,
                              workspace, workspace_bytes, stream);
}

int iabn_forward_train_noalloc(void* x_z, int dtype, const float* gamma, const float* beta,
                               float* running_mean, float* running_var, float* save_mean,
                               float* save_var, float eps, float momentum, float slope, int64_t N,
                               int64_t C, int64_t HW, void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    const size_t need = workspace_bytes_for(N, C, HW);
    const int vec = access_vec(HW, dtype, x_z, nullptr, nullptr);
    FusedPlan fp;
    const bool fused =
        plan_fused(C, make_geom(N, C, HW, dtype, vec), elem_bytes(dtype), false, true, &fp);
    if (!fused && need > kScratchBytes)
        return fail(IABN_ERR_WORKSPACE,
                    "this shape needs %zu bytes of scratch, more than the %zu the library "
                    "holds per device",
                    need, kScratchBytes);
    void* ws = nullptr;
    if ((rc = scratch_address(&ws))) return rc;
    return forward_train_impl(kFwdInPlace, x_z, nullptr, dtype, gamma, beta, running_mean,
                              running_var, save_mean, save_var, eps, momentum, slope, N, C, HW, ws,
                              kScratchBytes, stream, true);
}

int iabn_forward_eval(void* x_z, int dtype, const float* gamma, const float* beta,
                      const float* running_mean, const float* running_var, float eps,
                      float slope, int64_t N, int64_t C, int64_t HW, void* stream) {
    int rc = validate_common(dtype, N, C, HW, false);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!x_z || !gamma || !beta || !running_mean || !running_var)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    const int vec = access_vec(HW, dtype, x_z, nullptr, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec, eval_target_blocks(C));
    const FwdParams prm = {gamma, beta, const_cast<float*>(running_mean),
                           const_cast<float*>(running_var), nullptr, nullptr, nullptr, eps, 0.f,
                           slope};
    launch_fwd_apply(dtype, vec, x_z, g, static_cast<const Partial*>(nullptr), prm, false,
                     kFwdInPlace, static_cast<hipStream_t>(stream));
    return launched("fwd_eval");
}

int iabn_backward_reduce(const void* z, const void* dz, int dtype, const float* gamma,
                         const float* beta, float slope, int64_t N, int64_t C, int64_t HW,
                         void* workspace, size_t workspace_bytes, void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!z || !dz || !gamma || !beta)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if (!(slope > 0.f) || !std::isfinite(slope))
        return fail(IABN_ERR_PARAM, "slope must be finite and > 0 (the activation must be invertible)");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const int vec = access_vec(HW, dtype, z, dz, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, nullptr, nullptr, nullptr, nullptr, 1.f, slope, 0};
    launch_bwd_reduce(dtype, vec, z, static_cast<const void*>(nullptr), dz, g, prm, kBwdFromZ,
                      static_cast<Partial*>(workspace), static_cast<hipStream_t>(stream));
    return launched("bwd_reduce");
}

int iabn_backward_apply(const void* z, void* dz_dx, int dtype, const float* gamma,
                        const float* beta, const float* save_var, float* dgamma, float* dbeta,
                        float eps, float slope, int64_t N, int64_t C, int64_t HW,
                        void* workspace, size_t workspace_bytes, void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!z || !dz_dx || !gamma || !beta || !save_var || !dgamma || !dbeta)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const int vec = access_vec(HW, dtype, z, dz_dx, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, nullptr, save_var, dgamma, dbeta, eps, slope, 0};
    launch_bwd_apply(dtype, vec, z, static_cast<const void*>(nullptr), dz_dx, g,
                     static_cast<const Partial*>(workspace), prm, kBwdFromZ,
                     static_cast<hipStream_t>(stream));
    return launched("bwd_apply");
}

int iabn_backward(const void* z, void* dz_dx, int dtype, const float* gamma, const float* beta,
                  const float* save_var, float* dgamma, float* dbeta, float eps, float slope,
                  int64_t N, int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                  void* stream) {
    return backward_impl(kBwdFromZ, false, z, nullptr, dz_dx, dtype, gamma, beta, nullptr,
                         save_var, dgamma, dbeta, eps, slope, N, C, HW, workspace,
                         workspace_bytes, stream);
}

int iabn_backward_ii(const void* z, void* dz_dx, int dtype, const float* gamma,
                     const float* beta, const float* save_var, float* dgamma, float* dbeta,
                     float eps, float slope, int64_t N, int64_t C, int64_t HW, void* workspace,
                     size_t workspace_bytes, void* stream) {
    return backward_impl(kBwdFromZ, true, z, nullptr, dz_dx, dtype, gamma, beta, nullptr,
                         save_var, dgamma, dbeta, eps, slope, N, C, HW, workspace,
                         workspace_bytes, stream);
}

int iabn_std_forward_train(const void* x, void* z, int dtype, const float* gamma,
                           const float* beta, float* running_mean, float* running_var,
                           float* save_mean, float* save_var, float eps, float momentum,
                           float slope, int64_t N, int64_t C, int64_t HW, void* workspace,
                           size_t workspace_bytes, void* stream) {
    return forward_train_impl(kFwdOut, const_cast<void*>(x), z, dtype, gamma, beta, running_mean,
                              running_var, save_mean, save_var, eps, momentum, slope, N, C, HW,
                              workspace, workspace_bytes, stream);
}

int iabn_std_backward(const void* x, const void* z, void* dz_dx, int dtype, const float* gamma,
                      const float* beta, const float* save_mean, const float* save_var,
                      float* dgamma, float* dbeta, float eps, float slope, int64_t N, int64_t C,
                      int64_t HW, void* workspace, size_t workspace_bytes, void* stream) {
    return backward_impl(kBwdFromXZ, false, x, z, dz_dx, dtype, gamma, beta, save_mean, save_var,
                         dgamma, dbeta, eps, slope, N, C, HW, workspace, workspace_bytes, stream);
}

int iabn_ckpt_forward_train(void* x_xhat, void* z, int dtype, const float* gamma,
                            const float* beta, float* running_mean, float* running_var,
                            float* save_mean, float* save_var, float eps, float momentum,
                            float slope, int64_t N, int64_t C, int64_t HW, void* workspace,
                            size_t workspace_bytes, void* stream) {
    return forward_train_impl(kFwdCkpt, x_xhat, z, dtype, gamma, beta, running_mean, running_var,
                              save_mean, save_var, eps, momentum, slope, N, C, HW, workspace,
                              workspace_bytes, stream);
}

int iabn_ckpt_recompute(const void* xhat, void* z, int dtype, const float* gamma,
                        const float* beta, float slope, int64_t N, int64_t C, int64_t HW,
                        void* stream) {
    int rc = validate_common(dtype, N, C, HW, false);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!xhat || !z || !gamma || !beta)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(1.f, slope))) return rc;
    const int vec = access_vec(HW, dtype, xhat, z, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    launch_recompute(dtype, vec, xhat, z, g, gamma, beta, slope, static_cast<hipStream_t>(stream));
    return launched("recompute");
}

int iabn_ckpt_backward(const void* xhat, void* dz_dx, int dtype, const float* gamma,
                       const float* beta, const float* save_var, float* dgamma, float* dbeta,
                       float eps, float slope, int64_t N, int64_t C, int64_t HW,
                       void* workspace, size_t workspace_bytes, void* stream) {
    return backward_impl(kBwdFromXhat, false, xhat, nullptr, dz_dx, dtype, gamma, beta, nullptr,
                         save_var, dgamma, dbeta, eps, slope, N, C, HW, workspace,
                         workspace_bytes, stream);
}

}  // extern "C"
