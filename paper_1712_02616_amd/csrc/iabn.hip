// libiabn: InPlace-ABN (arXiv:1712.02616) for AMD Instinct MI355X (gfx950).
//
// Four streaming kernels, all bound by HBM bandwidth:
//   fwd_stats    reads x, writes per-(channel, slice) partial moments
//   fwd_apply    combines a channel's partials (fixed order), writes the
//                statistics, overwrites x with z = f(gamma*xhat + beta)
//   bwd_reduce   reads z and dz, writes per-(channel, slice) partial sums of
//                dy and dy*xhat, with y = f^-1(z) and xhat = (y - beta)/gamma
//   bwd_apply    combines the partial sums, writes dgamma/dbeta, overwrites
//                dz with dx
// plus fwd_apply in inference mode.
//
// Work decomposition.  A channel's m = N*HW values are N rows of HW
// contiguous elements, C*HW elements apart.  Each channel is cut into P
// slices of L elements (the last one shorter); one 256-thread block owns one
// (channel, slice) pair, so each block sees a single channel and reads its
// parameters once.  Slices are defined in elements, independent of the
// access width, so the partials of a slice mean the same thing whichever
// path wrote them.  Inside a slice a thread reads 16-byte vectors
// v = lo + tid, lo + tid + 256, ... (consecutive lanes touch consecutive 16
// bytes), U of them in flight before any arithmetic.  A vector never crosses
// a row because HW is a multiple of the vector width on the vector path;
// otherwise (odd HW, or a pointer not 16-byte aligned) the same kernels run
// with one element per access.
//
// In place.  Every element is read and then written by the same thread in
// the same kernel, so x -> z and dz -> dx need no synchronisation between
// threads.  The backward's apply kernel reads dz before overwriting it, and
// runs after the reduce kernel on the same stream.
//
// Determinism.  Each block reduces in a fixed shuffle tree, then across its
// four waves in a fixed order; the apply kernels combine a channel's P
// partials in a fixed tree.  Nothing depends on scheduling, so results are
// bit-identical from run to run.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <cmath>

#include "divmagic.h"
#include "iabn.h"

#define IABN_VERSION 10000

namespace {

constexpr int kThreads = 256;
constexpr int kWave = 64;
constexpr int kWaves = kThreads / kWave;

// ---------------------------------------------------------------- storage

template <int DT>
struct Elem;
template <>
struct Elem<IABN_F32> {
    using T = float;
};
template <>
struct Elem<IABN_F16> {
    using T = _Float16;
};
template <>
struct Elem<IABN_BF16> {
    using T = __bf16;
};

// VEC elements per access: 16 bytes on the vector path, 1 on the scalar path.
template <int DT, int VEC>
__device__ __forceinline__ void load_vec(const void* __restrict__ base, uint64_t idx,
                                         float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    if constexpr (VEC == 1) {
        v[0] = static_cast<float>(static_cast<const T*>(base)[idx]);
    } else {
        typedef T vt __attribute__((ext_vector_type(VEC)));
        typedef float vf __attribute__((ext_vector_type(VEC)));
        const vt r = static_cast<const vt*>(base)[idx];
        const vf f = __builtin_convertvector(r, vf);
#pragma unroll
        for (int k = 0; k < VEC; ++k) v[k] = f[k];
    }
}

// fp32 -> storage conversions round to nearest even.
template <int DT, int VEC>
__device__ __forceinline__ void store_vec(void* __restrict__ base, uint64_t idx,
                                          const float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    if constexpr (VEC == 1) {
        static_cast<T*>(base)[idx] = static_cast<T>(v[0]);
    } else {
        typedef T vt __attribute__((ext_vector_type(VEC)));
        typedef float vf __attribute__((ext_vector_type(VEC)));
        vf f;
#pragma unroll
        for (int k = 0; k < VEC; ++k) f[k] = v[k];
        static_cast<vt*>(base)[idx] = __builtin_convertvector(f, vt);
    }
}

// ---------------------------------------------------------------- geometry

struct Geom {
    uint32_t C;      // channels
    uint32_t P;      // slices per channel
    uint32_t vrow;   // accesses per row (HW / VEC)
    uint32_t vchan;  // accesses per channel (N * vrow)
    uint32_t lv;     // accesses per slice (the last slice may be shorter)
    uint32_t vec;    // elements per access
    iabn_divmagic_t row_div;  // division by vrow
    uint64_t nstride;         // accesses between samples of a channel (C * vrow)
    double m;                 // elements per channel (N * HW)
};

// Index (in accesses) of the v-th access of channel c.
__device__ __forceinline__ uint64_t access_index(const Geom& g, uint64_t cbase, uint32_t v) {
    const uint32_t n = iabn_divmagic_div(v, g.row_div);
    const uint32_t i = v - n * g.vrow;
    return static_cast<uint64_t>(n) * g.nstride + cbase + i;
}

struct Slice {
    uint32_t c, p, lo, hi;
};

__device__ __forceinline__ Slice block_slice(const Geom& g) {
    Slice s;
    s.c = blockIdx.x / g.P;
    s.p = blockIdx.x - s.c * g.P;
    s.lo = s.p * g.lv;
    s.hi = min(s.lo + g.lv, g.vchan);
    return s;
}

// Elements in slice p of a channel.
__device__ __forceinline__ double slice_count(const Geom& g, uint32_t p) {
    const uint32_t lo = p * g.lv;
    const uint32_t hi = min(lo + g.lv, g.vchan);
    return static_cast<double>(hi - lo) * static_cast<double>(g.vec);
}

// ---------------------------------------------------------------- reductions

// Count, mean and sum of squared deviations of a set of values, in double.
// Two sets combine with the pairwise update of Chan, Golub and LeVeque
// (1979).  Per-element work stays in fp32 (see fwd_stats_kernel); only the
// per-thread results and everything after them are double, which costs a few
// dozen instructions per thread and keeps large channel means from eating
// the fp32 mantissa.
struct Moments {
    double n, mean, m2;
};

__device__ __forceinline__ Moments chan_merge(const Moments& a, const Moments& b) {
    const double n = a.n + b.n;
    const double wb = n > 0.0 ? b.n / n : 0.0;
    const double d = b.mean - a.mean;
    Moments r;
    r.n = n;
    r.mean = fma(d, wb, a.mean);
    r.m2 = a.m2 + b.m2 + d * d * a.n * wb;
    return r;
}

// Fixed-order tree over a wave; lane 0 ends with the merge of all 64 lanes.
__device__ __forceinline__ Moments wave_merge(Moments a) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        Moments b;
        b.n = __shfl_down(a.n, off, kWave);
        b.mean = __shfl_down(a.mean, off, kWave);
        b.m2 = __shfl_down(a.m2, off, kWave);
        if ((threadIdx.x & (kWave - 1)) < static_cast<unsigned>(off)) a = chan_merge(a, b);
    }
    return a;
}

__device__ __forceinline__ double2 wave_sum(double2 a) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        a.x += __shfl_down(a.x, off, kWave);
        a.y += __shfl_down(a.y, off, kWave);
    }
    return a;
}

// Combine a channel's P partial moments (fixed order); run by one full wave,
// the result is valid in lane 0.
__device__ __forceinline__ Moments combine_channel_moments(const Geom& g,
                                                           const double2* __restrict__ part,
                                                           uint32_t c) {
    const uint32_t lane = threadIdx.x & (kWave - 1);
    Moments acc = {0.0, 0.0, 0.0};
    for (uint32_t p = lane; p < g.P; p += kWave) {
        const double2 pm = part[static_cast<uint64_t>(c) * g.P + p];
        const Moments b = {slice_count(g, p), pm.x, pm.y};
        acc = chan_merge(acc, b);
    }
    return wave_merge(acc);
}

__device__ __forceinline__ double2 combine_channel_sums(const Geom& g,
                                                        const double2* __restrict__ part,
                                                        uint32_t c) {
    const uint32_t lane = threadIdx.x & (kWave - 1);
    double2 acc = make_double2(0.0, 0.0);
    for (uint32_t p = lane; p < g.P; p += kWave) {
        const double2 s = part[static_cast<uint64_t>(c) * g.P + p];
        acc.x += s.x;
        acc.y += s.y;
    }
    return wave_sum(acc);
}

// ---------------------------------------------------------------- forward

// Partial moments of one (channel, slice): part[c*P + p] = (mean, M2).
//
// Each thread accumulates shifted sums S1 = sum(x - K), S2 = sum((x - K)^2)
// in fp32 with K = the first value it reads, which sits within a few standard
// deviations of the mean, so x - K carries the spread and not the offset
// (and is exact when x and K are within a factor of two).  The thread's
// moments are then mean = K + S1/n, M2 = S2 - S1^2/n, formed in double.
template <int DT, int VEC, int U>
__global__ __launch_bounds__(kThreads) void fwd_stats_kernel(const void* __restrict__ x, Geom g,
                                                             double2* __restrict__ part) {
    const Slice s = block_slice(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    float shift = 0.f, s1 = 0.f, s2 = 0.f;
    bool first = true;
    uint32_t nacc = 0;
    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float t[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) load_vec<DT, VEC>(x, access_index(g, cbase, v + u * kThreads), t[u]);
        if (first) shift = t[0][0];
        first = false;
        float a1 = 0.f, a2 = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                const float d = t[u][k] - shift;
                a1 += d;
                a2 = fmaf(d, d, a2);
            }
        }
        s1 += a1;
        s2 += a2;
        nacc += U;
    }
    for (; v < s.hi; v += kThreads) {
        float t[VEC];
        load_vec<DT, VEC>(x, access_index(g, cbase, v), t);
        if (first) shift = t[0];
        first = false;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const float d = t[k] - shift;
            s1 += d;
            s2 = fmaf(d, d, s2);
        }
        nacc += 1;
    }
    Moments acc = {0.0, 0.0, 0.0};
    if (nacc > 0) {
        const double n = static_cast<double>(nacc) * g.vec;
        const double d1 = s1, d2 = s2;
        acc.n = n;
        acc.mean = static_cast<double>(shift) + d1 / n;
        acc.m2 = fmax(d2 - d1 * d1 / n, 0.0);
    }
    acc = wave_merge(acc);

    __shared__ Moments wave_acc[kWaves];
    const uint32_t wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) wave_acc[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        Moments r = wave_acc[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) r = chan_merge(r, wave_acc[w]);
        part[static_cast<uint64_t>(s.c) * g.P + s.p] = make_double2(r.mean, r.m2);
    }
}

struct FwdParams {
    const float* gamma;
    const float* beta;
    float* running_mean;
    float* running_var;
    float* save_mean;
    float* save_var;
    float eps, momentum, slope;
};

// z = f(gamma * (x - mu) / sqrt(var + eps) + beta), in place.  TRAIN: mu and
// var are the batch statistics combined from the partials (slice 0 of each
// channel also writes them out and updates the running estimates); otherwise
// they are the running estimates.  mu is applied as a two-float sum
// hi + lo, so x - mu keeps fp32 relative accuracy even when |mu| >> sigma.
template <int DT, int VEC, int U, bool TRAIN>
__global__ __launch_bounds__(kThreads) void fwd_apply_kernel(void* __restrict__ xz, Geom g,
                                                             const double2* __restrict__ part,
                                                             FwdParams prm) {
    const Slice s = block_slice(g);
    __shared__ float coef[4];
    if (threadIdx.x < kWave) {
        double mean, var;
        if constexpr (TRAIN) {
            const Moments r = combine_channel_moments(g, part, s.c);
            mean = r.mean;
            var = fmax(r.m2, 0.0) / g.m;
        } else {
            mean = prm.running_mean[s.c];
            var = prm.running_var[s.c];
        }
        if (threadIdx.x == 0) {
            const double scale = static_cast<double>(prm.gamma[s.c]) / sqrt(var + static_cast<double>(prm.eps));
            const float mean_hi = static_cast<float>(mean);
            coef[0] = mean_hi;
            coef[1] = static_cast<float>(mean - static_cast<double>(mean_hi));
            coef[2] = static_cast<float>(scale);
            coef[3] = prm.beta[s.c];
            if constexpr (TRAIN) {
                if (s.p == 0) {
                    const double mom = prm.momentum;
                    const double m = g.m;
                    prm.save_mean[s.c] = mean_hi;
                    prm.save_var[s.c] = static_cast<float>(var);
                    prm.running_mean[s.c] = static_cast<float>(
                        (1.0 - mom) * static_cast<double>(prm.running_mean[s.c]) + mom * mean);
                    prm.running_var[s.c] = static_cast<float>(
                        (1.0 - mom) * static_cast<double>(prm.running_var[s.c]) +
                        mom * var * (m / (m - 1.0)));
                }
            }
        }
    }
    __syncthreads();
    const float mean_hi = coef[0], mean_lo = coef[1], scale = coef[2], shift = coef[3];
    const float slope = prm.slope;
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    auto act = [&](float xv) {
        const float y = fmaf((xv - mean_hi) - mean_lo, scale, shift);
        return y >= 0.f ? y : slope * y;
    };

    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float t[U][VEC];
        uint64_t idx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            idx[u] = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC>(xz, idx[u], t[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) t[u][k] = act(t[u][k]);
            store_vec<DT, VEC>(xz, idx[u], t[u]);
        }
    }
    for (; v < s.hi; v += kThreads) {
        float t[VEC];
        const uint64_t idx = access_index(g, cbase, v);
        load_vec<DT, VEC>(xz, idx, t);
#pragma unroll
        for (int k = 0; k < VEC; ++k) t[k] = act(t[k]);
        store_vec<DT, VEC>(xz, idx, t);
    }
}

// ---------------------------------------------------------------- backward

// Per-element reconstruction from the stored output (Algorithm 2):
//   dy = dz * f'(y) with f' = 1 where z >= 0, slope where z < 0
//   y = f^-1(z) = z (z >= 0) or z / slope (z < 0)
//   xhat = (y - beta) / gamma
struct BwdElem {
    float slope, inv_slope, beta, inv_gamma;
    __device__ __forceinline__ void operator()(float z, float dz, float& dy, float& xhat) const {
        const bool neg = z < 0.f;
        const float y = neg ? z * inv_slope : z;
        dy = neg ? dz * slope : dz;
        xhat = (y - beta) * inv_gamma;
    }
};

// Partial sums of dy and dy*xhat of one (channel, slice):
// part[c*P + p] = (sum dy, sum dy*xhat).  fp32 per batch of U accesses,
// double across batches and threads.
template <int DT, int VEC, int U>
__global__ __launch_bounds__(kThreads) void bwd_reduce_kernel(const void* __restrict__ z,
                                                              const void* __restrict__ dz, Geom g,
                                                              const float* __restrict__ gamma,
                                                              const float* __restrict__ beta,
                                                              float slope,
                                                              double2* __restrict__ part) {
    const Slice s = block_slice(g);
    const BwdElem el = {slope, 1.0f / slope, beta[s.c], 1.0f / gamma[s.c]};
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    double2 acc = make_double2(0.0, 0.0);
    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float tz[U][VEC], tg[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t idx = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC>(z, idx, tz[u]);
            load_vec<DT, VEC>(dz, idx, tg[u]);
        }
        float sdy = 0.f, sdyx = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                float dy, xhat;
                el(tz[u][k], tg[u][k], dy, xhat);
                sdy += dy;
                sdyx = fmaf(dy, xhat, sdyx);
            }
        }
        acc.x += sdy;
        acc.y += sdyx;
    }
    for (; v < s.hi; v += kThreads) {
        float tz[VEC], tg[VEC];
        const uint64_t idx = access_index(g, cbase, v);
        load_vec<DT, VEC>(z, idx, tz);
        load_vec<DT, VEC>(dz, idx, tg);
        float sdy = 0.f, sdyx = 0.f;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float dy, xhat;
            el(tz[k], tg[k], dy, xhat);
            sdy += dy;
            sdyx = fmaf(dy, xhat, sdyx);
        }
        acc.x += sdy;
        acc.y += sdyx;
    }
    acc = wave_sum(acc);

    __shared__ double2 wave_acc[kWaves];
    const uint32_t wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) wave_acc[wave] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double2 r = wave_acc[0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) {
            r.x += wave_acc[w].x;
            r.y += wave_acc[w].y;
        }
        part[static_cast<uint64_t>(s.c) * g.P + s.p] = r;
    }
}

struct BwdParams {
    const float* gamma;
    const float* beta;
    const float* save_var;
    float* dgamma;
    float* dbeta;
    float eps, slope;
};

// dx = (dy - dgamma*xhat/m - dbeta/m) * gamma/sqrt(var + eps), in place over dz,
// as dx = A*dy + B*xhat + Cc with per-channel A, B, Cc formed in double.
template <int DT, int VEC, int U>
__global__ __launch_bounds__(kThreads) void bwd_apply_kernel(const void* __restrict__ z,
                                                             void* __restrict__ dzdx, Geom g,
                                                             const double2* __restrict__ part,
                                                             BwdParams prm) {
    const Slice s = block_slice(g);
    __shared__ float coef[3];
    if (threadIdx.x < kWave) {
        const double2 sums = combine_channel_sums(g, part, s.c);
        if (threadIdx.x == 0) {
            const double dbeta = sums.x, dgamma = sums.y, m = g.m;
            const double a = static_cast<double>(prm.gamma[s.c]) /
                             sqrt(static_cast<double>(prm.save_var[s.c]) + static_cast<double>(prm.eps));
            coef[0] = static_cast<float>(a);
            coef[1] = static_cast<float>(-a * dgamma / m);
            coef[2] = static_cast<float>(-a * dbeta / m);
            if (s.p == 0) {
                prm.dgamma[s.c] = static_cast<float>(dgamma);
                prm.dbeta[s.c] = static_cast<float>(dbeta);
            }
        }
    }
    __syncthreads();
    const float ca = coef[0], cb = coef[1], cc = coef[2];
    const BwdElem el = {prm.slope, 1.0f / prm.slope, prm.beta[s.c], 1.0f / prm.gamma[s.c]};
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    auto dx_of = [&](float zv, float gv) {
        float dy, xhat;
        el(zv, gv, dy, xhat);
        return fmaf(ca, dy, fmaf(cb, xhat, cc));
    };

    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float tz[U][VEC], tg[U][VEC];
        uint64_t idx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            idx[u] = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC>(z, idx[u], tz[u]);
            load_vec<DT, VEC>(dzdx, idx[u], tg[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) tg[u][k] = dx_of(tz[u][k], tg[u][k]);
            store_vec<DT, VEC>(dzdx, idx[u], tg[u]);
        }
    }
    for (; v < s.hi; v += kThreads) {
        float tz[VEC], tg[VEC];
        const uint64_t idx = access_index(g, cbase, v);
        load_vec<DT, VEC>(z, idx, tz);
        load_vec<DT, VEC>(dzdx, idx, tg);
#pragma unroll
        for (int k = 0; k < VEC; ++k) tg[k] = dx_of(tz[k], tg[k]);
        store_vec<DT, VEC>(dzdx, idx, tg);
    }
}

// ---------------------------------------------------------------- host side

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
constexpr int64_t kTargetBlocks = 2048;    // 8 blocks of 4 waves per CU on 256 CUs
constexpr int64_t kMinSliceElems = 4096;   // at least 16 elements per thread
constexpr int64_t kMaxSlices = 1024;
constexpr int64_t kSliceAlign = 8;         // slices start on a 16-byte access of any dtype

int elem_bytes(int dtype) { return dtype == IABN_F32 ? 4 : 2; }

bool valid_dtype(int dtype) { return dtype == IABN_F32 || dtype == IABN_F16 || dtype == IABN_BF16; }

// Slices per channel and slice length in elements; depends on the shape only.
struct Split {
    int64_t P;
    int64_t L;
};

Split split_channel(int64_t m, int64_t C) {
    int64_t P = (kTargetBlocks + C - 1) / C;
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
    return static_cast<size_t>(C) * static_cast<size_t>(sp.P) * sizeof(double2);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// The access geometry.  vector=true uses 16-byte accesses (requires
// HW % (16/elem) == 0 and 16-byte aligned pointers).
Geom make_geom(int64_t N, int64_t C, int64_t HW, int dtype, bool vector) {
    const int64_t m = N * HW;
    const Split sp = split_channel(m, C);
    const int64_t vec = vector ? 16 / elem_bytes(dtype) : 1;
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
    return g;
}

bool use_vector(int64_t HW, int dtype, const void* a, const void* b) {
    const int64_t vec = 16 / elem_bytes(dtype);
    return HW % vec == 0 && aligned16(a) && (b == nullptr || aligned16(b));
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

dim3 grid_of(const Geom& g) { return dim3(g.C * g.P); }

// Dispatch on dtype and access width.
template <template <int, int> class Launch, typename... A>
void dispatch(int dtype, bool vector, A&&... args) {
    switch (dtype) {
        case IABN_F32:
            if (vector) Launch<IABN_F32, 4>::run(args...);
            else Launch<IABN_F32, 1>::run(args...);
            break;
        case IABN_F16:
            if (vector) Launch<IABN_F16, 8>::run(args...);
            else Launch<IABN_F16, 1>::run(args...);
            break;
        default:
            if (vector) Launch<IABN_BF16, 8>::run(args...);
            else Launch<IABN_BF16, 1>::run(args...);
            break;
    }
}

// Accesses in flight per thread: 4 x 16 bytes on the vector path, 8 single
// elements on the scalar path.
template <int VEC>
constexpr int unroll() {
    return VEC == 1 ? 8 : 4;
}

template <int DT, int VEC>
struct LaunchFwdStats {
    static void run(const void* x, const Geom& g, double2* part, hipStream_t st) {
        fwd_stats_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(x, g, part);
    }
};

template <int DT, int VEC>
struct LaunchFwdApply {
    static void run(void* xz, const Geom& g, const double2* part, const FwdParams& prm, bool train,
                    hipStream_t st) {
        if (train)
            fwd_apply_kernel<DT, VEC, unroll<VEC>(), true><<<grid_of(g), kThreads, 0, st>>>(
                xz, g, part, prm);
        else
            fwd_apply_kernel<DT, VEC, unroll<VEC>(), false><<<grid_of(g), kThreads, 0, st>>>(
                xz, g, part, prm);
    }
};

template <int DT, int VEC>
struct LaunchBwdReduce {
    static void run(const void* z, const void* dz, const Geom& g, const float* gamma,
                    const float* beta, float slope, double2* part, hipStream_t st) {
        bwd_reduce_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(
            z, dz, g, gamma, beta, slope, part);
    }
};

template <int DT, int VEC>
struct LaunchBwdApply {
    static void run(const void* z, void* dzdx, const Geom& g, const double2* part,
                    const BwdParams& prm, hipStream_t st) {
        bwd_apply_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(z, dzdx, g,
                                                                                   part, prm);
    }
};

int validate_common(int dtype, int64_t N, int64_t C, int64_t HW, bool train) {
    if (!valid_dtype(dtype)) return fail(IABN_ERR_DTYPE, "unknown dtype %d", dtype);
    return check_shape(N, C, HW, train);
}

bool empty(int64_t N, int64_t C, int64_t HW) { return C == 0 || N * HW == 0; }

}  // namespace

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

int iabn_forward_stats(const void* x, int dtype, int64_t N, int64_t C, int64_t HW,
                       void* workspace, size_t workspace_bytes, void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (x == nullptr) return fail(IABN_ERR_NULL, "x is NULL");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const bool vec = use_vector(HW, dtype, x, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    dispatch<LaunchFwdStats>(dtype, vec, x, g, static_cast<double2*>(workspace),
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
    const bool vec = use_vector(HW, dtype, x_z, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const FwdParams prm = {gamma, beta, running_mean, running_var, save_mean, save_var,
                           eps,   momentum, slope};
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const double2*>(workspace), prm, true,
                             static_cast<hipStream_t>(stream));
    return launched("fwd_apply");
}

int iabn_forward_train(void* x_z, int dtype, const float* gamma, const float* beta,
                       float* running_mean, float* running_var, float* save_mean,
                       float* save_var, float eps, float momentum, float slope, int64_t N,
                       int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                       void* stream) {
    // Validate everything before the first launch so that an error changes nothing.
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!x_z || !gamma || !beta || !running_mean || !running_var || !save_mean || !save_var)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if (!(momentum >= 0.f && momentum <= 1.f))
        return fail(IABN_ERR_PARAM, "momentum must lie in [0, 1]");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    if ((rc = iabn_forward_stats(x_z, dtype, N, C, HW, workspace, workspace_bytes, stream)))
        return rc;
    return iabn_forward_apply(x_z, dtype, gamma, beta, running_mean, running_var, save_mean,
                              save_var, eps, momentum, slope, N, C, HW, workspace,
                              workspace_bytes, stream);
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
    const bool vec = use_vector(HW, dtype, x_z, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const FwdParams prm = {gamma, beta, const_cast<float*>(running_mean),
                           const_cast<float*>(running_var), nullptr, nullptr, eps, 0.f, slope};
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const double2*>(nullptr), prm, false,
                             static_cast<hipStream_t>(stream));
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
    const bool vec = use_vector(HW, dtype, z, dz);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    dispatch<LaunchBwdReduce>(dtype, vec, z, dz, g, gamma, beta, slope,
                              static_cast<double2*>(workspace), static_cast<hipStream_t>(stream));
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
    const bool vec = use_vector(HW, dtype, z, dz_dx);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, save_var, dgamma, dbeta, eps, slope};
    dispatch<LaunchBwdApply>(dtype, vec, z, dz_dx, g, static_cast<const double2*>(workspace), prm,
                             static_cast<hipStream_t>(stream));
    return launched("bwd_apply");
}

int iabn_backward(const void* z, void* dz_dx, int dtype, const float* gamma, const float* beta,
                  const float* save_var, float* dgamma, float* dbeta, float eps, float slope,
                  int64_t N, int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                  void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!z || !dz_dx || !gamma || !beta || !save_var || !dgamma || !dbeta)
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    if ((rc = iabn_backward_reduce(z, dz_dx, dtype, gamma, beta, slope, N, C, HW, workspace,
                                   workspace_bytes, stream)))
        return rc;
    return iabn_backward_apply(z, dz_dx, dtype, gamma, beta, save_var, dgamma, dbeta, eps, slope,
                               N, C, HW, workspace, workspace_bytes, stream);
}

}  // extern "C"
