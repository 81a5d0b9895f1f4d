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
// Reductions.  Every wave of a reduction kernel writes one partial result
// (no block barrier); each wave of an apply kernel combines its channel's
// partials itself, while its first data loads are already in flight.  All
// combines run in a fixed order, so results are bit-identical from run to
// run.

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

// Cache hint of an access: kCached for data that is read again soon (it
// should stay in the caches), kStream for the last touch of a tensor in a
// pass (non-temporal: do not displace data that is reused).
constexpr int kCached = 0;
constexpr int kStream = 1;

// VEC elements per access: 16 bytes on the vector path, 1 on the scalar path.
template <int DT, int VEC, int HINT>
__device__ __forceinline__ void load_vec(const void* __restrict__ base, uint64_t idx,
                                         float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    if constexpr (VEC == 1) {
        const T* p = static_cast<const T*>(base) + idx;
        v[0] = static_cast<float>(HINT == kStream ? __builtin_nontemporal_load(p) : *p);
    } else {
        typedef T vt __attribute__((ext_vector_type(VEC)));
        typedef float vf __attribute__((ext_vector_type(VEC)));
        const vt* p = static_cast<const vt*>(base) + idx;
        const vt r = HINT == kStream ? __builtin_nontemporal_load(p) : *p;
        const vf f = __builtin_convertvector(r, vf);
#pragma unroll
        for (int k = 0; k < VEC; ++k) v[k] = f[k];
    }
}

// fp32 -> storage conversions round to nearest even.
template <int DT, int VEC, int HINT>
__device__ __forceinline__ void store_vec(void* __restrict__ base, uint64_t idx,
                                          const float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    if constexpr (VEC == 1) {
        T* p = static_cast<T*>(base) + idx;
        const T r = static_cast<T>(v[0]);
        if constexpr (HINT == kStream) __builtin_nontemporal_store(r, p);
        else *p = r;
    } else {
        typedef T vt __attribute__((ext_vector_type(VEC)));
        typedef float vf __attribute__((ext_vector_type(VEC)));
        vf f;
#pragma unroll
        for (int k = 0; k < VEC; ++k) f[k] = v[k];
        const vt r = __builtin_convertvector(f, vt);
        vt* p = static_cast<vt*>(base) + idx;
        if constexpr (HINT == kStream) __builtin_nontemporal_store(r, p);
        else *p = r;
    }
}

// Cache hints of the four passes.  x is read by the statistics pass and
// again by the forward apply pass; z and dz are read by the backward reduce
// pass and again by the backward apply pass.  z and dx are written for a
// consumer that runs much later (the backward / the previous layer).
constexpr int kHintStatsLoad = kCached;
constexpr int kHintFwdApplyLoad = kStream;
constexpr int kHintFwdApplyStore = kStream;
constexpr int kHintReduceLoad = kCached;
constexpr int kHintBwdApplyLoad = kStream;
constexpr int kHintBwdApplyStore = kStream;
// Apply passes visit the slices in reverse order of their reduction pass.
constexpr bool kReverseApply = false;

// ---------------------------------------------------------------- geometry

struct Geom {
    uint32_t C;      // channels
    uint32_t P;      // slices per channel (one block each)
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

// REVERSE walks the slices from the last to the first: an apply pass then
// starts on the data its reduction pass fetched most recently, which is the
// data most likely still in the caches.
template <bool REVERSE = false>
__device__ __forceinline__ Slice block_slice(const Geom& g) {
    Slice s;
    const uint32_t b = REVERSE ? gridDim.x - 1 - blockIdx.x : blockIdx.x;
    s.c = b / g.P;
    s.p = b - s.c * g.P;
    s.lo = s.p * g.lv;
    s.hi = min(s.lo + g.lv, g.vchan);
    return s;
}

// ---------------------------------------------------------------- partials

// One partial result per wave of a reduction kernel, 32 bytes:
//   forward:  k, s1 = sum(x - k), s2 = sum((x - k)^2), n   (shifted sums)
//   backward: sum dy, sum dy*xhat, 0, 0
// A channel's partials are part[(c*P + p)*kWaves + w].
struct alignas(16) Partial {
    double a, b, c, d;
};

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_down(v, off, kWave);
    return v;  // valid in lane 0
}

// Shifted sums re-expressed about another shift:
//   sum(x - k') = s1 + n d,  sum((x - k')^2) = s2 + d (2 s1 + n d),  d = k - k'.
__device__ __forceinline__ void reshift(double& s1, double& s2, double n, double k_from,
                                        double k_to) {
    const double d = k_from - k_to;
    s2 += d * (2.0 * s1 + n * d);
    s1 += n * d;
}

// Batch mean and biased variance of channel c from its P*kWaves partials,
// combined in a fixed order by every lane of the calling wave (all lanes get
// the result).  Everything is double: the shift k of the first partial is a
// value of the channel, so the final cancellation S2 - S1^2/n loses at most a
// few of double's 53 bits.
__device__ __forceinline__ void channel_moments(const Geom& g, const Partial* __restrict__ part,
                                                uint32_t c, double& mean, double& var) {
    const uint32_t np = g.P * kWaves;
    const Partial* cp = part + static_cast<uint64_t>(c) * np;
    const double kref = cp[0].a;
    double s1 = 0.0, s2 = 0.0, n = 0.0;
    for (uint32_t q = lane_id(); q < np; q += kWave) {
        const Partial pq = cp[q];
        double t1 = pq.b, t2 = pq.c;
        reshift(t1, t2, pq.d, pq.a, kref);
        s1 += t1;
        s2 += t2;
        n += pq.d;
    }
    s1 = __shfl(wave_sum(s1), 0, kWave);
    s2 = __shfl(wave_sum(s2), 0, kWave);
    n = __shfl(wave_sum(n), 0, kWave);
    mean = kref + s1 / n;
    var = fmax(s2 - s1 * s1 / n, 0.0) / n;
}

__device__ __forceinline__ void channel_sums(const Geom& g, const Partial* __restrict__ part,
                                             uint32_t c, double& sdy, double& sdyx) {
    const uint32_t np = g.P * kWaves;
    const Partial* cp = part + static_cast<uint64_t>(c) * np;
    double a = 0.0, b = 0.0;
    for (uint32_t q = lane_id(); q < np; q += kWave) {
        a += cp[q].a;
        b += cp[q].b;
    }
    sdy = __shfl(wave_sum(a), 0, kWave);
    sdyx = __shfl(wave_sum(b), 0, kWave);
}

// ---------------------------------------------------------------- forward

// Shifted sums of one wave's share of a (channel, slice).
//
// Each thread accumulates S1 = sum(x - K), S2 = sum((x - K)^2) in fp32 with
// K = the first value it reads, which sits within a few standard deviations
// of the mean, so x - K carries the spread and not the offset (and is exact
// when x and K are within a factor of two).  The thread's sums are then
// re-expressed about lane 0's K in double and summed over the wave.
template <int DT, int VEC, int U>
__global__ __launch_bounds__(kThreads) void fwd_stats_kernel(const void* __restrict__ x, Geom g,
                                                             Partial* __restrict__ part) {
    const Slice s = block_slice(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    float shift = 0.f, s1 = 0.f, s2 = 0.f;
    bool first = true;
    uint32_t nacc = 0;
    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float t[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u)
            load_vec<DT, VEC, kHintStatsLoad>(x, access_index(g, cbase, v + u * kThreads), t[u]);
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
        load_vec<DT, VEC, kHintStatsLoad>(x, access_index(g, cbase, v), t);
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
    // Lane 0 has the smallest index of its wave, so if it read nothing the
    // whole wave read nothing and its sums are zero.
    const double kw = __shfl(shift, 0, kWave);
    const double n = static_cast<double>(nacc) * g.vec;
    double d1 = s1, d2 = s2;
    reshift(d1, d2, n, shift, kw);
    d1 = wave_sum(d1);
    d2 = wave_sum(d2);
    const double nw = wave_sum(n);
    if (lane_id() == 0) {
        Partial r;
        r.a = kw;
        r.b = d1;
        r.c = d2;
        r.d = nw;
        part[(static_cast<uint64_t>(s.c) * g.P + s.p) * kWaves + threadIdx.x / kWave] = r;
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
                                                             const Partial* __restrict__ part,
                                                             FwdParams prm) {
    const Slice s = block_slice<kReverseApply>(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    // First batch in flight before the per-channel coefficients are known.
    uint32_t v = s.lo + threadIdx.x;
    float t[U][VEC];
    uint64_t idx[U];
    bool full = v + (U - 1) * kThreads < s.hi;
    if (full) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            idx[u] = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC, kHintFwdApplyLoad>(xz, idx[u], t[u]);
        }
    }

    double mean, var;
    if constexpr (TRAIN) {
        channel_moments(g, part, s.c, mean, var);
    } else {
        mean = prm.running_mean[s.c];
        var = prm.running_var[s.c];
    }
    const float mean_hi = static_cast<float>(mean);
    const float mean_lo = static_cast<float>(mean - static_cast<double>(mean_hi));
    const float scale = static_cast<float>(static_cast<double>(prm.gamma[s.c]) /
                                           sqrt(var + static_cast<double>(prm.eps)));
    const float shift = prm.beta[s.c];
    const float slope = prm.slope;
    if constexpr (TRAIN) {
        if (s.p == 0 && threadIdx.x == 0) {
            const double mom = prm.momentum;
            const double m = g.m;
            prm.save_mean[s.c] = mean_hi;
            prm.save_var[s.c] = static_cast<float>(var);
            prm.running_mean[s.c] = static_cast<float>(
                (1.0 - mom) * static_cast<double>(prm.running_mean[s.c]) + mom * mean);
            prm.running_var[s.c] = static_cast<float>(
                (1.0 - mom) * static_cast<double>(prm.running_var[s.c]) + mom * var * (m / (m - 1.0)));
        }
    }

    auto act = [&](float xv) {
        const float y = fmaf((xv - mean_hi) - mean_lo, scale, shift);
        return y >= 0.f ? y : slope * y;
    };

    while (full) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) t[u][k] = act(t[u][k]);
            store_vec<DT, VEC, kHintFwdApplyStore>(xz, idx[u], t[u]);
        }
        v += U * kThreads;
        full = v + (U - 1) * kThreads < s.hi;
        if (full) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                idx[u] = access_index(g, cbase, v + u * kThreads);
                load_vec<DT, VEC, kHintFwdApplyLoad>(xz, idx[u], t[u]);
            }
        }
    }
    for (; v < s.hi; v += kThreads) {
        float r[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintFwdApplyLoad>(xz, i1, r);
#pragma unroll
        for (int k = 0; k < VEC; ++k) r[k] = act(r[k]);
        store_vec<DT, VEC, kHintFwdApplyStore>(xz, i1, r);
    }
}

// ---------------------------------------------------------------- backward

// Per-element terms of Algorithm 2 from the stored output z, with the
// per-channel constants folded in (exact in real arithmetic; formed in double
// once per block):
//   dy   = dz * f'(z)                   f' = 1 where z >= 0, slope where z < 0
//   xhat = (f^-1(z) - beta) / gamma     = z * (z < 0 ? 1/(slope gamma) : 1/gamma) - beta/gamma
// and, for the apply pass, with A = gamma/sqrt(var + eps), B = -A dgamma/m,
// C = -A dbeta/m,
//   dx   = A dy + B xhat + C
//        = (z < 0 ? A slope : A) dz + (z < 0 ? B/(slope gamma) : B/gamma) z + (C - B beta/gamma).
struct BwdReduceElem {
    float slope, k_pos, k_neg, nb;
    __device__ __forceinline__ void operator()(float z, float dz, float& dy, float& xhat) const {
        const bool neg = z < 0.f;
        dy = neg ? dz * slope : dz;
        xhat = fmaf(z, neg ? k_neg : k_pos, nb);
    }
};

__device__ __forceinline__ BwdReduceElem make_reduce_elem(float slope, float gamma, float beta) {
    const double g = gamma, a = slope;
    BwdReduceElem el;
    el.slope = slope;
    el.k_pos = static_cast<float>(1.0 / g);
    el.k_neg = static_cast<float>(1.0 / (a * g));
    el.nb = static_cast<float>(-static_cast<double>(beta) / g);
    return el;
}

struct BwdApplyElem {
    float a_pos, a_neg, b_pos, b_neg, c0;
    __device__ __forceinline__ float operator()(float z, float dz) const {
        const bool neg = z < 0.f;
        return fmaf(neg ? a_neg : a_pos, dz, fmaf(neg ? b_neg : b_pos, z, c0));
    }
};

__device__ __forceinline__ BwdApplyElem make_apply_elem(double A, double dgamma, double dbeta,
                                                        double m, float slope, float gamma,
                                                        float beta) {
    const double B = -A * dgamma / m, C = -A * dbeta / m;
    const double g = gamma, a = slope;
    BwdApplyElem el;
    el.a_pos = static_cast<float>(A);
    el.a_neg = static_cast<float>(A * a);
    el.b_pos = static_cast<float>(B / g);
    el.b_neg = static_cast<float>(B / (a * g));
    el.c0 = static_cast<float>(C - B * static_cast<double>(beta) / g);
    return el;
}

// Sums of dy and dy*xhat of one wave's share of a (channel, slice): fp32 per
// batch of U accesses, double across batches and lanes.
template <int DT, int VEC, int U>
__global__ __launch_bounds__(kThreads) void bwd_reduce_kernel(const void* __restrict__ z,
                                                              const void* __restrict__ dz, Geom g,
                                                              const float* __restrict__ gamma,
                                                              const float* __restrict__ beta,
                                                              float slope,
                                                              Partial* __restrict__ part) {
    const Slice s = block_slice(g);
    const BwdReduceElem el = make_reduce_elem(slope, gamma[s.c], beta[s.c]);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    double acc_dy = 0.0, acc_dyx = 0.0;
    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float tz[U][VEC], tg[U][VEC];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint64_t i1 = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC, kHintReduceLoad>(z, i1, tz[u]);
            load_vec<DT, VEC, kHintReduceLoad>(dz, i1, tg[u]);
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
        acc_dy += sdy;
        acc_dyx += sdyx;
    }
    for (; v < s.hi; v += kThreads) {
        float tz[VEC], tg[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintReduceLoad>(z, i1, tz);
        load_vec<DT, VEC, kHintReduceLoad>(dz, i1, tg);
        float sdy = 0.f, sdyx = 0.f;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float dy, xhat;
            el(tz[k], tg[k], dy, xhat);
            sdy += dy;
            sdyx = fmaf(dy, xhat, sdyx);
        }
        acc_dy += sdy;
        acc_dyx += sdyx;
    }
    acc_dy = wave_sum(acc_dy);
    acc_dyx = wave_sum(acc_dyx);
    if (lane_id() == 0) {
        Partial r;
        r.a = acc_dy;
        r.b = acc_dyx;
        r.c = 0.0;
        r.d = 0.0;
        part[(static_cast<uint64_t>(s.c) * g.P + s.p) * kWaves + threadIdx.x / kWave] = r;
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
                                                             const Partial* __restrict__ part,
                                                             BwdParams prm) {
    const Slice s = block_slice<kReverseApply>(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    uint32_t v = s.lo + threadIdx.x;
    float tz[U][VEC], tg[U][VEC];
    uint64_t idx[U];
    bool full = v + (U - 1) * kThreads < s.hi;
    if (full) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            idx[u] = access_index(g, cbase, v + u * kThreads);
            load_vec<DT, VEC, kHintBwdApplyLoad>(z, idx[u], tz[u]);
            load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, idx[u], tg[u]);
        }
    }

    double dbeta, dgamma;
    channel_sums(g, part, s.c, dbeta, dgamma);
    const double A = static_cast<double>(prm.gamma[s.c]) /
                     sqrt(static_cast<double>(prm.save_var[s.c]) + static_cast<double>(prm.eps));
    const BwdApplyElem dx_of =
        make_apply_elem(A, dgamma, dbeta, g.m, prm.slope, prm.gamma[s.c], prm.beta[s.c]);
    if (s.p == 0 && threadIdx.x == 0) {
        prm.dgamma[s.c] = static_cast<float>(dgamma);
        prm.dbeta[s.c] = static_cast<float>(dbeta);
    }

    while (full) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) tg[u][k] = dx_of(tz[u][k], tg[u][k]);
            store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, idx[u], tg[u]);
        }
        v += U * kThreads;
        full = v + (U - 1) * kThreads < s.hi;
        if (full) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                idx[u] = access_index(g, cbase, v + u * kThreads);
                load_vec<DT, VEC, kHintBwdApplyLoad>(z, idx[u], tz[u]);
                load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, idx[u], tg[u]);
            }
        }
    }
    for (; v < s.hi; v += kThreads) {
        float rz[VEC], rg[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintBwdApplyLoad>(z, i1, rz);
        load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, i1, rg);
#pragma unroll
        for (int k = 0; k < VEC; ++k) rg[k] = dx_of(rz[k], rg[k]);
        store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, i1, rg);
    }
}

// ---------------------------------------------------------------- fused, channel-resident

// One block owns a whole channel and keeps the first R of each thread's
// 16-byte accesses in registers between the reduction and the apply phase,
// so those bytes cross HBM once on the way in and once on the way out (the
// forward reads x and writes z; the backward reads z and dz and writes dx).
// Accesses beyond R (channels larger than the block's registers) are read
// again in the apply phase.  Thread t handles accesses t, t + T, t + 2T, ...
// of its channel, so a wave touches consecutive 16-byte vectors.  The only
// synchronisation is the block barrier around the channel's reduction.

typedef uint32_t raw16_t __attribute__((ext_vector_type(4)));

// Hide a value from the optimiser (an empty asm that "may change" it).  Used
// after the reduction barrier so that the apply phase keeps only the raw
// 16-byte registers alive and converts them again, instead of keeping the
// twice-as-large fp32 values (and 64-bit addresses) from the first phase.
template <typename V>
__device__ __forceinline__ void opaque(V& v) {
    asm volatile("" : "+v"(v));
}

// Keep the scheduler from interleaving the per-access steps of the register-
// resident loops: interleaving them only raises register pressure (the loads
// are already all in flight), and past the block's register budget it spills.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

template <int HINT>
__device__ __forceinline__ raw16_t load_raw(const void* __restrict__ base, uint64_t idx) {
    const raw16_t* p = static_cast<const raw16_t*>(base) + idx;
    return HINT == kStream ? __builtin_nontemporal_load(p) : *p;
}

template <int DT, int VEC>
__device__ __forceinline__ void unpack(raw16_t r, float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    typedef T vt __attribute__((ext_vector_type(VEC)));
    typedef float vf __attribute__((ext_vector_type(VEC)));
    const vf f = __builtin_convertvector(__builtin_bit_cast(vt, r), vf);
#pragma unroll
    for (int k = 0; k < VEC; ++k) v[k] = f[k];
}

// Per-wave (shift, s1, s2, n) of a block, combined by wave 0 in a fixed
// order into the channel's mean and biased variance.
template <int T>
__device__ __forceinline__ void block_moments(float shift, float s1, float s2, uint32_t nacc,
                                              uint32_t vec, double& mean, double& var) {
    constexpr int W = T / kWave;
    __shared__ double red[W][4];
    __shared__ double out[2];
    const double kw = __shfl(shift, 0, kWave);
    const double n = static_cast<double>(nacc) * vec;
    double d1 = s1, d2 = s2;
    reshift(d1, d2, n, shift, kw);
    d1 = wave_sum(d1);
    d2 = wave_sum(d2);
    const double nw = wave_sum(n);
    const uint32_t wave = threadIdx.x / kWave;
    if (lane_id() == 0) {
        red[wave][0] = kw;
        red[wave][1] = d1;
        red[wave][2] = d2;
        red[wave][3] = nw;
    }
    __syncthreads();
    if (wave == 0) {
        const double kref = red[0][0];
        double t1 = 0.0, t2 = 0.0, tn = 0.0;
        if (lane_id() < W) {
            t1 = red[lane_id()][1];
            t2 = red[lane_id()][2];
            tn = red[lane_id()][3];
            reshift(t1, t2, tn, red[lane_id()][0], kref);
        }
        t1 = wave_sum(t1);
        t2 = wave_sum(t2);
        tn = wave_sum(tn);
        if (lane_id() == 0) {
            out[0] = kref + t1 / tn;
            out[1] = fmax(t2 - t1 * t1 / tn, 0.0) / tn;
        }
    }
    __syncthreads();
    mean = out[0];
    var = out[1];
}

template <int T>
__device__ __forceinline__ void block_sums(double a, double b, double& sa, double& sb) {
    constexpr int W = T / kWave;
    __shared__ double red[W][2];
    __shared__ double out[2];
    a = wave_sum(a);
    b = wave_sum(b);
    const uint32_t wave = threadIdx.x / kWave;
    if (lane_id() == 0) {
        red[wave][0] = a;
        red[wave][1] = b;
    }
    __syncthreads();
    if (wave == 0) {
        double t1 = lane_id() < W ? red[lane_id()][0] : 0.0;
        double t2 = lane_id() < W ? red[lane_id()][1] : 0.0;
        t1 = wave_sum(t1);
        t2 = wave_sum(t2);
        if (lane_id() == 0) {
            out[0] = t1;
            out[1] = t2;
        }
    }
    __syncthreads();
    sa = out[0];
    sb = out[1];
}

// Where each row of a channel holds a whole number of T-wide strips of
// 16-byte accesses (vrow % T == 0) and the channel has at least R strips,
// access k of every thread of the block lies in strip k: its index is a
// block-uniform strip offset plus the thread index, and every thread has an
// access in each of the vchan / T strips.  The strip offsets are scalar
// (SGPR) arithmetic and the R resident accesses need no bounds test, so the
// per-element path spends no vector instructions on addresses or bounds.
// STRIP = false is the general mapping (row division per access, bounds per
// lane).
struct StripPos {
    uint64_t off;  // index of the strip's first access
    uint32_t col;  // column of the strip within its row
};

__device__ __forceinline__ StripPos strip_begin(const Geom& g, uint32_t c) {
    StripPos s;
    s.off = static_cast<uint64_t>(c) * g.vrow;
    s.col = 0;
    return s;
}

template <int T>
__device__ __forceinline__ void strip_next(const Geom& g, StripPos& s) {
    s.col += T;
    s.off += T;
    if (s.col == g.vrow) {
        s.col = 0;
        s.off += g.nstride - g.vrow;
    }
}

// The same for a block-uniform strip position (kept in scalar registers):
// the apply phase walks the strips again instead of keeping every strip
// offset of the reduction phase alive.
__device__ __forceinline__ void opaque_uniform(StripPos& s) {
    asm volatile("" : "+s"(s.off), "+s"(s.col));
}

// The leaky ReLU as max(y, a*y) for a <= 1 and min(y, a*y) for a > 1: two
// instructions, and the same value as the definition's branch (including
// y = -0, which stays -0).
template <bool SMALL_SLOPE>
__device__ __forceinline__ float leaky(float y, float a) {
    return SMALL_SLOPE ? fmaxf(y, a * y) : fminf(y, a * y);
}

// Apply phase of the fused forward: z = f((x - mean_hi) * scale + bshift) for
// the thread's resident accesses (from registers) and the remainder (loaded
// again), stored over x.
template <int DT, int VEC, int T, int R, bool STRIP, bool SMALL_SLOPE>
__device__ __forceinline__ void fwd_fused_apply(void* __restrict__ xz, const Geom& g, uint32_t c,
                                                uint32_t tid, const raw16_t (&keep)[R],
                                                float mean_hi, float scale, float bshift,
                                                float slope) {
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    StripPos sq = strip_begin(g, c);
    opaque_uniform(sq);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        uint64_t idx = 0;
        bool live = true;
        if constexpr (STRIP) {
            idx = sq.off + tid;
            strip_next<T>(g, sq);
        } else {
            const uint32_t v = tid + k * T;
            live = v < g.vchan;
            if (live) idx = access_index(g, cbase, v);
        }
        if (live) {
            float t[VEC];
            unpack<DT, VEC>(keep[k], t);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                t[e] = leaky<SMALL_SLOPE>(fmaf(t[e] - mean_hi, scale, bshift), slope);
            store_vec<DT, VEC, kHintFwdApplyStore>(xz, idx, t);
        }
        sched_fence();
    }
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            const uint64_t idx = sq.off + tid;
            float t[VEC];
            unpack<DT, VEC>(load_raw<kStream>(xz, idx), t);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                t[e] = leaky<SMALL_SLOPE>(fmaf(t[e] - mean_hi, scale, bshift), slope);
            store_vec<DT, VEC, kHintFwdApplyStore>(xz, idx, t);
            strip_next<T>(g, sq);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T) {
            const uint64_t idx = access_index(g, cbase, v);
            float t[VEC];
            unpack<DT, VEC>(load_raw<kStream>(xz, idx), t);
#pragma unroll
            for (int e = 0; e < VEC; ++e)
                t[e] = leaky<SMALL_SLOPE>(fmaf(t[e] - mean_hi, scale, bshift), slope);
            store_vec<DT, VEC, kHintFwdApplyStore>(xz, idx, t);
        }
    }
}

// Training forward of one channel per block (statistics, running estimates,
// z over x), same arithmetic as fwd_stats_kernel + fwd_apply_kernel.
template <int DT, int VEC, int T, int R, bool STRIP>
__device__ __forceinline__ void fwd_fused_channel(void* __restrict__ xz, const Geom& g,
                                                  const FwdParams& prm, uint32_t c) {
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t tid = threadIdx.x;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    raw16_t* const xv = static_cast<raw16_t*>(xz);
    // Per-channel inputs before the data loads (see bwd_fused_channel).
    const float gamma_c = prm.gamma[c], beta_c = prm.beta[c];
    float rm_c = 0.f, rv_c = 0.f;
    if (tid == 0) {
        rm_c = prm.running_mean[c];
        rv_c = prm.running_var[c];
    }

    // The first R accesses per thread stay in registers until the apply, so
    // this is their only read: non-temporal.  Accesses past those are read
    // again by the apply and go through the caches.  (Measured: non-temporal
    // register-resident loads cut the forward over the backbone sweep by 12%
    // and the backward by 7%.)
    raw16_t keep[R];
    StripPos sp = strip_begin(g, c);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if constexpr (STRIP) {
            keep[k] = load_raw<kStream>(xv, sp.off + tid);
            strip_next<T>(g, sp);
        } else {
            const uint32_t v = tid + k * T;
            if (v < g.vchan) keep[k] = load_raw<kStream>(xz, access_index(g, cbase, v));
        }
    }
    float shift = 0.f, s1 = 0.f, s2 = 0.f;
    uint32_t nacc = 0;
    if (tid < g.vchan) {
        float t[VEC];
        unpack<DT, VEC>(keep[0], t);
        shift = t[0];
    }
    auto accumulate = [&](raw16_t r) {
        float t[VEC];
        unpack<DT, VEC>(r, t);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            const float d = t[e] - shift;
            s1 += d;
            s2 = fmaf(d, d, s2);
        }
        ++nacc;
    };
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if (STRIP || tid + k * T < g.vchan) {
            float t[VEC];
            unpack<DT, VEC>(keep[k], t);
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                const float d = t[e] - shift;
                s1 += d;
                s2 = fmaf(d, d, s2);
            }
            ++nacc;
        }
        sched_fence();
    }
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            accumulate((xv + sp.off)[tid]);
            strip_next<T>(g, sp);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T)
            accumulate(load_raw<kCached>(xz, access_index(g, cbase, v)));
    }

    double mean, var;
    block_moments<T>(shift, s1, s2, nacc, VEC, mean, var);
    uint32_t tid2 = tid;
    opaque(tid2);
#pragma unroll
    for (int k = 0; k < R; ++k) opaque(keep[k]);
    const double scale_d = static_cast<double>(gamma_c) / sqrt(var + static_cast<double>(prm.eps));
    const float mean_hi = static_cast<float>(mean);
    const double mean_lo = mean - static_cast<double>(mean_hi);
    const float scale = static_cast<float>(scale_d);
    // (x - mu) * scale + beta with mu = mean_hi + mean_lo: the low part goes into the shift.
    const float bshift = static_cast<float>(static_cast<double>(beta_c) - mean_lo * scale_d);
    const float slope = prm.slope;
    if (tid == 0) {
        const double mom = prm.momentum;
        const double m = g.m;
        prm.save_mean[c] = mean_hi;
        prm.save_var[c] = static_cast<float>(var);
        prm.running_mean[c] = static_cast<float>((1.0 - mom) * static_cast<double>(rm_c) + mom * mean);
        prm.running_var[c] = static_cast<float>((1.0 - mom) * static_cast<double>(rv_c) +
                                                mom * var * (m / (m - 1.0)));
    }

    if (slope <= 1.f)
        fwd_fused_apply<DT, VEC, T, R, STRIP, true>(xz, g, c, tid2, keep, mean_hi, scale, bshift, slope);
    else
        fwd_fused_apply<DT, VEC, T, R, STRIP, false>(xz, g, c, tid2, keep, mean_hi, scale, bshift, slope);
}

// Backward of one channel per block (sums of dy and dy*xhat, dgamma, dbeta,
// dx over dz), same arithmetic as bwd_reduce_kernel + bwd_apply_kernel.
template <int DT, int VEC, int T, int R, bool STRIP>
__device__ __forceinline__ void bwd_fused_channel(const void* __restrict__ z,
                                                  void* __restrict__ dzdx, const Geom& g,
                                                  const BwdParams& prm, uint32_t c) {
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t tid = threadIdx.x;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    const raw16_t* const zv = static_cast<const raw16_t*>(z);
    const raw16_t* const gv = static_cast<const raw16_t*>(dzdx);
    // All per-channel inputs first: a load issued after the data loads would
    // put another memory round trip after the reduction barrier.
    const float gamma_c = prm.gamma[c], beta_c = prm.beta[c], var_c = prm.save_var[c];
    const BwdReduceElem el = make_reduce_elem(prm.slope, gamma_c, beta_c);

    // Register-resident accesses non-temporal, the rest cached (see
    // fwd_fused_channel).
    raw16_t kz[R], kg[R];
    StripPos sp = strip_begin(g, c);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if constexpr (STRIP) {
            kz[k] = load_raw<kStream>(zv, sp.off + tid);
            kg[k] = load_raw<kStream>(gv, sp.off + tid);
            strip_next<T>(g, sp);
        } else {
            const uint32_t v = tid + k * T;
            if (v < g.vchan) {
                const uint64_t i1 = access_index(g, cbase, v);
                kz[k] = load_raw<kStream>(z, i1);
                kg[k] = load_raw<kStream>(dzdx, i1);
            }
        }
    }
    // fp32 within one access, fp64 across accesses (as the streaming reduce
    // does per unrolled step): a channel's sums of dy cancel to near zero and
    // an fp32 running sum over the whole register-resident part loses that.
    double acc_dy = 0.0, acc_dyx = 0.0;
    float sdy = 0.f, sdyx = 0.f;
    auto accumulate = [&](raw16_t rz, raw16_t rg) {
        float tz[VEC], tg[VEC];
        unpack<DT, VEC>(rz, tz);
        unpack<DT, VEC>(rg, tg);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            float dy, xhat;
            el(tz[e], tg[e], dy, xhat);
            sdy += dy;
            sdyx = fmaf(dy, xhat, sdyx);
        }
    };
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if (STRIP || tid + k * T < g.vchan) {
            float tz[VEC], tg[VEC];
            unpack<DT, VEC>(kz[k], tz);
            unpack<DT, VEC>(kg[k], tg);
            sdy = 0.f;
            sdyx = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                float dy, xhat;
                el(tz[e], tg[e], dy, xhat);
                sdy += dy;
                sdyx = fmaf(dy, xhat, sdyx);
            }
            acc_dy += sdy;
            acc_dyx += sdyx;
        }
        sched_fence();
    }
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            sdy = 0.f;
            sdyx = 0.f;
            accumulate((zv + sp.off)[tid], (gv + sp.off)[tid]);
            acc_dy += sdy;
            acc_dyx += sdyx;
            strip_next<T>(g, sp);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T) {
            const uint64_t i1 = access_index(g, cbase, v);
            sdy = 0.f;
            sdyx = 0.f;
            accumulate(load_raw<kCached>(z, i1), load_raw<kCached>(dzdx, i1));
            acc_dy += sdy;
            acc_dyx += sdyx;
        }
    }

    double dbeta, dgamma;
    block_sums<T>(acc_dy, acc_dyx, dbeta, dgamma);
    uint32_t tid2 = tid;
    opaque(tid2);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        opaque(kz[k]);
        opaque(kg[k]);
    }
    const double A = static_cast<double>(gamma_c) /
                     sqrt(static_cast<double>(var_c) + static_cast<double>(prm.eps));
    const BwdApplyElem dx_of = make_apply_elem(A, dgamma, dbeta, g.m, prm.slope, gamma_c, beta_c);
    if (tid == 0) {
        prm.dgamma[c] = static_cast<float>(dgamma);
        prm.dbeta[c] = static_cast<float>(dbeta);
    }
    auto emit = [&](raw16_t rz, raw16_t rg, uint64_t idx) {
        float tz[VEC], tg[VEC];
        unpack<DT, VEC>(rz, tz);
        unpack<DT, VEC>(rg, tg);
#pragma unroll
        for (int e = 0; e < VEC; ++e) tg[e] = dx_of(tz[e], tg[e]);
        store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, idx, tg);
    };
    StripPos sq = strip_begin(g, c);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if constexpr (STRIP) {
            emit(kz[k], kg[k], sq.off + tid2);
            strip_next<T>(g, sq);
        } else {
            const uint32_t v = tid2 + k * T;
            if (v < g.vchan) {
                const uint64_t i1 = access_index(g, cbase, v);
                float tz[VEC], tg[VEC];
                unpack<DT, VEC>(kz[k], tz);
                unpack<DT, VEC>(kg[k], tg);
#pragma unroll
                for (int e = 0; e < VEC; ++e) tg[e] = dx_of(tz[e], tg[e]);
                store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, i1, tg);
            }
        }
        sched_fence();
    }
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            const uint64_t i1 = sq.off + tid2;
            emit(load_raw<kStream>(z, i1), load_raw<kStream>(dzdx, i1), i1);
            strip_next<T>(g, sq);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid2 + R * T; v < g.vchan; v += T) {
            const uint64_t i1 = access_index(g, cbase, v);
            emit(load_raw<kStream>(z, i1), load_raw<kStream>(dzdx, i1), i1);
        }
    }
}

// One block per channel: c = blockIdx.x.  (Giving each XCD a contiguous
// range of channels, rather than every eighth channel as the round-robin
// hand-out of workgroups to the 8 XCDs does, was measured 4% slower.  Blocks
// that loop over several
// channels were measured slower, both plainly and with the next channel
// prefetched into a second register buffer: the second buffer limits a CU to
// one block, and at that occupancy the per-channel reduce-barrier-apply chain
// costs more than the overlap of one channel's stores with the next one's
// loads gains.)
template <int DT, int VEC, int T, int R, bool STRIP>
__global__ __launch_bounds__(T) void fwd_fused_kernel(void* __restrict__ xz, Geom g,
                                                      FwdParams prm) {
    fwd_fused_channel<DT, VEC, T, R, STRIP>(xz, g, prm, blockIdx.x);
}

template <int DT, int VEC, int T, int R, bool STRIP>
__global__ __launch_bounds__(T) void bwd_fused_kernel(const void* __restrict__ z,
                                                      void* __restrict__ dzdx, Geom g,
                                                      BwdParams prm) {
    bwd_fused_channel<DT, VEC, T, R, STRIP>(z, dzdx, g, prm, blockIdx.x);
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
constexpr int64_t kTargetBlocks = 512;     // 2 blocks of 4 waves per CU on 256 CUs (measured best)
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
    return static_cast<size_t>(C) * static_cast<size_t>(sp.P) * kWaves * sizeof(Partial);
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

// Accesses in flight per thread and batch: 2 x 16 bytes on the vector path
// (measured best on the backbone sweep), 8 single elements on the scalar path.
template <int VEC>
constexpr int unroll() {
    return VEC == 1 ? 8 : 2;
}

template <int DT, int VEC>
struct LaunchFwdStats {
    static void run(const void* x, const Geom& g, Partial* part, hipStream_t st) {
        fwd_stats_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(x, g, part);
    }
};

template <int DT, int VEC>
struct LaunchFwdApply {
    static void run(void* xz, const Geom& g, const Partial* part, const FwdParams& prm, bool train,
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
                    const float* beta, float slope, Partial* part, hipStream_t st) {
        bwd_reduce_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(
            z, dz, g, gamma, beta, slope, part);
    }
};

template <int DT, int VEC>
struct LaunchBwdApply {
    static void run(const void* z, void* dzdx, const Geom& g, const Partial* part,
                    const BwdParams& prm, hipStream_t st) {
        bwd_apply_kernel<DT, VEC, unroll<VEC>()><<<grid_of(g), kThreads, 0, st>>>(z, dzdx, g,
                                                                                   part, prm);
    }
};

// ---- fused (channel-resident) path

// Used when every channel gets a block of its own and at least one block per
// CU (C >= kFusedMinChannels) on the 16-byte path.
constexpr int64_t kFusedMinChannels = 256;

struct FusedPlan {
    int T;  // threads per block
    int R;  // 16-byte accesses per thread held in registers (per tensor)
};

dim3 fused_grid(const Geom& g, const FusedPlan&) { return dim3(g.C); }

// Resident blocks per CU of a fused launch (0: as many as registers allow).
// Fewer resident blocks run the channels in several rounds, so the loads of
// a later round overlap the stores of an earlier one instead of every block
// reading, then every block writing.  The cap is applied by reserving LDS.
constexpr int kFusedFwdBlocksPerCU = 0;
constexpr int kFusedBwdBlocksPerCU = 0;
constexpr size_t kLdsPerCU = 160 * 1024;

size_t fused_lds(int blocks_per_cu) {
    if (blocks_per_cu <= 0) return 0;
    return kLdsPerCU / blocks_per_cu - 2048;  // leaves room for the kernels' own reduction buffers
}

// Candidate (T, R) in order of preference (each one has a kernel built in
// launch_fwd_fused / launch_bwd_fused): the first whose threads hold the
// whole channel is used; larger channels take the last entry and re-read
// the remainder.  The backward holds two tensors, so its largest blocks keep
// half as many accesses per thread.
// Fused kernels use strip addressing where the shape allows it.
constexpr bool kUseStrips = true;

constexpr FusedPlan kFwdLadder[] = {{256, 4}, {512, 4}, {256, 16}, {512, 16}, {1024, 16}};
constexpr FusedPlan kBwdLadder[] = {{256, 4}, {512, 4}, {256, 16}, {512, 16}, {1024, 8}};

bool plan_fused(int64_t C, const Geom& g, bool vector, bool backward, FusedPlan* out) {
    if (!vector || C < kFusedMinChannels) return false;
    const int64_t A = g.vchan;
    const FusedPlan* ladder = backward ? kBwdLadder : kFwdLadder;
    const int n = backward ? int(sizeof kBwdLadder / sizeof kBwdLadder[0])
                           : int(sizeof kFwdLadder / sizeof kFwdLadder[0]);
    for (int i = 0; i < n; ++i) {
        if (A <= static_cast<int64_t>(ladder[i].T) * ladder[i].R || i == n - 1) {
            *out = ladder[i];
            return true;
        }
    }
    return false;
}

#define IABN_FUSED_CASE(KERNEL, TT, RR, ...)                                                   \
    if (fp.T == TT && fp.R == RR) {                                                           \
        if (kUseStrips && g.vrow % TT == 0 && g.vchan / TT >= RR)                             \
            KERNEL<DT, V, TT, RR, true><<<grid, TT, lds, st>>>(__VA_ARGS__);                  \
        else                                                                                  \
            KERNEL<DT, V, TT, RR, false><<<grid, TT, lds, st>>>(__VA_ARGS__);                 \
        return true;                                                                          \
    }

template <int DT>
bool launch_fwd_fused(void* xz, const Geom& g, const FusedPlan& fp, const FwdParams& prm,
                      hipStream_t st) {
    constexpr int V = 16 / sizeof(typename Elem<DT>::T);
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedFwdBlocksPerCU);
    IABN_FUSED_CASE(fwd_fused_kernel, 256, 4, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, 512, 4, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, 256, 16, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, 512, 16, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, 1024, 16, xz, g, prm)
    return false;
}

template <int DT>
bool launch_bwd_fused(const void* z, void* dzdx, const Geom& g, const FusedPlan& fp,
                      const BwdParams& prm, hipStream_t st) {
    constexpr int V = 16 / sizeof(typename Elem<DT>::T);
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedBwdBlocksPerCU);
    IABN_FUSED_CASE(bwd_fused_kernel, 256, 4, z, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, 512, 4, z, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, 256, 16, z, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, 512, 16, z, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, 1024, 8, z, dzdx, g, prm)
    return false;
}

#undef IABN_FUSED_CASE

// ---- end fused planning

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
    dispatch<LaunchFwdStats>(dtype, vec, x, g, static_cast<Partial*>(workspace),
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
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const Partial*>(workspace), prm, true,
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
    const bool vec = use_vector(HW, dtype, x_z, nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    FusedPlan fp;
    if (plan_fused(C, g, vec, false, &fp)) {
        const FwdParams prm = {gamma, beta, running_mean, running_var, save_mean, save_var,
                               eps,   momentum, slope};
        const hipStream_t st = static_cast<hipStream_t>(stream);
        const bool ok = dtype == IABN_F32   ? launch_fwd_fused<IABN_F32>(x_z, g, fp, prm, st)
                        : dtype == IABN_F16 ? launch_fwd_fused<IABN_F16>(x_z, g, fp, prm, st)
                                            : launch_fwd_fused<IABN_BF16>(x_z, g, fp, prm, st);
        if (!ok) return fail(IABN_ERR_HIP, "no forward kernel built for T=%d R=%d", fp.T, fp.R);
        return launched("fwd_fused");
    }
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
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const Partial*>(nullptr), prm, false,
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
    const bool vec = use_vector(HW, dtype, z, dz_dx);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, save_var, dgamma, dbeta, eps, slope};
    dispatch<LaunchBwdApply>(dtype, vec, z, dz_dx, g, static_cast<const Partial*>(workspace), prm,
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
    const bool vec = use_vector(HW, dtype, z, dz_dx);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    FusedPlan fp;
    if (plan_fused(C, g, vec, true, &fp)) {
        const BwdParams prm = {gamma, beta, save_var, dgamma, dbeta, eps, slope};
        const hipStream_t st = static_cast<hipStream_t>(stream);
        const bool ok = dtype == IABN_F32   ? launch_bwd_fused<IABN_F32>(z, dz_dx, g, fp, prm, st)
                        : dtype == IABN_F16 ? launch_bwd_fused<IABN_F16>(z, dz_dx, g, fp, prm, st)
                                            : launch_bwd_fused<IABN_BF16>(z, dz_dx, g, fp, prm, st);
        if (!ok) return fail(IABN_ERR_HIP, "no backward kernel built for T=%d R=%d", fp.T, fp.R);
        return launched("bwd_fused");
    }
    if ((rc = iabn_backward_reduce(z, dz_dx, dtype, gamma, beta, slope, N, C, HW, workspace,
                                   workspace_bytes, stream)))
        return rc;
    return iabn_backward_apply(z, dz_dx, dtype, gamma, beta, save_var, dgamma, dbeta, eps, slope,
                               N, C, HW, workspace, workspace_bytes, stream);
}

}  // extern "C"
