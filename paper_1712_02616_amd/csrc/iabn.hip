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
    void* out;  // z for kFwdOut and kFwdCkpt
    float eps, momentum, slope;
};

// Forward outputs.  kFwdInPlace: z over x (InPlace-ABN, Fig. 2(d)).
// kFwdOut: z to a separate buffer, x kept (the standard block, Fig. 2(a)).
// kFwdCkpt: xhat over x and z to a separate buffer (the proposed
// checkpointing, Fig. 2(c)); z is formed from xhat as stored, so the
// backward's recomputation of z from the stored xhat reproduces it exactly.
constexpr int kFwdInPlace = 0;
constexpr int kFwdOut = 1;
constexpr int kFwdCkpt = 2;

// A value rounded to the storage type and widened back.
template <int DT>
__device__ __forceinline__ float storage_round(float v) {
    return static_cast<float>(static_cast<typename Elem<DT>::T>(v));
}

// z = f(gamma * (x - mu) / sqrt(var + eps) + beta).  TRAIN: mu and var are
// the batch statistics combined from the partials (slice 0 of each channel
// also writes them out and updates the running estimates); otherwise they
// are the running estimates (inference, in place only).  mu is applied as a
// two-float sum hi + lo, so x - mu keeps fp32 relative accuracy even when
// |mu| >> sigma.
template <int DT, int VEC, int U, bool TRAIN, int FM>
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
        for (int q = 0; q < U; ++q) {
            idx[q] = access_index(g, cbase, v + q * kThreads);
            load_vec<DT, VEC, kHintFwdApplyLoad>(xz, idx[q], t[q]);
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
    const double invstd = 1.0 / sqrt(var + static_cast<double>(prm.eps));
    const float gamma = prm.gamma[s.c], beta = prm.beta[s.c];
    // kFwdCkpt normalises first (scale 1/sigma, shift beta applied after the
    // rounding of xhat); the others fold gamma into the scale.
    const float scale = static_cast<float>(FM == kFwdCkpt ? invstd : gamma * invstd);
    const float shift = FM == kFwdCkpt ? 0.f : beta;
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

    auto act = [&](float y) { return y >= 0.f ? y : slope * y; };
    // Writes the outputs of access i1 from its inputs r (overwritten).
    auto emit = [&](float (&r)[VEC], uint64_t i1) {
        if constexpr (FM == kFwdCkpt) {
            float zv[VEC];
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                r[k] = storage_round<DT>(fmaf((r[k] - mean_hi) - mean_lo, scale, shift));
                zv[k] = act(fmaf(r[k], gamma, beta));
            }
            store_vec<DT, VEC, kHintFwdApplyStore>(xz, i1, r);
            store_vec<DT, VEC, kHintFwdApplyStore>(prm.out, i1, zv);
        } else {
#pragma unroll
            for (int k = 0; k < VEC; ++k) r[k] = act(fmaf((r[k] - mean_hi) - mean_lo, scale, shift));
            store_vec<DT, VEC, kHintFwdApplyStore>(FM == kFwdOut ? prm.out : xz, i1, r);
        }
    };

    while (full) {
#pragma unroll
        for (int q = 0; q < U; ++q) emit(t[q], idx[q]);
        v += U * kThreads;
        full = v + (U - 1) * kThreads < s.hi;
        if (full) {
#pragma unroll
            for (int q = 0; q < U; ++q) {
                idx[q] = access_index(g, cbase, v + q * kThreads);
                load_vec<DT, VEC, kHintFwdApplyLoad>(xz, idx[q], t[q]);
            }
        }
    }
    for (; v < s.hi; v += kThreads) {
        float r[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintFwdApplyLoad>(xz, i1, r);
        emit(r, i1);
    }
}

// z = f(gamma * xhat + beta) from a stored xhat, out of place: the
// recomputation step of the proposed checkpointing (Fig. 2(c)).
template <int DT, int VEC>
__global__ __launch_bounds__(kThreads) void recompute_kernel(const void* __restrict__ xhat,
                                                             void* __restrict__ z, Geom g,
                                                             const float* __restrict__ gamma,
                                                             const float* __restrict__ beta,
                                                             float slope) {
    const Slice s = block_slice(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    const float gm = gamma[s.c], bt = beta[s.c];
    for (uint32_t v = s.lo + threadIdx.x; v < s.hi; v += kThreads) {
        float r[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kStream>(xhat, i1, r);
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            const float y = fmaf(r[k], gm, bt);
            r[k] = y >= 0.f ? y : slope * y;
        }
        store_vec<DT, VEC, kStream>(z, i1, r);
    }
}

// ---------------------------------------------------------------- backward

// Backward formulations.  Each reads a stored tensor u (plus dz) and
// recovers, per element, dy = dz * f'(y) and a weight w whose sum against dy
// gives dgamma:
//   kBwdFromZ     u = z (InPlace-ABN, Sec. 3.3, Algorithm 2).  f' from the
//                 sign of z.  Formulation I: w = xhat = (f^-1(z) - beta)/gamma.
//                 Formulation II (BN-dagger, the Appendix): w = y = f^-1(z),
//                 dgamma = (sum dy*y - beta sum dy)/gamma per channel.
//   kBwdFromXZ    u = x, plus the stored z for f' (the standard block of
//                 Fig. 2(a), which keeps x and z): w = xhat = (x - mu)/sigma.
//   kBwdFromXhat  u = xhat (the proposed checkpointing of Fig. 2(c)):
//                 f' from the sign of y = gamma*xhat + beta, w = xhat.
// With the per-channel constants folded in (exact in real arithmetic, formed
// in double once per block) every formulation is
//   w  = (u - off) * (neg ? k_neg : k_pos) + nb
//   dx = A dy + B xhat + C        (A = gamma/sqrt(var + eps), B = -A dgamma/m, C = -A dbeta/m)
//      = (neg ? a_neg : a_pos) dz + (neg ? b_neg : b_pos) (u - off) + c0
// e.g. for formulation I: k_pos = 1/gamma, k_neg = 1/(slope gamma),
// nb = -beta/gamma, b_pos = B/gamma, b_neg = B/(slope gamma),
// c0 = C - B beta/gamma.
constexpr int kBwdFromZ = 0;
constexpr int kBwdFromXZ = 1;
constexpr int kBwdFromXhat = 2;

// The sign test of f'(y): y < 0.  kBwdFromZ and kBwdFromXZ test the stored z
// (f preserves the sign and -0 stays on the identity side); kBwdFromXhat
// forms y = fma(xhat, gamma, beta), whose single rounding keeps the sign of
// the exact gamma*xhat + beta.
template <int BM>
struct BwdSign {
    float gamma, beta;
    __device__ __forceinline__ bool operator()(float u, float zv) const {
        if constexpr (BM == kBwdFromZ) return u < 0.f;
        else if constexpr (BM == kBwdFromXZ) return zv < 0.f;
        else return fmaf(u, gamma, beta) < 0.f;
    }
};

template <int BM>
struct BwdReduceElem {
    BwdSign<BM> sign;
    float slope, k_pos, k_neg, nb, off;
    __device__ __forceinline__ void with_neg(bool neg, float u, float dz, float& dy,
                                             float& w) const {
        dy = neg ? dz * slope : dz;
        if constexpr (BM == kBwdFromZ) w = fmaf(u, neg ? k_neg : k_pos, nb);
        else if constexpr (BM == kBwdFromXZ) w = fmaf(u - off, k_pos, nb);
        else w = u;
    }
    __device__ __forceinline__ void operator()(float u, float zv, float dz, float& dy,
                                               float& w) const {
        with_neg(sign(u, zv), u, dz, dy, w);
    }
};

// Per-channel constants of the reduction.  ii selects formulation II
// (w = y instead of xhat) for kBwdFromZ.
template <int BM>
__device__ __forceinline__ BwdReduceElem<BM> make_reduce_elem(float slope, float gamma, float beta,
                                                              float mean, double invstd, bool ii) {
    const double g = gamma, a = slope;
    BwdReduceElem<BM> el;
    el.sign.gamma = gamma;
    el.sign.beta = beta;
    el.slope = slope;
    el.k_pos = el.k_neg = 1.f;
    el.nb = 0.f;
    el.off = 0.f;
    if constexpr (BM == kBwdFromZ) {
        if (ii) {
            el.k_neg = static_cast<float>(1.0 / a);
        } else {
            el.k_pos = static_cast<float>(1.0 / g);
            el.k_neg = static_cast<float>(1.0 / (a * g));
            el.nb = static_cast<float>(-static_cast<double>(beta) / g);
        }
    } else if constexpr (BM == kBwdFromXZ) {
        el.off = mean;
        el.k_pos = el.k_neg = static_cast<float>(invstd);
    }
    return el;
}

template <int BM>
struct BwdApplyElem {
    BwdSign<BM> sign;
    float a_pos, a_neg, b_pos, b_neg, c0, off;
    __device__ __forceinline__ float operator()(float u, float zv, float dz) const {
        return with_neg(sign(u, zv), u, dz);
    }
    __device__ __forceinline__ float with_neg(bool neg, float u, float dz) const {
        if constexpr (BM == kBwdFromZ)
            return fmaf(neg ? a_neg : a_pos, dz, fmaf(neg ? b_neg : b_pos, u, c0));
        else if constexpr (BM == kBwdFromXZ)
            return fmaf(neg ? a_neg : a_pos, dz, fmaf(b_pos, u - off, c0));
        else
            return fmaf(neg ? a_neg : a_pos, dz, fmaf(b_pos, u, c0));
    }
};

// dgamma from the two sums (formulation II converts sum dy*y), then the
// apply constants.  sdyw is overwritten with dgamma.
template <int BM>
__device__ __forceinline__ BwdApplyElem<BM> make_apply_elem(double A, double& sdyw, double dbeta,
                                                            double m, float slope, float gamma,
                                                            float beta, float mean, double invstd,
                                                            bool ii) {
    const double g = gamma, a = slope, bt = beta;
    if (BM == kBwdFromZ && ii) sdyw = (sdyw - bt * dbeta) / g;
    const double dgamma = sdyw;
    const double B = -A * dgamma / m, C = -A * dbeta / m;
    BwdApplyElem<BM> el;
    el.sign.gamma = gamma;
    el.sign.beta = beta;
    el.a_pos = static_cast<float>(A);
    el.a_neg = static_cast<float>(A * a);
    el.off = 0.f;
    if constexpr (BM == kBwdFromZ) {
        el.b_pos = static_cast<float>(B / g);
        el.b_neg = static_cast<float>(B / (a * g));
        el.c0 = static_cast<float>(C - B * bt / g);
    } else if constexpr (BM == kBwdFromXZ) {
        el.off = mean;
        el.b_pos = el.b_neg = static_cast<float>(B * invstd);
        el.c0 = static_cast<float>(C);
    } else {
        el.b_pos = el.b_neg = static_cast<float>(B);
        el.c0 = static_cast<float>(C);
    }
    return el;
}

struct BwdParams {
    const float* gamma;
    const float* beta;
    const float* save_mean;  // kBwdFromXZ only
    const float* save_var;
    float* dgamma;
    float* dbeta;
    float eps, slope;
    int ii;  // formulation II (kBwdFromZ only)
};

__device__ __forceinline__ double chan_invstd(const BwdParams& prm, uint32_t c) {
    return 1.0 / sqrt(static_cast<double>(prm.save_var[c]) + static_cast<double>(prm.eps));
}

// Loads the z of access i1 for the sign test of kBwdFromXZ (nothing otherwise).
template <int DT, int VEC, int HINT, int BM>
__device__ __forceinline__ void load_sign(const void* __restrict__ zs, uint64_t i1,
                                          float (&v)[VEC]) {
    if constexpr (BM == kBwdFromXZ) {
        load_vec<DT, VEC, HINT>(zs, i1, v);
    } else {
#pragma unroll
        for (int k = 0; k < VEC; ++k) v[k] = 0.f;
    }
}

// Sums of dy and dy*w of one wave's share of a (channel, slice): fp32 per
// batch of U accesses, double across batches and lanes.  u is z, x or xhat
// (see BwdSign); zs is the stored z for kBwdFromXZ.
template <int DT, int VEC, int U, int BM>
__global__ __launch_bounds__(kThreads) void bwd_reduce_kernel(const void* __restrict__ u,
                                                              const void* __restrict__ zs,
                                                              const void* __restrict__ dz, Geom g,
                                                              BwdParams prm,
                                                              Partial* __restrict__ part) {
    const Slice s = block_slice(g);
    const double invstd = BM == kBwdFromXZ ? chan_invstd(prm, s.c) : 1.0;
    const BwdReduceElem<BM> el =
        make_reduce_elem<BM>(prm.slope, prm.gamma[s.c], prm.beta[s.c],
                             BM == kBwdFromXZ ? prm.save_mean[s.c] : 0.f, invstd, prm.ii != 0);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;
    double acc_dy = 0.0, acc_dyw = 0.0;
    uint32_t v = s.lo + threadIdx.x;
    for (; v + (U - 1) * kThreads < s.hi; v += U * kThreads) {
        float tu[U][VEC], tz[U][VEC], tg[U][VEC];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const uint64_t i1 = access_index(g, cbase, v + q * kThreads);
            load_vec<DT, VEC, kHintReduceLoad>(u, i1, tu[q]);
            load_sign<DT, VEC, kHintReduceLoad, BM>(zs, i1, tz[q]);
            load_vec<DT, VEC, kHintReduceLoad>(dz, i1, tg[q]);
        }
        float sdy = 0.f, sdyw = 0.f;
#pragma unroll
        for (int q = 0; q < U; ++q) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) {
                float dy, w;
                el(tu[q][k], tz[q][k], tg[q][k], dy, w);
                sdy += dy;
                sdyw = fmaf(dy, w, sdyw);
            }
        }
        acc_dy += sdy;
        acc_dyw += sdyw;
    }
    for (; v < s.hi; v += kThreads) {
        float tu[VEC], tz[VEC], tg[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintReduceLoad>(u, i1, tu);
        load_sign<DT, VEC, kHintReduceLoad, BM>(zs, i1, tz);
        load_vec<DT, VEC, kHintReduceLoad>(dz, i1, tg);
        float sdy = 0.f, sdyw = 0.f;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
            float dy, w;
            el(tu[k], tz[k], tg[k], dy, w);
            sdy += dy;
            sdyw = fmaf(dy, w, sdyw);
        }
        acc_dy += sdy;
        acc_dyw += sdyw;
    }
    acc_dy = wave_sum(acc_dy);
    acc_dyw = wave_sum(acc_dyw);
    if (lane_id() == 0) {
        Partial r;
        r.a = acc_dy;
        r.b = acc_dyw;
        r.c = 0.0;
        r.d = 0.0;
        part[(static_cast<uint64_t>(s.c) * g.P + s.p) * kWaves + threadIdx.x / kWave] = r;
    }
}

// dx = (dy - dgamma*xhat/m - dbeta/m) * gamma/sqrt(var + eps), in place over dz,
// with the per-channel constants of make_apply_elem.
template <int DT, int VEC, int U, int BM>
__global__ __launch_bounds__(kThreads) void bwd_apply_kernel(const void* __restrict__ u,
                                                             const void* __restrict__ zs,
                                                             void* __restrict__ dzdx, Geom g,
                                                             const Partial* __restrict__ part,
                                                             BwdParams prm) {
    const Slice s = block_slice<kReverseApply>(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    uint32_t v = s.lo + threadIdx.x;
    float tu[U][VEC], tz[U][VEC], tg[U][VEC];
    uint64_t idx[U];
    bool full = v + (U - 1) * kThreads < s.hi;
    if (full) {
#pragma unroll
        for (int q = 0; q < U; ++q) {
            idx[q] = access_index(g, cbase, v + q * kThreads);
            load_vec<DT, VEC, kHintBwdApplyLoad>(u, idx[q], tu[q]);
            load_sign<DT, VEC, kHintBwdApplyLoad, BM>(zs, idx[q], tz[q]);
            load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, idx[q], tg[q]);
        }
    }

    double dbeta, dgamma;
    channel_sums(g, part, s.c, dbeta, dgamma);
    const double invstd = chan_invstd(prm, s.c);
    const double A = static_cast<double>(prm.gamma[s.c]) * invstd;
    const BwdApplyElem<BM> dx_of = make_apply_elem<BM>(
        A, dgamma, dbeta, g.m, prm.slope, prm.gamma[s.c], prm.beta[s.c],
        BM == kBwdFromXZ ? prm.save_mean[s.c] : 0.f, invstd, prm.ii != 0);
    if (s.p == 0 && threadIdx.x == 0) {
        prm.dgamma[s.c] = static_cast<float>(dgamma);
        prm.dbeta[s.c] = static_cast<float>(dbeta);
    }

    while (full) {
#pragma unroll
        for (int q = 0; q < U; ++q) {
#pragma unroll
            for (int k = 0; k < VEC; ++k) tg[q][k] = dx_of(tu[q][k], tz[q][k], tg[q][k]);
            store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, idx[q], tg[q]);
        }
        v += U * kThreads;
        full = v + (U - 1) * kThreads < s.hi;
        if (full) {
#pragma unroll
            for (int q = 0; q < U; ++q) {
                idx[q] = access_index(g, cbase, v + q * kThreads);
                load_vec<DT, VEC, kHintBwdApplyLoad>(u, idx[q], tu[q]);
                load_sign<DT, VEC, kHintBwdApplyLoad, BM>(zs, idx[q], tz[q]);
                load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, idx[q], tg[q]);
            }
        }
    }
    for (; v < s.hi; v += kThreads) {
        float ru[VEC], rz[VEC], rg[VEC];
        const uint64_t i1 = access_index(g, cbase, v);
        load_vec<DT, VEC, kHintBwdApplyLoad>(u, i1, ru);
        load_sign<DT, VEC, kHintBwdApplyLoad, BM>(zs, i1, rz);
        load_vec<DT, VEC, kHintBwdApplyLoad>(dzdx, i1, rg);
#pragma unroll
        for (int k = 0; k < VEC; ++k) rg[k] = dx_of(ru[k], rz[k], rg[k]);
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

// Per-channel constants of the fused forward's apply phase.
struct FwdApplyK {
    float mean_hi, scale, bshift, slope;  // y = (x - mean_hi) * scale + bshift (kFwdCkpt: xhat)
    float gamma, beta;                    // kFwdCkpt: y = gamma * xhat + beta
    void* out;                            // kFwdOut / kFwdCkpt: z
};

// The outputs of one 16-byte access from its input values t (overwritten).
template <int DT, int VEC, int FM, bool SMALL_SLOPE>
__device__ __forceinline__ void fwd_fused_emit(void* __restrict__ xz, uint64_t idx,
                                               float (&t)[VEC], const FwdApplyK& k) {
    if constexpr (FM == kFwdCkpt) {
        float zv[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            t[e] = storage_round<DT>(fmaf(t[e] - k.mean_hi, k.scale, k.bshift));
            zv[e] = leaky<SMALL_SLOPE>(fmaf(t[e], k.gamma, k.beta), k.slope);
        }
        store_vec<DT, VEC, kHintFwdApplyStore>(xz, idx, t);
        store_vec<DT, VEC, kHintFwdApplyStore>(k.out, idx, zv);
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e)
            t[e] = leaky<SMALL_SLOPE>(fmaf(t[e] - k.mean_hi, k.scale, k.bshift), k.slope);
        store_vec<DT, VEC, kHintFwdApplyStore>(FM == kFwdOut ? k.out : xz, idx, t);
    }
}

// Apply phase of the fused forward for the thread's resident accesses (from
// registers) and the remainder (loaded again).
template <int DT, int VEC, int T, int R, bool STRIP, int FM, bool SMALL_SLOPE>
__device__ __forceinline__ void fwd_fused_apply(void* __restrict__ xz, const Geom& g, uint32_t c,
                                                uint32_t tid, const raw16_t (&keep)[R],
                                                const FwdApplyK& kk) {
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
            fwd_fused_emit<DT, VEC, FM, SMALL_SLOPE>(xz, idx, t, kk);
        }
        sched_fence();
    }
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            const uint64_t idx = sq.off + tid;
            float t[VEC];
            unpack<DT, VEC>(load_raw<kStream>(xz, idx), t);
            fwd_fused_emit<DT, VEC, FM, SMALL_SLOPE>(xz, idx, t, kk);
            strip_next<T>(g, sq);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T) {
            const uint64_t idx = access_index(g, cbase, v);
            float t[VEC];
            unpack<DT, VEC>(load_raw<kStream>(xz, idx), t);
            fwd_fused_emit<DT, VEC, FM, SMALL_SLOPE>(xz, idx, t, kk);
        }
    }
}

// Training forward of one channel per block (statistics, running estimates,
// z over x), same arithmetic as fwd_stats_kernel + fwd_apply_kernel.
template <int DT, int VEC, int T, int R, bool STRIP, int FM>
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
    const double invstd = 1.0 / sqrt(var + static_cast<double>(prm.eps));
    const double scale_d = FM == kFwdCkpt ? invstd : static_cast<double>(gamma_c) * invstd;
    const float mean_hi = static_cast<float>(mean);
    const double mean_lo = mean - static_cast<double>(mean_hi);
    // (x - mu) * scale + beta with mu = mean_hi + mean_lo: the low part goes
    // into the shift (kFwdCkpt: beta comes after the rounding of xhat).
    FwdApplyK kk;
    kk.mean_hi = mean_hi;
    kk.scale = static_cast<float>(scale_d);
    kk.bshift = static_cast<float>((FM == kFwdCkpt ? 0.0 : static_cast<double>(beta_c)) -
                                   mean_lo * scale_d);
    kk.slope = prm.slope;
    kk.gamma = gamma_c;
    kk.beta = beta_c;
    kk.out = prm.out;
    if (tid == 0) {
        const double mom = prm.momentum;
        const double m = g.m;
        prm.save_mean[c] = mean_hi;
        prm.save_var[c] = static_cast<float>(var);
        prm.running_mean[c] = static_cast<float>((1.0 - mom) * static_cast<double>(rm_c) + mom * mean);
        prm.running_var[c] = static_cast<float>((1.0 - mom) * static_cast<double>(rv_c) +
                                                mom * var * (m / (m - 1.0)));
    }

    if (kk.slope <= 1.f)
        fwd_fused_apply<DT, VEC, T, R, STRIP, FM, true>(xz, g, c, tid2, keep, kk);
    else
        fwd_fused_apply<DT, VEC, T, R, STRIP, FM, false>(xz, g, c, tid2, keep, kk);
}

// Backward of one channel per block (sums of dy and dy*w, dgamma, dbeta, dx
// over dz), same arithmetic as bwd_reduce_kernel + bwd_apply_kernel.  u is z,
// x or xhat (see BwdSign).  kBwdFromXZ reads the stored z as well but keeps
// only its signs (one bit per element) for the apply phase.
template <int DT, int VEC, int T, int R, bool STRIP, int BM>
__device__ __forceinline__ void bwd_fused_channel(const void* __restrict__ u,
                                                  const void* __restrict__ zs,
                                                  void* __restrict__ dzdx, const Geom& g,
                                                  const BwdParams& prm, uint32_t c) {
    constexpr bool XZ = BM == kBwdFromXZ;
    constexpr int NW = XZ ? (R * VEC + 31) / 32 : 1;
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t tid = threadIdx.x;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    const raw16_t* const uv = static_cast<const raw16_t*>(u);
    const raw16_t* const zsv = static_cast<const raw16_t*>(zs);
    const raw16_t* const gv = static_cast<const raw16_t*>(dzdx);
    // All per-channel inputs first: a load issued after the data loads would
    // put another memory round trip after the reduction barrier.
    const float gamma_c = prm.gamma[c], beta_c = prm.beta[c], var_c = prm.save_var[c];
    const float mean_c = XZ ? prm.save_mean[c] : 0.f;
    const double invstd =
        1.0 / sqrt(static_cast<double>(var_c) + static_cast<double>(prm.eps));
    const BwdReduceElem<BM> el =
        make_reduce_elem<BM>(prm.slope, gamma_c, beta_c, mean_c, invstd, prm.ii != 0);

    // Register-resident accesses non-temporal, the rest cached (see
    // fwd_fused_channel).  kBwdFromXZ first loads z (into the registers x
    // will use) and dz, turns z into sign bits, and only then loads x, so
    // that no more than two tensors' worth of registers is live.
    raw16_t ku[R], kg[R];
    uint32_t negm[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) negm[q] = 0u;
    auto resident_index = [&](int k, StripPos& p, bool& live) -> uint64_t {
        if constexpr (STRIP) {
            const uint64_t i = p.off + tid;
            strip_next<T>(g, p);
            live = true;
            return i;
        } else {
            const uint32_t v = tid + k * T;
            live = v < g.vchan;
            return live ? access_index(g, cbase, v) : 0;
        }
    };
    StripPos sp = strip_begin(g, c);
    if constexpr (XZ) {
        StripPos sz = sp;
#pragma unroll
        for (int k = 0; k < R; ++k) {
            bool live;
            const uint64_t i1 = resident_index(k, sz, live);
            if (live) {
                ku[k] = load_raw<kStream>(zs, i1);
                kg[k] = load_raw<kStream>(dzdx, i1);
            }
        }
#pragma unroll
        for (int k = 0; k < R; ++k) {
            if (STRIP || tid + k * T < g.vchan) {
                float tz[VEC];
                unpack<DT, VEC>(ku[k], tz);
#pragma unroll
                for (int e = 0; e < VEC; ++e)
                    negm[(k * VEC + e) / 32] |= static_cast<uint32_t>(tz[e] < 0.f)
                                                << ((k * VEC + e) % 32);
            }
        }
        // The bits must exist before the x loads are issued (a memory clobber
        // keeps the loads below this point and the bit arithmetic above it).
#pragma unroll
        for (int q = 0; q < NW; ++q) asm volatile("" : "+v"(negm[q])::"memory");
#pragma unroll
        for (int k = 0; k < R; ++k) {
            bool live;
            const uint64_t i1 = resident_index(k, sp, live);
            if (live) ku[k] = load_raw<kStream>(u, i1);
        }
    } else {
#pragma unroll
        for (int k = 0; k < R; ++k) {
            bool live;
            const uint64_t i1 = resident_index(k, sp, live);
            if (live) {
                ku[k] = load_raw<kStream>(u, i1);
                kg[k] = load_raw<kStream>(dzdx, i1);
            }
        }
    }
    // fp32 within one access, fp64 across accesses (as the streaming reduce
    // does per unrolled step): a channel's sums of dy cancel to near zero and
    // an fp32 running sum over the whole register-resident part loses that.
    double acc_dy = 0.0, acc_dyw = 0.0;
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if (STRIP || tid + k * T < g.vchan) {
            float tu[VEC], tg[VEC];
            unpack<DT, VEC>(ku[k], tu);
            unpack<DT, VEC>(kg[k], tg);
            float sdy = 0.f, sdyw = 0.f;
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                float dy, w;
                if constexpr (XZ) {
                    const bool neg = (negm[(k * VEC + e) / 32] >> ((k * VEC + e) % 32)) & 1u;
                    el.with_neg(neg, tu[e], tg[e], dy, w);
                } else {
                    el(tu[e], 0.f, tg[e], dy, w);
                }
                sdy += dy;
                sdyw = fmaf(dy, w, sdyw);
            }
            acc_dy += sdy;
            acc_dyw += sdyw;
        }
        sched_fence();
    }
    auto accumulate = [&](uint64_t i1) {
        float tu[VEC], tz[VEC], tg[VEC];
        unpack<DT, VEC>(load_raw<kCached>(u, i1), tu);
        if constexpr (XZ) unpack<DT, VEC>(load_raw<kCached>(zs, i1), tz);
        else
#pragma unroll
            for (int e = 0; e < VEC; ++e) tz[e] = 0.f;
        unpack<DT, VEC>(load_raw<kCached>(dzdx, i1), tg);
        float sdy = 0.f, sdyw = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            float dy, w;
            el(tu[e], tz[e], tg[e], dy, w);
            sdy += dy;
            sdyw = fmaf(dy, w, sdyw);
        }
        acc_dy += sdy;
        acc_dyw += sdyw;
    };
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            accumulate(sp.off + tid);
            strip_next<T>(g, sp);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T) accumulate(access_index(g, cbase, v));
    }

    double dbeta, sdyw;
    block_sums<T>(acc_dy, acc_dyw, dbeta, sdyw);
    uint32_t tid2 = tid;
    opaque(tid2);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        opaque(ku[k]);
        opaque(kg[k]);
    }
#pragma unroll
    for (int q = 0; q < NW; ++q) opaque(negm[q]);
    const double A = static_cast<double>(gamma_c) * invstd;
    const BwdApplyElem<BM> dx_of = make_apply_elem<BM>(A, sdyw, dbeta, g.m, prm.slope, gamma_c,
                                                       beta_c, mean_c, invstd, prm.ii != 0);
    if (tid == 0) {
        prm.dgamma[c] = static_cast<float>(sdyw);
        prm.dbeta[c] = static_cast<float>(dbeta);
    }
    auto emit = [&](raw16_t ru, raw16_t rz, raw16_t rg, uint64_t idx) {
        float tu[VEC], tz[VEC], tg[VEC];
        unpack<DT, VEC>(ru, tu);
        if constexpr (XZ) unpack<DT, VEC>(rz, tz);
        else
#pragma unroll
            for (int e = 0; e < VEC; ++e) tz[e] = 0.f;
        unpack<DT, VEC>(rg, tg);
#pragma unroll
        for (int e = 0; e < VEC; ++e) tg[e] = dx_of(tu[e], tz[e], tg[e]);
        store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, idx, tg);
    };
    // The resident accesses: dx from registers (kBwdFromXZ: signs from the bits).
    StripPos sq = strip_begin(g, c);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        uint64_t idx = 0;
        bool live = true;
        if constexpr (STRIP) {
            idx = sq.off + tid2;
            strip_next<T>(g, sq);
        } else {
            const uint32_t v = tid2 + k * T;
            live = v < g.vchan;
            if (live) idx = access_index(g, cbase, v);
        }
        if (live) {
            float tu[VEC], tg[VEC];
            unpack<DT, VEC>(ku[k], tu);
            unpack<DT, VEC>(kg[k], tg);
#pragma unroll
            for (int e = 0; e < VEC; ++e) {
                if constexpr (XZ) {
                    const bool neg = (negm[(k * VEC + e) / 32] >> ((k * VEC + e) % 32)) & 1u;
                    tg[e] = dx_of.with_neg(neg, tu[e], tg[e]);
                } else {
                    tg[e] = dx_of(tu[e], 0.f, tg[e]);
                }
            }
            store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, idx, tg);
        }
        sched_fence();
    }
    const raw16_t zero16 = {0u, 0u, 0u, 0u};
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            const uint64_t i1 = sq.off + tid2;
            emit(load_raw<kStream>(u, i1), XZ ? load_raw<kStream>(zs, i1) : zero16,
                 load_raw<kStream>(dzdx, i1), i1);
            strip_next<T>(g, sq);
        }
    } else {
#pragma unroll 1
        for (uint32_t v = tid2 + R * T; v < g.vchan; v += T) {
            const uint64_t i1 = access_index(g, cbase, v);
            emit(load_raw<kStream>(u, i1), XZ ? load_raw<kStream>(zs, i1) : zero16,
                 load_raw<kStream>(dzdx, i1), i1);
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
template <int DT, int VEC, int T, int R, bool STRIP, int FM>
__global__ __launch_bounds__(T) void fwd_fused_kernel(void* __restrict__ xz, Geom g,
                                                      FwdParams prm) {
    fwd_fused_channel<DT, VEC, T, R, STRIP, FM>(xz, g, prm, blockIdx.x);
}

template <int DT, int VEC, int T, int R, bool STRIP, int BM>
__global__ __launch_bounds__(T) void bwd_fused_kernel(const void* __restrict__ u,
                                                      const void* __restrict__ zs,
                                                      void* __restrict__ dzdx, Geom g,
                                                      BwdParams prm) {
    bwd_fused_channel<DT, VEC, T, R, STRIP, BM>(u, zs, dzdx, g, prm, blockIdx.x);
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

// train = false is inference (in place); otherwise fm is the output mode.
template <int DT, int VEC>
struct LaunchFwdApply {
    static void run(void* xz, const Geom& g, const Partial* part, const FwdParams& prm, bool train,
                    int fm, hipStream_t st) {
        constexpr int U = unroll<VEC>();
        const dim3 grid = grid_of(g);
        if (!train)
            fwd_apply_kernel<DT, VEC, U, false, kFwdInPlace><<<grid, kThreads, 0, st>>>(xz, g, part, prm);
        else if (fm == kFwdOut)
            fwd_apply_kernel<DT, VEC, U, true, kFwdOut><<<grid, kThreads, 0, st>>>(xz, g, part, prm);
        else if (fm == kFwdCkpt)
            fwd_apply_kernel<DT, VEC, U, true, kFwdCkpt><<<grid, kThreads, 0, st>>>(xz, g, part, prm);
        else
            fwd_apply_kernel<DT, VEC, U, true, kFwdInPlace><<<grid, kThreads, 0, st>>>(xz, g, part, prm);
    }
};

template <int DT, int VEC>
struct LaunchBwdReduce {
    static void run(const void* u, const void* zs, const void* dz, const Geom& g,
                    const BwdParams& prm, int bm, Partial* part, hipStream_t st) {
        constexpr int U = unroll<VEC>();
        const dim3 grid = grid_of(g);
        if (bm == kBwdFromXZ)
            bwd_reduce_kernel<DT, VEC, U, kBwdFromXZ><<<grid, kThreads, 0, st>>>(u, zs, dz, g, prm, part);
        else if (bm == kBwdFromXhat)
            bwd_reduce_kernel<DT, VEC, U, kBwdFromXhat><<<grid, kThreads, 0, st>>>(u, zs, dz, g, prm, part);
        else
            bwd_reduce_kernel<DT, VEC, U, kBwdFromZ><<<grid, kThreads, 0, st>>>(u, zs, dz, g, prm, part);
    }
};

template <int DT, int VEC>
struct LaunchBwdApply {
    static void run(const void* u, const void* zs, void* dzdx, const Geom& g, const Partial* part,
                    const BwdParams& prm, int bm, hipStream_t st) {
        constexpr int U = unroll<VEC>();
        const dim3 grid = grid_of(g);
        if (bm == kBwdFromXZ)
            bwd_apply_kernel<DT, VEC, U, kBwdFromXZ><<<grid, kThreads, 0, st>>>(u, zs, dzdx, g, part, prm);
        else if (bm == kBwdFromXhat)
            bwd_apply_kernel<DT, VEC, U, kBwdFromXhat><<<grid, kThreads, 0, st>>>(u, zs, dzdx, g, part, prm);
        else
            bwd_apply_kernel<DT, VEC, U, kBwdFromZ><<<grid, kThreads, 0, st>>>(u, zs, dzdx, g, part, prm);
    }
};

template <int DT, int VEC>
struct LaunchRecompute {
    static void run(const void* xhat, void* z, const Geom& g, const float* gamma, const float* beta,
                    float slope, hipStream_t st) {
        recompute_kernel<DT, VEC><<<grid_of(g), kThreads, 0, st>>>(xhat, z, g, gamma, beta, slope);
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

#define IABN_FUSED_CASE(KERNEL, MODE, TT, RR, ...)                                             \
    if (fp.T == TT && fp.R == RR) {                                                           \
        if (kUseStrips && g.vrow % TT == 0 && g.vchan / TT >= RR)                             \
            KERNEL<DT, V, TT, RR, true, MODE><<<grid, TT, lds, st>>>(__VA_ARGS__);            \
        else                                                                                  \
            KERNEL<DT, V, TT, RR, false, MODE><<<grid, TT, lds, st>>>(__VA_ARGS__);           \
        return true;                                                                          \
    }

template <int DT, int FM>
bool launch_fwd_fused(void* xz, const Geom& g, const FusedPlan& fp, const FwdParams& prm,
                      hipStream_t st) {
    constexpr int V = 16 / sizeof(typename Elem<DT>::T);
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedFwdBlocksPerCU);
    IABN_FUSED_CASE(fwd_fused_kernel, FM, 256, 4, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, FM, 512, 4, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, FM, 256, 16, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, FM, 512, 16, xz, g, prm)
    IABN_FUSED_CASE(fwd_fused_kernel, FM, 1024, 16, xz, g, prm)
    return false;
}

template <int DT, int BM>
bool launch_bwd_fused(const void* u, const void* zs, void* dzdx, const Geom& g,
                      const FusedPlan& fp, const BwdParams& prm, hipStream_t st) {
    constexpr int V = 16 / sizeof(typename Elem<DT>::T);
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedBwdBlocksPerCU);
    IABN_FUSED_CASE(bwd_fused_kernel, BM, 256, 4, u, zs, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, BM, 512, 4, u, zs, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, BM, 256, 16, u, zs, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, BM, 512, 16, u, zs, dzdx, g, prm)
    IABN_FUSED_CASE(bwd_fused_kernel, BM, 1024, 8, u, zs, dzdx, g, prm)
    return false;
}

#undef IABN_FUSED_CASE

template <int FM>
bool launch_fwd_fused_dt(int dtype, void* xz, const Geom& g, const FusedPlan& fp,
                         const FwdParams& prm, hipStream_t st) {
    return dtype == IABN_F32   ? launch_fwd_fused<IABN_F32, FM>(xz, g, fp, prm, st)
           : dtype == IABN_F16 ? launch_fwd_fused<IABN_F16, FM>(xz, g, fp, prm, st)
                               : launch_fwd_fused<IABN_BF16, FM>(xz, g, fp, prm, st);
}

template <int BM>
bool launch_bwd_fused_dt(int dtype, const void* u, const void* zs, void* dzdx, const Geom& g,
                         const FusedPlan& fp, const BwdParams& prm, hipStream_t st) {
    return dtype == IABN_F32   ? launch_bwd_fused<IABN_F32, BM>(u, zs, dzdx, g, fp, prm, st)
           : dtype == IABN_F16 ? launch_bwd_fused<IABN_F16, BM>(u, zs, dzdx, g, fp, prm, st)
                               : launch_bwd_fused<IABN_BF16, BM>(u, zs, dzdx, g, fp, prm, st);
}

// ---- end fused planning

int validate_common(int dtype, int64_t N, int64_t C, int64_t HW, bool train) {
    if (!valid_dtype(dtype)) return fail(IABN_ERR_DTYPE, "unknown dtype %d", dtype);
    return check_shape(N, C, HW, train);
}

bool empty(int64_t N, int64_t C, int64_t HW) { return C == 0 || N * HW == 0; }

bool vector_ok(int64_t HW, int dtype, const void* a, const void* b, const void* c) {
    return use_vector(HW, dtype, a, b) && (c == nullptr || aligned16(c));
}

const char* fwd_name(int fm) {
    return fm == kFwdOut ? "standard forward" : fm == kFwdCkpt ? "checkpointing forward" : "forward";
}

// Training forward of the three arms (fm: kFwdInPlace, kFwdOut, kFwdCkpt).
// x is the input (kFwdInPlace: z on return; kFwdCkpt: xhat on return); out
// receives z for kFwdOut and kFwdCkpt.  Everything is validated before the
// first launch, so an error changes nothing.
int forward_train_impl(int fm, void* x, void* out, int dtype, const float* gamma,
                       const float* beta, float* running_mean, float* running_var,
                       float* save_mean, float* save_var, float eps, float momentum, float slope,
                       int64_t N, int64_t C, int64_t HW, void* workspace, size_t workspace_bytes,
                       void* stream) {
    int rc = validate_common(dtype, N, C, HW, true);
    if (rc) return rc;
    if (empty(N, C, HW)) return ok();
    if (!x || !gamma || !beta || !running_mean || !running_var || !save_mean || !save_var ||
        (fm != kFwdInPlace && !out))
        return fail(IABN_ERR_NULL, "a tensor or parameter pointer is NULL");
    if ((rc = check_params(eps, slope))) return rc;
    if (!(momentum >= 0.f && momentum <= 1.f))
        return fail(IABN_ERR_PARAM, "momentum must lie in [0, 1]");
    if ((rc = check_workspace(N, C, HW, workspace, workspace_bytes))) return rc;
    const bool vec = use_vector(HW, dtype, x, fm == kFwdInPlace ? nullptr : out);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const FwdParams prm = {gamma,    beta, running_mean, running_var, save_mean, save_var,
                           fm == kFwdInPlace ? nullptr : out, eps, momentum, slope};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    FusedPlan fp;
    if (plan_fused(C, g, vec, false, &fp)) {
        const bool ok = fm == kFwdOut    ? launch_fwd_fused_dt<kFwdOut>(dtype, x, g, fp, prm, st)
                        : fm == kFwdCkpt ? launch_fwd_fused_dt<kFwdCkpt>(dtype, x, g, fp, prm, st)
                                         : launch_fwd_fused_dt<kFwdInPlace>(dtype, x, g, fp, prm, st);
        if (!ok)
            return fail(IABN_ERR_HIP, "no %s kernel built for T=%d R=%d", fwd_name(fm), fp.T, fp.R);
        return launched(fwd_name(fm));
    }
    Partial* part = static_cast<Partial*>(workspace);
    dispatch<LaunchFwdStats>(dtype, vec, static_cast<const void*>(x), g, part, st);
    if ((rc = launched("fwd_stats"))) return rc;
    dispatch<LaunchFwdApply>(dtype, vec, x, g, static_cast<const Partial*>(part), prm, true, fm, st);
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
    const bool vec = vector_ok(HW, dtype, u, dz_dx, bm == kBwdFromXZ ? zs : nullptr);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, save_mean, save_var, dgamma, dbeta, eps, slope, ii ? 1 : 0};
    const hipStream_t st = static_cast<hipStream_t>(stream);
    FusedPlan fp;
    if (plan_fused(C, g, vec, true, &fp)) {
        const bool ok =
            bm == kBwdFromXZ     ? launch_bwd_fused_dt<kBwdFromXZ>(dtype, u, zs, dz_dx, g, fp, prm, st)
            : bm == kBwdFromXhat ? launch_bwd_fused_dt<kBwdFromXhat>(dtype, u, zs, dz_dx, g, fp, prm, st)
                                 : launch_bwd_fused_dt<kBwdFromZ>(dtype, u, zs, dz_dx, g, fp, prm, st);
        if (!ok)
            return fail(IABN_ERR_HIP, "no %s kernel built for T=%d R=%d", bwd_name(bm, ii), fp.T, fp.R);
        return launched(bwd_name(bm, ii));
    }
    Partial* part = static_cast<Partial*>(workspace);
    dispatch<LaunchBwdReduce>(dtype, vec, u, zs, static_cast<const void*>(dz_dx), g, prm, bm, part, st);
    if ((rc = launched("bwd_reduce"))) return rc;
    dispatch<LaunchBwdApply>(dtype, vec, u, zs, dz_dx, g, static_cast<const Partial*>(part), prm, bm, st);
    return launched(bwd_name(bm, ii));
}

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
                           nullptr, eps, momentum, slope};
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const Partial*>(workspace), prm, true,
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
                           const_cast<float*>(running_var), nullptr, nullptr, nullptr, eps, 0.f,
                           slope};
    dispatch<LaunchFwdApply>(dtype, vec, x_z, g, static_cast<const Partial*>(nullptr), prm, false,
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
    const bool vec = use_vector(HW, dtype, z, dz);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    const BwdParams prm = {gamma, beta, nullptr, nullptr, nullptr, nullptr, 1.f, slope, 0};
    dispatch<LaunchBwdReduce>(dtype, vec, z, static_cast<const void*>(nullptr), dz, g, prm,
                              kBwdFromZ, static_cast<Partial*>(workspace),
                              static_cast<hipStream_t>(stream));
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
    const BwdParams prm = {gamma, beta, nullptr, save_var, dgamma, dbeta, eps, slope, 0};
    dispatch<LaunchBwdApply>(dtype, vec, z, static_cast<const void*>(nullptr), dz_dx, g,
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
    const bool vec = use_vector(HW, dtype, xhat, z);
    const Geom g = make_geom(N, C, HW, dtype, vec);
    dispatch<LaunchRecompute>(dtype, vec, xhat, z, g, gamma, beta, slope,
                              static_cast<hipStream_t>(stream));
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
