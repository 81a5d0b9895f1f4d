// Definitions shared by every kernel and the host side of libiabn:
// storage types and vector accesses, the access geometry of a layer, the
// per-wave partial results of the streaming reductions, the parameters and
// output modes of the forward, and the per-element forms of the backward
// formulations.  InPlace-ABN (arXiv:1712.02616) for AMD Instinct MI355X
// (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "divmagic.h"
#include "iabn.h"

namespace iabn_impl {

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

// VEC elements per access: 16, 8, 4 or 2 bytes, or a single element.
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
    double inv_m;             // 1 / m
    // Order of the channels (or slices) over the blocks of a launch (see
    // fused_channel and block_slice): xcd_order set, each XCD takes a
    // contiguous range of them; a channel-resident launch's XCDs take xcd_q
    // or xcd_q + 1 channels each.
    uint32_t xcd_order, xcd_q, xcd_r;
};

// XCDs (accelerator complex dies, each with its own L2) of the device.
constexpr uint32_t kXcds = 8;

// Index (in accesses) of the v-th access of channel c.
__device__ __forceinline__ uint64_t access_index(const Geom& g, uint64_t cbase, uint32_t v) {
    const uint32_t n = iabn_divmagic_div(v, g.row_div);
    const uint32_t i = v - n * g.vrow;
    return static_cast<uint64_t>(n) * g.nstride + cbase + i;
}

struct Slice {
    uint32_t c, p, lo, hi;
};

// The slice of this block: slice k = c*P + p covers part p of channel c.
// Block k takes slice k, or, with xcd_order (rows that do not end on a
// cache line), the blocks on each XCD (block b on XCD b mod 8) take a
// contiguous range of slices, so that neighbouring slices, which share the
// lines where their rows meet, read them through one L2 (the inference
// forward on (32, 2048, 7x7) fp16: 10.2 us against 14.5).
__device__ __forceinline__ Slice block_slice(const Geom& g) {
    Slice s;
    uint32_t b = blockIdx.x;
    if (g.xcd_order) {
        const uint32_t n = gridDim.x, x = b % kXcds, j = b / kXcds;
        b = x * (n / kXcds) + min(x, n % kXcds) + j;
    }
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

// One DPP move of a double (both halves; lanes without a source read 0).
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t bits = __builtin_bit_cast(uint64_t, v);
    const int lo = __builtin_amdgcn_update_dpp(0, static_cast<int>(bits & 0xffffffffu), CTRL,
                                               ROW_MASK, 0xF, true);
    const int hi = __builtin_amdgcn_update_dpp(0, static_cast<int>(bits >> 32), CTRL, ROW_MASK,
                                               0xF, true);
    return __builtin_bit_cast(
        double, (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo));
}

// Sum over the 64 lanes of a wave (every lane must be active), returned in
// every lane.  Register-to-register DPP steps: within each row of 16 lanes,
// shifts by 1, 2, 4 and 8 leave the row's sum in its lane 15; two row
// broadcasts then carry rows 0-1 and 2-3 into lane 63.  The order of the
// additions is fixed, so the result is the same on every run.
__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_f64<0x111, 0xF>(v);  // row_shr:1
    v += dpp_f64<0x112, 0xF>(v);  // row_shr:2
    v += dpp_f64<0x114, 0xF>(v);  // row_shr:4
    v += dpp_f64<0x118, 0xF>(v);  // row_shr:8
    v += dpp_f64<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_f64<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    const uint64_t bits = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = __builtin_amdgcn_readlane(static_cast<int>(bits & 0xffffffffu), 63);
    const uint32_t hi = __builtin_amdgcn_readlane(static_cast<int>(bits >> 32), 63);
    return __builtin_bit_cast(double, (static_cast<uint64_t>(hi) << 32) | lo);
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
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    n = wave_sum(n);
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
    sdy = wave_sum(a);
    sdyx = wave_sum(b);
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

// Reciprocals of the per-channel divisors, formed before the reduction so
// that the constants after it take multiplications only.
struct BwdRecip {
    double g, ag, m;  // 1/gamma, 1/(slope gamma), 1/m
};

__device__ __forceinline__ BwdRecip make_recip(float gamma, float slope, double inv_m) {
    const double g = gamma;
    BwdRecip r;
    r.g = 1.0 / g;
    r.ag = 1.0 / (static_cast<double>(slope) * g);
    r.m = inv_m;
    return r;
}

// dgamma from the two sums (formulation II converts sum dy*y), then the
// apply constants.  sdyw is overwritten with dgamma.
template <int BM>
__device__ __forceinline__ BwdApplyElem<BM> make_apply_elem(double A, double& sdyw, double dbeta,
                                                            const BwdRecip& rc, float slope,
                                                            float gamma, float beta, float mean,
                                                            double invstd, bool ii) {
    const double a = slope, bt = beta;
    if (BM == kBwdFromZ && ii) sdyw = (sdyw - bt * dbeta) * rc.g;
    const double dgamma = sdyw;
    const double B = -A * dgamma * rc.m, C = -A * dbeta * rc.m;
    BwdApplyElem<BM> el;
    el.sign.gamma = gamma;
    el.sign.beta = beta;
    el.a_pos = static_cast<float>(A);
    el.a_neg = static_cast<float>(A * a);
    el.off = 0.f;
    if constexpr (BM == kBwdFromZ) {
        el.b_pos = static_cast<float>(B * rc.g);
        el.b_neg = static_cast<float>(B * rc.ag);
        el.c0 = static_cast<float>(C - B * bt * rc.g);
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

// 1/sqrt(v) in double: the hardware estimate refined by one Newton step
// (relative error about 1e-14, far below the fp32 constants it feeds).
__device__ __forceinline__ double rsqrt_d(double v) {
    const double r = __builtin_amdgcn_rsq(v);
    return r * (1.5 - 0.5 * v * r * r);
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

}  // namespace iabn_impl
