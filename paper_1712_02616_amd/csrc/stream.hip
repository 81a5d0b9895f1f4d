// The streaming kernels of libiabn, all bound by HBM bandwidth:
//   fwd_stats    reads x, writes per-(channel, slice) partial moments
//   fwd_apply    combines a channel's partials (fixed order), writes the
//                statistics, writes z = f(gamma*xhat + beta) (over x, or to a
//                second buffer; the checkpointing mode writes xhat over x and
//                z to the second buffer); also inference with fixed statistics
//   recompute    z = f(gamma*xhat + beta) from a stored xhat
//   bwd_reduce   reads the stored tensor(s) and dz, writes per-(channel,
//                slice) partial sums of dy and dy*w (see the backward modes)
//   bwd_apply    combines the partial sums, writes dgamma/dbeta, overwrites
//                dz with dx
// They serve the phase entry points, and the fused entry points for shapes
// the channel-resident kernels do not take (few channels, odd rows).
//
// Work decomposition.  A channel's m = N*HW values are N rows of HW
// contiguous elements, C*HW elements apart.  Each channel is cut into P
// slices of L elements (the last one shorter); one 256-thread block owns one
// (channel, slice) pair, so each block sees a single channel and reads its
// parameters once.  Slices are defined in elements, independent of the
// access width, so the partials of a slice mean the same thing whichever
// path wrote them.  Inside a slice a thread reads vectors v = lo + tid,
// lo + tid + 256, ... (consecutive lanes touch consecutive vectors), U of
// them in flight before any arithmetic.  A vector is 16 bytes wide, or 8, 4
// or 2 bytes where HW or the pointers' alignment rule out the wider ones, or
// a single element (odd HW); it never crosses a row because HW is a multiple
// of the vector width.
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

#include "fused.h"
#include "launch.h"

namespace iabn_impl {
namespace {

// Index of access v of a slice's last, partial batch: accesses at or past
// the slice's end read the slice's first access instead (a line the block
// reads anyway) and are not used.  Loading every access of the batch
// unconditionally keeps all of them in flight at once; one at a time, a
// short slice of narrow accesses waited for each load in turn.
__device__ __forceinline__ uint64_t rest_index(const Geom& g, uint64_t cbase, const Slice& s,
                                               uint32_t v) {
    return access_index(g, cbase, v < s.hi ? v : s.lo);
}

// The accesses of a batch are loaded raw, all of them, before any is
// widened to fp32 (sched_fence between): left to itself the compiler
// interleaves each conversion, and the wait it needs, with the next load,
// which on narrow accesses (a dozen or more per batch) left one load in
// flight at a time.
template <int DT, int VEC, int U>
__device__ __forceinline__ void widen(const raw_t<DT, VEC> (&r)[U], float (&t)[U][VEC]) {
#pragma unroll
    for (int u = 0; u < U; ++u) unpack<DT, VEC>(r[u], t[u]);
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
        raw_t<DT, VEC> r[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            r[u] = load_raw<DT, VEC, kHintStatsLoad>(x, access_index(g, cbase, v + u * kThreads));
        sched_fence();
        float t[U][VEC];
        widen<DT, VEC, U>(r, t);
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
    // The last, partial batch: every load in flight at once (accesses past
    // the slice read its first access instead and are not used; see
    // rest_index).
    if (v < s.hi) {
        raw_t<DT, VEC> r[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            r[u] = load_raw<DT, VEC, kHintStatsLoad>(x, rest_index(g, cbase, s, v + u * kThreads));
        sched_fence();
        float t[U][VEC];
        widen<DT, VEC, U>(r, t);
        if (first) shift = t[0][0];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (v + u * kThreads < s.hi) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    const float d = t[u][k] - shift;
                    s1 += d;
                    s2 = fmaf(d, d, s2);
                }
                nacc += 1;
            }
        }
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
    const Slice s = block_slice(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    // First batch in flight before the per-channel coefficients are known.
    uint32_t v = s.lo + threadIdx.x;
    raw_t<DT, VEC> r[U];
    uint64_t idx[U];
    bool full = v + (U - 1) * kThreads < s.hi;
    if (full) {
#pragma unroll
        for (int q = 0; q < U; ++q) {
            idx[q] = access_index(g, cbase, v + q * kThreads);
            r[q] = load_raw<DT, VEC, kHintFwdApplyLoad>(xz, idx[q]);
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
        float t[U][VEC];
        widen<DT, VEC, U>(r, t);
#pragma unroll
        for (int q = 0; q < U; ++q) emit(t[q], idx[q]);
        v += U * kThreads;
        full = v + (U - 1) * kThreads < s.hi;
        if (full) {
#pragma unroll
            for (int q = 0; q < U; ++q) {
                idx[q] = access_index(g, cbase, v + q * kThreads);
                r[q] = load_raw<DT, VEC, kHintFwdApplyLoad>(xz, idx[q]);
            }
            sched_fence();
        }
    }
    if (v < s.hi) {
#pragma unroll
        for (int q = 0; q < U; ++q)
            r[q] = load_raw<DT, VEC, kHintFwdApplyLoad>(xz, rest_index(g, cbase, s, v + q * kThreads));
        sched_fence();
        float t[U][VEC];
        widen<DT, VEC, U>(r, t);
#pragma unroll
        for (int q = 0; q < U; ++q)
            if (v + q * kThreads < s.hi) emit(t[q], access_index(g, cbase, v + q * kThreads));
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

// One batch of the backward's tensors at accesses idx(0..U-1), raw: u, the
// stored z for kBwdFromXZ, dz.
template <int DT, int VEC, int HINT, int U, int BM, typename Index>
__device__ __forceinline__ void load_bwd_raw(const void* __restrict__ u,
                                             const void* __restrict__ zs,
                                             const void* __restrict__ dz, Index idx,
                                             raw_t<DT, VEC> (&ru)[U], raw_t<DT, VEC> (&rz)[U],
                                             raw_t<DT, VEC> (&rg)[U]) {
#pragma unroll
    for (int q = 0; q < U; ++q) {
        const uint64_t i1 = idx(q);
        ru[q] = load_raw<DT, VEC, HINT>(u, i1);
        if constexpr (BM == kBwdFromXZ) rz[q] = load_raw<DT, VEC, HINT>(zs, i1);
        rg[q] = load_raw<DT, VEC, HINT>(dz, i1);
    }
}

// The same widened to fp32 (z as zeros unless kBwdFromXZ).
template <int DT, int VEC, int U, int BM>
__device__ __forceinline__ void widen_bwd(const raw_t<DT, VEC> (&ru)[U],
                                          const raw_t<DT, VEC> (&rz)[U],
                                          const raw_t<DT, VEC> (&rg)[U], float (&tu)[U][VEC],
                                          float (&tz)[U][VEC], float (&tg)[U][VEC]) {
    widen<DT, VEC, U>(ru, tu);
    widen<DT, VEC, U>(rg, tg);
    if constexpr (BM == kBwdFromXZ) {
        widen<DT, VEC, U>(rz, tz);
    } else {
#pragma unroll
        for (int q = 0; q < U; ++q)
#pragma unroll
            for (int k = 0; k < VEC; ++k) tz[q][k] = 0.f;
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
        raw_t<DT, VEC> ru[U], rz[U], rg[U];
        load_bwd_raw<DT, VEC, kHintReduceLoad, U, BM>(
            u, zs, dz, [&](int q) { return access_index(g, cbase, v + q * kThreads); }, ru, rz, rg);
        sched_fence();
        float tu[U][VEC], tz[U][VEC], tg[U][VEC];
        widen_bwd<DT, VEC, U, BM>(ru, rz, rg, tu, tz, tg);
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
    if (v < s.hi) {
        raw_t<DT, VEC> ru[U], rz[U], rg[U];
        load_bwd_raw<DT, VEC, kHintReduceLoad, U, BM>(
            u, zs, dz, [&](int q) { return rest_index(g, cbase, s, v + q * kThreads); }, ru, rz, rg);
        sched_fence();
        float tu[U][VEC], tz[U][VEC], tg[U][VEC];
        widen_bwd<DT, VEC, U, BM>(ru, rz, rg, tu, tz, tg);
        float sdy = 0.f, sdyw = 0.f;
#pragma unroll
        for (int q = 0; q < U; ++q) {
            if (v + q * kThreads < s.hi) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) {
                    float dy, w;
                    el(tu[q][k], tz[q][k], tg[q][k], dy, w);
                    sdy += dy;
                    sdyw = fmaf(dy, w, sdyw);
                }
            }
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
    const Slice s = block_slice(g);
    const uint64_t cbase = static_cast<uint64_t>(s.c) * g.vrow;

    uint32_t v = s.lo + threadIdx.x;
    raw_t<DT, VEC> ru[U], rz[U], rg[U];
    uint64_t idx[U];
    bool full = v + (U - 1) * kThreads < s.hi;
    if (full) {
#pragma unroll
        for (int q = 0; q < U; ++q) idx[q] = access_index(g, cbase, v + q * kThreads);
        load_bwd_raw<DT, VEC, kHintBwdApplyLoad, U, BM>(
            u, zs, dzdx, [&](int q) { return idx[q]; }, ru, rz, rg);
    }

    double dbeta, dgamma;
    channel_sums(g, part, s.c, dbeta, dgamma);
    const double invstd = chan_invstd(prm, s.c);
    const double A = static_cast<double>(prm.gamma[s.c]) * invstd;
    const BwdApplyElem<BM> dx_of = make_apply_elem<BM>(
        A, dgamma, dbeta, make_recip(prm.gamma[s.c], prm.slope, g.inv_m), prm.slope,
        prm.gamma[s.c], prm.beta[s.c], BM == kBwdFromXZ ? prm.save_mean[s.c] : 0.f, invstd,
        prm.ii != 0);
    if (s.p == 0 && threadIdx.x == 0) {
        prm.dgamma[s.c] = static_cast<float>(dgamma);
        prm.dbeta[s.c] = static_cast<float>(dbeta);
    }

    while (full) {
        float tu[U][VEC], tz[U][VEC], tg[U][VEC];
        widen_bwd<DT, VEC, U, BM>(ru, rz, rg, tu, tz, tg);
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
            for (int q = 0; q < U; ++q) idx[q] = access_index(g, cbase, v + q * kThreads);
            load_bwd_raw<DT, VEC, kHintBwdApplyLoad, U, BM>(
                u, zs, dzdx, [&](int q) { return idx[q]; }, ru, rz, rg);
            sched_fence();
        }
    }
    if (v < s.hi) {
        load_bwd_raw<DT, VEC, kHintBwdApplyLoad, U, BM>(
            u, zs, dzdx, [&](int q) { return rest_index(g, cbase, s, v + q * kThreads); }, ru, rz,
            rg);
        sched_fence();
        float tu[U][VEC], tz[U][VEC], tg[U][VEC];
        widen_bwd<DT, VEC, U, BM>(ru, rz, rg, tu, tz, tg);
#pragma unroll
        for (int q = 0; q < U; ++q) {
            if (v + q * kThreads < s.hi) {
#pragma unroll
                for (int k = 0; k < VEC; ++k) tg[q][k] = dx_of(tu[q][k], tz[q][k], tg[q][k]);
                store_vec<DT, VEC, kHintBwdApplyStore>(dzdx, access_index(g, cbase, v + q * kThreads), tg[q]);
            }
        }
    }
}

dim3 grid_of(const Geom& g) { return dim3(g.C * g.P); }

// Dispatch on dtype and access width (elements per access: 16, 8, 4 or 2
// bytes' worth).
template <template <int, int> class Launch, int DT, typename... A>
void dispatch_vec(int vec, A&&... args) {
    constexpr int W = 16 / static_cast<int>(sizeof(typename Elem<DT>::T));
    if (vec == W) {
        Launch<DT, W>::run(args...);
    } else if (vec == W / 2) {
        Launch<DT, W / 2>::run(args...);
    } else if (W / 4 > 1 && vec == W / 4) {
        Launch<DT, (W / 4 > 1 ? W / 4 : 1)>::run(args...);
    } else {
        Launch<DT, 1>::run(args...);
    }
}

template <template <int, int> class Launch, typename... A>
void dispatch(int dtype, int vec, A&&... args) {
    switch (dtype) {
        case IABN_F32: dispatch_vec<Launch, IABN_F32>(vec, args...); break;
        case IABN_F16: dispatch_vec<Launch, IABN_F16>(vec, args...); break;
        default: dispatch_vec<Launch, IABN_BF16>(vec, args...); break;
    }
}

// Accesses in flight per thread and batch: 32 bytes' worth (2 x 16 bytes on
// the 16-byte path, measured best on the backbone sweep), at least 8.
template <int DT, int VEC>
constexpr int unroll() {
    constexpr int bytes = VEC * static_cast<int>(sizeof(typename Elem<DT>::T));
    return bytes >= 16 ? 2 : (32 / bytes < 8 ? 8 : 32 / bytes);
}

// Long slices: on the 16-byte path, a pass whose blocks own slices of at
// least the pass's threshold (in accesses) keeps kLongU accesses per tensor
// in flight per thread instead of unroll()'s 2.  Few-channel layers cut into
// many slices run 512 blocks, 2 waves per SIMD, and then need the deeper
// batches to keep enough bytes in flight; measured on (8, 64, 256x256) and
// (32, 64, 112x112) fp16 and (16, 32, 112x112) fp32: statistics up to 13%,
// training apply 7-12%, backward apply up to 3% faster from 8 accesses per
// thread up (the last, partial batch is loaded whole, so short slices lose
// nothing to a remainder loop); the backward's reduction, which reads two
// tensors, gains only from 32 up (6% on 32, 1-6% slower on 12 and 24).  The
// inference apply keeps 2: 8 made it 5% slower over the backbone sweep's
// layers and no faster on the few-channel ones.
constexpr int kLongU = 8;
constexpr uint32_t kLongStatsAccesses = 8 * kThreads;
constexpr uint32_t kLongApplyAccesses = 8 * kThreads;
constexpr uint32_t kLongReduceAccesses = 32 * kThreads;
constexpr uint32_t kLongBwdApplyAccesses = 8 * kThreads;

template <int DT, int VEC>
constexpr bool wide_access() {
    return VEC * sizeof(typename Elem<DT>::T) == 16;
}

// Whether a pass with threshold `min_accesses` takes the long batches.
template <int DT, int VEC>
bool long_slices(const Geom& g, uint32_t min_accesses) {
    return wide_access<DT, VEC>() && g.lv >= min_accesses;
}

// The long batch where the access width has one (16-byte accesses), else
// the default; both branches of a launch name a kernel that exists.
template <int DT, int VEC>
constexpr int long_unroll() {
    return wide_access<DT, VEC>() ? kLongU : unroll<DT, VEC>();
}

template <int DT, int VEC>
struct LaunchFwdStats {
    static void run(const void* x, const Geom& g, Partial* part, hipStream_t st) {
        if (long_slices<DT, VEC>(g, kLongStatsAccesses))
            fwd_stats_kernel<DT, VEC, long_unroll<DT, VEC>()><<<grid_of(g), kThreads, 0, st>>>(x, g, part);
        else
            fwd_stats_kernel<DT, VEC, unroll<DT, VEC>()><<<grid_of(g), kThreads, 0, st>>>(x, g, part);
    }
};

// train = false is inference (in place); otherwise fm is the output mode.
template <int DT, int VEC>
struct LaunchFwdApply {
    static void run(void* xz, const Geom& g, const Partial* part, const FwdParams& prm, bool train,
                    int fm, hipStream_t st) {
        if (train && long_slices<DT, VEC>(g, kLongApplyAccesses))
            go<long_unroll<DT, VEC>()>(xz, g, part, prm, train, fm, st);
        else
            go<unroll<DT, VEC>()>(xz, g, part, prm, train, fm, st);
    }
    template <int U>
    static void go(void* xz, const Geom& g, const Partial* part, const FwdParams& prm, bool train,
                   int fm, hipStream_t st) {
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
        if (long_slices<DT, VEC>(g, kLongReduceAccesses))
            go<long_unroll<DT, VEC>()>(u, zs, dz, g, prm, bm, part, st);
        else
            go<unroll<DT, VEC>()>(u, zs, dz, g, prm, bm, part, st);
    }
    template <int U>
    static void go(const void* u, const void* zs, const void* dz, const Geom& g,
                   const BwdParams& prm, int bm, Partial* part, hipStream_t st) {
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
        if (long_slices<DT, VEC>(g, kLongBwdApplyAccesses))
            go<long_unroll<DT, VEC>()>(u, zs, dzdx, g, part, prm, bm, st);
        else
            go<unroll<DT, VEC>()>(u, zs, dzdx, g, part, prm, bm, st);
    }
    template <int U>
    static void go(const void* u, const void* zs, void* dzdx, const Geom& g, const Partial* part,
                   const BwdParams& prm, int bm, hipStream_t st) {
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

}  // namespace

void launch_fwd_stats(int dtype, int vec, const void* x, const Geom& g, Partial* part,
                      hipStream_t st) {
    dispatch<LaunchFwdStats>(dtype, vec, x, g, part, st);
}

void launch_fwd_apply(int dtype, int vec, void* xz, const Geom& g, const Partial* part,
                      const FwdParams& prm, bool train, int fm, hipStream_t st) {
    dispatch<LaunchFwdApply>(dtype, vec, xz, g, part, prm, train, fm, st);
}

void launch_bwd_reduce(int dtype, int vec, const void* u, const void* zs, const void* dz,
                       const Geom& g, const BwdParams& prm, int bm, Partial* part, hipStream_t st) {
    dispatch<LaunchBwdReduce>(dtype, vec, u, zs, dz, g, prm, bm, part, st);
}

void launch_bwd_apply(int dtype, int vec, const void* u, const void* zs, void* dzdx,
                      const Geom& g, const Partial* part, const BwdParams& prm, int bm,
                      hipStream_t st) {
    dispatch<LaunchBwdApply>(dtype, vec, u, zs, dzdx, g, part, prm, bm, st);
}

void launch_recompute(int dtype, int vec, const void* xhat, void* z, const Geom& g,
                      const float* gamma, const float* beta, float slope, hipStream_t st) {
    dispatch<LaunchRecompute>(dtype, vec, xhat, z, g, gamma, beta, slope, st);
}

}  // namespace iabn_impl
