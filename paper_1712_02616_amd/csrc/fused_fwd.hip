// The channel-resident training forward: one block per channel holds the
// channel's accesses in registers (and, in 1024-thread blocks, LDS) from the
// statistics to the apply, so x crosses HBM once in and the outputs once out
// (what does not fit is read again).  Output modes as in
// common.h (InPlace-ABN, standard, checkpointing).

#include "fused.h"
#include "launch.h"

namespace iabn_impl {
namespace {

// Per-channel constants of the fused forward's apply phase.
struct FwdApplyK {
    float mean_hi, scale, bshift, slope;  // y = (x - mean_hi) * scale + bshift (kFwdCkpt: xhat)
    float gamma, beta;                    // kFwdCkpt: y = gamma * xhat + beta
    void* out;                            // kFwdOut / kFwdCkpt: z
};

// The outputs of one access from its input values t (overwritten).
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
template <int DT, int VEC, int T, int R, int S, bool STRIP, int FM, bool SMALL_SLOPE>
__device__ __forceinline__ void fwd_fused_apply(void* __restrict__ xz, const Geom& g, uint32_t c,
                                                uint32_t tid, const raw_t<DT, VEC> (&keep)[R],
                                                const raw_t<DT, VEC> (&lx)[S > 0 ? S : 1][T],
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
            unpack<DT, VEC>(S > 0 && k < R + S ? lx[k - R][tid] : load_raw<DT, VEC, kStream>(xz, idx), t);
            fwd_fused_emit<DT, VEC, FM, SMALL_SLOPE>(xz, idx, t, kk);
            strip_next<T>(g, sq);
        }
    } else {
        uint32_t j = 0;
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T, ++j) {
            const uint64_t idx = access_index(g, cbase, v);
            float t[VEC];
            unpack<DT, VEC>(S > 0 && j < S ? lx[j][tid] : load_raw<DT, VEC, kStream>(xz, idx), t);
            fwd_fused_emit<DT, VEC, FM, SMALL_SLOPE>(xz, idx, t, kk);
        }
    }
}

// Training forward of one channel per block (statistics, running estimates,
// z over x), same arithmetic as fwd_stats_kernel + fwd_apply_kernel in
// stream.hip.
template <int DT, int VEC, int T, int R, bool STRIP, int FM, int CPB = 1>
__device__ __forceinline__ void fwd_fused_channel(void* __restrict__ xz, const Geom& g,
                                                  const FwdParams& prm, uint32_t c) {
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t tid = CPB > 1 ? threadIdx.x % T : threadIdx.x;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    // The first R accesses per thread stay in registers until the apply, so
    // this is their only read: non-temporal.  Accesses past those are read
    // again by the apply and go through the caches.  (Measured: non-temporal
    // register-resident loads cut the forward over the backbone sweep by 12%
    // and the backward by 7%.)
    raw_t<DT, VEC> keep[R];
    // The first S accesses per thread past the registers (1024-thread
    // blocks) wait in LDS for the apply phase instead of being read again;
    // each thread reads back only its own slots.
    constexpr int S = fused_lds_accesses(T, false, false);
    __shared__ raw_t<DT, VEC> lx[S > 0 ? S : 1][T];
    StripPos sp = strip_begin(g, c);
#pragma unroll
    for (int k = 0; k < R; ++k) {
        if constexpr (STRIP) {
            keep[k] = load_raw<DT, VEC, kStream>(xz, sp.off + tid);
            strip_next<T>(g, sp);
        } else {
            // Slots past the channel read its first access instead (a line
            // the block reads anyway) and are not used: loads under a
            // condition make the compiler carry the whole buffer through
            // every join, copying it after each load.
            const uint32_t v = tid + k * T;
            keep[k] = load_raw<DT, VEC, kStream>(xz, access_index(g, cbase, v < g.vchan ? v : 0));
        }
    }
    // The per-channel inputs are read once the data loads are out (see
    // bwd_fused_channel), and waited for here, while the data is still on
    // its way (left to the compiler, the loads sink to their first use after
    // the data has arrived, and their round trip is paid then).
    sched_fence();
    const float gamma_c = prm.gamma[c], beta_c = prm.beta[c];
    const float rm_c = prm.running_mean[c], rv_c = prm.running_var[c];
    asm volatile("" ::"s"(gamma_c), "s"(beta_c), "s"(rm_c), "s"(rv_c));
    sched_fence();
    float shift = 0.f, s1 = 0.f, s2 = 0.f;
    uint32_t nacc = 0;
    if (tid < g.vchan) {
        float t[VEC];
        unpack<DT, VEC>(keep[0], t);
        shift = t[0];
    }
    auto accumulate = [&](raw_t<DT, VEC> r) {
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
    // Past the registers: kept in LDS (read once: non-temporal), or read
    // again by the apply phase (through the caches).
    auto accumulate_at = [&](uint64_t i1, uint32_t j) {
        if (S > 0 && j < S) {
            const raw_t<DT, VEC> r = load_raw<DT, VEC, kStream>(xz, i1);
            lx[j][tid] = r;
            accumulate(r);
        } else {
            accumulate(load_raw<DT, VEC, kCached>(xz, i1));
        }
    };
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            accumulate_at(sp.off + tid, k - R);
            strip_next<T>(g, sp);
        }
    } else {
        uint32_t j = 0;
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T, ++j)
            accumulate_at(access_index(g, cbase, v), j);
    }

    double mean, var;
    block_moments<T, CPB>(shift, s1, s2, nacc, VEC, g.inv_m, mean, var);
    uint32_t tid2 = tid;
    opaque(tid2);
#pragma unroll
    for (int k = 0; k < R; ++k) opaque(keep[k]);
    const double invstd = rsqrt_d(var + static_cast<double>(prm.eps));
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
        fwd_fused_apply<DT, VEC, T, R, S, STRIP, FM, true>(xz, g, c, tid2, keep, lx, kk);
    else
        fwd_fused_apply<DT, VEC, T, R, S, STRIP, FM, false>(xz, g, c, tid2, keep, lx, kk);
}

// One block per channel: c = blockIdx.x.  (Giving each XCD a contiguous
// range of channels, rather than every eighth channel as the round-robin
// hand-out of workgroups to the 8 XCDs does, was measured 4% slower.  Blocks
// that loop over several channels were measured slower, both plainly and
// with the next channel prefetched into a second register buffer: the second
// buffer limits a CU to one block, and at that occupancy the per-channel
// reduce-barrier-apply chain costs more than the overlap of one channel's
// stores with the next one's loads gains.)
template <int DT, int VEC, int T, int R, bool STRIP, int FM>
__global__ __launch_bounds__(T) void fwd_fused_kernel(void* __restrict__ xz, Geom g,
                                                      FwdParams prm) {
    fwd_fused_channel<DT, VEC, T, R, STRIP, FM>(xz, g, prm, fused_channel(g, blockIdx.x));
}

// CPB adjacent channels per block, T threads each (channel
// CPB * blockIdx.x + threadIdx.x / T): a block's rows are then CPB times as
// long in memory, and one barrier serves CPB reductions.  Rows of whole
// strips only (they end on a cache line, so no XCD order).
template <int DT, int VEC, int T, int R, bool STRIP, int FM, int CPB>
__global__ __launch_bounds__(T * CPB) void fwd_fused_multi_kernel(void* __restrict__ xz, Geom g,
                                                                  FwdParams prm) {
    // T is a multiple of the wave size, so the channel is uniform per wave.
    const uint32_t c = __builtin_amdgcn_readfirstlane(CPB * blockIdx.x + threadIdx.x / T);
    fwd_fused_channel<DT, VEC, T, R, STRIP, FM, CPB>(xz, g, prm, c);
}

#define IABN_FUSED_CASE(TT, RR)                                                              \
    if (fp.T == TT && fp.R == RR) {                                                           \
        if (fused_strips(g, fp, true))                                                        \
            fwd_fused_kernel<DT, V, TT, RR, true, FM><<<grid, TT, lds, st>>>(xz, g, prm);     \
        else                                                                                  \
            fwd_fused_kernel<DT, V, TT, RR, false, FM><<<grid, TT, lds, st>>>(xz, g, prm);    \
        return true;                                                                          \
    }
// Narrower accesses: rows of odd length rarely hold whole strips, so only
// the general mapping is built.
#define IABN_FUSED_CASE_GENERAL(TT, RR)                                                      \
    if (fp.T == TT && fp.R == RR) {                                                           \
        fwd_fused_kernel<DT, V, TT, RR, false, FM><<<grid, TT, lds, st>>>(xz, g, prm);        \
        return true;                                                                          \
    }

template <int DT, int V, int FM>
bool launch_v(void* xz, const Geom& g, const FusedPlan& fp, const FwdParams& prm, hipStream_t st) {
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedFwdBlocksPerCU);
    if (fp.cpb != 1) {
        if constexpr (V * sizeof(typename Elem<DT>::T) == 16) {
            if (fp.cpb == kFwdMultiChannels && fp.T == 256 && fp.R == 16 &&
                fused_strips(g, fp, true) && g.C % kFwdMultiChannels == 0) {
                fwd_fused_multi_kernel<DT, V, 256, 16, true, FM, kFwdMultiChannels>
                    <<<grid, 256 * kFwdMultiChannels, lds, st>>>(xz, g, prm);
                return true;
            }
        }
        return false;
    }
    if constexpr (V * sizeof(typename Elem<DT>::T) == 16) {
        IABN_FUSED_CASE(256, 4)
        IABN_FUSED_CASE(256, 8)
        IABN_FUSED_CASE(64, 32)
        IABN_FUSED_CASE(256, 16)
        IABN_FUSED_CASE(512, 16)
        IABN_FUSED_CASE(1024, 16)
    } else if constexpr (FM == kFwdInPlace) {
        IABN_FUSED_CASE_GENERAL(256, 4)
        IABN_FUSED_CASE_GENERAL(256, 8)
        IABN_FUSED_CASE_GENERAL(64, 32)
        IABN_FUSED_CASE_GENERAL(512, 4)
        IABN_FUSED_CASE_GENERAL(256, 16)
        IABN_FUSED_CASE_GENERAL(512, 16)
        IABN_FUSED_CASE_GENERAL(1024, 16)
    }
    return false;
}

#undef IABN_FUSED_CASE
#undef IABN_FUSED_CASE_GENERAL

// Elements per access: 16 bytes, or the narrower widths of rows that are not
// a multiple of 16 bytes.
template <int DT, int FM>
bool launch_dt(int vec, void* xz, const Geom& g, const FusedPlan& fp, const FwdParams& prm,
               hipStream_t st) {
    constexpr int W = 16 / static_cast<int>(sizeof(typename Elem<DT>::T));
    if (vec == W) return launch_v<DT, W, FM>(xz, g, fp, prm, st);
    if (vec == W / 2) return launch_v<DT, W / 2, FM>(xz, g, fp, prm, st);
    if constexpr (W / 4 > 1) {
        if (vec == W / 4) return launch_v<DT, W / 4, FM>(xz, g, fp, prm, st);
    }
    if (vec == 1) return launch_v<DT, 1, FM>(xz, g, fp, prm, st);
    return false;
}

template <int FM>
bool launch_fm(int dtype, void* xz, const Geom& g, const FusedPlan& fp, const FwdParams& prm,
               hipStream_t st) {
    return dtype == IABN_F32   ? launch_dt<IABN_F32, FM>(g.vec, xz, g, fp, prm, st)
           : dtype == IABN_F16 ? launch_dt<IABN_F16, FM>(g.vec, xz, g, fp, prm, st)
                               : launch_dt<IABN_BF16, FM>(g.vec, xz, g, fp, prm, st);
}

}  // namespace

bool launch_fwd_fused(int dtype, int fm, void* xz, const Geom& g, const FusedPlan& fp,
                      const FwdParams& prm, hipStream_t st) {
    return fm == kFwdOut    ? launch_fm<kFwdOut>(dtype, xz, g, fp, prm, st)
           : fm == kFwdCkpt ? launch_fm<kFwdCkpt>(dtype, xz, g, fp, prm, st)
                            : launch_fm<kFwdInPlace>(dtype, xz, g, fp, prm, st);
}

}  // namespace iabn_impl
