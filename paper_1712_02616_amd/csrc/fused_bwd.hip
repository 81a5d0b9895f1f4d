// The channel-resident backward: one block per channel holds the stored
// tensor(s) and dz in registers (and, in 1024-thread blocks, LDS) from the
// reduction to the apply, so each crosses HBM once in and dx once out (what
// does not fit is read again).  Formulations as in common.h
// (InPlace-ABN I and II from z, standard from x and the signs of z,
// checkpointing from xhat).

#include "fused.h"
#include "launch.h"

namespace iabn_impl {
namespace {

// Backward of one channel per block (sums of dy and dy*w, dgamma, dbeta, dx
// over dz), same arithmetic as bwd_reduce_kernel + bwd_apply_kernel in
// stream.hip.  u is z, x or xhat (see BwdSign).  kBwdFromXZ reads the stored
// z as well but keeps only its signs (one bit per element) for the apply
// phase.
template <int DT, int VEC, int T, int R, bool STRIP, int BM, int CPB = 1>
__device__ __forceinline__ void bwd_fused_channel(const void* __restrict__ u,
                                                  const void* __restrict__ zs,
                                                  void* __restrict__ dzdx, const Geom& g,
                                                  const BwdParams& prm, uint32_t c) {
    constexpr bool XZ = BM == kBwdFromXZ;
    constexpr int NW = XZ ? (R * VEC + 31) / 32 : 1;
    const uint64_t cbase = static_cast<uint64_t>(c) * g.vrow;
    const uint32_t tid = CPB > 1 ? threadIdx.x % T : threadIdx.x;
    const uint32_t nstrips = STRIP ? g.vchan / T : 0;
    // Register-resident accesses non-temporal, the rest cached (see
    // fwd_fused_channel).  kBwdFromXZ first loads z (into the registers x
    // will use) and dz, turns z into sign bits, and only then loads x, so
    // that no more than two tensors' worth of registers is live.
    raw_t<DT, VEC> ku[R], kg[R];
    // The first S accesses per thread past the registers (1024-thread blocks,
    // whose registers hold 11 per tensor) wait in LDS from the reduction to
    // the apply phase instead of being read again; each thread reads back
    // only its own slots.  kBwdFromXZ keeps its third tensor (z) there too.
    constexpr int S = fused_lds_accesses(T, true, XZ);
    __shared__ raw_t<DT, VEC> lu[S > 0 ? S : 1][T], lg[S > 0 ? S : 1][T];
    __shared__ raw_t<DT, VEC> lz[XZ && S > 0 ? S : 1][T];
    uint32_t negm[NW];
#pragma unroll
    for (int q = 0; q < NW; ++q) negm[q] = 0u;
    float gamma_c, beta_c, mean_c;
    double invstd;
    BwdReduceElem<BM> el;
    BwdRecip rc;
    auto channel_inputs = [&]() {
        gamma_c = prm.gamma[c];
        beta_c = prm.beta[c];
        const float var_c = prm.save_var[c];
        mean_c = XZ ? prm.save_mean[c] : 0.f;
        invstd = 1.0 / sqrt(static_cast<double>(var_c) + static_cast<double>(prm.eps));
        el = make_reduce_elem<BM>(prm.slope, gamma_c, beta_c, mean_c, invstd, prm.ii != 0);
        rc = make_recip(gamma_c, prm.slope, g.inv_m);
    };
    if constexpr (XZ) channel_inputs();
    // Index of the thread's k-th resident access (live: within the channel).
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
                ku[k] = load_raw<DT, VEC, kStream>(zs, i1);
                kg[k] = load_raw<DT, VEC, kStream>(dzdx, i1);
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
            if (live) ku[k] = load_raw<DT, VEC, kStream>(u, i1);
        }
    } else {
        // Slots past the channel (general mapping) read the channel's first
        // access instead, a line the block reads anyway, and are never used:
        // loads under a condition can make the compiler carry the whole
        // register buffer through every join, copying it after each load and
        // so waiting for each load in turn.  (The standard block's mode above
        // keeps its conditional loads, which need fewer registers there.)
#pragma unroll
        for (int k = 0; k < R; ++k) {
            bool live;
            const uint64_t i1 = STRIP ? resident_index(k, sp, live)
                                      : access_index(g, cbase, tid + k * T < g.vchan ? tid + k * T : 0);
            ku[k] = load_raw<DT, VEC, kStream>(u, i1);
            kg[k] = load_raw<DT, VEC, kStream>(dzdx, i1);
        }
    }
    // The per-channel inputs, read once the data loads are out: their round
    // trip then overlaps the data's (read before the data loads, every wave
    // waited for them before issuing its own), and they have arrived before
    // the first data does.  (The standard block's backward reads them first:
    // it holds three tensors, and reading them later costs it registers.)
    if constexpr (!XZ) {
        sched_fence();
        channel_inputs();
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
        unpack<DT, VEC>(load_raw<DT, VEC, kCached>(u, i1), tu);
        if constexpr (XZ) unpack<DT, VEC>(load_raw<DT, VEC, kCached>(zs, i1), tz);
        else
#pragma unroll
            for (int e = 0; e < VEC; ++e) tz[e] = 0.f;
        unpack<DT, VEC>(load_raw<DT, VEC, kCached>(dzdx, i1), tg);
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
    // The same for an access kept in LDS (read once: non-temporal).
    auto accumulate_keep = [&](uint64_t i1, uint32_t slot) {
        const raw_t<DT, VEC> ru = load_raw<DT, VEC, kStream>(u, i1);
        const raw_t<DT, VEC> rg = load_raw<DT, VEC, kStream>(dzdx, i1);
        float tu[VEC], tz[VEC], tg[VEC];
        if constexpr (XZ) {
            const raw_t<DT, VEC> rz = load_raw<DT, VEC, kStream>(zs, i1);
            lz[slot][tid] = rz;
            unpack<DT, VEC>(rz, tz);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) tz[e] = 0.f;
        }
        lu[slot][tid] = ru;
        lg[slot][tid] = rg;
        unpack<DT, VEC>(ru, tu);
        unpack<DT, VEC>(rg, tg);
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
            if (S > 0 && k < R + S) accumulate_keep(sp.off + tid, k - R);
            else accumulate(sp.off + tid);
            strip_next<T>(g, sp);
        }
    } else {
        uint32_t j = 0;
#pragma unroll 1
        for (uint32_t v = tid + R * T; v < g.vchan; v += T, ++j) {
            if (S > 0 && j < S) accumulate_keep(access_index(g, cbase, v), j);
            else accumulate(access_index(g, cbase, v));
        }
    }

    double dbeta, sdyw;
    block_sums<T, CPB>(acc_dy, acc_dyw, dbeta, sdyw);
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
    const BwdApplyElem<BM> dx_of = make_apply_elem<BM>(A, sdyw, dbeta, rc, prm.slope, gamma_c,
                                                       beta_c, mean_c, invstd, prm.ii != 0);
    if (tid == 0) {
        prm.dgamma[c] = static_cast<float>(sdyw);
        prm.dbeta[c] = static_cast<float>(dbeta);
    }
    auto emit = [&](raw_t<DT, VEC> ru, raw_t<DT, VEC> rz, raw_t<DT, VEC> rg, uint64_t idx) {
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
    const raw_t<DT, VEC> zero16 = {};
    if constexpr (STRIP) {
#pragma unroll 1
        for (uint32_t k = R; k < nstrips; ++k) {
            const uint64_t i1 = sq.off + tid2;
            if (S > 0 && k < R + S)
                emit(lu[k - R][tid2], XZ ? lz[k - R][tid2] : zero16, lg[k - R][tid2], i1);
            else
                emit(load_raw<DT, VEC, kStream>(u, i1), XZ ? load_raw<DT, VEC, kStream>(zs, i1) : zero16,
                     load_raw<DT, VEC, kStream>(dzdx, i1), i1);
            strip_next<T>(g, sq);
        }
    } else {
        uint32_t j = 0;
#pragma unroll 1
        for (uint32_t v = tid2 + R * T; v < g.vchan; v += T, ++j) {
            const uint64_t i1 = access_index(g, cbase, v);
            if (S > 0 && j < S)
                emit(lu[j][tid2], XZ ? lz[j][tid2] : zero16, lg[j][tid2], i1);
            else
                emit(load_raw<DT, VEC, kStream>(u, i1), XZ ? load_raw<DT, VEC, kStream>(zs, i1) : zero16,
                     load_raw<DT, VEC, kStream>(dzdx, i1), i1);
        }
    }
}

// One block per channel: c = blockIdx.x (see fwd_fused_kernel).
template <int DT, int VEC, int T, int R, bool STRIP, int BM>
__global__ __launch_bounds__(T) void bwd_fused_kernel(const void* __restrict__ u,
                                                      const void* __restrict__ zs,
                                                      void* __restrict__ dzdx, Geom g,
                                                      BwdParams prm) {
    bwd_fused_channel<DT, VEC, T, R, STRIP, BM>(u, zs, dzdx, g, prm, fused_channel(g, blockIdx.x));
}

// CPB adjacent channels per block, T threads each (channel
// CPB * blockIdx.x + threadIdx.x / T; see fwd_fused_multi_kernel).
template <int DT, int VEC, int T, int R, bool STRIP, int BM, int CPB>
__global__ __launch_bounds__(T * CPB) void bwd_fused_multi_kernel(const void* __restrict__ u,
                                                                  const void* __restrict__ zs,
                                                                  void* __restrict__ dzdx, Geom g,
                                                                  BwdParams prm) {
    const uint32_t c = __builtin_amdgcn_readfirstlane(CPB * blockIdx.x + threadIdx.x / T);
    bwd_fused_channel<DT, VEC, T, R, STRIP, BM, CPB>(u, zs, dzdx, g, prm, c);
}

#define IABN_FUSED_CASE(TT, RR)                                                              \
    if (fp.T == TT && fp.R == RR) {                                                           \
        if (fused_strips(g, fp, true))                                                        \
            bwd_fused_kernel<DT, V, TT, RR, true, BM><<<grid, TT, lds, st>>>(u, zs, dzdx, g, prm);  \
        else                                                                                  \
            bwd_fused_kernel<DT, V, TT, RR, false, BM><<<grid, TT, lds, st>>>(u, zs, dzdx, g, prm); \
        return true;                                                                          \
    }
// Narrower accesses: the general mapping only (see fused_fwd.hip).
#define IABN_FUSED_CASE_GENERAL(TT, RR)                                                      \
    if (fp.T == TT && fp.R == RR) {                                                           \
        bwd_fused_kernel<DT, V, TT, RR, false, BM><<<grid, TT, lds, st>>>(u, zs, dzdx, g, prm);     \
        return true;                                                                          \
    }

template <int DT, int V, int BM>
bool launch_v(const void* u, const void* zs, void* dzdx, const Geom& g, const FusedPlan& fp,
              const BwdParams& prm, hipStream_t st) {
    const dim3 grid = fused_grid(g, fp);
    const size_t lds = fused_lds(kFusedBwdBlocksPerCU);
    if (fp.cpb != 1) {
        if constexpr (V * sizeof(typename Elem<DT>::T) == 16) {
            if (fp.T == 256 && fp.R == 16 && fused_strips(g, fp, true) && g.C % fp.cpb == 0) {
                if (fp.cpb == 2) {
                    bwd_fused_multi_kernel<DT, V, 256, 16, true, BM, 2>
                        <<<grid, 512, lds, st>>>(u, zs, dzdx, g, prm);
                    return true;
                }
                if (fp.cpb == 3) {
                    bwd_fused_multi_kernel<DT, V, 256, 16, true, BM, 3>
                        <<<grid, 768, lds, st>>>(u, zs, dzdx, g, prm);
                    return true;
                }
            }
        }
        return false;
    }
    if constexpr (V * sizeof(typename Elem<DT>::T) == 16) {
        IABN_FUSED_CASE(256, 4)
        IABN_FUSED_CASE(256, 8)
        IABN_FUSED_CASE(256, 16)
        IABN_FUSED_CASE(512, 16)
        IABN_FUSED_CASE(1024, 11)
    } else if constexpr (BM == kBwdFromZ) {
        IABN_FUSED_CASE_GENERAL(256, 4)
        IABN_FUSED_CASE_GENERAL(256, 8)
        IABN_FUSED_CASE_GENERAL(512, 4)
        IABN_FUSED_CASE_GENERAL(256, 16)
        IABN_FUSED_CASE_GENERAL(512, 16)
        IABN_FUSED_CASE_GENERAL(1024, 16)
    }
    return false;
}

#undef IABN_FUSED_CASE
#undef IABN_FUSED_CASE_GENERAL

template <int DT, int BM>
bool launch_dt(int vec, const void* u, const void* zs, void* dzdx, const Geom& g,
               const FusedPlan& fp, const BwdParams& prm, hipStream_t st) {
    constexpr int W = 16 / static_cast<int>(sizeof(typename Elem<DT>::T));
    if (vec == W) return launch_v<DT, W, BM>(u, zs, dzdx, g, fp, prm, st);
    if (vec == W / 2) return launch_v<DT, W / 2, BM>(u, zs, dzdx, g, fp, prm, st);
    if constexpr (W / 4 > 1) {
        if (vec == W / 4) return launch_v<DT, W / 4, BM>(u, zs, dzdx, g, fp, prm, st);
    }
    if (vec == 1) return launch_v<DT, 1, BM>(u, zs, dzdx, g, fp, prm, st);
    return false;
}

template <int BM>
bool launch_bm(int dtype, const void* u, const void* zs, void* dzdx, const Geom& g,
               const FusedPlan& fp, const BwdParams& prm, hipStream_t st) {
    return dtype == IABN_F32   ? launch_dt<IABN_F32, BM>(g.vec, u, zs, dzdx, g, fp, prm, st)
           : dtype == IABN_F16 ? launch_dt<IABN_F16, BM>(g.vec, u, zs, dzdx, g, fp, prm, st)
                               : launch_dt<IABN_BF16, BM>(g.vec, u, zs, dzdx, g, fp, prm, st);
}

}  // namespace

bool launch_bwd_fused(int dtype, int bm, const void* u, const void* zs, void* dzdx, const Geom& g,
                      const FusedPlan& fp, const BwdParams& prm, hipStream_t st) {
    return bm == kBwdFromXZ     ? launch_bm<kBwdFromXZ>(dtype, u, zs, dzdx, g, fp, prm, st)
           : bm == kBwdFromXhat ? launch_bm<kBwdFromXhat>(dtype, u, zs, dzdx, g, fp, prm, st)
                                : launch_bm<kBwdFromZ>(dtype, u, zs, dzdx, g, fp, prm, st);
}

}  // namespace iabn_impl
