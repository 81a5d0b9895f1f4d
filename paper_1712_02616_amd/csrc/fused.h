// Device helpers of the channel-resident (fused) kernels: raw access
// registers, the block-level reductions of a channel, strip addressing, and
// the optimiser barriers that keep the register-resident loops at their
// register budget.
#pragma once

#include <type_traits>

#include "common.h"

namespace iabn_impl {

// One block owns a whole channel and keeps the first R of each thread's
// accesses in registers between the reduction and the apply phase,
// so those bytes cross HBM once on the way in and once on the way out (the
// forward reads x and writes z; the backward reads z and dz and writes dx).
// Accesses beyond R (channels larger than the block's registers) wait in LDS
// where 1024-thread blocks have room, and are read again in the apply phase
// otherwise.  Thread t handles accesses t, t + T, t + 2T, ...
// of its channel, so a wave touches consecutive vectors.  The only
// synchronisation is the block barrier around the channel's reduction.

// One access of VEC elements of storage type DT, kept raw (undecoded) in
// registers: 16 bytes as 4 dwords, 8 bytes as one 64-bit value (a 2-dword
// vector made the compiler shuffle registers through AGPRs), 4 bytes as one
// dword, and a 2-byte element in the low half of a dword.
template <int DT, int VEC>
struct RawAccess {
    using T = typename Elem<DT>::T;
    static constexpr int kBytes = VEC * static_cast<int>(sizeof(T));
    typedef uint32_t v4 __attribute__((ext_vector_type(4)));
    // What is held in registers.
    using reg = typename std::conditional<
        kBytes == 16, v4, typename std::conditional<kBytes == 8, uint64_t, uint32_t>::type>::type;
    // What is read from and written to memory.
    using mem = typename std::conditional<kBytes == 2, uint16_t, reg>::type;
};

template <int DT, int VEC>
using raw_t = typename RawAccess<DT, VEC>::reg;

// Hide a value from the optimiser (an empty asm that "may change" it).  Used
// after the reduction barrier so that the apply phase keeps only the raw
// registers alive and converts them again, instead of keeping the larger
// fp32 values (and 64-bit addresses) from the first phase.
template <typename V>
__device__ __forceinline__ void opaque(V& v) {
    asm volatile("" : "+v"(v));
}

// Keep the scheduler from interleaving the per-access steps of the register-
// resident loops: interleaving them only raises register pressure (the loads
// are already all in flight), and past the block's register budget it spills.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

template <int DT, int VEC, int HINT>
__device__ __forceinline__ raw_t<DT, VEC> load_raw(const void* __restrict__ base, uint64_t idx) {
    using mem = typename RawAccess<DT, VEC>::mem;
    const mem* p = static_cast<const mem*>(base) + idx;
    return static_cast<raw_t<DT, VEC>>(HINT == kStream ? __builtin_nontemporal_load(p) : *p);
}

template <int DT, int VEC>
__device__ __forceinline__ void unpack(raw_t<DT, VEC> r, float (&v)[VEC]) {
    using T = typename Elem<DT>::T;
    if constexpr (VEC == 1) {
        v[0] = static_cast<float>(
            __builtin_bit_cast(T, static_cast<typename RawAccess<DT, VEC>::mem>(r)));
    } else {
        typedef T vt __attribute__((ext_vector_type(VEC)));
        typedef float vf __attribute__((ext_vector_type(VEC)));
        const vf f = __builtin_convertvector(__builtin_bit_cast(vt, r), vf);
#pragma unroll
        for (int k = 0; k < VEC; ++k) v[k] = f[k];
    }
}

// Per-wave (shift, s1, s2, n) of a block, combined by wave 0 in a fixed
// order into the channel's mean and biased variance.
// Per-wave (shift, s1, s2, n) of a block, combined into the channel's mean
// and biased variance.  Each wave writes its partial to LDS; after the one
// barrier every wave combines all of them itself, in the same fixed order,
// so all waves hold the same result without a second barrier.  inv_m is
// 1/m for the block's m values (formed off the critical path).
// With CPB channels per block (CPB groups of T threads), each group's waves
// combine only their own group's partials.
template <int T, int CPB = 1>
__device__ __forceinline__ void block_moments(float shift, float s1, float s2, uint32_t nacc,
                                              uint32_t vec, double inv_m, double& mean,
                                              double& var) {
    constexpr int W = T / kWave;
    __shared__ double red[CPB * W][4];
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
    const uint32_t w0 = CPB > 1 ? (threadIdx.x / T) * W : 0;
    const double kref = red[w0][0];
    double t1 = 0.0, t2 = 0.0;
    if (lane_id() < W) {
        double tn = red[w0 + lane_id()][3];
        t1 = red[w0 + lane_id()][1];
        t2 = red[w0 + lane_id()][2];
        reshift(t1, t2, tn, red[w0 + lane_id()][0], kref);
    }
    t1 = wave_sum(t1);
    t2 = wave_sum(t2);
    mean = kref + t1 * inv_m;
    var = fmax(t2 - t1 * t1 * inv_m, 0.0) * inv_m;
}

// Two sums over a block, returned in every thread (one barrier, as above;
// with CPB channels per block, over the thread's group of T threads).
template <int T, int CPB = 1>
__device__ __forceinline__ void block_sums(double a, double b, double& sa, double& sb) {
    constexpr int W = T / kWave;
    __shared__ double red[CPB * W][2];
    a = wave_sum(a);
    b = wave_sum(b);
    const uint32_t wave = threadIdx.x / kWave;
    if (lane_id() == 0) {
        red[wave][0] = a;
        red[wave][1] = b;
    }
    __syncthreads();
    const uint32_t w0 = CPB > 1 ? (threadIdx.x / T) * W : 0;
    double t1 = lane_id() < W ? red[w0 + lane_id()][0] : 0.0;
    double t2 = lane_id() < W ? red[w0 + lane_id()][1] : 0.0;
    sa = wave_sum(t1);
    sb = wave_sum(t2);
}

// Where each row of a channel holds a whole number of T-wide strips of
// accesses (vrow % T == 0) and the channel has at least R strips,
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

// The channel of block b of a channel-resident launch.  The hardware hands
// consecutive workgroups to the 8 XCDs in turn, so in block order
// neighbouring channels run on different XCDs, each with its own L2.  Where
// rows do not end on a 128-byte line, a line at the end of one channel's row
// also holds the start of the next channel's row and is then fetched once
// per XCD; xcd_order gives each XCD a contiguous range of channels instead
// (C = 8q + r: XCD x takes q channels, plus one if x < r), so both halves of
// such lines are read through one L2.  Measured: 4-5% on 16x2048x28x28 bf16,
// 9-19% on 14x14 and 7x7 fp16 maps, but 3-11% slower on rows of whole lines
// (the backbone sweep), which keep block order.

__device__ __forceinline__ uint32_t fused_channel(const Geom& g, uint32_t b) {
    if (!g.xcd_order) return b;
    const uint32_t x = b % kXcds, j = b / kXcds;
    return x * g.xcd_q + min(x, g.xcd_r) + j;
}

// The leaky ReLU as max(y, a*y) for a <= 1 and min(y, a*y) for a > 1: two
// instructions, and the same value as the definition's branch (including
// y = -0, which stays -0).
template <bool SMALL_SLOPE>
__device__ __forceinline__ float leaky(float y, float a) {
    return SMALL_SLOPE ? fmaxf(y, a * y) : fminf(y, a * y);
}

}  // namespace iabn_impl
