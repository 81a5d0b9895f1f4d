// Host-side launchers of libiabn's kernels, one per kernel family, and the
// planning of the channel-resident (fused) kernels.  Each launcher picks the
// template instance for the storage type, access width and mode and enqueues
// it on the stream; it neither validates (the C ABI in api.hip does that
// before any launch) nor reports launch errors (the caller reads
// hipGetLastError).
#pragma once

#include "common.h"

namespace iabn_impl {

// ---- streaming kernels (stream.hip)

// vec: elements per access (Geom::vec).
void launch_fwd_stats(int dtype, int vec, const void* x, const Geom& g, Partial* part,
                      hipStream_t st);
// train = false is inference (in place); otherwise fm is the output mode.
void launch_fwd_apply(int dtype, int vec, void* xz, const Geom& g, const Partial* part,
                      const FwdParams& prm, bool train, int fm, hipStream_t st);
void launch_bwd_reduce(int dtype, int vec, const void* u, const void* zs, const void* dz,
                       const Geom& g, const BwdParams& prm, int bm, Partial* part, hipStream_t st);
void launch_bwd_apply(int dtype, int vec, const void* u, const void* zs, void* dzdx,
                      const Geom& g, const Partial* part, const BwdParams& prm, int bm,
                      hipStream_t st);
void launch_recompute(int dtype, int vec, const void* xhat, void* z, const Geom& g,
                      const float* gamma, const float* beta, float slope, hipStream_t st);

// ---- channel-resident kernels (fused_fwd.hip, fused_bwd.hip)

// Used when every channel gets a block of its own and at least one block per
// CU (C >= kFusedMinChannels): on the 16-byte path for every entry point,
// on the narrower paths for InPlace-ABN's own forward and backward.  With
// fewer channels than CUs, a block per channel still beats the two passes of
// the streaming kernels while the channel fits the largest block's registers
// (or, from 128 channels, up to twice that) and enough CUs get a channel:
// measured over C = 64..256 and channels of 4K..64K accesses, from C = 64
// for the forward (C = 128, 16K accesses: 15 us against 25; 25K fp32
// accesses: 25 against 31) and from C = 96 for the backward (C = 128, 16K
// accesses: 27 us against 33); with larger channels, or fewer, the
// streaming kernels are faster.
constexpr int64_t kFusedMinChannels = 256;
constexpr int64_t kFusedFewChannelsFwd = 64;
constexpr int64_t kFusedFewChannelsBwd = 96;
constexpr int64_t kFusedFewChannelsWide = 128;
constexpr int64_t kFusedFewChannelsMaxAccesses = 16384;

inline bool fused_few_channels_ok(int64_t C, uint32_t vchan, bool backward) {
    if (C < (backward ? kFusedFewChannelsBwd : kFusedFewChannelsFwd)) return false;
    const int64_t cap = kFusedFewChannelsMaxAccesses * (C >= kFusedFewChannelsWide ? 2 : 1);
    return static_cast<int64_t>(vchan) <= cap;
}

struct FusedPlan {
    int T;        // threads per channel
    int R;        // accesses per thread held in registers (per tensor)
    int cpb = 1;  // channels per block (T * cpb threads)
};

inline dim3 fused_grid(const Geom& g, const FusedPlan& fp) { return dim3(g.C / fp.cpb); }

// The forward's (256, 16) rung on rows of whole strips takes two adjacent
// channels per 512-thread block (each with its own 256 threads, one block
// barrier for both reductions) from 1024 up to 2047 channels: measured
// (8, C, 64x64) fp16, C = 1024 25.1 -> 24.2 us and C = 1536 38.5 -> 37.0
// (the backbone sweep's C = 1024 layers 24.8 -> 23.3), but C = 768 18.1 ->
// 20.6 and C = 2048 50.5 -> 51.3, and four channels per block no better.
constexpr int kFwdMultiChannels = 2;
constexpr int64_t kFwdMultiMinChannels = 1024;
constexpr int64_t kFwdMultiMaxChannels = 2047;

// The backward's (256, 16) rung (166 registers: up to 3 waves per SIMD)
// takes several adjacent channels per block where the launch is then one
// round of one block on every CU, C = 512 (two channels per 512-thread
// block) or 768 (three per 768-thread block) on the 256 CUs, and two per
// block for C = 1024 (two rounds): (8, C, 64x64) fp16, C = 512 20.6 -> 18.1
// us, C = 768 27.3 -> 25.7, C = 1024 37.6 -> 37.1 (the backbone sweep's
// C = 1024 layers 37.6 -> 36.8).  Where it adds rounds or leaves CUs with
// unequal shares it is slower: two per block C = 768 27.8 -> 31.2, 1280
// 44.6 -> 49.2, 1536 53.2 -> 56.7, 2048 72.4 -> 81.7; three per block
// C = 1536 53.7 -> 56.3.
constexpr int64_t kCUs = 256;

inline int bwd_channels_per_block(int64_t C) {
    return C == 2 * kCUs ? 2 : C == 3 * kCUs ? 3 : C == 4 * kCUs ? 2 : 1;
}

// Resident blocks per CU of a fused launch (0: as many as registers allow).
// Fewer resident blocks run the channels in several rounds, so the loads of
// a later round overlap the stores of an earlier one instead of every block
// reading, then every block writing.  The cap is applied by reserving LDS.
constexpr int kFusedFwdBlocksPerCU = 0;
constexpr int kFusedBwdBlocksPerCU = 0;
constexpr size_t kLdsPerCU = 160 * 1024;

inline size_t fused_lds(int blocks_per_cu) {
    if (blocks_per_cu <= 0) return 0;
    return kLdsPerCU / blocks_per_cu - 2048;  // leaves room for the kernels' own reduction buffers
}

// A launch's dynamic LDS is at most 64 KB (the runtime rejects a larger
// request and aborts the queue), so a cap takes at least 3 blocks per CU;
// and the 1024-thread kernels, whose static LDS holds up to 144 KB of
// accesses, leave no room for a cap's reservation at all.
constexpr bool cap_ok(int blocks_per_cu) {
    return blocks_per_cu == 0 || kLdsPerCU / blocks_per_cu - 2048 <= 65536;
}
static_assert(cap_ok(kFusedFwdBlocksPerCU) && cap_ok(kFusedBwdBlocksPerCU),
              "a residency cap needs more than 64 KB of dynamic LDS per block");
static_assert(kFusedFwdBlocksPerCU == 0 && kFusedBwdBlocksPerCU == 0,
              "a residency cap does not fit beside the LDS residency of the 1024-thread kernels");

// Candidate (T, R) in order of preference (each one has a kernel built in
// launch_fwd_fused / launch_bwd_fused): the first whose threads hold the
// whole channel is used; larger channels take the last entry, which keeps
// part of the remainder in LDS and reads the rest again.  The backward holds
// two tensors, so its largest blocks keep
// 11 accesses per thread of each (the most that fits a 1024-thread block's
// 128 registers per thread in every mode without spilling; 11 instead of 8
// took the 256-channel layers of the backbone sweep from 41 to 38 us).
// Channels of 1025-2048 accesses take (256, 8): 5% faster than (512, 4) on
// the forward of 16x2048x28x28 bf16, the same on its backward.
// Fused kernels use strip addressing where the shape allows it.
constexpr bool kUseStrips = true;

// Accesses per thread past the registers that the 1024-thread blocks keep in
// LDS (160 KB per CU, and such a block has the CU to itself): the forward 9
// of x (144 KB), the backward 4 of each of its two tensors (128 KB; the
// standard block's backward, which reads three, 3 of each: 144 KB).  Over
// the backbone sweep's C = 256 layers this cut the backward from 39.3 to
// 37.4 us (5 of 16 strips past the registers), on (32, 256, 56x56) fp32
// from 67.0 to 61.9.
constexpr int kFwdLdsAccesses = 9;
constexpr int kBwdLdsAccesses = 4;
constexpr int kBwdLdsAccessesXZ = 3;

// LDS slots per thread of a channel-resident kernel with T threads (xz: the
// standard block's backward, which keeps three tensors).
constexpr int fused_lds_accesses(int T, bool backward, bool xz) {
    return T != 1024 ? 0 : !backward ? kFwdLdsAccesses : xz ? kBwdLdsAccessesXZ : kBwdLdsAccesses;
}

constexpr FusedPlan kFwdLadder[] = {{256, 4}, {256, 8}, {256, 16}, {512, 16}, {1024, 16}};
constexpr FusedPlan kBwdLadder[] = {{256, 4}, {256, 8}, {256, 16}, {512, 16}, {1024, 11}};

// Accesses narrower than 16 bytes (rows whose length is not a multiple of
// 16 bytes: 14x14 or 7x7 maps in fp16, for instance) hold the same
// elements in more, smaller registers; one ladder serves both directions.
// Built for InPlace-ABN's own forward and backward only (the comparison
// blocks take the streaming kernels on such shapes).  (One wave per channel
// for the small channels of 7x7 maps measured no faster than these rungs.)
constexpr FusedPlan kNarrowLadder[] = {{256, 4}, {256, 8}, {256, 16}, {512, 16}, {1024, 16}};
// With at most one channel per CU, channels of 1025-2048 narrow accesses take
// 512-thread blocks instead (2-5% faster on 14x14 and 7x7 fp16 maps with 128
// to 256 channels; 3-7% slower with 512).
constexpr FusedPlan kNarrowLadderFew[] = {{256, 4}, {512, 4}, {256, 16}, {512, 16}, {1024, 16}};
static_assert(sizeof kNarrowLadderFew == sizeof kNarrowLadder, "the narrow ladders have one length");

// With at least two channels per SIMD (2048 on 1024 SIMDs), the forward's
// channels of 1025-2048 accesses take one wave each instead of (256, 8):
// each wave then reduces and writes its channel without waiting for other
// waves at a block barrier.  Measured: (16, 2048, 28x28) bf16 forward 19.7 us
// against 22.2, (8, 2048, 28x28) fp32 18.1 against 21.1, (32, 2048, 14x14)
// fp16 (8-byte accesses) 13.3 against 14.0; with fewer channels it is
// slower ((16, 1024, 28x28) fp16 12.6 against 11.0, (8, 300, 32x64) fp16
// 9.8 against 6.8).  The backward's two tensors do not fit one wave's
// registers ((128, 16) measured slower than (256, 8) there).
constexpr int64_t kOneWaveMinChannels = 2048;
constexpr FusedPlan kOneWaveRung = {64, 32};

// elem_bytes: storage size; narrow_ok: whether this entry point has narrow
// channel-resident kernels.
inline bool plan_fused(int64_t C, const Geom& g, int elem_bytes, bool backward, bool narrow_ok,
                       FusedPlan* out) {
    if (C < kFusedMinChannels && !fused_few_channels_ok(C, g.vchan, backward)) return false;
    const bool wide = static_cast<int>(g.vec) * elem_bytes == 16;
    if (!wide && !narrow_ok) return false;
    const FusedPlan* ladder = !wide ? (C <= kFusedMinChannels ? kNarrowLadderFew : kNarrowLadder)
                              : backward ? kBwdLadder
                                         : kFwdLadder;
    const int n = !wide      ? int(sizeof kNarrowLadder / sizeof kNarrowLadder[0])
                  : backward ? int(sizeof kBwdLadder / sizeof kBwdLadder[0])
                             : int(sizeof kFwdLadder / sizeof kFwdLadder[0]);
    const int64_t A = g.vchan;
    for (int i = 0; i < n; ++i) {
        if (A <= static_cast<int64_t>(ladder[i].T) * ladder[i].R || i == n - 1) {
            *out = ladder[i];
            if (!backward && C >= kOneWaveMinChannels && out->T == 256 && out->R == 8)
                *out = kOneWaveRung;
            if (!backward && wide && C >= kFwdMultiMinChannels && C <= kFwdMultiMaxChannels &&
                C % kFwdMultiChannels == 0 && !g.xcd_order && out->T == 256 && out->R == 16 &&
                g.vrow % 256 == 0 && g.vchan / 256 >= 16)
                out->cpb = kFwdMultiChannels;
            if (backward && wide && !g.xcd_order && out->T == 256 && out->R == 16 &&
                g.vrow % 256 == 0 && g.vchan / 256 >= 16)
                out->cpb = bwd_channels_per_block(C);
            return true;
        }
    }
    return false;
}

// Strip addressing: 16-byte accesses whose rows hold whole T-wide strips,
// at least R of them per channel.
inline bool fused_strips(const Geom& g, const FusedPlan& fp, bool wide) {
    return wide && kUseStrips && g.vrow % static_cast<uint32_t>(fp.T) == 0 &&
           g.vchan / static_cast<uint32_t>(fp.T) >= static_cast<uint32_t>(fp.R);
}

// False if no kernel is built for the plan's (T, R) (a planning bug).
bool launch_fwd_fused(int dtype, int fm, void* xz, const Geom& g, const FusedPlan& fp,
                      const FwdParams& prm, hipStream_t st);
bool launch_bwd_fused(int dtype, int bm, const void* u, const void* zs, void* dzdx, const Geom& g,
                      const FusedPlan& fp, const BwdParams& prm, hipStream_t st);

}  // namespace iabn_impl
