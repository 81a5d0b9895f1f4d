// Bandwidth probes for the benchmark: the HBM rate this part sustains for
// the access mixes of libiabn's kernels, over the same buffers and working
// set, with no arithmetic.  Not part of libiabn (built into a library of its
// own, libiabn_probe.so); the benchmark reports its kernels' rates against
// these measured ceilings as well as against the 8 TB/s peak.
//
// Every access is 16 bytes and non-temporal, as in the channel-resident
// kernels.  Mixes (a and b are two tensors of `bytes` each):
//   IABN_PROBE_READ        read a and b
//   IABN_PROBE_RW          read a, write a in place (the forward's 1:1 mix)
//   IABN_PROBE_RMW         read a and b, write b in place (the backward's 2:1)
//   IABN_PROBE_RES_RW      as IABN_PROBE_RW in the channel-resident pattern:
//                          a block loads 16 accesses per thread, waits at a
//                          block barrier, then stores them
//   IABN_PROBE_RES_RMW     as IABN_PROBE_RMW in the channel-resident pattern
// The streaming mixes are grid-stride loops with 4 accesses per tensor in
// flight per thread over `grid` blocks of 256 threads; the resident ones
// take one block per 16 x 256 accesses.  Written values equal the values
// read (key = 0), so a probe leaves its buffers as it found them.

#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

namespace {

typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int kProbeThreads = 256;
constexpr int kInFlight = 4;
constexpr int kResident = 16;

enum { kRead = 0, kRw = 1, kRmw = 2, kResRw = 3, kResRmw = 4 };

__device__ __forceinline__ u4 ld(const u4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st(u4* p, u4 v) { __builtin_nontemporal_store(v, p); }

template <int MIX>
__global__ __launch_bounds__(kProbeThreads) void stream_probe(u4* __restrict__ a,
                                                              u4* __restrict__ b, uint64_t n,
                                                              uint32_t key,
                                                              uint32_t* __restrict__ sink) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kProbeThreads;
    uint32_t acc = 0;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * kProbeThreads + threadIdx.x; i < n;
         i += kInFlight * stride) {
        u4 va[kInFlight], vb[kInFlight];
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) {
            const uint64_t j = i + u * stride;
            if (j < n) {
                va[u] = ld(a + j);
                if (MIX != kRw) vb[u] = ld(b + j);
            }
        }
#pragma unroll
        for (int u = 0; u < kInFlight; ++u) {
            const uint64_t j = i + u * stride;
            if (j < n) {
                if (MIX == kRead) acc ^= va[u].x ^ vb[u].w;
                else if (MIX == kRw) st(a + j, va[u] ^ key);
                else st(b + j, vb[u] + (va[u] & key));
            }
        }
    }
    // Keeps the read-only loads alive; the stored value is never compared.
    if (MIX == kRead && acc == key + 0x9e3779b9u) sink[0] = acc;
}

template <int MIX>
__global__ __launch_bounds__(kProbeThreads) void resident_probe(u4* __restrict__ a,
                                                                u4* __restrict__ b, uint64_t n,
                                                                uint32_t key) {
    const uint64_t base = static_cast<uint64_t>(blockIdx.x) * (kResident * kProbeThreads);
    u4 va[kResident], vb[kResident];
#pragma unroll
    for (int k = 0; k < kResident; ++k) {
        const uint64_t j = base + threadIdx.x + k * kProbeThreads;
        if (j < n) {
            va[k] = ld(a + j);
            if (MIX == kResRmw) vb[k] = ld(b + j);
        }
    }
    // One block-wide combine, as the channel-resident kernels' reduction.
    __shared__ uint32_t red[kProbeThreads / 64];
    uint32_t acc = 0;
#pragma unroll
    for (int k = 0; k < kResident; ++k) acc ^= va[k].x;
    if ((threadIdx.x & 63) == 0) red[threadIdx.x / 64] = acc;
    __syncthreads();
    const uint32_t add = (red[0] ^ red[1] ^ red[2] ^ red[3]) & key;
#pragma unroll
    for (int k = 0; k < kResident; ++k) {
        const uint64_t j = base + threadIdx.x + k * kProbeThreads;
        if (j < n) {
            if (MIX == kResRw) st(a + j, va[k] ^ add);
            else st(b + j, vb[k] + (va[k] & key) + add);
        }
    }
}

}  // namespace

extern "C" {

// Enqueues one probe over `bytes` bytes of a (and b) on `stream`.  bytes must
// be a positive multiple of 16 and a, b 16-byte aligned device pointers
// (b and sink are unused by the mixes that do not name them); grid is the
// block count of the streaming mixes (1..2^20).  key = 0 leaves the data
// unchanged.  Returns 0, or 1 for invalid arguments, 2 if the launch failed.
int iabn_probe_launch(int mix, void* a, void* b, size_t bytes, int grid, unsigned key,
                      void* sink, void* stream) {
    if (bytes == 0 || bytes % 16 != 0 || a == nullptr) return 1;
    if ((reinterpret_cast<uintptr_t>(a) | reinterpret_cast<uintptr_t>(b)) & 15u) return 1;
    if (mix != kRw && mix != kResRw && b == nullptr) return 1;
    if (mix == kRead && sink == nullptr) return 1;
    if (mix < kRead || mix > kResRmw) return 1;
    if (grid < 1 || grid > (1 << 20)) return 1;
    const uint64_t n = bytes / 16;
    u4* pa = static_cast<u4*>(a);
    u4* pb = static_cast<u4*>(b);
    uint32_t* ps = static_cast<uint32_t*>(sink);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    const dim3 res_grid(static_cast<uint32_t>((n + kResident * kProbeThreads - 1) /
                                              (kResident * kProbeThreads)));
    switch (mix) {
        case kRead: stream_probe<kRead><<<grid, kProbeThreads, 0, st>>>(pa, pb, n, key, ps); break;
        case kRw: stream_probe<kRw><<<grid, kProbeThreads, 0, st>>>(pa, pb, n, key, ps); break;
        case kRmw: stream_probe<kRmw><<<grid, kProbeThreads, 0, st>>>(pa, pb, n, key, ps); break;
        case kResRw: resident_probe<kResRw><<<res_grid, kProbeThreads, 0, st>>>(pa, pb, n, key); break;
        default: resident_probe<kResRmw><<<res_grid, kProbeThreads, 0, st>>>(pa, pb, n, key); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
