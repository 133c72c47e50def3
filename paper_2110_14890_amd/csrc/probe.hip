// probe.hip -- random-read ceiling of the device, for the benchmark.
//
// The sampler's reads are single 4-byte words at random places of large
// tables, and every one that misses L2 moves a whole line.  This kernel
// performs the same kind of read as fast as the device allows (eight
// independent reads in flight per lane, no dependence between them), so its
// rate is the practical ceiling the sampler's gathers are measured against.
#include <hip/hip_runtime.h>

#include "smore_internal.h"

namespace smore {
namespace {

constexpr int PROBE_WG = 256;
constexpr int PROBE_INFLIGHT = 8;
constexpr int PROBE_ITERS = 8;

__device__ __forceinline__ uint32_t probe_mix(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7FEB352Du;
    x ^= x >> 15;
    x *= 0x846CA68Bu;
    x ^= x >> 16;
    return x;
}

// Thread t reads PROBE_ITERS x PROBE_INFLIGHT words, each the first word of
// a line chosen by a hash of (t, read index) among `lines` 64-byte lines
// (lines is a power of two that fits the table).
__global__ __launch_bounds__(PROBE_WG) void k_gather_probe(const uint32_t* __restrict__ table,
                                                           uint32_t line_mask, int64_t threads,
                                                           uint32_t* __restrict__ sink)
{
    const int64_t t = (int64_t)blockIdx.x * PROBE_WG + threadIdx.x;
    if (t >= threads) return;
    uint32_t acc = 0;
    for (int i = 0; i < PROBE_ITERS; ++i) {
        uint32_t v[PROBE_INFLIGHT];
#pragma unroll
        for (int u = 0; u < PROBE_INFLIGHT; ++u) {
            const uint32_t h = probe_mix((uint32_t)t * 7919u + (uint32_t)(i * PROBE_INFLIGHT + u) * 104729u);
            v[u] = table[(size_t)(h & line_mask) * 16];
        }
#pragma unroll
        for (int u = 0; u < PROBE_INFLIGHT; ++u) acc ^= v[u];
    }
    sink[t] = acc;
}

}  // namespace

int64_t gather_probe_threads(int64_t n_reads)
{
    const int64_t per = (int64_t)PROBE_INFLIGHT * PROBE_ITERS;
    return (n_reads + per - 1) / per;
}

int launch_gather_probe(const void* table, int64_t table_bytes, int64_t n_reads, uint32_t* sink,
                        hipStream_t st, const char** err)
{
    uint64_t lines = 1;
    while (lines * 2 * 64 <= (uint64_t)table_bytes && lines * 2 <= (1ull << 32)) lines *= 2;
    const int64_t threads = gather_probe_threads(n_reads);
    const int64_t blocks = (threads + PROBE_WG - 1) / PROBE_WG;
    k_gather_probe<<<(unsigned)blocks, PROBE_WG, 0, st>>>((const uint32_t*)table,
                                                           (uint32_t)(lines - 1), threads, sink);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) { *err = hipGetErrorString(e); return SMORE_E_HIP; }
    return SMORE_OK;
}

}  // namespace smore
