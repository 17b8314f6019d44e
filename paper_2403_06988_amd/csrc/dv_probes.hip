// Roofline probes (declared in include/dv_probes.h): HBM streaming read and
// write, dependent random 2-byte gathers from global memory (L1/L2) and from
// LDS.  Used by the benchmark to put the hot-path kernels' rates next to what
// the same memory path reaches on its own.
#include "../../include/dv_probes.h"
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;
constexpr int kProbeBlocks = 2048;

__global__ __launch_bounds__(kThreads) void stream_read_kernel(const uint4 *__restrict__ src, size_t n16,
                                                               uint32_t *__restrict__ sink)
{
    constexpr int kU = 8;
    const size_t stride = (size_t)gridDim.x * kThreads;
    uint32_t acc = 0;
    size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + (kU - 1) * stride < n16; i += kU * stride) {
        uint4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            v[u] = src[i + u * stride];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9E3779B9u)  // practically never: keeps the loads alive
        sink[blockIdx.x & 4095] = acc;
}

__global__ __launch_bounds__(kThreads) void stream_write_kernel(uint4 *__restrict__ dst, size_t n16)
{
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += stride) {
        const uint32_t x = (uint32_t)i;
        dst[i] = make_uint4(x, x + 1, x + 2, x + 3);
    }
}

__device__ __forceinline__ uint32_t mix(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7FEB352Du;
    x ^= x >> 15;
    x *= 0x846CA68Bu;
    x ^= x >> 16;
    return x;
}

template <int CHAINS, bool LDS>
__global__ __launch_bounds__(kThreads) void gather_kernel(const uint32_t *__restrict__ table, int entries,
                                                          int steps, uint32_t *__restrict__ sink)
{
    extern __shared__ uint32_t lds_table[];
    const uint32_t *tab = table;
    if (LDS) {
        for (int i = threadIdx.x; i < entries; i += kThreads)
            lds_table[i] = table[i];
        __syncthreads();
        tab = lds_table;
    }
    const uint32_t lane = blockIdx.x * kThreads + threadIdx.x;
    uint32_t idx[CHAINS];
#pragma unroll
    for (int k = 0; k < CHAINS; ++k)
        idx[k] = mix(lane * CHAINS + k) % (uint32_t)entries;
    for (int s = 0; s < steps; ++s)
#pragma unroll
        for (int k = 0; k < CHAINS; ++k)
            idx[k] = min(tab[idx[k]], (uint32_t)entries - 1u);  // stays in bounds
    uint32_t acc = 0;
#pragma unroll
    for (int k = 0; k < CHAINS; ++k)
        acc += idx[k];
    sink[lane] = acc;
}

template <bool LDS>
hipError_t launch_gather(const uint32_t *table, int entries, int lanes, int chains, int steps,
                         uint32_t *sink, hipStream_t stream)
{
    const int grid = lanes / kThreads;
    const size_t lds = LDS ? (size_t)entries * 4 : 0;
    switch (chains) {
    case 1: gather_kernel<1, LDS><<<grid, kThreads, lds, stream>>>(table, entries, steps, sink); break;
    case 2: gather_kernel<2, LDS><<<grid, kThreads, lds, stream>>>(table, entries, steps, sink); break;
    case 4: gather_kernel<4, LDS><<<grid, kThreads, lds, stream>>>(table, entries, steps, sink); break;
    default: gather_kernel<8, LDS><<<grid, kThreads, lds, stream>>>(table, entries, steps, sink); break;
    }
    return hipGetLastError();
}

}  // namespace
}  // namespace dv

extern "C" {

int32_t dvprobe_stream_read(const void *src, size_t n_bytes, uint32_t *sink, void *stream)
{
    if (!src || !sink || n_bytes < 4096 || (n_bytes & 15) || (reinterpret_cast<uintptr_t>(src) & 15))
        return 1;
    dv::stream_read_kernel<<<dv::kProbeBlocks, dv::kThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const uint4 *>(src), n_bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

int32_t dvprobe_stream_write(void *dst, size_t n_bytes, void *stream)
{
    if (!dst || n_bytes < 4096 || (n_bytes & 15) || (reinterpret_cast<uintptr_t>(dst) & 15))
        return 1;
    dv::stream_write_kernel<<<dv::kProbeBlocks, dv::kThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<uint4 *>(dst), n_bytes / 16);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

static bool gather_args_ok(const uint32_t *table, int32_t entries, int32_t lanes, int32_t chains,
                           int32_t steps, const uint32_t *sink, int32_t max_entries)
{
    return table && sink && entries >= 1 && entries <= max_entries && lanes >= 256 && lanes % 256 == 0 &&
           (chains == 1 || chains == 2 || chains == 4 || chains == 8) && steps >= 1;
}

int32_t dvprobe_gather(const uint32_t *table, int32_t table_entries, int32_t lanes, int32_t chains,
                       int32_t steps, uint32_t *sink, void *stream)
{
    if (!gather_args_ok(table, table_entries, lanes, chains, steps, sink, 1 << 24))
        return 1;
    return dv::launch_gather<false>(table, table_entries, lanes, chains, steps, sink,
                                    static_cast<hipStream_t>(stream)) == hipSuccess ? 0 : 6;
}

int32_t dvprobe_lds_gather(const uint32_t *table, int32_t table_entries, int32_t lanes, int32_t chains,
                           int32_t steps, uint32_t *sink, void *stream)
{
    if (!gather_args_ok(table, table_entries, lanes, chains, steps, sink, 32768))
        return 1;
    static const hipError_t attr = [] {
        hipError_t e = hipSuccess;
        for (const void *k : {reinterpret_cast<const void *>(dv::gather_kernel<1, true>),
                              reinterpret_cast<const void *>(dv::gather_kernel<2, true>),
                              reinterpret_cast<const void *>(dv::gather_kernel<4, true>),
                              reinterpret_cast<const void *>(dv::gather_kernel<8, true>)})
            if (e == hipSuccess)
                e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, 32768 * 4);
        return e;
    }();
    if (attr != hipSuccess)
        return 6;
    return dv::launch_gather<true>(table, table_entries, lanes, chains, steps, sink,
                                   static_cast<hipStream_t>(stream)) == hipSuccess ? 0 : 6;
}

}  // extern "C"
