// Roofline probes (libdv_probes.so, declared in include/dv_probes.h): HBM
// streaming read and write, dependent random 2-byte gathers from global
// memory (L1/L2) and from LDS, and the floors of the bf16 masked step at its
// own launch shape.  Used by the benchmark to put the hot-path kernels'
// rates next to what the same memory path reaches on its own.  Measurement
// code: not part of libdv.so.
#include "../../include/dv_probes.h"
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;

// HBM streaming: each block reads (writes) one contiguous chunk of the
// buffer, four 16-byte vectors per lane in flight.  Against a grid-stride
// loop over the whole buffer (2,048 blocks of 256 lanes, cached loads) this
// form reaches about 7.2 TB/s of reads instead of 5.5, and 6.0-6.2 TB/s of
// writes instead of 5.0 (2 GiB buffers, one MI355X): a sweep over chunked
// and grid-stride forms, 256 to 4,096 blocks of 256 to 1,024 lanes, 1 to 8
// vectors in flight, cached and non-temporal, found these among the best.
constexpr int kStreamThreads = 512;
constexpr int kStreamU = 4;
constexpr int kStreamReadBlocks = 512;
constexpr int kStreamWriteBlocks = 2048;

typedef unsigned int stream_u32x4 __attribute__((ext_vector_type(4)));

// [begin, end) of block `blk`'s chunk of n16 vectors over `blocks` blocks
__device__ __forceinline__ void stream_chunk(size_t n16, int blocks, int blk, size_t &begin, size_t &end)
{
    const size_t per = n16 / (size_t)blocks, extra = n16 % (size_t)blocks;
    begin = (size_t)blk * per + ((size_t)blk < extra ? (size_t)blk : extra);
    end = begin + per + ((size_t)blk < extra ? 1 : 0);
}

__global__ __launch_bounds__(kStreamThreads) void stream_read_kernel(const uint4 *__restrict__ src, size_t n16,
                                                                     uint32_t *__restrict__ sink)
{
    const stream_u32x4 *p = reinterpret_cast<const stream_u32x4 *>(src);
    size_t begin, end;
    stream_chunk(n16, (int)gridDim.x, (int)blockIdx.x, begin, end);
    uint32_t acc = 0;
    size_t i = begin + threadIdx.x;
    for (; i + (size_t)(kStreamU - 1) * kStreamThreads < end; i += (size_t)kStreamU * kStreamThreads) {
        stream_u32x4 v[kStreamU];
#pragma unroll
        for (int u = 0; u < kStreamU; ++u)
            v[u] = __builtin_nontemporal_load(p + i + (size_t)u * kStreamThreads);
#pragma unroll
        for (int u = 0; u < kStreamU; ++u)
            acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < end; i += kStreamThreads) {
        const stream_u32x4 v = __builtin_nontemporal_load(p + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9E3779B9u)  // practically never: keeps the loads alive
        sink[blockIdx.x & 4095] = acc;
}

__global__ __launch_bounds__(kStreamThreads) void stream_write_kernel(uint4 *__restrict__ dst, size_t n16)
{
    size_t begin, end;
    stream_chunk(n16, (int)gridDim.x, (int)blockIdx.x, begin, end);
    size_t i = begin + threadIdx.x;
    for (; i + (size_t)(kStreamU - 1) * kStreamThreads < end; i += (size_t)kStreamU * kStreamThreads) {
#pragma unroll
        for (int u = 0; u < kStreamU; ++u) {
            const size_t j = i + (size_t)u * kStreamThreads;
            const uint32_t x = (uint32_t)j;
            dst[j] = make_uint4(x, x + 1, x + 2, x + 3);
        }
    }
    for (; i < end; i += kStreamThreads) {
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

// ------------------------------------------------- masked-step floors
//
// The grid and block size of the bf16 masked step (step_geometry): each
// block owns chunk c of row b.  MODE 0: the row's state is read and the
// outputs written, nothing else (the launch and its one dependent trip).
// MODE 1: the chunk's 16-byte vectors are streamed as the step streams
// them (512 lanes, two vectors per lane per batch, two batches in flight,
// non-temporal), with no mask and no arithmetic.  MODE 2: only the vectors
// whose mask byte is nonzero (the 128-byte lines holding an allowed token of
// the row's state): the row's state is read, its mask bytes are loaded two
// batches ahead of their logits and choose the offsets (a vector with no
// allowed token gets one past the buffer's records and is not read), as a loads-only
// kernel over exactly the lines the step must read.  Rows must be 16-byte
// aligned.
constexpr int kFloorThreads = 512;
constexpr int kFloorU = 2;
static_assert(kFloorThreads == kStepBigThreads, "the step's block size");

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// The step's loads: raw buffers over the chunk's vectors, so a lane past the
// chunk, and (MODE 2) a vector with no allowed token, which gets an offset
// past the records, read zeros without a memory access.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t floor_buffer(const char *p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(p), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ uint4 nt_load(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 2);  // non-temporal
    return make_uint4(x[0], x[1], x[2], x[3]);
}

__device__ __forceinline__ void floor_batch(uint4 (&d)[kFloorU], __amdgpu_buffer_rsrc_t r, int vb)
{
#pragma unroll
    for (int u = 0; u < kFloorU; ++u)
        d[u] = nt_load(r, (uint32_t)(vb + u * kFloorThreads + (int)threadIdx.x) * 16u);
}

__device__ __forceinline__ void floor_batch_sel(uint4 (&d)[kFloorU], __amdgpu_buffer_rsrc_t r, int vb,
                                                const uint32_t (&m)[kFloorU])
{
#pragma unroll
    for (int u = 0; u < kFloorU; ++u)
        d[u] = nt_load(r, m[u] ? (uint32_t)(vb + u * kFloorThreads + (int)threadIdx.x) * 16u : 0xFFFFFFF0u);
}

__device__ __forceinline__ void floor_masks(uint32_t (&m)[kFloorU], const uint8_t *mb, int vb, int n)
{
#pragma unroll
    for (int u = 0; u < kFloorU; ++u)
        m[u] = mb[min(vb + u * kFloorThreads + (int)threadIdx.x, n - 1)];
}

__device__ __forceinline__ uint32_t fold(const uint4 (&d)[kFloorU])
{
    uint32_t a = 0;
#pragma unroll
    for (int u = 0; u < kFloorU; ++u)
        a ^= d[u].x ^ d[u].y ^ d[u].z ^ d[u].w;
    return a;
}

template <int MODE>
__global__ __launch_bounds__(kFloorThreads) void step_floor_kernel(const void *__restrict__ logits, int V, int64_t ld,
                                                                   const uint32_t *__restrict__ allow, int S,
                                                                   const int32_t *__restrict__ states,
                                                                   int chunk_vec, int nchunks,
                                                                   int32_t *__restrict__ token,
                                                                   int32_t *__restrict__ new_state,
                                                                   uint32_t *__restrict__ sink)
{
    constexpr int K = kFloorThreads * kFloorU;
    const int b = blockIdx.x / nchunks, c = blockIdx.x - b * nchunks;
    const int s = states[b];
    const int nvec = V / 8;
    const int v0 = c * chunk_vec, n = min(nvec, v0 + chunk_vec) - v0;
    const char *crow = static_cast<const char *>(logits) + (size_t)b * ld * 2 + (size_t)v0 * 16;
    const __amdgpu_buffer_rsrc_t rb = floor_buffer(crow, (uint32_t)(n > 0 ? n : 0) * 16u);
    uint32_t acc = 0;
    if (MODE == 1 && n > 0) {
        uint4 da[kFloorU], db[kFloorU];
        floor_batch(da, rb, 0);
        for (int vb = 0; vb < n; vb += 2 * K) {
            floor_batch(db, rb, vb + K);
            acc ^= fold(da);
            floor_batch(da, rb, vb + 2 * K);
            acc ^= fold(db);
        }
    } else if (MODE == 2 && n > 0 && (uint32_t)s < (uint32_t)S) {
        const uint8_t *mb = reinterpret_cast<const uint8_t *>(allow + (size_t)s * ((V + 31) / 32)) + v0;
        uint4 da[kFloorU], db[kFloorU];
        uint32_t m0[kFloorU], m1[kFloorU], m2[kFloorU], m3[kFloorU];
        // the first two batches are read whole (issued before the state is
        // known); the issue order is pinned: the load counter is in order
        floor_batch(da, rb, 0);
        __builtin_amdgcn_sched_barrier(0);
        floor_masks(m2, mb, 2 * K, n);
        __builtin_amdgcn_sched_barrier(0);
        floor_masks(m3, mb, 3 * K, n);
        __builtin_amdgcn_sched_barrier(0);
        floor_batch(db, rb, K);
        __builtin_amdgcn_sched_barrier(0);
        acc ^= fold(da);
        floor_batch_sel(da, rb, 2 * K, m2);
        __builtin_amdgcn_sched_barrier(0);
        floor_masks(m0, mb, 4 * K, n);
        __builtin_amdgcn_sched_barrier(0);
        acc ^= fold(db);
        floor_batch_sel(db, rb, 3 * K, m3);
        __builtin_amdgcn_sched_barrier(0);
        floor_masks(m1, mb, 5 * K, n);
        __builtin_amdgcn_sched_barrier(0);
        for (int vb = 2 * K; vb < n; vb += 4 * K) {
            acc ^= fold(da);
            floor_batch_sel(da, rb, vb + 2 * K, m0);
            __builtin_amdgcn_sched_barrier(0);
            floor_masks(m2, mb, vb + 4 * K, n);
            __builtin_amdgcn_sched_barrier(0);
            acc ^= fold(db);
            floor_batch_sel(db, rb, vb + 3 * K, m1);
            __builtin_amdgcn_sched_barrier(0);
            floor_masks(m3, mb, vb + 5 * K, n);
            __builtin_amdgcn_sched_barrier(0);
            acc ^= fold(da);
            floor_batch_sel(da, rb, vb + 4 * K, m2);
            __builtin_amdgcn_sched_barrier(0);
            floor_masks(m0, mb, vb + 6 * K, n);
            __builtin_amdgcn_sched_barrier(0);
            acc ^= fold(db);
            floor_batch_sel(db, rb, vb + 5 * K, m3);
            __builtin_amdgcn_sched_barrier(0);
            floor_masks(m1, mb, vb + 7 * K, n);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    acc = wave_reduce<true>(acc);
    if (threadIdx.x == 0) {
        sink[blockIdx.x] = acc;
        if (c == 0) {
            token[b] = -1;
            new_state[b] = s;
        }
    }
}

// The alignment walk's own gather: a chase through a uint16 table [S][Cp]
// of states, st = table[st * Cp + c] with the byte class c drawn per step
// from the lane and step (2-byte reads at 32-bit byte offsets, as the walk
// makes them), CHAINS independent chases per lane, 1024-lane blocks.
template <int CHAINS>
__global__ __launch_bounds__(1024) void walk_gather_kernel(const uint16_t *__restrict__ table, int S, int Cp,
                                                           int steps, uint32_t *__restrict__ sink)
{
    const uint32_t lane = blockIdx.x * 1024 + threadIdx.x;
    const char *tb = reinterpret_cast<const char *>(table);
    uint32_t st[CHAINS];
#pragma unroll
    for (int k = 0; k < CHAINS; ++k)
        st[k] = mix(lane * CHAINS + k) % (uint32_t)S;
    uint32_t h = mix(lane);
    for (int i = 0; i < steps; ++i) {
        h = h * 1664525u + 1013904223u;
#pragma unroll
        for (int k = 0; k < CHAINS; ++k) {
            const uint32_t c = ((h >> (4 * k)) & 0xFFFu) % (uint32_t)Cp;
            const uint32_t v = *reinterpret_cast<const uint16_t *>(tb + (st[k] * (uint32_t)Cp + c) * 2u);
            st[k] = v < (uint32_t)S ? v : v % (uint32_t)S;  // stays in bounds
        }
    }
    uint32_t acc = 0;
#pragma unroll
    for (int k = 0; k < CHAINS; ++k)
        acc += st[k];
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
    dv::stream_read_kernel<<<dv::kStreamReadBlocks, dv::kStreamThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<const uint4 *>(src), n_bytes / 16, sink);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

int32_t dvprobe_stream_write(void *dst, size_t n_bytes, void *stream)
{
    if (!dst || n_bytes < 4096 || (n_bytes & 15) || (reinterpret_cast<uintptr_t>(dst) & 15))
        return 1;
    dv::stream_write_kernel<<<dv::kStreamWriteBlocks, dv::kStreamThreads, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<uint4 *>(dst), n_bytes / 16);
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

static bool gather_args_ok(const uint32_t *table, int32_t entries, int32_t lanes, int32_t chains,
                           int32_t steps, const uint32_t *sink, int32_t max_entries)
{
    return table && sink && entries >= 1 && entries <= max_entries && lanes >= 256 && lanes % 256 == 0 &&
           (chains == 1 || chains == 2 || chains == 4 || chains == 8) && steps >= 1;
}

int32_t dvprobe_step_floor(int32_t mode, const void *logits, int32_t num_tokens, int64_t ld_logits,
                           const uint32_t *allow, int32_t num_states, const int32_t *states, int32_t batch,
                           int32_t *token, int32_t *new_state, uint32_t *sink, int64_t sink_words, void *stream)
{
    if (mode < 0 || mode > 2 || !states || !token || !new_state || !sink || batch < 1 || num_tokens < 8 ||
        ld_logits < num_tokens || num_states < 1 || (mode > 0 && !logits) || (mode == 2 && !allow))
        return 1;
    if (mode > 0 && ((reinterpret_cast<uintptr_t>(logits) & 15) || (ld_logits * 2) % 16))
        return 1;  // rows must be 16-byte aligned
    const dv::StepGeometry g = dv::step_geometry(batch, num_tokens, 1);
    const int64_t grid = (int64_t)batch * g.nchunks;
    if (grid > sink_words || grid > (1 << 30))
        return 1;
    const hipStream_t st = static_cast<hipStream_t>(stream);
#define DV_FLOOR(M)                                                                                            \
    dv::step_floor_kernel<M><<<(unsigned)grid, dv::kFloorThreads, 0, st>>>(                                   \
        logits, num_tokens, ld_logits, allow, num_states, states, g.chunk_vec, g.nchunks, token, new_state, sink)
    if (mode == 0)
        DV_FLOOR(0);
    else if (mode == 1)
        DV_FLOOR(1);
    else
        DV_FLOOR(2);
#undef DV_FLOOR
    return hipGetLastError() == hipSuccess ? 0 : 6;
}

int32_t dvprobe_walk_gather(const uint16_t *table, int32_t num_states, int32_t num_classes, int32_t lanes,
                            int32_t chains, int32_t steps, uint32_t *sink, void *stream)
{
    if (!table || !sink || num_states < 1 || num_classes < 1 || (int64_t)num_states * num_classes > (1 << 24) ||
        lanes < 1024 || lanes % 1024 || (chains != 1 && chains != 3) || steps < 1)
        return 1;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (chains == 1)
        dv::walk_gather_kernel<1><<<lanes / 1024, 1024, 0, st>>>(table, num_states, num_classes, steps, sink);
    else
        dv::walk_gather_kernel<3><<<lanes / 1024, 1024, 0, st>>>(table, num_states, num_classes, steps, sink);
    return hipGetLastError() == hipSuccess ? 0 : 6;
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
