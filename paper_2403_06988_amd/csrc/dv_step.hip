// One masked greedy decoding step on CDNA4 (gfx950) (Algorithm 1: mask,
// apply, decode, update; Algorithm 3's argmax over the admissible set).
//
// The step streams B x V logits once: it is bound by HBM read bandwidth.
// Rows are split into chunks so that a launch has a few thousand blocks
// (256 CUs need >> 256 blocks).  A block streams its chunk with 16-byte
// loads, turns every allowed logit into an order-preserving unsigned key and
// keeps the per-lane best (strict '>' in increasing index order, so the
// lowest index wins ties).  Lanes combine (key << 32 | ~index) as one 64-bit
// maximum: a larger key wins, on equal keys the smaller index wins.  Chunks
// of a row meet in a 64-bit atomic maximum in the workspace; the last block
// of the row (arrival counter) writes token / new_state and re-zeroes the
// row's workspace slots for the next call.  The result does not depend on
// block order, so the step is deterministic.
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;
constexpr int kTargetBlocks = 2048;

// Order-preserving key of an fp32 bit pattern, after the value rules of the
// step: NaN ranks as -inf and -0.0 equals +0.0.  Every key of a real value is
// >= key(-inf) = 0x007FFFFF > 0, so 0 can stand for "not allowed".
__device__ __forceinline__ uint32_t f32_key(uint32_t u)
{
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        u = 0xFF800000u;
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int DT> struct Elt;
template <> struct Elt<0> {  // fp32
    static constexpr int kPerVec = 4;
    __device__ static uint32_t bits(const void *row, int64_t i) { return ((const uint32_t *)row)[i]; }
    __device__ static void unpack(const uint4 &v, uint32_t (&u)[kPerVec])
    {
        u[0] = v.x; u[1] = v.y; u[2] = v.z; u[3] = v.w;
    }
};
template <> struct Elt<1> {  // bf16: the high half of an fp32
    static constexpr int kPerVec = 8;
    __device__ static uint32_t bits(const void *row, int64_t i)
    {
        return (uint32_t)((const uint16_t *)row)[i] << 16;
    }
    __device__ static void unpack(const uint4 &v, uint32_t (&u)[kPerVec])
    {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            u[2 * k] = w[k] << 16;
            u[2 * k + 1] = w[k] & 0xFFFF0000u;
        }
    }
};

__device__ __forceinline__ uint64_t pack(uint32_t key, int idx)
{
    return key ? ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx) : 0ull;
}

__device__ __forceinline__ uint64_t block_max(uint64_t v)
{
    __shared__ uint64_t red[kThreads / kWave];
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        const uint64_t o = __shfl_xor(v, d);
        v = o > v ? o : v;
    }
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kThreads / kWave; ++w)
            v = red[w] > v ? red[w] : v;
    }
    return v;  // valid in thread 0
}

template <int DT>
__global__ __launch_bounds__(kThreads) void masked_step_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, int64_t ld, int chunk,
    int nchunks, int32_t *__restrict__ token, int32_t *__restrict__ new_state,
    uint64_t *__restrict__ ws_key, uint32_t *__restrict__ ws_cnt)
{
    using E = Elt<DT>;
    constexpr int kVec = E::kPerVec;
    constexpr int kEltBytes = DT == 0 ? 4 : 2;

    const int b = blockIdx.x / nchunks;
    const int c = blockIdx.x - b * nchunks;
    const int tid = threadIdx.x;
    const int s = states[b];
    const bool live = (uint32_t)s < (uint32_t)S;

    uint32_t best_key = 0;
    int best_idx = 0;
    if (live) {
        const int t0 = c * chunk;
        const int t1 = min(V, t0 + chunk);
        const char *row = static_cast<const char *>(logits) + (size_t)b * (size_t)ld * kEltBytes;
        const uint32_t *arow = allow + (size_t)s * W;
        if ((reinterpret_cast<uintptr_t>(row) & 15) == 0) {
            for (int t = t0 + tid * kVec; t < t1; t += kThreads * kVec) {
                uint32_t m = (arow[t >> 5] >> (t & 31)) & ((1u << kVec) - 1u);
                uint32_t u[kVec];
                if (t + kVec <= V) {
                    const uint4 v = *reinterpret_cast<const uint4 *>(row + (size_t)t * kEltBytes);
                    E::unpack(v, u);
                } else {
#pragma unroll
                    for (int e = 0; e < kVec; ++e)
                        u[e] = t + e < V ? E::bits(row, t + e) : 0u;
                    m &= (1u << (V - t)) - 1u;
                }
#pragma unroll
                for (int e = 0; e < kVec; ++e) {
                    const uint32_t k = ((m >> e) & 1u) ? f32_key(u[e]) : 0u;
                    if (k > best_key) {
                        best_key = k;
                        best_idx = t + e;
                    }
                }
            }
        } else {
            for (int t = t0 + tid; t < t1; t += kThreads) {
                if ((arow[t >> 5] >> (t & 31)) & 1u) {
                    const uint32_t k = f32_key(E::bits(row, t));
                    if (k > best_key) {
                        best_key = k;
                        best_idx = t;
                    }
                }
            }
        }
    }
    const uint64_t best = block_max(pack(best_key, best_idx));
    if (tid != 0)
        return;

    uint64_t final_key;
    if (nchunks == 1) {
        final_key = best;
    } else {
        if (best)
            atomicMax(reinterpret_cast<unsigned long long *>(ws_key + b), (unsigned long long)best);
        __threadfence();
        const uint32_t arrived = atomicAdd(ws_cnt + b, 1u);
        if (arrived != (uint32_t)nchunks - 1)
            return;
        __threadfence();
        final_key = atomicExch(reinterpret_cast<unsigned long long *>(ws_key + b), 0ull);
        atomicExch(ws_cnt + b, 0u);
    }
    const int tok = final_key ? (int)(0xFFFFFFFFu - (uint32_t)final_key) : -1;
    token[b] = tok;
    new_state[b] = tok >= 0 ? next_state[(size_t)s * V + tok] : -1;
}

}  // namespace

hipError_t launch_masked_step(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int B,
                              int64_t ld, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    const int W = (V + 31) / 32;
    const int vec = dtype == 0 ? 4 : 8;
    const int step = kThreads * vec;  // tokens per block-wide vector sweep
    const int max_chunks = (V + step - 1) / step;
    int want = (kTargetBlocks + B - 1) / B;
    want = want < 1 ? 1 : (want > max_chunks ? max_chunks : want);
    int chunk = (V + want - 1) / want;
    chunk = (chunk + step - 1) / step * step;
    const int nchunks = (V + chunk - 1) / chunk;

    uint8_t *ws = static_cast<uint8_t *>(workspace);
    uint64_t *ws_key = reinterpret_cast<uint64_t *>(ws);
    uint32_t *ws_cnt = reinterpret_cast<uint32_t *>(ws + step_counter_offset(B));
    const unsigned grid = (unsigned)B * (unsigned)nchunks;
    if (dtype == 0)
        masked_step_kernel<0><<<grid, kThreads, 0, stream>>>(next_state, allow, S, V, W, states, logits,
                                                             ld, chunk, nchunks, token, new_state,
                                                             ws_key, ws_cnt);
    else
        masked_step_kernel<1><<<grid, kThreads, 0, stream>>>(next_state, allow, S, V, W, states, logits,
                                                             ld, chunk, nchunks, token, new_state,
                                                             ws_key, ws_cnt);
    return hipGetLastError();
}

}  // namespace dv
