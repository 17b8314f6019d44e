// One masked greedy decoding step on CDNA4 (gfx950) (Algorithm 1: mask,
// apply, decode, update; Algorithm 3's argmax over the admissible set).
//
// The step reads B x V logits once: it is bound by HBM read bandwidth, so
// the design is about keeping enough bytes in flight and spending few ALU
// operations per element.
//   * Rows are split into chunks so that a launch has ~2048 blocks (256 CUs
//     need >> 256 blocks).  A block streams its chunk in batches: each lane
//     issues kU = 8 independent 16-byte loads (plus the matching allow-mask
//     words) before it touches any of them, so one CU keeps ~256 KB in
//     flight.
//   * bf16 rows use packed 16-bit arithmetic: per 32-bit word (two logits)
//     one v_pk_ashrrev_i16 and two bit operations give order-preserving
//     16-bit keys; each key is joined with its position in the lane's batch
//     and masked by its allow bit, and one unsigned max per element finds
//     the lane's best key with the lowest position.  The fast key differs
//     from the exact ordering only for NaN (which must rank as -inf) and
//     -0.0 (which must tie with +0.0); a lane whose batch maximum is one of
//     those few key values recomputes that batch exactly from memory.
//   * Lanes combine (exact 32-bit key << 32 | ~index) as one 64-bit maximum:
//     a larger key wins, on equal keys the smaller index wins.
//   * The chunks of one row are combined by a second, tiny kernel (one lane
//     per row) that also writes token / new_state: no atomics and no
//     device-wide fences inside the streaming kernel.  (A per-block release
//     fence at device scope writes back and invalidates the XCD's L2 on
//     gfx950 -- thousands of those per step cost more than the step.)
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;
constexpr int kU = 8;  // 16-byte vectors per lane per batch

// Order-preserving key of an fp32 bit pattern under the step's value rules:
// NaN ranks as -inf and -0.0 equals +0.0.  Every real value's key is
// >= key(-inf) = 0x007FFFFF > 0, so 0 can stand for "not allowed".
__device__ __forceinline__ uint32_t f32_key(uint32_t u)
{
    if ((u & 0x7FFFFFFFu) > 0x7F800000u)
        u = 0xFF800000u;
    if (u == 0x80000000u)
        u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

typedef short s16x2 __attribute__((ext_vector_type(2)));

// Fast 16-bit keys of the two bf16 values in w (flip all bits of negatives,
// set the sign bit of non-negatives).  Exact except: -0.0 -> 0x7FFF (+0.0 ->
// 0x8000), positive NaN -> (0xFF80, 0xFFFF], negative NaN -> [0x0000, 0x007F).
__device__ __forceinline__ uint32_t fast_key2(uint32_t w)
{
    const s16x2 x = __builtin_bit_cast(s16x2, w);
    const s16x2 sign = x >> (s16x2){15, 15};
    return w ^ (__builtin_bit_cast(uint32_t, sign) | 0x80008000u);
}

// All-ones if bit j of m is set, else zero.
__device__ __forceinline__ uint32_t bit_mask(uint32_t m, int j)
{
    return (uint32_t)(((int32_t)(m << (31 - j))) >> 31);
}

__device__ __forceinline__ uint64_t pack(uint32_t key, int idx)
{
    return key ? ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx) : 0ull;
}

__device__ __forceinline__ uint64_t wave_max(uint64_t v)
{
#pragma unroll
    for (int d = kWave / 2; d > 0; d >>= 1) {
        const uint64_t o = __shfl_xor(v, d);
        v = o > v ? o : v;
    }
    return v;
}

__device__ __forceinline__ uint64_t block_max(uint64_t v)
{
    __shared__ uint64_t red[kThreads / kWave];
    v = wave_max(v);
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

template <int DT> struct Elt;
template <> struct Elt<0> {  // fp32
    static constexpr int kVec = 4;
    static constexpr int kBytes = 4;
    __device__ static uint32_t bits(const char *row, int64_t i)
    {
        return reinterpret_cast<const uint32_t *>(row)[i];
    }
};
template <> struct Elt<1> {  // bf16: the high half of an fp32
    static constexpr int kVec = 8;
    static constexpr int kBytes = 2;
    __device__ static uint32_t bits(const char *row, int64_t i)
    {
        return (uint32_t)reinterpret_cast<const uint16_t *>(row)[i] << 16;
    }
};

// Exact scan of elements [e0, e1) with lane stride kThreads.
template <int DT>
__device__ __forceinline__ void scan_exact(const char *row, const uint32_t *arow, int e0, int e1,
                                           uint32_t &best_key, int &best_idx)
{
    for (int t = e0 + (int)threadIdx.x; t < e1; t += kThreads) {
        if ((arow[t >> 5] >> (t & 31)) & 1u) {
            const uint32_t k = f32_key(Elt<DT>::bits(row, t));
            if (k > best_key) {
                best_key = k;
                best_idx = t;
            }
        }
    }
}

// Vector path over the full vectors [v0, v1) of a 16-byte aligned row.
template <int DT>
__device__ __forceinline__ void scan_vectors(const char *row, const uint32_t *arow, int v0, int v1,
                                             uint32_t &best_key, int &best_idx)
{
    using E = Elt<DT>;
    constexpr int kVec = E::kVec;
    const int tid = threadIdx.x;
    for (int vb = v0; vb < v1; vb += kThreads * kU) {
        uint4 d[kU];
        uint32_t m[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int v = vb + u * kThreads + tid;
            if (v < v1) {
                d[u] = *reinterpret_cast<const uint4 *>(row + (size_t)v * 16);
                m[u] = (arow[(v * kVec) >> 5] >> ((v * kVec) & 31)) & ((1u << kVec) - 1u);
            } else {
                d[u] = make_uint4(0, 0, 0, 0);
                m[u] = 0;
            }
        }
        if constexpr (DT == 1) {
            // fast packed keys: (key16 << 16 | 63 - position) masked by the allow bit
            uint32_t bmax = 0, any = 0;
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                any |= m[u];
                const uint32_t w[4] = {d[u].x, d[u].y, d[u].z, d[u].w};
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const uint32_t key = fast_key2(w[k]);
                    const int p = u * 8 + 2 * k;
                    const uint32_t lo = ((key << 16) | (uint32_t)(63 - p)) & bit_mask(m[u], 2 * k);
                    const uint32_t hi = ((key & 0xFFFF0000u) | (uint32_t)(62 - p)) & bit_mask(m[u], 2 * k + 1);
                    bmax = max(bmax, max(lo, hi));
                }
            }
            if (any) {
                const uint32_t k16 = bmax >> 16;
                const bool special = k16 <= 0x007Fu || k16 == 0x7FFFu || k16 == 0x8000u || k16 > 0xFF80u;
                if (!special) {
                    const int p = 63 - (int)(bmax & 0xFFFFu);
                    const int v = vb + (p >> 3) * kThreads + tid;
                    const uint32_t h = (k16 & 0x8000u) ? (k16 & 0x7FFFu) : (~k16 & 0xFFFFu);
                    const uint32_t key = f32_key(h << 16);
                    if (key > best_key) {
                        best_key = key;
                        best_idx = v * kVec + (p & 7);
                    }
                } else {
                    // exact recompute of this lane's batch (NaN or signed zero at the top)
#pragma unroll 1
                    for (int u = 0; u < kU; ++u) {
                        const int v = vb + u * kThreads + tid;
                        for (int e = 0; e < kVec; ++e) {
                            if ((m[u] >> e) & 1u) {
                                const uint32_t key = f32_key(E::bits(row, (int64_t)v * kVec + e));
                                if (key > best_key) {
                                    best_key = key;
                                    best_idx = v * kVec + e;
                                }
                            }
                        }
                    }
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const int v = vb + u * kThreads + tid;
                const uint32_t w[4] = {d[u].x, d[u].y, d[u].z, d[u].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t key = ((m[u] >> e) & 1u) ? f32_key(w[e]) : 0u;
                    if (key > best_key) {
                        best_key = key;
                        best_idx = v * kVec + e;
                    }
                }
            }
        }
    }
}

template <int DT>
__global__ __launch_bounds__(kThreads) void masked_step_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, int64_t ld, int chunk_vec,
    int nchunks, int32_t *__restrict__ token, int32_t *__restrict__ new_state,
    uint64_t *__restrict__ partial)
{
    using E = Elt<DT>;
    constexpr int kVec = E::kVec;
    const int b = blockIdx.x / nchunks;
    const int c = blockIdx.x - b * nchunks;
    const int s = states[b];
    const bool live = (uint32_t)s < (uint32_t)S;

    uint32_t best_key = 0;
    int best_idx = 0;
    if (live) {
        const char *row = static_cast<const char *>(logits) + (size_t)b * (size_t)ld * E::kBytes;
        const uint32_t *arow = allow + (size_t)s * W;
        const int nvec = V / kVec;
        const int e0 = c * chunk_vec * kVec;
        const int e1 = c == nchunks - 1 ? V : min(V, (c + 1) * chunk_vec * kVec);
        if ((reinterpret_cast<uintptr_t>(row) & 15) == 0) {
            scan_vectors<DT>(row, arow, c * chunk_vec, min(nvec, (c + 1) * chunk_vec), best_key, best_idx);
            if (c == nchunks - 1)
                scan_exact<DT>(row, arow, nvec * kVec, V, best_key, best_idx);
        } else {
            scan_exact<DT>(row, arow, e0, e1, best_key, best_idx);
        }
    }
    const uint64_t best = block_max(pack(best_key, best_idx));
    if (threadIdx.x != 0)
        return;
    if (nchunks > 1) {
        partial[blockIdx.x] = best;
        return;
    }
    const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
    token[b] = tok;
    new_state[b] = tok >= 0 ? next_state[(size_t)s * V + tok] : -1;
}

// One lane per row: combine the row's chunk results and write the outputs.
__global__ __launch_bounds__(kThreads) void finalize_kernel(const int32_t *__restrict__ next_state, int S,
                                                           int V, const int32_t *__restrict__ states,
                                                           int B, int nchunks,
                                                           const uint64_t *__restrict__ partial,
                                                           int32_t *__restrict__ token,
                                                           int32_t *__restrict__ new_state)
{
    const int b = blockIdx.x * kThreads + threadIdx.x;
    if (b >= B)
        return;
    uint64_t best = 0;
    for (int c = 0; c < nchunks; ++c) {
        const uint64_t p = partial[(size_t)b * nchunks + c];
        best = p > best ? p : best;
    }
    const int s = states[b];
    const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
    token[b] = tok;
    new_state[b] = (tok >= 0 && (uint32_t)s < (uint32_t)S) ? next_state[(size_t)s * V + tok] : -1;
}

}  // namespace

StepGeometry step_geometry(int B, int V, int dtype)
{
    const int vec = dtype == 0 ? Elt<0>::kVec : Elt<1>::kVec;
    const int nvec = V / vec;
    const int per_block = kThreads;  // at least one vector per lane
    int want = (kStepTargetBlocks + B - 1) / (B > 0 ? B : 1);
    const int max_chunks = (nvec + per_block - 1) / per_block;
    want = want < 1 ? 1 : want;
    want = want > max_chunks ? (max_chunks > 0 ? max_chunks : 1) : want;
    want = want > kStepMaxChunks ? kStepMaxChunks : want;
    int chunk_vec = (nvec + want - 1) / want;
    chunk_vec = (chunk_vec + per_block - 1) / per_block * per_block;
    if (chunk_vec == 0)
        chunk_vec = per_block;
    int nchunks = (nvec + chunk_vec - 1) / chunk_vec;
    if (nchunks < 1)
        nchunks = 1;
    return {chunk_vec, nchunks};
}

hipError_t launch_masked_step(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int B,
                              int64_t ld, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    const int W = (V + 31) / 32;
    const StepGeometry g = step_geometry(B, V, dtype);
    uint64_t *partial = static_cast<uint64_t *>(workspace);
    const unsigned grid = (unsigned)B * (unsigned)g.nchunks;
    if (dtype == 0)
        masked_step_kernel<0><<<grid, kThreads, 0, stream>>>(next_state, allow, S, V, W, states, logits, ld,
                                                             g.chunk_vec, g.nchunks, token, new_state,
                                                             partial);
    else
        masked_step_kernel<1><<<grid, kThreads, 0, stream>>>(next_state, allow, S, V, W, states, logits, ld,
                                                             g.chunk_vec, g.nchunks, token, new_state,
                                                             partial);
    if (g.nchunks > 1)
        finalize_kernel<<<(B + kThreads - 1) / kThreads, kThreads, 0, stream>>>(next_state, S, V, states, B,
                                                                              g.nchunks, partial, token,
                                                                              new_state);
    return hipGetLastError();
}

}  // namespace dv
