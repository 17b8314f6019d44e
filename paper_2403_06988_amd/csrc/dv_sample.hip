// Masked sampling on CDNA4 (gfx950): the sampled decode of Algorithm 1 (the
// paper samples at temperature 1.0, Sec. 4) as a Gumbel-max draw over each
// row's admissible tokens:
//     token = argmax over allowed i of  fma(x_i, 1/T, G_i),  G_i = -ln(-ln U_i),
// with U_i from Philox4x32-10 (Salmon et al., SC 2011) keyed by the seed and
// counted by (i / 4, row, offset), and ln in binary32 by fixed steps that
// round alike on every IEEE implementation (no library log, no division), so
// the draw is reproducible bit for bit.
//
// The cost is arithmetic, not memory: a Philox call (ten rounds of two
// 32x32->64 multiplies) per 4 tokens and two logarithms per token.  Only
// admissible tokens need noise, so each wave compacts its 4-token groups
// that hold at least one allowed token into an LDS queue (one allow word of
// 32 tokens per lane, or half of one when few blocks are resident; ballot
// prefix sums for the queue offsets), then every
// lane takes one queued group: one Philox call per group, a logarithm pair
// per allowed token.  Where a wave's allowed tokens are hardly more than its
// groups (sparse masks) it queues single tokens instead, so that no lane
// waits on a neighbour's second logarithm pair; dense masks keep the groups
// and so one Philox call per 4 tokens.  Lanes combine exact
// (order-preserving fp32 key << 32 | ~index) maxima, so ties go to the lowest
// index and the result does not depend on the order of the work.
#include "dv_sample.h"

namespace dv {
namespace {

constexpr int kThreads = 256;       // split rows: several blocks per row, meeting in the workspace
constexpr int kRowThreads = 1024;   // one block per row once B >= kOneBlockRows
                                    // (below that, split rows keep more waves per CU, which this
                                    // latency-laden arithmetic needs more than it saves a launch)
constexpr int kOneBlockRows = 1024;  // four or more rows per CU keep enough waves resident
// A wave queues single tokens instead of 4-token groups when its allowed
// tokens number at most kTokenRatio4 / 4 times its allowed groups: a lane
// then pays one Philox call and one logarithm pair per trip, where a group
// trip pays as many pairs as the wave's fullest group holds (two or three
// on almost every trip of a sparse random mask, while its groups average
// 1.1 tokens).  Per trip a Philox call is about 63 instructions and a pair
// about 90, so single tokens cost less up to about twice as many tokens as
// groups; runs of allowed tokens (4 per group) keep the groups.
constexpr int kTokenRatio4 = 8;
constexpr int kTargetBlocks = 2048;
constexpr int kHalfSpanBlocks = 512;
constexpr int kMaxChunks = 64;

struct SampleGeometry {
    int threads;
    int chunk_tok;  // a multiple of threads * span tokens (span tokens per lane per iteration)
    int nchunks;
    int span;  // tokens per lane per iteration: 32 (a whole allow word) or 16
};

SampleGeometry sample_geometry(int B, int V)
{
    if (B >= kOneBlockRows) {
        const int per_iter = kRowThreads * 32;
        return {kRowThreads, (V + per_iter - 1) / per_iter * per_iter, 1, 32};
    }
    const int b = B > 0 ? B : 1;
    // Below two blocks per compute unit (a row of whole allow words per lane
    // giving fewer than kHalfSpanBlocks blocks), lanes take half a word each:
    // twice the waves for the same tokens, which this issue-bound kernel
    // needs when so few are resident (B = 64 x V = 32,000: 11-12 against
    // 15.5-16.5 us per step).  Above that the extra blocks only add their
    // start-up and their meeting in the workspace (B = 64 x V = 128,256:
    // 17.3 against 11.2 us).
    int span = 32;
    if ((int64_t)b * ((V + kThreads * 32 - 1) / (kThreads * 32)) < kHalfSpanBlocks)
        span = 16;
    const int per_iter = kThreads * span;
    const int iters = (V + per_iter - 1) / per_iter;
    int want = (kTargetBlocks + b - 1) / b;
    want = want > iters ? iters : want;
    want = want > kMaxChunks ? kMaxChunks : want;
    want = want < 1 ? 1 : want;
    const int per = (iters + want - 1) / want;
    return {kThreads, per * per_iter, (iters + per - 1) / per, span};
}

// a ^ b ^ c in one v_bitop3_b32 (truth table 0x96); the compiler leaves
// the Philox rounds' three-way XORs as two instructions otherwise.
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                               uint32_t k1)
{
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = xor3((uint32_t)(p1 >> 32), c1, k0);
        const uint32_t n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
    }
    return make_uint4(c0, c1, c2, c3);
}

// Word e (0 .. 3) of philox4x32_10's output, for a lane that needs only
// that word: the same ten rounds, the last of which computes only the
// product the word comes from (words 0 and 1 from the multiple of c2,
// words 2 and 3 from the multiple of c0) -- one 32 x 32 -> 64-bit
// multiply fewer per call.
__device__ __forceinline__ uint32_t philox4x32_10_word(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                       uint32_t k0, uint32_t k1, int e)
{
#pragma unroll
    for (int round = 0; round < 9; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = xor3((uint32_t)(p1 >> 32), c1, k0);
        const uint32_t n2 = xor3((uint32_t)(p0 >> 32), c3, k1);
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
    }
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
    const bool from_c2 = e < 2;
    const uint64_t p = (uint64_t)(from_c2 ? 0xCD9E8D57u : 0xD2511F53u) * (from_c2 ? c2 : c0);
    const uint32_t high = xor3((uint32_t)(p >> 32), from_c2 ? c1 : c3, from_c2 ? k0 : k1);
    return (e & 1) ? (uint32_t)p : high;
}

// ln of a positive normal binary32: x = m 2^e, m in [sqrt(1/2), sqrt(2));
// z = (m - 1) / (m + 1) with the reciprocal by four Newton steps from 1/2;
// ln m = 2 (z + z^3 (1/3 + w (1/5 + w (1/7 + w / 9)))), w = z^2;
// ln x = fma(e, ln 2, ln m).  Every operation is a rounded IEEE add,
// multiply or fused multiply-add, written out (no contraction).
__device__ __forceinline__ float ln_f32(float x)
{
#pragma clang fp contract(off)
    const uint32_t bits = __float_as_uint(x);
    int e = (int)(bits >> 23) - 127;
    uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
    if (mb > 0x3FB504F3u) {
        mb -= 0x00800000u;
        e += 1;
    }
    const float f = __uint_as_float(mb) - 1.0f;
    const float d = f + 2.0f;
    float r = 0.5f;
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const float t = __builtin_fmaf(-d, r, 1.0f);
        r = __builtin_fmaf(r, t, r);
    }
    const float z = f * r;
    const float w = z * z;
    float p = __builtin_fmaf(w, 0x1.c71c72p-4f, 0x1.24924ap-3f);
    p = __builtin_fmaf(w, p, 0x1.99999ap-3f);
    p = __builtin_fmaf(w, p, 0x1.555556p-2f);
    const float zw = z * w;
    const float half = __builtin_fmaf(zw, p, z);
    const float lnm = half + half;
    return __builtin_fmaf((float)e, 0x1.62e430p-1f, lnm);
}

__device__ __forceinline__ float gumbel_of_word(uint32_t w)
{
#pragma clang fp contract(off)
    const float u = (float)(2u * (w >> 9) + 1u) * 0x1p-24f;  // exact, strictly inside (0, 1)
    return -ln_f32(-ln_f32(u));
}

// Order-preserving key of a binary32 value: NaN ranks as -inf, -0.0 as
// +0.0; every value's key is > 0, so 0 stands for "nothing yet".  Adding
// +0.0 turns -0.0 into +0.0 and leaves every other value as it is (round to
// nearest); then negatives have all their bits flipped, the rest their sign.
__device__ __forceinline__ uint32_t order_key(float x)
{
#pragma clang fp contract(off)
    float c = x + 0.0f;
    c = c != c ? -__builtin_inff() : c;
    const uint32_t u = __float_as_uint(c);
    return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

__device__ __forceinline__ uint64_t max_u64(uint64_t a, uint64_t b) { return a > b ? a : b; }

template <int DT>
__device__ __forceinline__ float logit_at(const char *row, int i)
{
    if constexpr (DT == 0)
        return reinterpret_cast<const float *>(row)[i];
    else
        return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(row)[i] << 16);
}

// The 4 logits of group g (tokens 4g .. 4g+3) as binary32 bit patterns: one
// vector load when the row is aligned to a group and the group lies inside
// the row, else element loads of the allowed tokens only (the last group
// may run past V).
template <int DT>
__device__ __forceinline__ uint4 group_logits(const char *row, bool aligned, uint32_t g, uint32_t bits, int V)
{
    const int i0 = (int)(g * 4u);
    if (aligned && i0 + 3 < V) {
        if constexpr (DT == 0) {
            return reinterpret_cast<const uint4 *>(row)[g];
        } else {
            const uint2 h = reinterpret_cast<const uint2 *>(row)[g];
            return make_uint4(h.x << 16, h.x & 0xFFFF0000u, h.y << 16, h.y & 0xFFFF0000u);
        }
    }
    uint4 v = make_uint4(0, 0, 0, 0);
    if (bits & 1u)
        v.x = __float_as_uint(logit_at<DT>(row, i0));
    if (bits & 2u)
        v.y = __float_as_uint(logit_at<DT>(row, i0 + 1));
    if (bits & 4u)
        v.z = __float_as_uint(logit_at<DT>(row, i0 + 2));
    if (bits & 8u)
        v.w = __float_as_uint(logit_at<DT>(row, i0 + 3));
    return v;
}

// Exclusive prefix sum over the wave of a count in [0, 15], and the wave's
// total, from four ballots of the count's bits (no LDS, no waits).
__device__ __forceinline__ int wave_prefix_small(int cnt, int &total)
{
    int excl = 0, tot = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint64_t m = __ballot((cnt >> j) & 1);
        const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        excl += below << j;
        tot += __popcll(m) << j;
    }
    total = tot;
    return excl;
}

// The same for a count in [0, 32] (six ballots).
__device__ __forceinline__ int wave_prefix_word(int cnt, int &total)
{
    int excl = 0, tot = 0;
#pragma unroll
    for (int j = 0; j < 6; ++j) {
        const uint64_t m = __ballot((cnt >> j) & 1);
        const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        excl += below << j;
        tot += __popcll(m) << j;
    }
    total = tot;
    return excl;
}

template <int DT, int THREADS, int SPAN>
__global__ __launch_bounds__(THREADS) void masked_sample_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, int64_t ld, float inv_t, uint32_t seed_lo,
    uint32_t seed_hi, uint32_t off_lo, uint32_t off_hi, int chunk_tok, int nchunks, RowMeet meet,
    int32_t *__restrict__ token, int32_t *__restrict__ new_state)
{
#pragma clang fp contract(off)
    constexpr int kWaves = THREADS / kWave;
    static_assert(SPAN == 32 || SPAN == 16, "a whole allow word or one half of it per lane");
    constexpr int kTokPerIter = THREADS * SPAN;
    __shared__ uint32_t queue[kWaves][kWave * 8];  // up to 8 groups per lane per iteration, or 512 tokens
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int b = blockIdx.x / nchunks;
    const int c = blockIdx.x - b * nchunks;
    const int s = states[b];
    const bool live = (uint32_t)s < (uint32_t)S;  // block-uniform
    uint64_t best = 0;
    if (live) {
        const char *row = static_cast<const char *>(logits) + (size_t)b * (size_t)ld * (DT == 0 ? 4 : 2);
        const bool aligned = (reinterpret_cast<uintptr_t>(row) & (DT == 0 ? 15 : 7)) == 0;  // block-uniform
        const uint32_t *arow = allow + (size_t)s * W;
        const int t0 = c * chunk_tok;
        const int t1 = min(V, t0 + chunk_tok);
        for (int base = t0; base < t1; base += kTokPerIter) {  // block-uniform trip count
            const int tok0 = base + tid * SPAN;  // a multiple of SPAN: the word's low or high half
            uint32_t word = tok0 < t1 ? arow[tok0 >> 5] : 0u;
            if constexpr (SPAN == 16)
                word = (word >> (tok0 & 16)) & 0xFFFFu;
            if (tok0 < t1 && t1 - tok0 < SPAN)
                word &= (1u << (t1 - tok0)) - 1u;  // a chunk ends inside this span only at V
            // groups (4 tokens) holding an allowed token: bit 4k of `nz`
            uint32_t nz = (word | (word >> 1) | (word >> 2) | (word >> 3)) & 0x11111111u;
            int groups, toks;
            const int gpos = wave_prefix_small(__popc(nz), groups);  // at most 8 groups per lane
            const int tpos = wave_prefix_word(__popc(word), toks);
            // wave-uniform: single tokens when they fit the queue and are few per group
            const bool by_token = toks <= kWave * 8 && 4 * toks <= kTokenRatio4 * groups;
            if (by_token) {
                int pos = tpos;
                uint32_t w = word;
                while (w) {
                    queue[wave][pos++] = (uint32_t)(tok0 + __builtin_ctz(w));
                    w &= w - 1u;
                }
            } else {
                int pos = gpos;
                while (nz) {
                    const int k = __builtin_ctz(nz) >> 2;
                    nz &= nz - 1u;
                    // token group index (token / 4) and its 4 mask bits
                    queue[wave][pos++] = ((uint32_t)((tok0 >> 2) + k) << 4) | ((word >> (4 * k)) & 0xFu);
                }
            }
            wave_lds_sync();
            if (by_token) {
                for (int q = lane; q < toks; q += kWave) {
                    const uint32_t i = queue[wave][q];
                    const float x = logit_at<DT>(row, (int)i);  // in flight during the Philox rounds
                    const uint32_t word =
                        philox4x32_10_word(i >> 2, (uint32_t)b, off_lo, off_hi, seed_lo, seed_hi, (int)(i & 3u));
                    const float key = __builtin_fmaf(x, inv_t, gumbel_of_word(word));
                    const uint64_t packed =
                        ((uint64_t)order_key(key) << 32) | (uint64_t)(0xFFFFFFFFu - i);
                    best = max_u64(best, packed);
                }
            } else {
                for (int q = lane; q < groups; q += kWave) {
                    const uint32_t entry = queue[wave][q];
                    const uint32_t g = entry >> 4;
                    const uint32_t bitsg = entry & 0xFu;
                    // the logits first: their load is in flight during the Philox rounds
                    const uint4 xs = group_logits<DT>(row, aligned, g, bitsg, V);
                    const uint4 rnd = philox4x32_10(g, (uint32_t)b, off_lo, off_hi, seed_lo, seed_hi);
                    // one guarded pass per position of the group (a pass runs
                    // when any lane of the wave has that token allowed): the
                    // logit and the Philox word are then fixed registers
                    auto noise = [&](uint32_t x, uint32_t word, uint32_t e) {
                        const uint32_t i = g * 4u + e;
                        const float key = __builtin_fmaf(__uint_as_float(x), inv_t, gumbel_of_word(word));
                        const uint64_t packed =
                            ((uint64_t)order_key(key) << 32) | (uint64_t)(0xFFFFFFFFu - i);
                        best = max_u64(best, packed);
                    };
                    if (bitsg & 1u)
                        noise(xs.x, rnd.x, 0u);
                    if (bitsg & 2u)
                        noise(xs.y, rnd.y, 1u);
                    if (bitsg & 4u)
                        noise(xs.z, rnd.z, 2u);
                    if (bitsg & 8u)
                        noise(xs.w, rnd.w, 3u);
                }
            }
            wave_lds_sync();  // every lane has read its entries before the next iteration writes
        }
    }
    // block-wide maximum
    __shared__ uint64_t red[THREADS / kWave];
    best = wave_reduce<true>(best);
    if (lane == 0)
        red[wave] = best;
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kWaves; ++w)
            best = max_u64(best, red[w]);
        if (nchunks == 1 || meet_row(meet, b, c, nchunks, best, best)) {  // else another block finishes the row
            const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
            const bool found = live && tok >= 0 && tok < V;  // guards the read
            token[b] = found ? tok : -1;
            new_state[b] = found ? next_state[(size_t)s * V + tok] : -1;
        }
    }
}


}  // namespace

size_t sample_workspace_bytes(int B, int V)
{
    return row_meet_bytes(B, sample_geometry(B, V).nchunks);
}

hipError_t launch_masked_sample(const int32_t *next_state, const uint32_t *allow, int S, int V,
                                const int32_t *states, const void *logits, int dtype, int B, int64_t ld,
                                float inv_temperature, uint64_t seed, uint64_t offset, int32_t *token,
                                int32_t *new_state, void *workspace, hipStream_t stream)
{
    const int W = (V + 31) / 32;
    const SampleGeometry g = sample_geometry(B, V);
    const RowMeet meet = row_meet(workspace, B);
    const unsigned grid = (unsigned)B * (unsigned)g.nchunks;
    const uint32_t s_lo = (uint32_t)seed, s_hi = (uint32_t)(seed >> 32);
    const uint32_t o_lo = (uint32_t)offset, o_hi = (uint32_t)(offset >> 32);
#define DV_SAMPLE_LAUNCH(DT, T, SP)                                                                              \
    masked_sample_kernel<DT, T, SP><<<grid, T, 0, stream>>>(next_state, allow, S, V, W, states, logits, ld,      \
                                                            inv_temperature, s_lo, s_hi, o_lo, o_hi,             \
                                                            g.chunk_tok, g.nchunks, meet, token, new_state)
    if (g.threads == kRowThreads) {
        if (dtype == 0)
            DV_SAMPLE_LAUNCH(0, kRowThreads, 32);
        else
            DV_SAMPLE_LAUNCH(1, kRowThreads, 32);
    } else if (g.span == 32) {
        if (dtype == 0)
            DV_SAMPLE_LAUNCH(0, kThreads, 32);
        else
            DV_SAMPLE_LAUNCH(1, kThreads, 32);
    } else {
        if (dtype == 0)
            DV_SAMPLE_LAUNCH(0, kThreads, 16);
        else
            DV_SAMPLE_LAUNCH(1, kThreads, 16);
    }
#undef DV_SAMPLE_LAUNCH
    return hipGetLastError();
}

}  // namespace dv
