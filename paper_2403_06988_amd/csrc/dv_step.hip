// One masked greedy decoding step on CDNA4 (gfx950) (Algorithm 1: mask,
// apply, decode, update; Algorithm 3's argmax over the admissible set).
//
// The step reads B x V logits once: it is bound by HBM read bandwidth, so
// the design is about keeping enough bytes in flight and spending few ALU
// operations per element.
//   * Launch shape (bf16, step_geometry).  A row is one 512-lane block once
//     B >= 256 (every CU gets at least one row), or when B >= 64 and the row
//     holds at most 32768 logits (a second block per row buys nothing
//     there).  Otherwise each row is split into about 32 / sqrt(B) chunks,
//     one block each, and the chunks meet in the workspace (meet_row): up
//     to four chunks in pairs, each pair's second block learning both
//     values from one device-scope atomic maximum (one round trip per
//     level); more chunks through a device-scope atomic maximum and then an
//     atomic count whose operand depends on the maximum's result, the block
//     that counts last taking the row's result.  The finishing block puts
//     the entries back to zero.  For bf16 the 64-bit entry also carries the
//     winner's next state, so that block reads nothing more.  No second
//     kernel and no device-wide fences (a release fence at device scope
//     writes back and invalidates the XCD's L2 on gfx950).
//   * Each lane streams batches of 2 independent non-temporal 16-byte loads
//     with a register double buffer: batch i + 1 is in flight while batch i
//     is reduced.  Loads are branch-free and in a fixed order, because the
//     load counter is in order: waiting for one load waits for every earlier
//     one.  The first batch is issued before the row's state is known.
//     Rows that start on a 16-byte boundary are read as raw buffers whose
//     records end at the chunk's end: one add per load for the address, and
//     a lane past the chunk reads zeros (no clamp, no memory access).
//   * Mask bytes (one per 8 logits).  With two or more blocks per compute
//     unit, the block first copies its chunk's mask bytes into LDS; with one,
//     chunks of at least 8 batches read each batch's mask bytes from memory
//     two batches ahead of its logits.  Either way each later batch's
//     offsets are chosen from them: a vector with no allowed token gets an
//     offset past the buffer's records, which reads zeros without a memory
//     access, so a 128-byte line with no allowed token is never fetched.
//     Shorter chunks at one block per unit read their mask bytes beside
//     their logits, and every line.
//   * bf16 arithmetic, a batch at a time in two parts.  Fold: per 32-bit
//     word (two logits) a v_pk_ashrrev_i16 and two bit operations give the
//     order-preserving 16-bit keys ANDed with two 16-bit lane masks (from an
//     LDS table indexed by the mask byte, read a batch ahead), so disallowed
//     tokens key as 0; the loads of a later batch are issued right after it.
//     Reduce: v_pk_max_u16 over the masked keys and one wave-wide max per
//     batch (DPP moves, no LDS and no barrier); only the wave(s) holding the
//     maximum search their masked keys for its lowest index.  The fast key
//     differs from the exact ordering only for NaN (which must rank as -inf)
//     and -0.0 (which must tie with +0.0); a batch whose maximum is one of
//     those few key values is redone with exact keys.
//   * A bf16 row need not be 16-byte aligned (any row stride): the elements
//     before its first 16-byte boundary are read one by one and the mask
//     bits of each vector are taken from two mask bytes, shifted.
//   * fp32 rows (small workloads) use 256-lane blocks, the same head, vector
//     and tail split (4 elements per vector) and exact keys with the
//     index tracked per element.
//   * Lanes combine (exact 32-bit key << 32 | ~index) as one 64-bit maximum:
//     a larger key wins, on equal keys the smaller index wins.  The result
//     does not depend on block or lane order, so the step is deterministic.
#include <atomic>

#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kSmallThreads = kStepSmallThreads;  // fp32 rows
constexpr int kSmallU = 8;                         // 16-byte vectors per lane per batch
constexpr int kBigThreads = kStepBigThreads;       // lanes per bf16 block
constexpr int kBigU = 2;                           // vectors per lane per batch (x2: double-buffered)

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
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Fast 16-bit keys of the two bf16 values in w (flip all bits of negatives,
// set the sign bit of non-negatives).  Exact except: -0.0 -> 0x7FFF (+0.0 ->
// 0x8000), positive NaN -> (0xFF80, 0xFFFF], negative NaN -> [0x0000, 0x007F).
__device__ __forceinline__ uint32_t fast_key2(uint32_t w)
{
    const s16x2 x = __builtin_bit_cast(s16x2, w);
    const s16x2 sign = x >> (s16x2){15, 15};
    return w ^ (__builtin_bit_cast(uint32_t, sign) | 0x80008000u);
}

__device__ __forceinline__ uint64_t pack(uint32_t key, int idx)
{
    return key ? ((uint64_t)key << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx) : 0ull;
}

__device__ __forceinline__ uint64_t wave_max(uint64_t v) { return wave_reduce<true>(v); }

template <int THREADS>
__device__ __forceinline__ uint64_t block_max(uint64_t v)
{
    __shared__ uint64_t red[THREADS / kWave];
    v = wave_max(v);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    if (lane == 0)
        red[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < THREADS / kWave; ++w)
            v = red[w] > v ? red[w] : v;
    }
    return v;  // valid in thread 0
}

// "next state not loaded yet": the winner was not a vector-path best.
constexpr int kNsUnknown = INT_MIN;

// The meeting word of a bf16 row split over several blocks: the winner's
// 16-bit key (a bf16 value's exact 32-bit key is that key followed by 16
// fixed bits), 2^24 - 1 - its index (V <= 2^24), and its next state + 1 in
// the low 24 bits -- so the 64-bit maximum orders by key, then by lowest
// index, and hands the last block the winner's next state as well.  A next
// state outside [-1, 2^24 - 2] (a table not written by dv_align) is marked
// with the top value and read again.  0 = nothing allowed.
constexpr uint32_t kSplitNsReload = 0xFFFFFFu;

__device__ __forceinline__ uint64_t pack_split(uint64_t best, int tok, int ns)
{
    const uint32_t nsf = (ns >= -1 && ns < (int)kSplitNsReload - 1) ? (uint32_t)(ns + 1) : kSplitNsReload;
    return (best >> 48) << 48 | (uint64_t)(0xFFFFFFu - (uint32_t)tok) << 24 | nsf;
}

__device__ __forceinline__ void unpack_split(uint64_t w, int &tok, int &ns)
{
    if (!w) {
        tok = -1;
        ns = -1;
        return;
    }
    tok = (int)(0xFFFFFFu - (uint32_t)((w >> 24) & 0xFFFFFFu));
    const uint32_t nsf = (uint32_t)w & 0xFFFFFFu;
    ns = nsf == kSplitNsReload ? kNsUnknown : (int)nsf - 1;
}

// block_max, also returning (in thread 0) the next state of the winner when
// its wave had already loaded it: `vec_pack` is the wave's vector-path best
// (wave-uniform) and `vec_ns` its next state.
template <int THREADS>
__device__ __forceinline__ uint64_t block_max_ns(uint64_t v, uint64_t vec_pack, int vec_ns, int &ns)
{
    __shared__ uint64_t red[THREADS / kWave];
    __shared__ int red_ns[THREADS / kWave];
    v = wave_max(v);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    if (lane == 0) {
        red[wave] = v;
        red_ns[wave] = v != 0 && v == vec_pack ? vec_ns : kNsUnknown;
    }
    __syncthreads();
    ns = kNsUnknown;
    if (threadIdx.x == 0) {
        ns = red_ns[0];
        for (int w = 1; w < THREADS / kWave; ++w) {
            if (red[w] > v) {
                v = red[w];
                ns = red_ns[w];
            }
        }
    }
    return v;  // valid in thread 0
}

template <int DT> struct Elt;
template <> struct Elt<0> {  // fp32
    __device__ static uint32_t bits(const char *row, int64_t i)
    {
        return reinterpret_cast<const uint32_t *>(row)[i];
    }
};
template <> struct Elt<1> {  // bf16: the high half of an fp32
    __device__ static uint32_t bits(const char *row, int64_t i)
    {
        return (uint32_t)reinterpret_cast<const uint16_t *>(row)[i] << 16;
    }
};

// Exact scan of elements [e0, e1) with lane stride THREADS (with MASKED
// false every element counts as allowed and the mask is not read).
template <int DT, int THREADS, bool MASKED = true>
__device__ __forceinline__ void scan_exact(const char *row, const uint32_t *arow, int e0, int e1,
                                           uint32_t &best_key, int &best_idx)
{
    for (int t = e0 + (int)threadIdx.x; t < e1; t += THREADS) {
        if (!MASKED || ((arow[t >> 5] >> (t & 31)) & 1u)) {
            const uint32_t k = f32_key(Elt<DT>::bits(row, t));
            if (k > best_key) {
                best_key = k;
                best_idx = t;
            }
        }
    }
}

// fp32 rows are read as a head of `head` < 4 elements (up to the row's first
// 16-byte boundary), 16-byte vectors from element `head` on, and a tail of
// fewer than 4 elements.  Vector v holds elements i = head + 4v .. i + 3,
// whose mask bits straddle two mask words when i mod 32 > 28.
__device__ __forceinline__ int f32_head(const char *row, int V)
{
    return min(V, (int)(((16u - (uint32_t)(reinterpret_cast<uintptr_t>(row) & 15u)) & 15u) >> 2));
}

// Vector path over vectors [v0, v1) past the head; each lane takes U vectors
// per batch, strided by THREADS so loads coalesce.  Per lane, elements are
// visited in increasing index order and only a strictly larger key replaces
// the lane's best, so the lane keeps the lowest index of its maximum.
template <int THREADS, int U>
__device__ __forceinline__ void scan_vectors_f32(const char *row, const uint32_t *arow, int head, int v0, int v1,
                                                 uint32_t &best_key, int &best_idx)
{
    const char *vrow = row + 4 * head;  // 16-byte aligned
    const int tid = threadIdx.x;
    for (int vb = v0; vb < v1; vb += THREADS * U) {
        uint4 d[U];
        uint32_t m[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = vb + u * THREADS + tid;
            if (v < v1) {
                d[u] = *reinterpret_cast<const uint4 *>(vrow + (size_t)v * 16);
                const int i = head + 4 * v, w = i >> 5, sh = i & 31;
                uint32_t bits = arow[w] >> sh;
                if (sh > 28)  // element i + 3 < V, so word w + 1 is in the row
                    bits |= arow[w + 1] << (32 - sh);
                m[u] = bits & 0xFu;
            } else {
                d[u] = make_uint4(0, 0, 0, 0);
                m[u] = 0;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = head + 4 * (vb + u * THREADS + tid);
            const uint32_t w[4] = {d[u].x, d[u].y, d[u].z, d[u].w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t key = ((m[u] >> e) & 1u) ? f32_key(w[e]) : 0u;
                if (key > best_key) {
                    best_key = key;
                    best_idx = i + e;
                }
            }
        }
    }
}

// fp32 rows, 256-lane blocks, exact keys.
template <int THREADS, int U>
__global__ __launch_bounds__(THREADS) void masked_step_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, RowMap map, int chunk_vec,
    int nchunks, int32_t *__restrict__ token, int32_t *__restrict__ new_state, RowMeet meet)
{
    const int b = blockIdx.x / nchunks;
    const int c = blockIdx.x - b * nchunks;
    const int s = row_state(states, map, next_state, allow, S, V, b);
    const bool live = (uint32_t)s < (uint32_t)S;

    uint32_t best_key = 0;
    int best_idx = 0;
    if (live) {
        const char *row = static_cast<const char *>(logits) + (size_t)map.offset(b) * 4;
        const uint32_t *arow = allow + (size_t)s * W;
        const int head = f32_head(row, V);
        const int nvec = (V - head) / 4;
        // increasing index order per lane: head, vectors, tail
        if (c == 0)
            scan_exact<0, THREADS>(row, arow, 0, head, best_key, best_idx);
        scan_vectors_f32<THREADS, U>(row, arow, head, c * chunk_vec, min(nvec, (c + 1) * chunk_vec), best_key,
                                     best_idx);
        if (c == nchunks - 1)
            scan_exact<0, THREADS>(row, arow, head + nvec * 4, V, best_key, best_idx);
    }
    uint64_t best = block_max<THREADS>(pack(best_key, best_idx));
    if (threadIdx.x != 0)
        return;
    if (nchunks > 1 && !meet_row(meet, b, c, nchunks, best, best))
        return;  // another block of the row finishes it
    const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
    const bool found = tok >= 0 && tok < V;  // always true for a found token; guards the read
    token[b] = found ? tok : -1;
    new_state[b] = found ? next_state[(size_t)s * V + tok] : -1;
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pk_max_u16(uint32_t a, uint32_t b)
{
    return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(u16x2, a),
                                                                   __builtin_bit_cast(u16x2, b)));
}

__device__ __forceinline__ uint32_t wave_reduce_u32(uint32_t v, bool is_max)
{
    return is_max ? wave_reduce<true>(v) : wave_reduce<false>(v);  // in every lane of the wave
}

// bf16 rows.  Per batch of U vectors per lane:
//   pass 1: packed 16-bit fast keys, masked through an LDS table that turns
//           a mask byte into four 32-bit lane masks, folded with
//           v_pk_max_u16 -- two VALU operations per logit;
//   wave:   one wave-wide max of (lane max << 1 | lane has an allowed
//           element), by cross-lane shuffles (no barrier, so waves never
//           wait for each other inside the stream);
//   pass 2: only if the batch beats the wave's best so far: lanes holding
//           the maximum find its first position in their registers, and a
//           wave-wide min picks the lowest index.  A batch whose maximum is
//           one of the inexact fast keys (NaN, -0.0 / +0.0) is redone with
//           exact keys.
// The waves' results meet in one block-wide maximum at the end.  Without
// the mask (MASKED false: the model's own choice, for opportunistic
// masking) every element of the chunk counts as allowed and no mask byte is
// read.

// Block barrier ordering LDS only: global loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// mask byte -> two 16-bit lane masks per 32-bit word of logits
__device__ __forceinline__ void fill_lut(uint4 *lut)
{
    if (threadIdx.x < 256) {
        const uint32_t m = threadIdx.x;
        uint4 e;
        e.x = ((m & 1u) ? 0x0000FFFFu : 0u) | ((m & 2u) ? 0xFFFF0000u : 0u);
        e.y = ((m & 4u) ? 0x0000FFFFu : 0u) | ((m & 8u) ? 0xFFFF0000u : 0u);
        e.z = ((m & 16u) ? 0x0000FFFFu : 0u) | ((m & 32u) ? 0xFFFF0000u : 0u);
        e.w = ((m & 64u) ? 0x0000FFFFu : 0u) | ((m & 128u) ? 0xFFFF0000u : 0u);
        lut[m] = e;
    }
}

// Loads are branch-free: a lane past the chunk reloads its last vector and
// its mask byte counts as 0 when the batch is reduced.  (A load under a
// branch makes the compiler wait for every outstanding load at the join,
// which would serialise the double buffer.)
template <int THREADS, int U>
__device__ __forceinline__ void load_batch_bf16(uint4 (&d)[U], const char *row, int vb, int v1)
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int v = min(vb + u * THREADS + tid, v1 - 1);
        // logits are read once: a non-temporal load keeps them from
        // displacing reusable lines (mask rows, tables) in the caches
        const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(row + (size_t)v * 16));
        d[u] = make_uint4(x[0], x[1], x[2], x[3]);
    }
}

// Buffer loads for aligned rows: the row's vectors [0, v1) and their mask
// bytes as raw buffers whose records end at the chunk's end, so a lane past
// it reads zeros (an allowed-nothing mask byte) with no clamp and no memory
// access; the per-lane offset is one add per load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_buffer(const void *p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

template <int THREADS, int U>
__device__ __forceinline__ void load_batch_buf(uint4 (&d)[U], __amdgpu_buffer_rsrc_t r, int vb)
{
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t off = (uint32_t)(vb + u * THREADS + (int)threadIdx.x) * 16u;
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 2);  // non-temporal
        d[u] = make_uint4(x[0], x[1], x[2], x[3]);
    }
}

// As load_batch_buf for the staged scan: a vector whose mask byte `sel[u]`
// is 0 gets an offset past the records, which reads zeros without touching
// memory, so a 128-byte line none of whose vectors is needed is not fetched.
template <int THREADS, int U>
__device__ __forceinline__ void load_batch_buf_sel(uint4 (&d)[U], __amdgpu_buffer_rsrc_t r, int vb,
                                                   const uint32_t (&sel)[U])
{
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t off = sel[u] ? (uint32_t)(vb + u * THREADS + (int)threadIdx.x) * 16u : 0xFFFFFFF0u;
        const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 2);
        d[u] = make_uint4(x[0], x[1], x[2], x[3]);
    }
}

template <int THREADS, int U>
__device__ __forceinline__ void load_masks_buf(uint32_t (&m)[U], __amdgpu_buffer_rsrc_t r, int vb)
{
#pragma unroll
    for (int u = 0; u < U; ++u)
        m[u] = __builtin_amdgcn_raw_buffer_load_b8(r, vb + u * THREADS + (int)threadIdx.x, 0, 0);
}

// A row is read as a head of `head` < 8 elements (its first 16-byte
// boundary), then 16-byte vectors from element `head` on, then a tail of
// fewer than 8 elements.  Vector v holds elements head + 8v .. head + 8v + 7,
// whose mask bits are bits head .. head + 7 of allow bytes v and v + 1 (just
// byte v when head = 0).  Rows of any alignment (any row stride) thus take
// the vector path; the head and the tail are scanned element by element.
struct RowSplit {
    int head;  // elements before the first 16-byte boundary (< 8)
    int nvec;  // 16-byte vectors after the head
};

__device__ __forceinline__ RowSplit split_row(const char *row, int V)
{
    const int head = min(V, (int)(((16u - (uint32_t)(reinterpret_cast<uintptr_t>(row) & 15u)) & 15u) >> 1));
    return {head, (V - head) / 8};
}

// This lane's packed best (exact key << 32 | ~index, 0 if none) over the
// vectors [v0, v1) of `row` past its head, plus the head when `first` and
// the tail when `last`.  `da` holds the first batch (loaded by the caller,
// so it can be in flight before the row's state is known).  SHIFTED: the
// head is not empty, so mask bits straddle two bytes.  The entry of
// `ns_row` (the row state's next-state row) at the wave's vector-path best
// is loaded once the stream is done, before the block's maximum is known:
// `vec_pack` and `vec_ns` return that best and its next state
// (wave-uniform).  The mask byte of vector v (bits 8v .. 8v + 7 of the
// allow row) is mbytes[v - moff]: the allow row itself (moff = 0) or the
// chunk's bytes staged in LDS.  `db` holds the second batch when STAGED
// (issued by the caller before the staging finished).  SELECT (STAGED
// only): vectors with no allowed token are not read (see
// load_batch_buf_sel).  AHEAD2 (aligned rows streamed from memory): the
// mask bytes are read two batches ahead of their logits and choose the
// loads in the same way.
template <int THREADS, int U, bool MASKED, bool SHIFTED, bool STAGED, bool SELECT, bool AHEAD2 = false>
__device__ __forceinline__ uint64_t scan_bf16(const char *row, const uint32_t *arow, const uint8_t *mbytes,
                                              int moff, const int32_t *ns_row, RowSplit rs, int v0, int v1,
                                              bool first, bool last, int V, const uint4 *lut, uint4 (&da)[U],
                                              uint4 (&db)[U], uint64_t &vec_pack, int &vec_ns)
{
    static_assert(!SELECT || STAGED, "selection reads the staged mask bytes");
    static_assert(!AHEAD2 || (MASKED && !STAGED), "two batches ahead: the streamed mask bytes choose the loads");
    constexpr int kVec = 8;
    constexpr int kStep = THREADS * U;  // vectors per batch
    const int tid = threadIdx.x;
    const int head = SHIFTED ? rs.head : 0;
    const char *vrow = row + 2 * head;  // 16-byte aligned
    uint32_t best_key = 0;  // exact key of the wave's best vector-path element, wave-uniform
    int best_idx = 0;
    int best_ns = kNsUnknown;
    uint32_t lane_key = 0;  // exact key of this lane's head / tail elements
    int lane_idx = 0;
    if (v0 < v1) {
        const int last_byte = (V - 1) >> 3;
        auto mask_of = [&](int v) -> uint32_t {
            if constexpr (!MASKED) {
                return 0xFFu;
            } else if constexpr (!SHIFTED) {
                return mbytes[v - moff];
            } else {
                const uint32_t b0 = mbytes[v - moff], b1 = mbytes[min(v + 1, last_byte) - moff];
                return ((b0 | (b1 << 8)) >> head) & 0xFFu;
            }
        };
        auto load_masks = [&](uint32_t (&m)[U], int vb) {
#pragma unroll
            for (int u = 0; u < U; ++u)
                m[u] = mask_of(min(vb + u * THREADS + tid, v1 - 1));
        };
        // One batch is U vectors per lane, taken in two parts.  fold: the
        // batch's masked 16-bit keys (two per word, 0 where not allowed) from
        // its logits and the mask-table entries of its mask bytes; after it
        // the logits' registers are free, so the loads of a later batch are
        // issued right then.  reduce: the wave-wide maximum and, when it
        // beats the wave's best so far, the search for its lowest position,
        // both on the masked keys.  Loads are branch-free and in a fixed
        // order (the load counter is in order: waiting for one load waits
        // for every earlier one), so while a batch is reduced the next is in
        // flight.
        //
        // Mask bytes with the lanes past the chunk zeroed (the buffer loads
        // of the aligned streaming scans already read zeros there).
        constexpr bool kZeroPast = MASKED && !SHIFTED && !STAGED;
        auto live = [&](uint32_t (&m)[U], int vb) {
            if constexpr (!kZeroPast) {
#pragma unroll
                for (int u = 0; u < U; ++u)
                    m[u] = vb + u * THREADS + tid < v1 ? m[u] : 0u;
            }
        };
        // mask-table entries of live mask bytes: two 16-bit lane masks per word
        auto entries = [&](uint4 (&l)[U], const uint32_t (&m)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if constexpr (MASKED) {
                    l[u] = lut[m[u]];
                } else {
                    const uint32_t all = m[u] ? 0xFFFFFFFFu : 0u;
                    l[u] = make_uint4(all, all, all, all);
                }
            }
        };
        // masked keys of a batch; returns whether the lane has an allowed
        // element in it
        auto fold = [&](const uint4 (&d)[U], const uint4 (&l)[U], const uint32_t (&m)[U],
                        uint32_t (&km)[4 * U]) -> uint32_t {
            uint32_t any = 0;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                any |= m[u];
                km[4 * u + 0] = fast_key2(d[u].x) & l[u].x;
                km[4 * u + 1] = fast_key2(d[u].y) & l[u].y;
                km[4 * u + 2] = fast_key2(d[u].z) & l[u].z;
                km[4 * u + 3] = fast_key2(d[u].w) & l[u].w;
            }
            return any;
        };
        // The batch's wave-wide maximum against the wave's best so far.  Per
        // lane, elements are in increasing index order and a later batch
        // replaces the best only when strictly larger, so the wave keeps the
        // lowest index of its maximum.
        auto reduce = [&](const uint32_t (&km)[4 * U], uint32_t any, int vb) {
            uint32_t acc = 0;
#pragma unroll
            for (int i = 0; i < 4 * U; ++i)
                acc = pk_max_u16(acc, km[i]);
            const uint32_t lane_max = max(acc & 0xFFFFu, acc >> 16);
            const uint32_t top = wave_reduce_u32((lane_max << 1) | (any ? 1u : 0u), true);
            const uint32_t k16 = top >> 1;
            if (k16 == 0 && (top & 1u) == 0)
                return;  // nothing allowed in this batch
            const bool special = k16 <= 0x007Fu || k16 == 0x7FFFu || k16 == 0x8000u || k16 > 0xFF80u;
            if (!special) {
                const uint32_t h = (k16 & 0x8000u) ? (k16 & 0x7FFFu) : (~k16 & 0xFFFFu);
                const uint32_t key = f32_key(h << 16);
                if (key <= best_key)
                    return;  // an earlier batch of this wave (lower indices) is at least as good
                // first allowed element whose bits are h: a non-special k16
                // is not 0, and the fast key is one-to-one, so a masked key
                // equal to k16 is exactly that
                int pos = 0x7FFFFFFF;
                if (lane_max == k16) {
#pragma unroll
                    for (int i = 4 * U - 1; i >= 0; --i) {
                        const int e = head + (vb + (i / 4) * THREADS + tid) * kVec + 2 * (i % 4);
                        if ((km[i] >> 16) == k16)
                            pos = e + 1;
                        if ((km[i] & 0xFFFFu) == k16)
                            pos = e;
                    }
                }
                best_idx = (int)wave_reduce_u32((uint32_t)pos, false);
                best_key = key;
            } else {
                // exact keys for this batch (NaN or a signed zero at the top),
                // logits and mask bytes re-read from memory: a rare path, kept
                // out of the registers
                uint32_t bk = 0;
                int bi = 0;
#pragma unroll 1
                for (int u = 0; u < U; ++u) {
                    const int v = vb + u * THREADS + tid;
                    const uint32_t mb = v < v1 ? mask_of(v) : 0u;
#pragma unroll 1
                    for (int e = 0; e < kVec; ++e) {
                        if ((mb >> e) & 1u) {
                            const int i = head + v * kVec + e;
                            const uint32_t key = f32_key(Elt<1>::bits(row, i));
                            if (key > bk) {
                                bk = key;
                                bi = i;
                            }
                        }
                    }
                }
                const uint32_t kmax = wave_reduce_u32(bk, true);
                if (kmax > best_key) {
                    best_idx = (int)wave_reduce_u32(bk == kmax ? (uint32_t)bi : 0x7FFFFFFFu, false);
                    best_key = kmax;
                }
            }
        };
        uint32_t ma[U], mb[U];
        uint4 la[U], lb[U];  // mask-table entries of the batch being folded and of the next
        if constexpr (STAGED) {
            // Both first batches are in flight (issued by the caller) and the
            // mask bytes are in LDS: reading them costs no memory trip, so
            // with SELECT every later batch's addresses are chosen from them.
            // Each batch's mask bytes are read from LDS once, two batches
            // ahead, and serve both its addresses and its fold.
            const __amdgpu_buffer_rsrc_t rl = raw_buffer(vrow, (uint32_t)v1 * 16u);
            auto issue = [&](uint4 (&d)[U], int vb, const uint32_t (&sel)[U]) {
                if constexpr (SELECT && MASKED && !SHIFTED)
                    load_batch_buf_sel<THREADS, U>(d, rl, vb, sel);
                else
                    load_batch_bf16<THREADS, U>(d, vrow, vb, v1);
            };
            uint32_t na[U], nb[U];
            load_masks(ma, v0);
            live(ma, v0);
            load_masks(mb, v0 + kStep);
            live(mb, v0 + kStep);
            entries(la, ma);
            for (int vb = v0; vb < v1; vb += 2 * kStep) {
                load_masks(na, vb + 2 * kStep);
                live(na, vb + 2 * kStep);
                {
                    uint32_t km[4 * U];
                    const uint32_t any = fold(da, la, ma, km);
                    __builtin_amdgcn_sched_barrier(0);
                    issue(da, vb + 2 * kStep, na);
                    __builtin_amdgcn_sched_barrier(0);
                    entries(lb, mb);
                    reduce(km, any, vb);
                }
                load_masks(nb, vb + 3 * kStep);
                live(nb, vb + 3 * kStep);
                {
                    uint32_t km[4 * U];
                    const bool in = vb + kStep < v1;  // block-uniform
                    const uint32_t any = in ? fold(db, lb, mb, km) : 0u;
                    __builtin_amdgcn_sched_barrier(0);
                    issue(db, vb + 3 * kStep, nb);
                    __builtin_amdgcn_sched_barrier(0);
                    entries(la, na);
                    if (in)
                        reduce(km, any, vb + kStep);
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    ma[u] = na[u];
                    mb[u] = nb[u];
                }
                // the best so far's next state, loaded outside any branch (a
                // load under a branch would make the compiler wait for every
                // load in flight where the branches join)
                best_ns = ns_row[best_idx];
            }
        } else if constexpr (MASKED && !SHIFTED && !AHEAD2) {
            // Mask bytes one batch ahead, each issued before its batch's
            // logits, so reading a batch's table entries waits for no logits.
            const __amdgpu_buffer_rsrc_t rl = raw_buffer(vrow, (uint32_t)v1 * 16u);
            const __amdgpu_buffer_rsrc_t rm = raw_buffer(mbytes - moff, (uint32_t)v1);
            load_masks_buf<THREADS, U>(ma, rm, v0);
            load_masks_buf<THREADS, U>(mb, rm, v0 + kStep);
            __builtin_amdgcn_sched_barrier(0);
            load_batch_buf<THREADS, U>(db, rl, v0 + kStep);
            __builtin_amdgcn_sched_barrier(0);
            entries(la, ma);
#define DV_STREAM_BATCH(D, L, LN, M, MN, K)                                                                    \
    {                                                                                                          \
        uint32_t km[4 * U];                                                                                    \
        const bool in = vb + (K) * kStep < v1; /* block-uniform */                                             \
        const uint32_t any = in ? fold(D, L, M, km) : 0u;                                                      \
        __builtin_amdgcn_sched_barrier(0);                                                                     \
        load_masks_buf<THREADS, U>(M, rm, vb + ((K) + 2) * kStep);                                             \
        load_batch_buf<THREADS, U>(D, rl, vb + ((K) + 2) * kStep);                                             \
        __builtin_amdgcn_sched_barrier(0);                                                                     \
        entries(LN, MN);                                                                                       \
        if (in)                                                                                                \
            reduce(km, any, vb + (K) * kStep);                                                                 \
    }
            for (int vb = v0; vb < v1; vb += 2 * kStep) {
                DV_STREAM_BATCH(da, la, lb, ma, mb, 0)
                DV_STREAM_BATCH(db, lb, la, mb, ma, 1)
                best_ns = ns_row[best_idx];  // as above
            }
#undef DV_STREAM_BATCH
        } else if constexpr (MASKED && !SHIFTED) {
            // Mask bytes two batches ahead of their logits: each batch from
            // the third on is issued with its vectors' offsets chosen by
            // them, so a vector with no allowed token is not read.  Four
            // batches per trip, so no register holding a load in flight is
            // ever copied (a copy would wait for the load).
            const __amdgpu_buffer_rsrc_t rl = raw_buffer(vrow, (uint32_t)v1 * 16u);
            const __amdgpu_buffer_rsrc_t rm = raw_buffer(mbytes - moff, (uint32_t)v1);
            uint32_t mc[U], md[U];
            // (the mask bytes that choose the third and fourth batches are
            // issued ahead of the second batch, so choosing them waits for
            // no logits)
            load_masks_buf<THREADS, U>(ma, rm, v0);
            load_masks_buf<THREADS, U>(mb, rm, v0 + kStep);
            load_masks_buf<THREADS, U>(mc, rm, v0 + 2 * kStep);
            load_masks_buf<THREADS, U>(md, rm, v0 + 3 * kStep);
            __builtin_amdgcn_sched_barrier(0);
            load_batch_buf<THREADS, U>(db, rl, v0 + kStep);
            __builtin_amdgcn_sched_barrier(0);
            entries(la, ma);
#define DV_AHEAD2_BATCH(D, L, LN, M, MN, MSEL, K)                                                              \
    {                                                                                                          \
        uint32_t km[4 * U];                                                                                    \
        const bool in = vb + (K) * kStep < v1; /* block-uniform */                                             \
        const uint32_t any = in ? fold(D, L, M, km) : 0u;                                                      \
        __builtin_amdgcn_sched_barrier(0);                                                                     \
        load_batch_buf_sel<THREADS, U>(D, rl, vb + ((K) + 2) * kStep, MSEL);                                   \
        __builtin_amdgcn_sched_barrier(0);                                                                     \
        load_masks_buf<THREADS, U>(M, rm, vb + ((K) + 4) * kStep);                                             \
        __builtin_amdgcn_sched_barrier(0);                                                                     \
        entries(LN, MN);                                                                                       \
        if (in)                                                                                                \
            reduce(km, any, vb + (K) * kStep);                                                                 \
    }
            for (int vb = v0; vb < v1; vb += 4 * kStep) {
                DV_AHEAD2_BATCH(da, la, lb, ma, mb, mc, 0)
                DV_AHEAD2_BATCH(db, lb, la, mb, mc, md, 1)
                DV_AHEAD2_BATCH(da, la, lb, mc, md, ma, 2)
                DV_AHEAD2_BATCH(db, lb, la, md, ma, mb, 3)
                best_ns = ns_row[best_idx];  // as above
            }
#undef DV_AHEAD2_BATCH
        } else {
            // rows of any alignment, and the unmasked scan: the same parts
            // in sequence, the next batch's loads issued ahead of each
            auto process_batch = [&](const uint4 (&d)[U], uint32_t (&m)[U], int vb) {
                live(m, vb);
                uint4 l[U];
                entries(l, m);
                uint32_t km[4 * U];
                const uint32_t any = fold(d, l, m, km);
                reduce(km, any, vb);
            };
            load_masks(ma, v0);
            for (int vb = v0; vb < v1; vb += 2 * kStep) {
                load_batch_bf16<THREADS, U>(db, vrow, vb + kStep, v1);
                load_masks(mb, vb + kStep);
                process_batch(da, ma, vb);
                load_batch_bf16<THREADS, U>(da, vrow, vb + 2 * kStep, v1);
                load_masks(ma, vb + 2 * kStep);
                if (vb + kStep < v1)  // block-uniform
                    process_batch(db, mb, vb + kStep);
                best_ns = ns_row[best_idx];  // as above
            }
        }
    }
    if (first)
        scan_exact<1, THREADS, MASKED>(row, arow, 0, rs.head, lane_key, lane_idx);
    if (last)
        scan_exact<1, THREADS, MASKED>(row, arow, rs.head + rs.nvec * kVec, V, lane_key, lane_idx);
    const uint64_t mine = pack(lane_key, lane_idx);
    const uint64_t vec_best = pack(best_key, best_idx);
    vec_pack = vec_best;
    vec_ns = best_ns;
    return vec_best > mine ? vec_best : mine;
}

// The scan of a row's chunk with the right mask alignment (block-uniform).
// ANY_ALIGN false: the caller has checked that every row is 16-byte aligned,
// so only the aligned scan is compiled (fewer registers: more resident
// blocks where several share a CU).
template <int THREADS, int U, bool MASKED, bool ANY_ALIGN, bool STAGED, bool SELECT, bool AHEAD2 = false>
__device__ __forceinline__ uint64_t scan_chunk_bf16(const char *row, const uint32_t *arow, const uint8_t *mbytes,
                                                    int moff, const int32_t *ns_row, RowSplit rs, int v0, int v1,
                                                    bool first, bool last, int V, const uint4 *lut, uint4 (&da)[U],
                                                    uint4 (&db)[U], uint64_t &vec_pack, int &vec_ns)
{
    if (!ANY_ALIGN || rs.head == 0)
        return scan_bf16<THREADS, U, MASKED, false, STAGED, SELECT, AHEAD2>(
            row, arow, mbytes, moff, ns_row, rs, v0, v1, first, last, V, lut, da, db, vec_pack, vec_ns);
    return scan_bf16<THREADS, U, MASKED, true, STAGED, SELECT>(row, arow, mbytes, moff, ns_row, rs, v0, v1, first,
                                                               last, V, lut, da, db, vec_pack, vec_ns);
}

// Mask words staged per block: the chunk's mask bytes (one per vector, plus
// one for a shifted head) in at most kStageWords words, so chunks are capped
// at kStepMaxChunkVec vectors.
constexpr int kStageWords = kStepStageWords;

// Copies allow-row words [w0, w0 + nwords) (nwords <= kStageWords) of `arow`
// (a row of W words) into LDS: every lane's loads first (clamped into the
// row, branch-free), then `between` (loads that must not queue behind the
// LDS writes' waits), then the writes.
template <int THREADS, typename F>
__device__ __forceinline__ void stage_mask_words(uint32_t *lds, const uint32_t *arow, int w0, int nwords, int W,
                                                 F between)
{
    constexpr int kPerLane = kStageWords / THREADS;
    static_assert(kPerLane * THREADS == kStageWords, "whole words per lane");
    uint32_t t[kPerLane];
#pragma unroll
    for (int k = 0; k < kPerLane; ++k)
        t[k] = arow[min(w0 + min(k * THREADS + (int)threadIdx.x, nwords - 1), W - 1)];
    between();
#pragma unroll
    for (int k = 0; k < kPerLane; ++k) {
        const int i = k * THREADS + (int)threadIdx.x;
        if (i < nwords)
            lds[i] = t[k];
    }
}

// LDS bytes of a launch's staged mask words (chunks of chunk_vec vectors).
inline size_t staged_mask_bytes(int chunk_vec) { return ((size_t)chunk_vec / 4 + 1) * 4; }

template <int THREADS, int U, bool ANY_ALIGN, bool SELECT, bool AHEAD2>
__global__ __launch_bounds__(THREADS) void masked_step_bf16_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, RowMap map, int chunk_vec,
    int nchunks, int32_t *__restrict__ token, int32_t *__restrict__ new_state, RowMeet meet)
{
    extern __shared__ uint32_t staged[];  // the chunk's mask words
    __shared__ uint4 lut[256];
    const int b = blockIdx.x / nchunks;
    const int c = blockIdx.x - b * nchunks;
    const char *row = static_cast<const char *>(logits) + (size_t)map.offset(b) * 2;
    const RowSplit rs = split_row(row, V);  // block-uniform
    const int v0 = c * chunk_vec;            // a multiple of 4: staging starts at word v0 / 4
    const int v1 = min(rs.nvec, v0 + chunk_vec);
    const char *vrow = row + 2 * rs.head;

    // The first batch of logits does not depend on the row's state: it is in
    // flight before the state lookup returns.  With SELECT the chunk's mask
    // bytes are then staged in LDS (their loads issued ahead of the second
    // batch, so waiting for them does not wait for it) and vectors with no
    // allowed token are not read; without, mask bytes stream beside their
    // logits.  Either way the mask table is built meanwhile.
    uint4 da[U], db[U];
    if (v0 < v1)
        load_batch_bf16<THREADS, U>(da, vrow, v0, v1);
    const int s = row_state(states, map, next_state, allow, S, V, b);
    const bool live = (uint32_t)s < (uint32_t)S;  // block-uniform
    const uint32_t *arow = allow + (size_t)(live ? s : 0) * W;
    uint64_t mine = 0, vec_pack = 0;
    int vec_ns = kNsUnknown;
    if constexpr (SELECT) {
        // The streaming scan is reached only on this path, so the loads the
        // compiler sees in flight at its loop head are the two batches'.
        if (live && v0 < v1) {
            const int w0 = v0 >> 2, nwords = min(W, (v1 >> 2) + 1) - w0;  // bytes v0 .. v1
            stage_mask_words<THREADS>(staged, arow, w0, nwords, W,
                                      [&] { load_batch_bf16<THREADS, U>(db, vrow, v0 + THREADS * U, v1); });
            fill_lut(lut);
            lds_barrier();
            mine = scan_chunk_bf16<THREADS, U, true, ANY_ALIGN, true, true>(
                row, arow, reinterpret_cast<const uint8_t *>(staged), v0, next_state + (size_t)s * V, rs, v0, v1,
                c == 0, c == nchunks - 1, V, lut, da, db, vec_pack, vec_ns);
        } else if (live) {  // no whole vector in this chunk: the head and tail elements only
            uint32_t key = 0;
            int idx = 0;
            if (c == 0)
                scan_exact<1, THREADS>(row, arow, 0, rs.head, key, idx);
            if (c == nchunks - 1)
                scan_exact<1, THREADS>(row, arow, rs.head + rs.nvec * 8, V, key, idx);
            mine = pack(key, idx);
        }
    } else {
        // Mask bytes read from the allow row batch by batch, right behind
        // their logits: nothing to wait for before the first batch.
        fill_lut(lut);
        lds_barrier();
        if (live)
            mine = scan_chunk_bf16<THREADS, U, true, ANY_ALIGN, false, false, AHEAD2>(
                row, arow, reinterpret_cast<const uint8_t *>(arow), 0, next_state + (size_t)s * V, rs, v0, v1,
                c == 0, c == nchunks - 1, V, lut, da, db, vec_pack, vec_ns);
    }
    int ns;
    const uint64_t best = block_max_ns<THREADS>(mine, vec_pack, vec_ns, ns);
    if (threadIdx.x != 0)
        return;
    const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
    const bool found = tok >= 0 && tok < V;  // always true for a found token; guards the read
    const int nsv = !found ? -1 : ns != kNsUnknown ? ns : next_state[(size_t)s * V + tok];
    if (nchunks == 1) {
        token[b] = found ? tok : -1;
        new_state[b] = nsv;
        return;
    }
    // Split rows: the meeting word carries the winner's next state, so the
    // block that arrives last needs no further read.
    uint64_t fin;
    if (!meet_row(meet, b, c, nchunks, found ? pack_split(best, tok, nsv) : 0ull, fin))
        return;  // another block of the row finishes it
    int ftok, fns;
    unpack_split(fin, ftok, fns);
    token[b] = ftok;
    new_state[b] = fns != kNsUnknown ? fns : next_state[(size_t)s * V + ftok];
}

// Opportunistic masking (Sec. 3.5, further optimizations), one block per
// row: the model's own choice over the whole row is found first, without
// reading the mask; only when the mask does not allow it is the row scanned
// again with the mask.  Same result as masked_step_bf16_kernel.
template <int THREADS, int U, bool ANY_ALIGN>
__global__ __launch_bounds__(THREADS) void opportunistic_step_bf16_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V, int W,
    const int32_t *__restrict__ states, const void *__restrict__ logits, RowMap map,
    int32_t *__restrict__ token, int32_t *__restrict__ new_state)
{
    __shared__ uint4 lut[256];
    __shared__ int miss;
    const int b = blockIdx.x;
    const char *row = static_cast<const char *>(logits) + (size_t)map.offset(b) * 2;
    const RowSplit rs = split_row(row, V);  // block-uniform

    uint4 da[U], db[U];  // db: scratch of the scan
    if (rs.nvec > 0)
        load_batch_bf16<THREADS, U>(da, row + 2 * rs.head, 0, rs.nvec);
    const int s = states[b];
    fill_lut(lut);
    lds_barrier();
    const bool live = (uint32_t)s < (uint32_t)S;  // block-uniform
    const uint32_t *arow = allow + (size_t)(live ? s : 0) * W;
    const int32_t *ns_row = next_state + (size_t)(live ? s : 0) * V;
    uint64_t mine = 0, vec_pack = 0;
    int vec_ns = kNsUnknown, ns;
    if (live)
        mine = scan_chunk_bf16<THREADS, U, false, ANY_ALIGN, false, false>(
            row, arow, reinterpret_cast<const uint8_t *>(arow), 0, ns_row, rs, 0, rs.nvec, true, true, V, lut, da, db,
            vec_pack, vec_ns);
    uint64_t best = block_max_ns<THREADS>(mine, vec_pack, vec_ns, ns);
    if (threadIdx.x == 0) {
        const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
        const bool ok = tok >= 0 && tok < V && ((arow[tok >> 5] >> (tok & 31)) & 1u);
        miss = live && !ok;
    }
    __syncthreads();
    if (miss) {  // block-uniform
        if (rs.nvec > 0)
            load_batch_bf16<THREADS, U>(da, row + 2 * rs.head, 0, rs.nvec);
        mine = scan_chunk_bf16<THREADS, U, true, ANY_ALIGN, false, false>(
            row, arow, reinterpret_cast<const uint8_t *>(arow), 0, ns_row, rs, 0, rs.nvec, true, true, V, lut, da, db,
            vec_pack, vec_ns);
        best = block_max_ns<THREADS>(mine, vec_pack, vec_ns, ns);
    }
    if (threadIdx.x != 0)
        return;
    const int tok = best ? (int)(0xFFFFFFFFu - (uint32_t)best) : -1;
    const bool found = live && tok >= 0 && tok < V;  // guards the read
    token[b] = found ? tok : -1;
    new_state[b] = !found ? -1 : ns != kNsUnknown ? ns : next_state[(size_t)s * V + tok];
}

}  // namespace

// Whether a bf16 launch of `blocks` blocks stages its mask bytes in LDS and
// skips lines with no allowed token.  Staging puts the whole chunk's mask
// row ahead of the first reduction; with two or more blocks per compute
// unit other blocks hide that and the saved bytes win (B = 1024 x V =
// 256000: 82 against 85 us per step), with one block per unit it shows
// (B = 256 x V = 128256: 15.0 against 13.9 us).
// Chunks of at least 8 batches per lane (8 x 512 lanes x 2 vectors = 64K
// tokens) instead choose their loads from mask bytes read two batches ahead
// when the launch has at most four blocks per compute unit (B = 1024 x V =
// 256000: 80.4-81.0 against 82.3 us; the speculative verification of B =
// 64 x 9 positions x V = 128256 24.7 against 28.6); at nine per unit the
// staged form, with fewer registers and so more resident blocks, stays
// ahead (B = 256 x 9 x 128256: 70.2-70.7 against 71.9-72.5).  Shorter
// chunks are over before the two-ahead form pays for its longer start.
constexpr int kAhead2MinVec = 8 * kBigThreads * kBigU;

static bool skip_unread_lines(unsigned blocks)
{
    const int n = device_compute_units();  // unknown: never skip
    return n > 0 && blocks >= 2u * (unsigned)n;
}

hipError_t launch_masked_rows(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int B,
                              RowMap map, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    const int W = (V + 31) / 32;
    const StepGeometry g = step_geometry(B, V, dtype);
    const RowMeet meet = row_meet(workspace, B);
    const unsigned grid = (unsigned)B * (unsigned)g.nchunks;
    if (dtype == 0)
        masked_step_kernel<kSmallThreads, kSmallU><<<grid, kSmallThreads, 0, stream>>>(
            next_state, allow, S, V, W, states, logits, map, g.chunk_vec, g.nchunks, token, new_state, meet);
    else {
        const bool aligned = map.rows_aligned(logits, 2);
        // long chunks at up to four blocks per compute unit choose their
        // loads from mask bytes read two batches ahead; more blocks per unit
        // stage the mask bytes in LDS (the two-ahead scan's registers allow
        // fewer resident blocks)
        const int cus = device_compute_units();
        const bool ahead2 = g.chunk_vec >= kAhead2MinVec && (cus <= 0 || grid <= 4u * (unsigned)cus);
        const bool select = !ahead2 && skip_unread_lines(grid);
        const size_t lds = select ? staged_mask_bytes(g.chunk_vec) : 0;
#define DV_STEP_BF16(A, SEL, A2)                                                                               \
    masked_step_bf16_kernel<kBigThreads, kBigU, A, SEL, A2><<<grid, kBigThreads, lds, stream>>>(              \
        next_state, allow, S, V, W, states, logits, map, g.chunk_vec, g.nchunks, token, new_state, meet)
        if (aligned && select)
            DV_STEP_BF16(false, true, false);
        else if (aligned && ahead2)
            DV_STEP_BF16(false, false, true);
        else if (aligned)
            DV_STEP_BF16(false, false, false);
        else if (select)
            DV_STEP_BF16(true, true, false);
        else if (ahead2)
            DV_STEP_BF16(true, false, true);
        else
            DV_STEP_BF16(true, false, false);
#undef DV_STEP_BF16
    }
    return hipGetLastError();
}

hipError_t launch_masked_step_opportunistic(const int32_t *next_state, const uint32_t *allow, int S, int V,
                                            const int32_t *states, const void *logits, int dtype, int B,
                                            int64_t ld, int32_t *token, int32_t *new_state,
                                            void *workspace, hipStream_t stream)
{
    // Where a bf16 row is one block the check runs first; elsewhere (fp32
    // rows, rows split over several blocks, where checking first would need
    // an extra pass over the chunks) the plain masked step gives the same
    // result.
    if (dtype == 1 && step_geometry(B, V, 1).nchunks == 1) {
        const RowMap map{ld, 0, 1, nullptr, 0};
        if (map.rows_aligned(logits, 2))
            opportunistic_step_bf16_kernel<kBigThreads, kBigU, false><<<(unsigned)B, kBigThreads, 0, stream>>>(
                next_state, allow, S, V, (V + 31) / 32, states, logits, map, token, new_state);
        else
            opportunistic_step_bf16_kernel<kBigThreads, kBigU, true><<<(unsigned)B, kBigThreads, 0, stream>>>(
                next_state, allow, S, V, (V + 31) / 32, states, logits, map, token, new_state);
        return hipGetLastError();
    }
    return launch_masked_rows(next_state, allow, S, V, states, logits, dtype, B, RowMap{ld, 0, 1, nullptr, 0}, token,
                              new_state, workspace, stream);
}

hipError_t launch_masked_step(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int B,
                              int64_t ld, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    return launch_masked_rows(next_state, allow, S, V, states, logits, dtype, B, RowMap{ld, 0, 1, nullptr, 0}, token,
                              new_state, workspace, stream);
}

}  // namespace dv
