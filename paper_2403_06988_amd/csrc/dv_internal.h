// Internal declarations shared by the translation units of libdv.so.
// Not installed; the public interface is include/dv.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace dv {

constexpr int kWave = 64;

// ---------------------------------------------------------- wave reductions
//
// Maximum or minimum over the 64 lanes of a wave, the same value returned in
// every lane: inside each 16-lane row by DPP moves (swap neighbours in a
// quad, swap quad pairs, mirror each half-row, mirror the row: no LDS traffic
// and no waits), then across the four rows by reading lanes 0, 16, 32 and
// 48.  Every lane of the wave must be active.
constexpr int kDppQuadSwap1 = 0xB1;       // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadSwap2 = 0x4E;       // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;  // lane i of each 8 reads lane 7 - i
constexpr int kDppRowMirror = 0x140;      // lane i of each 16 reads lane 15 - i

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_move(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, false);
}

template <bool MAX, typename T>
__device__ __forceinline__ T pick(T a, T b)
{
    return MAX ? (a > b ? a : b) : (a < b ? a : b);
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_move64(uint64_t v)
{
    return (uint64_t)dpp_move<CTRL>((uint32_t)(v >> 32)) << 32 | dpp_move<CTRL>((uint32_t)v);
}

__device__ __forceinline__ uint32_t lane_value(uint32_t v, int lane)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ uint64_t lane_value(uint64_t v, int lane)
{
    return (uint64_t)lane_value((uint32_t)(v >> 32), lane) << 32 | lane_value((uint32_t)v, lane);
}

template <bool MAX, typename T>
__device__ __forceinline__ T wave_reduce(T v)
{
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit lanes");
    if constexpr (sizeof(T) == 4) {
        v = pick<MAX>(v, (T)dpp_move<kDppQuadSwap1>(v));
        v = pick<MAX>(v, (T)dpp_move<kDppQuadSwap2>(v));
        v = pick<MAX>(v, (T)dpp_move<kDppRowHalfMirror>(v));
        v = pick<MAX>(v, (T)dpp_move<kDppRowMirror>(v));
    } else {
        v = pick<MAX>(v, (T)dpp_move64<kDppQuadSwap1>(v));
        v = pick<MAX>(v, (T)dpp_move64<kDppQuadSwap2>(v));
        v = pick<MAX>(v, (T)dpp_move64<kDppRowHalfMirror>(v));
        v = pick<MAX>(v, (T)dpp_move64<kDppRowMirror>(v));
    }
    return pick<MAX>(pick<MAX>((T)lane_value(v, 0), (T)lane_value(v, 16)),
                     pick<MAX>((T)lane_value(v, 32), (T)lane_value(v, 48)));
}

// Compute units of the current device (read once per device), or -1 when
// the runtime cannot say: launch shapes that depend on it fall back to
// their plain form.
inline int device_compute_units()
{
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cus[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return -1;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
            n = -1;
        cus[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// Lanes of one wave hand data to each other through LDS: the wave's LDS
// operations run in order, so a compiler barrier with wavefront-scope
// ordering is all that is needed (no block barrier: waves do not wait for
// each other).
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ---------------------------------------------------------------- alignment
//
// Workspace of dv_align (all offsets 256-byte aligned):
//   [0, 4)        int32  number of live byte columns C
//   [4, 8)        int32  row stride Cp of the compacted table (C + 1 rounded up
//                        to even; 256 when every byte is live)
//   [256, 512)    uint8  class of each byte (the bytes dead from every state
//                        share class C, whose table column is all DEAD)
//   [512, 768)    uint8  byte of each class
//   [1024, ...)   uint32 per-block live-column bit sets, 8 words per block
//   [table, ...)  uint16 compacted table [S][Cp], DEAD = 0xFFFF
//   [tokinfo, ...) uint4 per token: classes of bytes 0-3, 4-7, length, offset
constexpr int kAlignMetaBytes = 1024;
constexpr int kLiveRowsPerBlock = 16;
constexpr uint16_t kDead16 = 0xFFFF;

constexpr size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline size_t align_live_blocks(int S) { return (size_t)(S + kLiveRowsPerBlock - 1) / kLiveRowsPerBlock; }
inline size_t align_table_offset(int S) { return align_up(kAlignMetaBytes + align_live_blocks(S) * 32, 256); }
inline size_t align_tokinfo_offset(int S) { return align_up(align_table_offset(S) + (size_t)S * 256 * sizeof(uint16_t), 256); }
// per token: byte classes of its first 8 bytes (4 per word), its length, its offset
inline size_t align_workspace_bytes(int S, int V) { return align_tokinfo_offset(S) + (size_t)V * 16; }

// first_bad <- the smallest t at which the CSR layout of the vocabulary
// breaks, or -1 (dv_validate_vocab).
hipError_t launch_validate_vocab(const int32_t *offsets, int V, int64_t num_bytes, int32_t *first_bad,
                                 hipStream_t stream);

// eos_token = -1: no end-of-sequence token; accepting may then be NULL.
hipError_t launch_align(const int32_t *trans, int S, const int32_t *offsets, const uint8_t *bytes,
                        int V, const uint8_t *accepting, int eos_token, int32_t *next_state,
                        uint32_t *allow, void *workspace, hipStream_t stream);

// ----------------------------------------------------- split rows meet here
//
// When a row is split over several blocks, the blocks meet in the
// workspace, whose words are all zero between calls; one lane per block
// takes part, and no block ever waits for another.
//
// Up to kMeetTreeChunks chunks the blocks meet in pairs, as a binary tree
// over the chunk indices: per row nchunks - 1 64-bit words, pair p of
// level l at word (pairs below level l) + p.  A block folds its value into
// its pair's word with a device-scope atomic maximum; the block that
// finds the word zero arrived first and leaves, the other one has both
// values (the maximum of the old word and its own), puts the word back to
// zero and goes on to the next level; a chunk without a partner at a level
// (an odd count) goes on without a trip.  The value of a block with
// nothing allowed is 1, which every found value exceeds, so that zero
// always means "not arrived".  The last block thus learns the row's
// maximum after ceil(log2 nchunks) round trips, one per level.
//
// More chunks use two words per row: a 64-bit maximum and a 32-bit count
// of the blocks that have arrived.  Each block folds its value into the
// maximum and then counts itself; the block that arrives last reads the
// maximum and puts both back to zero: three round trips.
//
// Layout: pairs [B][nchunks - 1] uint64 from 0 (up to kMeetTreeChunks
// chunks); otherwise best [B] uint64 at 0 and arrived [B] uint32 at
// row_meet_count_offset.
constexpr int kMeetTreeChunks = 4;
constexpr size_t row_meet_count_offset(int B) { return align_up((size_t)(B > 0 ? B : 1) * 8, 256); }
constexpr size_t row_meet_bytes(int B) { return row_meet_count_offset(B) + align_up((size_t)(B > 0 ? B : 1) * 4, 256); }
// the bytes a launch of B rows split into nchunks chunks needs (either layout)
constexpr size_t row_meet_bytes(int B, int nchunks)
{
    const size_t pairs = nchunks >= 2 && nchunks <= kMeetTreeChunks
                             ? align_up((size_t)(B > 0 ? B : 1) * (size_t)(nchunks - 1) * 8, 256)
                             : 0;
    return pairs > row_meet_bytes(B) ? pairs : row_meet_bytes(B);
}

struct RowMeet {
    uint64_t *best;
    uint32_t *arrived;
};

inline RowMeet row_meet(void *workspace, int B)
{
    char *w = static_cast<char *>(workspace);
    return {reinterpret_cast<uint64_t *>(w), reinterpret_cast<uint32_t *>(w + row_meet_count_offset(B))};
}

// Called by one lane of each of the `nchunks` (>= 2) blocks of row b (this
// block holds chunk c) with the block's best value, 0 when it found nothing.
// All updates are device-scope atomics (performed where every XCD sees
// them); each step's operand depends on the value the previous one
// returned.  Returns true in the block that finishes the row, with the
// row's maximum in `fin` (0 when nothing was found) and the row's words
// back at zero.
__device__ __forceinline__ bool meet_row(RowMeet m, int b, int c, int nchunks, uint64_t best, uint64_t &fin)
{
    if (nchunks <= kMeetTreeChunks) {
        static_assert(kMeetTreeChunks == 4, "two levels at most");
        uint64_t *pairs = m.best + (size_t)b * (size_t)(nchunks - 1);
        uint64_t v = best ? best : 1ull;
        // level 1: chunks 2k and 2k + 1 at word k (with three chunks, chunk 2
        // has no partner there); level 2: the two survivors at word n / 2
        if (nchunks != 3 || c < 2) {
            uint64_t *w = pairs + (c >> 1);
            const uint64_t other = __hip_atomic_fetch_max(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (!other)
                return false;  // the partner carries both values on
            (void)__hip_atomic_exchange(w, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            v = other > v ? other : v;
        }
        if (nchunks > 2) {
            uint64_t *w = pairs + (nchunks >> 1);
            const uint64_t other = __hip_atomic_fetch_max(w, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (!other)
                return false;
            (void)__hip_atomic_exchange(w, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            v = other > v ? other : v;
        }
        fin = v == 1ull ? 0ull : v;
        return true;
    }
    const uint64_t before = __hip_atomic_fetch_max(m.best + b, best, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    uint32_t one = 1u;
    asm volatile("" : "+v"(one) : "v"(before) : "memory");
    const uint32_t n = __hip_atomic_fetch_add(m.arrived + b, one, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (n != (uint32_t)nchunks - 1u)
        return false;
    fin = __hip_atomic_exchange(m.best + b, (uint64_t)0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    (void)__hip_atomic_exchange(m.arrived + b, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
}

// ------------------------------------------------------------- masked step
//
// A row of V logits is split into `nchunks` chunks of `chunk_vec` 16-byte
// vectors, one block of `threads` lanes each; with more than one chunk the
// blocks meet in the workspace (above).  bf16 rows use 512-lane blocks, one
// per row once B >= kStepOneBlockRows (a block per compute unit already) or
// when B >= 64 and a row holds at most kStepSingleBlockRowBytes (a second
// block per row buys nothing there); otherwise about 32 / sqrt(B) chunks per
// row.  fp32 rows use 256-lane blocks and the same chunk rule.
constexpr int kStepOneBlockRows = 256;
constexpr int kStepSmallThreads = 256;   // fp32 rows
constexpr int kStepBigThreads = 512;     // bf16 rows
constexpr int kStepStageWords = 8192;    // mask words a bf16 block may stage in LDS
constexpr int kStepMaxChunkVec = (kStepStageWords - 1) * 4 / kStepBigThreads * kStepBigThreads;
constexpr int64_t kStepSingleBlockRowBytes = 65536;
static_assert(kStepMaxChunkVec % kStepBigThreads == 0, "chunks are whole batches of lanes");

struct StepGeometry {
    int chunk_vec;
    int nchunks;
    int threads;
};

inline StepGeometry step_geometry(int B, int V, int dtype)
{
    const bool bf16 = dtype == 1;
    const int vec = bf16 ? 8 : 4;  // elements per 16-byte vector
    const int threads = bf16 ? kStepBigThreads : kStepSmallThreads;
    const int nvec = V / vec;
    int want;
    if (bf16 && B >= kStepOneBlockRows) {
        want = 1;
    } else if (bf16 && B >= 64 && (int64_t)V * 2 <= kStepSingleBlockRowBytes) {
        want = 1;
    } else {
        // Chunks per row ~ 32 / sqrt(B): about 32 sqrt(B) blocks per launch
        // (at most 256).  Since split rows meet in the workspace instead of a
        // second kernel, this is what measures fastest from B = 1 to 128 at
        // V = 32000 .. 256000: fewer blocks leave bandwidth unused, more
        // make each block's stream too short for its fixed start-up cost.
        int r = 1;
        while (r * r < B)
            ++r;  // ceil(sqrt(B))
        const int blocks = 32 * r < 256 ? 32 * r : 256;
        want = (blocks + B / 2) / (B > 0 ? B : 1);
    }
    // at least one vector per lane per chunk
    const int max_chunks = nvec / threads > 1 ? nvec / threads : 1;
    want = want > max_chunks ? max_chunks : want;
    want = want < 1 ? 1 : want;
    int chunk_vec = (nvec + want - 1) / want;
    chunk_vec = (chunk_vec + threads - 1) / threads * threads;
    if (chunk_vec == 0)
        chunk_vec = threads;
    if (bf16 && chunk_vec > kStepMaxChunkVec)  // the staged mask bytes must fit
        chunk_vec = kStepMaxChunkVec;
    int nchunks = (nvec + chunk_vec - 1) / chunk_vec;
    if (nchunks < 1)
        nchunks = 1;
    return {chunk_vec, nchunks, threads};
}

// either dtype's launch shape
inline size_t step_workspace_bytes(int B, int V)
{
    const size_t a = row_meet_bytes(B, step_geometry(B, V, 0).nchunks);
    const size_t b = row_meet_bytes(B, step_geometry(B, V, 1).nchunks);
    return a > b ? a : b;
}

hipError_t launch_masked_step(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int B,
                              int64_t ld, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream);

// Opportunistic masking: the same outputs as launch_masked_step (and the
// same workspace).
hipError_t launch_masked_step_opportunistic(const int32_t *next_state, const uint32_t *allow, int S, int V,
                                            const int32_t *states, const void *logits, int dtype, int B,
                                            int64_t ld, int32_t *token, int32_t *new_state,
                                            void *workspace, hipStream_t stream);

// How the rows of a masked-step launch map to logits and states.  Rows come
// in groups of `per` (a sequence's positions): row r is position j = r % per
// of group g = r / per.  Its logits start at element g * ld_row + j * ld_pos;
// its state is the group's state advanced by the group's first j proposals
// prop[g * ld_prop + i] (DEAD once one is not allowed).  A plain batch is
// {ld, 0, 1, nullptr, 0}: row r's state is states[r].
struct RowMap {
    int64_t ld_row;
    int64_t ld_pos;
    int per;
    const int32_t *prop;
    int64_t ld_prop;
    __host__ __device__ int64_t offset(int r) const
    {
        if (per == 1)  // a plain batch: no division ahead of the first loads
            return (int64_t)r * ld_row;
        const int g = r / per;
        return (int64_t)g * ld_row + (int64_t)(r - g * per) * ld_pos;
    }
    // Every row of `base` starts on a 16-byte boundary.
    bool rows_aligned(const void *base, int elt) const
    {
        return reinterpret_cast<uintptr_t>(base) % 16 == 0 && (ld_row * elt) % 16 == 0 &&
               (per == 1 || (ld_pos * elt) % 16 == 0);
    }
};

// One move of the speculative chain: the state after proposal t from state
// st (-1 if st is DEAD, t is not a token id or its allow bit is clear; a
// table entry outside [0, S) also reads as -1).  The mask word and the
// table entry are loaded together at clamped addresses.
__device__ __forceinline__ int spec_hop(const int32_t *next_state, const uint32_t *allow, int S, int V, int st,
                                        int t, bool &legal)
{
    const bool ok = st >= 0 && (uint32_t)t < (uint32_t)V;
    const size_t si = ok ? (size_t)st : 0, ti = ok ? (size_t)t : 0;
    const size_t W = ((size_t)V + 31) / 32;
    const uint32_t word = allow[si * W + (ti >> 5)];
    const int nx = next_state[si * (size_t)V + ti];
    legal = ok && ((word >> (ti & 31)) & 1u);
    return legal && (uint32_t)nx < (uint32_t)S ? nx : -1;
}

// State of row r under `m` (for a plain batch the raw states[r]; the caller
// treats anything outside [0, S) as DEAD).
__device__ __forceinline__ int row_state(const int32_t *states, const RowMap &m, const int32_t *next_state,
                                         const uint32_t *allow, int S, int V, int r)
{
    if (m.per == 1)
        return states[r];
    const int g = r / m.per, j = r - g * m.per;
    int st = states[g];
    st = (uint32_t)st < (uint32_t)S ? st : -1;
    const int32_t *p = m.prop + (size_t)g * (size_t)m.ld_prop;
    for (int i = 0; i < j; ++i) {
        bool legal;
        st = spec_hop(next_state, allow, S, V, st, p[i], legal);
    }
    return st;
}

// The masked step over R rows addressed through `map` (workspace as above,
// for R rows).
hipError_t launch_masked_rows(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const void *logits, int dtype, int R,
                              RowMap map, int32_t *token, int32_t *new_state, void *workspace,
                              hipStream_t stream);

// ------------------------------------------------ speculative chain check
//
// Workspace of the verification, for B rows of s proposals (R = B (s + 1)
// positions), 256-byte aligned parts:
//   [0, ...)     int32 state after each position's choice [B][s+1]
//   [meet..)     the masked step's workspace for R rows (zero between calls)
inline size_t spec_positions(int B, int s) { return (size_t)B * (size_t)(s + 1); }
inline size_t spec_partial_offset(int B, int s) { return align_up(spec_positions(B, s) * 4, 256); }
inline size_t spec_workspace_bytes(int B, int s, int V)
{
    return spec_partial_offset(B, s) + step_workspace_bytes((int)spec_positions(B, s), V);
}

hipError_t launch_spec_walk(const int32_t *next_state, const uint32_t *allow, int S, int V,
                            const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                            int B, int32_t *accepted, int32_t *final_state, hipStream_t stream);

hipError_t launch_spec_verify(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                              const void *logits, int dtype, int64_t ld_row, int64_t ld_pos, int B,
                              int32_t *token, int32_t *accepted, int32_t *new_state, void *workspace,
                              hipStream_t stream);

}  // namespace dv
