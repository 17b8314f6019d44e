// Vocabulary alignment on CDNA4 (gfx950): for every DFA state and every
// token, walk the token's bytes through the DFA (Sec. 3.3 / Algorithm 2 at
// full depth, Sec. 3.5).  Output next_state[S][V] int32 and the allow
// bitmask [S][ceil(V/32)] uint32.
//
// Pipeline (all on the caller's stream, no host synchronisation):
//   1. live_columns: which byte columns have at least one live move.
//   2. byte_classes: rank the live columns; dead columns get no storage.
//   3. compact: uint16 table [S][Cp] over the live columns only (DEAD = 0xFFFF).
//      Random printable-ASCII DFAs keep ~95 of 256 columns, so the table is
//      ~2.7x smaller than the int32 input and stays resident in each XCD's L2.
//   4. walk: one lane per (state, token) pair.  A block owns a tile of 32
//      states x 1024 tokens: the 32 compacted rows are staged in LDS, so the
//      first move of every walk (every pair takes it) is an LDS read; later
//      moves (about half the pairs survive each byte) read the L2-resident
//      compacted table.  Each lane carries 4 tokens whose walks advance in
//      lock-step for memory-level parallelism; the wave stops as soon as all
//      64 lanes' walks have ended.  Stores are coalesced along tokens, and
//      the allow words come from a wave ballot (64 tokens -> 2 words).
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;
constexpr int kTokPerLane = 4;
constexpr int kTokTile = kThreads * kTokPerLane;  // 1024 tokens = 32 allow words
constexpr int kStateTile = 32;

__device__ __forceinline__ bool in_range(int32_t v, int S) { return (uint32_t)v < (uint32_t)S; }

// 1. per block of 64 rows: bit b set if some row has a live move on byte b.
__global__ __launch_bounds__(kThreads) void live_columns_kernel(const int32_t *__restrict__ trans,
                                                                int S, uint32_t *__restrict__ partial)
{
    const int b = threadIdx.x;
    const int r0 = blockIdx.x * kLiveRowsPerBlock;
    const int r1 = min(S, r0 + kLiveRowsPerBlock);
    bool live = false;
    for (int s = r0; s < r1; ++s)
        live |= in_range(trans[(size_t)s * 256 + b], S);
    const uint64_t m = __ballot(live);
    const int lane = b & (kWave - 1), wave = b / kWave;
    if (lane < 2)
        partial[(size_t)blockIdx.x * 8 + wave * 2 + lane] = (uint32_t)(m >> (32 * lane));
}

// 2. one block: class id of each live byte (in byte order) and the inverse map.
__global__ __launch_bounds__(kThreads) void byte_classes_kernel(const uint32_t *__restrict__ partial,
                                                                int nblocks, uint8_t *__restrict__ ws)
{
    __shared__ int wave_count[kThreads / kWave];
    const int b = threadIdx.x;
    uint32_t any = 0;
    for (int k = 0; k < nblocks; ++k)
        any |= partial[(size_t)k * 8 + b / 32];
    const bool live = (any >> (b % 32)) & 1u;
    const uint64_t m = __ballot(live);
    const int lane = b & (kWave - 1), wave = b / kWave;
    if (lane == 0)
        wave_count[wave] = __popcll(m);
    __syncthreads();
    int rank = __popcll(m & ((1ull << lane) - 1ull));
    int total = 0;
    for (int w = 0; w < kThreads / kWave; ++w) {
        if (w < wave)
            rank += wave_count[w];
        total += wave_count[w];
    }
    uint8_t *cls = ws + 256;
    uint8_t *byte_of = ws + 512;
    cls[b] = live ? (uint8_t)rank : kDeadClass;
    if (live)
        byte_of[rank] = (uint8_t)b;
    if (b == 0) {
        int32_t *meta = reinterpret_cast<int32_t *>(ws);
        meta[0] = total;
        meta[1] = (total + 1) & ~1;
    }
}

// 3. compacted uint16 table [S][Cp]; padding columns are DEAD.
__global__ __launch_bounds__(kThreads) void compact_kernel(const int32_t *__restrict__ trans, int S,
                                                           const uint8_t *__restrict__ ws,
                                                           uint16_t *__restrict__ table)
{
    const int32_t *meta = reinterpret_cast<const int32_t *>(ws);
    const int C = meta[0], Cp = meta[1];
    const int c = threadIdx.x;
    if (c >= Cp)
        return;
    const int byte = c < C ? ws[512 + c] : 0;
    const int r0 = blockIdx.x * 16;
    const int r1 = min(S, r0 + 16);
    for (int s = r0; s < r1; ++s) {
        uint16_t v = kDead16;
        if (c < C) {
            const int32_t x = trans[(size_t)s * 256 + byte];
            v = in_range(x, S) ? (uint16_t)x : kDead16;
        }
        table[(size_t)s * Cp + c] = v;
    }
}

// 4. the walk.
__global__ __launch_bounds__(kThreads) void walk_kernel(const uint8_t *__restrict__ ws,
                                                        const uint16_t *__restrict__ table, int S,
                                                        const int32_t *__restrict__ offsets,
                                                        const uint8_t *__restrict__ bytes, int V,
                                                        int W, int32_t *__restrict__ next_state,
                                                        uint32_t *__restrict__ allow)
{
    __shared__ uint16_t rows[kStateTile * 256];
    __shared__ uint8_t cls[256];

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int Cp = reinterpret_cast<const int32_t *>(ws)[1];
    const int s0 = blockIdx.y * kStateTile;
    const int nS = min(kStateTile, S - s0);
    const int t_base = blockIdx.x * kTokTile;

    cls[tid] = ws[256 + tid];
    for (int i = tid; i < nS * Cp; i += kThreads)
        rows[i] = table[(size_t)s0 * Cp + i];

    int off[kTokPerLane], len[kTokPerLane];
#pragma unroll
    for (int j = 0; j < kTokPerLane; ++j) {
        const int t = t_base + j * kThreads + tid;
        if (t < V) {
            off[j] = offsets[t];
            len[j] = offsets[t + 1] - off[j];
        } else {
            off[j] = 0;
            len[j] = -1;  // past the end: not stored, allow bit 0
        }
    }
    __syncthreads();

    int c0[kTokPerLane];
#pragma unroll
    for (int j = 0; j < kTokPerLane; ++j)
        c0[j] = len[j] > 0 ? cls[bytes[off[j]]] : kDeadClass;

    for (int si = 0; si < nS; ++si) {
        const int s = s0 + si;
        uint32_t st[kTokPerLane];
#pragma unroll
        for (int j = 0; j < kTokPerLane; ++j) {
            if (len[j] > 0)
                st[j] = c0[j] == kDeadClass ? kDead16 : rows[si * Cp + c0[j]];
            else
                st[j] = len[j] == 0 ? (uint32_t)s : kDead16;  // empty token keeps the state
        }
        for (int h = 1;; ++h) {
            bool more = false;
#pragma unroll
            for (int j = 0; j < kTokPerLane; ++j) {
                if (st[j] != kDead16 && h < len[j]) {
                    const int c = cls[bytes[off[j] + h]];
                    st[j] = c == kDeadClass ? kDead16 : table[(size_t)st[j] * Cp + c];
                    more |= st[j] != kDead16 && h + 1 < len[j];
                }
            }
            if (!__any(more))
                break;
        }
        int32_t *ns_row = next_state + (size_t)s * V;
        uint32_t *al_row = allow + (size_t)s * W;
#pragma unroll
        for (int j = 0; j < kTokPerLane; ++j) {
            const int t = t_base + j * kThreads + tid;
            const bool alive = len[j] >= 0 && st[j] != kDead16;
            if (t < V)
                ns_row[t] = alive ? (int32_t)st[j] : -1;
            const uint64_t m = __ballot(alive);
            const int w = (t_base + j * kThreads + wave * kWave) / 32 + lane;
            if (lane < 2 && w < W)
                al_row[w] = (uint32_t)(m >> (32 * lane));
        }
    }
}

}  // namespace

hipError_t launch_align(const int32_t *trans, int S, const int32_t *offsets, const uint8_t *bytes,
                        int V, int32_t *next_state, uint32_t *allow, void *workspace,
                        hipStream_t stream)
{
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    uint32_t *partial = reinterpret_cast<uint32_t *>(ws + kAlignMetaBytes);
    uint16_t *table = reinterpret_cast<uint16_t *>(ws + align_table_offset(S));
    const int nblk = (int)align_live_blocks(S);
    const int W = (V + 31) / 32;

    live_columns_kernel<<<nblk, kThreads, 0, stream>>>(trans, S, partial);
    byte_classes_kernel<<<1, kThreads, 0, stream>>>(partial, nblk, ws);
    compact_kernel<<<(S + 15) / 16, kThreads, 0, stream>>>(trans, S, ws, table);
    dim3 grid((V + kTokTile - 1) / kTokTile, (S + kStateTile - 1) / kStateTile);
    walk_kernel<<<grid, kThreads, 0, stream>>>(ws, table, S, offsets, bytes, V, W, next_state, allow);
    return hipGetLastError();
}

}  // namespace dv
