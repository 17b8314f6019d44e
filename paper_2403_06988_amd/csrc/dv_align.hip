// Vocabulary alignment on CDNA4 (gfx950): for every DFA state and every
// token, walk the token's bytes through the DFA (Sec. 3.3 / Algorithm 2 at
// full depth, Sec. 3.5).  Output next_state[S][V] int32 and the allow
// bitmask [S][ceil(V/32)] uint32.
//
// Pipeline (all on the caller's stream, no host synchronisation):
//   1. live_columns: which byte columns have at least one live move.
//   2. byte_classes: rank the live columns; the bytes dead from every state
//      share one extra class whose column is all DEAD (it exists only when
//      some byte is dead, so the C <= 256 classes always fit in a byte).
//   3. compact: uint16 table [S][Cp] over the live columns, then the DEAD
//      column (DEAD = 0xFFFF).  (3 and 4 run in one launch.)
//      Random printable-ASCII DFAs keep ~95 of 256 columns, so the table is
//      ~2.7x smaller than the int32 input and stays resident in each XCD's L2.
//      The walks write their outputs (4.125 bytes per pair) with
//      non-temporal stores: that stream passes the caches by, so it neither
//      evicts the compacted table the walks gather from nor leaves the
//      caches full of dirty lines for the kernels that follow to write back.
//   4. token_info: each token's first 8 byte classes, length and offset.
//   5. walk (tables of at most 98 columns that do not fit in LDS whole, e.g.
//      random printable-ASCII DFAs of more than ~330 states): the prefix-table
//      walk, kernel 6 below.  Otherwise the tile walk: a block owns 16 states
//      x 256 tokens (one token per lane), with the whole table in LDS when it
//      fits, else the tile's 16 rows; the byte classes of each token's first
//      8 bytes are looked up once and kept in registers.  A lane walks its
//      token from 8 of the tile's states at once, one byte per iteration, so
//      a long walk is a chain of 8 independent reads per byte, not one
//      dependent read per move of every state: from LDS when the table is
//      whole (a dead state reads an all-DEAD sentinel row), else the first
//      move from the row tile and later ones from the cache-resident table
//      at 32-bit offsets (a dead state skips its read).  Stores are coalesced
//      along tokens; the allow words come from a wave ballot (64 tokens -> 2
//      words).
#include <algorithm>

#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kThreads = 256;
constexpr int kTokTile = kThreads;                // a multiple of 64 tokens = 2 allow words
constexpr int kStateTile = 16;                    // states per tile
constexpr int kLockG = 8;                         // of which a lane walks this many at once
constexpr int kRegBytes = 8;                      // token bytes whose classes sit in registers
constexpr int kRowsLds = kStateTile * 256 * 2;    // worst-case bytes of the row tile
constexpr int kSentinelLds = 256 * 2;             // the whole table's all-DEAD sentinel row
constexpr int kWholeLdsMax = 64 * 1024;           // LDS budget for a whole table
static_assert(kStateTile >= 1 && kLockG >= 1, "tile shape");
constexpr int kLiveRows = kLiveRowsPerBlock;

// the prefix-table walk: states per block, block size, and the largest
// column count whose per-state table [Cp][Cp] uint16
// (19.2 KB at 98 columns: printable ASCII, tab, newline and the dead class)
// it takes.  Three states (57 KB of LDS) leave room for two 1024-lane blocks
// per compute unit; measured against two and four states, and against two
// tokens per lane per round.
constexpr int kPrefR = 3;
constexpr int kPrefThreads = 1024;
constexpr int kPrefixMaxCp = 98;
constexpr int kPrefStride = kPrefixMaxCp * kPrefixMaxCp + kPrefixMaxCp;  // entries per state
constexpr int kPrefWaveSpan = 1024;  // tokens per wave between allow-word writes: 32 words per state
constexpr int kPrefWordsOffset = 256 + kPrefR * kPrefStride * 2;  // 4-byte aligned: the stride is even
constexpr int kPrefLds = kPrefWordsOffset + kPrefThreads / 64 * kPrefR * 32 * 4;
// Token ranges per state group: at least enough for kPrefTargetBlocks
// blocks, and enough that no block walks more than kPrefMaxChunks rounds of
// its 16 waves (64K tokens), so the last, partly filled round of resident
// blocks stays short; each block builds its prefix tables once for them.
constexpr int kPrefTargetBlocks = 2048;  // four rounds of two resident blocks per compute unit
constexpr int kPrefMaxChunks = 4;
constexpr int kTileDeferGrid = 8192;
constexpr int kLdsPerCu = 160 * 1024;  // gfx950
static_assert(kPrefR >= 1 && 2 * kPrefLds <= 160 * 1024, "two blocks per compute unit");
static_assert(kPrefThreads >= 256, "one byte class per thread in the first 256");

// token lengths with a special meaning in the walk
constexpr int kPastEnd = -1;  // a lane slot past the last token: never stored
constexpr int kEosLen = -2;   // the end-of-sequence token

__device__ __forceinline__ bool in_range(int32_t v, int S) { return (uint32_t)v < (uint32_t)S; }

// 1. per block of rows: bit b set if some row has a live move on byte b.
__global__ __launch_bounds__(kThreads) void live_columns_kernel(const int32_t *__restrict__ trans,
                                                                int S, uint32_t *__restrict__ partial)
{
    const int b = threadIdx.x;
    const int r0 = blockIdx.x * kLiveRows;
    const int r1 = min(S, r0 + kLiveRows);
    bool live = false;
#pragma unroll 8
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
    __shared__ uint32_t words[kThreads][9];
    __shared__ int wave_count[kThreads / kWave];
    const int tid = threadIdx.x;
    uint32_t acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int k = tid; k < nblocks; k += kThreads)
#pragma unroll
        for (int w = 0; w < 8; ++w)
            acc[w] |= partial[(size_t)k * 8 + w];
#pragma unroll
    for (int w = 0; w < 8; ++w)
        words[tid][w] = acc[w];
    __syncthreads();
    for (int half = kThreads / 2; half > 0; half >>= 1) {
        if (tid < half)
#pragma unroll
            for (int w = 0; w < 8; ++w)
                words[tid][w] |= words[tid + half][w];
        __syncthreads();
    }
    const int b = tid;
    const bool live = (words[0][b / 32] >> (b % 32)) & 1u;
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
    // a dead byte exists only when total < 256, so class `total` fits in a byte
    cls[b] = (uint8_t)(live ? rank : total);
    if (live)
        byte_of[rank] = (uint8_t)b;
    if (b == 0) {
        int32_t *meta = reinterpret_cast<int32_t *>(ws);
        meta[0] = total;
        meta[1] = total < 256 ? (total + 2) & ~1 : 256;  // room for the DEAD column, even
    }
}

// 3. compacted uint16 table [S][Cp]; columns C .. Cp-1 (the dead bytes'
// class and padding) are DEAD.
__device__ __forceinline__ void compact_rows(const int32_t *__restrict__ trans, int S,
                                             const uint8_t *__restrict__ ws, uint16_t *__restrict__ table,
                                             int block)
{
    const int32_t *meta = reinterpret_cast<const int32_t *>(ws);
    const int C = meta[0], Cp = meta[1];
    const int c = threadIdx.x;
    if (c >= Cp)
        return;
    const int byte = c < C ? ws[512 + c] : 0;
    const int r0 = block * 16;
    const int r1 = min(S, r0 + 16);
#pragma unroll 4
    for (int s = r0; s < r1; ++s) {
        uint16_t v = kDead16;
        if (c < C) {
            const int32_t x = trans[(size_t)s * 256 + byte];
            v = in_range(x, S) ? (uint16_t)x : kDead16;
        }
        table[(size_t)s * Cp + c] = v;
    }
}

// 4. per token: the classes of its first kRegBytes bytes (four per word),
// its length and offset -- read once per block by the walk instead of
// re-deriving them from the bytes in every block.
__device__ __forceinline__ void token_records(const int32_t *__restrict__ offsets,
                                              const uint8_t *__restrict__ bytes, int V, int eos_token,
                                              const uint8_t *__restrict__ ws, uint4 *__restrict__ tokinfo,
                                              uint8_t *cls, int block)
{
    cls[threadIdx.x] = ws[256 + threadIdx.x];
    __syncthreads();
    const int t = block * kThreads + threadIdx.x;
    if (t >= V)
        return;
    if (t == eos_token) {  // its bytes are ignored: allowed exactly in accepting states
        tokinfo[t] = make_uint4(0, 0, (uint32_t)kEosLen, 0);
        return;
    }
    const int off = offsets[t];
    const int len = max(0, offsets[t + 1] - off);  // a decreasing pair reads as an empty token
    uint32_t lo = 0, hi = 0;
    const int n = min(len, kRegBytes);
    for (int h = 0; h < n; ++h) {
        const uint32_t c = cls[bytes[off + h]];
        if (h < 4)
            lo |= c << (8 * h);
        else
            hi |= c << (8 * (h - 4));
    }
    tokinfo[t] = make_uint4(lo, hi, (uint32_t)len, (uint32_t)off);
}

// 3 and 4 share one launch (both need only the byte classes): the first
// ceil(S / 16) blocks compact the table, the rest build the token records.
__global__ __launch_bounds__(kThreads) void compact_and_tokens_kernel(
    const int32_t *__restrict__ trans, int S, const int32_t *__restrict__ offsets,
    const uint8_t *__restrict__ bytes, int V, int eos_token, const uint8_t *__restrict__ ws,
    uint16_t *__restrict__ table, uint4 *__restrict__ tokinfo)
{
    __shared__ uint8_t cls[256];
    const int ncompact = (S + 15) / 16;
    if ((int)blockIdx.x < ncompact)
        compact_rows(trans, S, ws, table, blockIdx.x);
    else
        token_records(offsets, bytes, V, eos_token, ws, tokinfo, cls, blockIdx.x - ncompact);
}

// 5. the tile walk.  One block owns a tile of kStateTile states x kThreads
// tokens (one per lane, so stores are coalesced).  Dynamic LDS holds the
// byte-class map and the table: the whole table when S * Cp * 2 fits in
// `lds_table_bytes` (then followed by an all-DEAD sentinel row), else the
// tile's rows.  Either way a lane walks its token from kLockG of the tile's
// states at once.

// The tile walk when the whole table is in LDS: a lane walks its token from
// kLockG of the tile's states at once, one byte per iteration (the class
// shared by the states, kLockG independent LDS reads per iteration instead
// of one dependent read per move), until every one of them is dead or the
// token ends.  A dead state is row S, an all-DEAD sentinel row, which every
// read maps back to S, so the walk needs no branch per state.  Each group's
// results go straight to coalesced stores; a wave ballot packs the allow
// words.
__device__ __forceinline__ void walk_tile_whole(const uint16_t *tab, const uint8_t *cls, int Cp, int S, int s0,
                                                int nS, const uint8_t *__restrict__ bytes, int t_base, int V,
                                                int W, const uint4 *__restrict__ tokinfo,
                                                const uint8_t *__restrict__ accepting,
                                                int32_t *__restrict__ next_state, uint32_t *__restrict__ allow)
{
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int t = t_base + tid;
    const uint4 ti = t < V ? tokinfo[t] : make_uint4(0, 0, (uint32_t)kPastEnd, 0);
    const int len = (int)ti.z;
    const uint64_t classes = ((uint64_t)ti.y << 32) | ti.x;  // the first kRegBytes byte classes
    const uint32_t dead = (uint32_t)S;
    const int t0 = t_base + wave * kWave;  // a multiple of 64
    const int w = t0 / 32 + lane;
    for (int g = 0; g < nS; g += kLockG) {
        uint32_t st[kLockG];
#pragma unroll
        for (int k = 0; k < kLockG; ++k) {
            const int s = s0 + g + k;
            st[k] = g + k < nS ? (uint32_t)s : dead;
            if (len < 0)  // EOS: only where the scanner may stop; past the last token: dead
                st[k] = g + k < nS && len == kEosLen && accepting != nullptr && accepting[s] != 0 ? (uint32_t)s
                                                                                                : dead;
        }
        uint32_t m = st[0];
#pragma unroll
        for (int k = 1; k < kLockG; ++k)
            m = min(m, st[k]);
        bool go = len > 0 && m != dead;  // an empty token keeps the state
        uint64_t cr = classes;
        uint32_t h = 0;
        while (go) {
            uint32_t c;
            if (h < (uint32_t)kRegBytes) {
                c = (uint32_t)cr & 0xFFu;
                cr >>= 8;
            } else {
                c = cls[bytes[ti.w + h]];
            }
#pragma unroll
            for (int k = 0; k < kLockG; ++k)
                st[k] = min((uint32_t)tab[st[k] * (uint32_t)Cp + c], dead);
            h += 1;
            m = st[0];
#pragma unroll
            for (int k = 1; k < kLockG; ++k)
                m = min(m, st[k]);
            go = m != dead && h < (uint32_t)len;
        }
#pragma unroll
        for (int k = 0; k < kLockG; ++k) {
            if (g + k >= nS)
                break;
            const int s = s0 + g + k;
            const bool alive = st[k] != dead;
            if (t < V)
                __builtin_nontemporal_store(alive ? (int32_t)st[k] : -1, &next_state[(size_t)s * V + t]);
            const uint64_t mask = __ballot(alive);
            if (lane < 2 && w < W)
                __builtin_nontemporal_store((uint32_t)(mask >> (32 * lane)), &allow[(size_t)s * W + w]);
        }
    }
}

// The tile walk when only the tile's rows are in LDS, in lockstep: a lane
// walks its token from kLockG of the tile's states at once, the first move
// from the LDS rows, later ones from the cache-resident table at 32-bit
// offsets (a dead state skips its read under the exec mask), so a long walk
// costs a chain of independent reads rather than one dependent read per
// move of every state.  Results go straight to coalesced stores.
__device__ __forceinline__ void walk_tile_rows(const uint16_t *tab, const uint16_t *__restrict__ table,
                                               const uint8_t *cls, int Cp, int s0, int nS,
                                               const uint8_t *__restrict__ bytes, int t_base, int V, int W,
                                               const uint4 *__restrict__ tokinfo,
                                               const uint8_t *__restrict__ accepting,
                                               int32_t *__restrict__ next_state, uint32_t *__restrict__ allow)
{
    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int t = t_base + tid;
    const uint4 ti = t < V ? tokinfo[t] : make_uint4(0, 0, (uint32_t)kPastEnd, 0);
    const int len = (int)ti.z;
    const uint64_t classes = ((uint64_t)ti.y << 32) | ti.x;  // the first kRegBytes byte classes
    const char *tab_bytes = reinterpret_cast<const char *>(table);
    const uint32_t Cp2 = 2u * (uint32_t)Cp;
    const int t0 = t_base + wave * kWave;  // a multiple of 64
    const int w = t0 / 32 + lane;
    for (int g = 0; g < nS; g += kLockG) {
        uint32_t st[kLockG];
        const uint32_t c0 = ti.x & 0xFFu;
#pragma unroll
        for (int k = 0; k < kLockG; ++k) {
            const int s = s0 + g + k;
            uint32_t v = kDead16;
            if (g + k < nS) {
                if (len > 0)
                    v = tab[(g + k) * Cp + c0];  // the first move, from the row tile
                else if (len == 0)
                    v = (uint32_t)s;  // an empty token keeps the state
                else if (len == kEosLen && accepting != nullptr && accepting[s] != 0)
                    v = (uint32_t)s;  // EOS: only where the scanner may stop
            }
            st[k] = v;
        }
        uint32_t m = st[0];
#pragma unroll
        for (int k = 1; k < kLockG; ++k)
            m = min(m, st[k]);
        bool go = len > 1 && m != kDead16;
        uint64_t cr = classes >> 8;
        uint32_t h = 1;
        while (go) {
            uint32_t c;
            if (h < (uint32_t)kRegBytes) {
                c = (uint32_t)cr & 0xFFu;
                cr >>= 8;
            } else {
                c = cls[bytes[ti.w + h]];
            }
#pragma unroll
            for (int k = 0; k < kLockG; ++k)
                if (st[k] != kDead16) {
                    const uint32_t boff = __umul24(st[k], Cp2) + 2u * c;  // < 2^32: S <= 65535, Cp <= 256
                    st[k] = *reinterpret_cast<const uint16_t *>(tab_bytes + boff);
                }
            h += 1;
            m = st[0];
#pragma unroll
            for (int k = 1; k < kLockG; ++k)
                m = min(m, st[k]);
            go = m != kDead16 && h < (uint32_t)len;
        }
#pragma unroll
        for (int k = 0; k < kLockG; ++k) {
            if (g + k >= nS)
                break;
            const int s = s0 + g + k;
            const bool alive = st[k] != kDead16;
            if (t < V)
                __builtin_nontemporal_store(alive ? (int32_t)st[k] : -1, &next_state[(size_t)s * V + t]);
            const uint64_t mask = __ballot(alive);
            if (lane < 2 && w < W)
                __builtin_nontemporal_store((uint32_t)(mask >> (32 * lane)), &allow[(size_t)s * W + w]);
        }
    }
}

__global__ __launch_bounds__(kThreads) void walk_kernel(const uint8_t *__restrict__ ws,
                                                        const uint16_t *__restrict__ table, int S,
                                                        const uint4 *__restrict__ tokinfo,
                                                        const uint8_t *__restrict__ bytes, int V,
                                                        int W, int lds_table_bytes, int defer,
                                                        const uint8_t *__restrict__ accepting,
                                                        int32_t *__restrict__ next_state,
                                                        uint32_t *__restrict__ allow)
{
    extern __shared__ __align__(16) uint8_t smem[];
    uint8_t *cls = smem;
    uint16_t *tab = reinterpret_cast<uint16_t *>(smem + 256);

    const int tid = threadIdx.x;
    const int Cp = reinterpret_cast<const int32_t *>(ws)[1];
    const bool whole = (size_t)S * Cp * 2 <= (size_t)lds_table_bytes;
    if (defer && !whole && Cp <= kPrefixMaxCp)
        return;  // the prefix-table walk owns this table
    const int ntx = (V + kTokTile - 1) / kTokTile;
    const int ntiles = ntx * ((S + kStateTile - 1) / kStateTile);

    cls[tid] = ws[256 + tid];
    if (whole) {
        const int n32 = S * Cp / 2;  // Cp is even
        const uint32_t *src = reinterpret_cast<const uint32_t *>(table);
        uint32_t *dst = reinterpret_cast<uint32_t *>(tab);
        for (int i = tid; i < n32; i += kThreads)
            dst[i] = src[i];
        // the sentinel row S (all DEAD) right after the table: Cp * 2 <= kSentinelLds
        for (int i = tid; i < Cp; i += kThreads)
            tab[S * Cp + i] = kDead16;
    }
    // a grid smaller than the tile count (launched beside the prefix-table
    // walk, so that it exits cheaply when that one owns the table) strides
    for (int tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int s0 = (tile / ntx) * kStateTile;
        const int nS = min(kStateTile, S - s0);
        const int t_base = (tile % ntx) * kTokTile;
        if (!whole) {
            if (tile != (int)blockIdx.x)
                __syncthreads();  // the previous tile's rows are no longer read
            const int n32 = nS * Cp / 2;
            const uint32_t *src = reinterpret_cast<const uint32_t *>(table + (size_t)s0 * Cp);
            uint32_t *dst = reinterpret_cast<uint32_t *>(tab);
            for (int i = tid; i < n32; i += kThreads)
                dst[i] = src[i];
        }
        __syncthreads();
        if (whole)
            walk_tile_whole(tab, cls, Cp, S, s0, nS, bytes, t_base, V, W, tokinfo, accepting, next_state, allow);
        else
            walk_tile_rows(tab, table, cls, Cp, s0, nS, bytes, t_base, V, W, tokinfo, accepting, next_state, allow);
    }
}

// 6. the prefix-table walk, for tables of at most kPrefixMaxCp columns that
// do not fit in LDS whole.  A block owns kPrefR states and a range of tokens.
// It first builds, per state s, the table P_s[c0][c1] = state after the byte
// classes c0 c1 from s (the rows of the states one move from s, copied from
// the compacted table: coalesced reads) followed by s's own row, so that the
// first two moves of every pair are one LDS read; only walks still live
// after two bytes (about a fifth of the pairs for random printable DFAs)
// read the cache-resident table.  The walk is bound by instruction issue
// and L1 accesses, so the later moves run in lockstep: a lane walks its
// token from all the block's states at once, one byte per iteration; the
// byte class, doubled to a byte offset, is shifted out of a 64-bit register
// and shared by the states; each live state costs one compare, one
// multiply-add and one table read at a 32-bit offset, and a dead one skips
// its read under the exec mask (reading an all-DEAD row instead costs an L1
// access per lane); the lane stops when every state is dead or the token
// ends.  A wave takes 64 consecutive tokens per round, one per lane, over a
// run of kPrefWaveSpan tokens; the results stay in registers until the
// round's coalesced stores, and the alive compare gives both the stored
// value and, as a wave mask, the allow bits, which wait in LDS until the
// run's words are written together.
__global__ __launch_bounds__(kPrefThreads) void walk_prefix_kernel(
    const uint8_t *__restrict__ ws, const uint16_t *__restrict__ table, int S, const uint4 *__restrict__ tokinfo,
    const uint8_t *__restrict__ bytes, int V, int W, int lds_table_bytes, int range,
    const uint8_t *__restrict__ accepting, int32_t *__restrict__ next_state, uint32_t *__restrict__ allow)
{
    extern __shared__ __align__(16) uint8_t smem[];
    const int Cp = reinterpret_cast<const int32_t *>(ws)[1];
    if (Cp > kPrefixMaxCp || (size_t)S * Cp * 2 <= (size_t)lds_table_bytes)
        return;  // the tile walk owns this table
    uint8_t *cls = smem;                                     // [256]
    uint16_t *pt = reinterpret_cast<uint16_t *>(smem + 256);  // [kPrefR][kPrefStride]: P_s, then s's row
    const int CC = Cp * Cp;

    const int tid = threadIdx.x;
    const int lane = tid & (kWave - 1), wave = tid / kWave;
    const int s0 = blockIdx.y * kPrefR;
    const int nS = min(kPrefR, S - s0);
    const int t_lo = blockIdx.x * range;
    const int t_hi = min(V, t_lo + range);

    if (tid < 256)
        cls[tid] = ws[256 + tid];
    for (int i = tid; i < kPrefR * Cp; i += kPrefThreads) {
        const int si = i / Cp, c = i - si * Cp;
        pt[si * kPrefStride + CC + c] = si < nS ? table[(size_t)(s0 + si) * Cp + c] : kDead16;
    }
    __syncthreads();
    for (int row = wave; row < kPrefR * Cp; row += kPrefThreads / kWave) {
        const int si = row / Cp, c0 = row - si * Cp;
        const uint32_t f = pt[si * kPrefStride + CC + c0];
        const bool live = f != kDead16;
        uint16_t *dst = pt + si * kPrefStride + c0 * Cp;
        const uint16_t *src = table + (size_t)(live ? f : 0u) * Cp;  // row 0 stands in for DEAD
        for (int c = lane; c < Cp; c += kWave) {
            const uint16_t v = src[c];
            dst[c] = live ? v : kDead16;
        }
    }
    __syncthreads();

    uint32_t acc_bits = 0;  // accepting flags of the block's states
#pragma unroll
    for (int si = 0; si < kPrefR; ++si)
        if (si < nS && accepting != nullptr && accepting[s0 + si] != 0)
            acc_bits |= 1u << si;
    const char *tab_bytes = reinterpret_cast<const char *>(table);
    const uint32_t Cp2 = 2u * (uint32_t)Cp;  // row stride in bytes

    // Each wave walks kPrefWaveSpan consecutive tokens, 64 per round, and
    // then writes its allow words for them as runs of 32 words (128 bytes)
    // per state from LDS: whole L2 lines where the row is aligned, instead
    // of 8-byte pieces from every wave of the block.
    uint32_t *words = reinterpret_cast<uint32_t *>(smem + kPrefWordsOffset) + wave * (kPrefR * 32);
    for (int sc = t_lo; sc < t_hi; sc += kPrefThreads / kWave * kPrefWaveSpan) {
        const int wb = sc + wave * kPrefWaveSpan;  // a multiple of kPrefWaveSpan
        if (wb >= t_hi)
            continue;
        const int we = min(t_hi, wb + kPrefWaveSpan);
        for (int t0 = wb; t0 < we; t0 += kWave) {
            const int t = t0 + lane;
            const uint4 ti = t < we ? tokinfo[t] : make_uint4(0, 0, (uint32_t)kPastEnd, 0);
            const int len = (int)ti.z;
            const uint32_t c0 = ti.x & 0xFFu, c1 = (ti.x >> 8) & 0xFFu;
            const uint32_t idx = len >= 2 ? c0 * (uint32_t)Cp + c1 : (uint32_t)CC + c0;
            // the first two moves of every pair: one LDS read
            uint32_t st[kPrefR];
#pragma unroll
            for (int si = 0; si < kPrefR; ++si)
                st[si] = pt[si * kPrefStride + idx];
            if (__any(len <= 0)) {  // empty, EOS and past-the-end tokens
#pragma unroll
                for (int si = 0; si < kPrefR; ++si)
                    if (len <= 0) {
                        const bool keep = si < nS && (len == 0 || (len == kEosLen && ((acc_bits >> si) & 1u)));
                        st[si] = keep ? (uint32_t)(s0 + si) : kDead16;  // EOS: where the scanner may stop
                    }
            }

            // the later moves, every state in lockstep
            uint32_t m = st[0];
#pragma unroll
            for (int si = 1; si < kPrefR; ++si)
                m = min(m, st[si]);
            bool go = m != kDead16 && len > 2;
            if (__any(go)) {
                uint64_t crem = (((uint64_t)ti.y << 16) | (ti.x >> 16)) << 1;  // classes 2..7, doubled
                uint32_t h = 2;
                while (go) {
                    uint32_t c2;
                    if (h < (uint32_t)kRegBytes) {
                        c2 = (uint32_t)crem & 0xFFu;
                        crem >>= 8;
                    } else {
                        c2 = 2u * cls[bytes[ti.w + h]];
                    }
#pragma unroll
                    for (int si = 0; si < kPrefR; ++si)
                        if (st[si] != kDead16) {
                            const uint32_t boff = __umul24(st[si], Cp2) + c2;  // < 2^24: S <= 65535, Cp <= 98
                            st[si] = *reinterpret_cast<const uint16_t *>(tab_bytes + boff);
                        }
                    h += 1;
                    m = st[0];
#pragma unroll
                    for (int si = 1; si < kPrefR; ++si)
                        m = min(m, st[si]);
                    go = m != kDead16 && h < (uint32_t)len;
                }
            }

            // coalesced stores; the alive compare is also the wave's allow mask
            const int k = (t0 - wb) / 32;  // this round's first word in the wave's run
#pragma unroll
            for (int si = 0; si < kPrefR; ++si) {
                if (si >= nS)
                    break;
                const bool alive = st[si] != kDead16;  // past-the-end slots are DEAD
                if (t < we)
                    __builtin_nontemporal_store(alive ? (int32_t)st[si] : -1, &next_state[(size_t)(s0 + si) * V + t]);
                const uint64_t mask = __ballot(alive);
                if (lane < 2)
                    words[si * 32 + k + lane] = (uint32_t)(mask >> (32 * lane));
            }
        }
        wave_lds_sync();
        const int w0 = wb / 32, nw = min((we - wb + 31) / 32, W - w0);
        for (int i = lane; i < kPrefR * 32; i += kWave) {
            const int si = i / 32, k = i % 32;
            if (si < nS && k < nw)
                __builtin_nontemporal_store(words[i], &allow[(size_t)(s0 + si) * W + w0 + k]);
        }
        wave_lds_sync();  // read before the next run's words are written
    }
}

}  // namespace

// The vocabulary's CSR layout: the smallest t in [0, V] at which it breaks
// (offsets[0] != 0 at t = 0; offsets[t] < offsets[t - 1] or offsets[t] >
// num_bytes at t >= 1), or -1.  The answer is an unsigned minimum over the
// broken indices, started at all ones (= -1 as int32) by a one-lane kernel.
__global__ void validate_vocab_init_kernel(uint32_t *first_bad) { *first_bad = 0xFFFFFFFFu; }

__global__ __launch_bounds__(256) void validate_vocab_kernel(const int32_t *__restrict__ offsets, int V,
                                                             int64_t num_bytes, uint32_t *__restrict__ first_bad)
{
    const int stride = gridDim.x * blockDim.x;
    for (int t = blockIdx.x * blockDim.x + (int)threadIdx.x; t <= V; t += stride) {
        const int o = offsets[t];
        const bool broken = t == 0 ? o != 0 : (o < offsets[t - 1] || (int64_t)o > num_bytes);
        if (broken)
            atomicMin(first_bad, (uint32_t)t);
    }
}

hipError_t launch_validate_vocab(const int32_t *offsets, int V, int64_t num_bytes, int32_t *first_bad,
                                 hipStream_t stream)
{
    uint32_t *out = reinterpret_cast<uint32_t *>(first_bad);
    validate_vocab_init_kernel<<<1, 1, 0, stream>>>(out);
    const int blocks = (int)std::min<int64_t>(((int64_t)V + 256) / 256, 4096);
    validate_vocab_kernel<<<blocks, 256, 0, stream>>>(offsets, V, num_bytes, out);
    return hipGetLastError();
}

hipError_t launch_align(const int32_t *trans, int S, const int32_t *offsets, const uint8_t *bytes,
                        int V, const uint8_t *accepting, int eos_token, int32_t *next_state,
                        uint32_t *allow, void *workspace, hipStream_t stream)
{
    uint8_t *ws = static_cast<uint8_t *>(workspace);
    uint32_t *partial = reinterpret_cast<uint32_t *>(ws + kAlignMetaBytes);
    uint16_t *table = reinterpret_cast<uint16_t *>(ws + align_table_offset(S));
    uint4 *tokinfo = reinterpret_cast<uint4 *>(ws + align_tokinfo_offset(S));
    const int nblk = (int)align_live_blocks(S);
    const int W = (V + 31) / 32;

    // LDS for the table.  The column count C is only known on the device, so
    // for small S the launch reserves up to kWholeLdsMax bytes and the kernel
    // stages the whole table when S * Cp * 2 fits; otherwise (and always for
    // S > 512, where a whole table would leave too little LDS for occupancy)
    // it stages only the block's row tile.
    int lds_table = kRowsLds;
    if (S <= 512) {
        const size_t whole_worst = (size_t)S * 256 * 2;
        lds_table = (int)(whole_worst < (size_t)kWholeLdsMax ? whole_worst : (size_t)kWholeLdsMax);
        if (lds_table < kRowsLds)
            lds_table = kRowsLds;
    }

    // LDS beyond the default 64 KB per block must be opted into once.
    static const hipError_t lds_attr = hipFuncSetAttribute(
        reinterpret_cast<const void *>(walk_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
        256 + kWholeLdsMax + kSentinelLds);
    if (lds_attr != hipSuccess)
        return lds_attr;
    static const hipError_t prefix_lds_attr = hipFuncSetAttribute(
        reinterpret_cast<const void *>(walk_prefix_kernel), hipFuncAttributeMaxDynamicSharedMemorySize, kPrefLds);
    if (prefix_lds_attr != hipSuccess)
        return prefix_lds_attr;

    live_columns_kernel<<<nblk, kThreads, 0, stream>>>(trans, S, partial);
    byte_classes_kernel<<<1, kThreads, 0, stream>>>(partial, nblk, ws);
    compact_and_tokens_kernel<<<(S + 15) / 16 + (V + kThreads - 1) / kThreads, kThreads, 0, stream>>>(
        trans, S, offsets, bytes, V, eos_token, ws, table, tokinfo);
    // Tables of at most kPrefixMaxCp columns that are not staged whole go to
    // the prefix-table walk; the column count is known only on the device,
    // so when such a table is possible both walks are launched and each
    // block of the one that does not own the table exits at once (the tile
    // walk then runs a strided grid of at most kTileDeferGrid blocks).
    const bool prefix = (size_t)S * kPrefixMaxCp * 2 > (size_t)lds_table;
    if (prefix) {
        const int rows = (S + kPrefR - 1) / kPrefR;
        const int chunk = kPrefThreads / kWave * kPrefWaveSpan;
        const int nchunks = (V + chunk - 1) / chunk;
        int nr = max((kPrefTargetBlocks + rows - 1) / rows, (nchunks + kPrefMaxChunks - 1) / kPrefMaxChunks);
        nr = max(1, min(nr, nchunks));
        const int range = (int)align_up((size_t)((V + nr - 1) / nr), chunk);  // whole rounds of every wave
        nr = (V + range - 1) / range;
        walk_prefix_kernel<<<dim3(nr, rows), kPrefThreads, kPrefLds, stream>>>(
            ws, table, S, tokinfo, bytes, V, W, lds_table, range, accepting, next_state, allow);
    }
    // The tile walk strides over its tiles; when the whole table may be
    // staged (S <= 512), at most one round of resident blocks is launched,
    // so that each block stages the table once for several tiles.
    const long long ntiles = (long long)((V + kTokTile - 1) / kTokTile) * ((S + kStateTile - 1) / kStateTile);
    long long cap = prefix ? kTileDeferGrid : ntiles;
    const int cus = device_compute_units();
    if (S <= 512 && cus > 0) {
        const int per_cu = kLdsPerCu / (256 + lds_table + kSentinelLds);
        cap = min(cap, (long long)(per_cu > 1 ? per_cu : 1) * cus);
    }
    const int grid = (int)(ntiles < cap ? ntiles : cap);
    walk_kernel<<<grid, kThreads, 256 + lds_table + kSentinelLds, stream>>>(ws, table, S, tokinfo, bytes, V, W,
                                                                       lds_table, prefix ? 1 : 0, accepting,
                                                                       next_state, allow);
    return hipGetLastError();
}

}  // namespace dv
