/*
 * dv_probes.h -- roofline probes (libdv_probes.so: measurement, not the hot
 * path; libdv.so does not contain them).
 *
 * Each probe enqueues one kernel on `stream` that exercises one memory path
 * of the GPU the way the alignment and masked-step kernels do, so the rates
 * they reach can be compared with what those kernels reach:
 *
 *   dvprobe_stream_read  16-byte loads over `n_bytes` of device memory (HBM
 *                        read bandwidth, the masked step's bound);
 *   dvprobe_stream_write 16-byte stores over `n_bytes` (HBM write bandwidth,
 *                        the alignment table's output bound);
 *   dvprobe_gather       dependent random gathers from a device table of
 *                        `table_entries` uint32 values (L1/L2 gather rate,
 *                        the alignment walk's later moves, which read one
 *                        small table entry per request);
 *   dvprobe_lds_gather   the same chase inside LDS (the walk's first move).
 *
 * All pointers are device pointers owned by the caller; sizes are checked on
 * the host before any HIP call.  `sink` receives a value derived from every
 * load so that no load can be optimised away (its contents are meaningless).
 * Returns 0 on success, 1 for a bad argument, 6 for a HIP error.
 */
#ifndef DV_PROBES_H
#define DV_PROBES_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define DVPROBE_API __attribute__((visibility("default")))
#else
#define DVPROBE_API
#endif

/* src: n_bytes (multiple of 16, >= 4096) of device memory; sink: 4096 uint32. */
DVPROBE_API int32_t dvprobe_stream_read(const void *src, size_t n_bytes, uint32_t *sink,
                                        void *stream);

/* dst: n_bytes (multiple of 16, >= 4096) of device memory, overwritten. */
DVPROBE_API int32_t dvprobe_stream_write(void *dst, size_t n_bytes, void *stream);

/* table: table_entries (<= 2^24) uint32 values, normally a random chase
 * permutation of [0, table_entries) (values outside are clamped into range);
 * lanes * chains independent chases of `steps` dependent loads each.
 * lanes: a multiple of 256; chains: 1, 2, 4 or 8.  sink: lanes uint32. */
DVPROBE_API int32_t dvprobe_gather(const uint32_t *table, int32_t table_entries, int32_t lanes,
                                   int32_t chains, int32_t steps, uint32_t *sink, void *stream);

/* As dvprobe_gather with the table copied into each block's LDS first
 * (table_entries <= 32768, i.e. up to 128 KB of LDS). */
DVPROBE_API int32_t dvprobe_lds_gather(const uint32_t *table, int32_t table_entries,
                                       int32_t lanes, int32_t chains, int32_t steps,
                                       uint32_t *sink, void *stream);

/* The alignment walk's later moves in isolation: lanes * chains chases of
 * `steps` dependent 2-byte reads st = table[st * num_classes + c] through a
 * uint16 state table [num_states][num_classes] (values >= num_states are
 * folded back in range), c a per-step pseudo-random byte class; 1024-lane
 * blocks.  lanes: a multiple of 1024; chains: 1 or 3 (the prefix walk's
 * states per lane); num_states * num_classes <= 2^24.  sink: lanes uint32. */
DVPROBE_API int32_t dvprobe_walk_gather(const uint16_t *table, int32_t num_states, int32_t num_classes,
                                        int32_t lanes, int32_t chains, int32_t steps, uint32_t *sink,
                                        void *stream);

/* Floors of the bf16 masked step (dv_masked_step) at its own launch shape
 * for `batch` rows of `num_tokens` logits (the same blocks and block size):
 *   mode 0  each block reads its row's state and writes the outputs
 *           (token = -1, new_state = the state): the launch and one
 *           dependent trip, nothing streamed;
 *   mode 1  loads of every 16-byte vector of the rows, streamed as the step
 *           streams them, with no mask and no arithmetic;
 *   mode 2  loads of exactly the 128-byte lines holding an allowed token of
 *           each row's state (allow [S][ceil(V/32)] as for dv_masked_step),
 *           the mask bytes read first and choosing the addresses.
 * logits: [batch][ld_logits] bf16, rows 16-byte aligned; states [batch];
 * token, new_state [batch]; sink: at least batch * 64 uint32 (contents
 * meaningless).  Returns 0, 1 for a bad argument, 6 for a HIP error. */
DVPROBE_API int32_t dvprobe_step_floor(int32_t mode, const void *logits, int32_t num_tokens,
                                       int64_t ld_logits, const uint32_t *allow, int32_t num_states,
                                       const int32_t *states, int32_t batch, int32_t *token,
                                       int32_t *new_state, uint32_t *sink, int64_t sink_words,
                                       void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DV_PROBES_H */
