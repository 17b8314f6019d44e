/*
 * dv.h -- vocabulary alignment and masked greedy decoding on one MI355X.
 *
 * C ABI of libdv.so.  Two operations, from "Guiding LLMs The Right Way: Fast,
 * Non-Invasive Constrained Generation" (DOMINO, ICML 2024):
 *
 *   dv_align        the offline vocabulary alignment of Sec. 3.3 /
 *                   Algorithm 2 for a regular (DFA) constraint walked to full
 *                   depth (Sec. 3.5, lookahead k = infinity): every scanner
 *                   state is walked through every token's bytes.
 *   dv_masked_step  one step of Algorithm 1: look up the mask of each
 *                   sequence's current state, apply it to the logits, decode
 *                   greedily (Algorithm 3's argmax over the admissible set)
 *                   and advance the state with the chosen token.
 *   dv_align_eos    dv_align with an end-of-sequence token that is allowed
 *                   exactly in accepting states.
 *   dv_masked_step_opportunistic
 *                   dv_masked_step that checks the model's own choice first
 *                   (opportunistic masking, Sec. 3.5).
 *   dv_masked_sample
 *                   the sampled decode at temperature T over the allowed
 *                   tokens, reproducible from a seed and an offset.
 *   dv_spec_walk,   the speculative chain check of Sec. 3.6: how many
 *   dv_spec_verify  proposed tokens the constraint admits, and greedy
 *                   verification of the proposals against the model's logits
 *                   at every proposed position.
 *
 * Conventions shared by every call:
 *   - Every array argument is a DEVICE pointer (hipMalloc'd or a torch CUDA
 *     tensor's data_ptr) owned by the caller.  The library allocates nothing,
 *     keeps no pointer after it returns, and has no global state except a
 *     per-thread error message.
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream)
 *     and runs asynchronously to the host.  Outputs are valid once the stream
 *     has reached the call; inputs must stay unchanged until then.  Two calls
 *     that share a workspace must be ordered on one stream.
 *   - Arguments are checked on the host before any HIP call.  On a failed
 *     check nothing is enqueued and the call returns an error status; a
 *     message is available from dv_last_error() on the calling thread.
 *   - The alphabet is bytes (256 symbols).  DV_DEAD (-1) is the dead state:
 *     a sentinel, never a table row.  A transition target or an input state
 *     outside [0, num_states) reads as DV_DEAD; nothing leaves DV_DEAD.
 */
#ifndef DV_H
#define DV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define DV_API __attribute__((visibility("default")))
#else
#define DV_API
#endif

#define DV_DEAD (-1)

/* Limits checked by every call (inclusive). */
#define DV_MAX_STATES 65535        /* num_states  in [1, DV_MAX_STATES]  */
#define DV_MAX_TOKENS 16777216     /* num_tokens  in [1, DV_MAX_TOKENS]  */
#define DV_MAX_BATCH  1048576      /* batch       in [0, DV_MAX_BATCH]   */
#define DV_MAX_PROPOSED 1024       /* num_proposed in [0, DV_MAX_PROPOSED];
                                      batch * (num_proposed + 1) <= DV_MAX_BATCH */
#define DV_NOALLOC_MAX_BATCH 65536 /* batch of dv_masked_step_noalloc          */

typedef enum dv_status {
    DV_OK = 0,
    DV_ERR_INVALID_ARG = 1,  /* a required pointer is NULL                         */
    DV_ERR_SHAPE = 2,        /* a size is outside its limit or ld_logits < V       */
    DV_ERR_DTYPE = 3,        /* unknown logits dtype                               */
    DV_ERR_ALIAS = 4,        /* an output overlaps an input or another output      */
    DV_ERR_WORKSPACE = 5,    /* workspace missing, too small or misaligned         */
    DV_ERR_HIP = 6           /* a HIP launch or runtime call failed                */
} dv_status;

typedef enum dv_dtype {
    DV_F32 = 0,              /* IEEE binary32 logits                               */
    DV_BF16 = 1              /* bfloat16 logits (high half of a binary32)          */
} dv_dtype;

/*
 * dv_align_workspace_bytes -- device workspace dv_align / dv_align_eos need
 * for `num_states` states and `num_tokens` tokens (the compacted transition
 * table, the byte-class map and per-token byte classes).  Returns 0 when a
 * size is outside its limit.
 */
DV_API size_t dv_align_workspace_bytes(int32_t num_states, int32_t num_tokens);

/*
 * dv_align -- the vocabulary alignment table (Sec. 3.3, Algorithm 2, at
 * full depth as in Sec. 3.5).
 *
 * For every state s in [0, S) and every token t in [0, V):
 *     next_state[s*V + t] = the state reached by reading the bytes of token t
 *                           one by one from s, or DV_DEAD if a transition on
 *                           the way is dead (the walk stops there);
 *     bit (t % 32) of allow[s*W + t/32] = 1 exactly when next_state != DV_DEAD,
 * with W = ceil(V/32).  Bits for t >= V are written as 0.  A zero-length
 * token leaves the state unchanged (next_state = s, allowed).
 *
 * Inputs (device, read only):
 *   trans      [S][256] int32, row-major: trans[s*256 + b] is the move of
 *              state s on byte b.  Values outside [0, S) read as DV_DEAD.
 *   offsets    [V+1] int32, offsets[0] = 0, non-decreasing, offsets[V] <=
 *              the size of bytes (a precondition this call does not check:
 *              dv_validate_vocab does): token t is bytes[offsets[t] ..
 *              offsets[t+1]); a decreasing pair reads as an empty token.
 *   bytes      [offsets[V]] uint8, the concatenated token strings.  May be
 *              NULL only when every token is empty.
 * Outputs (device, written in full):
 *   next_state [S][V] int32; allow [S][W] uint32.
 * Workspace: at least dv_align_workspace_bytes(S, V) bytes of device memory,
 *   256-byte aligned; contents on entry are ignored, on exit undefined.
 * Errors: DV_ERR_INVALID_ARG (NULL pointer), DV_ERR_SHAPE (S or V out of
 *   range), DV_ERR_ALIAS (next_state/allow overlap each other or an input,
 *   checked on the address ranges implied by S and V), DV_ERR_WORKSPACE,
 *   DV_ERR_HIP.
 */
DV_API dv_status dv_align(const int32_t *trans, int32_t num_states,
                   const int32_t *offsets, const uint8_t *bytes, int32_t num_tokens,
                   int32_t *next_state, uint32_t *allow,
                   void *workspace, size_t workspace_bytes, void *stream);

/*
 * dv_align_eos -- dv_align with an end-of-sequence token (Algorithm 1 stops
 * on EOS; Sec. 3.2 treats EOS as one more terminal of the scanner, so it may
 * follow wherever a terminal sequence may end).
 *
 * Every token except `eos_token` is aligned exactly as by dv_align.  For the
 * EOS column (its bytes are ignored):
 *     next_state[s*V + eos_token] = s        if accepting[s] != 0,
 *                                   DV_DEAD  otherwise,
 * with the allow bit set exactly when it is not DV_DEAD, so the masked step
 * can choose EOS only where the constraint may end; the state is left
 * unchanged and the caller stops decoding the sequence.
 *
 * accepting  [S] uint8 (device), nonzero for states where the constraint may
 *            end (accepting states; the start state if the empty output is
 *            valid).  NULL means no state accepts: EOS is never allowed.
 * eos_token  in [0, V).
 * Workspace, outputs and errors as dv_align (DV_ERR_SHAPE also for an
 * eos_token outside [0, V)).
 */
DV_API dv_status dv_align_eos(const int32_t *trans, int32_t num_states,
                       const int32_t *offsets, const uint8_t *bytes, int32_t num_tokens,
                       const uint8_t *accepting, int32_t eos_token,
                       int32_t *next_state, uint32_t *allow,
                       void *workspace, size_t workspace_bytes, void *stream);

/*
 * dv_validate_vocab -- checks the CSR layout of a vocabulary on the device:
 * the precondition of dv_align / dv_align_eos, whose kernels read
 * bytes[offsets[t] .. offsets[t+1]) without bounds checks.
 *
 * Writes to *first_bad (device, one int32) -1 when offsets[0] = 0, offsets
 * is non-decreasing and offsets[V] <= num_bytes; otherwise the smallest t
 * in [0, V] at which that fails (t = 0: offsets[0] != 0; t >= 1:
 * offsets[t] < offsets[t-1] or offsets[t] > num_bytes).  The result is
 * valid once the stream has reached the call.
 *
 * offsets    [V+1] int32 (device), num_tokens = V in [1, DV_MAX_TOKENS];
 * num_bytes  the number of bytes the caller's bytes array holds (>= 0).
 * (dv_align itself reads a decreasing pair as an empty token, never as
 * anything else; bytes past the array are the case only this check
 * catches.)
 * Errors: DV_ERR_INVALID_ARG (NULL), DV_ERR_SHAPE, DV_ERR_ALIAS (first_bad
 *   inside offsets), DV_ERR_HIP.
 */
DV_API dv_status dv_validate_vocab(const int32_t *offsets, int32_t num_tokens, int64_t num_bytes,
                                   int32_t *first_bad, void *stream);

/*
 * dv_masked_step_workspace_bytes -- device workspace dv_masked_step needs for
 * `batch` rows of `num_tokens` logits, for either dtype: where a row is
 * split over several blocks, they meet there (up to four blocks per row in
 * pairs, one 64-bit word per pair; more through a running maximum and an
 * arrival count per row; the block that finishes the row writes its
 * outputs and puts its words back to zero).  Returns 0 when a size is
 * outside its limit.
 */
DV_API size_t dv_masked_step_workspace_bytes(int32_t batch, int32_t num_tokens);

/*
 * dv_masked_step -- one greedy constrained decoding step (Algorithm 1:
 * mask, apply, decode, update; the argmax of Algorithm 3 restricted to the
 * admissible tokens).
 *
 * For every row b in [0, B):
 *     s = states[b];  if s is outside [0, S) the row is dead;
 *     token[b] = the index i in [0, V) with allow bit (s, i) set whose logit
 *                logits[b*ld_logits + i] is largest; ties go to the lowest
 *                index; NaN ranks as -infinity; -0.0 equals +0.0;
 *                -1 when the row is dead or has no allowed token;
 *     new_state[b] = next_state[s*V + token[b]], or DV_DEAD when token = -1.
 *
 * Inputs (device, read only):
 *   next_state [S][V] int32 and allow [S][ceil(V/32)] uint32 as written by
 *              dv_align (any table with that layout is accepted; new_state
 *              is read from it as is).
 *   states     [B] int32.
 *   logits     [B][ld_logits] of `dtype` (dv_dtype), row stride ld_logits
 *              elements (ld_logits >= V); the pointer must be aligned to
 *              the element size.  bf16 rows of any such alignment take the
 *              vector path (up to 7 elements before the row's first 16-byte
 *              boundary are read one by one); fp32 rows not 16-byte aligned
 *              take a scalar path with the same results.
 * Outputs (device): token [B] int32, new_state [B] int32.  They must not
 *   overlap each other or any input (callers ping-pong two state buffers).
 * Workspace: at least dv_masked_step_workspace_bytes(B, V) bytes of device
 *   memory, 256-byte aligned, all zero before its first use (clear it once,
 *   e.g. with hipMemset); every call leaves it all zero again, so it can be
 *   reused by any later call of any size without clearing.  Calls that share
 *   a workspace must be ordered on one stream.
 * B = 0 is valid and enqueues nothing; states, logits, token and new_state
 *   may then be NULL (the pointers of empty tensors).
 * Errors: DV_ERR_INVALID_ARG (also for logits not aligned to the element
 *   size), DV_ERR_SHAPE (S, V, B out of range or ld_logits < V),
 *   DV_ERR_DTYPE, DV_ERR_ALIAS, DV_ERR_WORKSPACE, DV_ERR_HIP.
 */
DV_API dv_status dv_masked_step(const int32_t *next_state, const uint32_t *allow,
                         int32_t num_states, int32_t num_tokens,
                         const int32_t *states, const void *logits, int32_t dtype,
                         int32_t batch, int64_t ld_logits,
                         int32_t *token, int32_t *new_state,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * dv_masked_step_noalloc -- dv_masked_step without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation).  Results are
 * exactly those of dv_masked_step.
 *
 * Split rows meet in a scratch array the library holds on each GPU it runs
 * on (768 KiB, enough for DV_NOALLOC_MAX_BATCH rows; kept until the process
 * ends).  The first call on a device looks the array up and enqueues a
 * kernel on `stream` that clears it; every call leaves it all zero.  The
 * call allocates nothing.  All calls on one GPU share the array: calls that
 * may overlap on one GPU (other streams, other threads) race and must be
 * ordered by the caller; give concurrent work dv_masked_step with a
 * workspace each.
 *
 * Arguments as dv_masked_step, without workspace and workspace_bytes.
 * Errors as dv_masked_step; DV_ERR_SHAPE also for batch >
 *   DV_NOALLOC_MAX_BATCH; DV_ERR_HIP if the scratch array cannot be found or
 *   cleared.
 */
DV_API dv_status dv_masked_step_noalloc(const int32_t *next_state, const uint32_t *allow,
                         int32_t num_states, int32_t num_tokens,
                         const int32_t *states, const void *logits, int32_t dtype,
                         int32_t batch, int64_t ld_logits,
                         int32_t *token, int32_t *new_state, void *stream);

/*
 * dv_masked_step_opportunistic -- dv_masked_step with opportunistic masking
 * (Sec. 3.5, further optimizations): the model's own greedy choice over all
 * V logits is found first, without reading the mask, and checked against
 * the mask; only when it is not allowed is the masked choice computed.
 *
 * The outputs are exactly those of dv_masked_step (an allowed overall
 * maximum at the lowest index is also the masked one), so the two are
 * interchangeable; this one reads less memory when the model mostly picks
 * allowed tokens and reads a row twice when it does not.  The check runs
 * first for bf16 rows that one block covers (batch >= 256, or batch >= 64
 * with rows of at most 32768 tokens); other shapes (fp32 rows, rows split
 * over several blocks) take dv_masked_step's kernels.
 * Arguments, workspace (dv_masked_step_workspace_bytes) and errors as
 *   dv_masked_step.
 */
DV_API dv_status dv_masked_step_opportunistic(const int32_t *next_state, const uint32_t *allow,
                         int32_t num_states, int32_t num_tokens,
                         const int32_t *states, const void *logits, int32_t dtype,
                         int32_t batch, int64_t ld_logits,
                         int32_t *token, int32_t *new_state,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * dv_masked_sample_workspace_bytes -- device workspace dv_masked_sample needs
 * for `batch` rows of `num_tokens` logits.  Returns 0 when a size is outside
 * its limit.
 */
DV_API size_t dv_masked_sample_workspace_bytes(int32_t batch, int32_t num_tokens);

/*
 * dv_masked_sample -- one sampled constrained decoding step (Algorithm 1's
 * decode "argmax or sample"; the paper samples at temperature 1.0, Sec. 4).
 *
 * For every row b with a live state s (as dv_masked_step), the token is
 * drawn from softmax(logits / T) restricted to the allowed tokens, as the
 * Gumbel-max choice
 *     token[b] = argmax over allowed i of  fma(x_i, inv_temperature, G_i)
 * in binary32 (x_i the logit, widened exactly from bf16), NaN ranking as
 * -infinity and ties going to the lowest index, with the noise
 *     G_i = -ln(-ln U_i),  U_i = (2 (w >> 9) + 1) 2^-24,
 *     w = word (i mod 4) of Philox4x32-10 (Salmon et al., SC 2011) with
 *         key (seed mod 2^32, seed >> 32) and
 *         counter (i / 4, b, offset mod 2^32, offset >> 32),
 * and ln evaluated in binary32 by fixed IEEE steps (x = m 2^e with m in
 * [sqrt(1/2), sqrt(2)); z = (m - 1) r, r = 1/(m + 1) by four Newton steps
 * t = fma(-d, r, 1), r = fma(r, t, r) from r = 1/2; ln m = 2 h with
 * h = fma(z^3, p, z), p = 1/3 + w (1/5 + w (1/7 + w/9)) by fused
 * multiply-adds, w = z^2; ln x = fma(e, ln 2, ln m)), so the draw is the
 * same on every device.  new_state[b] = next_state[s*V + token[b]]; a dead
 * row or a row with nothing allowed gives token -1 and DV_DEAD.  Rows are
 * independent draws; use a different `offset` for every step (the pair
 * (seed, offset) names one draw of the whole batch).
 *
 * inv_temperature = 1/T, finite and > 0 (T -> 0 approaches dv_masked_step).
 * Other arguments and errors as dv_masked_step (DV_ERR_SHAPE also for a
 * bad inv_temperature); workspace: dv_masked_sample_workspace_bytes(B, V),
 * zero before its first use and left zero, as for dv_masked_step.
 */
DV_API dv_status dv_masked_sample(const int32_t *next_state, const uint32_t *allow,
                         int32_t num_states, int32_t num_tokens,
                         const int32_t *states, const void *logits, int32_t dtype,
                         int32_t batch, int64_t ld_logits, float inv_temperature,
                         uint64_t seed, uint64_t offset,
                         int32_t *token, int32_t *new_state,
                         void *workspace, size_t workspace_bytes, void *stream);

/*
 * dv_spec_walk -- speculative chain check (Sec. 3.6): how many of a row's
 * proposed tokens the constraint admits, one after the other.
 *
 * For every row b in [0, B), with s = num_proposed proposals
 * p_j = proposals[b*ld_proposals + j] and q_0 = states[b] (DV_DEAD if
 * outside [0, S)):
 *     p_j is admitted when q_j is a state in [0, S), p_j is in [0, V) and
 *         the allow bit (q_j, p_j) is set; then q_{j+1} = next_state[q_j*V + p_j];
 *     accepted[b]    = the number a of leading admitted proposals;
 *     final_state[b] = the table entry reached by the last admitted proposal
 *                      (q_0 when a = 0).
 * Proposal ids outside [0, V) are not errors: they are not admitted.
 *
 * Inputs (device, read only): next_state, allow, states as for
 *   dv_masked_step; proposals [B][ld_proposals] int32 (ld_proposals >= s;
 *   may be NULL when s = 0).
 * Outputs (device): accepted [B], final_state [B] int32; they must not
 *   overlap each other or any input.  No workspace.
 * B = 0 is valid and enqueues nothing (then only next_state and allow must
 *   be non-NULL).
 * Errors: DV_ERR_INVALID_ARG, DV_ERR_SHAPE (S, V, B or s out of range,
 *   ld_proposals < s), DV_ERR_ALIAS, DV_ERR_HIP.
 */
DV_API dv_status dv_spec_walk(const int32_t *next_state, const uint32_t *allow,
                       int32_t num_states, int32_t num_tokens,
                       const int32_t *states, const int32_t *proposals,
                       int32_t num_proposed, int64_t ld_proposals, int32_t batch,
                       int32_t *accepted, int32_t *final_state, void *stream);

/*
 * dv_spec_verify_workspace_bytes -- device workspace dv_spec_verify needs for
 * `batch` rows of `num_proposed` proposals over `num_tokens` logits (the
 * state of every position and the masked step's meeting entries).  Returns 0
 * when a size is outside its limit.
 */
DV_API size_t dv_spec_verify_workspace_bytes(int32_t batch, int32_t num_proposed,
                                             int32_t num_tokens);

/*
 * dv_spec_verify -- verification of proposed tokens with greedy decoding
 * (Sec. 3.6: the model scores all proposed positions in one pass and the
 * proposals it does not confirm are discarded; its choice at a position is
 * the masked greedy decode of Algorithm 1).
 *
 * Row b proposes s = num_proposed tokens p_j = proposals[b*ld_proposals + j].
 * The logits the model gives at position j (j = 0 .. s, after reading the
 * first j proposals) are V elements at logits[b*ld_row + j*ld_pos].  With
 * q_j the state after the first j proposals as defined by dv_spec_walk, and
 * DV_DEAD once a proposal was not admitted:
 *     token[b*(s+1) + j] = the masked greedy choice of dv_masked_step in
 *                          state q_j for position j's logits (-1 when q_j is
 *                          DV_DEAD or allows nothing);
 *     accepted[b]        = the first j < s whose choice is -1 or differs from
 *                          p_j, else s: the proposals p_0 .. p_{a-1} agree with
 *                          the model and token[b][0 .. a] are the tokens
 *                          plain greedy decoding emits (a + 1 of them, a if
 *                          token[b][a] = -1);
 *     new_state[b]       = next_state[q_a*V + token[b][a]], or DV_DEAD when
 *                          token[b][a] = -1.
 * The tokens emitted are exactly those of one-step-at-a-time decoding with
 * dv_masked_step on the same logits; an end-of-sequence token among them
 * ends the sequence at that point (the caller truncates there).
 *
 * Inputs (device, read only): next_state, allow, states as for
 *   dv_masked_step; proposals [B][ld_proposals] int32 (ld_proposals >= s;
 *   may be NULL when s = 0; ids outside [0, V) are never confirmed);
 *   logits of `dtype`, aligned to the element size, any non-negative
 *   ld_row and ld_pos (a model's [B][s+1][V] output is ld_row = (s+1)*V,
 *   ld_pos = V).
 * Outputs (device): token [B][s+1], accepted [B], new_state [B] int32; they
 *   must not overlap each other, an input or the workspace.
 * Workspace: at least dv_spec_verify_workspace_bytes(B, s, V) bytes of
 *   device memory, 256-byte aligned, all zero before its first use and left
 *   all zero by every call (as for dv_masked_step).  Calls that share a
 *   workspace must be ordered on one stream.
 * B = 0 is valid and enqueues nothing.
 * Errors: DV_ERR_INVALID_ARG (also for misaligned logits), DV_ERR_SHAPE
 *   (S, V, B or s out of range, B*(s+1) > DV_MAX_BATCH, ld_proposals < s,
 *   a negative or too large stride), DV_ERR_DTYPE, DV_ERR_ALIAS,
 *   DV_ERR_WORKSPACE, DV_ERR_HIP.
 */
DV_API dv_status dv_spec_verify(const int32_t *next_state, const uint32_t *allow,
                         int32_t num_states, int32_t num_tokens,
                         const int32_t *states, const int32_t *proposals,
                         int32_t num_proposed, int64_t ld_proposals,
                         const void *logits, int32_t dtype, int64_t ld_row, int64_t ld_pos,
                         int32_t batch, int32_t *token, int32_t *accepted, int32_t *new_state,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Static, human-readable name of a status code ("DV_OK", ...). */
DV_API const char *dv_status_string(int32_t status);

/* Detail of the last error returned on the calling thread ("" if none).
 * The string stays valid until the next dv_* call on that thread. */
DV_API const char *dv_last_error(void);

/* Library ABI version: major * 10000 + minor * 100 + patch. */
DV_API int32_t dv_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DV_H */
