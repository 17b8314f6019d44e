/*
 * CPU oracle for vocabulary alignment and masked greedy decoding.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * statement of what the GPU path computes.  Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or constant with the HIP library and never includes it.
 *
 * Definitions followed (paper: "Guiding LLMs The Right Way", DOMINO):
 *   - Alignment (Sec. 3.3, Algorithm 2): for every scanner state q and every
 *     vocabulary token, follow the scanner's transitions on the token's
 *     characters and record where the token leads.  For a regular constraint
 *     walked to full depth (Sec. 3.5, k = infinity) the landing state of a
 *     token is all that matters: the token is a valid continuation exactly
 *     when the walk does not die.
 *   - Mask (Sec. 2, Algorithm 1, "compute mask"): the set of tokens that are
 *     valid continuations of the current state.
 *   - Decode (Algorithm 1 "decode", Appendix B Algorithm 3): argmax of the
 *     logits restricted to the admissible token set.
 *
 * Readings where the paper is silent (listed again in the design notes):
 *   - Alphabet: bytes (256 symbols); tokens are byte strings.
 *   - DEAD = -1 is a sentinel, never a row.  Any transition target or input
 *     state outside [0, S) reads as DEAD; walking from DEAD stays DEAD.
 *   - A zero-length token leaves the state unchanged.
 *   - Ties go to the lowest token index.  NaN logits rank as -infinity.
 *     -0.0 and +0.0 compare equal (IEEE), so they tie.
 *   - A row whose state is DEAD or that has no allowed token yields
 *     token = -1 and new_state = DEAD.
 *   - Allow bitmask: word t/32, bit t%32 (least significant bit first),
 *     row stride ceil(V/32) words, bits for t >= V are zero.
 *   - Logit values are compared in double precision after exact conversion
 *     (fp32 -> double, bf16 -> fp32 by placing the 16 bits in the high half).
 *
 * Build: gcc -O2 -shared -fPIC -o libdv_oracle.so dv_oracle.c
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define ORACLE_DEAD (-1)

/* Any value outside [0, S) is the dead sentinel. */
static int32_t oracle_canon(int64_t x, int32_t num_states)
{
    if (x >= 0 && x < num_states)
        return (int32_t)x;
    return ORACLE_DEAD;
}

/* Walk one byte string through the DFA from state s (Algorithm 2, the
 * q.traverse(token) step, restricted to a deterministic scanner). */
int32_t oracle_walk(const int32_t *trans, int32_t num_states, int32_t s,
                    const uint8_t *str, int64_t len)
{
    int32_t st = oracle_canon(s, num_states);
    for (int64_t i = 0; i < len; ++i) {
        if (st == ORACLE_DEAD)
            return ORACLE_DEAD;
        st = oracle_canon(trans[(int64_t)st * 256 + str[i]], num_states);
    }
    return st;
}

/* next_state / allow rows for an explicit list of source states, with an
 * optional end-of-sequence token (eos_token >= 0).  Algorithm 1 stops on
 * EOS, and Sec. 3.2 makes EOS one more terminal of the scanner, so EOS may
 * follow wherever a terminal sequence may end: it is allowed exactly in
 * the states flagged in `accepting` (NULL: none), and leaves the state
 * unchanged; its bytes are ignored.
 * next_state is [nrows][V] and allow is [nrows][ceil(V/32)]. */
void oracle_align_rows_eos(const int32_t *trans, int32_t num_states,
                           const int32_t *offsets, const uint8_t *bytes,
                           int32_t num_tokens, const uint8_t *accepting,
                           int32_t eos_token, const int32_t *rows, int64_t nrows,
                           int32_t *next_state, uint32_t *allow)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    for (int64_t r = 0; r < nrows; ++r) {
        int32_t s = rows[r];
        int32_t *ns_row = next_state + r * (int64_t)num_tokens;
        uint32_t *al_row = allow + r * words;
        memset(al_row, 0, (size_t)words * sizeof(uint32_t));
        for (int32_t t = 0; t < num_tokens; ++t) {
            int32_t ns;
            if (t == eos_token) {
                int32_t cs = oracle_canon(s, num_states);
                ns = (cs != ORACLE_DEAD && accepting != NULL && accepting[cs]) ? cs : ORACLE_DEAD;
            } else {
                int64_t begin = offsets[t];
                int64_t len = (int64_t)offsets[t + 1] - begin;
                ns = oracle_walk(trans, num_states, s, bytes + begin, len);
            }
            ns_row[t] = ns;
            if (ns != ORACLE_DEAD)
                al_row[t / 32] |= (uint32_t)1u << (t % 32);
        }
    }
}

/* The same rows without an end-of-sequence token. */
void oracle_align_rows(const int32_t *trans, int32_t num_states,
                       const int32_t *offsets, const uint8_t *bytes,
                       int32_t num_tokens, const int32_t *rows, int64_t nrows,
                       int32_t *next_state, uint32_t *allow)
{
    oracle_align_rows_eos(trans, num_states, offsets, bytes, num_tokens, NULL, -1,
                          rows, nrows, next_state, allow);
}

/* The whole table: every state 0..S-1 in order. */
void oracle_align(const int32_t *trans, int32_t num_states,
                  const int32_t *offsets, const uint8_t *bytes,
                  int32_t num_tokens, int32_t *next_state, uint32_t *allow)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    for (int32_t s = 0; s < num_states; ++s)
        oracle_align_rows(trans, num_states, offsets, bytes, num_tokens, &s, 1,
                          next_state + (int64_t)s * num_tokens,
                          allow + (int64_t)s * words);
}

/* Exact conversion of one logit to double.  dtype 0 = fp32, 1 = bf16. */
static double oracle_logit(const void *row, int64_t i, int dtype)
{
    float f;
    if (dtype == 0) {
        f = ((const float *)row)[i];
    } else {
        uint32_t bits = (uint32_t)((const uint16_t *)row)[i] << 16;
        memcpy(&f, &bits, sizeof f);
    }
    return (double)f;
}

/* Masked greedy choice over one row: argmax of the logits over the tokens
 * whose allow bit is set (Algorithm 1 mask/apply/decode, Algorithm 3's
 * set-restricted argmax).  Returns -1 when no token is allowed. */
int32_t oracle_masked_argmax(const uint32_t *allow_row, const void *logits_row,
                             int dtype, int32_t num_tokens)
{
    int32_t best = -1;
    double best_v = 0.0;
    for (int32_t i = 0; i < num_tokens; ++i) {
        if (((allow_row[i / 32] >> (i % 32)) & 1u) == 0)
            continue;
        double v = oracle_logit(logits_row, i, dtype);
        if (isnan(v))
            v = -INFINITY;
        if (best == -1 || v > best_v) {
            best = i;
            best_v = v;
        }
    }
    return best;
}

/* One masked decode step for a batch (Algorithm 1: mask, apply, decode,
 * then update the constraint state with the chosen token). */
void oracle_masked_step(const int32_t *next_state, const uint32_t *allow,
                        int32_t num_states, int32_t num_tokens,
                        const int32_t *states, const void *logits, int dtype,
                        int32_t batch, int64_t ld_logits, int32_t *token,
                        int32_t *new_state)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    size_t elt = dtype == 0 ? 4 : 2;
    for (int32_t b = 0; b < batch; ++b) {
        int32_t s = oracle_canon(states[b], num_states);
        int32_t tok = -1;
        if (s != ORACLE_DEAD) {
            const void *row = (const char *)logits + (size_t)b * (size_t)ld_logits * elt;
            tok = oracle_masked_argmax(allow + (int64_t)s * words, row, dtype, num_tokens);
        }
        token[b] = tok;
        new_state[b] = tok == -1 ? ORACLE_DEAD
                                 : next_state[(int64_t)s * num_tokens + tok];
    }
}

/* Count the transitions a walk takes (the lookups an implementation must
 * make): the number of bytes consumed before the walk ends or dies. */
int64_t oracle_walk_lookups(const int32_t *trans, int32_t num_states,
                            const int32_t *offsets, const uint8_t *bytes,
                            int32_t num_tokens, const int32_t *rows, int64_t nrows)
{
    int64_t total = 0;
    for (int64_t r = 0; r < nrows; ++r) {
        for (int32_t t = 0; t < num_tokens; ++t) {
            int32_t st = oracle_canon(rows[r], num_states);
            for (int64_t i = offsets[t]; i < offsets[t + 1]; ++i) {
                if (st == ORACLE_DEAD)
                    break;
                st = oracle_canon(trans[(int64_t)st * 256 + bytes[i]], num_states);
                ++total;
            }
        }
    }
    return total;
}

/* Histogram of walk lengths: hist[k] counts the (row state, token) walks
 * that take exactly k transitions before they end or die (k >= max_len
 * counts in hist[max_len]).  From it, the lookups past a given depth d are
 * the sum over k of hist[k] * max(k - d, 0). */
void oracle_walk_length_hist(const int32_t *trans, int32_t num_states,
                             const int32_t *offsets, const uint8_t *bytes,
                             int32_t num_tokens, const int32_t *rows, int64_t nrows,
                             int64_t *hist, int32_t max_len)
{
    for (int32_t k = 0; k <= max_len; ++k)
        hist[k] = 0;
    for (int64_t r = 0; r < nrows; ++r) {
        for (int32_t t = 0; t < num_tokens; ++t) {
            int32_t st = oracle_canon(rows[r], num_states);
            int64_t n = 0;
            for (int64_t i = offsets[t]; i < offsets[t + 1]; ++i) {
                if (st == ORACLE_DEAD)
                    break;
                st = oracle_canon(trans[(int64_t)st * 256 + bytes[i]], num_states);
                ++n;
            }
            hist[n < max_len ? n : max_len] += 1;
        }
    }
}

/* Whether proposal t may follow state s (a live state, t a token id whose
 * allow bit is set): the mask of Algorithm 1 applied to a proposed token. */
static int oracle_legal(const uint32_t *allow, int32_t num_states, int32_t num_tokens,
                        int32_t s, int64_t t)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    if (oracle_canon(s, num_states) == ORACLE_DEAD || t < 0 || t >= num_tokens)
        return 0;
    return (int)((allow[(int64_t)s * words + t / 32] >> (t % 32)) & 1u);
}

/* Speculative chain check (Sec. 3.6): the proposals of row b are
 * proposals[b*ld_proposals + j], j < num_proposed.  accepted[b] is the number
 * of leading proposals that are each allowed in the state the earlier ones
 * lead to; final_state[b] is the state after them (states[b], or DEAD if it
 * is not a state, when none is accepted; else the table entry of the last
 * accepted proposal). */
void oracle_spec_walk(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                      int32_t num_tokens, const int32_t *states, const int32_t *proposals,
                      int32_t num_proposed, int64_t ld_proposals, int32_t batch,
                      int32_t *accepted, int32_t *final_state)
{
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t *prop = proposals + (int64_t)b * ld_proposals;
        int32_t st = oracle_canon(states[b], num_states);
        int32_t fin = st;
        int32_t a = 0;
        while (a < num_proposed && oracle_legal(allow, num_states, num_tokens, st, prop[a])) {
            fin = next_state[(int64_t)st * num_tokens + prop[a]];
            st = oracle_canon(fin, num_states);
            ++a;
        }
        accepted[b] = a;
        final_state[b] = fin;
    }
}

/* Speculative verification with greedy decoding (Sec. 3.6 with Algorithm 1
 * as the decoder).  Row b proposes num_proposed tokens; the model's logits
 * for its position j (j = 0 .. num_proposed, scored after the first j
 * proposals) are at element b*ld_row + j*ld_pos of `logits`.
 *
 * Decoding goes through the positions in order, as Algorithm 1 would one
 * step at a time: at position j the masked greedy choice is made in the
 * state the first j proposals lead to; while it equals proposal j the
 * proposal is accepted and decoding moves on.  The first position whose
 * choice differs (or has no allowed token, or j = num_proposed) ends the
 * row: its choice is the one extra token the model contributes.
 *   token[b*(num_proposed+1) + j]  the masked greedy choice at position j in
 *                                  the state reached by proposals 0..j-1
 *                                  (-1 where that state is DEAD: an earlier
 *                                  proposal was not allowed);
 *   accepted[b]                    the number of accepted proposals a; the
 *                                  tokens emitted are token[b][0..a] (a + 1
 *                                  of them, a if token[b][a] = -1);
 *   new_state[b]                   the state after the emitted tokens
 *                                  (table entry of token[b][a]; DEAD if -1). */
void oracle_spec_verify(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                        int32_t num_tokens, const int32_t *states, const int32_t *proposals,
                        int32_t num_proposed, int64_t ld_proposals, const void *logits, int dtype,
                        int64_t ld_row, int64_t ld_pos, int32_t batch, int32_t *token,
                        int32_t *accepted, int32_t *new_state)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    size_t elt = dtype == 0 ? 4 : 2;
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t *prop = proposals + (int64_t)b * ld_proposals;
        int32_t *tok_row = token + (int64_t)b * (num_proposed + 1);
        int32_t st = oracle_canon(states[b], num_states);
        int32_t a = -1, ns = ORACLE_DEAD;
        for (int32_t j = 0; j <= num_proposed; ++j) {
            const void *row = (const char *)logits + (size_t)(b * ld_row + j * ld_pos) * elt;
            int32_t tok = -1;
            if (st != ORACLE_DEAD)
                tok = oracle_masked_argmax(allow + (int64_t)st * words, row, dtype, num_tokens);
            tok_row[j] = tok;
            if (a < 0 && (j == num_proposed || tok == -1 || tok != prop[j])) {
                a = j;
                ns = tok == -1 ? ORACLE_DEAD : next_state[(int64_t)st * num_tokens + tok];
            }
            if (j < num_proposed) {
                if (oracle_legal(allow, num_states, num_tokens, st, prop[j]))
                    st = oracle_canon(next_state[(int64_t)st * num_tokens + prop[j]], num_states);
                else
                    st = ORACLE_DEAD;
            }
        }
        accepted[b] = a;
        new_state[b] = ns;
    }
}

/* Opportunistic masking (Sec. 3.5, further optimizations): decode first
 * without the constraint, check the model's own choice against the mask,
 * and compute the masked choice only when that check fails.  The
 * unconstrained choice follows the same value rules as the masked one
 * (NaN ranks as -inf, ties to the lowest index). */
void oracle_masked_step_opportunistic(const int32_t *next_state, const uint32_t *allow,
                                      int32_t num_states, int32_t num_tokens,
                                      const int32_t *states, const void *logits, int dtype,
                                      int32_t batch, int64_t ld_logits, int32_t *token,
                                      int32_t *new_state, uint8_t *unconstrained_ok)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    size_t elt = dtype == 0 ? 4 : 2;
    for (int32_t b = 0; b < batch; ++b) {
        int32_t s = oracle_canon(states[b], num_states);
        const void *row = (const char *)logits + (size_t)b * (size_t)ld_logits * elt;
        int32_t tok = -1;
        int ok = 0;
        if (s != ORACLE_DEAD) {
            /* the model's own greedy choice: argmax over every token */
            int32_t free_tok = 0;
            double best_v = 0.0;
            for (int32_t i = 0; i < num_tokens; ++i) {
                double v = oracle_logit(row, i, dtype);
                if (isnan(v))
                    v = -INFINITY;
                if (i == 0 || v > best_v) {
                    free_tok = i;
                    best_v = v;
                }
            }
            const uint32_t *arow = allow + (int64_t)s * words;
            ok = (int)((arow[free_tok / 32] >> (free_tok % 32)) & 1u);
            tok = ok ? free_tok : oracle_masked_argmax(arow, row, dtype, num_tokens);
        }
        token[b] = tok;
        new_state[b] = tok == -1 ? ORACLE_DEAD : next_state[(int64_t)s * num_tokens + tok];
        if (unconstrained_ok)
            unconstrained_ok[b] = (uint8_t)ok;
    }
}

/* ------------------------------------------------------------------------
 * Masked sampling.  The paper samples at temperature 1.0 (Sec. 4, setup) and
 * Algorithm 1's decode may be "argmax or sample".  The sampled token is the
 * Gumbel-max choice over the admissible set:
 *     token = argmax over allowed i of  x_i / T + G_i,   G_i ~ Gumbel(0, 1),
 * which draws i with probability softmax(x / T) restricted to the allowed
 * tokens.  G_i = -ln(-ln U_i) with U_i from a counter-based generator, so the
 * draw is reproducible and the same on every device:
 *   - Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random
 *     numbers: as easy as 1, 2, 3", SC 2011), key = (seed low, seed high),
 *     counter = (i / 4, row, offset low, offset high), word i % 4 -> w;
 *   - U = (2 (w >> 9) + 1) 2^-24, exactly, strictly inside (0, 1);
 *   - ln in binary32 by fixed steps that every IEEE implementation rounds
 *     alike (no library log, no division):  x = m 2^e with m in
 *     [sqrt(1/2), sqrt(2)); f = m - 1; r = 1 / (2 + f) by four Newton steps
 *     from 1/2 (each t = fma(-d, r, 1), r = fma(r, t, r)); z = f r;
 *     ln m = 2 (z + z^3 (1/3 + w (1/5 + w (1/7 + w / 9)))), w = z^2, with
 *     the polynomial by fused multiply-adds; ln x = fma(e, ln 2, ln m);
 *   - the key is fma(x_i, 1/T, G_i) in binary32, NaN ranks as -infinity,
 *     ties go to the lowest index.
 * ------------------------------------------------------------------------ */

void oracle_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {            /* the key is bumped between rounds */
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

static float oracle_bits_f32(uint32_t u)
{
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static uint32_t oracle_f32_bits(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    return u;
}

/* Natural log of a positive normal binary32 by the fixed steps above. */
float oracle_ln_f32(float x)
{
    uint32_t bits = oracle_f32_bits(x);
    int32_t e = (int32_t)(bits >> 23) - 127;
    uint32_t mb = (bits & 0x007FFFFFu) | 0x3F800000u;
    if (mb > 0x3FB504F3u) {         /* m above sqrt(2): halve it */
        mb -= 0x00800000u;
        e += 1;
    }
    float f = oracle_bits_f32(mb) - 1.0f;
    float d = f + 2.0f;
    float r = 0.5f;
    for (int it = 0; it < 4; ++it) {
        float t = fmaf(-d, r, 1.0f);
        r = fmaf(r, t, r);
    }
    float z = f * r;
    float w = z * z;
    float p = fmaf(w, 0x1.c71c72p-4f, 0x1.24924ap-3f);  /* 1/9, 1/7 */
    p = fmaf(w, p, 0x1.99999ap-3f);                       /* 1/5 */
    p = fmaf(w, p, 0x1.555556p-2f);                       /* 1/3 */
    float zw = z * w;
    float half = fmaf(zw, p, z);
    float lnm = half + half;
    return fmaf((float)e, 0x1.62e430p-1f, lnm);           /* ln 2 */
}

/* The Gumbel noise of (seed, offset, row, token). */
float oracle_gumbel(uint64_t seed, uint64_t offset, uint32_t row, uint32_t token)
{
    uint32_t ctr[4] = {token / 4u, row, (uint32_t)offset, (uint32_t)(offset >> 32)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t out[4];
    oracle_philox4x32_10(ctr, key, out);
    uint32_t w = out[token % 4u];
    float u = (float)(2u * (w >> 9) + 1u) * 0x1p-24f;
    return -oracle_ln_f32(-oracle_ln_f32(u));
}

/* One sampled masked step: as oracle_masked_step with the Gumbel-max draw
 * in place of the argmax.  inv_temperature = 1 / T > 0. */
void oracle_masked_sample(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                          int32_t num_tokens, const int32_t *states, const void *logits, int dtype,
                          int32_t batch, int64_t ld_logits, float inv_temperature, uint64_t seed,
                          uint64_t offset, int32_t *token, int32_t *new_state)
{
    int64_t words = ((int64_t)num_tokens + 31) / 32;
    size_t elt = dtype == 0 ? 4 : 2;
    for (int32_t b = 0; b < batch; ++b) {
        int32_t s = oracle_canon(states[b], num_states);
        int32_t best = -1;
        float best_key = 0.0f;
        if (s != ORACLE_DEAD) {
            const void *row = (const char *)logits + (size_t)b * (size_t)ld_logits * elt;
            const uint32_t *arow = allow + (int64_t)s * words;
            for (int32_t i = 0; i < num_tokens; ++i) {
                if (((arow[i / 32] >> (i % 32)) & 1u) == 0)
                    continue;
                float x = (float)oracle_logit(row, i, dtype);   /* exact: the logit is binary32 or bf16 */
                float key = fmaf(x, inv_temperature, oracle_gumbel(seed, offset, (uint32_t)b, (uint32_t)i));
                if (isnan(key))
                    key = -INFINITY;
                if (best == -1 || key > best_key) {
                    best = i;
                    best_key = key;
                }
            }
        }
        token[b] = best;
        new_state[b] = best == -1 ? ORACLE_DEAD : next_state[(int64_t)s * num_tokens + best];
    }
}
