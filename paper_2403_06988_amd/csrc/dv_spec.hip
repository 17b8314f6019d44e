// Speculative chain check (Sec. 3.6) on CDNA4 (gfx950).
//
// A row proposes s tokens; the model scores all s + 1 positions in one pass.
//   * Legality walk (dv_spec_walk): one lane per row follows its proposals
//     through the alignment table -- the allow bit says whether a proposal
//     may follow, next_state where it leads.  Each hop's two loads (mask word
//     and table entry) are issued together at clamped, always-valid
//     addresses, so a hop costs one memory round trip.
//   * Verification (dv_spec_verify): the same walk writes the state of every
//     position (DEAD after a proposal that is not allowed), then the masked
//     greedy step runs over all B (s + 1) positions at once as independent
//     rows -- the HBM-bound part, with dead positions costing no logit
//     reads -- and a last lane-per-row pass finds the first position whose
//     choice differs from its proposal.
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kSpecThreads = 256;

// One lane per row: walk the row's proposals.  Writes, when non-NULL, the
// state of each position [B][s+1], the number of leading allowed proposals
// and the table entry reached by the last of them.
__global__ __launch_bounds__(kSpecThreads) void spec_chain_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V,
    const int32_t *__restrict__ states, const int32_t *__restrict__ proposals, int s, int64_t ld_prop,
    int B, int32_t *__restrict__ pos_state, int32_t *__restrict__ accepted, int32_t *__restrict__ final_state)
{
    const int b = blockIdx.x * kSpecThreads + threadIdx.x;
    if (b >= B)
        return;
    const size_t W = ((size_t)V + 31) / 32;
    const int32_t *prop = proposals + (size_t)b * (size_t)ld_prop;
    int32_t *pos = pos_state ? pos_state + (size_t)b * (size_t)(s + 1) : nullptr;
    int st = states[b];
    st = (uint32_t)st < (uint32_t)S ? st : -1;
    int fin = st, a = 0;
    for (int j = 0; j < s; ++j) {
        if (pos)
            pos[j] = st;
        const int t = prop[j];
        const bool ok = st >= 0 && (uint32_t)t < (uint32_t)V;
        const size_t si = ok ? (size_t)st : 0, ti = ok ? (size_t)t : 0;
        const uint32_t word = allow[si * W + (ti >> 5)];
        const int nx = next_state[si * (size_t)V + ti];
        const bool legal = ok && ((word >> (ti & 31)) & 1u);
        if (legal) {
            ++a;
            fin = nx;
        }
        st = legal && (uint32_t)nx < (uint32_t)S ? nx : -1;
    }
    if (pos)
        pos[s] = st;
    if (accepted)
        accepted[b] = a;
    if (final_state)
        final_state[b] = fin;
}

// One lane per row: the first position whose choice is not its proposal (or
// is -1) ends the row; its choice is the model's own token.
__global__ __launch_bounds__(kSpecThreads) void spec_accept_kernel(
    const int32_t *__restrict__ token, const int32_t *__restrict__ proposals, int s, int64_t ld_prop, int B,
    const int32_t *__restrict__ pos_new, int32_t *__restrict__ accepted, int32_t *__restrict__ new_state)
{
    const int b = blockIdx.x * kSpecThreads + threadIdx.x;
    if (b >= B)
        return;
    const int32_t *prop = proposals + (size_t)b * (size_t)ld_prop;
    const int32_t *tok = token + (size_t)b * (size_t)(s + 1);
    int a = 0;
    while (a < s && tok[a] != -1 && tok[a] == prop[a])
        ++a;
    accepted[b] = a;
    new_state[b] = pos_new[(size_t)b * (size_t)(s + 1) + a];
}

unsigned lanes_grid(int B) { return (unsigned)((B + kSpecThreads - 1) / kSpecThreads); }

}  // namespace

hipError_t launch_spec_walk(const int32_t *next_state, const uint32_t *allow, int S, int V,
                            const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                            int B, int32_t *accepted, int32_t *final_state, hipStream_t stream)
{
    spec_chain_kernel<<<lanes_grid(B), kSpecThreads, 0, stream>>>(next_state, allow, S, V, states, proposals, s,
                                                                  ld_prop, B, nullptr, accepted, final_state);
    return hipGetLastError();
}

hipError_t launch_spec_verify(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                              const void *logits, int dtype, int64_t ld_row, int64_t ld_pos, int B,
                              int32_t *token, int32_t *accepted, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    char *ws = static_cast<char *>(workspace);
    int32_t *pos_state = reinterpret_cast<int32_t *>(ws);
    int32_t *pos_new = reinterpret_cast<int32_t *>(ws + spec_pos_new_offset(B, s));
    void *partial = ws + spec_partial_offset(B, s);
    const int R = (int)spec_positions(B, s);
    spec_chain_kernel<<<lanes_grid(B), kSpecThreads, 0, stream>>>(next_state, allow, S, V, states, proposals, s,
                                                                  ld_prop, B, pos_state, nullptr, nullptr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    e = launch_masked_rows(next_state, allow, S, V, pos_state, logits, dtype, R, RowMap{ld_row, ld_pos, s + 1},
                           token, pos_new, partial, stream);
    if (e != hipSuccess)
        return e;
    spec_accept_kernel<<<lanes_grid(B), kSpecThreads, 0, stream>>>(token, proposals, s, ld_prop, B, pos_new,
                                                                   accepted, new_state);
    return hipGetLastError();
}

}  // namespace dv
