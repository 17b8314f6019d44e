// Speculative chain check (Sec. 3.6) on CDNA4 (gfx950).
//
// A row proposes s tokens; the model scores all s + 1 positions in one pass.
//   * Legality walk (dv_spec_walk): one lane per row follows its proposals
//     through the alignment table -- the allow bit says whether a proposal
//     may follow, next_state where it leads.  Each hop's two loads (mask word
//     and table entry) are issued together at clamped, always-valid
//     addresses, so a hop costs one memory round trip.
//   * Verification (dv_spec_verify): the masked greedy step runs over all
//     B (s + 1) positions at once as independent rows -- the HBM-bound part,
//     with positions past a proposal that is not allowed costing no logit
//     reads.  Each position's block walks its own j proposals after its
//     first batch of logits is in flight, so the walk's round trips overlap
//     other blocks' streaming instead of forming a serial kernel of their
//     own.  A last lane-per-row pass finds the first position whose choice
//     differs from its proposal.
#include "dv_internal.h"

namespace dv {
namespace {

constexpr int kSpecThreads = 256;

// One lane per row: walk the row's proposals.  Writes the number of leading
// allowed proposals and the table entry reached by the last of them.
__global__ __launch_bounds__(kSpecThreads) void spec_chain_kernel(
    const int32_t *__restrict__ next_state, const uint32_t *__restrict__ allow, int S, int V,
    const int32_t *__restrict__ states, const int32_t *__restrict__ proposals, int s, int64_t ld_prop,
    int B, int32_t *__restrict__ accepted, int32_t *__restrict__ final_state)
{
    const int b = blockIdx.x * kSpecThreads + threadIdx.x;
    if (b >= B)
        return;
    const int32_t *prop = proposals + (size_t)b * (size_t)ld_prop;
    int st = states[b];
    st = (uint32_t)st < (uint32_t)S ? st : -1;
    int fin = st, a = 0;
#pragma unroll 4
    for (int j = 0; j < s; ++j) {
        const int t = prop[j];
        bool legal;
        const int nx = spec_hop(next_state, allow, S, V, st, t, legal);
        if (legal) {
            ++a;
            // the table entry as stored (spec_hop maps entries outside [0, S) to -1)
            fin = next_state[(size_t)st * (size_t)V + (size_t)t];
        }
        st = nx;
    }
    accepted[b] = a;
    final_state[b] = fin;
}

// One lane per row: the first position whose choice is not its proposal (or
// is -1) ends the row; its choice is the model's own token.
__global__ __launch_bounds__(kSpecThreads) void spec_accept_kernel(
    const int32_t *__restrict__ token, const int32_t *__restrict__ proposals, int s, int64_t ld_prop, int B,
    int32_t *__restrict__ pos_new, int32_t *__restrict__ accepted, int32_t *__restrict__ new_state)
{
    const int b = blockIdx.x * kSpecThreads + threadIdx.x;
    if (b >= B)
        return;
    const int32_t *prop = proposals + (size_t)b * (size_t)ld_prop;
    const int32_t *tok = token + (size_t)b * (size_t)(s + 1);
    int32_t *pn = pos_new + (size_t)b * (size_t)(s + 1);
    // no early exit, and every position's state read alongside its token:
    // the loads of several positions are in flight together, in one round
    // trip instead of one per position
    int a = s, ns = pn[s];
#pragma unroll 8
    for (int j = 0; j < s; ++j) {
        const int t = tok[j], p = prop[j], n = pn[j];
        if (a == s && (t == -1 || t != p)) {
            a = j;
            ns = n;
        }
    }
    accepted[b] = a;
    new_state[b] = ns;
    // the workspace is handed back all zero, like the step's part of it
#pragma unroll 8
    for (int j = 0; j <= s; ++j)
        pn[j] = 0;
}

unsigned lanes_grid(int B) { return (unsigned)((B + kSpecThreads - 1) / kSpecThreads); }

}  // namespace

hipError_t launch_spec_walk(const int32_t *next_state, const uint32_t *allow, int S, int V,
                            const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                            int B, int32_t *accepted, int32_t *final_state, hipStream_t stream)
{
    spec_chain_kernel<<<lanes_grid(B), kSpecThreads, 0, stream>>>(next_state, allow, S, V, states, proposals, s,
                                                                  ld_prop, B, accepted, final_state);
    return hipGetLastError();
}

hipError_t launch_spec_verify(const int32_t *next_state, const uint32_t *allow, int S, int V,
                              const int32_t *states, const int32_t *proposals, int s, int64_t ld_prop,
                              const void *logits, int dtype, int64_t ld_row, int64_t ld_pos, int B,
                              int32_t *token, int32_t *accepted, int32_t *new_state, void *workspace,
                              hipStream_t stream)
{
    char *ws = static_cast<char *>(workspace);
    int32_t *pos_new = reinterpret_cast<int32_t *>(ws);
    void *meet = ws + spec_partial_offset(B, s);  // the step's meeting slots for R rows
    const int R = (int)spec_positions(B, s);
    const RowMap map{ld_row, ld_pos, s + 1, proposals, ld_prop};
    hipError_t e = launch_masked_rows(next_state, allow, S, V, states, logits, dtype, R, map, token, pos_new,
                                      meet, stream);
    if (e != hipSuccess)
        return e;
    spec_accept_kernel<<<lanes_grid(B), kSpecThreads, 0, stream>>>(token, proposals, s, ld_prop, B, pos_new,
                                                                   accepted, new_state);
    return hipGetLastError();
}

}  // namespace dv
