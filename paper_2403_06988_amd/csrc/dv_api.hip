// C ABI of libdv.so (declared in include/dv.h): argument checks, then the
// launches.  Every check runs on the host before any HIP call, so a rejected
// call enqueues nothing and touches no device state.
#include <stdarg.h>
#include <stdio.h>

#include <atomic>
#include <mutex>

#include "../../include/dv.h"
#include "dv_internal.h"
#include "dv_sample.h"

namespace {

thread_local char g_error[512] = "";

dv_status fail(dv_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return st;
}

// Byte range [p, p + n) of a device pointer, for overlap checks.
struct Range {
    uintptr_t lo, hi;
};
Range range_of(const void *p, size_t n) { return {reinterpret_cast<uintptr_t>(p), reinterpret_cast<uintptr_t>(p) + n}; }
bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi && a.lo != a.hi && b.lo != b.hi; }

dv_status hip_status(hipError_t e, const char *what)
{
    if (e == hipSuccess)
        return DV_OK;
    return fail(DV_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

extern "C" {

int32_t dv_version(void) { return 100; }

const char *dv_status_string(int32_t status)
{
    switch (status) {
    case DV_OK: return "DV_OK";
    case DV_ERR_INVALID_ARG: return "DV_ERR_INVALID_ARG";
    case DV_ERR_SHAPE: return "DV_ERR_SHAPE";
    case DV_ERR_DTYPE: return "DV_ERR_DTYPE";
    case DV_ERR_ALIAS: return "DV_ERR_ALIAS";
    case DV_ERR_WORKSPACE: return "DV_ERR_WORKSPACE";
    case DV_ERR_HIP: return "DV_ERR_HIP";
    default: return "DV_ERR_UNKNOWN";
    }
}

const char *dv_last_error(void) { return g_error; }

size_t dv_align_workspace_bytes(int32_t num_states, int32_t num_tokens)
{
    if (num_states < 1 || num_states > DV_MAX_STATES || num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return 0;
    return dv::align_workspace_bytes(num_states, num_tokens);
}

static dv_status align_common(const char *name, const int32_t *trans, int32_t num_states,
                              const int32_t *offsets, const uint8_t *bytes, int32_t num_tokens,
                              const uint8_t *accepting, int32_t eos_token, int32_t *next_state,
                              uint32_t *allow, void *workspace, size_t workspace_bytes, void *stream)
{
    g_error[0] = '\0';
    if (!trans || !offsets || !next_state || !allow)
        return fail(DV_ERR_INVALID_ARG, "%s: trans, offsets, next_state and allow must be non-NULL", name);
    if (num_states < 1 || num_states > DV_MAX_STATES)
        return fail(DV_ERR_SHAPE, "%s: num_states=%d outside [1, %d]", name, num_states, DV_MAX_STATES);
    if (num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return fail(DV_ERR_SHAPE, "%s: num_tokens=%d outside [1, %d]", name, num_tokens, DV_MAX_TOKENS);
    if (eos_token < -1 || eos_token >= num_tokens)
        return fail(DV_ERR_SHAPE, "%s: eos_token=%d outside [0, %d)", name, eos_token, num_tokens);
    const size_t S = (size_t)num_states, V = (size_t)num_tokens, W = (V + 31) / 32;
    const Range r_ns = range_of(next_state, S * V * 4), r_al = range_of(allow, S * W * 4);
    const Range r_tr = range_of(trans, S * 256 * 4), r_off = range_of(offsets, (V + 1) * 4);
    const Range r_acc = range_of(accepting, accepting ? S : 0);
    if (overlap(r_ns, r_al) || overlap(r_ns, r_tr) || overlap(r_ns, r_off) || overlap(r_al, r_tr) ||
        overlap(r_al, r_off) || overlap(r_ns, r_acc) || overlap(r_al, r_acc))
        return fail(DV_ERR_ALIAS, "%s: next_state / allow overlap each other or an input", name);
    const size_t need = dv::align_workspace_bytes(num_states, num_tokens);
    if (!workspace || workspace_bytes < need)
        return fail(DV_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", name, workspace_bytes, need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(DV_ERR_WORKSPACE, "%s: workspace must be 256-byte aligned", name);
    const Range r_ws = range_of(workspace, need);
    if (overlap(r_ws, r_ns) || overlap(r_ws, r_al) || overlap(r_ws, r_tr) || overlap(r_ws, r_off) ||
        overlap(r_ws, r_acc))
        return fail(DV_ERR_ALIAS, "%s: workspace overlaps an input or output", name);
    // bytes == NULL is accepted; the kernels read it only for non-empty tokens.
    return hip_status(dv::launch_align(trans, num_states, offsets, bytes, num_tokens, accepting, eos_token,
                                       next_state, allow, workspace, static_cast<hipStream_t>(stream)),
                      "launch");
}

dv_status dv_align(const int32_t *trans, int32_t num_states, const int32_t *offsets,
                   const uint8_t *bytes, int32_t num_tokens, int32_t *next_state, uint32_t *allow,
                   void *workspace, size_t workspace_bytes, void *stream)
{
    return align_common("dv_align", trans, num_states, offsets, bytes, num_tokens, nullptr, -1, next_state,
                        allow, workspace, workspace_bytes, stream);
}

dv_status dv_align_eos(const int32_t *trans, int32_t num_states, const int32_t *offsets,
                       const uint8_t *bytes, int32_t num_tokens, const uint8_t *accepting,
                       int32_t eos_token, int32_t *next_state, uint32_t *allow, void *workspace,
                       size_t workspace_bytes, void *stream)
{
    if (eos_token < 0) {
        g_error[0] = '\0';
        return fail(DV_ERR_SHAPE, "dv_align_eos: eos_token=%d must be a token id", eos_token);
    }
    return align_common("dv_align_eos", trans, num_states, offsets, bytes, num_tokens, accepting, eos_token,
                        next_state, allow, workspace, workspace_bytes, stream);
}

dv_status dv_validate_vocab(const int32_t *offsets, int32_t num_tokens, int64_t num_bytes, int32_t *first_bad,
                            void *stream)
{
    g_error[0] = '\0';
    const char *name = "dv_validate_vocab";
    if (!offsets || !first_bad)
        return fail(DV_ERR_INVALID_ARG, "%s: offsets and first_bad must be non-NULL", name);
    if (num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return fail(DV_ERR_SHAPE, "%s: num_tokens=%d outside [1, %d]", name, num_tokens, DV_MAX_TOKENS);
    if (num_bytes < 0)
        return fail(DV_ERR_SHAPE, "%s: num_bytes=%lld must be >= 0", name, (long long)num_bytes);
    if (overlap(range_of(first_bad, 4), range_of(offsets, ((size_t)num_tokens + 1) * 4)))
        return fail(DV_ERR_ALIAS, "%s: first_bad overlaps offsets", name);
    return hip_status(dv::launch_validate_vocab(offsets, num_tokens, num_bytes, first_bad,
                                                static_cast<hipStream_t>(stream)),
                      "dv_validate_vocab launch");
}

size_t dv_masked_step_workspace_bytes(int32_t batch, int32_t num_tokens)
{
    if (batch < 0 || batch > DV_MAX_BATCH || num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return 0;
    return dv::step_workspace_bytes(batch, num_tokens);
}

// How a step call decodes: greedy, greedy with the check first, or sampled.
struct StepMode {
    int kind;  // 0 greedy, 1 opportunistic, 2 sampled, 3 argument checks only
    float inv_temperature;
    uint64_t seed, offset;
};

static dv_status step_common(const char *name, StepMode mode, const int32_t *next_state,
                             const uint32_t *allow, int32_t num_states, int32_t num_tokens, const int32_t *states,
                             const void *logits, int32_t dtype, int32_t batch, int64_t ld_logits, int32_t *token,
                             int32_t *new_state, void *workspace, size_t workspace_bytes, void *stream)
{
    g_error[0] = '\0';
    if (!next_state || !allow)
        return fail(DV_ERR_INVALID_ARG, "%s: next_state and allow must be non-NULL", name);
    if (batch > 0 && (!states || !logits || !token || !new_state))
        return fail(DV_ERR_INVALID_ARG, "%s: states, logits, token and new_state must be "
                                        "non-NULL when batch > 0", name);
    if (num_states < 1 || num_states > DV_MAX_STATES)
        return fail(DV_ERR_SHAPE, "%s: num_states=%d outside [1, %d]", name, num_states, DV_MAX_STATES);
    if (num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return fail(DV_ERR_SHAPE, "%s: num_tokens=%d outside [1, %d]", name, num_tokens, DV_MAX_TOKENS);
    if (batch < 0 || batch > DV_MAX_BATCH)
        return fail(DV_ERR_SHAPE, "%s: batch=%d outside [0, %d]", name, batch, DV_MAX_BATCH);
    if (ld_logits < num_tokens || ld_logits > ((int64_t)1 << 40))
        return fail(DV_ERR_SHAPE, "%s: ld_logits=%lld must be >= num_tokens=%d", name,
                    (long long)ld_logits, num_tokens);
    if (dtype != DV_F32 && dtype != DV_BF16)
        return fail(DV_ERR_DTYPE, "%s: unknown dtype %d", name, dtype);
    if (mode.kind == 2 && !(mode.inv_temperature > 0.0f && mode.inv_temperature <= 3.0e38f))
        return fail(DV_ERR_SHAPE, "%s: inv_temperature=%g must be finite and > 0", name,
                    (double)mode.inv_temperature);
    if (batch == 0)
        return DV_OK;
    const size_t S = (size_t)num_states, V = (size_t)num_tokens, W = (V + 31) / 32, B = (size_t)batch;
    const size_t elt = dtype == DV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(logits) % elt)
        return fail(DV_ERR_INVALID_ARG, "%s: logits must be aligned to their element size (%zu bytes)", name, elt);
    const Range r_tok = range_of(token, B * 4), r_new = range_of(new_state, B * 4);
    const Range r_ns = range_of(next_state, S * V * 4), r_al = range_of(allow, S * W * 4);
    const Range r_st = range_of(states, B * 4);
    const Range r_lg = range_of(logits, ((B - 1) * (size_t)ld_logits + V) * elt);
    if (overlap(r_tok, r_new))
        return fail(DV_ERR_ALIAS, "%s: token and new_state overlap", name);
    for (Range out : {r_tok, r_new})
        if (overlap(out, r_ns) || overlap(out, r_al) || overlap(out, r_st) || overlap(out, r_lg))
            return fail(DV_ERR_ALIAS, "%s: an output overlaps an input "
                                      "(ping-pong two state buffers instead of updating in place)", name);
    if (mode.kind == 3)
        return DV_OK;  // argument checks only (the scratch-backed step checks before its set-up)
    const size_t need = mode.kind == 2 ? dv::sample_workspace_bytes(batch, num_tokens)
                                       : dv::step_workspace_bytes(batch, num_tokens);
    if (!workspace || workspace_bytes < need)
        return fail(DV_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", name, workspace_bytes,
                    need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(DV_ERR_WORKSPACE, "%s: workspace must be 256-byte aligned", name);
    const Range r_ws = range_of(workspace, need);
    for (Range r : {r_tok, r_new, r_ns, r_al, r_st, r_lg})
        if (overlap(r_ws, r))
            return fail(DV_ERR_ALIAS, "%s: workspace overlaps an input or output", name);
    const hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e;
    if (mode.kind == 2)
        e = dv::launch_masked_sample(next_state, allow, num_states, num_tokens, states, logits, dtype, batch,
                                     ld_logits, mode.inv_temperature, mode.seed, mode.offset, token, new_state,
                                     workspace, st);
    else if (mode.kind == 1)
        e = dv::launch_masked_step_opportunistic(next_state, allow, num_states, num_tokens, states, logits, dtype,
                                                 batch, ld_logits, token, new_state, workspace, st);
    else
        e = dv::launch_masked_step(next_state, allow, num_states, num_tokens, states, logits, dtype, batch,
                                   ld_logits, token, new_state, workspace, st);
    return hip_status(e, "launch");
}

dv_status dv_masked_step(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                         int32_t num_tokens, const int32_t *states, const void *logits, int32_t dtype,
                         int32_t batch, int64_t ld_logits, int32_t *token, int32_t *new_state,
                         void *workspace, size_t workspace_bytes, void *stream)
{
    return step_common("dv_masked_step", StepMode{0, 1.0f, 0, 0}, next_state, allow, num_states, num_tokens, states, logits,
                       dtype, batch, ld_logits, token, new_state, workspace, workspace_bytes, stream);
}

// ------------------------------------------------ step without allocation
//
// dv_masked_step_noalloc meets split rows in `scratch`, a device array of
// the library, instead of a caller's workspace.  Its size covers
// DV_NOALLOC_MAX_BATCH rows that meet through a maximum and a count (12
// bytes a row); rows that meet in pairs need up to 24 bytes a row but occur
// only below 256 rows, and the workspace check below refuses any call the
// array would not cover.
// Each GPU holds its own copy until the process ends.  Host code never uses
// the array's name as an address: the device address of each GPU's copy is
// looked up once per device and kept in g_scratch_ptr.
namespace {

constexpr size_t kScratchBytes = dv::row_meet_bytes(DV_NOALLOC_MAX_BATCH);
__device__ __align__(256) uint4 scratch[kScratchBytes / sizeof(uint4)];

constexpr int kMaxScratchDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxScratchDevices];
std::mutex g_scratch_mu;

__global__ void clear_scratch_kernel(uint4 *p, size_t n)
{
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = make_uint4(0, 0, 0, 0);
}

// The current device's scratch address; on a device's first call, looked up
// and cleared with a kernel on `stream` (a kernel, not a memset, so that a
// first call under graph capture records a plain kernel node).
dv_status scratch_for_current_device(const char *name, hipStream_t stream, void **out)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return fail(DV_ERR_HIP, "%s: hipGetDevice: %s", name, hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(DV_ERR_HIP, "%s: device %d beyond the %d devices the scratch table covers", name, dev,
                    kMaxScratchDevices);
    void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p) {
        *out = p;
        return DV_OK;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (!p) {
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(DV_ERR_HIP, "%s: hipGetSymbolAddress(scratch): %s", name, hipGetErrorString(e));
        const size_t n = kScratchBytes / sizeof(uint4);
        clear_scratch_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(static_cast<uint4 *>(p), n);
        e = hipGetLastError();
        if (e != hipSuccess)
            return fail(DV_ERR_HIP, "%s: clearing the scratch array: %s", name, hipGetErrorString(e));
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = p;
    return DV_OK;
}

}  // namespace

dv_status dv_masked_step_noalloc(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                                 int32_t num_tokens, const int32_t *states, const void *logits, int32_t dtype,
                                 int32_t batch, int64_t ld_logits, int32_t *token, int32_t *new_state,
                                 void *stream)
{
    const char *name = "dv_masked_step_noalloc";
    g_error[0] = '\0';
    if (batch > DV_NOALLOC_MAX_BATCH)
        return fail(DV_ERR_SHAPE, "%s: batch=%d exceeds DV_NOALLOC_MAX_BATCH=%d (the scratch array's size); "
                                  "use dv_masked_step with a workspace", name, batch, DV_NOALLOC_MAX_BATCH);
    // The same checks as dv_masked_step, with a stand-in workspace address
    // (never dereferenced: a failed check enqueues nothing) so that no HIP
    // call happens before the arguments are known good.
    const dv_status pre = step_common(name, StepMode{3, 1.0f, 0, 0}, next_state, allow, num_states, num_tokens,
                                      states, logits, dtype, batch, ld_logits, token, new_state, nullptr, 0,
                                      stream);
    if (pre != DV_OK || batch == 0)
        return pre;
    void *ws = nullptr;
    const dv_status got = scratch_for_current_device(name, static_cast<hipStream_t>(stream), &ws);
    if (got != DV_OK)
        return got;
    return step_common(name, StepMode{0, 1.0f, 0, 0}, next_state, allow, num_states, num_tokens, states, logits,
                       dtype, batch, ld_logits, token, new_state, ws, kScratchBytes, stream);
}

dv_status dv_masked_step_opportunistic(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                                       int32_t num_tokens, const int32_t *states, const void *logits,
                                       int32_t dtype, int32_t batch, int64_t ld_logits, int32_t *token,
                                       int32_t *new_state, void *workspace, size_t workspace_bytes,
                                       void *stream)
{
    return step_common("dv_masked_step_opportunistic", StepMode{1, 1.0f, 0, 0}, next_state, allow, num_states, num_tokens, states,
                       logits, dtype, batch, ld_logits, token, new_state, workspace, workspace_bytes, stream);
}

size_t dv_masked_sample_workspace_bytes(int32_t batch, int32_t num_tokens)
{
    if (batch < 0 || batch > DV_MAX_BATCH || num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return 0;
    return dv::sample_workspace_bytes(batch, num_tokens);
}

dv_status dv_masked_sample(const int32_t *next_state, const uint32_t *allow, int32_t num_states, int32_t num_tokens,
                           const int32_t *states, const void *logits, int32_t dtype, int32_t batch,
                           int64_t ld_logits, float inv_temperature, uint64_t seed, uint64_t offset,
                           int32_t *token, int32_t *new_state, void *workspace, size_t workspace_bytes,
                           void *stream)
{
    return step_common("dv_masked_sample", StepMode{2, inv_temperature, seed, offset}, next_state, allow,
                       num_states, num_tokens, states, logits, dtype, batch, ld_logits, token, new_state, workspace,
                       workspace_bytes, stream);
}

static dv_status spec_shape_checks(const char *name, int32_t num_states, int32_t num_tokens, int32_t batch,
                                   int32_t num_proposed, int64_t ld_proposals)
{
    if (num_states < 1 || num_states > DV_MAX_STATES)
        return fail(DV_ERR_SHAPE, "%s: num_states=%d outside [1, %d]", name, num_states, DV_MAX_STATES);
    if (num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return fail(DV_ERR_SHAPE, "%s: num_tokens=%d outside [1, %d]", name, num_tokens, DV_MAX_TOKENS);
    if (batch < 0 || batch > DV_MAX_BATCH)
        return fail(DV_ERR_SHAPE, "%s: batch=%d outside [0, %d]", name, batch, DV_MAX_BATCH);
    if (num_proposed < 0 || num_proposed > DV_MAX_PROPOSED)
        return fail(DV_ERR_SHAPE, "%s: num_proposed=%d outside [0, %d]", name, num_proposed, DV_MAX_PROPOSED);
    if ((int64_t)batch * (num_proposed + 1) > DV_MAX_BATCH)
        return fail(DV_ERR_SHAPE, "%s: batch * (num_proposed + 1) = %lld exceeds %d", name,
                    (long long)batch * (num_proposed + 1), DV_MAX_BATCH);
    if (num_proposed > 0 && (ld_proposals < num_proposed || ld_proposals > ((int64_t)1 << 40)))
        return fail(DV_ERR_SHAPE, "%s: ld_proposals=%lld must be >= num_proposed=%d", name,
                    (long long)ld_proposals, num_proposed);
    return DV_OK;
}

dv_status dv_spec_walk(const int32_t *next_state, const uint32_t *allow, int32_t num_states, int32_t num_tokens,
                       const int32_t *states, const int32_t *proposals, int32_t num_proposed,
                       int64_t ld_proposals, int32_t batch, int32_t *accepted, int32_t *final_state, void *stream)
{
    g_error[0] = '\0';
    const char *name = "dv_spec_walk";
    if (!next_state || !allow)
        return fail(DV_ERR_INVALID_ARG, "%s: next_state and allow must be non-NULL", name);
    if (batch > 0 && (!states || !accepted || !final_state || (num_proposed > 0 && !proposals)))
        return fail(DV_ERR_INVALID_ARG, "%s: states, proposals, accepted and final_state must be non-NULL "
                                        "when batch > 0", name);
    const dv_status st = spec_shape_checks(name, num_states, num_tokens, batch, num_proposed, ld_proposals);
    if (st != DV_OK)
        return st;
    if (batch == 0)
        return DV_OK;
    const size_t S = (size_t)num_states, V = (size_t)num_tokens, W = (V + 31) / 32, B = (size_t)batch;
    const size_t np = (size_t)num_proposed;
    const Range r_acc = range_of(accepted, B * 4), r_fin = range_of(final_state, B * 4);
    const Range r_ns = range_of(next_state, S * V * 4), r_al = range_of(allow, S * W * 4);
    const Range r_st = range_of(states, B * 4);
    const Range r_pr = range_of(proposals, np ? ((B - 1) * (size_t)ld_proposals + np) * 4 : 0);
    if (overlap(r_acc, r_fin))
        return fail(DV_ERR_ALIAS, "%s: accepted and final_state overlap", name);
    for (Range out : {r_acc, r_fin})
        if (overlap(out, r_ns) || overlap(out, r_al) || overlap(out, r_st) || overlap(out, r_pr))
            return fail(DV_ERR_ALIAS, "%s: an output overlaps an input", name);
    return hip_status(dv::launch_spec_walk(next_state, allow, num_states, num_tokens, states, proposals,
                                           num_proposed, num_proposed ? ld_proposals : 0, batch, accepted,
                                           final_state, static_cast<hipStream_t>(stream)),
                      "dv_spec_walk launch");
}

size_t dv_spec_verify_workspace_bytes(int32_t batch, int32_t num_proposed, int32_t num_tokens)
{
    if (batch < 0 || batch > DV_MAX_BATCH || num_proposed < 0 || num_proposed > DV_MAX_PROPOSED ||
        (int64_t)batch * (num_proposed + 1) > DV_MAX_BATCH || num_tokens < 1 || num_tokens > DV_MAX_TOKENS)
        return 0;
    return dv::spec_workspace_bytes(batch, num_proposed, num_tokens);
}

dv_status dv_spec_verify(const int32_t *next_state, const uint32_t *allow, int32_t num_states,
                         int32_t num_tokens, const int32_t *states, const int32_t *proposals,
                         int32_t num_proposed, int64_t ld_proposals, const void *logits, int32_t dtype,
                         int64_t ld_row, int64_t ld_pos, int32_t batch, int32_t *token, int32_t *accepted,
                         int32_t *new_state, void *workspace, size_t workspace_bytes, void *stream)
{
    g_error[0] = '\0';
    const char *name = "dv_spec_verify";
    if (!next_state || !allow)
        return fail(DV_ERR_INVALID_ARG, "%s: next_state and allow must be non-NULL", name);
    if (batch > 0 && (!states || !logits || !token || !accepted || !new_state || (num_proposed > 0 && !proposals)))
        return fail(DV_ERR_INVALID_ARG, "%s: states, proposals, logits, token, accepted and new_state must be "
                                        "non-NULL when batch > 0", name);
    dv_status st = spec_shape_checks(name, num_states, num_tokens, batch, num_proposed, ld_proposals);
    if (st != DV_OK)
        return st;
    const int64_t kMaxStride = (int64_t)1 << 40;
    if (ld_row < 0 || ld_row > kMaxStride || ld_pos < 0 || ld_pos > kMaxStride)
        return fail(DV_ERR_SHAPE, "%s: ld_row=%lld and ld_pos=%lld must be in [0, 2^40]", name,
                    (long long)ld_row, (long long)ld_pos);
    if (dtype != DV_F32 && dtype != DV_BF16)
        return fail(DV_ERR_DTYPE, "%s: unknown dtype %d", name, dtype);
    if (batch == 0)
        return DV_OK;
    const size_t S = (size_t)num_states, V = (size_t)num_tokens, W = (V + 31) / 32, B = (size_t)batch;
    const size_t np = (size_t)num_proposed, P = np + 1;
    const size_t elt = dtype == DV_F32 ? 4 : 2;
    if (reinterpret_cast<uintptr_t>(logits) % elt)
        return fail(DV_ERR_INVALID_ARG, "%s: logits must be aligned to their element size (%zu bytes)", name, elt);
    const Range r_tok = range_of(token, B * P * 4), r_acc = range_of(accepted, B * 4),
                r_new = range_of(new_state, B * 4);
    const Range r_ns = range_of(next_state, S * V * 4), r_al = range_of(allow, S * W * 4);
    const Range r_st = range_of(states, B * 4);
    const Range r_pr = range_of(proposals, np ? ((B - 1) * (size_t)ld_proposals + np) * 4 : 0);
    const Range r_lg = range_of(logits, ((B - 1) * (size_t)ld_row + np * (size_t)ld_pos + V) * elt);
    if (overlap(r_tok, r_acc) || overlap(r_tok, r_new) || overlap(r_acc, r_new))
        return fail(DV_ERR_ALIAS, "%s: token, accepted and new_state overlap", name);
    for (Range out : {r_tok, r_acc, r_new})
        if (overlap(out, r_ns) || overlap(out, r_al) || overlap(out, r_st) || overlap(out, r_pr) ||
            overlap(out, r_lg))
            return fail(DV_ERR_ALIAS, "%s: an output overlaps an input", name);
    const size_t need = dv::spec_workspace_bytes(batch, num_proposed, num_tokens);
    if (!workspace || workspace_bytes < need)
        return fail(DV_ERR_WORKSPACE, "%s: workspace of %zu bytes given, %zu needed", name, workspace_bytes, need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(DV_ERR_WORKSPACE, "%s: workspace must be 256-byte aligned", name);
    const Range r_ws = range_of(workspace, need);
    for (Range r : {r_tok, r_acc, r_new, r_ns, r_al, r_st, r_pr, r_lg})
        if (overlap(r_ws, r))
            return fail(DV_ERR_ALIAS, "%s: workspace overlaps an input or output", name);
    return hip_status(dv::launch_spec_verify(next_state, allow, num_states, num_tokens, states, proposals,
                                             num_proposed, num_proposed ? ld_proposals : 0, logits, dtype, ld_row,
                                             ld_pos, batch, token, accepted, new_state, workspace,
                                             static_cast<hipStream_t>(stream)),
                      "dv_spec_verify launch");
}

}  // extern "C"
