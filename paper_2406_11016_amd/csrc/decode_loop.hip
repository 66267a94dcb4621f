// A decoding loop around the fused verification step: one call per
// iteration replays the step for the iteration's number of drafts from a
// HIP graph captured once per gamma (the verification followed by the copy of
// the accepted lengths and next tokens to pinned host memory), waits for it,
// and returns the next gamma by the draft-length rule of the paper's
// experiments (Sec. 4, hyperparameters: gamma starts at 5, grows by 2 after
// an iteration that accepts every draft, otherwise shrinks by 1; here kept
// within 1 .. gamma_max, and with several batch elements every element must
// accept every draft to grow).
//
// In the exact mode each step runs either the single pass or the early exit
// (Sec. 3.1 stops at the first rejection): as the descriptor says, or chosen
// from the previous step's acceptance (early_exit_pays).
//
// Host code only: the device work is the library's verification kernel and
// three copies.  All device and pinned buffers belong to the caller; the loop
// object holds the descriptor, one pinned word for the workspace's error flag
// and the instantiated graphs.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <new>
#include <vector>

#include "plan.hpp"
#include "spec_verify.h"

struct sv_loop {
    sv_loop_desc_t d;
    uint32_t* flag = nullptr;          // pinned: the workspace's sticky error flag (from the first step on)
    std::vector<hipGraphExec_t> exec;  // by 2 gamma + early exit (0, 1 unused); null until first use
    bool early = false;                // the next step's choice (exact mode)
    int32_t last_early = -1;           // the last step's choice
};

// Byte offset of the sticky error flag in the workspace header.
constexpr size_t kErrorFlagOffset = 4;

namespace {

// The verification of the leading [B, gamma, V] parts of the static buffers
// and the copy of its outputs to host_out and of the workspace's error flag,
// enqueued on the loop's stream.
sv_status_t enqueue(const sv_loop_desc_t& d, uint32_t* flag, int32_t gamma, bool early) {
    sv_status_t st;
    if (d.mode == 0 && early)
        st = spec_verify_exact_early_exit(d.draft, d.target, d.dtype, d.tokens, d.uniforms, d.batch, gamma, d.vocab,
                                          d.temperature, d.accepted_len, d.next_token, d.workspace,
                                          d.workspace_bytes, d.stream);
    else if (d.mode == 0)
        st = spec_verify_exact(d.draft, d.target, d.dtype, d.tokens, d.uniforms, d.batch, gamma, d.vocab,
                               d.temperature, d.accepted_len, d.next_token, d.workspace, d.workspace_bytes,
                               d.stream);
    else
        st = spec_verify_sigmoid(d.draft, d.target, d.dtype, d.tokens, d.uniforms, d.batch, gamma, d.vocab,
                                 d.temperature, d.alpha, d.beta, d.accepted_len, d.next_token, d.workspace,
                                 d.workspace_bytes, d.stream);
    if (st != SV_OK) return st;
    const size_t n = sizeof(int32_t) * (size_t)d.batch;
    if (hipMemcpyAsync(d.host_out, d.accepted_len, n, hipMemcpyDeviceToHost, d.stream) != hipSuccess ||
        hipMemcpyAsync(d.host_out + d.batch, d.next_token, n, hipMemcpyDeviceToHost, d.stream) != hipSuccess ||
        hipMemcpyAsync(flag, static_cast<const char*>(d.workspace) + kErrorFlagOffset, sizeof(uint32_t),
                       hipMemcpyDeviceToHost, d.stream) != hipSuccess)
        return SV_ERR_HIP;
    return SV_OK;
}

sv_status_t capture(sv_loop* loop, int32_t gamma, bool early) {
    const sv_loop_desc_t& d = loop->d;
    if (hipStreamBeginCapture(d.stream, hipStreamCaptureModeThreadLocal) != hipSuccess) return SV_ERR_HIP;
    const sv_status_t st = enqueue(d, loop->flag, gamma, early);
    hipGraph_t graph = nullptr;
    const hipError_t end = hipStreamEndCapture(d.stream, &graph);
    if (st != SV_OK || end != hipSuccess || graph == nullptr) {
        if (graph != nullptr) (void)hipGraphDestroy(graph);
        return st != SV_OK ? st : SV_ERR_HIP;
    }
    hipGraphExec_t exec = nullptr;
    const hipError_t inst = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (inst != hipSuccess) return SV_ERR_HIP;
    loop->exec[2 * gamma + (early ? 1 : 0)] = exec;
    return SV_OK;
}

}  // namespace

extern "C" {

sv_status_t spec_verify_loop_create(const sv_loop_desc_t* desc, sv_loop** out) {
    if (desc == nullptr || out == nullptr) return SV_ERR_NULL;
    *out = nullptr;
    const sv_loop_desc_t& d = *desc;
    if (d.draft == nullptr || d.target == nullptr || d.tokens == nullptr || d.uniforms == nullptr ||
        d.accepted_len == nullptr || d.next_token == nullptr || d.host_out == nullptr || d.workspace == nullptr)
        return SV_ERR_NULL;
    if ((d.mode != 0 && d.mode != 1) || d.early_exit < 0 || d.early_exit > 2) return SV_ERR_PARAM;
    if (d.batch < 1 || d.gamma_max < 1 || d.vocab < 1) return SV_ERR_SHAPE;
    for (int32_t g = 1; g <= d.gamma_max; ++g) {
        const size_t need = spec_verify_workspace_bytes(d.batch, g, d.vocab, d.dtype);
        if (need == 0) return SV_ERR_SHAPE;
        if (d.workspace_bytes < need) return SV_ERR_WORKSPACE;
    }
    sv_loop* loop = new (std::nothrow) sv_loop;
    if (loop == nullptr) return SV_ERR_ALLOC;
    loop->d = d;
    loop->exec.assign(2 * ((size_t)d.gamma_max + 1), nullptr);
    loop->early = d.mode == 0 && d.early_exit == 1;
    *out = loop;
    return SV_OK;
}

sv_status_t spec_verify_loop_step(sv_loop* loop, int32_t gamma, int32_t* next_gamma) {
    if (loop == nullptr || next_gamma == nullptr) return SV_ERR_NULL;
    const sv_loop_desc_t& d = loop->d;
    if (gamma < 1 || gamma > d.gamma_max) return SV_ERR_PARAM;
    if (loop->flag == nullptr) {
        // the pinned word the flag is copied to, allocated once (a step needs
        // the GPU anyway; creating the loop does not)
        void* flag = nullptr;
        if (hipHostMalloc(&flag, sizeof(uint32_t), hipHostMallocDefault) != hipSuccess || flag == nullptr)
            return SV_ERR_HIP;
        loop->flag = static_cast<uint32_t*>(flag);
    }
    *loop->flag = 0;
    const bool early = loop->early;
    if (d.use_graphs) {
        hipGraphExec_t& e = loop->exec[2 * gamma + (early ? 1 : 0)];
        if (e == nullptr) {
            const sv_status_t st = capture(loop, gamma, early);
            if (st != SV_OK) return st;
        }
        if (hipGraphLaunch(e, d.stream) != hipSuccess) return SV_ERR_HIP;
    } else {
        const sv_status_t st = enqueue(d, loop->flag, gamma, early);
        if (st != SV_OK) return st;
    }
    loop->last_early = (d.mode == 0 && early) ? 1 : 0;
    if (hipStreamSynchronize(d.stream) != hipSuccess) return SV_ERR_HIP;
    if (*loop->flag != 0) return SV_ERR_TIMEOUT;
    bool all = true;
    long long accepted = 0;
    for (int32_t b = 0; b < d.batch; ++b) {
        all = all && d.host_out[b] == gamma;
        accepted += (d.host_out[b] > 0) ? d.host_out[b] : 0;
    }
    if (d.mode == 0 && d.early_exit == 2) loop->early = sv::early_exit_pays(accepted, d.batch, gamma);
    *next_gamma = all ? (gamma + 2 < d.gamma_max ? gamma + 2 : d.gamma_max) : (gamma > 1 ? gamma - 1 : 1);
    return SV_OK;
}

int32_t spec_verify_loop_last_early_exit(const sv_loop* loop) { return loop == nullptr ? -1 : loop->last_early; }

sv_status_t spec_verify_loop_destroy(sv_loop* loop) {
    if (loop == nullptr) return SV_OK;
    sv_status_t st = SV_OK;
    for (hipGraphExec_t e : loop->exec)
        if (e != nullptr && hipGraphExecDestroy(e) != hipSuccess) st = SV_ERR_HIP;
    if (loop->flag != nullptr && hipHostFree(loop->flag) != hipSuccess) st = SV_ERR_HIP;
    delete loop;
    return st;
}

}  // extern "C"
