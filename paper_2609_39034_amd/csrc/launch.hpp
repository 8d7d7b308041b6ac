// Internal launch interface between the C-ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace swila {

// Pointers and sizes of one forward or decode call (decode uses T = 1).
struct LayerArgs {
    const void *q, *k, *v, *lb, *lk, *lq;  // inputs, fp32 or bf16 (in_bf16)
    const float *state_in;                 // nullptr = zeros
    float *state_out;                      // nullptr = not written
    void *o;                               // fp32 or bf16 (out_bf16)
    float *resp;                           // nullptr = not written
    int B, H, T, Dk, Dv, J;
    bool in_bf16, out_bf16;
    // Temporal SwiLA (App. B.3): gate logits [B,T,H,Dv] (in_bf16 like the other
    // inputs; both set, or neither for the plain form) and the prior state
    // [B,H,2,J,Dv] fp32 (part 0: r_{t-1}, part 1: rhobar_{t-1}; nullptr = 1/J).
    const void *gk = nullptr, *gq = nullptr;
    const float *prior_in = nullptr;
    float *prior_out = nullptr;
    // Gated SwiLA (App. B.4, eq. pre-decay): decay logits [B,T,H,J,Dk] (in_bf16),
    // a = sigmoid, one gate per key dimension and component; nullptr = no decay.
    const void *decay = nullptr;
    // Backward support (token-by-token scan in its AX mode, or the chunk scan in
    // exact mode): delta_{tjd} per token ([B,T,H,J,Dv] fp32; the chunk scan then
    // writes no responsibilities, and o may be nullptr) and the state before every
    // kBwdChunk-th token ([B,H,NCH,Dv,J,Dk] fp32, NCH = ceil(T / kBwdChunk));
    // nullptr = not written.
    float *delta_out = nullptr;
    float *ckpt = nullptr;
};

// Tokens per checkpoint interval of the backward pass.
constexpr int kBwdChunk = 32;

// Largest J * Dk of the gated token-by-token scan (its per-round gate tile in
// LDS is [16 tokens][J][Dk] fp32).
constexpr int kMaxGatedJDk = 1024;

// Largest J of the matrix-core chunk scan (all J components of at least 8
// output dims in one 64-lane sequential wave).
constexpr int kMaxChunkJ = 8;

// Pointers and sizes of one backward call: the forward's inputs (f.o, f.resp,
// f.state_out unused), the loss gradients of its outputs, the input gradients
// (fp32) and the workspace.
struct BackwardArgs {
    LayerArgs f;
    const void *grad_o;          // [B,T,H,Dv], bf16 when f.out_bf16
    const float *grad_state;     // [B,H,J,Dk,Dv]; nullptr = zeros
    float *dq, *dk, *dv;         // [B,T,H,Dk], [B,T,H,Dk], [B,T,H,Dv]
    float *dlb, *dlk, *dlq;      // [B,T,H,J,Dv]
    float *dstate;               // [B,H,J,Dk,Dv]; nullptr = not written
    float *delta;                // workspace, [B,T,H,J,Dv]: the recomputed errors
    // workspace: the chunk pass's per-(token, column) operands, written by the
    // reverse scan in the pass's tile order, [B,H,NCH,Dv/DT,kBwdChunk,DT,J] with
    // DT output dims per tile: c = beta r delta, dpred and pi^q; and dL/do as
    // [B,H,NCH,Dv/DT,kBwdChunk,DT] fp32
    float *cpk, *ppk, *qpk, *dopk;
    float *wck, *eck;            // workspace, [B,H,NCH,Dv,J,Dk] each
};

// Parameters of the chunkwise quasi-Newton form (App. D).
struct NewtonArgs {
    float *pred;        // workspace: predictions of the current iterate, per block
    int *iters;         // nullptr, or 2 ints: most sweeps of any block, blocks not converged
    int max_iters;      // sweeps at most (>= 1)
    float tol;          // stop when the change is <= tol * max(1, |pred|); < 0: max_iters sweeps
    bool clamp;         // clamp g to [0, 2 / |k_t|^2]
    bool unnorm;        // App. D.2 variant: responsibilities without their normaliser
};

// Token-by-token scan with fp32 state in registers.  Returns the HIP status of
// the launch; hipErrorInvalidValue if the shape has no instantiation.
hipError_t launch_scan_direct(const LayerArgs &a, hipStream_t stream);

// Exact chunk scan on the matrix cores, pipelined (one sequential wave plus
// matrix-core waves); bf16 inputs, T > 0.  With gate logits (a.gk) it runs the
// temporal form.
hipError_t launch_scan_pipe(const LayerArgs &a, hipStream_t stream);
// Gated SwiLA (App. B.4) in chunks of 16 tokens on the matrix cores: bf16
// inputs, no temporal priors, J <= 4, J * Dk <= 256 (gated_chunk_supported).
bool gated_chunk_supported(const LayerArgs &a);
hipError_t launch_scan_gated_chunk(const LayerArgs &a, hipStream_t stream);
hipError_t launch_scan_pipe_temporal(const LayerArgs &a, hipStream_t stream);

// Chunkwise quasi-Newton evaluation (App. D) on the same pipelined kernel;
// bf16 inputs, T > 0, resp must be nullptr.  na.pred holds
// newton_workspace_bytes(...) bytes.
hipError_t launch_newton(const LayerArgs &a, const NewtonArgs &na, hipStream_t stream);
size_t newton_workspace_bytes(int B, int H, int T, int Dv, int J);

// Token-by-token forward that writes a.delta_out and a.ckpt (both required)
// and no output or final state: the first step of the backward pass.
hipError_t launch_scan_direct_aux(const LayerArgs &a, hipStream_t stream);

// Backward pass of the plain forward (every pointer of b set except
// b.grad_state and b.dstate, which may be nullptr; T > 0).
hipError_t launch_backward(const BackwardArgs &b, hipStream_t stream);
size_t backward_workspace_bytes(int B, int H, int T, int Dk, int Dv, int J);

// One-token decode step streaming the state through registers.
hipError_t launch_decode(const LayerArgs &a, hipStream_t stream);

// state <- src (or zeros when src is nullptr); n floats.
hipError_t launch_state_fill(float *state, const float *src, size_t n, hipStream_t stream);

// dst <- src (or the constant value when src is nullptr); n floats.
hipError_t launch_fill(float *dst, const float *src, size_t n, float value, hipStream_t stream);

}  // namespace swila
