/*
 * swila.h -- C ABI of libswila.so, the MI355X (gfx950) hot path of Switching
 * Linear Attention (SwiLA).
 *
 * What is computed (per batch b, head h, token t, output dimension d and
 * mixture component j; Sec. 3.2 of the paper, with beta and the priors
 * produced from logits as App. B.2 states):
 *
 *   beta_{tjd}   = sigmoid(beta_logit_{tjd})
 *   pi^k_{tjd}   = softmax over j of prior_k_logit_{t.d}
 *   pi^q_{tjd}   = softmax over j of prior_q_logit_{t.d}
 *   delta_{tjd}  = v_{td} - w_{t-1,jd} . k_t                     (prediction error)
 *   r_{tjd}      = pi^k_{tjd} exp(-delta^2/2) / sum_j' (same)   (eq. responsibility)
 *   w_{tjd}      = w_{t-1,jd} + beta_{tjd} r_{tjd} delta_{tjd} k_t (eq. recurrence)
 *   o_{td}       = sum_j pi^q_{tjd} w_{tjd} . q_t              (eq. retrieval, updated state)
 *
 * The op applies no scaling, normalisation or activation to q, k or v: the
 * caller supplies them as the layer produces them (the paper L2-normalises
 * the keys, App. E).
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer, owned by the caller; the library
 *     allocates no device memory and keeps no pointer after the call returns.
 *   - Tensors are dense, row-major and 16-byte aligned:
 *       q, k                 [B, T, H, Dk]      (decode: [B, H, Dk])
 *       v, o                 [B, T, H, Dv]      (decode: [B, H, Dv])
 *       beta_logit, prior_k_logit, prior_q_logit, resp
 *                            [B, T, H, J, Dv]   (decode: [B, H, J, Dv])
 *       state                [B, H, J, Dk, Dv]  fp32; element (b,h,j,i,d) is key
 *                            weight i of component j for output dimension d,
 *                            i.e. (W_j)_{d,i} in the paper's notation (App. B.4)
 *   - q, k, v and the logits share one dtype (opts->in_dtype); o has
 *     opts->out_dtype; the state, the scalar recurrence and every accumulation
 *     are fp32 (the matrix-core forms multiply fp32 operands as a bf16 high part
 *     and a bf16 residual, see swila_algo).  bf16 values are widened exactly; o
 *     is rounded to nearest-even when it is bf16.
 *   - stream is a hipStream_t (NULL = the null stream).  Work is enqueued and
 *     the call returns; device faults surface at the caller's next sync.
 *   - Return value: SWILA_OK, or a negative status.  Argument errors are found
 *     before anything is enqueued.  swila_last_error() then describes the
 *     failure (thread-local text, valid until this thread's next call).
 *   - Supported shapes: Dk in {16, 32, 64, 128}, Dv in {16, 32, 64, 128},
 *     J in {1, 2, 3, 4, 8, 16} (every J of the paper's Sec. 5.1 sweep, and 3),
 *     1 <= B, H <= 65535 with B * H <= 2^26, T >= 0.  Others give
 *     SWILA_EUNSUPPORTED.  Narrower limits:
 *     the chunked forms (SWILA_ALGO_CHUNK_EXACT, SWILA_ALGO_NEWTON) and the
 *     backward pass take J <= 8 (SWILA_ALGO_AUTO then picks the token-by-token
 *     scan), and the gated forward takes J * Dk <= 1024 (its chunked form
 *     J <= 4 and J * Dk <= 512; see swila_forward_gated).
 */
#ifndef SWILA_H
#define SWILA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct swila_shape {
    int32_t B, H, T, Dk, Dv, J;   /* J: number of mixture components */
} swila_shape;

enum swila_dtype { SWILA_F32 = 0, SWILA_BF16 = 1 };

enum swila_algo {
    SWILA_ALGO_AUTO = 0,        /* CHUNK_EXACT for bf16 inputs with J <= 8, else RECURRENT */
    SWILA_ALGO_RECURRENT = 1,   /* token-by-token scan on the vector ALUs */
    SWILA_ALGO_CHUNK_EXACT = 2, /* the same recurrence evaluated 16 tokens at a time with
                                   the Dk-long products on the matrix cores (bf16 inputs
                                   only; fp32 operands split into bf16 high + residual) */
    SWILA_ALGO_NEWTON = 3       /* App. D: chunkwise parallel quasi-Newton iteration.  Each
                                   sweep linearises the recurrence around the previous
                                   sweep's predictions k_t . w_{t-1} (eq. jacobian_coeff,
                                   eq. effective_input) and solves the linear recurrence
                                   (eq. linearized) chunk by chunk (App. D.3), on the matrix
                                   cores like CHUNK_EXACT.  The first sweep linearises
                                   around w_t = W_0 for all t.  bf16 inputs only; needs a
                                   workspace; resp_out must be NULL. */
};

/* opts->flags bits */
enum swila_flags {
    SWILA_FLAG_NEWTON_NO_CLAMP = 1, /* SWILA_ALGO_NEWTON: use g of eq. jacobian_coeff as it
                                       is.  By default g is clamped to [0, 2 / |k_t|^2], which
                                       keeps every linearised transition I - g k k^T
                                       non-expansive; the fixed point does not depend on the
                                       Jacobian approximation (App. D.2). */
    SWILA_FLAG_NEWTON_SYNC = 2,     /* SWILA_ALGO_NEWTON, for callers that want a status:
                                       swila_forward waits for the stream after the launch,
                                       reads iters_out (then required) and returns
                                       SWILA_ENOTCONVERGED if some block of columns stopped
                                       at max_iters without meeting tol.  Its outputs are
                                       written either way.  Without the flag the call only
                                       enqueues, and iters_out is the report. */
    SWILA_FLAG_UNNORMALIZED = 4     /* SWILA_ALGO_NEWTON only (other algorithms and entry
                                       points return SWILA_EUNSUPPORTED): evaluate App. D.2's
                                       variant of the recurrence whose responsibilities drop
                                       the denominator of eq. responsibility,
                                       r = pi^k exp(-delta^2/2).  Its Jacobian is exact,
                                       g = beta r (1 - delta^2), so the sweeps are Newton's
                                       method proper.  It is a different recurrence: the
                                       outputs are those of the variant. */
};

typedef struct swila_opts {
    int32_t in_dtype;    /* enum swila_dtype of q, k, v and the three logits */
    int32_t out_dtype;   /* enum swila_dtype of o */
    int32_t algo;        /* enum swila_algo */
    int32_t chunk;       /* chunk length of the chunked forms: 0 (default) or 16 */
    int32_t max_iters;   /* SWILA_ALGO_NEWTON: most sweeps; 0 = 64.  Ignored otherwise. */
    float tol;           /* SWILA_ALGO_NEWTON: a block of columns stops once the largest
                            change of its predictions in a sweep is <= tol * max(1, largest
                            |prediction|); 0 = 1e-3; < 0 = run exactly max_iters sweeps.
                            Ignored otherwise.  NaN is an error. */
    uint32_t flags;      /* enum swila_flags; other bits must be 0 */
} swila_opts;

enum swila_status {
    SWILA_OK = 0,
    SWILA_EINVAL = -1,        /* null or misaligned pointer, bad size or dtype */
    SWILA_EUNSUPPORTED = -2,  /* valid but outside the supported set */
    SWILA_EHIP = -3,          /* the HIP runtime reported an error */
    SWILA_ENOTCONVERGED = -4  /* SWILA_ALGO_NEWTON with SWILA_FLAG_NEWTON_SYNC: some block of
                                 columns did not meet tol within max_iters sweeps */
};

/* Library ABI version (currently 1). */
int swila_version(void);

/* Bytes of one state tensor: B*H*J*Dk*Dv*4.  0 if shape is NULL or invalid. */
size_t swila_state_bytes(const swila_shape *shape);

/*
 * Initial state W_0 (Sec. 3.2: the recurrence starts from a given state).
 * Writes state [B,H,J,Dk,Dv] fp32 with a copy of src (same layout, device),
 * or zeros when src is NULL.  src may equal state (no-op).  T is ignored.
 */
int swila_state_init(const swila_shape *shape, float *state, const float *src, void *stream);

/*
 * Forward over a whole sequence (Sec. 3.2: eq. recurrence, eq. responsibility,
 * eq. retrieval; App. B.2 for the logits).  Runs all T tokens of every (b, h).
 *   q, k, v, beta_logit, prior_k_logit, prior_q_logit: inputs, in_dtype.
 *   state_in:  W_0 [B,H,J,Dk,Dv] fp32, or NULL for zeros.
 *   state_out: W_T, or NULL to discard it; may equal state_in (updated in place).
 *   o:         output [B,T,H,Dv], out_dtype.  Must not overlap any input.
 *   resp_out:  NULL, or [B,T,H,J,Dv] fp32 receiving the key-side
 *              responsibilities r_{tjd} (for routing diagnostics).
 *   workspace, ws_bytes: device scratch for forms that need it, at least
 *              swila_forward_workspace_bytes bytes, 16-byte aligned, disjoint
 *              from every tensor argument (SWILA_ALGO_NEWTON: the predictions
 *              of the current iterate, overwritten).  Other forms ignore both.
 *   iters_out: NULL, or a device int32[2] (SWILA_ALGO_NEWTON only; ignored
 *              otherwise): [0] = the most sweeps any block of columns ran,
 *              [1] = how many blocks stopped at max_iters without meeting tol
 *              (0 when tol < 0).  Columns of different output dimensions are
 *              independent, so each block of them stops on its own test; the
 *              outputs and W_T are those of each block's last sweep.
 * T == 0 copies state_in (or zeros) to state_out and writes nothing else.
 */
int swila_forward(const swila_shape *shape, const swila_opts *opts,
                  const void *q, const void *k, const void *v,
                  const void *beta_logit, const void *prior_k_logit,
                  const void *prior_q_logit,
                  const float *state_in, float *state_out, void *o, float *resp_out,
                  void *workspace, size_t ws_bytes, int32_t *iters_out, void *stream);

/* Workspace bytes swila_forward needs for these options (0 if none):
 * SWILA_ALGO_NEWTON needs B*H*J*Dv*(16*ceil(T/16))*4. */
size_t swila_forward_workspace_bytes(const swila_shape *shape, const swila_opts *opts);

/*
 * One decode step: the recurrence and retrieval for a single new token per
 * sequence (shape->T must be 1), streaming the state from state_in to
 * state_out.  q, k [B,H,Dk]; v [B,H,Dv]; logits [B,H,J,Dv]; o [B,H,Dv].
 * state_in NULL means a zero state.  state_out may equal state_in (in
 * place); otherwise they must not overlap; NULL discards the new state.
 * The same token's result equals swila_forward with T = 1.
 */
int swila_decode_step(const swila_shape *shape, const swila_opts *opts,
                      const void *q, const void *k, const void *v,
                      const void *beta_logit, const void *prior_k_logit,
                      const void *prior_q_logit,
                      const float *state_in, float *state_out, void *o, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): swila_forward without
 * the workspace arguments.  The arguments, results and errors are those of
 * swila_forward; the forms that need scratch (SWILA_ALGO_NEWTON: the
 * predictions of the current iterate) use a device array of
 * SWILA_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on
 * until the process ends, so the call allocates nothing.
 *   - Limit: B*H*J*Dv*16*ceil(T/16)*4 <= SWILA_NOALLOC_SCRATCH_BYTES (64 MiB, e.g.
 *     B=4 H=8 T=2048 Dv=64 J=4) for SWILA_ALGO_NEWTON; larger calls return
 *     SWILA_EUNSUPPORTED before anything is enqueued.  Other forms need none.
 *   - The stream must belong to the current device (hipGetDevice).  The first
 *     call on a device looks up that device's copy of the array.
 *   - Every call on a GPU shares that GPU's array, which keeps the last call's
 *     contents (nothing in it needs to start at zero): calls that overlap on one
 *     GPU, on different streams or threads, race.
 */
#define SWILA_NOALLOC_SCRATCH_BYTES (64u << 20)
int swila_forward_noalloc(const swila_shape *shape, const swila_opts *opts,
                          const void *q, const void *k, const void *v,
                          const void *beta_logit, const void *prior_k_logit,
                          const void *prior_q_logit,
                          const float *state_in, float *state_out, void *o, float *resp_out,
                          int32_t *iters_out, void *stream);

/*
 * Temporal SwiLA (Sec. 3.3, App. B.3): the two priors become running mixtures
 * over time, per (b, h, j, d),
 *
 *   g^k_{td}     = sigmoid(gate_k_logit_{td}),  g^q_{td} = sigmoid(gate_q_logit_{td})
 *   rbar_{tjd}   = (1 - g^k_{td}) r_{t-1,jd}      + g^k_{td} pi^k_{tjd}
 *   rhobar_{tjd} = (1 - g^q_{td}) rhobar_{t-1,jd} + g^q_{td} pi^q_{tjd}
 *
 * rbar replaces pi^k in eq. responsibility and rhobar replaces pi^q in
 * eq. retrieval.  The key side mixes in the previous token's responsibilities
 * r_{t-1} (the filtered posterior), the query side its own previous prior.
 *   gate_k_logit, gate_q_logit: [B,T,H,Dv] (decode: [B,H,Dv]), in_dtype, 16-byte
 *              aligned; required when T > 0.
 *   prior_in:  the prior state [B,H,2,J,Dv] fp32 carried from a previous call
 *              (part 0: r_{t-1}, part 1: rhobar_{t-1}), or NULL for the uniform
 *              1/J (the paper gives no initial value).
 *   prior_out: NULL, or the prior state after the last token; may equal
 *              prior_in (updated in place), otherwise disjoint from everything.
 * The gate tensors and prior_in must not overlap any output.
 */
typedef struct swila_temporal {
    const void *gate_k_logit;
    const void *gate_q_logit;
    const float *prior_in;
    float *prior_out;
} swila_temporal;

/*
 * swila_forward with the temporal priors above.  The other arguments are those
 * of swila_forward (no workspace: SWILA_ALGO_NEWTON, whose linearisation is
 * that of the plain recurrence, returns SWILA_EUNSUPPORTED).  SWILA_ALGO_AUTO
 * picks the matrix-core chunk scan for bf16 inputs and the token-by-token scan
 * for fp32, as swila_forward does.  T == 0 copies state_in and prior_in (or
 * zeros and 1/J) to the outputs.
 */
int swila_forward_temporal(const swila_shape *shape, const swila_opts *opts,
                           const void *q, const void *k, const void *v,
                           const void *beta_logit, const void *prior_k_logit,
                           const void *prior_q_logit, const swila_temporal *temporal,
                           const float *state_in, float *state_out, void *o,
                           float *resp_out, void *stream);

/* swila_decode_step with the temporal priors (gate logits [B,H,Dv]); its
 * result equals swila_forward_temporal with T = 1. */
int swila_decode_step_temporal(const swila_shape *shape, const swila_opts *opts,
                               const void *q, const void *k, const void *v,
                               const void *beta_logit, const void *prior_k_logit,
                               const void *prior_q_logit, const swila_temporal *temporal,
                               const float *state_in, float *state_out, void *o,
                               void *stream);

/*
 * Gated SwiLA (Sec. 3.4, App. B.4), in the form of eq. pre-decay with one
 * gate per key dimension (tied across output dims, as in the paper's language
 * models): before the prediction of token t the state decays,
 *
 *   a_{tj}      = sigmoid(decay_logit_{tj})          in (0, 1)^Dk
 *   wbar_{jd}   = a_{tj} (.) w_{t-1,jd}              (elementwise over key index i)
 *   delta_{tjd} = v_{td} - wbar_{jd} . k_t,  r from these errors (eq. responsibility)
 *   w_{tjd}     = wbar_{jd} + beta r delta k_t
 *
 *   decay_logit: [B,T,H,J,Dk] (decode: [B,H,J,Dk]), in_dtype, 16-byte aligned;
 *                required when T > 0; must not overlap any output.
 */
typedef struct swila_gated {
    const void *decay_logit;
} swila_gated;

/*
 * swila_forward with the gated decay above; temporal may be NULL (plain
 * priors) or the temporal priors of swila_forward_temporal (Gated Temporal
 * SwiLA).  Algorithms:
 *   SWILA_ALGO_CHUNK_EXACT: the same recurrence 16 tokens at a time on the
 *     matrix cores (App. B.4 with the chunk algebra of the plain form; exact
 *     up to rounding order).  It takes bf16 inputs, no temporal priors,
 *     J <= 4 and J * Dk <= 512; other calls return SWILA_EUNSUPPORTED.
 *   SWILA_ALGO_RECURRENT: the token-by-token scan (either input dtype, with
 *     or without temporal priors, J * Dk <= 1024).
 *   SWILA_ALGO_AUTO: CHUNK_EXACT where it applies, else RECURRENT.
 *   SWILA_ALGO_NEWTON returns SWILA_EUNSUPPORTED.
 * T == 0 copies the states.
 */
int swila_forward_gated(const swila_shape *shape, const swila_opts *opts,
                        const void *q, const void *k, const void *v,
                        const void *beta_logit, const void *prior_k_logit,
                        const void *prior_q_logit, const swila_gated *gated,
                        const swila_temporal *temporal, const float *state_in,
                        float *state_out, void *o, float *resp_out, void *stream);

/* swila_decode_step with the gated decay (decay logits [B,H,J,Dk]); temporal
 * may be NULL.  Its result equals swila_forward_gated with T = 1. */
int swila_decode_step_gated(const swila_shape *shape, const swila_opts *opts,
                            const void *q, const void *k, const void *v,
                            const void *beta_logit, const void *prior_k_logit,
                            const void *prior_q_logit, const swila_gated *gated,
                            const swila_temporal *temporal, const float *state_in,
                            float *state_out, void *o, void *stream);

/*
 * Backward pass of swila_forward (plain form; Sec. 3.2: eq. recurrence,
 * eq. responsibility, eq. retrieval, with the logits of App. B.2): the exact
 * gradient of a scalar loss L through the forward, for training.  The paper
 * trains through the sequential evaluation and gives no backward formulas;
 * this is the chain rule of that forward, evaluated with fp32 values and
 * accumulation (with bf16 inputs the reverse scan's Dk-long products take fp32
 * operands as a bf16 high part and residual on the matrix cores; the final
 * pass multiplies in fp32 on the matrix cores).
 *   q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in: the forward's
 *              inputs, as in swila_forward (state_in NULL = zeros).
 *   grad_o:    dL/do [B,T,H,Dv], out_dtype; required when T > 0.
 *   grad_state_out: dL/dW_T [B,H,J,Dk,Dv] fp32, or NULL for zeros.
 *   grad_q, grad_k: [B,T,H,Dk] fp32;  grad_v: [B,T,H,Dv] fp32;
 *   grad_beta_logit, grad_prior_k_logit, grad_prior_q_logit: [B,T,H,J,Dv] fp32
 *              (all six required when T > 0, overwritten).
 *   grad_state_in: dL/dW_0 [B,H,J,Dk,Dv] fp32, or NULL to discard it.
 *   workspace, ws_bytes: at least swila_backward_workspace_bytes bytes,
 *              16-byte aligned; holds the recomputed errors delta, the state
 *              every 32 tokens and the per-token operands the reverse scan
 *              hands to the final pass, and is overwritten.
 * Every output, the workspace and the inputs are pairwise disjoint.  The
 * algorithm field of opts is ignored: the backward recomputes the forward
 * with the matrix-core chunk scan for bf16 inputs and the token-by-token scan
 * for fp32 inputs.  T == 0 copies grad_state_out (or zeros) to grad_state_in.
 */
int swila_backward(const swila_shape *shape, const swila_opts *opts,
                   const void *q, const void *k, const void *v,
                   const void *beta_logit, const void *prior_k_logit,
                   const void *prior_q_logit, const float *state_in,
                   const void *grad_o, const float *grad_state_out,
                   float *grad_q, float *grad_k, float *grad_v,
                   float *grad_beta_logit, float *grad_prior_k_logit,
                   float *grad_prior_q_logit, float *grad_state_in,
                   void *workspace, size_t ws_bytes, void *stream);

/* Workspace bytes swila_backward needs (0 if shape is NULL or invalid), with
 * N = ceil(T/32) and each part rounded up to a multiple of 256:
 * B*T*H*J*Dv*4 + 3*(B*H*N*32*J*Dv*4) + B*H*N*32*Dv*4 + 2*(B*H*N*J*Dk*Dv*4). */
size_t swila_backward_workspace_bytes(const swila_shape *shape);

/* Text of this thread's last error ("" if none). */
const char *swila_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SWILA_H */
