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
 *     opts->out_dtype; the state and all arithmetic are fp32.  bf16 values are
 *     widened exactly; o is rounded to nearest-even when it is bf16.
 *   - stream is a hipStream_t (NULL = the null stream).  Work is enqueued and
 *     the call returns; device faults surface at the caller's next sync.
 *   - Return value: SWILA_OK, or a negative status.  Argument errors are found
 *     before anything is enqueued.  swila_last_error() then describes the
 *     failure (thread-local text, valid until this thread's next call).
 *   - Supported shapes: Dk in {16, 32, 64, 128}, Dv in {16, 32, 64, 128},
 *     J in {1, 2, 3, 4, 8}, B, H >= 1, T >= 0.  Others give SWILA_EUNSUPPORTED.
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
    SWILA_ALGO_AUTO = 0,        /* CHUNK_EXACT for bf16 inputs, RECURRENT for fp32 */
    SWILA_ALGO_RECURRENT = 1,   /* token-by-token scan on the vector ALUs */
    SWILA_ALGO_CHUNK_EXACT = 2  /* the same recurrence evaluated 16 tokens at a time with
                                   the Dk-long products on the matrix cores (bf16 inputs
                                   only; fp32 operands split into bf16 high + residual) */
};

typedef struct swila_opts {
    int32_t in_dtype;    /* enum swila_dtype of q, k, v and the three logits */
    int32_t out_dtype;   /* enum swila_dtype of o */
    int32_t algo;        /* enum swila_algo */
    int32_t chunk;       /* chunk length of chunked forms; 0 = default */
    int32_t max_iters;   /* reserved, 0 */
    float tol;           /* reserved, 0 */
    uint32_t flags;      /* reserved, 0 */
} swila_opts;

enum swila_status {
    SWILA_OK = 0,
    SWILA_EINVAL = -1,        /* null or misaligned pointer, bad size or dtype */
    SWILA_EUNSUPPORTED = -2,  /* valid but outside the supported set */
    SWILA_EHIP = -3           /* the HIP runtime reported an error */
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
 *   workspace, ws_bytes: scratch for forms that need it; see
 *              swila_forward_workspace_bytes (0 for the recurrent scan, where
 *              both may be NULL/0).
 *   iters_out: reserved, may be NULL.
 * T == 0 copies state_in (or zeros) to state_out and writes nothing else.
 */
int swila_forward(const swila_shape *shape, const swila_opts *opts,
                  const void *q, const void *k, const void *v,
                  const void *beta_logit, const void *prior_k_logit,
                  const void *prior_q_logit,
                  const float *state_in, float *state_out, void *o, float *resp_out,
                  void *workspace, size_t ws_bytes, int32_t *iters_out, void *stream);

/* Workspace bytes swila_forward needs for these options (0 if none). */
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

/* Text of this thread's last error ("" if none). */
const char *swila_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SWILA_H */
