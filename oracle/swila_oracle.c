/*
 * SwiLA reference oracle -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, fp64 CPU implementation of the Switching Linear Attention
 * recurrence exactly as the paper states it (Sec. 3.2: eq. recurrence,
 * eq. responsibility, eq. retrieval; App. B.2 for how beta and the two
 * priors are produced from logits).  Only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or helper with the GPU library, and it never calls into it.
 *
 * Notation follows the paper.  For one head, the state is J matrices
 * W_j in R^{Dv x Dk}; row d of W_j is the regression weight w_{jd} in R^{Dk}
 * of mixture component j for output dimension d (App. B.4, "rows index
 * output dimensions and columns index key dimensions").  Per token t:
 *
 *   pi^k_{jd}  = softmax over j of the key-prior logits          (App. B.2)
 *   beta_{tjd} = sigmoid(beta logit)                              (App. B.2)
 *   delta_{tjd} = v_{td} - w_{t-1,jd}^T k_t                       (Sec. 3.2)
 *   r_{tjd} = pi^k_{jd} exp(-delta^2/2) / sum_j' (same)           (eq. responsibility)
 *             (evaluated with every exp(-delta^2/2) divided by the largest)
 *   w_{tjd} = w_{t-1,jd} + beta_{tjd} r_{tjd} delta_{tjd} k_t     (eq. recurrence)
 *   pi^q_{jd}  = softmax over j of the query-prior logits         (App. B.2)
 *   o_{td} = sum_j pi^q_{jd} w_{tjd}^T q_t   (updated state)      (eq. retrieval)
 *
 * Tensor layouts (row-major, every array is double):
 *   q, k          [B, T, H, Dk]
 *   v, o          [B, T, H, Dv]
 *   *_logit, resp [B, T, H, J, Dv]
 *   state         [B, H, J, Dk, Dv]   element (b,h,j,i,d) = (W_j)_{d,i}
 * The state layout is the storage convention of the library under test; the
 * oracle converts it to its own W[j][d][i] on entry and back on exit.
 *
 * Decode (one token with state in and out) is this same function with T = 1.
 *
 * Temporal SwiLA (Sec. 3.3, App. B.3), when gate logits are given: the two
 * priors become running mixtures over time, per (j, d),
 *
 *   g^k_{td} = sigmoid(gate_k_logit_{td}),  g^q_{td} = sigmoid(gate_q_logit_{td})
 *   rbar_{tjd}   = (1 - g^k_{td}) r_{t-1,jd}      + g^k_{td} pi^k_{tjd}
 *   rhobar_{tjd} = (1 - g^q_{td}) rhobar_{t-1,jd} + g^q_{td} pi^q_{tjd}
 *
 * and rbar replaces pi^k in the E-step, rhobar replaces pi^q in the retrieval.
 * Note the key side mixes in the previous token's responsibilities r (the
 * filtered posterior), the query side its own previous prior.  The carried
 * pair (r_{t-1}, rhobar_{t-1}) is the "prior state" [B, H, 2, J, Dv]: part 0
 * is r, part 1 is rhobar.  Without an input prior state both start uniform,
 * 1/J (the paper gives no initial value).  Gate logits are [B, T, H, Dv].
 *
 * Gated SwiLA (Sec. 3.4, App. B.4), when decay logits are given: a decay
 * a_{tj} = sigmoid(decay_logit_{tj}) in [0,1]^{Dk}, one gate per key dimension
 * and component, tied across the output dims (the form of the paper's
 * language-model runs).  Pre-decay (eq. pre-decay, the form the paper uses):
 *
 *   wbar_{jd}   = a_{tj} (.) w_{t-1,jd}                 (elementwise over i)
 *   delta_{tjd} = v_{td} - wbar_{jd} . k_t,  r from these errors
 *   w_{tjd}     = wbar_{jd} + beta r delta k_t
 *
 * Post-decay (eq. post-decay; kept here for the J = 1 equivalence the paper
 * states): delta and r from w_{t-1}, then w_{tjd} = a_{tj} (.) w_{t-1,jd} +
 * beta r delta k_t.  Decay logits are [B, T, H, J, Dk].
 *
 * Unnormalised responsibilities (App. D.2), when asked for: the variant of the
 * recurrence whose Jacobian has no cross-component terms, obtained by dropping
 * the denominator of eq. responsibility,
 *
 *   r_{tjd} = pi^k_{jd} exp(-delta_{tjd}^2 / 2),
 *
 * so that the update is beta times the gradient of the mixture likelihood
 * sum_j pi_j exp(-delta_j^2/2) itself rather than of its logarithm.  Everything
 * else (prediction, retrieval) is unchanged.  It is defined for the plain form
 * only.
 */
#include <math.h>
#include <pthread.h>
#include <stddef.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

typedef struct {
    int B, H, T, Dk, Dv, J;
    const double *q, *k, *v, *lb, *lk, *lq, *state_in;
    double *state_out, *o, *resp, *delta_out;
    const double *gk, *gq, *prior_in;   /* temporal form: gate logits, prior state */
    double *prior_out;
    const double *decay;                 /* gated form: decay logits */
    int post_decay;
    int unnormalized;                    /* App. D.2 variant: r without its normaliser */
    int next_head;              /* work counter, guarded by mu */
    int status;                 /* first error seen, guarded by mu */
    pthread_mutex_t mu;
} job_t;

/* One (b, h) sequence, straight from the definitions above. */
static int run_head(job_t *a, int b, int h)
{
    const int H = a->H, T = a->T, Dk = a->Dk, Dv = a->Dv, J = a->J;
    double *W = (double *)malloc(sizeof(double) * (size_t)J * Dv * Dk);
    double *prior = (double *)malloc(sizeof(double) * (size_t)J);
    double *num = (double *)malloc(sizeof(double) * (size_t)J);
    double *delta = (double *)malloc(sizeof(double) * (size_t)J);
    const int temporal = a->gk != NULL;
    /* temporal form: r_{t-1,jd} and rhobar_{t-1,jd}, [j][d] */
    double *rprev = (double *)malloc(sizeof(double) * (size_t)J * Dv);
    double *rho = (double *)malloc(sizeof(double) * (size_t)J * Dv);
    if (!W || !prior || !num || !delta || !rprev || !rho) {
        free(W); free(prior); free(num); free(delta); free(rprev); free(rho);
        return -2;
    }
    int rc = 0;
    for (int j = 0; j < J; ++j)
        for (int d = 0; d < Dv; ++d) {
            const size_t p = (((size_t)b * H + h) * 2 * J + j) * Dv + d;
            rprev[(size_t)j * Dv + d] = a->prior_in ? a->prior_in[p] : 1.0 / J;
            rho[(size_t)j * Dv + d] = a->prior_in ? a->prior_in[p + (size_t)J * Dv] : 1.0 / J;
        }

    /* initial state W_0 (zeros when none is given) */
    for (int j = 0; j < J; ++j)
        for (int d = 0; d < Dv; ++d)
            for (int i = 0; i < Dk; ++i) {
                size_t s = ((((size_t)b * H + h) * J + j) * Dk + i) * Dv + d;
                W[((size_t)j * Dv + d) * Dk + i] = a->state_in ? a->state_in[s] : 0.0;
            }

    for (int t = 0; t < T && rc == 0; ++t) {
        const size_t row = ((size_t)b * T + t) * H + h;
        const double *kt = a->k + row * Dk;
        const double *qt = a->q + row * Dk;
        const double *vt = a->v + row * Dv;
        const double *lbt = a->lb + row * (size_t)J * Dv;
        const double *lkt = a->lk + row * (size_t)J * Dv;
        const double *lqt = a->lq + row * (size_t)J * Dv;

        for (int d = 0; d < Dv; ++d) {
            /* key-side prior pi^k_{jd} = softmax_j(logit) */
            double m = -INFINITY, z = 0.0;
            for (int j = 0; j < J; ++j) m = fmax(m, lkt[(size_t)j * Dv + d]);
            for (int j = 0; j < J; ++j) z += exp(lkt[(size_t)j * Dv + d] - m);
            for (int j = 0; j < J; ++j) prior[j] = exp(lkt[(size_t)j * Dv + d] - m) / z;
            if (temporal) {
                /* App. B.3: mix in the previous token's responsibilities */
                const double g = 1.0 / (1.0 + exp(-a->gk[row * Dv + d]));
                for (int j = 0; j < J; ++j)
                    prior[j] = (1.0 - g) * rprev[(size_t)j * Dv + d] + g * prior[j];
            }

            /* gated, pre-decay: the state decays before the prediction */
            if (a->decay && !a->post_decay)
                for (int j = 0; j < J; ++j) {
                    double *w = W + ((size_t)j * Dv + d) * Dk;
                    const double *dl = a->decay + (row * J + j) * (size_t)Dk;
                    for (int i = 0; i < Dk; ++i) w[i] *= 1.0 / (1.0 + exp(-dl[i]));
                }

            /* prediction errors with the previous (pre-decay: decayed) state */
            for (int j = 0; j < J; ++j) {
                const double *w = W + ((size_t)j * Dv + d) * Dk;
                double pred = 0.0;
                for (int i = 0; i < Dk; ++i) pred += w[i] * kt[i];
                delta[j] = vt[d] - pred;
            }

            /* E-step: responsibilities, pi * N(v; w^T k, 1) normalised over j.
             * Numerator and denominator are both divided by the largest
             * exp(-delta^2/2), which leaves r unchanged and keeps the
             * normaliser finite when every exp(-delta^2/2) underflows. */
            double shift = -INFINITY;
            for (int j = 0; j < J; ++j) shift = fmax(shift, -0.5 * delta[j] * delta[j]);
            double Z = 0.0;
            for (int j = 0; j < J; ++j) {
                num[j] = prior[j] * exp(-0.5 * delta[j] * delta[j] - shift);
                Z += num[j];
            }
            if (!(Z > 0.0) || !isfinite(Z)) { rc = -1; break; }

            /* M-step: one gradient step of size beta on the log-likelihood
             * (unnormalised variant: on the likelihood, r without Z) */
            for (int j = 0; j < J; ++j) {
                double r = num[j] / Z;
                if (a->unnormalized) r = prior[j] * exp(-0.5 * delta[j] * delta[j]);
                const double beta = 1.0 / (1.0 + exp(-lbt[(size_t)j * Dv + d]));
                double *w = W + ((size_t)j * Dv + d) * Dk;
                if (a->decay && a->post_decay) {   /* gated, post-decay */
                    const double *dl = a->decay + (row * J + j) * (size_t)Dk;
                    for (int i = 0; i < Dk; ++i) w[i] *= 1.0 / (1.0 + exp(-dl[i]));
                }
                for (int i = 0; i < Dk; ++i) w[i] += beta * r * delta[j] * kt[i];
                if (a->resp) a->resp[(row * J + j) * Dv + d] = r;
                if (temporal) rprev[(size_t)j * Dv + d] = r;
                if (a->delta_out) a->delta_out[(row * J + j) * Dv + d] = delta[j];
            }

            /* retrieval from the updated state, query-side prior softmax_j */
            m = -INFINITY; z = 0.0;
            for (int j = 0; j < J; ++j) m = fmax(m, lqt[(size_t)j * Dv + d]);
            for (int j = 0; j < J; ++j) z += exp(lqt[(size_t)j * Dv + d] - m);
            double out = 0.0;
            const double gq = temporal ? 1.0 / (1.0 + exp(-a->gq[row * Dv + d])) : 0.0;
            for (int j = 0; j < J; ++j) {
                double pq = exp(lqt[(size_t)j * Dv + d] - m) / z;
                if (temporal) {
                    /* App. B.3: running mixture of the query-side priors */
                    double *rq = rho + (size_t)j * Dv + d;
                    *rq = (1.0 - gq) * *rq + gq * pq;
                    pq = *rq;
                }
                const double *w = W + ((size_t)j * Dv + d) * Dk;
                double y = 0.0;
                for (int i = 0; i < Dk; ++i) y += w[i] * qt[i];
                out += pq * y;
            }
            a->o[row * Dv + d] = out;
        }
    }

    if (rc == 0 && a->state_out)
        for (int j = 0; j < J; ++j)
            for (int d = 0; d < Dv; ++d)
                for (int i = 0; i < Dk; ++i) {
                    size_t s = ((((size_t)b * H + h) * J + j) * Dk + i) * Dv + d;
                    a->state_out[s] = W[((size_t)j * Dv + d) * Dk + i];
                }
    if (rc == 0 && temporal && a->prior_out)
        for (int j = 0; j < J; ++j)
            for (int d = 0; d < Dv; ++d) {
                const size_t p = (((size_t)b * H + h) * 2 * J + j) * Dv + d;
                a->prior_out[p] = rprev[(size_t)j * Dv + d];
                a->prior_out[p + (size_t)J * Dv] = rho[(size_t)j * Dv + d];
            }

    free(W); free(prior); free(num); free(delta); free(rprev); free(rho);
    return rc;
}

static void *worker(void *p)
{
    job_t *a = (job_t *)p;
    for (;;) {
        pthread_mutex_lock(&a->mu);
        int hh = a->next_head++;
        int stop = a->status != 0;
        pthread_mutex_unlock(&a->mu);
        if (stop || hh >= a->B * a->H) break;
        int rc = run_head(a, hh / a->H, hh % a->H);
        if (rc != 0) {
            pthread_mutex_lock(&a->mu);
            if (a->status == 0) a->status = rc;
            pthread_mutex_unlock(&a->mu);
        }
    }
    return NULL;
}

static int run_all(job_t *ap, int nthreads);
int swila_oracle_forward_ext(int B, int H, int T, int Dk, int Dv, int J,
                             const double *q, const double *k, const double *v,
                             const double *beta_logit, const double *prior_k_logit,
                             const double *prior_q_logit, const double *gate_k_logit,
                             const double *gate_q_logit, const double *decay_logit,
                             int post_decay, int unnormalized,
                             const double *state_in, const double *prior_in,
                             double *state_out, double *prior_out, double *o, double *resp_out,
                             double *delta_out, int nthreads);

/*
 * Forward over T tokens for every (b, h).  state_in may be NULL (zeros);
 * state_out, resp_out and delta_out may be NULL (not written).  state_out
 * must not alias state_in.  nthreads <= 0 uses every online core.
 * Returns 0, -1 if a responsibility normaliser is zero or not finite,
 * -2 on allocation failure, -3 on bad sizes.
 */
int swila_oracle_forward(int B, int H, int T, int Dk, int Dv, int J,
                         const double *q, const double *k, const double *v,
                         const double *beta_logit, const double *prior_k_logit,
                         const double *prior_q_logit, const double *state_in,
                         double *state_out, double *o, double *resp_out,
                         double *delta_out, int nthreads)
{
    return swila_oracle_forward_ext(B, H, T, Dk, Dv, J, q, k, v, beta_logit, prior_k_logit,
                                    prior_q_logit, NULL, NULL, NULL, 0, 0, state_in, NULL,
                                    state_out, NULL, o, resp_out, delta_out, nthreads);
}

/*
 * The same with the temporal priors of App. B.3 when gate_k_logit and
 * gate_q_logit are given ([B, T, H, Dv]; both or neither), and with the
 * gated decay of App. B.4 when decay_logit is given ([B, T, H, J, Dk];
 * post_decay selects eq. post-decay instead of eq. pre-decay).  prior_in is the
 * prior state [B, H, 2, J, Dv] or NULL (uniform); prior_out receives the
 * final one, or is NULL.  Without either this is the plain forward.
 * unnormalized selects App. D.2's unnormalised responsibilities (plain form
 * only: -3 with gates or decay).
 */
int swila_oracle_forward_ext(int B, int H, int T, int Dk, int Dv, int J,
                             const double *q, const double *k, const double *v,
                             const double *beta_logit, const double *prior_k_logit,
                             const double *prior_q_logit, const double *gate_k_logit,
                             const double *gate_q_logit, const double *decay_logit,
                             int post_decay, int unnormalized,
                             const double *state_in, const double *prior_in,
                             double *state_out, double *prior_out, double *o, double *resp_out,
                             double *delta_out, int nthreads)
{
    if (B < 0 || H < 0 || T < 0 || Dk <= 0 || Dv <= 0 || J <= 0) return -3;
    if ((gate_k_logit == NULL) != (gate_q_logit == NULL)) return -3;
    if (unnormalized && (gate_k_logit || decay_logit)) return -3;
    job_t a;
    memset(&a, 0, sizeof a);
    a.B = B; a.H = H; a.T = T; a.Dk = Dk; a.Dv = Dv; a.J = J;
    a.q = q; a.k = k; a.v = v;
    a.lb = beta_logit; a.lk = prior_k_logit; a.lq = prior_q_logit;
    a.state_in = state_in; a.state_out = state_out; a.o = o;
    a.resp = resp_out; a.delta_out = delta_out;
    a.gk = gate_k_logit; a.gq = gate_q_logit;
    a.prior_in = prior_in; a.prior_out = prior_out;
    a.decay = decay_logit; a.post_decay = post_decay;
    a.unnormalized = unnormalized;
    return run_all(&a, nthreads);
}

static int run_all(job_t *ap, int nthreads)
{
    job_t a = *ap;
    pthread_mutex_init(&a.mu, NULL);

    int n = nthreads;
    if (n <= 0) n = (int)sysconf(_SC_NPROCESSORS_ONLN);
    if (n < 1) n = 1;
    if (n > a.B * a.H) n = a.B * a.H;
    if (n <= 1) {
        worker(&a);
    } else {
        pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n);
        if (!th) { pthread_mutex_destroy(&a.mu); return -2; }
        int started = 0;
        for (int i = 0; i < n; ++i)
            if (pthread_create(&th[i], NULL, worker, &a) == 0) ++started;
        if (started == 0) worker(&a);
        for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
        free(th);
    }
    pthread_mutex_destroy(&a.mu);
    return a.status;
}
