// C ABI of libswila.so: argument checks, then dispatch to the kernels.
// Every check runs before anything is enqueued, so a failing call leaves the
// stream untouched.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "launch.hpp"
#include "swila.h"

// Device scratch of swila_forward_noalloc: each GPU the library runs on holds
// its own copy until the process ends.  In host code this name is a stand-in,
// not a device address; host code uses the address hipGetSymbolAddress returns
// for the current device (scratch_address below).
static __device__ __align__(256) unsigned char scratch[SWILA_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local char g_err[512];

int fail(int code, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

void clear_error() { g_err[0] = 0; }

bool dim_ok(int x) { return x == 16 || x == 32 || x == 64 || x == 128; }
constexpr int64_t kMaxHeads = int64_t(1) << 26;
// every J the paper uses (its Sec. 5.1 sweep: powers of two up to 16), and 3
bool j_ok(int j) { return j == 1 || j == 2 || j == 3 || j == 4 || j == 8 || j == 16; }

int check_shape(const swila_shape *s, bool decode) {
    if (!s) return fail(SWILA_EINVAL, "shape is NULL");
    if (s->B < 1 || s->H < 1 || s->T < 0 || s->Dk < 1 || s->Dv < 1 || s->J < 1)
        return fail(SWILA_EINVAL, "invalid shape B=%d H=%d T=%d Dk=%d Dv=%d J=%d", s->B, s->H,
                    s->T, s->Dk, s->Dv, s->J);
    if (decode && s->T != 1) return fail(SWILA_EINVAL, "decode needs T == 1 (got %d)", s->T);
    if (!dim_ok(s->Dk) || !dim_ok(s->Dv))
        return fail(SWILA_EUNSUPPORTED, "Dk=%d Dv=%d: supported sizes are 16, 32, 64, 128", s->Dk,
                    s->Dv);
    if (!j_ok(s->J))
        return fail(SWILA_EUNSUPPORTED, "J=%d: supported are 1, 2, 3, 4, 8, 16", s->J);
    if (s->B > 65535 || s->H > 65535)
        return fail(SWILA_EUNSUPPORTED, "B=%d H=%d: at most 65535 each", s->B, s->H);
    // the matrix-core kernels launch (Dv / 8) * B * H blocks or fewer on a 1-D
    // grid and index heads with 32-bit integers
    if ((int64_t)s->B * s->H > kMaxHeads)
        return fail(SWILA_EUNSUPPORTED, "B*H=%lld: at most %lld heads per call",
                    (long long)s->B * s->H, (long long)kMaxHeads);
    return SWILA_OK;
}

int check_opts(const swila_opts *o) {
    if (!o) return fail(SWILA_EINVAL, "opts is NULL");
    if (o->in_dtype != SWILA_F32 && o->in_dtype != SWILA_BF16)
        return fail(SWILA_EINVAL, "in_dtype %d is not SWILA_F32 or SWILA_BF16", o->in_dtype);
    if (o->out_dtype != SWILA_F32 && o->out_dtype != SWILA_BF16)
        return fail(SWILA_EINVAL, "out_dtype %d is not SWILA_F32 or SWILA_BF16", o->out_dtype);
    if (o->algo != SWILA_ALGO_AUTO && o->algo != SWILA_ALGO_RECURRENT &&
        o->algo != SWILA_ALGO_CHUNK_EXACT && o->algo != SWILA_ALGO_NEWTON)
        return fail(SWILA_EUNSUPPORTED, "algo %d is not available", o->algo);
    if (o->algo == SWILA_ALGO_CHUNK_EXACT && o->in_dtype != SWILA_BF16)
        return fail(SWILA_EUNSUPPORTED, "SWILA_ALGO_CHUNK_EXACT needs bf16 inputs");
    if (o->algo == SWILA_ALGO_NEWTON && o->in_dtype != SWILA_BF16)
        return fail(SWILA_EUNSUPPORTED, "SWILA_ALGO_NEWTON needs bf16 inputs");
    if (o->chunk < 0) return fail(SWILA_EINVAL, "chunk %d < 0", o->chunk);
    if ((o->algo == SWILA_ALGO_CHUNK_EXACT || o->algo == SWILA_ALGO_NEWTON) && o->chunk != 0 &&
        o->chunk != 16)
        return fail(SWILA_EUNSUPPORTED, "chunk %d: the chunked forms use 16 (or 0)", o->chunk);
    if (o->max_iters < 0) return fail(SWILA_EINVAL, "max_iters %d < 0", o->max_iters);
    if (o->tol != o->tol) return fail(SWILA_EINVAL, "tol is NaN");
    if (o->flags & ~(uint32_t)(SWILA_FLAG_NEWTON_NO_CLAMP | SWILA_FLAG_NEWTON_SYNC |
                               SWILA_FLAG_UNNORMALIZED))
        return fail(SWILA_EINVAL, "unknown flags 0x%x", o->flags);
    if ((o->flags & SWILA_FLAG_UNNORMALIZED) && o->algo != SWILA_ALGO_NEWTON)
        return fail(SWILA_EUNSUPPORTED, "SWILA_FLAG_UNNORMALIZED needs SWILA_ALGO_NEWTON");
    return SWILA_OK;
}

// The matrix-core chunk scan takes bf16 inputs and J <= kMaxChunkJ; AUTO picks
// it whenever it can, the token-by-token scan otherwise.
bool use_chunk(const swila_shape *s, const swila_opts *o) {
    if (o->algo == SWILA_ALGO_CHUNK_EXACT) return true;
    return o->algo == SWILA_ALGO_AUTO && o->in_dtype == SWILA_BF16 && s->J <= swila::kMaxChunkJ;
}

// The chunked forms (exact chunk scan, App. D) hold all J components of eight or
// more output dims in one wave: J <= kMaxChunkJ.
int check_chunk_j(const swila_shape *s, const swila_opts *o) {
    if ((o->algo == SWILA_ALGO_CHUNK_EXACT || o->algo == SWILA_ALGO_NEWTON) &&
        s->J > swila::kMaxChunkJ)
        return fail(SWILA_EUNSUPPORTED, "J=%d: the chunked forms support J <= %d", s->J,
                    swila::kMaxChunkJ);
    return SWILA_OK;
}

struct Span {
    const char *name;
    const void *p;
    size_t bytes;
};

// Pointer present (when required), 16-byte aligned, and disjoint from the
// given inputs.
int check_ptr(const Span &s, bool required) {
    if (!s.p) return required ? fail(SWILA_EINVAL, "%s is NULL", s.name) : SWILA_OK;
    if (reinterpret_cast<uintptr_t>(s.p) % 16 != 0)
        return fail(SWILA_EINVAL, "%s is not 16-byte aligned", s.name);
    return SWILA_OK;
}

bool overlap(const Span &a, const Span &b) {
    if (!a.p || !b.p || a.bytes == 0 || b.bytes == 0) return false;
    const char *a0 = static_cast<const char *>(a.p), *b0 = static_cast<const char *>(b.p);
    return a0 < b0 + b.bytes && b0 < a0 + a.bytes;
}

int map_hip(hipError_t e, const char *what) {
    if (e == hipSuccess) return SWILA_OK;
    return fail(SWILA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// SWILA_FLAG_NEWTON_SYNC: wait for the Newton launch and report whether every
// block of columns met the tolerance (iters_out[1] counts those that did not).
int newton_status(const int32_t *iters_out, hipStream_t st) {
    int32_t it[2] = {0, 0};
    int rc = map_hip(hipMemcpyAsync(it, iters_out, sizeof it, hipMemcpyDeviceToHost, st),
                     "iteration count copy");
    if (rc) return rc;
    rc = map_hip(hipStreamSynchronize(st), "stream synchronize");
    if (rc) return rc;
    if (it[1] > 0)
        return fail(SWILA_ENOTCONVERGED, "%d blocks of columns did not converge in %d sweeps",
                    it[1], it[0]);
    return SWILA_OK;
}

// Shared checks of forward and decode; fills the launch arguments.
int prepare(const swila_shape *shape, const swila_opts *opts, bool decode, const void *q,
            const void *k, const void *v, const void *lb, const void *lk, const void *lq,
            const float *state_in, float *state_out, void *o, float *resp,
            swila::LayerArgs *a) {
    int rc = check_shape(shape, decode);
    if (rc) return rc;
    rc = check_opts(opts);
    if (rc) return rc;
    const size_t B = shape->B, H = shape->H, T = shape->T, Dk = shape->Dk, Dv = shape->Dv,
                 J = shape->J;
    const size_t ie = opts->in_dtype == SWILA_BF16 ? 2 : 4;
    const size_t oe = opts->out_dtype == SWILA_BF16 ? 2 : 4;
    const bool need = T > 0;
    const Span in[] = {
        {"q", q, B * T * H * Dk * ie},          {"k", k, B * T * H * Dk * ie},
        {"v", v, B * T * H * Dv * ie},          {"beta_logit", lb, B * T * H * J * Dv * ie},
        {"prior_k_logit", lk, B * T * H * J * Dv * ie},
        {"prior_q_logit", lq, B * T * H * J * Dv * ie},
        {"state_in", state_in, B * H * J * Dk * Dv * 4},
    };
    const int n_in = sizeof in / sizeof in[0];
    for (int i = 0; i < n_in; ++i) {
        rc = check_ptr(in[i], need && i < 6);  // state_in may be NULL (zeros)
        if (rc) return rc;
    }
    const Span outs[] = {
        {"o", o, B * T * H * Dv * oe},
        {"state_out", state_out, B * H * J * Dk * Dv * 4},
        {"resp_out", resp, B * T * H * J * Dv * 4},
    };
    for (int x = 0; x < 3; ++x) {
        rc = check_ptr(outs[x], need && x == 0);  // o is required when T > 0
        if (rc) return rc;
        for (int i = 0; i < n_in; ++i) {
            // the state may be updated in place: state_out == state_in exactly
            if (x == 1 && i == 6 && state_out == state_in) continue;
            if (overlap(outs[x], in[i]))
                return fail(SWILA_EINVAL, "%s overlaps %s", outs[x].name, in[i].name);
        }
    }
    if (overlap(outs[0], outs[1]) || overlap(outs[0], outs[2]) || overlap(outs[1], outs[2]))
        return fail(SWILA_EINVAL, "output tensors overlap");
    *a = swila::LayerArgs{q, k, v, lb, lk, lq, state_in, state_out, o, resp,
                          shape->B, shape->H, shape->T, shape->Dk, shape->Dv, shape->J,
                          opts->in_dtype == SWILA_BF16, opts->out_dtype == SWILA_BF16};
    return SWILA_OK;
}

// Temporal SwiLA arguments (App. B.3): the two gate-logit tensors (inputs,
// in_dtype, [B,T,H,Dv]) and the prior state in and out ([B,H,2,J,Dv] fp32).
// prior_out may equal prior_in; every other pair is disjoint, and none of them
// overlaps a tensor of the base call.
int check_temporal(const swila_shape *shape, const swila_opts *opts, const swila_temporal *tp,
                   const void *q, const void *k, const void *v, const void *lb, const void *lk,
                   const void *lq, const float *state_in, float *state_out, void *o, float *resp,
                   swila::LayerArgs *a) {
    if (!tp) return fail(SWILA_EINVAL, "temporal is NULL");
    const size_t B = shape->B, H = shape->H, T = shape->T, Dk = shape->Dk, Dv = shape->Dv,
                 J = shape->J;
    const size_t ie = opts->in_dtype == SWILA_BF16 ? 2 : 4;
    const size_t oe = opts->out_dtype == SWILA_BF16 ? 2 : 4;
    const bool need = T > 0;
    const Span t_in[] = {
        {"gate_k_logit", tp->gate_k_logit, B * T * H * Dv * ie},
        {"gate_q_logit", tp->gate_q_logit, B * T * H * Dv * ie},
        {"prior_in", tp->prior_in, B * H * 2 * J * Dv * 4},
    };
    const Span p_out{"prior_out", tp->prior_out, B * H * 2 * J * Dv * 4};
    for (int i = 0; i < 3; ++i) {
        int rc = check_ptr(t_in[i], need && i < 2);
        if (rc) return rc;
    }
    int rc = check_ptr(p_out, false);
    if (rc) return rc;
    const Span base_in[] = {
        {"q", q, B * T * H * Dk * ie},          {"k", k, B * T * H * Dk * ie},
        {"v", v, B * T * H * Dv * ie},          {"beta_logit", lb, B * T * H * J * Dv * ie},
        {"prior_k_logit", lk, B * T * H * J * Dv * ie},
        {"prior_q_logit", lq, B * T * H * J * Dv * ie},
        {"state_in", state_in, B * H * J * Dk * Dv * 4},
    };
    const Span base_out[] = {
        {"o", o, B * T * H * Dv * oe},
        {"state_out", state_out, B * H * J * Dk * Dv * 4},
        {"resp_out", resp, B * T * H * J * Dv * 4},
    };
    for (const Span &x : base_out) {
        for (const Span &t : t_in)
            if (overlap(t, x)) return fail(SWILA_EINVAL, "%s overlaps %s", t.name, x.name);
        if (overlap(p_out, x)) return fail(SWILA_EINVAL, "prior_out overlaps %s", x.name);
    }
    for (const Span &x : base_in)
        if (overlap(p_out, x)) return fail(SWILA_EINVAL, "prior_out overlaps %s", x.name);
    for (int i = 0; i < 3; ++i) {
        if (i == 2 && tp->prior_out == tp->prior_in) continue;   // updated in place
        if (overlap(p_out, t_in[i]))
            return fail(SWILA_EINVAL, "prior_out overlaps %s", t_in[i].name);
    }
    a->gk = tp->gate_k_logit;
    a->gq = tp->gate_q_logit;
    a->prior_in = tp->prior_in;
    a->prior_out = tp->prior_out;
    return SWILA_OK;
}

// Gated SwiLA argument (App. B.4): the decay logits, an input of in_dtype,
// [B,T,H,J,Dk]; disjoint from every output.
int check_gated(const swila_shape *shape, const swila_opts *opts, const swila_gated *gd,
                const swila_temporal *tp, void *o, float *state_out, float *resp,
                swila::LayerArgs *a) {
    if (!gd) return fail(SWILA_EINVAL, "gated is NULL");
    const size_t B = shape->B, H = shape->H, T = shape->T, Dk = shape->Dk, Dv = shape->Dv,
                 J = shape->J;
    const size_t ie = opts->in_dtype == SWILA_BF16 ? 2 : 4;
    const size_t oe = opts->out_dtype == SWILA_BF16 ? 2 : 4;
    const Span dec{"decay_logit", gd->decay_logit, B * T * H * J * Dk * ie};
    int rc = check_ptr(dec, T > 0);
    if (rc) return rc;
    const Span outs[] = {
        {"o", o, B * T * H * Dv * oe},
        {"state_out", state_out, B * H * J * Dk * Dv * 4},
        {"resp_out", resp, B * T * H * J * Dv * 4},
        {"prior_out", tp ? tp->prior_out : nullptr, B * H * 2 * J * Dv * 4},
    };
    for (const Span &x : outs)
        if (overlap(dec, x)) return fail(SWILA_EINVAL, "decay_logit overlaps %s", x.name);
    a->decay = gd->decay_logit;
    return SWILA_OK;
}

// Address of this device's copy of the scratch array, looked up once per device
// with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_at[kMaxDevices];

int scratch_address(void **out) {
    int dev = 0;
    int rc = map_hip(hipGetDevice(&dev), "hipGetDevice");
    if (rc) return rc;
    if (dev < 0 || dev >= kMaxDevices)
        return fail(SWILA_EUNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_at[dev]) {
        void *p = nullptr;
        rc = map_hip(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "scratch symbol address");
        if (rc) return rc;
        if (!p) return fail(SWILA_EHIP, "scratch symbol address is NULL");
        g_scratch_at[dev] = p;
    }
    *out = g_scratch_at[dev];
    return SWILA_OK;
}

}  // namespace

extern "C" {

int swila_version(void) { return 1; }

const char *swila_last_error(void) { return g_err; }

size_t swila_state_bytes(const swila_shape *s) {
    if (!s || s->B < 1 || s->H < 1 || s->Dk < 1 || s->Dv < 1 || s->J < 1) return 0;
    return (size_t)s->B * s->H * s->J * s->Dk * s->Dv * sizeof(float);
}

int swila_state_init(const swila_shape *shape, float *state, const float *src, void *stream) {
    clear_error();
    if (!shape) return fail(SWILA_EINVAL, "shape is NULL");
    const size_t bytes = swila_state_bytes(shape);
    if (bytes == 0) return fail(SWILA_EINVAL, "invalid shape");
    if (!state) return fail(SWILA_EINVAL, "state is NULL");
    if (reinterpret_cast<uintptr_t>(state) % 16 || reinterpret_cast<uintptr_t>(src) % 16)
        return fail(SWILA_EINVAL, "state or src is not 16-byte aligned");
    const Span a{"state", state, bytes}, b{"src", src, bytes};
    if (src && src != state && overlap(a, b)) return fail(SWILA_EINVAL, "state overlaps src");
    return map_hip(swila::launch_state_fill(state, src, bytes / sizeof(float),
                                            static_cast<hipStream_t>(stream)),
                   "state_init launch");
}

size_t swila_forward_workspace_bytes(const swila_shape *shape, const swila_opts *opts) {
    if (!shape || !opts || opts->algo != SWILA_ALGO_NEWTON) return 0;
    if (shape->B < 1 || shape->H < 1 || shape->T < 1 || shape->Dv < 1 || shape->J < 1) return 0;
    return swila::newton_workspace_bytes(shape->B, shape->H, shape->T, shape->Dv, shape->J);
}

int swila_forward(const swila_shape *shape, const swila_opts *opts, const void *q, const void *k,
                  const void *v, const void *beta_logit, const void *prior_k_logit,
                  const void *prior_q_logit, const float *state_in, float *state_out, void *o,
                  float *resp_out, void *workspace, size_t ws_bytes, int32_t *iters_out,
                  void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, false, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, resp_out, &a);
    if (rc) return rc;
    rc = check_chunk_j(shape, opts);
    if (rc) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const bool newton = opts->algo == SWILA_ALGO_NEWTON;
    if (newton && shape->T > 0) {
        if (resp_out)
            return fail(SWILA_EUNSUPPORTED, "resp_out is not produced by SWILA_ALGO_NEWTON");
        const size_t need = swila_forward_workspace_bytes(shape, opts);
        if (!workspace) return fail(SWILA_EINVAL, "SWILA_ALGO_NEWTON needs a workspace");
        if (reinterpret_cast<uintptr_t>(workspace) % 16)
            return fail(SWILA_EINVAL, "workspace is not 16-byte aligned");
        if (ws_bytes < need)
            return fail(SWILA_EINVAL, "workspace holds %zu bytes, %zu needed", ws_bytes, need);
        if (iters_out && reinterpret_cast<uintptr_t>(iters_out) % 4)
            return fail(SWILA_EINVAL, "iters_out is not 4-byte aligned");
        if ((opts->flags & SWILA_FLAG_NEWTON_SYNC) && !iters_out)
            return fail(SWILA_EINVAL, "SWILA_FLAG_NEWTON_SYNC needs iters_out");
        const size_t B = shape->B, H = shape->H, T = shape->T, Dk = shape->Dk, Dv = shape->Dv,
                     J = shape->J;
        const size_t ie = 2, oe = opts->out_dtype == SWILA_BF16 ? 2 : 4;
        const Span ws{"workspace", workspace, need}, it{"iters_out", iters_out, 8};
        const Span all[] = {
            {"q", q, B * T * H * Dk * ie},          {"k", k, B * T * H * Dk * ie},
            {"v", v, B * T * H * Dv * ie},          {"beta_logit", beta_logit, B * T * H * J * Dv * ie},
            {"prior_k_logit", prior_k_logit, B * T * H * J * Dv * ie},
            {"prior_q_logit", prior_q_logit, B * T * H * J * Dv * ie},
            {"state_in", state_in, B * H * J * Dk * Dv * 4},
            {"state_out", state_out, B * H * J * Dk * Dv * 4},
            {"o", o, B * T * H * Dv * oe},
        };
        for (const Span &x : all) {
            if (overlap(ws, x)) return fail(SWILA_EINVAL, "workspace overlaps %s", x.name);
            if (overlap(it, x)) return fail(SWILA_EINVAL, "iters_out overlaps %s", x.name);
        }
        if (overlap(ws, it)) return fail(SWILA_EINVAL, "iters_out overlaps workspace");
    }
    if (shape->T == 0) {
        if (!state_out) return SWILA_OK;
        return map_hip(swila::launch_state_fill(state_out, state_in,
                                                swila_state_bytes(shape) / sizeof(float), st),
                       "state copy");
    }
    if (newton) {
        // App. D defaults: at most 64 sweeps, tolerance 1e-3 (bf16 inputs)
        swila::NewtonArgs na{static_cast<float *>(workspace), iters_out,
                             opts->max_iters > 0 ? opts->max_iters : 64,
                             opts->tol == 0.f ? 1e-3f : opts->tol,
                             (opts->flags & SWILA_FLAG_NEWTON_NO_CLAMP) == 0,
                             (opts->flags & SWILA_FLAG_UNNORMALIZED) != 0};
        rc = map_hip(swila::launch_newton(a, na, st), "Newton launch");
        if (rc || !(opts->flags & SWILA_FLAG_NEWTON_SYNC)) return rc;
        return newton_status(iters_out, st);
    }
    if (use_chunk(shape, opts)) return map_hip(swila::launch_scan_pipe(a, st), "chunk scan launch");
    return map_hip(swila::launch_scan_direct(a, st), "scan launch");
}

int swila_forward_noalloc(const swila_shape *shape, const swila_opts *opts, const void *q,
                          const void *k, const void *v, const void *beta_logit,
                          const void *prior_k_logit, const void *prior_q_logit,
                          const float *state_in, float *state_out, void *o, float *resp_out,
                          int32_t *iters_out, void *stream) {
    clear_error();
    if (!shape) return fail(SWILA_EINVAL, "shape is NULL");
    if (!opts) return fail(SWILA_EINVAL, "opts is NULL");
    const size_t need = swila_forward_workspace_bytes(shape, opts);
    if (need > SWILA_NOALLOC_SCRATCH_BYTES)
        return fail(SWILA_EUNSUPPORTED,
                    "swila_forward_noalloc: this call needs %zu bytes of scratch, the library "
                    "holds %zu (B*H*J*Dv*16*ceil(T/16)*4 <= %zu)", need,
                    (size_t)SWILA_NOALLOC_SCRATCH_BYTES, (size_t)SWILA_NOALLOC_SCRATCH_BYTES);
    void *ws = nullptr;
    if (need > 0) {
        int rc = scratch_address(&ws);
        if (rc) return rc;
    }
    return swila_forward(shape, opts, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                         state_in, state_out, o, resp_out, ws,
                         need > 0 ? (size_t)SWILA_NOALLOC_SCRATCH_BYTES : 0, iters_out, stream);
}

int swila_forward_temporal(const swila_shape *shape, const swila_opts *opts, const void *q,
                           const void *k, const void *v, const void *beta_logit,
                           const void *prior_k_logit, const void *prior_q_logit,
                           const swila_temporal *temporal, const float *state_in,
                           float *state_out, void *o, float *resp_out, void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, false, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, resp_out, &a);
    if (rc) return rc;
    rc = check_temporal(shape, opts, temporal, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                        state_in, state_out, o, resp_out, &a);
    if (rc) return rc;
    rc = check_chunk_j(shape, opts);
    if (rc) return rc;
    if (opts->algo == SWILA_ALGO_NEWTON)
        return fail(SWILA_EUNSUPPORTED,
                    "SWILA_ALGO_NEWTON linearises the plain recurrence; not the temporal form");
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (shape->T == 0) {
        if (state_out) {
            rc = map_hip(swila::launch_state_fill(state_out, state_in,
                                                  swila_state_bytes(shape) / sizeof(float), st),
                         "state copy");
            if (rc) return rc;
        }
        if (!temporal->prior_out) return SWILA_OK;
        const size_t n = (size_t)shape->B * shape->H * 2 * shape->J * shape->Dv;
        return map_hip(swila::launch_fill(temporal->prior_out, temporal->prior_in, n,
                                          1.0f / shape->J, st),
                       "prior state copy");
    }
    if (use_chunk(shape, opts)) return map_hip(swila::launch_scan_pipe(a, st), "chunk scan launch");
    return map_hip(swila::launch_scan_direct(a, st), "scan launch");
}

int swila_decode_step_temporal(const swila_shape *shape, const swila_opts *opts, const void *q,
                               const void *k, const void *v, const void *beta_logit,
                               const void *prior_k_logit, const void *prior_q_logit,
                               const swila_temporal *temporal, const float *state_in,
                               float *state_out, void *o, void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, true, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, nullptr, &a);
    if (rc) return rc;
    if (opts->flags & SWILA_FLAG_UNNORMALIZED)
        return fail(SWILA_EUNSUPPORTED, "decode evaluates the plain recurrence");
    rc = check_temporal(shape, opts, temporal, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                        state_in, state_out, o, nullptr, &a);
    if (rc) return rc;
    return map_hip(swila::launch_decode(a, static_cast<hipStream_t>(stream)), "decode launch");
}

int swila_forward_gated(const swila_shape *shape, const swila_opts *opts, const void *q,
                        const void *k, const void *v, const void *beta_logit,
                        const void *prior_k_logit, const void *prior_q_logit,
                        const swila_gated *gated, const swila_temporal *temporal,
                        const float *state_in, float *state_out, void *o, float *resp_out,
                        void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, false, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, resp_out, &a);
    if (rc) return rc;
    if (temporal) {
        rc = check_temporal(shape, opts, temporal, q, k, v, beta_logit, prior_k_logit,
                            prior_q_logit, state_in, state_out, o, resp_out, &a);
        if (rc) return rc;
    }
    rc = check_gated(shape, opts, gated, temporal, o, state_out, resp_out, &a);
    if (rc) return rc;
    if (opts->algo == SWILA_ALGO_NEWTON)
        return fail(SWILA_EUNSUPPORTED,
                    "the gated form runs on SWILA_ALGO_CHUNK_EXACT or SWILA_ALGO_RECURRENT");
    const bool chunk_ok = swila::gated_chunk_supported(a);
    if (opts->algo == SWILA_ALGO_CHUNK_EXACT && !chunk_ok)
        return fail(SWILA_EUNSUPPORTED,
                    "the gated chunk form takes bf16 inputs without temporal priors, J <= 4 "
                    "and J * Dk <= 512 (J=%d, Dk=%d)",
                    shape->J, shape->Dk);
    const bool use_chunk = chunk_ok && opts->algo != SWILA_ALGO_RECURRENT;
    if (!use_chunk && shape->J * shape->Dk > swila::kMaxGatedJDk)
        return fail(SWILA_EUNSUPPORTED, "gated forward: J * Dk = %d exceeds %d",
                    shape->J * shape->Dk, swila::kMaxGatedJDk);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (shape->T == 0) {
        if (state_out) {
            rc = map_hip(swila::launch_state_fill(state_out, state_in,
                                                  swila_state_bytes(shape) / sizeof(float), st),
                         "state copy");
            if (rc) return rc;
        }
        if (!temporal || !temporal->prior_out) return SWILA_OK;
        const size_t n = (size_t)shape->B * shape->H * 2 * shape->J * shape->Dv;
        return map_hip(swila::launch_fill(temporal->prior_out, temporal->prior_in, n,
                                          1.0f / shape->J, st),
                       "prior state copy");
    }
    if (use_chunk) return map_hip(swila::launch_scan_gated_chunk(a, st), "gated chunk launch");
    return map_hip(swila::launch_scan_direct(a, st), "scan launch");
}

int swila_decode_step_gated(const swila_shape *shape, const swila_opts *opts, const void *q,
                            const void *k, const void *v, const void *beta_logit,
                            const void *prior_k_logit, const void *prior_q_logit,
                            const swila_gated *gated, const swila_temporal *temporal,
                            const float *state_in, float *state_out, void *o, void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, true, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, nullptr, &a);
    if (rc) return rc;
    if (opts->flags & SWILA_FLAG_UNNORMALIZED)
        return fail(SWILA_EUNSUPPORTED, "decode evaluates the plain recurrence");
    if (temporal) {
        rc = check_temporal(shape, opts, temporal, q, k, v, beta_logit, prior_k_logit,
                            prior_q_logit, state_in, state_out, o, nullptr, &a);
        if (rc) return rc;
    }
    rc = check_gated(shape, opts, gated, temporal, o, state_out, nullptr, &a);
    if (rc) return rc;
    return map_hip(swila::launch_decode(a, static_cast<hipStream_t>(stream)), "decode launch");
}

int swila_decode_step(const swila_shape *shape, const swila_opts *opts, const void *q,
                      const void *k, const void *v, const void *beta_logit,
                      const void *prior_k_logit, const void *prior_q_logit,
                      const float *state_in, float *state_out, void *o, void *stream) {
    clear_error();
    swila::LayerArgs a;
    int rc = prepare(shape, opts, true, q, k, v, beta_logit, prior_k_logit, prior_q_logit,
                     state_in, state_out, o, nullptr, &a);
    if (rc) return rc;
    if (opts->flags & SWILA_FLAG_UNNORMALIZED)
        return fail(SWILA_EUNSUPPORTED, "decode evaluates the plain recurrence");
    return map_hip(swila::launch_decode(a, static_cast<hipStream_t>(stream)), "decode launch");
}

size_t swila_backward_workspace_bytes(const swila_shape *s) {
    if (!s || s->B < 1 || s->H < 1 || s->T < 0 || s->Dk < 1 || s->Dv < 1 || s->J < 1) return 0;
    return swila::backward_workspace_bytes(s->B, s->H, s->T, s->Dk, s->Dv, s->J);
}

int swila_backward(const swila_shape *shape, const swila_opts *opts, const void *q,
                   const void *k, const void *v, const void *beta_logit,
                   const void *prior_k_logit, const void *prior_q_logit, const float *state_in,
                   const void *grad_o, const float *grad_state_out, float *grad_q, float *grad_k,
                   float *grad_v, float *grad_beta_logit, float *grad_prior_k_logit,
                   float *grad_prior_q_logit, float *grad_state_in, void *workspace,
                   size_t ws_bytes, void *stream) {
    clear_error();
    int rc = check_shape(shape, false);
    if (rc) return rc;
    rc = check_opts(opts);
    if (rc) return rc;
    if (shape->J > swila::kMaxChunkJ)
        return fail(SWILA_EUNSUPPORTED, "backward: J=%d, supported J <= %d", shape->J,
                    swila::kMaxChunkJ);
    if (opts->flags & SWILA_FLAG_UNNORMALIZED)
        return fail(SWILA_EUNSUPPORTED, "backward: the plain recurrence only");
    const size_t B = shape->B, H = shape->H, T = shape->T, Dk = shape->Dk, Dv = shape->Dv,
                 J = shape->J;
    const size_t ie = opts->in_dtype == SWILA_BF16 ? 2 : 4;
    const size_t oe = opts->out_dtype == SWILA_BF16 ? 2 : 4;
    const bool need = T > 0;
    const size_t nst = B * H * J * Dk * Dv * 4;
    const Span in[] = {
        {"q", q, B * T * H * Dk * ie},          {"k", k, B * T * H * Dk * ie},
        {"v", v, B * T * H * Dv * ie},          {"beta_logit", beta_logit, B * T * H * J * Dv * ie},
        {"prior_k_logit", prior_k_logit, B * T * H * J * Dv * ie},
        {"prior_q_logit", prior_q_logit, B * T * H * J * Dv * ie},
        {"grad_o", grad_o, B * T * H * Dv * oe},
        {"state_in", state_in, nst},
        {"grad_state_out", grad_state_out, nst},
    };
    for (int i = 0; i < 9; ++i) {
        rc = check_ptr(in[i], need && i < 7);   // the two states may be NULL (zeros)
        if (rc) return rc;
    }
    const size_t need_ws = swila_backward_workspace_bytes(shape);
    const Span outs[] = {
        {"grad_q", grad_q, B * T * H * Dk * 4},
        {"grad_k", grad_k, B * T * H * Dk * 4},
        {"grad_v", grad_v, B * T * H * Dv * 4},
        {"grad_beta_logit", grad_beta_logit, B * T * H * J * Dv * 4},
        {"grad_prior_k_logit", grad_prior_k_logit, B * T * H * J * Dv * 4},
        {"grad_prior_q_logit", grad_prior_q_logit, B * T * H * J * Dv * 4},
        {"grad_state_in", grad_state_in, nst},
        {"workspace", workspace, need_ws},
    };
    const int n_out = sizeof outs / sizeof outs[0];
    for (int x = 0; x < n_out; ++x) {
        rc = check_ptr(outs[x], need && x != 6);   // grad_state_in may be NULL
        if (rc) return rc;
        for (int i = 0; i < 9; ++i)
            if (overlap(outs[x], in[i]))
                return fail(SWILA_EINVAL, "%s overlaps %s", outs[x].name, in[i].name);
        for (int y = 0; y < x; ++y)
            if (overlap(outs[x], outs[y]))
                return fail(SWILA_EINVAL, "%s overlaps %s", outs[x].name, outs[y].name);
    }
    if (need && ws_bytes < need_ws)
        return fail(SWILA_EINVAL, "workspace holds %zu bytes, %zu needed", ws_bytes, need_ws);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (T == 0) {
        if (!grad_state_in) return SWILA_OK;
        return map_hip(swila::launch_state_fill(grad_state_in, grad_state_out, nst / 4, st),
                       "state copy");
    }
    // workspace: delta ([B,T,H,J,Dv]); the chunk pass's operands c, dpred, pi^q
    // and dL/do in its tile order (tokens padded to whole checkpoint intervals);
    // state checkpoints W_n, E_n
    const size_t nch = (T + swila::kBwdChunk - 1) / swila::kBwdChunk;
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    char *ws = static_cast<char *>(workspace);
    const size_t per_tok = up(B * T * H * J * Dv * 4), ck = up(B * H * nch * Dv * J * Dk * 4);
    const size_t pk = up(B * H * nch * swila::kBwdChunk * J * Dv * 4),
                 dpk = up(B * H * nch * swila::kBwdChunk * Dv * 4);
    swila::BackwardArgs ba;
    ba.f = swila::LayerArgs{q, k, v, beta_logit, prior_k_logit, prior_q_logit, state_in,
                            nullptr, nullptr, nullptr, shape->B, shape->H, shape->T,
                            shape->Dk, shape->Dv, shape->J,
                            opts->in_dtype == SWILA_BF16, opts->out_dtype == SWILA_BF16};
    ba.grad_o = grad_o;
    ba.grad_state = grad_state_out;
    ba.dq = grad_q;
    ba.dk = grad_k;
    ba.dv = grad_v;
    ba.dlb = grad_beta_logit;
    ba.dlk = grad_prior_k_logit;
    ba.dlq = grad_prior_q_logit;
    ba.dstate = grad_state_in;
    ba.delta = reinterpret_cast<float *>(ws);
    ws += per_tok;
    ba.cpk = reinterpret_cast<float *>(ws);
    ba.ppk = reinterpret_cast<float *>(ws + pk);
    ba.qpk = reinterpret_cast<float *>(ws + 2 * pk);
    ba.dopk = reinterpret_cast<float *>(ws + 3 * pk);
    ws += 3 * pk + dpk;
    ba.wck = reinterpret_cast<float *>(ws);
    ba.eck = reinterpret_cast<float *>(ws + ck);
    return map_hip(swila::launch_backward(ba, st), "backward launch");
}

}  // extern "C"
