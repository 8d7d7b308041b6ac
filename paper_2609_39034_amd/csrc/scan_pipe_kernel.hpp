// Exact chunk scan on the matrix cores (bf16 inputs, fp32 state), pipelined
// over one sequential wave and the matrix-core waves.
//
// Every update of eq. recurrence adds a multiple of k_t to w_{jd}, so inside a
// chunk of 16 tokens starting from state S_n the state before token t is
//   w_{t-1,jd} = S_{n,jd} + sum_{s<t in chunk} c_{s,jd} k_s,   c = beta r delta.
// Hence, exactly up to rounding order,
//   pred_t   = k_t . S_n + sum_{s<t} (k_t . k_s) c_s           (prediction)
//   w_t . q_t = q_t . S_n + sum_{s<=t} (q_t . k_s) c_s          (eq. retrieval)
//   S_{n+1}  = S_n + sum_s c_s k_s^T.
// The Dk-long contractions are 16 x 16 matrix-core products per chunk; only
// the scalar recurrence of the coefficients over the 16 tokens of a chunk (a
// <= 15-term right-looking update plus the E-step, per token) is sequential.
// This is the algebra of the delta-rule chunk form that App. D builds on,
// applied to the exact nonlinear recurrence one chunk at a time.  The
// schedule puts only a 16 x 16 product between the recurrence of one chunk
// and that of the next.  With C_n the coefficients of chunk n:
//   P_{n+1} = K_{n+1} S_{n+1} = K_{n+1} S_n + (K_{n+1} K_n^T) C_n.
// While the sequential wave runs the recurrence of chunk n (phase B), the
// matrix-core waves do everything that does not need C_n:
//   S_n = S_{n-1} + K_{n-1}^T C_{n-1}          (state update of the previous chunk)
//   Y_{n-1} += tril(A_{n-1}) C_{n-1}; pi^q Y    (retrieval of the previous chunk)
//   o_{n-2} = sum_j pi^q Y                      (output of the chunk before)
//   Y0_n = Q_n S_n,  X_{n+1} = K_{n+1} S_n,  G'_n = K_{n+1} K_n^T (each wave,
//   in registers),  G_{n+1} = K_{n+1} K_{n+1}^T,  pi^q_n, beta_{n+1}, ...
//   and the HBM -> LDS transfer of chunk n+2 (direct global-to-LDS loads).
// After C_n is published they form P_{n+1} = X_{n+1} + G'_n C_n (three
// 16 x 16 x 16 products) and the next recurrence starts.  Two block barriers
// per chunk.
//
// Precision.  bf16 q and k enter the matrix cores unrounded.  fp32 operands
// (the state, the coefficients, the Gram products) are split into a bf16 high
// part and a bf16 residual and the products that matter are summed (hi*hi +
// hi*lo [+ lo*hi]), about 2^-16 relative error per product; fp32 accumulation.
//
// Layout.  Block = one head (b, h) and DB output dims with all J components,
// N = J * DB columns (col = j * DB + dl); NW = N / 16 matrix-core waves, wave
// w holding the Dk x 16 state tile of columns 16w..16w+15 in MFMA accumulator
// layout; wave NW is the sequential wave.  Raw chunk inputs sit in LDS rings
// of a few chunk slots each; K and Q rows are stored with their 16-byte pieces permuted
// by row (piece p of row t at slot p ^ (t mod pieces)) so that the 16 lanes
// reading one column range hit distinct banks.
//
// Newton mode (App. D).  The same kernel evaluates the chunkwise quasi-Newton
// iteration of App. D.1-D.3.  Sweep i linearises the recurrence around the
// predictions pred^(i)_t = k_t . w^(i)_{t-1} of the previous sweep
// (eq. jacobian_coeff, eq. effective_input) and solves the linear recurrence
// eq. linearized exactly, chunk by chunk.  In solve form (per column, the
// output index d kept):
//   pred_t = k_t . S_n + sum_{s<t} (k_t . k_s) x_s,   x_t = p_t - g_t pred_t,
//   S_{n+1} = S_n + sum_s x_s k_s^T,
// which is the (I - Lambda)^{-1} of eq. aggregate_transition and
// eq. aggregate_history applied by forward substitution.  The matrix-core
// schedule above is unchanged; the sequential wave runs the linear step
// x_t = g_t (pred^(i)_t - pred_t) + beta r delta instead of the E-step.  The
// predictions of every sweep go to a workspace and are read back, chunk by
// chunk, by the next sweep.  Each block iterates until the largest change of
// its predictions is at most tol * max(1, largest prediction), or until
// max_iters sweeps; outputs and the final state are those of the last sweep.
//
// This header holds the kernel template and its launch dispatch; the three
// modes are instantiated in separate translation units (scan_pipe.hip,
// scan_pipe_newton.hip, scan_pipe_temporal.hip) so that they compile in
// parallel.
#pragma once
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kC = 16;    // tokens per chunk
// LDS ring slots per input, by how long a chunk stays in use after it lands
// (it lands two chunks ahead of the sequential wave):
constexpr int kRingKQ = 4;  // K, Q: chunks n-1 .. n+2 (state update, retrieval of n-1)
constexpr int kRingQP = 3;  // query-prior logits, Newton predictions: n .. n+2
constexpr int kRingS = 2;   // beta and key-prior logits, v: n+1, n+2 (staged one chunk ahead)
constexpr int kTP = kC + 4;  // row of a column-major [column][token] staging array
constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// The sequential wave works in scaled units: with s^2 = log2(e) / 2,
// d = s (v - pred) makes the E-step exponent log2(e) (lk - delta^2 / 2) a
// single fused multiply-add, -d * d + log2(e) lk, and the coefficient
// s c = beta r d feeds the scaled predictions s pred.
constexpr float kS = 0.84932180028801904272f;      // sqrt(log2(e) / 2)
constexpr float kInvS = 1.17741002251547469101f;   // 1 / kS

__device__ __forceinline__ floatx4 mfma32(bf16x8 a, bf16x8 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma16(short4v a, short4v b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
// bf16 high part (round to nearest) and bf16 residual of two values, each
// converted as a pair (a in the low half)
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float floatx2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split_pk(float a, float b, uint32_t &hi, uint32_t &lo) {
    hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2v{a, b}, bf16x2v));
    const float ah = __uint_as_float(hi << 16), bh = __uint_as_float(hi & 0xffff0000u);
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2v{a - ah, b - bh}, bf16x2v));
}
// split of four values into short4v operands
__device__ __forceinline__ void split4v(float x0, float x1, float x2, float x3, short4v &hi,
                                        short4v &lo) {
    uint32_t h0, l0, h1, l1;
    split_pk(x0, x1, h0, l0);
    split_pk(x2, x3, h1, l1);
    hi = __builtin_bit_cast(short4v, make_uint2(h0, h1));
    lo = __builtin_bit_cast(short4v, make_uint2(l0, l1));
}
// Wait for this wave's outstanding vector-memory operations (the direct
// HBM -> LDS transfers among them).  Issued through the builtin so that the
// compiler's own wait insertion knows the transfers have landed and does not
// add waits of its own before later LDS reads (such a wait would also wait for
// every global store in flight).
template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};
template <int V>
struct IntTag {
    static constexpr int value = V;
};

__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Padding rows after each component's block of DB columns in a column-major
// [column][token] staging array of PITCH floats a row.  The sequential wave's
// lane l holds column (l % JP) DB + (l / JP) % DB: the J components of an
// output dim are DB rows apart, and with DB * PITCH a multiple of 64 floats
// their 16-byte accesses would all start in one bank.  Over paddings 0 .. 15,
// the one with the fewest sequential lanes of a 16-lane group starting in one
// four-bank group (64 banks of 4 bytes), then the fewest of a tile wave's 16
// consecutive columns, then the smallest.
template <int DB, int J, int JP, int N, int PITCH>
constexpr int skew_ways(int x, bool seq) {
    int worst = 0;
    for (int g = 0; g < (seq ? 4 : N / 16); ++g) {
        int cnt[16] = {};
        for (int u = 0; u < 16; ++u) {
            const int l = 16 * g + u, bj = l % JP, bdl = (l / JP) % DB;
            if (seq && (l >= DB * JP || bj >= J)) continue;   // idle lanes: no access of their own
            const int col = seq ? bj * DB + bdl : l;
            const int grp = ((col + x * (col / DB)) * PITCH % 64) / 4;
            worst = ++cnt[grp] > worst ? cnt[grp] : worst;
        }
    }
    return worst;
}
template <int DB, int J, int JP, int N, int PITCH>
constexpr int skew_rows() {
    int best = 0, bs = 64, bt = 64;
    for (int x = 0; x < 16; ++x) {
        const int s = skew_ways<DB, J, JP, N, PITCH>(x, true), t = skew_ways<DB, J, JP, N, PITCH>(x, false);
        if (s < bs || (s == bs && t < bt)) best = x, bs = s, bt = t;
    }
    return best;
}

template <int DK, int J, int DB>
struct PCfg {
    static constexpr int N = J * DB;
    static constexpr int NW = N / 16;
    static constexpr int NT = 64 * (NW + 1);
    static constexpr int NMT = 64 * NW;           // matrix-core threads
    static constexpr int JP = J == 3 ? 4 : J;
    static constexpr int IT = DK / 16;
    static constexpr int NP = N + 4;
    static constexpr int KPC = DK / 8;            // 16-byte pieces per K row
    static constexpr int KPIECES = kC * DK / 8;   // per K (or Q) chunk
    static constexpr int LPIECES = kC * N / 8;    // per logit tensor chunk
    static constexpr int VPIECES = kC * DB / 8;   // v chunk
    static constexpr int PPIECES = kC * N / 4;    // fp32 predictions of a chunk (Newton)
    static_assert(N % 16 == 0 && N <= 64 && DB % 8 == 0, "column block");
    static_assert(DB * JP <= 64, "one sequential wave");
    // rows of the column-major arrays: p and c (kTP floats a row), sq (kC + 2
    // float2), with the padding of skew_rows after each component's block
    static constexpr int XP = skew_rows<DB, J, JP, N, kTP>();
    static constexpr int XS = skew_rows<DB, J, JP, N, 2 * (kC + 2)>();
    static constexpr int NRP = N + J * XP, NRS = N + J * XS;
    __device__ static constexpr int prow(int col) { return col + XP * (col / DB); }
    __device__ static constexpr int srow(int col) { return col + XS * (col / DB); }
};

// MD: 0 exact scan, 1 Newton sweeps (App. D), 2 exact scan of Temporal SwiLA
// (App. B.3).
template <int DK, int J, int DB, int MD>
struct PSmem {
    static constexpr bool NT = MD == 1, TP = MD == 2;
    using C = PCfg<DK, J, DB>;
    uint4 k[kRingKQ][C::KPIECES];
    uint4 q[kRingKQ][C::KPIECES];
    uint4 lb[kRingS][C::LPIECES];
    uint4 lk[kRingS][C::LPIECES];
    uint4 lq[kRingQP][C::LPIECES];
    uint4 v[kRingS][C::VPIECES];
    uint4 pw[NT ? kRingQP : 1][NT ? C::PPIECES : 1];  // Newton: previous sweep's predictions
    uint4 gk[TP ? kRingS : 1][TP ? C::VPIECES : 1];    // temporal: key gate logits, [t][dl]
    uint4 gq[TP ? kRingQP : 1][TP ? C::VPIECES : 1];   // temporal: query gate logits
    union {
        // exact: {beta, log2(e) key-prior logit}, [column][token]; a column's
        // 16 tokens are 128 contiguous bytes, padded so that the sequential
        // wave's 16-byte reads of adjacent columns fall in distinct banks
        alignas(16) float2 sq[2][C::NRS][kC + 2];
        struct {
            float beta[2][kC][C::NP];   // Newton: g (before the clamp)
            float lks[2][kC][C::NP];    // Newton: beta r delta
        };
    };
    alignas(16) float vs[NT ? 1 : 2][DB][kC + 4];   // exact: s v, [dim][token]
    alignas(16) float gs[TP ? 2 : 1][TP ? DB : 1][kC + 4];   // temporal: 1 - g^k, [dim][token]
    float gqs[TP ? 3 : 1][kC][TP ? DB : 1];                  // temporal: g^q, [token][dim]
    float pq[TP ? 3 : 2][kC][C::NP];    // query prior (temporal: the running prior, 3 slots)
    alignas(16) float g[2][kC][kC + 4];    // K_n K_n^T, for the sequential wave
    // chunk-start predictions and coefficients, [C::prow(column)][token]
    // (C::prow(N): the idle lanes' row of c)
    float p[2][C::NRP][kTP];
    float c[2][C::NRP + 1][kTP];
    float r[NT ? 1 : 2][kC][C::NP];  // responsibilities (exact mode)
    float py[2][kC][C::NP];    // pi^q * retrieval
    int flag;                  // Newton: this sweep met the tolerance
    int near;                  // Newton: its change was within 4 tol (the next may be the last)
};

// Four consecutive bf16 (as raw bits) of row t from element i (i % 4 == 0)
// of a row-permuted K or Q tile.
template <int DK>
__device__ __forceinline__ uint2 tile4(const uint4 *tile, int t, int i) {
    constexpr int KPC = DK / 8;
    const int slot = t * KPC + ((i >> 3) ^ (t & (KPC - 1)));
    return reinterpret_cast<const uint2 *>(tile + slot)[(i >> 2) & 1];
}

// Transposed 16 x 16 block of a row-permuted K tile, as the A operand of a
// 16x16x16 matrix-core step: lane (tl, lg) receives K[4 lg + mm][16 it + tl],
// mm = 0..3, from one transposing LDS load.  In each group of 16 lanes the
// load hands lane i element mm of the 8 bytes addressed by lane 4 mm + i / 4
// (element i mod 4), so lane (tl, lg) addresses row 4 lg + tl / 4, key
// indices 16 it + 4 (tl mod 4) .. + 3.
typedef short short4vs __attribute__((__vector_size__(8)));
template <int DK>
__device__ __forceinline__ short4v tile_tr(const uint4 *tile, int it, int tl, int lg) {
    constexpr int KPC = DK / 8;
    const int t = 4 * lg + (tl >> 2), q = tl & 3;
    const int slot = t * KPC + ((2 * it + (q >> 1)) ^ (t & (KPC - 1)));
    const char *p = reinterpret_cast<const char *>(tile + slot) + 8 * (q & 1);
    const short4vs v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) short4vs *)(p));
    return __builtin_bit_cast(short4v, v);
}

// A-operand fragment of rows 0..15 of a K or Q tile for the matrix-core step
// covering key indices [32 s, 32 s + 32) (slot 8 g + m <-> key 32 s + 4 g + m,
// and 32 s + 16 + 4 g + m - 4), or all 16 for Dk = 16.
template <int DK>
__device__ __forceinline__ uint4 frag32(const uint4 *tile, int tl, int lg, int s) {
    const uint2 x0 = tile4<DK>(tile, tl, 32 * s + 4 * lg);
    const uint2 x1 = tile4<DK>(tile, tl, 32 * s + 16 + 4 * lg);
    return make_uint4(x0.x, x0.y, x1.x, x1.y);
}

// One wave-wide HBM -> LDS transfer: lane L moves 16 bytes from src to
// dst + 16 L (dst is the same for the whole wave).  Issued as inline
// assembly so that the compiler does not track it: it would otherwise wait
// for every transfer in flight before any later LDS access it cannot prove
// disjoint, and the transfers could not overlap a chunk's work.  Every wait
// for them is explicit (wait_vm before the barrier that publishes the data).
// lds is the LDS byte address of dst (wave-uniform).  M0 carries it; the
// compiler's value of M0 is saved and restored around the transfer, and
// writing M0 needs one wait state before the transfer reads it.
__device__ __forceinline__ void dma16(const void *src, uint32_t lds) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
        "global_load_lds_dwordx4 %2, off\n\ts_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(__builtin_amdgcn_readfirstlane(lds)), "v"((uint64_t)(uintptr_t)src)
        : "memory");
}

// First transfer index >= base that falls to wave mw in a round-robin deal.
__device__ __forceinline__ int first_for(int base, int mw, int nw) {
    return base + ((mw - base) % nw + nw) % nw;
}

// Issue the HBM -> LDS transfer of chunk m (starting at token t0) into its
// ring slots.  The chunk is cut into wave-wide transfers of 64 x 16 bytes
// (K, Q, the three logit tensors, v), dealt round-robin to the NIW waves that
// do the block's bookkeeping; each tensor has its own loop so its base address
// stays a scalar.
// Tokens past T re-read token T - 1 (in range); the recurrence gives them
// beta = 0.  In Newton mode the chunk's predictions from the previous sweep
// ([kC][N] fp32 at pred + t0 N, the block's workspace) come along.
template <int DK, int J, int DB, int MD, int NIW>
__device__ __forceinline__ void issue_chunk(const LayerArgs &a, PSmem<DK, J, DB, MD> &sm,
                                            uint32_t lds_base, int m, int t0, int b, int h,
                                            int d0, int mw, int lane, const float *pred) {
    constexpr bool NT = MD == 1, TP = MD == 2;
    // LDS byte address of a destination inside sm
    auto at = [&](const uint4 *dst) {
        return lds_base + (uint32_t)(reinterpret_cast<const char *>(dst) -
                                     reinterpret_cast<const char *>(&sm));
    };
    const int skq = m % kRingKQ, sqp = m % kRingQP, ss = m % kRingS;
    using C = PCfg<DK, J, DB>;
    const int T = a.T, H = a.H, Dv = a.Dv;
    constexpr int nk = (C::KPIECES + 63) / 64, nl = (C::LPIECES + 63) / 64;
    constexpr int nv = (C::VPIECES + 63) / 64;
    if (t0 + kC <= T) {
        // Whole chunk in range: a scalar base per tensor (row t0 of this head)
        // plus a 32-bit per-lane byte offset.
        const size_t row0 = ((size_t)b * T + t0) * H + h;
        // K and Q rows: piece p of row t goes to slot p ^ (t mod pieces)
        auto kq = [&](const void *base, uint4 *tile, int ibase) {
            const char *src = static_cast<const char *>(base) + row0 * DK * 2;
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nk; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::KPIECES) {
                    const int t = s / C::KPC, p = s % C::KPC, gp = p ^ (t & (C::KPC - 1));
                    dma16(src + (uint32_t)(t * H * DK * 2 + 16 * gp), at(tile + part * 64));
                }
            }
        };
        // logits, [t][j][dl]
        auto logit = [&](const void *base, uint4 *dstv, int ibase) {
            const char *src = static_cast<const char *>(base) + (row0 * J * Dv + d0) * 2;
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nl; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::LPIECES) {
                    const int t = s / (C::N / 8), rem = s % (C::N / 8);
                    const int j = rem / (DB / 8), qd = rem % (DB / 8);
                    dma16(src + (uint32_t)((t * H * J + j) * Dv * 2 + 16 * qd), at(dstv + part * 64));
                }
            }
        };
        kq(a.k, sm.k[skq], 0);
        kq(a.q, sm.q[skq], nk);
        logit(a.lb, sm.lb[ss], 2 * nk);
        logit(a.lk, sm.lk[ss], 2 * nk + nl);
        logit(a.lq, sm.lq[sqp], 2 * nk + 2 * nl);
        // [t][dl] tensors of one value per (token, output dim): v, and the gates
        auto vrow = [&](const void *base, uint4 *dstv, int ibase) {
            const char *src = static_cast<const char *>(base) + (row0 * Dv + d0) * 2;
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nv; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::VPIECES) {
                    const int t = s / (DB / 8), qd = s % (DB / 8);
                    dma16(src + (uint32_t)(t * H * Dv * 2 + 16 * qd), at(dstv + part * 64));
                }
            }
        };
        vrow(a.v, sm.v[ss], 2 * nk + 3 * nl);
        if constexpr (TP) {
            vrow(a.gk, sm.gk[ss], 2 * nk + 3 * nl + nv);
            vrow(a.gq, sm.gq[sqp], 2 * nk + 3 * nl + 2 * nv);
        }
    } else {
        const size_t row0 = (size_t)b * T;
        // K and Q rows: piece p of row t goes to slot p ^ (t mod pieces)
        auto kq = [&](const void *base, uint4 *tile, int ibase) {
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nk; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::KPIECES) {
                    const int t = s / C::KPC, p = s % C::KPC;
                    const int tc = min(t0 + t, T - 1);
                    const int gp = p ^ (t & (C::KPC - 1));
                    dma16(static_cast<const uint16_t *>(base) + ((row0 + tc) * H + h) * DK + 8 * gp,
                          at(tile + part * 64));
                }
            }
        };
        // logits, [t][j][dl]
        auto logit = [&](const void *base, uint4 *dstv, int ibase) {
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nl; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::LPIECES) {
                    const int t = s / (C::N / 8), rem = s % (C::N / 8);
                    const int j = rem / (DB / 8), qd = rem % (DB / 8);
                    const int tc = min(t0 + t, T - 1);
                    dma16(static_cast<const uint16_t *>(base) +
                              (((row0 + tc) * H + h) * J + j) * Dv + d0 + 8 * qd,
                          at(dstv + part * 64));
                }
            }
        };
        kq(a.k, sm.k[skq], 0);
        kq(a.q, sm.q[skq], nk);
        logit(a.lb, sm.lb[ss], 2 * nk);
        logit(a.lk, sm.lk[ss], 2 * nk + nl);
        logit(a.lq, sm.lq[sqp], 2 * nk + 2 * nl);
        auto vrow = [&](const void *base, uint4 *dstv, int ibase) {
            for (int ins = first_for(ibase, mw, NIW); ins < ibase + nv; ins += NIW) {
                const int part = ins - ibase, s = part * 64 + lane;
                if (s < C::VPIECES) {
                    const int t = s / (DB / 8), qd = s % (DB / 8);
                    const int tc = min(t0 + t, T - 1);
                    dma16(static_cast<const uint16_t *>(base) + ((row0 + tc) * H + h) * Dv + d0 +
                              8 * qd,
                          at(dstv + part * 64));
                }
            }
        };
        vrow(a.v, sm.v[ss], 2 * nk + 3 * nl);
        if constexpr (TP) {
            vrow(a.gk, sm.gk[ss], 2 * nk + 3 * nl + nv);
            vrow(a.gq, sm.gq[sqp], 2 * nk + 3 * nl + 2 * nv);
        }
    }
    if constexpr (NT) {
        constexpr int ib = 2 * nk + 3 * nl + nv, np = (C::PPIECES + 63) / 64;
        for (int ins = first_for(ib, mw, NIW); ins < ib + np; ins += NIW) {
            const int part = ins - ib, s = part * 64 + lane;
            if (s < C::PPIECES) dma16(pred + (size_t)t0 * C::N + 4 * s, at(sm.pw[sqp] + part * 64));
        }
    }
}

// Four consecutive bf16 elements (idx % 4 == 0) of an LDS tile, widened.
__device__ __forceinline__ float4 bf16x4_at(const uint4 *base, int idx) {
    const uint2 u = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(base) + idx);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}
// L consecutive bf16 (L in {1, 2, 4}, element index aligned to L) of an LDS
// tile, widened; L consecutive floats loaded or stored (aligned to L); L
// floats rounded to bf16 and stored.
template <int L>
__device__ __forceinline__ void bf16_row(const uint4 *base, int idx, float (&x)[L]) {
    const uint16_t *p = reinterpret_cast<const uint16_t *>(base) + idx;
    if constexpr (L == 4) {
        const uint2 u = *reinterpret_cast<const uint2 *>(p);
        x[0] = __uint_as_float(u.x << 16), x[1] = __uint_as_float(u.x & 0xffff0000u);
        x[2] = __uint_as_float(u.y << 16), x[3] = __uint_as_float(u.y & 0xffff0000u);
    } else if constexpr (L == 2) {
        const uint32_t u = *reinterpret_cast<const uint32_t *>(p);
        x[0] = __uint_as_float(u << 16), x[1] = __uint_as_float(u & 0xffff0000u);
    } else {
        x[0] = __uint_as_float((uint32_t)p[0] << 16);
    }
}
template <int L>
__device__ __forceinline__ void f32_load(const float *p, float (&x)[L]) {
    if constexpr (L == 4) {
        const float4 v = *reinterpret_cast<const float4 *>(p);
        x[0] = v.x, x[1] = v.y, x[2] = v.z, x[3] = v.w;
    } else if constexpr (L == 2) {
        const float2 v = *reinterpret_cast<const float2 *>(p);
        x[0] = v.x, x[1] = v.y;
    } else {
        x[0] = p[0];
    }
}
template <int L>
__device__ __forceinline__ void f32_row(float *p, const float (&x)[L]) {
    if constexpr (L == 4)
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    else if constexpr (L == 2)
        *reinterpret_cast<float2 *>(p) = make_float2(x[0], x[1]);
    else
        p[0] = x[0];
}
template <int L>
__device__ __forceinline__ void bf16_store(uint16_t *p, const float (&x)[L]) {
    typedef __bf16 bf16v __attribute__((ext_vector_type(L)));
    typedef float f32v __attribute__((ext_vector_type(L)));
    f32v f;
#pragma unroll
    for (int u = 0; u < L; ++u) f[u] = x[u];
    const bf16v hv = __builtin_convertvector(f, bf16v);
    if constexpr (L == 4)
        *reinterpret_cast<uint2 *>(p) = __builtin_bit_cast(uint2, hv);
    else if constexpr (L == 2)
        *reinterpret_cast<uint32_t *>(p) = __builtin_bit_cast(uint32_t, hv);
    else
        p[0] = __builtin_bit_cast(uint16_t, hv);
}

// Same block-to-(head, column block) map as the chunk scan: every column block
// of a head on one XCD when the head count is a multiple of 8.
__device__ __forceinline__ void pipe_coords(int id, int ndb, int nheads, int &db, int &head) {
    if (nheads % 8 == 0) {
        const int xcd = id % 8, k = id / 8;
        head = xcd + 8 * (k / ndb);
        db = k % ndb;
    } else {
        head = id / ndb;
        db = id % ndb;
    }
}

// LDS (over 60 KB a block) allows at most two blocks on a compute unit, so at
// most two waves share a SIMD: the compiler may use every register for that.
template <int DK, int J, int DB, int MD, int NH>
__global__ __launch_bounds__(512)
void scan_pipe_kernel(LayerArgs a, NewtonArgs na) {
    using C = PCfg<DK, J, DB>;
    constexpr int IT = C::IT, N = C::N, NW = C::NW, JP = C::JP;
    constexpr bool NT = MD == 1, TP = MD == 2;
    __shared__ PSmem<DK, J, DB, MD> sm;
    const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) void *)&sm;

    const int tid = threadIdx.x;
    // the wave index, as a scalar: role branches and transfer slots stay scalar
    const int w = __builtin_amdgcn_readfirstlane(tid / 64), lane = tid % 64;
    const int tl = lane % 16, lg = lane / 16;
    const int H = a.H, T = a.T, Dv = a.Dv;
    int db, hh;
    pipe_coords(blockIdx.x, Dv / DB, a.B * H, db, hh);
    const int d0 = db * DB, h = hh % H, b = hh / H;
    const int NCH = (T + kC - 1) / kC;
    const bool seq = (w == NW);
    // Roles: waves 0 .. NW-1 hold the state tiles (matrix-core products);
    // wave NW is the sequential wave; with NH > 0, waves NW+1 .. NW+NH do the
    // per-chunk bookkeeping (transfers, priors, input prep, outputs), which the
    // tile waves do themselves when NH = 0.
    const bool tile = w < NW;
    const bool book = NH == 0 ? tile : w > NW;        // this wave does the bookkeeping
    constexpr int NBW = NH == 0 ? NW : NH;            // bookkeeping waves
    constexpr int NBT = 64 * NBW;                     // bookkeeping threads
    const int bw = NH == 0 ? w : w - (NW + 1);        // index among them
    // The compiler cannot bound bt (the wave index comes from readfirstlane), so
    // loops strided by NBT count 0 .. ceil(n / NBT) from bt and stop at n: a
    // trip count it can see, and fully unrolled loops.
    const int bt = 64 * bw + lane;
    // The loops below deal n items over the NBT bookkeeping threads; when n is
    // not a multiple of NBT the first threads take one item more.  Each loop
    // starts its deal at a different bookkeeping wave (brot(k)), so those extra
    // items fall on different waves.  (Called only by bookkeeping threads, for
    // which 0 <= bt < NBT.)
    auto brot = [&](int k) { return (bt + (k % NBW) * 64) % NBT; };
    // the wave that forms the Gram matrix of the next chunk for the sequential wave
    const bool gwave = NH == 0 ? w == 1 % NW : w == NW + 1;
    // Newton mode: this block's predictions, [NCH * kC][N] fp32
    float *const pred = NT ? na.pred + ((size_t)hh * (Dv / DB) + db) * NCH * kC * N : nullptr;
    // Newton mode: only the last sweep's outputs are kept, so a sweep forms the
    // query side (Q S, the retrieval product, pi^q, the output stores) only when
    // it can be the last: the max_iters-th sweep, or one that follows a sweep
    // whose change was within 4 tol.  A sweep that meets tol without it is
    // followed by one more that has it.  Every role reads the sequential wave's
    // verdict after the sweep's last barrier and takes the same decision.
    auto next_sweep = [&](int sweeps, bool &qs, bool &done) {
        const bool met = sm.flag != 0, near = sm.near != 0;
        done = (met && qs) || sweeps >= na.max_iters;
        qs = near || met || sweeps + 1 >= na.max_iters;
    };

    // ---- matrix-core wave state: W^T tile rows 16 it + 4 lg + r, column col
    const int col = 16 * (seq ? 0 : w) + tl;
    const int jc = col / DB, dc = d0 + col % DB;
    const size_t sbase = (((size_t)b * H + h) * J + jc) * DK * Dv + dc;
    floatx4 W[IT];
    // Exact mode keeps the state, and with it every product the sequential wave
    // consumes (predictions, coefficients), in the scaled units s = sqrt(log2(e)/2)
    // of its recurrence, so that the critical path carries no conversions; the
    // state is converted on the way in and out, the retrieval by the query prior.
    constexpr float kWS = NT ? 1.f : kS, kInvWS = NT ? 1.f : kInvS;
    auto load_state = [&]() {
#pragma unroll
        for (int it = 0; it < IT; ++it) W[it] = floatx4{0.f, 0.f, 0.f, 0.f};
        if (tile && a.state_in) {
            // Newton mode reloads W_0 every sweep: an opaque copy of the row
            // stride keeps the compiler from holding all IT * 4 addresses in
            // registers across the sweeps.
            int dv = Dv;
            asm volatile("" : "+s"(dv));
            const float *src = a.state_in + sbase + (size_t)(4 * lg) * dv;
#pragma unroll
            for (int it = 0; it < IT; ++it)
#pragma unroll
                for (int r = 0; r < 4; ++r) W[it][r] = kWS * src[(size_t)(16 * it + r) * dv];
        }
    };
    load_state();
    floatx4 Yacc = {0.f, 0.f, 0.f, 0.f}, Xacc = Yacc;
    short4v chi = {0, 0, 0, 0}, clo = chi, ghi = chi, glo = chi;

    // ---- sequential wave identity: lanes of one output dim are adjacent
    const int sl = lane;
    const int bdl = (sl / JP) % DB, bj = sl % JP;
    const bool bact = seq && sl < DB * JP && bj < J;
    const bool bpad = seq && sl < DB * JP && bj >= J;   // padding component (J = 3)
    // Backward support (exact mode): with delta_out the per-token LDS ring that
    // carries r for resp carries delta instead, to delta_out, and the tile waves
    // store the state every second chunk to ckpt.
    const bool dmode = MD == 0 && a.delta_out != nullptr;
    float *const rdst = dmode ? a.delta_out : a.resp;
    const bool want_r = rdst != nullptr;   // (the temporal form always keeps r)
    const int bcol = bact ? bj * DB + bdl : 0;
    const int bsto = bact ? bcol : N;

    // split of the state tile into bf16 (hi, lo) B operands, per k-step
    auto split_state = [&](bf16x8 (&whi)[IT / 2 > 0 ? IT / 2 : 1],
                           bf16x8 (&wlo)[IT / 2 > 0 ? IT / 2 : 1], short4v &w16hi,
                           short4v &w16lo) {
        if constexpr (DK == 16) {
            split4v(W[0][0], W[0][1], W[0][2], W[0][3], w16hi, w16lo);
        } else {
#pragma unroll
            for (int s = 0; s < DK / 32; ++s) {
                // elements m = 0..3 from W[2 s], 4..7 from W[2 s + 1]
                uint32_t h[4], l[4];
                split_pk(W[2 * s][0], W[2 * s][1], h[0], l[0]);
                split_pk(W[2 * s][2], W[2 * s][3], h[1], l[1]);
                split_pk(W[2 * s + 1][0], W[2 * s + 1][1], h[2], l[2]);
                split_pk(W[2 * s + 1][2], W[2 * s + 1][3], h[3], l[3]);
                whi[s] = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
                wlo[s] = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
            }
        }
    };
    // acc += (rows of tile) x S, with S split as above
    auto tile_times_state = [&](const uint4 *tile, floatx4 acc, const bf16x8 (&whi)[IT / 2 > 0 ? IT / 2 : 1],
                                const bf16x8 (&wlo)[IT / 2 > 0 ? IT / 2 : 1], short4v w16hi,
                                short4v w16lo) {
        if constexpr (DK == 16) {
            const uint2 x = tile4<DK>(tile, tl, 4 * lg);
            const short4v av = __builtin_bit_cast(short4v, x);
            acc = mfma16(av, w16hi, acc);
            acc = mfma16(av, w16lo, acc);
        } else {
#pragma unroll
            for (int s = 0; s < DK / 32; ++s) {
                const bf16x8 av = __builtin_bit_cast(bf16x8, frag32<DK>(tile, tl, lg, s));
                acc = mfma32(av, whi[s], acc);
                acc = mfma32(av, wlo[s], acc);
            }
        }
        return acc;
    };
    // rows(x) . rows(y)^T for two 16-row tiles (Gram-type product), exact products
    auto gram = [&](const uint4 *x, const uint4 *y) {
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
        if constexpr (DK == 16) {
            const short4v ax = __builtin_bit_cast(short4v, tile4<DK>(x, tl, 4 * lg));
            const short4v ay = __builtin_bit_cast(short4v, tile4<DK>(y, tl, 4 * lg));
            acc = mfma16(ax, ay, acc);
        } else {
#pragma unroll
            for (int s = 0; s < DK / 32; ++s) {
                const bf16x8 ax = __builtin_bit_cast(bf16x8, frag32<DK>(x, tl, lg, s));
                const bf16x8 ay = __builtin_bit_cast(bf16x8, frag32<DK>(y, tl, lg, s));
                acc = mfma32(ax, ay, acc);
            }
        }
        return acc;
    };
    // Per-chunk bookkeeping works on groups of four consecutive columns (or
    // output dims), so that every thread makes one round trip to LDS.
    // Work per (t, dl) over the J components (priors, outputs, Newton
    // linearisation) is spread over every matrix-core thread: PE consecutive
    // output dims per thread.
    constexpr int PE = J == 1 ? 4 : J == 2 ? 2 : 1;
    constexpr int NPG = kC * DB / PE;   // (t, dl) groups per chunk
    // When the groups fill at most half of the threads (J = 8), the query
    // prior takes the first half and the outputs the second.
    constexpr int OUT0 = 2 * NPG <= NBT ? NBT - NPG : 0;
    // derived inputs of chunk m (parity pr) for the sequential wave
    auto prep_seq_inputs = [&](int m, int pr) {
        const int rs = m % kRingS;
        if constexpr (TP) {
            // Temporal (App. B.3), per (t, dl) over the J components: beta,
            // g^k pi^k (pi^k = softmax_j of the key-prior logits) and 1 - g^k for
            // the key prior (1 - g^k) r_{t-1} + g^k pi^k the sequential wave
            // forms; padded tokens carry no mass and keep r_{t-1}.
#pragma unroll
            for (int i_ = 0; i_ < ceil_div(NPG, NBT); ++i_) {
                const int gi = brot(0) + i_ * NBT;
                if (gi >= NPG) break;
                const int e = PE * gi, t = e / DB, dl = e % DB;
                const bool ok = m * kC + t < T;
                float lbj[J][PE], lkj[J][PE], mk[PE], zk[PE], gv[PE], vv[PE];
                bf16_row<PE>(sm.gk[rs], e, gv);
                bf16_row<PE>(sm.v[rs], e, vv);
#pragma unroll
                for (int u = 0; u < PE; ++u) mk[u] = -INFINITY, zk[u] = 0.f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    bf16_row<PE>(sm.lb[rs], t * N + j * DB + dl, lbj[j]);
                    bf16_row<PE>(sm.lk[rs], t * N + j * DB + dl, lkj[j]);
#pragma unroll
                    for (int u = 0; u < PE; ++u) mk[u] = fmaxf(mk[u], lkj[j][u]);
                }
#pragma unroll
                for (int j = 0; j < J; ++j)
#pragma unroll
                    for (int u = 0; u < PE; ++u) {
                        lkj[j][u] = exp_fast(lkj[j][u] - mk[u]);
                        zk[u] += lkj[j][u];
                    }
#pragma unroll
                for (int u = 0; u < PE; ++u) {
                    const float g = ok ? sigmoid(gv[u]) : 0.f;
                    const float gz = g * rcp_fast(zk[u]);
#pragma unroll
                    for (int j = 0; j < J; ++j)
                        sm.sq[pr][C::srow(j * DB + dl + u)][t] =
                            make_float2(ok ? sigmoid(lbj[j][u]) : 0.f, gz * lkj[j][u]);
                    sm.gs[pr][dl + u][t] = 1.f - g;
                    sm.vs[pr][dl + u][t] = kS * vv[u];
                }
            }
        } else if constexpr (!NT) {
#pragma unroll
          for (int i_ = 0; i_ < ceil_div(kC * N / 4, NBT); ++i_) {
            const int g4 = brot(0) + i_ * NBT;
            if (g4 >= kC * N / 4) break;
            // four consecutive columns (dims dl .. dl+3 of one component) of token
            // t.  Item g4 = 16 a + i takes token i and column group (a + i) mod
            // N/4: the 16 lanes of a group then read 16 distinct bank pairs of
            // the logit rows and store to 16 distinct bank pairs of sq (a plain
            // row-major deal put them on two).
            const int t = g4 % kC, cc = 4 * ((g4 / kC + t) % (N / 4)), e4 = t * N + cc;
            const bool ok = m * kC + t < T;
            float lbv[4], lkv[4];
            bf16_row<4>(sm.lb[rs], e4, lbv);
            bf16_row<4>(sm.lk[rs], e4, lkv);
#pragma unroll
            for (int u = 0; u < 4; ++u)
                sm.sq[pr][C::srow(cc + u)][t] = make_float2(ok ? sigmoid(lbv[u]) : 0.f, lkv[u] * kLog2e);
          }
#pragma unroll
          for (int i_ = 0; i_ < ceil_div(kC * DB / 4, NBT); ++i_) {
            const int g4 = brot(1) + i_ * NBT;
            if (g4 >= kC * DB / 4) break;
                const int e4 = 4 * g4;
                float vv[4];
                bf16_row<4>(sm.v[rs], e4, vv);
#pragma unroll
                for (int u = 0; u < 4; ++u) sm.vs[pr][e4 % DB + u][e4 / DB] = kS * vv[u];
          }
        } else {
            // Linearisation around the previous sweep's predictions (App. D.2),
            // per (t, dl) over the J components: delta, r (eq. responsibility),
            // g (eq. jacobian_coeff) and the part beta r delta of the effective
            // input (eq. effective_input); the sequential wave adds g pred^(i).
            const float *po = reinterpret_cast<const float *>(sm.pw[m % kRingQP]);
#pragma unroll
            for (int i_ = 0; i_ < ceil_div(NPG, NBT); ++i_) {
            const int gi = brot(0) + i_ * NBT;
            if (gi >= NPG) break;
                const int e = PE * gi, t = e / DB, dl = e % DB;
                const bool ok = m * kC + t < T;
                float vv[PE];
                bf16_row<PE>(sm.v[rs], e, vv);
                float dj[J][PE], xj[J][PE], lka[J][PE], mx[PE], z[PE];
#pragma unroll
                for (int u = 0; u < PE; ++u) mx[u] = -INFINITY, z[u] = 0.f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    float pj[PE];
                    f32_load<PE>(po + t * N + j * DB + dl, pj);
                    bf16_row<PE>(sm.lk[rs], t * N + j * DB + dl, lka[j]);
#pragma unroll
                    for (int u = 0; u < PE; ++u) {
                        dj[j][u] = vv[u] - pj[u];
                        xj[j][u] = kLog2e * fmaf(-0.5f * dj[j][u], dj[j][u], lka[j][u]);
                        mx[u] = fmaxf(mx[u], xj[j][u]);
                    }
                }
                if (na.unnorm) {
                    // App. D.2's variant: r = pi^k e^{-delta^2/2} with no
                    // normaliser, pi^k = softmax_j of the logits; the exponent
                    // log2(e) (lk - max lk - delta^2/2) is at most 0
#pragma unroll
                    for (int u = 0; u < PE; ++u) mx[u] = -INFINITY;
#pragma unroll
                    for (int j = 0; j < J; ++j)
#pragma unroll
                        for (int u = 0; u < PE; ++u) mx[u] = fmaxf(mx[u], lka[j][u]);
#pragma unroll
                    for (int j = 0; j < J; ++j)
#pragma unroll
                        for (int u = 0; u < PE; ++u) {
                            z[u] += exp_fast(lka[j][u] - mx[u]);
                            xj[j][u] = __builtin_amdgcn_exp2f(fmaf(-kLog2e, mx[u], xj[j][u]));
                        }
                } else {
#pragma unroll
                    for (int j = 0; j < J; ++j)
#pragma unroll
                        for (int u = 0; u < PE; ++u) {
                            xj[j][u] = __builtin_amdgcn_exp2f(xj[j][u] - mx[u]);
                            z[u] += xj[j][u];
                        }
                }
#pragma unroll
                for (int u = 0; u < PE; ++u) z[u] = rcp_fast(z[u]);
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    float lbj[PE], gv[PE], bv[PE];
                    bf16_row<PE>(sm.lb[rs], t * N + j * DB + dl, lbj);
#pragma unroll
                    for (int u = 0; u < PE; ++u) {
                        const float r = xj[j][u] * z[u];
                        const float br = sigmoid(lbj[u]) * r;
                        const float d = dj[j][u];
                        // eq. jacobian_coeff; the variant's exact coefficient drops
                        // the factor 1 - r that the normaliser contributes
                        const float c1 = na.unnorm ? 1.f : 1.f - r;
                        gv[u] = ok ? br * fmaf(-d * d, c1, 1.f) : 0.f;
                        bv[u] = ok ? br * d : 0.f;
                    }
                    f32_row<PE>(&sm.beta[pr][t][j * DB + dl], gv);
                    f32_row<PE>(&sm.lks[pr][t][j * DB + dl], bv);
                }
            }
        }
    };
    // pi^q of chunk m: softmax over j of the query-prior logits, per (t, dl)
    auto prep_query_prior = [&](int m, int pr) {
        const int rs = m % kRingQP;
        // temporal: pi^q itself (the scan below forms rhobar and scales it)
        constexpr float kQS = TP ? 1.f : kInvWS;
#pragma unroll
        for (int i_ = 0; i_ < ceil_div(NPG, NBT); ++i_) {
            const int gi = (OUT0 ? bt : brot(2)) + i_ * NBT;
            if (gi >= NPG) break;
            const int e = PE * gi, t = e / DB, dl = e % DB;
            float x[J][PE], mq[PE], z[PE];
#pragma unroll
            for (int u = 0; u < PE; ++u) mq[u] = -INFINITY, z[u] = 0.f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                bf16_row<PE>(sm.lq[rs], t * N + j * DB + dl, x[j]);
#pragma unroll
                for (int u = 0; u < PE; ++u) mq[u] = fmaxf(mq[u], x[j][u]);
            }
#pragma unroll
            for (int j = 0; j < J; ++j)
#pragma unroll
                for (int u = 0; u < PE; ++u) {
                    x[j][u] = exp_fast(x[j][u] - mq[u]);
                    z[u] += x[j][u];
                }
#pragma unroll
            for (int u = 0; u < PE; ++u) z[u] = kQS * rcp_fast(z[u]);
#pragma unroll
            for (int j = 0; j < J; ++j) {
#pragma unroll
                for (int u = 0; u < PE; ++u) x[j][u] *= z[u];
                f32_row<PE>(&sm.pq[pr][t][j * DB + dl], x[j]);
            }
            if constexpr (TP) {
                float gv[PE];
                bf16_row<PE>(sm.gq[rs], e, gv);
#pragma unroll
                for (int u = 0; u < PE; ++u) sm.gqs[pr][t][dl + u] = sigmoid(gv[u]);
            }
        }
    };
    // Temporal: the running query prior rhobar_t = (1 - g^q_t) rhobar_{t-1} +
    // g^q_t pi^q_t (App. B.3) over chunk m, one bookkeeping thread per column
    // (the last N of them, which have the least other work), carried in rho from
    // chunk to chunk; written in place of pi^q (scaled like the plain prior).
    // Padded tokens leave it unchanged.  All loads first, then the 16 dependent
    // steps in registers, then the stores.
    const int qc = bt - (NBT - N);   // this thread's column in the scan, if >= 0
    float rho = 1.f / J;
    if constexpr (TP) {
        if (book && qc >= 0 && a.prior_in)
            rho = a.prior_in[(((size_t)b * H + h) * 2 * J + J + qc / DB) * Dv + d0 + qc % DB];
    }
    auto scan_query_prior = [&](int m) {
        if (qc >= 0) {
            const int slot = m % 3, dl = qc % DB;
            float pi[kC], g[kC];
#pragma unroll
            for (int t = 0; t < kC; ++t) pi[t] = sm.pq[slot][t][qc], g[t] = sm.gqs[slot][t][dl];
            const int nt = T - m * kC;   // tokens of this chunk in range
#pragma unroll
            for (int t = 0; t < kC; ++t) {
                if (t < nt) rho = fmaf(g[t], pi[t] - rho, rho);
                pi[t] = kInvWS * rho;
            }
#pragma unroll
            for (int t = 0; t < kC; ++t) sm.pq[slot][t][qc] = pi[t];
        }
    };
    // o of chunk m: sum over j of pi^q * retrieval
    auto store_output = [&](int m, int pr) {
        if (!a.o) return;   // (the backward's recompute keeps no output)
#pragma unroll
        for (int i_ = 0; i_ < ceil_div(NPG, NBT); ++i_) {
            const int gi = (OUT0 ? bt - OUT0 : brot(1)) + i_ * NBT;
            if (gi < 0 || gi >= NPG) break;   // gi < 0: a thread of the query-prior half
            const int e = PE * gi, t = e / DB, dl = e % DB;
            if (m * kC + t < T) {
                float o[PE], y[PE];
#pragma unroll
                for (int u = 0; u < PE; ++u) o[u] = 0.f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    f32_load<PE>(&sm.py[pr][t][j * DB + dl], y);
#pragma unroll
                    for (int u = 0; u < PE; ++u) o[u] += y[u];
                }
                const size_t idx = (((size_t)b * T + m * kC + t) * H + h) * Dv + d0 + dl;
                if (a.out_bf16)
                    bf16_store<PE>(static_cast<uint16_t *>(a.o) + idx, o);
                else
                    f32_row<PE>(static_cast<float *>(a.o) + idx, o);
            }
        }
    };
    auto store_resp = [&](int m, int pr) {
        if constexpr (!NT) {
#pragma unroll
          for (int i_ = 0; i_ < ceil_div(kC * N / 4, NBT); ++i_) {
            const int g4 = brot(2) + i_ * NBT;
            if (g4 >= kC * N / 4) break;
            const int e4 = 4 * g4, t = e4 / N, cc = e4 % N;
            if (m * kC + t < T)
                *reinterpret_cast<float4 *>(
                    rdst + ((((size_t)b * T + m * kC + t) * H + h) * J + cc / DB) * Dv + d0 +
                    cc % DB) = *reinterpret_cast<const float4 *>(&sm.r[pr][t][cc]);
          }
        }
    };
    // Backward support: the state before chunk 2 m, unscaled, into
    // ckpt [B, H, ceil(T / 32), Dv, J, Dk] (rows 16 it + 4 lg .. + 3 of column col)
    auto store_ckpt = [&](int m) {
        static_assert(kBwdChunk == 2 * kC, "checkpoints every second chunk");
        const int NC2 = (T + 2 * kC - 1) / (2 * kC);
        float *dst = a.ckpt + ((((size_t)b * H + h) * NC2 + m) * Dv + dc) * J * DK +
                     (size_t)jc * DK + 4 * lg;
#pragma unroll
        for (int it = 0; it < IT; ++it)
            *reinterpret_cast<float4 *>(dst + 16 * it) =
                make_float4(kInvWS * W[it][0], kInvWS * W[it][1], kInvWS * W[it][2],
                            kInvWS * W[it][3]);
    };
    // W += K_m^T C_m and Y += tril(A_m) C_m (C_m split in chi/clo); then
    // stage pi^q * Y of chunk m
    auto finish_chunk = [&](int m, bool qs) {
        const int rs = m % kRingKQ, pr = m & 1;
#pragma unroll
        for (int it = 0; it < IT; ++it) {
            // A operand K^T: lane (tl, lg) needs K[4 lg + mm][16 it + tl], mm = 0..3
            const short4v ak = tile_tr<DK>(sm.k[rs], it, tl, lg);
            W[it] = mfma16(ak, chi, W[it]);
            W[it] = mfma16(ak, clo, W[it]);
        }
        if (!qs) return;   // (Newton: a sweep without the query side)
        // (K_m Q_m^T)[s][t] in accumulator layout is lane (t = tl, s = 4 lg + r):
        // exactly the A operand of tril(A_m) C_m, A_m = Q_m K_m^T
        const floatx4 at = gram(sm.k[rs], sm.q[rs]);
        short4v ahi, alo;
        split4v(4 * lg <= tl ? at[0] : 0.f, 4 * lg + 1 <= tl ? at[1] : 0.f,
                4 * lg + 2 <= tl ? at[2] : 0.f, 4 * lg + 3 <= tl ? at[3] : 0.f, ahi, alo);
        Yacc = mfma16(ahi, chi, Yacc);
        Yacc = mfma16(ahi, clo, Yacc);
        Yacc = mfma16(alo, chi, Yacc);
#pragma unroll
        for (int r = 0; r < 4; ++r)
            sm.py[pr][4 * lg + r][col] = Yacc[r] * sm.pq[TP ? m % 3 : pr][4 * lg + r][col];
    };

    if constexpr (NT) {
        // Iterate 0 (the initial guess w_t = W_0 for every t): pred_t = k_t . W_0,
        // straight from HBM rows of K, chunk by chunk.
        if (tile) {
            bf16x8 whi[IT / 2 > 0 ? IT / 2 : 1], wlo[IT / 2 > 0 ? IT / 2 : 1];
            short4v w16hi, w16lo;
            split_state(whi, wlo, w16hi, w16lo);
            const uint16_t *kb = static_cast<const uint16_t *>(a.k);
            for (int n = 0; n < NCH; ++n) {
                const int tc = min(n * kC + tl, T - 1);
                const uint16_t *row = kb + (((size_t)b * T + tc) * H + h) * DK;
                floatx4 acc = {0.f, 0.f, 0.f, 0.f};
                if constexpr (DK == 16) {
                    const short4v av =
                        __builtin_bit_cast(short4v, *reinterpret_cast<const uint2 *>(row + 4 * lg));
                    acc = mfma16(av, w16hi, acc);
                    acc = mfma16(av, w16lo, acc);
                } else {
#pragma unroll
                    for (int s = 0; s < DK / 32; ++s) {
                        const uint2 x0 = *reinterpret_cast<const uint2 *>(row + 32 * s + 4 * lg);
                        const uint2 x1 = *reinterpret_cast<const uint2 *>(row + 32 * s + 16 + 4 * lg);
                        const bf16x8 av = __builtin_bit_cast(bf16x8, make_uint4(x0.x, x0.y, x1.x, x1.y));
                        acc = mfma32(av, whi[s], acc);
                        acc = mfma32(av, wlo[s], acc);
                    }
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) pred[(size_t)(n * kC + 4 * lg + r) * N + col] = acc[r];
            }
            wait_vm();   // stores done before any wave reads them back
        }
        block_sync_lds();
    }

    // The two roles run separate loops with the same barriers, so that the
    // sequential wave's registers and the matrix-core waves' do not add up.
    if (seq) {
        int sweeps = 0;
        bool done = false, qs = na.max_iters <= 1;
        while (!done) {
            ++sweeps;
            float dmax = 0.f, pmax = 0.f;   // Newton: largest change, largest prediction
            // Exact mode: the per-token inputs of the next chunk and the first row
            // of its Gram matrix, read while the matrix-core waves form its
            // predictions (between the two barriers), off the critical path.
            // Temporal: lkvN holds g^k pi^k and gsN 1 - g^k of the key prior
            // (1 - g^k) r_{t-1} + g^k pi^k (App. B.3); rprev is r_{t-1} of this
            // lane's column, carried from chunk to chunk.
            float vvN[kC], lkvN[kC], bevN[kC], growN[kC], gsN[TP ? kC : 1];
            float rprev = 0.f;
            if constexpr (TP) {
                if (bact)
                    rprev = a.prior_in ? a.prior_in[(((size_t)b * H + h) * 2 * J + bj) * Dv + d0 + bdl]
                                       : 1.f / J;
            }
            auto fetch_inputs = [&](int prn) {
                // 16-byte reads: few enough to be in flight together
                const float4 *sq4 = reinterpret_cast<const float4 *>(sm.sq[prn][C::srow(bcol)]);
                const float4 *vs4 = reinterpret_cast<const float4 *>(sm.vs[prn][bdl]);
                const float4 *g4 = reinterpret_cast<const float4 *>(sm.g[prn][0]);
#pragma unroll
                for (int i = 0; i < kC / 2; ++i) {
                    const float4 x = sq4[i];
                    bevN[2 * i] = x.x, lkvN[2 * i] = x.y, bevN[2 * i + 1] = x.z, lkvN[2 * i + 1] = x.w;
                }
#pragma unroll
                for (int i = 0; i < kC / 4; ++i) {
                    const float4 x = vs4[i], y = g4[i];
                    vvN[4 * i] = x.x, vvN[4 * i + 1] = x.y, vvN[4 * i + 2] = x.z, vvN[4 * i + 3] = x.w;
                    growN[4 * i] = y.x, growN[4 * i + 1] = y.y, growN[4 * i + 2] = y.z, growN[4 * i + 3] = y.w;
                }
                if constexpr (TP) {
                    const float4 *gs4 = reinterpret_cast<const float4 *>(sm.gs[prn][bdl]);
#pragma unroll
                    for (int i = 0; i < kC / 4; ++i) {
                        const float4 x = gs4[i];
                        gsN[4 * i] = x.x, gsN[4 * i + 1] = x.y, gsN[4 * i + 2] = x.z, gsN[4 * i + 3] = x.w;
                    }
                }
            };
            block_sync_lds();               // prologue: ring filled
            block_sync_lds();               // prologue: P_0, G_0
            if constexpr (!NT) fetch_inputs(0);
            for (int n = 0; n < NCH; ++n) {
                const int pr = n & 1;
                float grow[kC];
                if constexpr (NT) {
#pragma unroll
                    for (int u = 1; u < kC; ++u) grow[u] = sm.g[pr][0][u];
                }
                if constexpr (!NT) {
                    // ---- B: the token recurrence of chunk n, in scaled units.
                    // The softmax over j runs without subtracting its maximum: for
                    // logits and errors of ordinary size its sum z stays far inside
                    // the fp32 range.  Should z of some column and token leave
                    // [2^-100, 2^100], the chunk is run again with the maximum
                    // subtracted.  Inside that range a component whose term was
                    // lost to underflow (true value below 2^-126) has r below
                    // 2^-126 / 2^-100 = 2^-26, and no term exceeds 2^100, so
                    // beta delta times a term stays finite.
                    float P[kC], vv[kC], lkv[kC], bev[kC], gs[TP ? kC : 1];
#pragma unroll
                    for (int t = 0; t < kC; ++t) {
                        // padding component of J = 3: no mass; idle lanes: harmless
                        vv[t] = vvN[t];
                        lkv[t] = bpad ? (TP ? 0.f : -INFINITY) : lkvN[t];
                        bev[t] = bact ? bevN[t] : 0.f;
                        if constexpr (TP) gs[t] = bpad ? 0.f : gsN[t];
                    }
                    const float rprev0 = rprev;   // for a rerun of the chunk
#pragma unroll
                    for (int u = 1; u < kC; ++u) grow[u] = growN[u];
                    auto load_pred = [&]() {
#pragma unroll
                        for (int t = 0; t < kC; t += 4) {
                            const float4 p4 = *reinterpret_cast<const float4 *>(&sm.p[pr][C::prow(bcol)][t]);
                            P[t] = p4.x, P[t + 1] = p4.y, P[t + 2] = p4.z, P[t + 3] = p4.w;
                        }
                    };
                    load_pred();
                    // Software-pipelined: token t updates only P[t+1] at once; its
                    // other updates (P[u], u > t+1) run during token t+1, between
                    // the exponential and the sum over j, where they fill the wait.
                    // The scheduling barriers and the empty asm pins keep the compiler
                    // from sinking them into the dependent chain of a later token.
                    // The coefficients go out four tokens at a time; the branch on
                    // whether r is wanted is taken once per chunk.
                    auto run = [&](auto want) {
                        constexpr bool R = decltype(want)::value;
                        // chk is the largest z and 1/z seen (one max3 per token):
                        // above 2^100 iff some z left [2^-100, 2^100]
                        float chk = 0.f, cprev = 0.f, gprev[kC], cb[4];
#pragma unroll
                        for (int t = 0; t < kC; ++t) {
                            // row t+1 of G from column t+2 on, in 16-byte reads
                            float gnext[kC];
#pragma unroll
                            for (int q4 = (t + 2) / 4; q4 < kC / 4; ++q4) {
                                const float4 x = *reinterpret_cast<const float4 *>(&sm.g[pr][t + 1][4 * q4]);
                                gnext[4 * q4] = x.x, gnext[4 * q4 + 1] = x.y;
                                gnext[4 * q4 + 2] = x.z, gnext[4 * q4 + 3] = x.w;
                            }
                            // The deferred updates of this token (c_{t-1} into P[u],
                            // u > t) in four parts, one in each latency gap of the
                            // dependent chain d, exponent, exp2, sum over j, 1 / z,
                            // P[t+1]; the scheduling barriers keep every part in its
                            // gap and the empty asm pins keep the compiler from
                            // sinking the updates into a later token.
                            auto defer = [&](int part) {
                                if (t >= 1) {
                                    const int F = kC - 1 - t;
                                    const int lo = t + 1 + F * part / 4, hi = t + 1 + F * (part + 1) / 4;
#pragma unroll
                                    for (int u = lo; u < hi; ++u) {
                                        P[u] = fmaf(gprev[u], cprev, P[u]);
                                        asm volatile("" : "+v"(P[u]));
                                    }
                                }
                            };
                            const float d = vv[t] - P[t];
                            const float bd = bev[t] * d;
                            float ex;
                            if constexpr (TP)   // key prior (1 - g^k) r_{t-1} + g^k pi^k
                                ex = fmaf(gs[t], rprev, lkv[t]) * __builtin_amdgcn_exp2f(-d * d);
                            else
                                ex = __builtin_amdgcn_exp2f(fmaf(-d, d, lkv[t]));
                            __builtin_amdgcn_sched_barrier(0);
                            defer(0);
                            __builtin_amdgcn_sched_barrier(0);
                            float z = ex;
                            if constexpr (JP >= 2) z += dpp_mov<0xb1>(z);   // lane ^ 1
                            const float bdex = bd * ex;
                            const float gb = t + 1 < kC ? grow[t + 1] * bdex : 0.f;
                            __builtin_amdgcn_sched_barrier(0);
                            defer(1);
                            __builtin_amdgcn_sched_barrier(0);
                            if constexpr (JP >= 4) z += dpp_mov<0x4e>(z);   // lane ^ 2
                            if constexpr (JP >= 8) z += dpp_mov<0x141>(z);  // other quad of 8
                            if constexpr (JP >= 16) z += dpp_mov<0x140>(z); // other half of 16
                            __builtin_amdgcn_sched_barrier(0);
                            defer(2);
                            __builtin_amdgcn_sched_barrier(0);
                            const float iz = rcp_fast(z);
                            __builtin_amdgcn_sched_barrier(0);
                            defer(3);
                            __builtin_amdgcn_sched_barrier(0);
                            if (t + 1 < kC) P[t + 1] = fmaf(gb, iz, P[t + 1]);
                            const float cs = bdex * iz;                  // s c
                            cb[t & 3] = cs;
                            if ((t & 3) == 3)
                                *reinterpret_cast<float4 *>(&sm.c[pr][C::prow(bsto)][t - 3]) =
                                    make_float4(cb[0], cb[1], cb[2], cb[3]);
                            if constexpr (R) {
                                const float rt = ex * iz;
                                sm.r[pr][t][bsto] = dmode ? kInvWS * d : rt;
                                if constexpr (TP) rprev = rt;
                            }
                            chk = fmaxf(chk, fmaxf(z, iz));
                            cprev = cs;
#pragma unroll
                            for (int u = t + 2; u < kC; ++u) gprev[u] = grow[u], grow[u] = gnext[u];
                        }
                        // (an integer test on bits the compiler cannot trace back to a
                        // float: the file is compiled without NaN semantics, and a NaN,
                        // whose magnitude bits exceed those of 2^100, must fail it too)
                        uint32_t chk_bits = __float_as_uint(chk);
                        asm volatile("" : "+v"(chk_bits));
                        const bool bad = (chk_bits & 0x7fffffffu) > 0x71800000u;   // 2^100
                        if (__builtin_amdgcn_ballot_w64(bact && bad) != 0) {
                            // some softmax sum left the range: the chunk again, maximum subtracted
#pragma unroll
                            for (int u = 1; u < kC; ++u) grow[u] = sm.g[pr][0][u];
                            load_pred();
                            if constexpr (TP) rprev = rprev0;
#pragma unroll
                            for (int t = 0; t < kC; ++t) {
                                float gnext[kC];
#pragma unroll
                                for (int u = t + 2; u < kC; ++u) gnext[u] = sm.g[pr][t + 1][u];
                                const float d = vv[t] - P[t];
                                const float bd = bev[t] * d;
                                const float e = TP ? (bpad ? -INFINITY : -d * d) : fmaf(-d, d, lkv[t]);
                                float ex = __builtin_amdgcn_exp2f(e - group_max<JP>(e));
                                if constexpr (TP) ex *= fmaf(gs[t], rprev, lkv[t]);
                                const float iz = rcp_fast(group_sum<JP>(ex));
                                const float cs = (bd * ex) * iz;
#pragma unroll
                                for (int u = t + 1; u < kC; ++u) P[u] = fmaf(grow[u], cs, P[u]);
                                sm.c[pr][C::prow(bsto)][t] = cs;
                                if constexpr (R) {
                                    const float rt = ex * iz;
                                    sm.r[pr][t][bsto] = dmode ? kInvWS * d : rt;
                                    if constexpr (TP) rprev = rt;
                                }
#pragma unroll
                                for (int u = t + 2; u < kC; ++u) grow[u] = gnext[u];
                            }
                        }
                    };
                    if (TP || want_r) run(BoolTag<true>{});
                    else run(BoolTag<false>{});
                } else {
                    // ---- B: forward substitution of the linearised recurrence
                    // (eq. linearized) over chunk n; g clamped to [0, 2 / |k_t|^2]
                    // unless disabled
                    const float *po = reinterpret_cast<const float *>(sm.pw[n % kRingQP]);
                    float P[kC], gc[kC], bb[kC], pold[kC];
                    const float glo_t = na.clamp ? 0.f : -INFINITY;
#pragma unroll
                    for (int t = 0; t < kC; ++t) {
                        P[t] = sm.p[pr][C::prow(bcol)][t];
                        const float ghi_t = na.clamp ? 2.f * rcp_fast(sm.g[pr][t][t]) : INFINITY;
                        gc[t] = fminf(fmaxf(sm.beta[pr][t][bcol], glo_t), ghi_t);
                        bb[t] = sm.lks[pr][t][bcol];
                        pold[t] = po[t * N + bcol];
                    }
#pragma unroll
                    for (int t = 0; t < kC; ++t) {
                        float gnext[kC];
#pragma unroll
                        for (int u = t + 2; u < kC; ++u) gnext[u] = sm.g[pr][t + 1][u];
                        const float pt = P[t];
                        const float x = fmaf(gc[t], pold[t] - pt, bb[t]);
#pragma unroll
                        for (int u = t + 1; u < kC; ++u) P[u] = fmaf(grow[u], x, P[u]);
                        sm.c[pr][C::prow(bsto)][t] = x;
                        const int tok = n * kC + t;
                        if (bact) {
                            pred[(size_t)tok * N + bcol] = pt;
                            if (tok < T) {
                                dmax = fmaxf(dmax, fabsf(pt - pold[t]));
                                pmax = fmaxf(pmax, fabsf(pt));
                            }
                        }
#pragma unroll
                        for (int u = t + 2; u < kC; ++u) grow[u] = gnext[u];
                    }
                }
                block_sync_lds();   // e(n): C_n published
                if constexpr (!NT) {
                    if (n + 1 < NCH) fetch_inputs(pr ^ 1);
                    // i(n+1), P_{n+1} ready.  This wave has no LDS stores in
                    // flight here, and nothing rewrites the slots it is reading
                    // before i(n+2): its reads may land after the barrier.
                    asm volatile("s_barrier" ::: "memory");
                } else {
                    block_sync_lds();   // i(n+1): P_{n+1} ready
                }
            }
            block_sync_lds();       // epilogue
            if constexpr (NT) {
                // stopping rule, decided here for the whole block
#pragma unroll
                for (int off = 32; off >= 1; off >>= 1) {
                    dmax = fmaxf(dmax, __shfl_xor(dmax, off));
                    pmax = fmaxf(pmax, __shfl_xor(pmax, off));
                }
                if (lane == 0) {
                    sm.flag = (na.tol >= 0.f && dmax <= na.tol * fmaxf(1.f, pmax)) ? 1 : 0;
                    sm.near = (na.tol >= 0.f && dmax <= 4.f * na.tol * fmaxf(1.f, pmax)) ? 1 : 0;
                }
                wait_vm();          // this sweep's predictions are in memory
                block_sync_lds();
                next_sweep(sweeps, qs, done);   // as the matrix-core waves decide
            } else {
                done = true;
            }
        }
        if constexpr (TP) {
            // r of the last token: part 0 of the prior state
            if (bact && a.prior_out)
                a.prior_out[(((size_t)b * H + h) * 2 * J + bj) * Dv + d0 + bdl] =
                    sm.r[(NCH - 1) & 1][T - 1 - (NCH - 1) * kC][bsto];
        }
        return;
    }

    // The matrix-core side, one copy per role: with NH = 0 the tile waves also
    // do the bookkeeping; with NH > 0 the tile waves and the helper waves run
    // copies of their own that meet the same barriers.
    if constexpr (NH == 0) {
        constexpr bool DT = true, DBK = true;
#include "scan_pipe_mfma_side.inc"
    } else if (tile) {
        constexpr bool DT = true, DBK = false;
#include "scan_pipe_mfma_side.inc"
    } else {
        constexpr bool DT = false, DBK = true;
#include "scan_pipe_mfma_side.inc"
    }
}

__global__ void int_fill_kernel(int *p, int n, int value) {
    if ((int)threadIdx.x < n) p[threadIdx.x] = value;
}

template <int DK, int J, int DB, int MD>
hipError_t launch_cfg(const LayerArgs &a, const NewtonArgs &na, hipStream_t stream) {
    using C = PCfg<DK, J, DB>;
    constexpr size_t lds = sizeof(PSmem<DK, J, DB, MD>);
    static_assert(lds <= 160 * 1024, "LDS");
    const long blocks = (long)(a.Dv / DB) * a.H * a.B;
    // Enough blocks to put two on every compute unit (LDS permitting): their
    // waves hide each other's latencies, so the tile waves keep the
    // bookkeeping.  Otherwise helper waves take it over.
    // (the temporal form has more per-chunk bookkeeping: always three helpers)
    // (a block over 80 KB of LDS is never two to a compute unit: only the
    // variant with helpers is built for it)
    constexpr int NH = MD == 2 ? 3 : (C::NW < 3 ? C::NW : 3);
    if constexpr (lds <= 80 * 1024) {
        if (blocks >= 512) {
            hipLaunchKernelGGL((scan_pipe_kernel<DK, J, DB, MD, 0>), dim3((unsigned)blocks),
                               dim3(64 * (C::NW + 1)), 0, stream, a, na);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((scan_pipe_kernel<DK, J, DB, MD, NH>), dim3((unsigned)blocks),
                       dim3(64 * (C::NW + 1 + NH)), 0, stream, a, na);
    return hipGetLastError();
}

template <int DK, int MD>
hipError_t launch_dk(const LayerArgs &a, const NewtonArgs &na, hipStream_t stream) {
    // At most 64 columns (one wave of sequential lanes).  J = 4 takes 32
    // columns (DB = 8): twice the blocks, the sequential wave on a SIMD of its
    // own, and two blocks' LDS fit one compute unit.
    switch (a.J) {
        case 1:
            // (the temporal form's extra staging does not fit 64 columns of Dk = 128)
            if constexpr (MD != 2 || DK < 128)
                if (a.Dv >= 64) return launch_cfg<DK, 1, 64, MD>(a, na, stream);
            if (a.Dv >= 32) return launch_cfg<DK, 1, 32, MD>(a, na, stream);
            return launch_cfg<DK, 1, 16, MD>(a, na, stream);
        case 2:
            if (a.Dv >= 32) return launch_cfg<DK, 2, 32, MD>(a, na, stream);
            return launch_cfg<DK, 2, 16, MD>(a, na, stream);
        case 3: return launch_cfg<DK, 3, 16, MD>(a, na, stream);
        case 4:
            // With enough heads to fill the chip twice over at 32 columns, 64
            // columns per block halve the blocks: the sequential wave's time per
            // token does not depend on its column count, so fewer, wider blocks
            // finish the batch in fewer rounds.
            if ((long)(a.Dv / 8) * a.H * a.B >= 512 && a.Dv >= 16)
                return launch_cfg<DK, 4, 16, MD>(a, na, stream);
            return launch_cfg<DK, 4, 8, MD>(a, na, stream);
        case 8: return launch_cfg<DK, 8, 8, MD>(a, na, stream);
        default: return hipErrorInvalidValue;
    }
}

template <int MD>
hipError_t launch_mode(const LayerArgs &a, const NewtonArgs &na, hipStream_t stream) {
    if (!a.in_bf16 || a.T <= 0) return hipErrorInvalidValue;
    switch (a.Dk) {
        case 16: return launch_dk<16, MD>(a, na, stream);
        case 32: return launch_dk<32, MD>(a, na, stream);
        case 64: return launch_dk<64, MD>(a, na, stream);
        case 128: return launch_dk<128, MD>(a, na, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace
}  // namespace swila
