// Chunk form of Gated SwiLA on the matrix cores (App. B.4, eq. pre-decay with
// one gate per key dimension, eq. gate-elementwise tied across the output
// index): bf16 inputs, fp32 state.
//
// Per component j and output dim d the recurrence is
//   w~_t = a_t (.) w_{t-1},   delta_t = v_t - k_t . w~_t,   w_t = w~_t + c_t k_t,
// c_t = beta r delta (r from eq. responsibility at the decayed state), with
// a_t = sigmoid(decay logit) in (0,1)^Dk.  Inside a chunk of 16 tokens that
// starts from S, with L_t = sum_{u<=t} log a_u (per key index, from the chunk
// start) and E_t = e^{L_t}:
//   w~_t = E_t (.) S + sum_{s<t} (E_t / E_s) (.) k_s c_s
//   pred_t  = (k_t (.) E_t) . S + sum_{s<t} G_ts c_s,   G_ts = sum_i k_ti k_si e^{L_ti - L_si}
//   q_t.w_t = (q_t (.) E_t) . S + sum_{s<=t} QG_ts c_s, QG_ts = sum_i q_ti k_si e^{L_ti - L_si}
//   S'      = E_C (.) S + sum_s (k_s (.) E_C / E_s) c_s.
// G and QG are formed as (K (.) E)(K (.) E^-1)^T on the matrix cores while
// every E^-1 stays below e^{40}.  E^-1 is the running product of 1 + e^{-x}
// over the chunk's decay logits x (1 / sigmoid), one exponential per element,
// and E its reciprocal; a chunk whose gates decay further (some E^-1_C above
// e^{40}) forms its cumulative log gates L instead and the Gram products with
// the per-pair exponent.  The scaled operands are fp32: each is split into a
// bf16 high part and a bf16 residual, and the hi*hi + hi*lo + lo*hi products
// are summed (about 2^-16 relative per product, fp32 accumulation).  A
// component's gates differ from the others', so each component has its own
// Gram matrices and scaled operands: tile wave j holds the state columns of
// component j.
//
// Block = one head (b, h) and DB output dims with all J components (J <= 4,
// J * Dk <= 512): J tile waves (wave j: the Dk x DB state tile of component j
// in accumulator registers), one sequential wave (one lane per column, the J
// components of an output dim in adjacent lanes), three helper waves.  Per
// chunk n, between two block barriers:
//   phase A  sequential wave: the chunk's 16-token recurrence -> C_n
//            tile waves: retrieval of chunk n-1 (needs C_{n-1}); Q_n S_n and
//              the update operand of chunk n; E^-1 of chunk n+1 (wave j:
//              component j's), K_{n+1} (.) E_{n+1}, Q_{n+1} (.) E_{n+1},
//              G_{n+1} for the next recurrence and QG_{n+1}
//            helper waves: pi^q_n, the output of chunk n-2, and the inputs of
//              chunk n+2 but its decay logits (HBM -> registers -> LDS)
//   phase B  tile waves: S_{n+1} = E_C (.) S_n + U_n^T C_n and
//              P_{n+1} = (K_{n+1} (.) E_{n+1}) S_{n+1} for the next recurrence;
//            sequential wave: beta, key-prior logits and v of chunk n+1;
//            helper waves: the decay logits of chunk n+2, the loads of n+3.
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

typedef short short4v __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kGC = 16;              // tokens per chunk
constexpr int kGH = 3;               // helper waves
constexpr float kGramEinv = 2.35385266837019985e17f;   // e^40: factorised Gram products while every E^-1 <= this
// The sequential wave works in scaled units: with s^2 = log2(e) / 2, d = s (v - pred)
// makes the E-step exponent log2(e) (lk - delta^2 / 2) a single fused multiply-add,
// -d * d + log2(e) lk, and the coefficient s c = beta r d feeds s pred.
constexpr float kS = 0.84932180028801904272f;      // sqrt(log2(e) / 2)
constexpr float kInvS = 1.17741002251547469101f;   // 1 / kS
constexpr int ceil_div_c(int x, int y) { return (x + y - 1) / y; }

__device__ __forceinline__ floatx4 mfma16(short4v a, short4v b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}

// Four fp32 values as bf16 high parts (round to nearest) and bf16 residuals,
// converted two at a time.
struct S4 {
    short4v hi, lo;
};
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void split2(float a, float b, uint32_t &hi, uint32_t &lo) {
    hi = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{a, b}, bf16x2v));
    const float ah = __uint_as_float(hi << 16), bh = __uint_as_float(hi & 0xffff0000u);
    lo = __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{a - ah, b - bh}, bf16x2v));
}
__device__ __forceinline__ S4 split4(float x0, float x1, float x2, float x3) {
    uint32_t h0, l0, h1, l1;
    split2(x0, x1, h0, l0);
    split2(x2, x3, h1, l1);
    S4 s;
    s.hi = __builtin_bit_cast(short4v, make_uint2(h0, h1));
    s.lo = __builtin_bit_cast(short4v, make_uint2(l0, l1));
    return s;
}
__device__ __forceinline__ S4 split4(floatx4 x) { return split4(x[0], x[1], x[2], x[3]); }
__device__ __forceinline__ S4 zero4() {
    S4 s;
    s.hi = short4v{0, 0, 0, 0};
    s.lo = short4v{0, 0, 0, 0};
    return s;
}
// a b with both operands split: hi hi + hi lo + lo hi
__device__ __forceinline__ floatx4 mm3(const S4 &a, const S4 &b, floatx4 acc) {
    acc = mfma16(a.hi, b.hi, acc);
    acc = mfma16(a.hi, b.lo, acc);
    acc = mfma16(a.lo, b.hi, acc);
    return acc;
}
// The same over two 16-wide k tiles at once (a0 b0 + a1 b1), on the 32-deep
// instruction: a lane's eight k elements are its four of tile 0, then its four
// of tile 1, in both operands.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ bf16x8 join8(short4v x, short4v y) {
    return __builtin_bit_cast(bf16x8, make_uint4(__builtin_bit_cast(uint2, x).x,
                                                 __builtin_bit_cast(uint2, x).y,
                                                 __builtin_bit_cast(uint2, y).x,
                                                 __builtin_bit_cast(uint2, y).y));
}
__device__ __forceinline__ floatx4 mm3x2(const S4 &a0, const S4 &a1, const S4 &b0, const S4 &b1,
                                         floatx4 acc) {
    const bf16x8 ah = join8(a0.hi, a1.hi), al = join8(a0.lo, a1.lo);
    const bf16x8 bh = join8(b0.hi, b1.hi), bl = join8(b0.lo, b1.lo);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ float bf(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// log sigmoid(x) = min(x, 0) - log(1 + e^{-|x|})
__device__ __forceinline__ float log_sigmoid(float x) {
    const float e = __builtin_amdgcn_exp2f(-fabsf(x) * kLog2e);
    return fminf(x, 0.0f) - __builtin_amdgcn_logf(1.0f + e) * 0.69314718055994531f;
}

template <int DK, int J, int DB>
struct GCfg {
    static constexpr int IT = DK / 16;       // 16-row key tiles
    static constexpr int N = J * DB;         // columns, col = j * DB + dd
    static constexpr int JP = J == 3 ? 4 : J;
    static constexpr int NWAVE = J + 1 + kGH;
    static constexpr int KP = DK + 4;        // bf16 row pitch of the K, Q tiles
    static constexpr int LP = DK + 4;        // fp32 row pitch of E^-1 (or L)
    static constexpr int TP = kGC + 4;       // [column][token] row pitch
    static constexpr int NP = N + 4;         // [token][column] row pitch
    static_assert(J >= 1 && J <= 4 && J * DK <= 512, "LDS budget of the gated chunk form");
    static_assert(DB == 8 || DB == 16, "column block");
    static_assert(DB * JP <= 64, "one sequential wave");
};

template <int DK, int J, int DB>
struct GSmem {
    using C = GCfg<DK, J, DB>;
    // chunk inputs, chunk m in slot m % 3
    alignas(16) uint16_t k[3][kGC][C::KP];
    alignas(16) uint16_t q[3][kGC][C::KP];
    alignas(16) uint16_t lq[3][kGC][C::N];   // [token][j * DB + dd]
    alignas(16) uint16_t g[kGC][J * DK];     // decay logits of the next chunk to take its gates
    // E^-1 of chunk m (its cumulative log gates L in a deep chunk), written and
    // read by tile wave j only; E_C, chunk m in m & 1
    alignas(16) float ei[J][kGC][C::LP];
    alignas(16) float ec[2][J][DK];
    // for the sequential wave, chunk m in m & 1: {beta, log2(e) key-prior logit}
    // [column][token] (beta = 0 past the end) and s v [dim][token]
    alignas(16) float2 sq[2][C::N][kGC + 2];
    alignas(16) float vs[2][DB][kGC + 4];
    alignas(16) float gt[2][J][kGC][kGC + 4];   // gt[.][j][s][t] = G_ts (t > s), chunk m in m & 1
    alignas(16) float p[C::N][C::TP];        // chunk-start predictions, times s [column][token]
    alignas(16) float c[2][C::N][C::TP];     // coefficients [column][token], chunk m in m & 1
    float pq[2][kGC][C::NP];                 // pi^q [token][column]
    float py[2][kGC][C::NP];                 // pi^q * retrieval [token][column]
};

// Block -> (column block, head): the column blocks of a head on one XCD
// (workgroups go to the eight XCDs round-robin by index, each with its own L2),
// so that the head's K, Q and gate rows are fetched from HBM once.
__device__ __forceinline__ void gated_coords(int id, int ndb, int nheads, int &db, int &head) {
    if (nheads % 8 == 0) {
        const int k = id / 8;
        head = id % 8 + 8 * (k / ndb);
        db = k % ndb;
    } else {
        head = id / ndb;
        db = id % ndb;
    }
}

// Each role runs its whole chunk loop in a branch of its own, so that the
// registers one role keeps across chunks are not held by the others; every
// role meets the same block barriers in the same order: four in the prologue,
// two per chunk (e(n): C_n and chunk n + 2 published; i(n+1): P_{n+1}
// published), one in the epilogue.
template <int DK, int J, int DB>
__global__ __launch_bounds__(512) void scan_gated_chunk_kernel(LayerArgs a) {
    using C = GCfg<DK, J, DB>;
    constexpr int IT = C::IT, N = C::N, JP = C::JP;
    __shared__ GSmem<DK, J, DB> sm;

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64), lane = tid % 64;
    const int tl = lane % 16, lg = lane / 16;
    const int H = a.H, T = a.T, Dv = a.Dv;
    int db, hh;
    gated_coords(blockIdx.x, Dv / DB, a.B * H, db, hh);
    const int d0 = db * DB, h = hh % H, b = hh / H;
    const int NCH = (T + kGC - 1) / kGC;

    if (w < J) {
        // ================= tile wave j: the state of component j =================
        // state S^j rows 16 it + 4 lg + r, column tl (a real column when tl < DB)
        const int tj = w;
        const bool tvalid = tl < DB;
        const int tcol = tj * DB + (tvalid ? tl : 0);
        float (*const EI)[C::LP] = sm.ei[tj];
        floatx4 W[IT];
        S4 Kp[IT];   // K_m (.) E_m for the next chunk m, A operand (rows t = tl)
        S4 Qe[IT];   // Q_m (.) E_m for the next chunk m (rows t = tl)
        S4 U[IT];    // update operand of chunk n: rows i = 16 it + tl, columns s = 4 lg + m
        // Q S and tril(QG) (A operand) of the chunk whose retrieval is pending
        // (r), and of the chunk after it (q)
        floatx4 Y0r = floatx4{0.f, 0.f, 0.f, 0.f}, Y0q = floatx4{0.f, 0.f, 0.f, 0.f};
        S4 QGr = zero4(), QGq = zero4();
        bool deep_n = false, deep_n1 = false;   // chunk n, n+1 past the factorised Gram products

        // E^-1 (or, in a deep chunk, L) and E_C of chunk m for component tj from
        // its decay logits (lane: key index lane, or 2 lane and 2 lane + 1 when
        // Dk = 128); returns whether the chunk is deep.
        auto log_gates = [&](int m) {
            const int nt = min(kGC, T - m * kGC);
            bool deep = false;
            if constexpr (DK == 128) {
                // two adjacent key indices per lane
                const int i = 2 * lane;
                uint32_t x[kGC];
#pragma unroll
                for (int t = 0; t < kGC; ++t)
                    x[t] = *reinterpret_cast<const uint32_t *>(&sm.g[t][tj * DK + i]);
                float c0 = 1.0f, c1 = 1.0f;
#pragma unroll
                for (int t = 0; t < kGC; ++t) {
                    const float f0 = 1.0f + __builtin_amdgcn_exp2f(-kLog2e * __uint_as_float(x[t] << 16));
                    const float f1 =
                        1.0f + __builtin_amdgcn_exp2f(-kLog2e * __uint_as_float(x[t] & 0xffff0000u));
                    c0 *= t < nt ? f0 : 1.0f;
                    c1 *= t < nt ? f1 : 1.0f;
                    *reinterpret_cast<float2 *>(&EI[t][i]) = make_float2(c0, c1);
                }
                *reinterpret_cast<float2 *>(&sm.ec[m & 1][tj][i]) = make_float2(rcp_fast(c0), rcp_fast(c1));
                deep = !(c0 <= kGramEinv) || !(c1 <= kGramEinv);
                if (__any(deep) == 0) return false;
                // deep chunk: L = the running sum of log sigmoid, in place of E^-1
                float l0 = 0.0f, l1 = 0.0f;
#pragma unroll
                for (int t = 0; t < kGC; ++t) {
                    l0 += t < nt ? log_sigmoid(__uint_as_float(x[t] << 16)) : 0.0f;
                    l1 += t < nt ? log_sigmoid(__uint_as_float(x[t] & 0xffff0000u)) : 0.0f;
                    *reinterpret_cast<float2 *>(&EI[t][i]) = make_float2(l0, l1);
                }
                *reinterpret_cast<float2 *>(&sm.ec[m & 1][tj][i]) =
                    make_float2(__builtin_amdgcn_exp2f(kLog2e * l0), __builtin_amdgcn_exp2f(kLog2e * l1));
                return true;
            } else {
                // one key index per lane (lanes past Dk idle)
                const int i = lane, ic = DK >= 64 || i < DK ? i : 0;
                float x[kGC];
#pragma unroll
                for (int t = 0; t < kGC; ++t) x[t] = bf(sm.g[t][tj * DK + ic]);
                // tokens past the end decay nothing: the chunk's last row is the
                // product over its last token
                float cum = 1.0f, e[kGC];
#pragma unroll
                for (int t = 0; t < kGC; ++t) {
                    const float f = 1.0f + __builtin_amdgcn_exp2f(-kLog2e * x[t]);
                    cum *= t < nt ? f : 1.0f;
                    e[t] = cum;
                }
                if (DK >= 64 || i < DK) {
#pragma unroll
                    for (int t = 0; t < kGC; ++t) EI[t][i] = e[t];
                    sm.ec[m & 1][tj][i] = rcp_fast(cum);
                    deep = !(cum <= kGramEinv);
                }
                if (__any(deep) == 0) return false;
                if (DK >= 64 || i < DK) {
                    float l = 0.0f;
#pragma unroll
                    for (int t = 0; t < kGC; ++t) {
                        l += t < nt ? log_sigmoid(x[t]) : 0.0f;
                        EI[t][i] = l;
                    }
                    sm.ec[m & 1][tj][i] = __builtin_amdgcn_exp2f(kLog2e * l);
                }
                return true;
            }
        };

        // four bf16 of row tl of X, key indices 16 it + 4 lg .. + 3, times f
        auto row4 = [&](const uint16_t (*X)[C::KP], int it, float4 f) {
            const uint2 raw = *reinterpret_cast<const uint2 *>(&X[tl][16 * it + 4 * lg]);
            return split4(__uint_as_float(raw.x << 16) * f.x,
                          __uint_as_float(raw.x & 0xffff0000u) * f.y,
                          __uint_as_float(raw.y << 16) * f.z,
                          __uint_as_float(raw.y & 0xffff0000u) * f.w);
        };
        // per-pair exponent (deep chunk m, L in EI): sum_i X[t][i] K[s][i] e^{L_ti - L_si}
        auto pair_dot = [&](const uint16_t (*X)[C::KP], int m, int t, int s) {
            float acc = 0.0f;
#pragma unroll 1
            for (int i = 0; i < DK; ++i)
                acc = fmaf(bf(X[t][i]) * bf(sm.k[m % 3][s][i]),
                           __builtin_amdgcn_exp2f(kLog2e * (EI[t][i] - EI[s][i])), acc);
            return acc;
        };
        // the operands of chunk m: Kp, Qe, G_m (for the sequential wave) and QG_m
        auto gram = [&](int m, bool pair) {
            const int s3 = m % 3;
            floatx4 g = floatx4{0.f, 0.f, 0.f, 0.f}, qg = floatx4{0.f, 0.f, 0.f, 0.f};
            if (!pair) {
                // E^-1 and E at rows tl, key indices 16 it + 4 lg .. + 3; K (.) E^-1
                // at rows s = tl
                auto operands = [&](int it) {
                    const float4 x = *reinterpret_cast<const float4 *>(&EI[tl][16 * it + 4 * lg]);
                    const float4 er = make_float4(rcp_fast(x.x), rcp_fast(x.y), rcp_fast(x.z), rcp_fast(x.w));
                    Kp[it] = row4(sm.k[s3], it, er);
                    Qe[it] = row4(sm.q[s3], it, er);
                    return row4(sm.k[s3], it, x);
                };
                if constexpr (IT == 1) {
                    const S4 kinv = operands(0);
                    g = mm3(Kp[0], kinv, g);      // D[t = 4 lg + r][s = tl] = G_ts
                    qg = mm3(kinv, Qe[0], qg);    // D[s = 4 lg + r][t = tl] = QG_ts
                } else {
#pragma unroll
                    for (int it = 0; it < IT; it += 2) {
                        const S4 k0 = operands(it), k1 = operands(it + 1);
                        g = mm3x2(Kp[it], Kp[it + 1], k0, k1, g);
                        qg = mm3x2(k0, k1, Qe[it], Qe[it + 1], qg);
                    }
                }
                // lane (tl, lg) holds QG[t = tl][s = 4 lg + r]: the A operand of the retrieval
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (4 * lg + r > tl) qg[r] = 0.0f;
            } else {
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const float4 x = *reinterpret_cast<const float4 *>(&EI[tl][16 * it + 4 * lg]);
                    const float4 er = make_float4(__builtin_amdgcn_exp2f(kLog2e * x.x),
                                                  __builtin_amdgcn_exp2f(kLog2e * x.y),
                                                  __builtin_amdgcn_exp2f(kLog2e * x.z),
                                                  __builtin_amdgcn_exp2f(kLog2e * x.w));
                    Kp[it] = row4(sm.k[s3], it, er);
                    Qe[it] = row4(sm.q[s3], it, er);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 4 * lg + r;   // row of G
                    const int s = 4 * lg + r;   // column of QG
                    g[r] = t > tl ? pair_dot(sm.k[s3], m, t, tl) : 0.0f;
                    qg[r] = s <= tl ? pair_dot(sm.q[s3], m, tl, s) : 0.0f;
                }
            }
            *reinterpret_cast<float4 *>(&sm.gt[m & 1][tj][tl][4 * lg]) =
                make_float4(g[0], g[1], g[2], g[3]);
            QGq = split4(qg);
        };
        // for the next chunk, from its start state S: the predictions P = Kp S
        // for the sequential wave, in its units, and Q S (Y0q)
        auto predict = [&]() {
            floatx4 pacc = floatx4{0.f, 0.f, 0.f, 0.f}, y0 = floatx4{0.f, 0.f, 0.f, 0.f};
            if constexpr (IT == 1) {
                const S4 ws = split4(W[0]);
                pacc = mm3(Kp[0], ws, pacc);   // D[t][col]
                y0 = mm3(Qe[0], ws, y0);
            } else {
#pragma unroll
                for (int it = 0; it < IT; it += 2) {
                    const S4 w0 = split4(W[it]), w1 = split4(W[it + 1]);
                    pacc = mm3x2(Kp[it], Kp[it + 1], w0, w1, pacc);
                    y0 = mm3x2(Qe[it], Qe[it + 1], w0, w1, y0);
                }
            }
            if (tvalid)
                *reinterpret_cast<float4 *>(&sm.p[tcol][4 * lg]) =
                    make_float4(kS * pacc[0], kS * pacc[1], kS * pacc[2], kS * pacc[3]);
            Y0q = y0;
        };
        // C of chunk m as the B operand: rows s = 4 lg .. + 3, column tl
        auto coeffs = [&](int m) {
            const float4 c4 = *reinterpret_cast<const float4 *>(&sm.c[m & 1][tcol][4 * lg]);
            return tvalid ? split4(c4.x, c4.y, c4.z, c4.w) : zero4();
        };
        // retrieval of chunk m: Y = Y0 + tril(QG) C, times pi^q, to py
        auto retrieve = [&](int m) {
            const floatx4 y = mm3(QGr, coeffs(m), Y0r);   // D[t = 4 lg + r][col]
            if (tvalid) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 4 * lg + r;
                    sm.py[m & 1][t][tcol] = sm.pq[m & 1][t][tcol] * y[r];
                }
            }
        };
        // what chunk n needs besides C_n: its Q S and tril(QG) for the retrieval
        // (from Y0q and QGq) and U_n (EI holds chunk n's E^-1 or L)
        auto prepare = [&](int n, bool pair) {
            const int s3 = n % 3;
            Y0r = Y0q;
            QGr = QGq;
            // U[i][s] = K[s][i] E_C,i / E_s,i, i = 16 it + tl, s = 4 lg + m
            if (!pair) {
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int i = 16 * it + tl;
                    const float ecv = sm.ec[n & 1][tj][i];
                    float u[4];
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const int s = 4 * lg + m;
                        u[m] = bf(sm.k[s3][s][i]) * (ecv * EI[s][i]);
                    }
                    U[it] = split4(u[0], u[1], u[2], u[3]);
                }
            } else {
#pragma unroll
                for (int it = 0; it < IT; ++it) {
                    const int i = 16 * it + tl;
                    const float lc = EI[kGC - 1][i];
                    float u[4];
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        const int s = 4 * lg + m;
                        u[m] = bf(sm.k[s3][s][i]) * __builtin_amdgcn_exp2f(kLog2e * (lc - EI[s][i]));
                    }
                    U[it] = split4(u[0], u[1], u[2], u[3]);
                }
            }
        };

#pragma unroll
        for (int it = 0; it < IT; ++it)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                W[it][r] = tvalid && a.state_in
                               ? a.state_in[(((size_t)b * H + h) * J + tj) * DK * Dv +
                                            (size_t)(16 * it + 4 * lg + r) * Dv + d0 + tl]
                               : 0.0f;
        block_sync_lds();   // prologue 1
        block_sync_lds();   // prologue 2: chunks 0 and 1 in LDS (the decay logits of 0)
        deep_n = log_gates(0);
        gram(0, deep_n);
        predict();          // P_0, Q_0 S_0
        block_sync_lds();   // prologue 3: the decay logits of chunk 0 read
        block_sync_lds();   // prologue 4: those of chunk 1 in LDS
        for (int n = 0; n < NCH; ++n) {
            // ---- phase A: everything that does not need C_n
            if (n >= 1) retrieve(n - 1);
            prepare(n, deep_n);
            if (n + 1 < NCH) {
                deep_n1 = log_gates(n + 1);
                gram(n + 1, deep_n1);
            }
            block_sync_lds();   // e(n)
            // ---- phase B: S_{n+1} = E_C (.) S_n + U_n^T C_n, then P_{n+1}, Q_{n+1} S_{n+1}
            const S4 cb = coeffs(n);
#pragma unroll
            for (int it = 0; it < IT; ++it) {
                const float4 e4 = *reinterpret_cast<const float4 *>(&sm.ec[n & 1][tj][16 * it + 4 * lg]);
                W[it][0] *= e4.x;
                W[it][1] *= e4.y;
                W[it][2] *= e4.z;
                W[it][3] *= e4.w;
                W[it] = mm3(U[it], cb, W[it]);
            }
            if (n + 1 < NCH) predict();
            deep_n = deep_n1;
            block_sync_lds();   // i(n+1)
        }
        retrieve(NCH - 1);
        block_sync_lds();   // epilogue
        if (tvalid && a.state_out) {
#pragma unroll
            for (int it = 0; it < IT; ++it)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    a.state_out[(((size_t)b * H + h) * J + tj) * DK * Dv +
                                (size_t)(16 * it + 4 * lg + r) * Dv + d0 + tl] = W[it][r];
        }
    } else if (w == J) {
        // ================= sequential wave: one lane per column =================
        const int sdd = lane / JP, sj = lane % JP;
        const bool sact = sdd < DB && sj < J;
        const int scol = sact ? sj * DB + sdd : 0, gj = sact ? sj : 0;
        const bool wres = a.resp && sact;
        float sbeta[kGC], slk[kGC], sv[kGC];
        const int vdd = sact ? sdd : 0;
        // beta, key-prior logits and v of chunk m (idle lanes read column 0)
        auto seq_inputs = [&](int m) {
#pragma unroll
            for (int t2 = 0; t2 < kGC; t2 += 2) {
                const float4 x = *reinterpret_cast<const float4 *>(&sm.sq[m & 1][scol][t2]);
                // idle lanes (and the padding component of J = 3) carry no mass
                sbeta[t2] = sact ? x.x : 0.0f, slk[t2] = sact ? x.y : -INFINITY;
                sbeta[t2 + 1] = sact ? x.z : 0.0f, slk[t2 + 1] = sact ? x.w : -INFINITY;
            }
#pragma unroll
            for (int t4 = 0; t4 < kGC; t4 += 4) {
                const float4 x = *reinterpret_cast<const float4 *>(&sm.vs[m & 1][vdd][t4]);
                sv[t4] = x.x, sv[t4 + 1] = x.y, sv[t4 + 2] = x.z, sv[t4 + 3] = x.w;
            }
        };
        block_sync_lds();   // prologue 1
        block_sync_lds();   // prologue 2
        seq_inputs(0);
        block_sync_lds();   // prologue 3
        block_sync_lds();   // prologue 4
        for (int n = 0; n < NCH; ++n) {
            const int t0 = n * kGC, nt = min(kGC, T - t0), gs = n & 1;
            // ---- the token recurrence of chunk n, in scaled units.  The softmax
            // over j runs without subtracting its maximum: for logits and errors
            // of ordinary size its sum z stays far inside the fp32 range.  Should
            // z of some column and token leave [2^-100, 2^100], the chunk is run
            // again with the maximum subtracted (the bound of the plain chunk scan).
            float P[kGC], cc[kGC], grow[kGC];
            auto load_pred = [&]() {
#pragma unroll
                for (int t4 = 0; t4 < kGC; t4 += 4) {
                    const float4 p4 = *reinterpret_cast<const float4 *>(&sm.p[scol][t4]);
                    P[t4] = p4.x, P[t4 + 1] = p4.y, P[t4 + 2] = p4.z, P[t4 + 3] = p4.w;
                }
#pragma unroll
                for (int u4 = 0; u4 < kGC; u4 += 4) {   // row 0 of gt: G_u0
                    const float4 x = *reinterpret_cast<const float4 *>(&sm.gt[gs][gj][0][u4]);
                    grow[u4] = x.x, grow[u4 + 1] = x.y, grow[u4 + 2] = x.z, grow[u4 + 3] = x.w;
                }
            };
            load_pred();
            // Software-pipelined: token t updates only P[t+1] at once; its other
            // updates (P[u], u > t+1) run during token t+1, in the latency gaps of
            // its chain, pinned there by scheduling barriers and empty asm.
            float chk = 0.f, cprev = 0.f, gprev[kGC];
#pragma unroll
            for (int t = 0; t < kGC; ++t) {
                // row t+1 of gt (G_{u,t+1}) from column t+2 on, in 16-byte reads
                float gnext[kGC];
#pragma unroll
                for (int q4 = (t + 2) / 4; q4 < kGC / 4; ++q4) {
                    const float4 x = *reinterpret_cast<const float4 *>(&sm.gt[gs][gj][t + 1 < kGC ? t + 1 : t][4 * q4]);
                    gnext[4 * q4] = x.x, gnext[4 * q4 + 1] = x.y;
                    gnext[4 * q4 + 2] = x.z, gnext[4 * q4 + 3] = x.w;
                }
                auto defer = [&](int part) {   // c_{t-1} into P[u], u > t, in four parts
                    if (t >= 1) {
                        const int F = kGC - 1 - t;
                        const int lo = t + 1 + F * part / 4, hi = t + 1 + F * (part + 1) / 4;
#pragma unroll
                        for (int u = lo; u < hi; ++u) {
                            P[u] = fmaf(gprev[u], cprev, P[u]);
                            asm volatile("" : "+v"(P[u]));
                        }
                    }
                };
                const float d = sv[t] - P[t];
                const float bd = sbeta[t] * d;
                const float ex = __builtin_amdgcn_exp2f(fmaf(-d, d, slk[t]));
                __builtin_amdgcn_sched_barrier(0);
                defer(0);
                __builtin_amdgcn_sched_barrier(0);
                float z = ex;
                if constexpr (JP >= 2) z += dpp_mov<0xb1>(z);   // lane ^ 1
                const float bdex = bd * ex;
                const float gb = t + 1 < kGC ? grow[t + 1] * bdex : 0.f;
                __builtin_amdgcn_sched_barrier(0);
                defer(1);
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (JP >= 4) z += dpp_mov<0x4e>(z);   // lane ^ 2
                __builtin_amdgcn_sched_barrier(0);
                defer(2);
                __builtin_amdgcn_sched_barrier(0);
                const float iz = rcp_fast(z);
                __builtin_amdgcn_sched_barrier(0);
                defer(3);
                __builtin_amdgcn_sched_barrier(0);
                if (t + 1 < kGC) P[t + 1] = fmaf(gb, iz, P[t + 1]);
                const float cs = bdex * iz;   // s c
                cc[t] = cs;
                if (wres) {   // (tokens past the end stay in registers)
                    if (t < nt)
                        a.resp[((((size_t)b * T + t0 + t) * H + h) * J + sj) * Dv + d0 + sdd] = ex * iz;
                }
                chk = fmaxf(chk, fmaxf(z, iz));
                cprev = cs;
#pragma unroll
                for (int u = t + 2; u < kGC; ++u) gprev[u] = grow[u], grow[u] = gnext[u];
            }
            // (an integer test on bits the compiler cannot trace back to a float:
            // a NaN, whose magnitude bits exceed those of 2^100, must fail it too)
            uint32_t chk_bits = __float_as_uint(chk);
            asm volatile("" : "+v"(chk_bits));
            const bool bad = (chk_bits & 0x7fffffffu) > 0x71800000u;   // 2^100
            if (__builtin_amdgcn_ballot_w64(sact && bad) != 0) {
                // some softmax sum left the range: the chunk again, maximum subtracted
                load_pred();
#pragma unroll
                for (int t = 0; t < kGC; ++t) {
                    float gnext[kGC];
#pragma unroll
                    for (int u = t + 2; u < kGC; ++u) gnext[u] = sm.gt[gs][gj][t + 1 < kGC ? t + 1 : t][u];
                    const float d = sv[t] - P[t];
                    const float e = fmaf(-d, d, slk[t]);
                    const float mx = group_max<JP>(e);
                    const float ex = sact ? __builtin_amdgcn_exp2f(e - mx) : 0.0f;
                    const float iz = rcp_fast(group_sum<JP>(ex));
                    const float cs = sact ? sbeta[t] * d * ex * iz : 0.0f;
#pragma unroll
                    for (int u = t + 1; u < kGC; ++u) P[u] = fmaf(grow[u], cs, P[u]);
                    cc[t] = cs;
                    if (wres) {
                        if (t < nt)
                            a.resp[((((size_t)b * T + t0 + t) * H + h) * J + sj) * Dv + d0 + sdd] = ex * iz;
                    }
#pragma unroll
                    for (int u = t + 2; u < kGC; ++u) grow[u] = gnext[u];
                }
            }
            if (sact) {
#pragma unroll
                for (int t4 = 0; t4 < kGC; t4 += 4)
                    *reinterpret_cast<float4 *>(&sm.c[n & 1][scol][t4]) =
                        make_float4(kInvS * cc[t4], kInvS * cc[t4 + 1], kInvS * cc[t4 + 2],
                                    kInvS * cc[t4 + 3]);
            }
            block_sync_lds();   // e(n)
            if (n + 1 < NCH) seq_inputs(n + 1);
            block_sync_lds();   // i(n+1)
        }
        block_sync_lds();   // epilogue
    } else {
        // ================= helper waves: inputs, priors, outputs =================
        const int bt = tid - 64 * (J + 1);
        constexpr int NBT = 64 * kGH;
        const bool obf = a.out_bf16;
        const uint16_t *const Kg = static_cast<const uint16_t *>(a.k);
        const uint16_t *const Qg = static_cast<const uint16_t *>(a.q);
        const uint16_t *const Vg = static_cast<const uint16_t *>(a.v);
        const uint16_t *const LBg = static_cast<const uint16_t *>(a.lb);
        const uint16_t *const LKg = static_cast<const uint16_t *>(a.lk);
        const uint16_t *const LQg = static_cast<const uint16_t *>(a.lq);
        const uint16_t *const Gg = static_cast<const uint16_t *>(a.decay);
        // one chunk's raw inputs, in registers from fetch to land
        constexpr int NKQ = ceil_div_c(kGC * DK / 8, NBT);   // uint4 of K (and of Q)
        constexpr int NLG = ceil_div_c(kGC * N / 8, NBT);    // uint4 of each logit tensor
        constexpr int NV = ceil_div_c(kGC * DB / 8, NBT);
        constexpr int NG = ceil_div_c(kGC * J * DK / 8, NBT);   // uint4 of the decay logits
        uint4 rk[NKQ], rq[NKQ], rlb[NLG], rlk[NLG], rlq[NLG], rv[NV], rg[NG];
        // Every thread loads every item it owns, from a clamped row (the last
        // token of the chunk, the last item): the loads go out back to back,
        // with no branch each.  land() zeroes what lies past the end, a phase
        // later, so that nothing here waits for the data.
        auto fetch = [&](int m) {
            const int t0 = m * kGC, nt = min(kGC, T - t0);
            const size_t row0 = (size_t)b * T + t0;
#pragma unroll
            for (int x = 0; x < NKQ; ++x) {
                const int e = min(bt + NBT * x, kGC * DK / 8 - 1);
                const int t = min(e / (DK / 8), nt - 1), p = e % (DK / 8);
                const size_t off = ((row0 + t) * H + h) * DK + 8 * p;
                rk[x] = *reinterpret_cast<const uint4 *>(Kg + off);
                rq[x] = *reinterpret_cast<const uint4 *>(Qg + off);
            }
#pragma unroll
            for (int x = 0; x < NLG; ++x) {
                const int e = min(bt + NBT * x, kGC * N / 8 - 1);
                const int t = min(e / (N / 8), nt - 1), rem = e % (N / 8);
                const int j = rem / (DB / 8), p = rem % (DB / 8);
                const size_t off = (((row0 + t) * H + h) * J + j) * Dv + d0 + 8 * p;
                rlb[x] = *reinterpret_cast<const uint4 *>(LBg + off);
                rlk[x] = *reinterpret_cast<const uint4 *>(LKg + off);
                rlq[x] = *reinterpret_cast<const uint4 *>(LQg + off);
            }
#pragma unroll
            for (int x = 0; x < NV; ++x) {
                const int e = min(bt + NBT * x, kGC * DB / 8 - 1);
                const int t = min(e / (DB / 8), nt - 1), p = e % (DB / 8);
                rv[x] = *reinterpret_cast<const uint4 *>(Vg + ((row0 + t) * H + h) * Dv + d0 + 8 * p);
            }
#pragma unroll
            for (int x = 0; x < NG; ++x) {
                const int e = min(bt + NBT * x, kGC * J * DK / 8 - 1);
                const int t = min(e / (J * DK / 8), nt - 1), p = e % (J * DK / 8);
                rg[x] = *reinterpret_cast<const uint4 *>(Gg + ((row0 + t) * H + h) * J * DK + 8 * p);
            }
        };
        // r, or zero when !keep (a mask: a select of the whole vector would be
        // made on addresses and put the registers in scratch memory)
        auto mask4 = [](const uint4 &r, bool keep) {
            const uint32_t m = keep ? 0xffffffffu : 0u;
            return make_uint4(r.x & m, r.y & m, r.z & m, r.w & m);
        };
        // chunk m's inputs but its decay logits to its slot
        auto land = [&](int m) {
            const int s3 = m % 3, nt = min(kGC, T - m * kGC);
#pragma unroll
            for (int x = 0; x < NKQ; ++x) {
                const int e = bt + NBT * x, t = e / (DK / 8), p = e % (DK / 8);
                if (e < kGC * DK / 8) {
                    // rows past the end are zero; two 8-byte stores (the padded
                    // rows are 8-byte aligned)
                    const uint4 kk = mask4(rk[x], t < nt), qq = mask4(rq[x], t < nt);
                    uint2 *dk = reinterpret_cast<uint2 *>(&sm.k[s3][t][8 * p]);
                    uint2 *dq = reinterpret_cast<uint2 *>(&sm.q[s3][t][8 * p]);
                    dk[0] = make_uint2(kk.x, kk.y);
                    dk[1] = make_uint2(kk.z, kk.w);
                    dq[0] = make_uint2(qq.x, qq.y);
                    dq[1] = make_uint2(qq.z, qq.w);
                }
            }
            // query-prior logits to the slot; beta = sigmoid(beta logit) and the
            // key-prior logits, and v, straight to the sequential wave's arrays
            // (chunk m's pair of them was last read in phase B of chunk m - 3)
#pragma unroll
            for (int x = 0; x < NLG; ++x) {
                const int e = bt + NBT * x, t = e / (N / 8), col8 = e % (N / 8);
                if (e < kGC * N / 8) {
                    const bool in = t < nt;
                    *reinterpret_cast<uint4 *>(&sm.lq[s3][t][8 * col8]) = mask4(rlq[x], in);
                    const uint32_t bw[4] = {rlb[x].x, rlb[x].y, rlb[x].z, rlb[x].w};
                    const uint32_t kw[4] = {rlk[x].x, rlk[x].y, rlk[x].z, rlk[x].w};
#pragma unroll
                    for (int y = 0; y < 8; ++y) {
                        const uint16_t hb = (uint16_t)(bw[y / 2] >> (16 * (y % 2)));
                        const uint16_t hk = (uint16_t)(kw[y / 2] >> (16 * (y % 2)));
                        sm.sq[m & 1][8 * col8 + y][t] =
                            make_float2(in ? sigmoid(bf(hb)) : 0.0f, in ? kLog2e * bf(hk) : 0.0f);
                    }
                }
            }
#pragma unroll
            for (int x = 0; x < NV; ++x) {
                const int e = bt + NBT * x, t = e / (DB / 8), p = e % (DB / 8);
                if (e < kGC * DB / 8) {
                    const uint32_t vw[4] = {rv[x].x, rv[x].y, rv[x].z, rv[x].w};
#pragma unroll
                    for (int y = 0; y < 8; ++y)
                        sm.vs[m & 1][8 * p + y][t] =
                            t < nt ? kS * bf((uint16_t)(vw[y / 2] >> (16 * (y % 2)))) : 0.0f;
                }
            }
        };
        // chunk m's decay logits, once the tile waves have taken chunk m - 1's
        auto land_g = [&](int m) {
            const int nt = min(kGC, T - m * kGC);
#pragma unroll
            for (int x = 0; x < NG; ++x) {
                const int e = bt + NBT * x, t = e / (J * DK / 8), p = e % (J * DK / 8);
                if (e < kGC * J * DK / 8)
                    *reinterpret_cast<uint4 *>(&sm.g[t][8 * p]) = mask4(rg[x], t < nt);
            }
        };
        // pi^q of chunk m: softmax over j of the query-prior logits, per (t, dd)
        auto priors = [&](int m) {
            const int s3 = m % 3;
            for (int e = bt; e < kGC * DB; e += NBT) {
                const int t = e / DB, dd = e % DB;
                float x[J], mx = -INFINITY, z = 0.0f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    x[j] = bf(sm.lq[s3][t][j * DB + dd]);
                    mx = fmaxf(mx, x[j]);
                }
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    x[j] = __builtin_amdgcn_exp2f(kLog2e * (x[j] - mx));
                    z += x[j];
                }
                const float iz = rcp_fast(z);
#pragma unroll
                for (int j = 0; j < J; ++j) sm.pq[m & 1][t][j * DB + dd] = J == 1 ? 1.0f : x[j] * iz;
            }
        };
        // output of chunk m: o = sum_j pi^q y
        auto output = [&](int m) {
            const int mt0 = m * kGC, nt = min(kGC, T - mt0);
            for (int e = bt; e < kGC * DB; e += NBT) {
                const int t = e / DB, dd = e % DB;
                if (t >= nt) continue;
                float o = 0.0f;
#pragma unroll
                for (int j = 0; j < J; ++j) o += sm.py[m & 1][t][j * DB + dd];
                store1(a.o, (((size_t)b * T + mt0 + t) * H + h) * Dv + d0 + dd, o, obf);
            }
        };

        block_sync_lds();   // prologue 1
        fetch(0);
        land(0);
        land_g(0);
        if (NCH > 1) {
            fetch(1);
            land(1);
        }
        block_sync_lds();   // prologue 2
        block_sync_lds();   // prologue 3: the tile waves have read chunk 0's decay logits
        if (NCH > 1) land_g(1);
        if (NCH > 2) fetch(2);
        block_sync_lds();   // prologue 4
        for (int n = 0; n < NCH; ++n) {
            priors(n);
            if (n >= 2) output(n - 2);
            // chunk n + 2 lands in the slots of chunk n - 1
            if (n + 2 < NCH) land(n + 2);
            block_sync_lds();   // e(n)
            // its decay logits in phase B, when those of chunk n + 1 have been read
            if (n + 2 < NCH) land_g(n + 2);
            if (n + 3 < NCH) fetch(n + 3);
            block_sync_lds();   // i(n+1)
        }
        if (NCH >= 2) output(NCH - 2);
        block_sync_lds();   // epilogue
        output(NCH - 1);
    }
}

template <int DK, int J, int DB>
hipError_t launch_g(const LayerArgs &a, hipStream_t stream) {
    using C = GCfg<DK, J, DB>;
    static_assert(sizeof(GSmem<DK, J, DB>) <= 160 * 1024, "LDS");
    const long blocks = (long)(a.Dv / DB) * a.H * a.B;
    hipLaunchKernelGGL((scan_gated_chunk_kernel<DK, J, DB>), dim3((unsigned)blocks),
                       dim3(64 * C::NWAVE), 0, stream, a);
    return hipGetLastError();
}

template <int DK, int J>
hipError_t launch_gj(const LayerArgs &a, hipStream_t stream) {
    if constexpr (J * DK > 512) {
        return hipErrorInvalidValue;
    } else {
        // 16 output dims per block once that grid fills the chip; 8 below
        if (a.Dv % 16 == 0 && (long)(a.Dv / 16) * a.H * a.B >= 256)
            return launch_g<DK, J, 16>(a, stream);
        return launch_g<DK, J, 8>(a, stream);
    }
}

template <int DK>
hipError_t launch_gdk(const LayerArgs &a, hipStream_t stream) {
    switch (a.J) {
        case 1: return launch_gj<DK, 1>(a, stream);
        case 2: return launch_gj<DK, 2>(a, stream);
        case 3: return launch_gj<DK, 3>(a, stream);
        case 4: return launch_gj<DK, 4>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

bool gated_chunk_supported(const LayerArgs &a) {
    return a.in_bf16 && a.decay && !a.gk && !a.delta_out && !a.ckpt && a.J >= 1 && a.J <= 4 &&
           a.J * a.Dk <= 512 && a.Dv % 8 == 0 &&
           (a.Dk == 16 || a.Dk == 32 || a.Dk == 64 || a.Dk == 128);
}

hipError_t launch_scan_gated_chunk(const LayerArgs &a, hipStream_t stream) {
    if (!gated_chunk_supported(a) || a.T <= 0) return hipErrorInvalidValue;
    switch (a.Dk) {
        case 16: return launch_gdk<16>(a, stream);
        case 32: return launch_gdk<32>(a, stream);
        case 64: return launch_gdk<64>(a, stream);
        case 128: return launch_gdk<128>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace swila
