// Backward pass of the plain SwiLA forward (Sec. 3.2: eq. recurrence,
// eq. responsibility, eq. retrieval; beta and the priors from logits as in
// App. B.2): the gradients of a loss L with respect to q, k, v, the three
// logit tensors and the initial state, given dL/do and dL/dW_T.  The paper
// trains through its sequential evaluation; this is the exact gradient of
// that forward, in three launches.
//
// 1. Forward recompute: delta_{tjd} of every token and the state W_n before
//    every kBwdChunk-th token.  bf16 inputs run the matrix-core chunk scan with
//    these outputs in place of o, fp32 inputs the token-by-token scan in its AX
//    mode, as their forwards do.
//
// 2. Reverse scan.  With G_{jd} = dL/dw_{t,jd}, per token in reverse:
//      dy_j = do pi^q_j;  G_j += dy_j q_t;  dc_j = G_j . k_t
//      r = softmax_j(lk - delta^2/2) and beta recomputed from delta and logits
//      dlb_j = dc_j r_j delta_j beta_j (1 - beta_j)
//      dr_j = dc_j beta_j delta_j;  da_j = r_j (dr_j - sum_i r_i dr_i) = dlk_j
//      ddelta_j = dc_j beta_j r_j - delta_j da_j;  dv = sum_j ddelta_j
//      dpred_j = -ddelta_j;  G_j += dpred_j k_t          (now dL/dw_{t-1,jd})
//    evaluated a chunk at a time (reverse_chunk_kernel below).  It writes dv,
//    dlb, dlk, dL/dW_0 (G after token 0), and E_n, the part of dL/dw at the
//    last token of checkpoint interval n that comes from later tokens; and, for
//    the chunk pass, c = beta r delta, dpred, pi^q and dL/do in that pass's tile
//    order, so that each of its tiles reads one contiguous run per operand.
//
// 3. Chunk pass, one block per (b, h, chunk of kBwdChunk tokens), no
//    sequential dependence.  Inside chunk n, with S = W_n, columns col = (j, d)
//    and per-(token, column) scalars C = c = beta r delta, P = dpred, Y = dy:
//      w_t     = S + sum_{s<=t} C_s k_s,     w_{t-1} = S + sum_{s<t} C_s k_s
//      G_t     = E_n + sum_{s>t} P_s k_s + sum_{s>=t} Y_s q_s
//    so the two sums over columns that need the per-token state become
//      dq_t = Y_t.S + sum_{s<=t} (Y_t.C_s) k_s
//      dk_t = C_t.E_n + P_t.S + sum_{s>t} (C_t.P_s) k_s + sum_{s<t} (P_t.C_s) k_s
//             + sum_{s>=t} (C_t.Y_s) q_s
//    (X_t.Z_s = sum over columns of X_{t,col} Z_{s,col}): contractions of
//    chunk-sized operands.  The query-prior logit gradient needs the
//    retrievals y_{tjd} = w_{t,jd} . q_t = (Q S + tril(Q K^T) C)_{t,col}:
//    dlq_j = pi^q_j do (y_j - sum_i pi^q_i y_i).  Column tiles of all J
//    components of DT output dims stream through LDS; every product runs on the
//    matrix cores in fp32 (16 x 16 output tiles spread over the four waves),
//    and the intra-chunk sums become three masked C x C coefficient matrices
//    applied to the chunk's K and Q at the end.
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

constexpr int kThreads = 256;
constexpr int kCB = kBwdChunk;    // tokens per chunk of the chunk pass

template <bool B>
struct BTag {
    static constexpr bool value = B;
};
template <int N>
struct ITag {
    static constexpr int value = N;
};

// The kernels below order only LDS traffic at their barriers (block_sync_lds):
// a full __syncthreads would also wait for every global load in flight, and
// with it for the next chunk's prefetch.  Their staging loads raw bits
// (raw1, raw4) and converts later.

// Output dims per column tile of the chunk pass: tiles of all J components of
// DT dims, 16 to 32 columns.
template <int J>
constexpr int chunk_tile_dims() { return J == 1 ? 16 : J == 3 ? 8 : 32 / J; }

// Chunked reverse scan.  The recurrence of the reverse sweep has the shape of
// the forward's chunk form run backwards: inside a chunk of kRC tokens, with E
// the gradient w.r.t. the state after the chunk's last token from the tokens
// that follow it,
//   dc_t = k_t . E + sum_{s>=t} (k_t . q_s) dy_s + sum_{s>t} (k_t . k_s) dpred_s
// and dpred_t is linear in the J values dc_t of its output dim.  So per chunk:
// the Gram products K K^T, K Q^T and the base K E + triu(K Q^T) Y in parallel;
// one wave then runs the chunk's tokens in reverse, one lane per column (all J
// components of DB output dims, J lanes adjacent), with the later tokens'
// dpred folded in as deferred updates; last E += Q^T Y + K^T P.  With fp32
// inputs every product is fp32 on the vector ALUs.  With bf16 inputs the
// products run on the matrix cores: K and Q are exact in bf16, so K K^T and
// K Q^T are single products; E, Y, P and the Gram values are fp32, split into
// a bf16 high part and a bf16 residual (about 2^-17 relative per operand,
// fp32 accumulation).
constexpr int kRC = 16;   // tokens per chunk of the reverse scan

typedef short short4v __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
typedef float floatx2v __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// two fp32 values to packed bf16 (round to nearest; a in the low half), and
// their residuals
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2v{a, b}, bf16x2v));
}
__device__ __forceinline__ void split_pk(float a, float b, uint32_t &hi, uint32_t &lo) {
    hi = pk_bf16(a, b);
    lo = pk_bf16(a - __uint_as_float(hi << 16), b - __uint_as_float(hi & 0xffff0000u));
}
// The k operand of a lane: M values (4 for the 16-deep product, 8 for the
// 32-deep one) as bf16, or as high parts and residuals
template <int M>
struct KOp {
    uint32_t hi[M / 2], lo[M / 2];
};
template <int M>
__device__ __forceinline__ KOp<M> kop_exact(const float *x) {
    KOp<M> o;
#pragma unroll
    for (int m = 0; m < M / 2; ++m) o.hi[m] = pk_bf16(x[2 * m], x[2 * m + 1]), o.lo[m] = 0u;
    return o;
}
template <int M>
__device__ __forceinline__ KOp<M> kop_split(const float *x) {
    KOp<M> o;
#pragma unroll
    for (int m = 0; m < M / 2; ++m) split_pk(x[2 * m], x[2 * m + 1], o.hi[m], o.lo[m]);
    return o;
}
__device__ __forceinline__ floatx4 mma(const uint32_t (&a)[2], const uint32_t (&b)[2], floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(short4v, make_uint2(a[0], a[1])),
                                                     __builtin_bit_cast(short4v, make_uint2(b[0], b[1])),
                                                     c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mma(const uint32_t (&a)[4], const uint32_t (&b)[4], floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        __builtin_bit_cast(bf16x8, make_uint4(a[0], a[1], a[2], a[3])),
        __builtin_bit_cast(bf16x8, make_uint4(b[0], b[1], b[2], b[3])), c, 0, 0, 0);
}

// J consecutive floats to global memory (16-byte stores where J allows).
template <int J>
__device__ __forceinline__ void st_row(float *p, const float (&v)[J]) {
    if constexpr (J % 4 == 0) {
#pragma unroll
        for (int x = 0; x < J; x += 4)
            *reinterpret_cast<float4 *>(p + x) = make_float4(v[x], v[x + 1], v[x + 2], v[x + 3]);
    } else if constexpr (J == 2) {
        *reinterpret_cast<float2 *>(p) = make_float2(v[0], v[1]);
    } else {
#pragma unroll
        for (int x = 0; x < J; ++x) p[x] = v[x];
    }
}

// IBF: bf16 inputs (the input dtype is fixed per instantiation, so that the
// prefetch has one load variant; dL/do's dtype stays a run-time choice).
//
// Schedule.  fp32 inputs: per chunk, every thread stages the chunk, then the
// Gram products, the base, the sequential wave's tokens, and the update of E,
// each step between block barriers.  bf16 inputs: the staged inputs have two slots (chunk m in
// slot m & 1) and three barriers per chunk:
//   A  the sequential wave runs chunk n's tokens; the other waves store
//      chunk n+1's dv and the chunk pass's dpred of chunk n+1,
//      stage chunk n-1 into the other slot from registers (storing its pi^q, c
//      and dL/do for the chunk pass) and issue the loads of chunk n-2
//   B  E += Q_n^T Y_n + K_n^T P_n; waves 2 and 3 also the Gram products of
//      chunk n-1
//   C  the base of chunk n-1 from the new E (one wave per 16-column tile);
//      chunk n's outputs on waves 2 and 3 when there are two tiles or fewer,
//      else in B.
template <int DK, int J, int DB, bool IBF>
__global__ __launch_bounds__(kThreads) void reverse_chunk_kernel(BackwardArgs a) {
    constexpr int JP = J == 3 ? 4 : J;   // lanes per output dim (J = 3 padded)
    constexpr int N = J * DB;            // columns, col = j * DB + dd
    constexpr int NL = JP * DB;          // sequential lanes, lane = dd * JP + j
    constexpr int KP = DK + 4;           // row pitches keep 16-byte rows
    constexpr int CP = N + 4, GP = kRC + 4;
    static_assert(NL <= 64 && kBwdChunk % kRC == 0 && N % 4 == 0, "one sequential wave");
    static_assert(DB % chunk_tile_dims<J>() == 0 || chunk_tile_dims<J>() % DB == 0,
                  "a block covers whole tiles of the chunk pass, or a part of one");
    constexpr int NS = IBF ? 2 : 1;      // slots of the staged inputs
    constexpr int KT = IBF ? 1 : DK;     // rows of K and Q transposed (fp32 products only)

    __shared__ __align__(16) float sE[DK][CP];
    __shared__ __align__(16) float sK[NS][kRC][KP], sQ[NS][kRC][KP];   // rows t
    __shared__ __align__(16) float sKt[KT][GP], sQt[KT][GP];           // the same, [i][t]
    __shared__ __align__(16) float sGkk[kRC][GP];                      // k_t . k_s (symmetric)
    __shared__ __align__(16) float sGkqT[kRC][GP];                     // [s][t] = k_t . q_s
    __shared__ __align__(16) float sBase[kRC][CP], sY[NS][kRC][CP], sP[NS][kRC][CP];
    __shared__ float sDelta[NS][kRC][CP], sBeta[NS][kRC][CP], sR[NS][kRC][CP];
    __shared__ float sDc[kRC][CP], sDlk[kRC][CP];   // dc, da

    const LayerArgs &f = a.f;
    const int tid = threadIdx.x, lane = tid % 64;
    // matrix-core lane coordinates: row / column tl, k slot lg
    const int wv = __builtin_amdgcn_readfirstlane(tid / 64), tl = lane % 16, lg = lane / 16;
    constexpr int NTC = (N + 15) / 16;    // 16-column tiles
    constexpr int KM = DK >= 32 ? 8 : 4;  // k values per lane: 32- or 16-deep products
    const int H = f.H, T = f.T, Dv = f.Dv;
    // Workgroups go to the eight XCDs (each with its own L2) round-robin by
    // index; every column block of a head is placed on the same XCD, so that
    // the head's K and Q rows and the shared cache lines of its per-token
    // scalars are fetched from HBM once.
    const int NDB = Dv / DB, NH = f.B * H, L = blockIdx.x;
    int hh, db;
    if (NH % 8 == 0) {
        const int xs = L / 8;
        hh = 8 * (xs / NDB) + L % 8;
        db = xs % NDB;
    } else {
        hh = L / NDB;
        db = L % NDB;
    }
    const int d0 = db * DB, h = hh % H, b = hh / H;
    constexpr bool ibf = IBF;
    const bool obf = f.out_bf16;
    const int NCH = (T + kRC - 1) / kRC;
    const int NC2 = (T + kBwdChunk - 1) / kBwdChunk;
    constexpr int R2 = kBwdChunk / kRC;   // reverse chunks per checkpoint interval
    const size_t sbase = ((size_t)b * H + h) * J * DK * Dv;

    // E = dL/dW_T (or 0), [i][col]
    for (int e = tid; e < DK * N; e += kThreads) {
        const int i = e / N, col = e % N, j = col / DB, dd = col % DB;
        sE[i][col] = a.grad_state ? a.grad_state[sbase + ((size_t)j * DK + i) * Dv + d0 + dd] : 0.0f;
    }
    // this lane's column in the sequential wave
    const int sj = lane % JP, sdd = lane / JP;
    const bool sact = tid < 64 && lane < NL && sj < J;
    const int scol = sact ? sj * DB + sdd : 0;

    // Each chunk's HBM inputs are fetched into registers while a later chunk
    // computes: K and Q rows as float4, and per (token, output dim) the J
    // errors and logits and dL/do.  The staging threads (F0 .. kThreads - 1)
    // load them and later stage them.  Every such thread loads every item it
    // owns, from a clamped row (the chunk's last token, the last item), with the
    // input dtype fixed at compile time: no load sits behind a branch (a load
    // there is waited for at the join); staging zeroes what lies past the end.
    constexpr int F0 = IBF ? 64 : 0, FT = kThreads - F0;
    constexpr int NKQ = (kRC * (DK / 4) + FT - 1) / FT;
    constexpr int NSC = (kRC * DB + FT - 1) / FT;
    uint4 pk[NKQ] = {}, pq[NKQ] = {};   // (bf16: halves x and y)
    float pdl[NSC][J];
    uint32_t plk[NSC][J], plq[NSC][J], plb[NSC][J], pdo[NSC];
    const int ft = tid - F0;   // index among the staging threads (when >= 0)
    auto fetch_as = [&](int n, auto otag) {
        constexpr bool BF = IBF, OBF = decltype(otag)::value;
        const int t0 = n * kRC, nt = min(kRC, T - t0);
#pragma unroll
        for (int x = 0; x < NKQ; ++x) {
            const int e = min(ft + FT * x, kRC * (DK / 4) - 1);
            const int t = min(e / (DK / 4), nt - 1), i = (e % (DK / 4)) * 4;
            const size_t off = ((size_t)(b * T + t0 + t) * H + h) * DK + i;
            if constexpr (BF) {
                const uint2 kk = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(f.k) + off);
                const uint2 qq = *reinterpret_cast<const uint2 *>(static_cast<const uint16_t *>(f.q) + off);
                pk[x].x = kk.x, pk[x].y = kk.y;
                pq[x].x = qq.x, pq[x].y = qq.y;
            } else {
                pk[x] = *reinterpret_cast<const uint4 *>(static_cast<const float *>(f.k) + off);
                pq[x] = *reinterpret_cast<const uint4 *>(static_cast<const float *>(f.q) + off);
            }
        }
#pragma unroll
        for (int x = 0; x < NSC; ++x) {
            const int e = min(ft + FT * x, kRC * DB - 1);
            const int t = min(e / DB, nt - 1), dd = e % DB;
            const size_t row = (size_t)(b * T + t0 + t) * H + h;
            // dL/do has the output dtype
            if constexpr (OBF) pdo[x] = static_cast<const uint16_t *>(a.grad_o)[row * Dv + d0 + dd];
            else pdo[x] = static_cast<const uint32_t *>(a.grad_o)[row * Dv + d0 + dd];
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const size_t idx = (row * J + j) * Dv + d0 + dd;
                pdl[x][j] = a.delta[idx];
                if constexpr (BF) {
                    plk[x][j] = static_cast<const uint16_t *>(f.lk)[idx];
                    plq[x][j] = static_cast<const uint16_t *>(f.lq)[idx];
                    plb[x][j] = static_cast<const uint16_t *>(f.lb)[idx];
                } else {
                    plk[x][j] = static_cast<const uint32_t *>(f.lk)[idx];
                    plq[x][j] = static_cast<const uint32_t *>(f.lq)[idx];
                    plb[x][j] = static_cast<const uint32_t *>(f.lb)[idx];
                }
            }
        }
    };
    auto fetch = [&](int n) {
        if (obf) fetch_as(n, BTag<true>{});
        else fetch_as(n, BTag<false>{});
    };
    // The chunk pass's operands, in its tile order [b, h, interval, tile, token,
    // dd, j]: the rows of one tile and consecutive tokens are contiguous, so each
    // store run covers whole lines.  This block's dims cover TW dims of each tile
    // it touches (all of them, or a part when the block is narrower than a
    // tile).  Threads first .. first + nthr - 1 store X[t][col] for the chunk's
    // tokens (trip counts and divisors compile-time; tokens past the end skipped).
    constexpr int CT = chunk_tile_dims<J>();
    constexpr int TW = DB < CT ? DB : CT;
    auto pack_index = [&](int t0, int t, int d) {
        const size_t pbase = ((size_t)b * H + h) * NC2 + t0 / kBwdChunk;
        return ((pbase * (Dv / CT) + d / CT) * kBwdChunk + t0 % kBwdChunk + t) * CT + d % CT;
    };
    // chunk n's registers to slot sl: K, Q (and their transposes for the fp32
    // products), delta, r, beta and dy = dL/do pi^q; and, from the same
    // registers, the chunk pass's operands pi^q, c = beta r delta and dL/do (a
    // thread's J components are adjacent there)
    auto stage = [&](int n, int sl) {
        const int t0 = n * kRC, nt = min(kRC, T - t0);
#pragma unroll
        for (int x = 0; x < NKQ; ++x) {
            const int e = ft + FT * x, t = e / (DK / 4), i = (e % (DK / 4)) * 4;
            if ((kRC * (DK / 4)) % FT == 0 || e < kRC * (DK / 4)) {
                float4 kv = cvt4(pk[x], ibf), qv = cvt4(pq[x], ibf);
                if (t >= nt) kv.x = kv.y = kv.z = kv.w = qv.x = qv.y = qv.z = qv.w = 0.0f;
                *reinterpret_cast<float4 *>(&sK[sl][t][i]) = kv;
                *reinterpret_cast<float4 *>(&sQ[sl][t][i]) = qv;
                if constexpr (!IBF) {
                    sKt[i][t] = kv.x, sKt[i + 1][t] = kv.y, sKt[i + 2][t] = kv.z, sKt[i + 3][t] = kv.w;
                    sQt[i][t] = qv.x, sQt[i + 1][t] = qv.y, sQt[i + 2][t] = qv.z, sQt[i + 3][t] = qv.w;
                }
            }
        }
#pragma unroll
        for (int x = 0; x < NSC; ++x) {
            const int e = ft + FT * x, t = e / DB, dd = e % DB;
            if ((kRC * DB) % FT != 0 && e >= kRC * DB) continue;
            float dl[J], ee[J], lq[J], be[J];
            const float dov = t < nt ? cvt1(pdo[x], obf) : 0.0f;
            if (t < nt) {
                float m = -INFINITY, mq = -INFINITY;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    dl[j] = pdl[x][j];
                    ee[j] = cvt1(plk[x][j], ibf) - 0.5f * dl[j] * dl[j];
                    lq[j] = cvt1(plq[x][j], ibf);
                    be[j] = 1.0f / (1.0f + exp_fast(-cvt1(plb[x][j], ibf)));
                    m = fmaxf(m, ee[j]);
                    mq = fmaxf(mq, lq[j]);
                }
                float z = 0.0f, zq = 0.0f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    ee[j] = exp_fast(ee[j] - m);
                    z += ee[j];
                    lq[j] = exp_fast(lq[j] - mq);
                    zq += lq[j];
                }
                const float iz = 1.0f / z, izq = 1.0f / zq;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    ee[j] = J == 1 ? 1.0f : ee[j] * iz;       // r
                    lq[j] = J == 1 ? 1.0f : lq[j] * izq;      // pi^q
                }
            } else {
#pragma unroll
                for (int j = 0; j < J; ++j) dl[j] = ee[j] = lq[j] = be[j] = 0.0f;
            }
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int col = j * DB + dd;
                sDelta[sl][t][col] = dl[j];
                sR[sl][t][col] = ee[j];
                sBeta[sl][t][col] = be[j];
                sY[sl][t][col] = dov * lq[j];
            }
            if (t < nt) {
                const size_t pr = pack_index(t0, t, d0 + dd);
                float cv[J];
#pragma unroll
                for (int j = 0; j < J; ++j) cv[j] = be[j] * ee[j] * dl[j];
                st_row<J>(a.qpk + pr * J, lq);
                st_row<J>(a.cpk + pr * J, cv);
                a.dopk[pr] = dov;
            }
        }
    };
    // dst[(tile row of (t, d)) * JJ + j] = val(t, j, dd) for the chunk's tokens,
    // by threads first .. first + nthr - 1 (compile-time: the loop is unrolled
    // and every LDS read is issued before the first store)
    auto pack_store = [&](float *dst, auto jj, auto val, int t0, int nt, auto first, auto nthr) {
        constexpr int JJ = decltype(jj)::value, F = decltype(first)::value;
        constexpr int NT = decltype(nthr)::value, NE = kRC * JJ * DB, NI = (NE + NT - 1) / NT;
        float v[NI];
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = min(tid - F + NT * x, NE - 1);
            const int j = e % JJ, w = (e / JJ) % TW, t = (e / (JJ * TW)) % kRC,
                      kk = e / (JJ * TW * kRC);
            v[x] = val(t, j, kk * TW + w);
        }
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = tid - F + NT * x;
            const int j = e % JJ, w = (e / JJ) % TW, t = (e / (JJ * TW)) % kRC,
                      kk = e / (JJ * TW * kRC);
            if ((NE % NT == 0 || e < NE) && t < nt)
                dst[pack_index(t0, t, d0 + kk * TW + w) * JJ + j] = v[x];
        }
    };
    // dv of chunk n = -(sum over j of its dpred, slot sl), summed in the pairs
    // of a J-lane reduction, by threads first .. first + nthr - 1
    auto dv_store = [&](int n, int sl, auto first, auto nthr) {
        constexpr int F = decltype(first)::value, NT = decltype(nthr)::value;
        constexpr int NE = kRC * DB, NI = (NE + NT - 1) / NT;
        const int t0 = n * kRC, nt = min(kRC, T - t0);
        float v[NI];
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = min(tid - F + NT * x, NE - 1), t = e / DB, dd = e % DB;
            float p[JP];
#pragma unroll
            for (int j = 0; j < JP; ++j) p[j] = j < J ? sP[sl][t][j * DB + dd] : 0.0f;
#pragma unroll
            for (int w = 1; w < JP; w *= 2)
#pragma unroll
                for (int j = 0; j < JP; j += 2 * w) p[j] += p[j + w];
            v[x] = -p[0];
        }
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = tid - F + NT * x, t = e / DB, dd = e % DB;
            if ((NE % NT == 0 || e < NE) && t < nt)
                a.dv[((size_t)(b * T + t0 + t) * H + h) * Dv + d0 + dd] = v[x];
        }
    };
    // dpred of chunk n (its tokens' results in slot sl)
    auto packs_dpred = [&](int n, int sl, auto first, auto nthr) {
        const int t0 = n * kRC, nt = min(kRC, T - t0);
        pack_store(a.ppk, ITag<J>{}, [&](int t, int j, int dd) { return sP[sl][t][j * DB + dd]; },
                   t0, nt, first, nthr);
    };
    // E_m (the gradient from the tokens after checkpoint interval m) before
    // the interval's last reverse chunk runs: [.., m, d, j, i], four key indices
    // per store, all LDS reads issued first
    auto checkpoint = [&](int n, auto first, auto nthr) {
        constexpr int F = decltype(first)::value, NT = decltype(nthr)::value;
        constexpr int NE4 = DB * J * DK / 4, NI = (NE4 + NT - 1) / NT;
        if (n % R2 == R2 - 1 || n == NCH - 1) {
            const int m = n / R2;
            float *ck = a.eck + ((((size_t)b * H + h) * NC2 + m) * Dv + d0) * J * DK;
            float4 v[NI];
#pragma unroll
            for (int x = 0; x < NI; ++x) {
                const int e = min(tid - F + NT * x, NE4 - 1);
                const int dd = e / (J * DK / 4), j = (e / (DK / 4)) % J, i = (e % (DK / 4)) * 4;
                const int col = j * DB + dd;
                v[x] = make_float4(sE[i][col], sE[i + 1][col], sE[i + 2][col], sE[i + 3][col]);
            }
#pragma unroll
            for (int x = 0; x < NI; ++x) {
                const int e = tid - F + NT * x;
                if (NE4 % NT == 0 || e < NE4) reinterpret_cast<float4 *>(ck)[e] = v[x];
            }
        }
    };
    // Gram products of the chunk in slot sl: on the matrix cores (bf16 inputs;
    // wave 2 K K^T, wave 3 K Q^T), else one (t, s) pair per thread
    auto gram = [&](int sl) {
        if constexpr (IBF) {
            if (wv >= 2) {
                // D[row][col] = sum_i A[row][i] K[col][i], A = K (D[t][s]) or Q
                // (D[s][t] = k_t . q_s); lane: row / col tl, k slot lg
                const float (*A)[KP] = wv == 2 ? sK[sl] : sQ[sl];
                floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i0 = 0; i0 < DK; i0 += KM * 4) {
                    const KOp<KM> a8 = kop_exact<KM>(&A[tl][i0 + KM * lg]);
                    const KOp<KM> b8 = kop_exact<KM>(&sK[sl][tl][i0 + KM * lg]);
                    acc = mma(a8.hi, b8.hi, acc);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (wv == 2) sGkk[4 * lg + r][tl] = acc[r];
                    else sGkqT[4 * lg + r][tl] = acc[r];
                }
            }
        } else {
            const int t = tid / kRC, s2 = tid % kRC;
            float gkk = 0.0f, gkq = 0.0f;
#pragma unroll 4
            for (int i = 0; i < DK; i += 4) {
                const float4 kt = *reinterpret_cast<const float4 *>(&sK[sl][t][i]);
                const float4 ks = *reinterpret_cast<const float4 *>(&sK[sl][s2][i]);
                const float4 qs = *reinterpret_cast<const float4 *>(&sQ[sl][s2][i]);
                gkk = fmaf(kt.x, ks.x, fmaf(kt.y, ks.y, fmaf(kt.z, ks.z, fmaf(kt.w, ks.w, gkk))));
                gkq = fmaf(kt.x, qs.x, fmaf(kt.y, qs.y, fmaf(kt.z, qs.z, fmaf(kt.w, qs.w, gkq))));
            }
            sGkk[t][s2] = gkk;
            sGkqT[s2][t] = gkq;
        }
    };
    // base_t = k_t . E + sum_{s>=t} (k_t . q_s) dy_s for the chunk in slot sl: a
    // 16-column tile per wave on the matrix cores (bf16 inputs), else four
    // tokens per thread
    auto base = [&](int sl) {
        if constexpr (IBF) {
            for (int ct = wv; ct < NTC; ct += kThreads / 64) {
                const int col = 16 * ct + tl;
                const bool cv = col < N;
                floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int i0 = 0; i0 < DK; i0 += KM * 4) {
                    const KOp<KM> a8 = kop_exact<KM>(&sK[sl][tl][i0 + KM * lg]);   // K[t = tl][i]
                    float ev[KM];
#pragma unroll
                    for (int m = 0; m < KM; ++m) ev[m] = cv ? sE[i0 + KM * lg + m][col] : 0.0f;
                    const KOp<KM> b8 = kop_split<KM>(ev);
                    acc = mma(a8.hi, b8.hi, acc);
                    acc = mma(a8.hi, b8.lo, acc);
                }
                // triu: A[t = tl][s = 4 lg + m] = k_t . q_s for s >= t, B = dy[s][col]
                float gv[4], yv[4];
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const int s2 = 4 * lg + m;
                    gv[m] = s2 >= tl ? sGkqT[s2][tl] : 0.0f;
                    yv[m] = cv ? sY[sl][s2][col] : 0.0f;
                }
                const KOp<4> ga = kop_split<4>(gv), yb = kop_split<4>(yv);
                acc = mma(ga.hi, yb.hi, acc);
                acc = mma(ga.hi, yb.lo, acc);
                acc = mma(ga.lo, yb.hi, acc);
                if (cv) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) sBase[4 * lg + r][col] = acc[r];
                }
            }
        } else {
            for (int e = tid; e < (kRC / 4) * N; e += kThreads) {
                const int t4 = (e / N) * 4, col = e % N;
                float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
                for (int i = 0; i < DK; ++i) {
                    const float4 kv = *reinterpret_cast<const float4 *>(&sKt[i][t4]);
                    const float ev = sE[i][col];
                    acc[0] = fmaf(kv.x, ev, acc[0]);
                    acc[1] = fmaf(kv.y, ev, acc[1]);
                    acc[2] = fmaf(kv.z, ev, acc[2]);
                    acc[3] = fmaf(kv.w, ev, acc[3]);
                }
                for (int s2 = t4; s2 < kRC; ++s2) {
                    const float4 gq = *reinterpret_cast<const float4 *>(&sGkqT[s2][t4]);
                    const float yv = sY[sl][s2][col];
                    // only s >= t: token t4 + x takes s2 >= t4 + x
                    acc[0] = fmaf(gq.x, yv, acc[0]);
                    if (s2 >= t4 + 1) acc[1] = fmaf(gq.y, yv, acc[1]);
                    if (s2 >= t4 + 2) acc[2] = fmaf(gq.z, yv, acc[2]);
                    if (s2 >= t4 + 3) acc[3] = fmaf(gq.w, yv, acc[3]);
                }
#pragma unroll
                for (int x = 0; x < 4; ++x) sBase[t4 + x][col] = acc[x];
            }
        }
    };
    // the chunk's tokens in reverse, by the sequential wave (tid < 64)
    // With c_j = beta_j r_j delta_j and sdr = sum_i c_i dc_i over the token's J
    // components, the per-token step above reads
    //   da_j = c_j dc_j - r_j sdr
    //   ddelta_j = beta_j r_j (1 - delta_j^2) dc_j + r_j delta_j sdr
    // (one component: ddelta = beta dc), so that the dependent chain from one
    // token's dc to the next is a product, the J-lane sum and two fused
    // multiply-adds.
    auto tokens = [&](int sl) {
        // dfr[u] starts at base_u and collects sum_{s>u} (k_u . k_s) dpred_s: dc_u
        float dfr[kRC], vd[kRC], vbe[kRC], vr[kRC];
        const int scw = sact ? scol : N;
#pragma unroll
        for (int u = 0; u < kRC; ++u) {
            dfr[u] = sact ? sBase[u][scol] : 0.0f;
            vd[u] = sact ? sDelta[sl][u][scol] : 0.0f;
            vbe[u] = sact ? sBeta[sl][u][scol] : 0.0f;
            vr[u] = sact ? sR[sl][u][scol] : 0.0f;
        }
        // rows of K K^T (= columns), the part u < t: row t - 1 is read while
        // token t runs, a token ahead of its use
        float grow[2][kRC];
#pragma unroll
        for (int u4 = 0; u4 < kRC / 4; ++u4) {
            const float4 x = *reinterpret_cast<const float4 *>(&sGkk[kRC - 1][4 * u4]);
            float *g = grow[(kRC - 1) & 1];
            g[4 * u4] = x.x, g[4 * u4 + 1] = x.y, g[4 * u4 + 2] = x.z, g[4 * u4 + 3] = x.w;
        }
#pragma unroll
        for (int t = kRC - 1; t >= 0; --t) {
#pragma unroll
            for (int u4 = 0; u4 < (t + 2) / 4; ++u4) {   // row t - 1
                const float4 x = *reinterpret_cast<const float4 *>(&sGkk[t - 1][4 * u4]);
                float *g = grow[(t - 1) & 1];
                g[4 * u4] = x.x, g[4 * u4 + 1] = x.y, g[4 * u4 + 2] = x.z, g[4 * u4 + 3] = x.w;
            }
            // (the scheduler would sink these loads to their use: no LDS read may
            // cross here; arithmetic and LDS writes may)
            __builtin_amdgcn_sched_barrier(0x207);
            const float dc = dfr[t];
            const float dl = vd[t], br = vbe[t] * vr[t], r = vr[t];
            float da = 0.0f, ddelta = br * dc;
            if constexpr (J > 1) {
                const float c = br * dl, g = fmaf(-c, dl, br);   // beta r (1 - delta^2)
                const float cdc = c * dc;
                const float sdr = group_sum<JP>(cdc);
                da = fmaf(-r, sdr, cdc);
                ddelta = fmaf(r * dl, sdr, g * dc);
            }
            const float dpred = -ddelta;
            // (the next token's dc first: it is on the dependent chain)
#pragma unroll
            for (int u = t - 1; u >= 0; --u) dfr[u] = fmaf(grow[t & 1][u], dpred, dfr[u]);
            // every lane stores to LDS (idle lanes to a padding column), so that
            // no branch hides from the compiler how many LDS operations are in
            // flight when the next row of K K^T is waited for
            sP[sl][t][scw] = dpred;
            sDc[t][scw] = dc;
            sDlk[t][scw] = da;
        }
    };
    // E += Q^T Y + K^T P for the chunk in slot sl (E then holds the gradient
    // from the tokens after the previous chunk): 16 x 16 tiles of E on the
    // matrix cores (bf16 inputs), else four columns per thread
    auto update_e = [&](int sl) {
        if constexpr (IBF) {
            // tiles wv, wv + 4, ..., two at a time with every LDS read of both
            // issued before their products (a clamped duplicate past the end
            // is computed and not stored)
            constexpr int NTL = (DK / 16) * NTC, NU = (NTL + 3) / 4;
#pragma unroll
            for (int u0 = 0; u0 < NU; u0 += 2) {
                constexpr int NP2 = NU > 1 ? 2 : 1;
                floatx4 acc[NP2];
                KOp<4> qa[NP2], ka[NP2], yb[NP2], pb[NP2];
#pragma unroll
                for (int x = 0; x < NP2; ++x) {
                    const int tile = min(wv + 4 * (u0 + x), NTL - 1);
                    const int ti = tile / NTC, col = 16 * (tile % NTC) + tl;
                    const bool cv = col < N;
                    const int cc = cv ? col : 0;
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[x][r] = cv ? sE[16 * ti + 4 * lg + r][cc] : 0.0f;
                    // A = Q^T, K^T: rows i = 16 ti + tl, k = t = 4 lg .. + 3
                    float qv[4], kv[4], yv[4], pv[4];
#pragma unroll
                    for (int m = 0; m < 4; ++m) {
                        qv[m] = sQ[sl][4 * lg + m][16 * ti + tl];
                        kv[m] = sK[sl][4 * lg + m][16 * ti + tl];
                        yv[m] = cv ? sY[sl][4 * lg + m][cc] : 0.0f;
                        pv[m] = cv ? sP[sl][4 * lg + m][cc] : 0.0f;
                    }
                    qa[x] = kop_exact<4>(qv), ka[x] = kop_exact<4>(kv);
                    yb[x] = kop_split<4>(yv), pb[x] = kop_split<4>(pv);
                }
#pragma unroll
                for (int x = 0; x < NP2; ++x) {
                    acc[x] = mma(qa[x].hi, yb[x].hi, acc[x]);
                    acc[x] = mma(qa[x].hi, yb[x].lo, acc[x]);
                    acc[x] = mma(ka[x].hi, pb[x].hi, acc[x]);
                    acc[x] = mma(ka[x].hi, pb[x].lo, acc[x]);
                }
#pragma unroll
                for (int x = 0; x < NP2; ++x) {
                    const int tile = wv + 4 * (u0 + x);
                    const int ti = tile / NTC, col = 16 * (tile % NTC) + tl;
                    if (u0 + x < NU && tile < NTL && col < N) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) sE[16 * ti + 4 * lg + r][col] = acc[x][r];
                    }
                }
            }
        } else {
            for (int e = tid; e < DK * (N / 4); e += kThreads) {
                const int i = e / (N / 4), c4 = (e % (N / 4)) * 4;
                float4 acc = *reinterpret_cast<const float4 *>(&sE[i][c4]);
#pragma unroll
                for (int t4 = 0; t4 < kRC; t4 += 4) {
                    const float4 qv = *reinterpret_cast<const float4 *>(&sQt[i][t4]);
                    const float4 kv = *reinterpret_cast<const float4 *>(&sKt[i][t4]);
                    const float qa[4] = {qv.x, qv.y, qv.z, qv.w}, ka[4] = {kv.x, kv.y, kv.z, kv.w};
#pragma unroll
                    for (int x = 0; x < 4; ++x) {
                        const float4 y = *reinterpret_cast<const float4 *>(&sY[sl][t4 + x][c4]);
                        const float4 p = *reinterpret_cast<const float4 *>(&sP[sl][t4 + x][c4]);
                        acc.x = fmaf(qa[x], y.x, fmaf(ka[x], p.x, acc.x));
                        acc.y = fmaf(qa[x], y.y, fmaf(ka[x], p.y, acc.y));
                        acc.z = fmaf(qa[x], y.z, fmaf(ka[x], p.z, acc.z));
                        acc.w = fmaf(qa[x], y.w, fmaf(ka[x], p.w, acc.w));
                    }
                }
                *reinterpret_cast<float4 *>(&sE[i][c4]) = acc;
            }
        }
    };
    // chunk n's per-token outputs, coalesced over output dims: dL/dlb and dL/dlk
    // (from the tokens' dc and da and the staged inputs in slot sl), by threads
    // first .. first + nthr - 1; all LDS reads are issued before the stores
    auto outputs = [&](int n, int sl, auto first, auto nthr) {
        constexpr int F = decltype(first)::value, NT = decltype(nthr)::value;
        const int t0 = n * kRC, nt = min(kRC, T - t0), lt = tid - F;
        constexpr int NE = kRC * J * DB, NI = (NE + NT - 1) / NT;
        float vb[NI], vk[NI];
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = min(lt + NT * x, NE - 1);
            const int t = e / (J * DB), col = e % (J * DB);
            const float be = sBeta[sl][t][col];
            vb[x] = sDc[t][col] * sR[sl][t][col] * sDelta[sl][t][col] * be * (1.0f - be);
            vk[x] = sDlk[t][col];
        }
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int e = lt + NT * x;
            const int t = e / (J * DB), j = (e / DB) % J, dd = e % DB;
            if ((NE % NT == 0 || e < NE) && t < nt) {
                const size_t idx = (((size_t)(b * T + t0 + t) * H + h) * J + j) * Dv + d0 + dd;
                a.dlb[idx] = vb[x];
                a.dlk[idx] = vk[x];
            }
        }
    };
    constexpr ITag<64> kF1{};               // the staging threads of the bf16 schedule
    constexpr ITag<kThreads - 64> kN1{};
    constexpr ITag<0> kF0{};                // every thread
    constexpr ITag<kThreads> kN0{};
    constexpr ITag<128> kF2{};              // waves 2 and 3
    constexpr ITag<kThreads - 128> kN2{};


    if constexpr (IBF) {
        if (NCH > 0) {
            const int n0 = NCH - 1;
            if (tid >= F0) {
                fetch(n0);
                stage(n0, n0 & 1);
                if (n0 > 0) fetch(n0 - 1);
            }
            block_sync_lds();
            gram(n0 & 1);
            block_sync_lds();
            base(n0 & 1);
            for (int n = n0; n >= 0; --n) {
                const int sl = n & 1;
                block_sync_lds();   // A: the base of chunk n and E are complete
                if (tid < 64) {
                    tokens(sl);
                } else {
                    checkpoint(n, kF1, kN1);
                    if (n < n0) {
                        packs_dpred(n + 1, sl ^ 1, kF1, kN1);
                        dv_store(n + 1, sl ^ 1, kF1, kN1);
                    }
                    if (n > 0) {
                        stage(n - 1, sl ^ 1);
                        if (n > 1) fetch(n - 2);   // lands during chunks n and n - 1
                    }
                }
                block_sync_lds();   // B: chunk n's dpred published
                update_e(sl);
                if (n > 0) gram(sl ^ 1);   // waves 2 and 3
                if constexpr (NTC > 2) outputs(n, sl, kF0, kN0);
                block_sync_lds();   // C: E now from the tokens after chunk n - 1
                if (n > 0) base(sl ^ 1);   // waves 0 .. NTC - 1
                // (with two column tiles, waves 2 and 3 store the outputs meanwhile)
                if constexpr (NTC <= 2) {
                    if (wv >= 2) outputs(n, sl, kF2, kN2);
                }
            }
            // chunk 0's tokens ended before the last barrier B
            packs_dpred(0, 0, kF0, kN0);
            dv_store(0, 0, kF0, kN0);
        }
    } else {
        if (NCH > 0) fetch(NCH - 1);
        for (int n = NCH - 1; n >= 0; --n) {
            block_sync_lds();   // E is complete; the previous chunk's staging is consumed
            checkpoint(n, kF0, kN0);
            stage(n, 0);
            block_sync_lds();
            if (n > 0) fetch(n - 1);   // lands while this chunk computes
            gram(0);
            block_sync_lds();
            base(0);
            block_sync_lds();
            if (tid < 64) tokens(0);
            block_sync_lds();
            update_e(0);
            outputs(n, 0, kF0, kN0);
            packs_dpred(n, 0, kF0, kN0);
            dv_store(n, 0, kF0, kN0);
        }
    }
    block_sync_lds();
    if (a.dstate) {
        for (int e = tid; e < J * DK * DB; e += kThreads) {
            const int j = e / (DK * DB), i = (e / DB) % DK, dd = e % DB;
            a.dstate[sbase + ((size_t)j * DK + i) * Dv + d0 + dd] = sE[i][j * DB + dd];
        }
    }
}

// J consecutive floats from global memory (16-byte loads where J allows).
template <int J>
__device__ __forceinline__ void ld_row(const float *p, float (&v)[J]) {
    if constexpr (J % 4 == 0) {
#pragma unroll
        for (int x = 0; x < J; x += 4) {
            const float4 w = *reinterpret_cast<const float4 *>(p + x);
            v[x] = w.x; v[x + 1] = w.y; v[x + 2] = w.z; v[x + 3] = w.w;
        }
    } else if constexpr (J == 2) {
        const float2 w = *reinterpret_cast<const float2 *>(p);
        v[0] = w.x; v[1] = w.y;
    } else {
#pragma unroll
        for (int x = 0; x < J; ++x) v[x] = p[x];
    }
}

// fp32 product on the matrix cores, D (16 x 16) += A (16 x 4) B (4 x 16): lane l
// supplies A[l % 16][l / 16] and B[l / 16][l % 16], and holds D[4 (l / 16) + r][l % 16]
// in element r.  Over a 16-deep block the lane group g = l / 16 supplies depth
// index 4 g + s at step s, so that an operand stored depth-contiguous is read
// with one 16-byte load per lane and block (a4), one stored depth-major with
// four 4-byte loads (b4).
__device__ __forceinline__ floatx4 mma4(float a, float b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 a4(const float *row, int k0, int g) {
    return *reinterpret_cast<const floatx4 *>(row + k0 + 4 * g);
}
template <int P>
__device__ __forceinline__ floatx4 b4(const float (*m)[P], int k0, int g, int col) {
    const int k = k0 + 4 * g;
    return floatx4{m[k][col], m[k + 1][col], m[k + 2][col], m[k + 3][col]};
}
__device__ __forceinline__ floatx4 mma16(floatx4 a, floatx4 b, floatx4 c) {
    c = mma4(a[0], b[0], c);
    c = mma4(a[1], b[1], c);
    c = mma4(a[2], b[2], c);
    return mma4(a[3], b[3], c);
}

// Chunk pass on the matrix cores (fp32 products, fp32 accumulation; one
// instantiation for both input dtypes).  The chunk's 32 tokens are two 16-token
// halves; every product is a set of 16 x 16 output tiles spread over the four
// waves:
//   dq, dk (tokens x key indices): per wave both token halves of key block w
//     (and w + 4, ...), accumulated over all column tiles and the intra-chunk
//     terms; with Dk = 32 one tile per wave, with Dk = 16 waves 0 and 1 only
//   the column Gram products Y_t.C_s (needed for s <= t) and C_t.P_s (s >= t):
//     three 16 x 16 tiles each, accumulated over the column tiles
//   the retrievals (Q S + tril(Q K^T) C), per column tile.
template <int DK, int J>
__global__ __launch_bounds__(kThreads) void bwd_chunk_kernel(BackwardArgs a) {
    constexpr int DT = chunk_tile_dims<J>();
    constexpr int NCT = J * DT;                  // columns per tile: 16, 24 or 32
    constexpr int NCP = (NCT + 15) / 16 * 16;    // columns held (J = 3: 8 zero columns)
    constexpr int NIB = DK / 16;                 // 16-wide key-index blocks
    constexpr int NTH = NIB >= 4 ? 2 : 1;        // token halves per wave (dq, dk)
    constexpr int NIW = NIB >= 4 ? NIB / 4 : 1;  // key blocks per wave
    constexpr int KP = DK + 4, CP = NCP + 4, GP = kCB + 4;   // row pitches (16-byte rows)
    static_assert(kCB == 32 && kThreads == 256, "two token halves, four waves");

    __shared__ __align__(16) float sK[kCB][KP];
    __shared__ __align__(16) float sQ[kCB][KP];
    __shared__ __align__(16) float sQK[kCB][GP];   // tril(Q K^T)
    // The column tiles' buffers and the final coefficient matrices are never
    // live together: they share LDS, which keeps two blocks per compute unit
    // up to Dk = 64.
    struct TileBufs {
        alignas(16) float S[NCP][KP], E[NCP][KP];                // [column][key index]
        alignas(16) float C[kCB][CP], P[kCB][CP], Y[kCB][CP];    // [token][column]
        float Pq[kCB][CP], Yv[kCB][CP];                          // pi^q and the retrievals y
        float Do[kCB][DT];
    };
    struct EndBufs {
        alignas(16) float M[3][kCB][GP];   // masked intra-chunk coefficients
    };
    __shared__ union {
        TileBufs t;
        EndBufs e;
    } lds;
    auto &sS = lds.t.S;
    auto &sE = lds.t.E;
    auto &sC = lds.t.C;
    auto &sP = lds.t.P;
    auto &sY = lds.t.Y;
    auto &sPq = lds.t.Pq;
    auto &sYv = lds.t.Yv;
    auto &sDo = lds.t.Do;
    auto &sM = lds.e.M;

    const LayerArgs &f = a.f;
    const int n = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int lr = tid % 16, g = (tid % 64) / 16;   // MFMA lane row/column and depth group
    const int H = f.H, T = f.T, Dv = f.Dv;
    const int NCH = (T + kCB - 1) / kCB;
    const int t0 = n * kCB, nt = min(kCB, T - t0);
    const bool ibf = f.in_bf16;

    for (int e = tid; e < kCB * (DK / 4); e += kThreads) {
        const int t = e / (DK / 4), i = (e % (DK / 4)) * 4;
        uint4 kr = make_uint4(0u, 0u, 0u, 0u), qr = kr;
        if (t < nt) {
            const size_t off = ((size_t)(b * T + t0 + t) * H + h) * DK + i;
            kr = raw4(f.k, off, ibf);
            qr = raw4(f.q, off, ibf);
        }
        *reinterpret_cast<float4 *>(&sK[t][i]) = cvt4(kr, ibf);
        *reinterpret_cast<float4 *>(&sQ[t][i]) = cvt4(qr, ibf);
    }
    if constexpr (NCP > NCT) {   // the padding columns stay zero
        for (int e = tid; e < (NCP - NCT) * (kCB + DK); e += kThreads) {
            const int c = NCT + e % (NCP - NCT), r = e / (NCP - NCT);
            if (r < kCB) {
                sC[r][c] = 0.0f;
                sP[r][c] = 0.0f;
                sY[r][c] = 0.0f;
            } else {
                sS[c][r - kCB] = 0.0f;
                sE[c][r - kCB] = 0.0f;
            }
        }
    }
    block_sync_lds();
    if constexpr (J > 1) {   // tril(Q K^T): wave w has tile (w / 2, w % 2)
        const int th = w >> 1, sh = w & 1;
        floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
        if (sh <= th) {
#pragma unroll 4
            for (int k0 = 0; k0 < DK; k0 += 16)
                acc = mma16(a4(sQ[16 * th + lr], k0, g), a4(sK[16 * sh + lr], k0, g), acc);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * th + 4 * g + r, s = 16 * sh + lr;
            sQK[t][s] = s <= t ? acc[r] : 0.0f;
        }
    }

    // this wave's dq and dk tiles: (token half, key block) = (x, w + 4 y) for
    // Dk >= 64, (w / 2, w % 2) for Dk = 32, (w, 0) on waves 0 and 1 for Dk = 16
    const bool dwave = NIB >= 2 || w < 2;
    auto tile_th = [&](int x) { return NIB >= 4 ? x : NIB == 2 ? w >> 1 : w; };
    auto tile_ib = [&](int y) { return NIB >= 4 ? w + 4 * y : NIB == 2 ? (w & 1) : 0; };
    floatx4 dq[NTH][NIW], dk[NTH][NIW];
    // Gram tiles: index w and w + 4 of ga(0,0), gb(0,0), ga(1,0), gb(0,1), ga(1,1),
    // gb(1,1); ga = Y_t.C_s, gb = C_t.P_s
    floatx4 gr[2];
#pragma unroll
    for (int x = 0; x < NTH; ++x)
#pragma unroll
        for (int y = 0; y < NIW; ++y) dq[x][y] = dk[x][y] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    gr[0] = gr[1] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
    auto gram_tile = [&](int slot, int &kind, int &th, int &sh) {
        const int idx = w + 4 * slot, pos = idx >> 1;
        kind = idx & 1;
        th = kind ? pos == 2 : pos > 0;
        sh = kind ? pos > 0 : pos == 2;
        return idx < 6;
    };

    // checkpoints of this chunk, [Dv][J][DK]
    const size_t ck0 = (((size_t)b * H + h) * NCH + n) * Dv * J * DK;
    // A tile's HBM operands are loaded into registers while the previous tile
    // computes: its state checkpoints S and E, and its per-(token, column)
    // operands, contiguous in the reverse scan's tile order [token][dd][j].
    // Every thread loads every item it owns (tokens past the end from the
    // chunk's last row); the store to LDS zeroes them.
    constexpr int NSE4 = DT * J * (DK / 4);                  // float4 of S (and of E)
    constexpr int NSE = (NSE4 + kThreads - 1) / kThreads;
    constexpr int NOP = (kCB * DT + kThreads - 1) / kThreads;
    floatx4 rS[NSE], rE[NSE];   // (native vectors: an array of float4 went to scratch memory)
    float rc[NOP][J], rp[NOP][J], rq[NOP][J], rd[NOP];
    auto fetch_tile = [&](int dt0) {
#pragma unroll
        for (int x = 0; x < NSE; ++x) {
            const size_t src = ck0 + (size_t)dt0 * J * DK + 4 * min(tid + kThreads * x, NSE4 - 1);
            rS[x] = *reinterpret_cast<const floatx4 *>(a.wck + src);
            rE[x] = *reinterpret_cast<const floatx4 *>(a.eck + src);
        }
        const size_t tb = ((((size_t)b * H + h) * NCH + n) * (Dv / DT) + dt0 / DT) * kCB;
#pragma unroll
        for (int x = 0; x < NOP; ++x) {
            const int e = min(tid + kThreads * x, kCB * DT - 1);
            const int t = min(e / DT, nt - 1), dd = e % DT;
            const size_t row = (tb + t) * DT + dd;
            ld_row<J>(a.cpk + row * J, rc[x]);
            ld_row<J>(a.ppk + row * J, rp[x]);
            ld_row<J>(a.qpk + row * J, rq[x]);
            rd[x] = a.dopk[row];
        }
    };
    fetch_tile(0);
    for (int dt0 = 0; dt0 < Dv; dt0 += DT) {
        block_sync_lds();   // the previous tile is consumed
#pragma unroll
        for (int x = 0; x < NSE; ++x) {
            const int e = 4 * (tid + kThreads * x);
            const int dd = e / (J * DK), j = (e / DK) % J, i = e % DK;
            if (NSE4 % kThreads == 0 || e < 4 * NSE4) {
                *reinterpret_cast<floatx4 *>(&sS[j * DT + dd][i]) = rS[x];
                *reinterpret_cast<floatx4 *>(&sE[j * DT + dd][i]) = rE[x];
            }
        }
#pragma unroll
        for (int x = 0; x < NOP; ++x) {
            const int e = tid + kThreads * x;
            const int t = e / DT, dd = e % DT;
            const bool in = t < nt;
            const float dov = in ? rd[x] : 0.0f;
            if ((kCB * DT) % kThreads == 0 || e < kCB * DT) {
                sDo[t][dd] = dov;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    const int cc = j * DT + dd;
                    const float pq = in ? rq[x][j] : 0.0f;
                    sC[t][cc] = in ? rc[x][j] : 0.0f;
                    sP[t][cc] = in ? rp[x][j] : 0.0f;
                    sY[t][cc] = dov * pq;
                    sPq[t][cc] = pq;
                }
            }
        }
        block_sync_lds();
        if (dt0 + DT < Dv) fetch_tile(dt0 + DT);   // lands while this tile computes

        // dq += Y S; dk += P S + C E (this tile's columns)
        if (dwave) {
#pragma unroll
            for (int k0 = 0; k0 < NCP; k0 += 16) {
                floatx4 ya[NTH], pa[NTH], ca[NTH], sb[NIW], eb[NIW];
#pragma unroll
                for (int x = 0; x < NTH; ++x) {
                    const int row = 16 * tile_th(x) + lr;
                    ya[x] = a4(sY[row], k0, g);
                    pa[x] = a4(sP[row], k0, g);
                    ca[x] = a4(sC[row], k0, g);
                }
#pragma unroll
                for (int y = 0; y < NIW; ++y) {
                    sb[y] = b4(sS, k0, g, 16 * tile_ib(y) + lr);
                    eb[y] = b4(sE, k0, g, 16 * tile_ib(y) + lr);
                }
#pragma unroll
                for (int x = 0; x < NTH; ++x)
#pragma unroll
                    for (int y = 0; y < NIW; ++y) {
                        dq[x][y] = mma16(ya[x], sb[y], dq[x][y]);
                        dk[x][y] = mma16(pa[x], sb[y], dk[x][y]);
                        dk[x][y] = mma16(ca[x], eb[y], dk[x][y]);
                    }
            }
        }
        // the Gram tiles of this wave
#pragma unroll
        for (int slot = 0; slot < 2; ++slot) {
            int kind, th, sh;
            if (gram_tile(slot, kind, th, sh)) {
                const float *ar = kind ? sC[16 * th + lr] : sY[16 * th + lr];
                const float *br = kind ? sP[16 * sh + lr] : sC[16 * sh + lr];
#pragma unroll
                for (int k0 = 0; k0 < NCP; k0 += 16)
                    gr[slot] = mma16(a4(ar, k0, g), a4(br, k0, g), gr[slot]);
            }
        }
        // retrievals y = Q S + tril(Q K^T) C: tile (token half, column block)
        // (w / 2, w % 2) for 32 columns, (w - 2, 0) on waves 2 and 3 for 16
        if constexpr (J > 1) {
            constexpr int NCB = NCP / 16;
            const int th = NCB == 2 ? w >> 1 : w - 2, cb = NCB == 2 ? (w & 1) : 0;
            if (th >= 0) {
                floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll 4
                for (int k0 = 0; k0 < DK; k0 += 16)
                    acc = mma16(a4(sQ[16 * th + lr], k0, g), a4(sS[16 * cb + lr], k0, g), acc);
                for (int s0 = 0; s0 <= 16 * th; s0 += 16)
                    acc = mma16(a4(sQK[16 * th + lr], s0, g), b4(sC, s0, g, 16 * cb + lr), acc);
#pragma unroll
                for (int r = 0; r < 4; ++r) sYv[16 * th + 4 * g + r][16 * cb + lr] = acc[r];
            }
        }
        block_sync_lds();
        // dL/dlq_j = pi^q_j do (y_j - sum_i pi^q_i y_i); zero for one component
        for (int e = tid; e < nt * DT; e += kThreads) {
            const int t = e / DT, dd = e % DT;
            const size_t row = (size_t)(b * T + t0 + t) * H + h;
            float mean = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) mean = fmaf(sPq[t][j * DT + dd], sYv[t][j * DT + dd], mean);
            const float dov = sDo[t][dd];
#pragma unroll
            for (int j = 0; j < J; ++j)
                a.dlq[(row * J + j) * Dv + dt0 + dd] =
                    J == 1 ? 0.0f : sPq[t][j * DT + dd] * dov * (sYv[t][j * DT + dd] - mean);
        }
    }

    // The intra-chunk terms as three masked C x C coefficient matrices (in the
    // tile buffers' LDS: the last tile is consumed first):
    //   M0[t][s] = (Y_t.C_s) for s <= t          (dq, times k_s)
    //   M1[t][s] = (C_t.P_s) for s > t, (P_t.C_s) for s < t   (dk, times k_s)
    //   M2[t][s] = (C_t.Y_s) for s >= t          (dk, times q_s)
    // A ga element (t, s) with s <= t gives M0[t][s] and M2[s][t]; a gb element
    // with s > t gives M1[t][s] and M1[s][t].  M0's upper and M2's lower
    // off-diagonal blocks are zero.
    block_sync_lds();
    for (int e = tid; e < 16 * 16; e += kThreads) {
        sM[0][e / 16][16 + e % 16] = 0.0f;
        sM[2][16 + e / 16][e % 16] = 0.0f;
    }
#pragma unroll
    for (int slot = 0; slot < 2; ++slot) {
        int kind, th, sh;
        if (gram_tile(slot, kind, th, sh)) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * th + 4 * g + r, s = 16 * sh + lr;
                const float v = gr[slot][r];
                if (kind == 0) {
                    sM[0][t][s] = s <= t ? v : 0.0f;
                    sM[2][s][t] = s <= t ? v : 0.0f;
                } else if (s >= t) {
                    sM[1][t][s] = s > t ? v : 0.0f;
                    sM[1][s][t] = s > t ? v : 0.0f;
                }
            }
        }
    }
    block_sync_lds();
    if (dwave) {
        // dq += M0 K (s up to the end of the token half); dk += M1 K + M2 Q
        // (M2 from the token half's start)
#pragma unroll
        for (int x = 0; x < NTH; ++x) {
            const int th = tile_th(x), row = 16 * th + lr;
#pragma unroll
            for (int y = 0; y < NIW; ++y) {
                const int col = 16 * tile_ib(y) + lr;
                for (int s0 = 0; s0 < kCB; s0 += 16) {
                    const floatx4 kb = b4(sK, s0, g, col);
                    if (s0 <= 16 * th) dq[x][y] = mma16(a4(sM[0][row], s0, g), kb, dq[x][y]);
                    dk[x][y] = mma16(a4(sM[1][row], s0, g), kb, dk[x][y]);
                    if (s0 >= 16 * th)
                        dk[x][y] = mma16(a4(sM[2][row], s0, g), b4(sQ, s0, g, col), dk[x][y]);
                }
            }
        }
#pragma unroll
        for (int x = 0; x < NTH; ++x)
#pragma unroll
            for (int y = 0; y < NIW; ++y)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * tile_th(x) + 4 * g + r;
                    if (t >= nt) continue;
                    const size_t off =
                        ((size_t)(b * T + t0 + t) * H + h) * DK + 16 * tile_ib(y) + lr;
                    a.dq[off] = dq[x][y][r];
                    a.dk[off] = dk[x][y][r];
                }
    }
}

template <int DK, int J, int DB>
hipError_t launch_reverse(const BackwardArgs &a, hipStream_t stream) {
    if constexpr ((J == 3 ? 4 : J) * DB > 64) {
        return hipErrorInvalidValue;
    } else {
        const dim3 grid((unsigned)((a.f.Dv / DB) * a.f.H * a.f.B));
        if (a.f.in_bf16)
            hipLaunchKernelGGL((reverse_chunk_kernel<DK, J, DB, true>), grid, dim3(kThreads), 0,
                               stream, a);
        else
            hipLaunchKernelGGL((reverse_chunk_kernel<DK, J, DB, false>), grid, dim3(kThreads), 0,
                               stream, a);
        return hipGetLastError();
    }
}

template <int DK, int J>
hipError_t launch_bwd_dk_j(const BackwardArgs &a, hipStream_t stream) {
    const LayerArgs &f = a.f;
    LayerArgs fa = f;
    fa.o = nullptr;
    fa.state_out = nullptr;
    fa.resp = nullptr;
    fa.delta_out = a.delta;
    fa.ckpt = a.wck;
    // bf16 inputs: the matrix-core chunk scan recomputes the forward; fp32 inputs
    // take the token-by-token scan, as their forward does
    hipError_t e = f.in_bf16 ? launch_scan_pipe(fa, stream) : launch_scan_direct_aux(fa, stream);
    if (e != hipSuccess) return e;
    // reverse scan: 64 sequential lanes per block (DB = 64 / JP output dims), or
    // half as many (and twice the blocks) while the grid would leave compute
    // units idle
    constexpr int JP = J == 3 ? 4 : J;
    int db = 64 / JP < f.Dv ? 64 / JP : f.Dv;
    if ((long)(f.Dv / db) * f.H * f.B < 256 && db >= 16) db /= 2;
    switch (db) {
        case 64: e = launch_reverse<DK, J, 64>(a, stream); break;
        case 32: e = launch_reverse<DK, J, 32>(a, stream); break;
        case 16: e = launch_reverse<DK, J, 16>(a, stream); break;
        case 8: e = launch_reverse<DK, J, 8>(a, stream); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    const int NCH = (f.T + kCB - 1) / kCB;
    hipLaunchKernelGGL((bwd_chunk_kernel<DK, J>), dim3(NCH, f.H, f.B), dim3(kThreads), 0, stream,
                       a);
    return hipGetLastError();
}

template <int DK>
hipError_t launch_bwd_dk(const BackwardArgs &a, hipStream_t stream) {
    switch (a.f.J) {
        case 1: return launch_bwd_dk_j<DK, 1>(a, stream);
        case 2: return launch_bwd_dk_j<DK, 2>(a, stream);
        case 3: return launch_bwd_dk_j<DK, 3>(a, stream);
        case 4: return launch_bwd_dk_j<DK, 4>(a, stream);
        case 8: return launch_bwd_dk_j<DK, 8>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

size_t backward_workspace_bytes(int B, int H, int T, int Dk, int Dv, int J) {
    const size_t nch = ((size_t)T + kCB - 1) / kCB;
    const size_t per_tok = (size_t)B * T * H * J * Dv * sizeof(float);
    const size_t pk = (size_t)B * H * nch * kCB * J * Dv * sizeof(float);
    const size_t ck = (size_t)B * H * nch * Dv * J * Dk * sizeof(float);
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    return up(per_tok) + 3 * up(pk) + up(pk / J) + 2 * up(ck);
}

hipError_t launch_backward(const BackwardArgs &a, hipStream_t stream) {
    const LayerArgs &f = a.f;
    if (f.T < 1 || f.gk || f.decay || !a.grad_o || !a.dq || !a.dk || !a.dv || !a.dlb || !a.dlk ||
        !a.dlq || !a.delta || !a.cpk || !a.ppk || !a.qpk || !a.dopk || !a.wck || !a.eck)
        return hipErrorInvalidValue;
    if (f.Dv % 16 != 0) return hipErrorInvalidValue;   // every column tile divides Dv
    switch (f.Dk) {
        case 16: return launch_bwd_dk<16>(a, stream);
        case 32: return launch_bwd_dk<32>(a, stream);
        case 64: return launch_bwd_dk<64>(a, stream);
        case 128: return launch_bwd_dk<128>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace swila
