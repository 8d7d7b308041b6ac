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
// 2. Reverse scan, one (b, h, d) column per L lanes as in the forward, with
//    G_{jd} = dL/dw_{t,jd} in registers (each lane a key slice).  Per token,
//    in reverse:
//      dy_j = do pi^q_j;  G_j += dy_j q_t;  dc_j = G_j . k_t
//      r = softmax_j(lk - delta^2/2) and beta recomputed from delta and logits
//      dlb_j = dc_j r_j delta_j beta_j (1 - beta_j)
//      dr_j = dc_j beta_j delta_j;  da_j = r_j (dr_j - sum_i r_i dr_i) = dlk_j
//      ddelta_j = dc_j beta_j r_j - delta_j da_j;  dv = sum_j ddelta_j
//      dpred_j = -ddelta_j;  G_j += dpred_j k_t          (now dL/dw_{t-1,jd})
//    It writes dv, dlb, dlk, dpred, dL/dW_0 (G after token 0), and E_n, the
//    part of dL/dw at the last token of chunk n that comes from later tokens.
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
//    components of DT output dims stream through LDS; each thread accumulates a
//    TM x TN block of (token, key index) outputs in registers, and the
//    intra-chunk sums become three masked C x C coefficient matrices applied to
//    the chunk's K and Q at the end.
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

constexpr int kThreads = 256;
constexpr int kTC = 16;           // tokens staged per round of the reverse scan
constexpr int kMaxCols = 128;
constexpr int kCB = kBwdChunk;    // tokens per chunk of the chunk pass

// Columns of one reverse-scan block: bounded by the block size, the largest Dv
// and 64 KiB of staged per-(token, column) inputs.
constexpr int rev_cols(int L, int J) {
    int n = kThreads / L < kMaxCols ? kThreads / L : kMaxCols;
    while (n > 16 && kTC * (4 * J + 1) * n * 4 > 65536) n /= 2;
    return n;
}

template <int DK, int J, int S>
__global__ __launch_bounds__(kThreads) void scan_reverse_kernel(BackwardArgs a, int ncol) {
    constexpr int L = DK / S;             // lanes per output column
    constexpr int NCM = rev_cols(L, J);
    constexpr int SP = S + 4;

    __shared__ __align__(16) float sK[kTC][L][SP];
    __shared__ __align__(16) float sQ[kTC][L][SP];
    __shared__ float sDo[kTC][NCM];
    __shared__ float sDelta[kTC][J][NCM];
    __shared__ float sBeta[kTC][J][NCM];
    __shared__ float sLk[kTC][J][NCM];
    __shared__ float sPq[kTC][J][NCM];

    const LayerArgs &f = a.f;
    const int tid = threadIdx.x;
    const int nthr = ncol * L;
    const int dl = tid / L, l = tid % L;
    const int d0 = blockIdx.x * ncol;
    const int h = blockIdx.y, b = blockIdx.z;
    const int H = f.H, T = f.T, Dv = f.Dv;
    const int d = d0 + dl;
    const bool ibf = f.in_bf16, obf = f.out_bf16;
    const int NCH = (T + kCB - 1) / kCB;

    float G[J][S];
    const size_t sbase = ((size_t)b * H + h) * J * DK * Dv;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int s = 0; s < S; ++s)
            G[j][s] = a.grad_state ? a.grad_state[sbase + ((size_t)j * DK + l * S + s) * Dv + d]
                                   : 0.0f;

    const int nr = (T + kTC - 1) / kTC;
    for (int rr = nr - 1; rr >= 0; --rr) {
        const int t0 = rr * kTC;
        const int nt = min(kTC, T - t0);
        __syncthreads();
        for (int g = tid; g < nt * (DK / 4); g += nthr) {
            const int tt = g / (DK / 4), i = (g % (DK / 4)) * 4;
            const size_t off = ((size_t)(b * T + t0 + tt) * H + h) * DK + i;
            *reinterpret_cast<float4 *>(&sK[tt][i / S][i % S]) = load4(f.k, off, ibf);
            *reinterpret_cast<float4 *>(&sQ[tt][i / S][i % S]) = load4(f.q, off, ibf);
        }
        for (int g = tid; g < nt * ncol; g += nthr) {
            const int tt = g / ncol, c = g % ncol;
            const size_t row = (size_t)(b * T + t0 + tt) * H + h;
            sDo[tt][c] = load1(a.grad_o, row * Dv + d0 + c, obf);
            float lq[J];
            float m = -INFINITY;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const size_t idx = (row * J + j) * Dv + d0 + c;
                sDelta[tt][j][c] = a.delta[idx];
                sBeta[tt][j][c] = 1.0f / (1.0f + exp_fast(-load1(f.lb, idx, ibf)));
                sLk[tt][j][c] = load1(f.lk, idx, ibf);
                lq[j] = load1(f.lq, idx, ibf);
                m = fmaxf(m, lq[j]);
            }
            float z = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                lq[j] = exp_fast(lq[j] - m);
                z += lq[j];
            }
            const float iz = 1.0f / z;
#pragma unroll
            for (int j = 0; j < J; ++j) sPq[tt][j][c] = lq[j] * iz;
        }
        __syncthreads();

        for (int tt = nt - 1; tt >= 0; --tt) {
            const int t = t0 + tt;
            if (t % kCB == kCB - 1 || t == T - 1) {
                // E_n: dL/dw_t from the tokens after t (the last token of chunk n)
                float *ck = a.eck + ((((size_t)b * H + h) * NCH + t / kCB) * Dv + d) * J * DK;
#pragma unroll
                for (int j = 0; j < J; ++j)
#pragma unroll
                    for (int s = 0; s < S; s += 4)
                        *reinterpret_cast<float4 *>(ck + j * DK + l * S + s) =
                            make_float4(G[j][s], G[j][s + 1], G[j][s + 2], G[j][s + 3]);
            }
            float kv[S], qv[S];
#pragma unroll
            for (int s = 0; s < S; s += 4) {
                const float4 x = *reinterpret_cast<const float4 *>(&sK[tt][l][s]);
                const float4 y = *reinterpret_cast<const float4 *>(&sQ[tt][l][s]);
                kv[s] = x.x; kv[s + 1] = x.y; kv[s + 2] = x.z; kv[s + 3] = x.w;
                qv[s] = y.x; qv[s + 1] = y.y; qv[s + 2] = y.z; qv[s + 3] = y.w;
            }
            const float dov = sDo[tt][dl];
            // retrieval: o = sum_j pi^q_j w_{t,j} . q_t adds dy_j q_t to G_j
            float dc[J];
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const float dy = dov * sPq[tt][j][dl];
                float acc = 0.0f;
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    G[j][s] = fmaf(dy, qv[s], G[j][s]);
                    acc = fmaf(G[j][s], kv[s], acc);
                }
                dc[j] = acc;
            }
#pragma unroll
            for (int j = 0; j < J; ++j) dc[j] = group_sum<L>(dc[j]);

            // r of token t from its errors, as in the forward
            float delta[J], e[J];
            float m = -INFINITY;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                delta[j] = sDelta[tt][j][dl];
                e[j] = sLk[tt][j][dl] - 0.5f * delta[j] * delta[j];
                m = fmaxf(m, e[j]);
            }
            float z = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                e[j] = exp_fast(e[j] - m);
                z += e[j];
            }
            const float iz = 1.0f / z;
            float r[J], dr[J];
            float sdr = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                r[j] = J == 1 ? 1.0f : e[j] * iz;
                dr[j] = dc[j] * sBeta[tt][j][dl] * delta[j];
                sdr = fmaf(r[j], dr[j], sdr);
            }
            const size_t row = (size_t)(b * T + t) * H + h;
            float dvv = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const float beta = sBeta[tt][j][dl];
                // (J = 1: a softmax over one component is constant; written as
                // 0 because the contracted dr - sum r dr leaves a rounding residue)
                const float da = J == 1 ? 0.0f : r[j] * (dr[j] - sdr);
                const float ddelta = dc[j] * beta * r[j] - delta[j] * da;
                dvv += ddelta;
                const float dpred = -ddelta;
#pragma unroll
                for (int s = 0; s < S; ++s) G[j][s] = fmaf(dpred, kv[s], G[j][s]);
                if (l == 0) {
                    const size_t idx = (row * J + j) * Dv + d;
                    a.dlb[idx] = dc[j] * r[j] * delta[j] * beta * (1.0f - beta);
                    a.dlk[idx] = da;
                    a.dpred[idx] = dpred;
                }
            }
            if (l == 0) a.dv[row * Dv + d] = dvv;
        }
    }
    if (a.dstate) {
#pragma unroll
        for (int j = 0; j < J; ++j)
#pragma unroll
            for (int s = 0; s < S; ++s)
                a.dstate[sbase + ((size_t)j * DK + l * S + s) * Dv + d] = G[j][s];
    }
}

// Output dims per column tile of the chunk pass: tiles of all J components of
// DT dims, 16 to 32 columns.
template <int J>
constexpr int chunk_tile_dims() { return J == 1 ? 16 : J == 3 ? 8 : 32 / J; }

template <int N>
__device__ __forceinline__ void lds_vec(const float *p, float (&v)[N]) {
    if constexpr (N == 4) {
        const float4 x = *reinterpret_cast<const float4 *>(p);
        v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    } else {
        const float2 x = *reinterpret_cast<const float2 *>(p);
        v[0] = x.x; v[1] = x.y;
    }
}

template <int DK, int J>
__global__ __launch_bounds__(kThreads) void bwd_chunk_kernel(BackwardArgs a) {
    constexpr int DT = chunk_tile_dims<J>();
    constexpr int NCT = J * DT;               // columns per tile
    constexpr int NO = kCB * DK / kThreads;   // (token, key index) outputs per thread
    constexpr int TN = NO < 4 ? NO : 4;       // consecutive key indices per thread
    constexpr int TM = NO / TN;               // tokens per thread
    constexpr int NIB = DK / TN;
    static_assert(TN >= 2 && NIB * (kCB / TM) == kThreads, "thread tiling");
    static_assert(kCB * kCB == 4 * kThreads, "Gram tiling: 4 entries per thread");
    constexpr int KP = DK + 4, GP = kCB + 4, CP = NCT + 1;   // row pitches (16-byte rows)

    __shared__ __align__(16) float sK[kCB][KP];
    __shared__ __align__(16) float sQ[kCB][KP];
    __shared__ __align__(16) float sS[NCT][KP];
    __shared__ __align__(16) float sE[NCT][KP];
    __shared__ float sC[kCB][CP], sP[kCB][CP], sY[kCB][CP];
    __shared__ __align__(16) float sCt[NCT][GP];   // C and P transposed: [column][token]
    __shared__ __align__(16) float sPt[NCT][GP];
    __shared__ float sA[kCB][GP], sB[kCB][GP];
    __shared__ __align__(16) float sM[3][kCB][GP]; // masked intra-chunk coefficients
    __shared__ float sQK[kCB][GP];                 // q_t . k_s
    __shared__ float sPq[kCB][CP], sYv[kCB][CP];   // pi^q and the retrievals y
    __shared__ float sDo[kCB][DT];

    const LayerArgs &f = a.f;
    const int n = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x;
    const int H = f.H, T = f.T, Dv = f.Dv;
    const int NCH = (T + kCB - 1) / kCB;
    const int t0 = n * kCB, nt = min(kCB, T - t0);
    const bool ibf = f.in_bf16, obf = f.out_bf16;
    const int i0 = (tid % NIB) * TN, tA = (tid / NIB) * TM;   // this thread's outputs
    const int gt = tid / 8, gs = (tid % 8) * 4;               // its Gram entries
    const int gt8 = tid % 8;                                  // its retrieval columns

    for (int g = tid; g < kCB * (DK / 4); g += kThreads) {
        const int t = g / (DK / 4), i = (g % (DK / 4)) * 4;
        float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), qv = kv;
        if (t < nt) {
            const size_t off = ((size_t)(b * T + t0 + t) * H + h) * DK + i;
            kv = load4(f.k, off, ibf);
            qv = load4(f.q, off, ibf);
        }
        *reinterpret_cast<float4 *>(&sK[t][i]) = kv;
        *reinterpret_cast<float4 *>(&sQ[t][i]) = qv;
    }
    __syncthreads();
    {   // Q K^T: row gt, columns gt8 + 8 x
        float qk[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
        for (int i = 0; i < DK; i += 4) {
            float qv[4];
            lds_vec<4>(&sQ[gt][i], qv);
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                float kv[4];
                lds_vec<4>(&sK[gt8 + 8 * x][i], kv);
#pragma unroll
                for (int z = 0; z < 4; ++z) qk[x] = fmaf(qv[z], kv[z], qk[x]);
            }
        }
#pragma unroll
        for (int x = 0; x < 4; ++x) sQK[gt][gt8 + 8 * x] = qk[x];
    }

    float dq[TM][TN], dk[TM][TN], ga[4], gb[4];
#pragma unroll
    for (int m = 0; m < TM; ++m)
#pragma unroll
        for (int x = 0; x < TN; ++x) dq[m][x] = dk[m][x] = 0.0f;
#pragma unroll
    for (int x = 0; x < 4; ++x) ga[x] = gb[x] = 0.0f;

    // checkpoints of this chunk, [Dv][J][DK]
    const size_t ck0 = (((size_t)b * H + h) * NCH + n) * Dv * J * DK;
    for (int dt0 = 0; dt0 < Dv; dt0 += DT) {
        __syncthreads();   // the previous tile is consumed
        for (int g = tid; g < DT * J * (DK / 4); g += kThreads) {
            const int e = 4 * g;
            const int dd = e / (J * DK), j = (e / DK) % J, i = e % DK;
            const size_t src = ck0 + (size_t)dt0 * J * DK + e;
            *reinterpret_cast<float4 *>(&sS[j * DT + dd][i]) =
                *reinterpret_cast<const float4 *>(a.wck + src);
            *reinterpret_cast<float4 *>(&sE[j * DT + dd][i]) =
                *reinterpret_cast<const float4 *>(a.eck + src);
        }
        for (int g = tid; g < kCB * DT; g += kThreads) {
            const int t = g / DT, dd = g % DT;
            float c[J], p[J], y[J], pq[J];
            if (t < nt) {
                const size_t row = (size_t)(b * T + t0 + t) * H + h;
                const float dov = load1(a.grad_o, row * Dv + dt0 + dd, obf);
                float delta[J], e[J], lq[J];
                float m = -INFINITY, mq = -INFINITY;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    const size_t idx = (row * J + j) * Dv + dt0 + dd;
                    delta[j] = a.delta[idx];
                    e[j] = load1(f.lk, idx, ibf) - 0.5f * delta[j] * delta[j];
                    lq[j] = load1(f.lq, idx, ibf);
                    m = fmaxf(m, e[j]);
                    mq = fmaxf(mq, lq[j]);
                }
                float z = 0.0f, zq = 0.0f;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    e[j] = exp_fast(e[j] - m);
                    z += e[j];
                    lq[j] = exp_fast(lq[j] - mq);
                    zq += lq[j];
                }
                const float iz = 1.0f / z, izq = 1.0f / zq;
#pragma unroll
                for (int j = 0; j < J; ++j) {
                    const size_t idx = (row * J + j) * Dv + dt0 + dd;
                    const float beta = 1.0f / (1.0f + exp_fast(-load1(f.lb, idx, ibf)));
                    c[j] = beta * (J == 1 ? 1.0f : e[j] * iz) * delta[j];
                    p[j] = a.dpred[idx];
                    pq[j] = J == 1 ? 1.0f : lq[j] * izq;
                    y[j] = dov * pq[j];
                }
                sDo[t][dd] = dov;
            } else {
#pragma unroll
                for (int j = 0; j < J; ++j) c[j] = p[j] = y[j] = pq[j] = 0.0f;
                sDo[t][dd] = 0.0f;
            }
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int cc = j * DT + dd;
                sC[t][cc] = c[j];
                sP[t][cc] = p[j];
                sY[t][cc] = y[j];
                sCt[cc][t] = c[j];
                sPt[cc][t] = p[j];
                sPq[t][cc] = pq[j];
            }
        }
        __syncthreads();

        // dq += Y S; dk += P S + C E (this tile's columns)
#pragma unroll 4
        for (int cc = 0; cc < NCT; ++cc) {
            float sv[TN], ev[TN];
            lds_vec<TN>(&sS[cc][i0], sv);
            lds_vec<TN>(&sE[cc][i0], ev);
#pragma unroll
            for (int m = 0; m < TM; ++m) {
                const float yv = sY[tA + m][cc], pv = sP[tA + m][cc], cv = sC[tA + m][cc];
#pragma unroll
                for (int x = 0; x < TN; ++x) {
                    dq[m][x] = fmaf(yv, sv[x], dq[m][x]);
                    dk[m][x] = fmaf(pv, sv[x], fmaf(cv, ev[x], dk[m][x]));
                }
            }
        }
        // Gram products over the columns: ga = Y_t . C_s, gb = C_t . P_s
#pragma unroll 4
        for (int cc = 0; cc < NCT; ++cc) {
            float ct[4], pt[4];
            lds_vec<4>(&sCt[cc][gs], ct);
            lds_vec<4>(&sPt[cc][gs], pt);
            const float yv = sY[gt][cc], cv = sC[gt][cc];
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                ga[x] = fmaf(yv, ct[x], ga[x]);
                gb[x] = fmaf(cv, pt[x], gb[x]);
            }
        }
        // retrievals y = Q S + tril(Q K^T) C: row gt, columns gt8 + 8 x
        if constexpr (J > 1) {
            constexpr int NY = NCT / 8;
            float yr[NY];
#pragma unroll
            for (int x = 0; x < NY; ++x) yr[x] = 0.0f;
#pragma unroll 4
            for (int i = 0; i < DK; i += 4) {
                float qv[4];
                lds_vec<4>(&sQ[gt][i], qv);
#pragma unroll
                for (int x = 0; x < NY; ++x) {
                    float sv[4];
                    lds_vec<4>(&sS[gt8 + 8 * x][i], sv);
#pragma unroll
                    for (int z = 0; z < 4; ++z) yr[x] = fmaf(qv[z], sv[z], yr[x]);
                }
            }
            for (int s2 = 0; s2 <= gt; ++s2) {
                const float qk = sQK[gt][s2];
#pragma unroll
                for (int x = 0; x < NY; ++x) yr[x] = fmaf(qk, sC[s2][gt8 + 8 * x], yr[x]);
            }
#pragma unroll
            for (int x = 0; x < NY; ++x) sYv[gt][gt8 + 8 * x] = yr[x];
        }
        __syncthreads();
        // dL/dlq_j = pi^q_j do (y_j - sum_i pi^q_i y_i); zero for one component
        for (int g = tid; g < nt * DT; g += kThreads) {
            const int t = g / DT, dd = g % DT;
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

    // the intra-chunk terms, as three masked C x C coefficient matrices
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        sA[gt][gs + x] = ga[x];
        sB[gt][gs + x] = gb[x];
    }
    __syncthreads();
    for (int g = tid; g < kCB * kCB; g += kThreads) {
        const int t = g / kCB, s = g % kCB;
        sM[0][t][s] = s <= t ? sA[t][s] : 0.0f;                          // (Y_t . C_s) k_s
        sM[1][t][s] = s > t ? sB[t][s] : (s < t ? sB[s][t] : 0.0f);      // (C_t.P_s), (P_t.C_s) k_s
        sM[2][t][s] = s >= t ? sA[s][t] : 0.0f;                          // (C_t . Y_s) q_s
    }
    __syncthreads();
#pragma unroll 4
    for (int s = 0; s < kCB; ++s) {
        float kv[TN], qv[TN];
        lds_vec<TN>(&sK[s][i0], kv);
        lds_vec<TN>(&sQ[s][i0], qv);
#pragma unroll
        for (int m = 0; m < TM; ++m) {
            const float mq = sM[0][tA + m][s], m1 = sM[1][tA + m][s], m2 = sM[2][tA + m][s];
#pragma unroll
            for (int x = 0; x < TN; ++x) {
                dq[m][x] = fmaf(mq, kv[x], dq[m][x]);
                dk[m][x] = fmaf(m1, kv[x], fmaf(m2, qv[x], dk[m][x]));
            }
        }
    }
#pragma unroll
    for (int m = 0; m < TM; ++m) {
        const int t = tA + m;
        if (t >= nt) continue;
        const size_t off = ((size_t)(b * T + t0 + t) * H + h) * DK + i0;
#pragma unroll
        for (int x = 0; x < TN; ++x) {
            a.dq[off + x] = dq[m][x];
            a.dk[off + x] = dk[m][x];
        }
    }
}

template <int DK, int J>
hipError_t launch_bwd_dk_j(const BackwardArgs &a, hipStream_t stream) {
    constexpr int S = (J <= 4) ? (DK < 16 ? DK : 16) : (DK < 8 ? DK : 8);
    constexpr int L = DK / S;
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
    const int ncol = f.Dv < rev_cols(L, J) ? f.Dv : rev_cols(L, J);
    hipLaunchKernelGGL((scan_reverse_kernel<DK, J, S>), dim3(f.Dv / ncol, f.H, f.B),
                       dim3(ncol * L), 0, stream, a, ncol);
    e = hipGetLastError();
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
    const size_t ck = (size_t)B * H * nch * Dv * J * Dk * sizeof(float);
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    return 2 * up(per_tok) + 2 * up(ck);
}

hipError_t launch_backward(const BackwardArgs &a, hipStream_t stream) {
    const LayerArgs &f = a.f;
    if (f.T < 1 || f.gk || f.decay || !a.grad_o || !a.dq || !a.dk || !a.dv || !a.dlb || !a.dlk ||
        !a.dlq || !a.delta || !a.dpred || !a.wck || !a.eck)
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
