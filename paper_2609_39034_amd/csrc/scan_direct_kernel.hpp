// Token-by-token SwiLA scan (Sec. 3.2: eq. recurrence, eq. responsibility,
// eq. retrieval), fp32 state held in VGPRs for the whole sequence.
//
// Work split.  Every (b, h, d) output column is independent except that the
// E-step normalises over the J components of the same d.  One column's state,
// w_{jd} for all j (J x Dk floats), is spread over L consecutive lanes, each
// lane holding an S = Dk / L slice of the key dimension for every j.  Per token:
//   pred_j = w_j . k and y_j = w_j . q   (S FMAs per lane, DPP sum over L lanes)
//   r      = softmax_j(lk_j - delta_j^2 / 2)   (in-lane over J; see below)
//   w_j   += beta_j r_j delta_j k          (S FMAs per lane)
//   o      = sum_j pi^q_j (y_j + c_j (k . q))
// The key prior pi^k = softmax_j(lk) enters the E-step only through
// pi^k_j e^{-delta_j^2/2}, so its normaliser cancels and r is a softmax of
// lk_j - delta_j^2/2.  The retrieval uses the updated state:
// w_new . q = w_old . q + c (k . q).
//
// Inputs are staged through LDS kTC tokens at a time: k and q as fp32 slices
// padded so the L lanes of a column read distinct banks, and the per-(token,
// column) scalars beta = sigmoid(logit), lk and pi^q = softmax_j already formed,
// so the sequential loop does only the dependent arithmetic.
//
// Temporal SwiLA (TP; Sec. 3.3, App. B.3).  The key prior is the gated mixture
// rbar_j = (1 - g^k) r_{t-1,j} + g^k pi^k_j of the previous token's
// responsibilities and pi^k = softmax_j(lk), so pi^k is staged normalised and
// r = rbar_j e^{-delta_j^2/2} / sum (the exponent shifted by its maximum over j);
// the query prior rhobar_j = (1 - g^q) rhobar_{t-1,j} + g^q pi^q_j replaces
// pi^q.  Both running priors live in registers, J per column, from the prior
// state (or 1/J) to the prior state written at the end.
//
// Gated SwiLA (GT; Sec. 3.4, App. B.4, eq. pre-decay).  Each token first
// decays the state, w_j (.)= a_{tj} with a = sigmoid(decay logit) one gate per
// key dimension, and the prediction, E-step, update and retrieval then use the
// decayed state.  The gates of a token round are formed once, in fp32, into
// LDS ([token][j][key index], each lane reading its slice).
//
// Backward support (AX): the same plain scan writes delta_{tjd} of every token
// and the state before every kBwdChunk-th token (layout [.., chunk, d, j, i], so
// that each lane stores its key slice contiguously), and no output.
//
// This header holds the kernel template and its launch rules; each key size Dk
// is instantiated in a translation unit of its own (scan_direct_dk*.hip) so that
// they compile in parallel, and scan_direct.hip dispatches on Dk.
#pragma once
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

constexpr int kThreads = 256;
constexpr int kTC = 16;
constexpr int kMaxCols = 128;  // largest supported Dv

// Columns one block holds: bounded by the block size, the largest Dv, and a
// 64 KiB budget for the per-(token, column) scalars staged in LDS.
constexpr int max_cols(int L, int J, bool tp) {
    int n = kThreads / L < kMaxCols ? kThreads / L : kMaxCols;
    while (n > 16 && kTC * (3 * J + (tp ? 4 : 2)) * n * 4 > 65536) n /= 2;
    return n;
}

// IBF: bf16 inputs.  The input dtype is fixed per instantiation, so that every
// staging load has one form and none sits in a branch on it (a load in one arm
// of a branch is waited for where the arms join).
template <int DK, int J, int S, bool TP, bool GT, bool AX, bool IBF>
__global__ __launch_bounds__(kThreads) void scan_direct_kernel(LayerArgs a, int ncol) {
    static_assert(kBwdChunk % kTC == 0, "checkpoints fall on round starts");
    constexpr int L = DK / S;             // lanes per output column
    constexpr int NCM = max_cols(L, J, TP);
    constexpr int SP = S + 4;             // padded slice stride in LDS

    __shared__ __align__(16) float sK[kTC][L][SP];
    __shared__ __align__(16) float sQ[kTC][L][SP];
    __shared__ float sV[kTC][NCM];
    __shared__ float sBeta[kTC][J][NCM];
    __shared__ float sLk[kTC][J][NCM];
    __shared__ float sPq[kTC][J][NCM];
    __shared__ float sO[kTC][NCM];
    __shared__ float sG[TP ? 2 : 1][kTC][TP ? NCM : 1];   // temporal: g^k, g^q
    __shared__ __align__(16) float sA[GT ? kTC : 1][GT ? J : 1][GT ? DK : 4];   // gated: decay

    const int tid = threadIdx.x;
    const int nthr = ncol * L;
    const int dl = tid / L, l = tid % L;
    // Workgroups go to the eight XCDs (each with its own L2) round-robin by
    // linear index.  Every column block of a head is placed on the same XCD, so
    // that the head's K, Q and decay rows, which each of its column blocks
    // stages, come from HBM once.
    const int NDB = gridDim.x, NH = gridDim.y * gridDim.z;
    const int lin = blockIdx.x + NDB * (blockIdx.y + gridDim.y * blockIdx.z);
    int hh = blockIdx.y + gridDim.y * blockIdx.z, db = blockIdx.x;
    if (NDB > 1 && NH % 8 == 0) {
        const int xs = lin / 8;
        hh = 8 * (xs / NDB) + lin % 8;
        db = xs % NDB;
    }
    const int d0 = db * ncol;
    const int h = hh % gridDim.y, b = hh / gridDim.y;
    const int H = a.H, T = a.T, Dv = a.Dv;
    const int d = d0 + dl;
    constexpr bool ibf = IBF;
    const bool obf = a.out_bf16;

    float w[J][S];
    const size_t sbase = ((size_t)b * H + h) * J * DK * Dv;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
        for (int s = 0; s < S; ++s)
            w[j][s] = a.state_in ? a.state_in[sbase + ((size_t)j * DK + l * S + s) * Dv + d] : 0.0f;
    // temporal: r_{t-1} and rhobar_{t-1} of this column
    float rprev[J], rho[J];
    const size_t pbase = ((size_t)b * H + h) * 2 * J * Dv + d;
    if constexpr (TP) {
#pragma unroll
        for (int j = 0; j < J; ++j) {
            rprev[j] = a.prior_in ? a.prior_in[pbase + (size_t)j * Dv] : 1.0f / J;
            rho[j] = a.prior_in ? a.prior_in[pbase + (size_t)(J + j) * Dv] : 1.0f / J;
        }
    }

    // Per-(token, column) scalars of one staged item: v, beta = sigmoid, the
    // key-prior logits (temporal: pi^k itself), pi^q = softmax_j, and the
    // temporal gates.
    auto stage_item = [&](int tt, int c, uint32_t rv, const uint32_t *rb, const uint32_t *rlk,
                          const uint32_t *rlq, uint32_t rgk, uint32_t rgq) {
        sV[tt][c] = cvt1(rv, ibf);
        float lq[J], lk[J];
        float m = -INFINITY, mk = -INFINITY;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            sBeta[tt][j][c] = 1.0f / (1.0f + exp_fast(-cvt1(rb[j], ibf)));
            lk[j] = cvt1(rlk[j], ibf);
            lq[j] = cvt1(rlq[j], ibf);
            m = fmaxf(m, lq[j]);
            mk = fmaxf(mk, lk[j]);
        }
        float z = 0.0f, zk = 0.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            lq[j] = exp_fast(lq[j] - m);
            z += lq[j];
            if constexpr (TP) {
                lk[j] = exp_fast(lk[j] - mk);
                zk += lk[j];
            }
        }
        const float iz = 1.0f / z;
        const float izk = TP ? 1.0f / zk : 1.0f;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            sPq[tt][j][c] = lq[j] * iz;
            sLk[tt][j][c] = TP ? lk[j] * izk : lk[j];
        }
        if constexpr (TP) {
            sG[0][tt][c] = 1.0f / (1.0f + exp_fast(-cvt1(rgk, ibf)));
            sG[1][tt][c] = 1.0f / (1.0f + exp_fast(-cvt1(rgq, ibf)));
        }
    };

    // Prefetch (PF): when the raw loads of a whole 16-token round fit in a
    // register budget, the loads of round n+1 are issued right after round n
    // is published to LDS, and so are in flight during round n's token loop;
    // they are converted and stored at the top of round n+1.  Without PF a
    // round's loads are issued and converted in batches before its token loop,
    // and the HBM latency of every batch sits on the sequential path.
    constexpr int NKQ = S / 4;                // K/Q pieces per thread at most (ncol >= 16)
    constexpr int ND = GT ? J * S / 4 : 0;    // decay pieces per thread at most
    constexpr int NI = kTC / L;               // scalar items per thread at most
    constexpr int NSC = 1 + 3 * J + (TP ? 2 : 0);
    constexpr bool PF = NKQ * 8 + NI * NSC + ND * 4 <= 128;
    uint4 pk[PF ? NKQ : 1], pq[PF ? NKQ : 1], pd[PF && ND ? ND : 1];
    uint32_t pv[PF ? NI : 1], pb[PF ? NI : 1][J], plk[PF ? NI : 1][J], plq[PF ? NI : 1][J];
    uint32_t pgk[PF ? NI : 1], pgq[PF ? NI : 1];
    // decay piece x of a thread in a round of un tokens: token, component, key index
    auto dpiece_n = [&](int x, int un, int &tt, int &j, int &i) {
        const int g = tid + x * nthr;
        tt = g / (J * (DK / 4));
        const int rem = g % (J * (DK / 4));
        j = rem / (DK / 4), i = (rem % (DK / 4)) * 4;
        return g < un * J * (DK / 4);
    };
    // Every thread loads every item it may own, from a clamped index (the
    // round's last item past the end), with no branch around the load: a load
    // behind a branch is waited for where the branch joins, which would put the
    // HBM latency of each load back on the sequential path.  commit stores only
    // the items that exist.
    auto issue = [&](int u0) {   // the raw loads of the round that starts at token u0
        const int un = min(kTC, T - u0);
#pragma unroll
        for (int x = 0; x < NKQ; ++x) {
            const int g = min(tid + x * nthr, un * (DK / 4) - 1);
            const size_t off = ((size_t)(b * T + u0 + g / (DK / 4)) * H + h) * DK +
                               (g % (DK / 4)) * 4;
            pk[x] = raw4(a.k, off, ibf);
            pq[x] = raw4(a.q, off, ibf);
        }
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int g = min(tid + x * nthr, un * ncol - 1);
            const int tt = g / ncol, c = g % ncol;
            const size_t row = (size_t)(b * T + u0 + tt) * H + h;
            pv[x] = raw1(a.v, row * Dv + d0 + c, ibf);
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const size_t idx = (row * J + j) * Dv + d0 + c;
                pb[x][j] = raw1(a.lb, idx, ibf);
                plk[x][j] = raw1(a.lk, idx, ibf);
                plq[x][j] = raw1(a.lq, idx, ibf);
            }
            if constexpr (TP) {
                pgk[x] = raw1(a.gk, row * Dv + d0 + c, ibf);
                pgq[x] = raw1(a.gq, row * Dv + d0 + c, ibf);
            }
        }
#pragma unroll
        for (int x = 0; x < ND; ++x) {
            const int g = min(tid + x * nthr, un * J * (DK / 4) - 1);
            const int tt = g / (J * (DK / 4)), rem = g % (J * (DK / 4));
            const int j = rem / (DK / 4), i = (rem % (DK / 4)) * 4;
            pd[x] = raw4(a.decay, (((size_t)(b * T + u0 + tt) * H + h) * J + j) * DK + i, ibf);
        }
    };
    auto commit = [&](int u0) {   // convert the issued round and store it to LDS
        const int un = min(kTC, T - u0);
#pragma unroll
        for (int x = 0; x < NKQ; ++x) {
            const int g = tid + x * nthr;
            if (g < un * (DK / 4)) {
                const int tt = g / (DK / 4), i = (g % (DK / 4)) * 4;
                *reinterpret_cast<float4 *>(&sK[tt][i / S][i % S]) = cvt4(pk[x], ibf);
                *reinterpret_cast<float4 *>(&sQ[tt][i / S][i % S]) = cvt4(pq[x], ibf);
            }
        }
#pragma unroll
        for (int x = 0; x < NI; ++x) {
            const int g = tid + x * nthr;
            if (g < un * ncol)
                stage_item(g / ncol, g % ncol, pv[x], pb[x], plk[x], plq[x], pgk[x], pgq[x]);
        }
#pragma unroll
        for (int x = 0; x < ND; ++x) {
            int tt, j, i;
            if (dpiece_n(x, un, tt, j, i)) {
                const float4 v4 = cvt4(pd[x], ibf);
                *reinterpret_cast<float4 *>(&sA[tt][j][i]) = make_float4(
                    sigmoid(v4.x), sigmoid(v4.y), sigmoid(v4.z), sigmoid(v4.w));
            }
        }
    };
    // The token loop leaves each token's output in sO and, where they are
    // asked for, r in the token's beta slot and delta in its key-prior slot,
    // both read for the last time by that token.  They go to HBM at the top
    // of the next round (and after the last one), so that the token loop
    // holds no global store: with one in it, the compiler waits for every
    // load in flight before the loop starts, the next round's prefetch
    // included.  A thread writes out the items g = tid + x nthr, which are
    // the ones it also stages, so none is overwritten before it is read.
    auto flush = [&](int u0, int un) {
        for (int g = tid; g < un * ncol; g += nthr) {
            const int tt = g / ncol, c = g % ncol;
            const size_t row = (size_t)(b * T + u0 + tt) * H + h;
            if constexpr (!AX) store1(a.o, row * Dv + d0 + c, sO[tt][c], obf);
            if (a.resp) {
#pragma unroll
                for (int j = 0; j < J; ++j) a.resp[(row * J + j) * Dv + d0 + c] = sBeta[tt][j][c];
            }
            if constexpr (AX) {
#pragma unroll
                for (int j = 0; j < J; ++j) a.delta_out[(row * J + j) * Dv + d0 + c] = sLk[tt][j][c];
            }
        }
    };
    if constexpr (PF) {
        if (T > 0) issue(0);
    }
    // The state (and the temporal priors) must have landed before the first
    // token; waiting for them here, behind the first round's loads, keeps the
    // compiler from placing a wait for every load in flight inside the token
    // loop, where the next round's prefetch would be waited for.
#pragma unroll
    for (int j = 0; j < J; ++j) {
#pragma unroll
        for (int s = 0; s < S; ++s) asm volatile("" : "+v"(w[j][s]));
        if constexpr (TP) asm volatile("" : "+v"(rprev[j]), "+v"(rho[j]));
    }

    for (int t0 = 0; t0 < T; t0 += kTC) {
        const int nt = min(kTC, T - t0);
        if constexpr (AX) {
            if (t0 % kBwdChunk == 0) {   // the state before token t0
                const int NCH = (T + kBwdChunk - 1) / kBwdChunk;
                float *ck = a.ckpt + ((((size_t)b * H + h) * NCH + t0 / kBwdChunk) * Dv + d) * J * DK;
#pragma unroll
                for (int j = 0; j < J; ++j)
#pragma unroll
                    for (int s = 0; s < S; s += 4)
                        *reinterpret_cast<float4 *>(ck + j * DK + l * S + s) =
                            make_float4(w[j][s], w[j][s + 1], w[j][s + 2], w[j][s + 3]);
            }
        }
        block_sync_lds();
        if (t0 > 0) flush(t0 - kTC, kTC);   // the previous (full) round
        // Staging issues every load of a batch before it converts anything:
        // loading and converting element by element would make each load wait
        // for its data before the next one is issued.  The block barriers order
        // LDS traffic only: the global stores of outputs need no ordering here,
        // and a full barrier would wait for them.
        if constexpr (PF) {
            commit(t0);
        } else {
            // K and Q rows and the first batch of per-(token, column) scalars are
            // all issued before anything converts; the decay gates follow in
            // batches of their own.
            // scalar items loaded together: a register budget over the values
            // of an item
            constexpr int NBR = 56 / (1 + 3 * J + (TP ? 2 : 0));
            constexpr int NB = NBR < 1 ? 1 : (NBR < NI ? NBR : NI);
            constexpr int NDB = ND < 4 ? ND : 4;      // decay pieces loaded together
            uint4 rk[NKQ], rq[NKQ];
#pragma unroll
            for (int x = 0; x < NKQ; ++x) {
                const int g = tid + x * nthr;
                if (g < nt * (DK / 4)) {
                    const int tt = g / (DK / 4), i = (g % (DK / 4)) * 4;
                    const size_t off = ((size_t)(b * T + t0 + tt) * H + h) * DK + i;
                    rk[x] = raw4(a.k, off, ibf);
                    rq[x] = raw4(a.q, off, ibf);
                }
            }
            auto dpiece = [&](int x, int &tt, int &j, int &i) { return dpiece_n(x, nt, tt, j, i); };
            for (int i0 = 0; i0 < NI; i0 += NB) {
                uint32_t rv[NB], rb[NB][J], rlk[NB][J], rlq[NB][J], rgk[NB], rgq[NB];
#pragma unroll
                for (int x = 0; x < NB; ++x) {
                    const int g = tid + (i0 + x) * nthr;
                    if (g < nt * ncol) {
                        const int tt = g / ncol, c = g % ncol;
                        const size_t row = (size_t)(b * T + t0 + tt) * H + h;
                        rv[x] = raw1(a.v, row * Dv + d0 + c, ibf);
#pragma unroll
                        for (int j = 0; j < J; ++j) {
                            const size_t idx = (row * J + j) * Dv + d0 + c;
                            rb[x][j] = raw1(a.lb, idx, ibf);
                            rlk[x][j] = raw1(a.lk, idx, ibf);
                            rlq[x][j] = raw1(a.lq, idx, ibf);
                        }
                        if constexpr (TP) {
                            rgk[x] = raw1(a.gk, row * Dv + d0 + c, ibf);
                            rgq[x] = raw1(a.gq, row * Dv + d0 + c, ibf);
                        }
                    }
                }
                if (i0 == 0) {
#pragma unroll
                    for (int x = 0; x < NKQ; ++x) {
                        const int g = tid + x * nthr;
                        if (g < nt * (DK / 4)) {
                            const int tt = g / (DK / 4), i = (g % (DK / 4)) * 4;
                            *reinterpret_cast<float4 *>(&sK[tt][i / S][i % S]) = cvt4(rk[x], ibf);
                            *reinterpret_cast<float4 *>(&sQ[tt][i / S][i % S]) = cvt4(rq[x], ibf);
                        }
                    }
                }
#pragma unroll
                for (int x = 0; x < NB; ++x) {
                    const int g = tid + (i0 + x) * nthr;
                    if (g >= nt * ncol) continue;
                    stage_item(g / ncol, g % ncol, rv[x], rb[x], rlk[x], rlq[x], rgk[x], rgq[x]);
                }
            }
            if constexpr (GT) {   // decay gates, in batches of their own
                for (int x0 = 0; x0 < ND; x0 += NDB) {
                    uint4 rd[NDB];
#pragma unroll
                    for (int x = 0; x < NDB; ++x) {
                        int tt, j, i;
                        if (x0 + x < ND && dpiece(x0 + x, tt, j, i))
                            rd[x] = raw4(a.decay, (((size_t)(b * T + t0 + tt) * H + h) * J + j) * DK + i,
                                         ibf);
                    }
#pragma unroll
                    for (int x = 0; x < NDB; ++x) {
                        int tt, j, i;
                        if (x0 + x < ND && dpiece(x0 + x, tt, j, i)) {
                            const float4 v4 = cvt4(rd[x], ibf);
                            *reinterpret_cast<float4 *>(&sA[tt][j][i]) = make_float4(
                                sigmoid(v4.x), sigmoid(v4.y), sigmoid(v4.z), sigmoid(v4.w));
                        }
                    }
                }
            }
        }
        block_sync_lds();
        if constexpr (PF) {
            if (t0 + kTC < T) issue(t0 + kTC);
        }

        for (int tt = 0; tt < nt; ++tt) {
            float kv[S], qv[S];
#pragma unroll
            for (int s = 0; s < S; s += 4) {
                const float4 x = *reinterpret_cast<const float4 *>(&sK[tt][l][s]);
                const float4 y = *reinterpret_cast<const float4 *>(&sQ[tt][l][s]);
                kv[s] = x.x; kv[s + 1] = x.y; kv[s + 2] = x.z; kv[s + 3] = x.w;
                qv[s] = y.x; qv[s + 1] = y.y; qv[s + 2] = y.z; qv[s + 3] = y.w;
            }
            if constexpr (GT) {
                // eq. pre-decay: the state decays before the prediction
#pragma unroll
                for (int j = 0; j < J; ++j)
#pragma unroll
                    for (int s = 0; s < S; s += 4) {
                        const float4 x = *reinterpret_cast<const float4 *>(&sA[tt][j][l * S + s]);
                        w[j][s] *= x.x, w[j][s + 1] *= x.y, w[j][s + 2] *= x.z, w[j][s + 3] *= x.w;
                    }
            }
            float p[J], y[J];
            float kq = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                p[j] = 0.0f;
                y[j] = 0.0f;
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    p[j] = fmaf(w[j][s], kv[s], p[j]);
                    y[j] = fmaf(w[j][s], qv[s], y[j]);
                }
            }
#pragma unroll
            for (int s = 0; s < S; ++s) kq = fmaf(kv[s], qv[s], kq);
#pragma unroll
            for (int j = 0; j < J; ++j) {
                p[j] = group_sum<L>(p[j]);
                y[j] = group_sum<L>(y[j]);
            }
            kq = group_sum<L>(kq);

            const float vd = sV[tt][dl];
            float delta[J], e[J];
            float m = -INFINITY;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                delta[j] = vd - p[j];
                e[j] = (TP ? 0.0f : sLk[tt][j][dl]) - 0.5f * delta[j] * delta[j];
                m = fmaxf(m, e[j]);
            }
            float z = 0.0f;
            const float gk = TP ? sG[0][tt][dl] : 0.0f, gq = TP ? sG[1][tt][dl] : 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                e[j] = exp_fast(e[j] - m);
                // temporal key prior: (1 - g^k) r_{t-1} + g^k pi^k
                if constexpr (TP) e[j] *= fmaf(gk, sLk[tt][j][dl] - rprev[j], rprev[j]);
                z += e[j];
            }
            const float iz = rcp_fast(z);
            float o = 0.0f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const float r = e[j] * iz;
                const float c = sBeta[tt][j][dl] * r * delta[j];
#pragma unroll
                for (int s = 0; s < S; ++s) w[j][s] = fmaf(c, kv[s], w[j][s]);
                float pq = sPq[tt][j][dl];
                if constexpr (TP) {
                    rprev[j] = r;
                    rho[j] = fmaf(gq, pq - rho[j], rho[j]);   // (1 - g^q) rhobar + g^q pi^q
                    pq = rho[j];
                }
                o = fmaf(pq, fmaf(c, kq, y[j]), o);
                // r and delta wait in slots that this token has read for the last
                // time (every lane of the column writes the same value)
                sBeta[tt][j][dl] = r;
                if constexpr (AX) sLk[tt][j][dl] = delta[j];
            }
            if (l == 0) sO[tt][dl] = o;
        }
    }

    block_sync_lds();
    if (T > 0) {
        const int tl = ((T - 1) / kTC) * kTC;
        flush(tl, T - tl);
    }
    if (a.state_out) {
#pragma unroll
        for (int j = 0; j < J; ++j)
#pragma unroll
            for (int s = 0; s < S; ++s)
                a.state_out[sbase + ((size_t)j * DK + l * S + s) * Dv + d] = w[j][s];
    }
    if constexpr (TP) {
        if (a.prior_out && l == 0) {
#pragma unroll
            for (int j = 0; j < J; ++j) {
                a.prior_out[pbase + (size_t)j * Dv] = rprev[j];
                a.prior_out[pbase + (size_t)(J + j) * Dv] = rho[j];
            }
        }
    }
}

template <int DK, int J, int S, bool TP, bool GT, bool AX>
hipError_t launch_s(const LayerArgs &a, hipStream_t stream) {
    constexpr int L = DK / S;
    const int ncol = a.Dv < max_cols(L, J, TP) ? a.Dv : max_cols(L, J, TP);
    dim3 grid(a.Dv / ncol, a.H, a.B);
    dim3 block(ncol * L);
    if (a.in_bf16)
        hipLaunchKernelGGL((scan_direct_kernel<DK, J, S, TP, GT, AX, true>), grid, block, 0, stream, a,
                           ncol);
    else
        hipLaunchKernelGGL((scan_direct_kernel<DK, J, S, TP, GT, AX, false>), grid, block, 0, stream, a,
                           ncol);
    return hipGetLastError();
}

// Blocks of the launch with S key rows per lane.
template <int DK, int J, int S, bool TP>
size_t grid_blocks(const LayerArgs &a) {
    const int ncol = a.Dv < max_cols(DK / S, J, TP) ? a.Dv : max_cols(DK / S, J, TP);
    return (size_t)(a.Dv / ncol) * a.H * a.B;
}

template <int DK, int J, bool TP, bool GT, bool AX = false>
hipError_t launch_dk_j_tp(const LayerArgs &a, hipStream_t stream) {
    constexpr int S = (J <= 4) ? (DK < 16 ? DK : 16) : (DK < 8 ? DK : 8);
    {
        // A wave's time per token is bound by its own instruction stream, which
        // shrinks with its rows per lane, and a grid of fewer blocks than
        // compute units leaves the rest idle: halve S (down to 4 rows, and to
        // at most 16 lanes per column, which keeps every block at 16 columns or
        // more) while the grid is under 256 blocks.  The gated form rescales
        // every state row of a lane each token, so its rows cost more than the
        // wider reductions that fewer rows bring: it halves S while the grid is
        // under 1024 blocks (four per compute unit).  At B=4 H=8 Dk=Dv=64 J=4
        // that is S = 4: 128 blocks of 16 columns instead of 32 of 64; gated at
        // B=8 H=16 Dk=Dv=128 J=4, S = 8: 1024 blocks instead of 512.  The
        // backward's checkpoints store key index l * S + s at its own position,
        // so their layout does not depend on S.
        constexpr size_t kFill = GT ? 1024 : 256;
        constexpr int S2 = S / 2 >= 4 && DK / (S / 2) <= 16 ? S / 2 : S;
        constexpr int S4 = S2 / 2 >= 4 && DK / (S2 / 2) <= 16 ? S2 / 2 : S2;
        if (grid_blocks<DK, J, S, TP>(a) < kFill) {
            if (S4 != S2 && grid_blocks<DK, J, S2, TP>(a) < kFill)
                return launch_s<DK, J, S4, TP, GT, AX>(a, stream);
            if constexpr (S2 != S) return launch_s<DK, J, S2, TP, GT, AX>(a, stream);
        }
    }
    return launch_s<DK, J, S, TP, GT, AX>(a, stream);
}

template <int DK, int J>
hipError_t launch_dk_j(const LayerArgs &a, hipStream_t stream) {
    if (a.decay) {
        // The gated form stages a round's gates as [token][j][key index] in LDS:
        // J * Dk <= 1024 keeps that tile at 64 KiB.
        if constexpr (J * DK > kMaxGatedJDk) {
            return hipErrorInvalidValue;
        } else {
            return a.gk ? launch_dk_j_tp<DK, J, true, true>(a, stream)
                        : launch_dk_j_tp<DK, J, false, true>(a, stream);
        }
    }
    return a.gk ? launch_dk_j_tp<DK, J, true, false>(a, stream)
                : launch_dk_j_tp<DK, J, false, false>(a, stream);
}

template <int DK>
hipError_t launch_dk(const LayerArgs &a, hipStream_t stream) {
    switch (a.J) {
        case 1: return launch_dk_j<DK, 1>(a, stream);
        case 2: return launch_dk_j<DK, 2>(a, stream);
        case 3: return launch_dk_j<DK, 3>(a, stream);
        case 4: return launch_dk_j<DK, 4>(a, stream);
        case 8: return launch_dk_j<DK, 8>(a, stream);
        case 16: return launch_dk_j<DK, 16>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

template <int DK>
hipError_t launch_aux_dk(const LayerArgs &a, hipStream_t stream) {
    switch (a.J) {
        case 1: return launch_dk_j_tp<DK, 1, false, false, true>(a, stream);
        case 2: return launch_dk_j_tp<DK, 2, false, false, true>(a, stream);
        case 3: return launch_dk_j_tp<DK, 3, false, false, true>(a, stream);
        case 4: return launch_dk_j_tp<DK, 4, false, false, true>(a, stream);
        case 8: return launch_dk_j_tp<DK, 8, false, false, true>(a, stream);
        case 16: return launch_dk_j_tp<DK, 16, false, false, true>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

}  // namespace swila
