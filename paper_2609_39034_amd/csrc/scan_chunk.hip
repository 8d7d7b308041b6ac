// Exact chunked SwiLA scan on the matrix cores (bf16 inputs, fp32 state).
//
// Every update of eq. recurrence adds a multiple of k_t to w_{jd}, so inside a
// chunk of C tokens that starts from state W_n the state before token t is
//   w_{t-1,jd} = w_{n,jd} + sum_{s<t, s in chunk} c_{s,jd} k_s,   c = beta r delta.
// Hence, exactly (up to rounding order),
//   pred_{t,jd} = k_t . w_{n,jd} + sum_{s<t} (k_t . k_s) c_{s,jd}
//   w_{t,jd}.q_t = q_t . w_{n,jd} + sum_{s<=t} (q_t . k_s) c_{s,jd}     (eq. retrieval)
//   W_{n+1}     = W_n + sum_s c_s k_s^T.
// The Dk-long contractions become 16 x 16 matrix products per chunk
// (U = K W^T, Y = Q W^T, G = K K^T, A = Q K^T, W += C^T K, Y += tril(A) C);
// only the scalar recurrence of the coefficients c over the C = 16 tokens of a
// chunk stays sequential (a <= 15-term update and the E-step per token).
// This is the same algebra as the delta-rule chunk form the paper builds on
// (App. D.1), applied to the exact nonlinear recurrence, one chunk at a time.
//
// Precision.  q and k are bf16 and enter the matrix cores unrounded.  fp32
// operands (the state W, the coefficients C, the products A) are split into a
// bf16 high part and a bf16 residual, and the products that matter are summed
// (hi*hi + hi*lo [+ lo*hi]), leaving about 2^-16 relative error per product;
// accumulation is fp32.
//
// Work split.  One block owns one head (b, h) and a block of DB output dims d
// with all J components: N = J * DB <= 64 columns, column index
// col = j * DB + dl.  Wave w owns the 16-column tile w of the state W^T
// (Dk x 16 fp32, kept in the MFMA accumulator layout for the whole sequence).
// Per chunk:
//   A  (all waves) U and Y0 for the wave's tile; wave 0 also forms G and A.
//   B  (wave 0)    the 16-token recurrence; lanes of one d hold its J
//                  components and reduce over them with DPP.
//   C  (all waves) W += K^T C; Y += tril(A) C; stage pi^q * Y.
//   D  (all)       o = sum_j pi^q y; stage the next chunk's inputs, which were
//                  fetched from HBM into registers at the start of the chunk.
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kC = 16;  // tokens per chunk: one matrix-core tile

__device__ __forceinline__ floatx4 mfma32(bf16x8 a, bf16x8 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ floatx4 mfma16(short4v a, short4v b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ short bf16_bits(__bf16 x) { return __builtin_bit_cast(short, x); }

// x = hi + lo with hi = bf16(x) and lo = bf16(x - hi).
__device__ __forceinline__ void split(float x, __bf16 &hi, __bf16 &lo) {
    hi = (__bf16)x;
    lo = (__bf16)(x - (float)hi);
}

template <int DK, int J, int DB>
struct Cfg {
    static constexpr int N = J * DB;               // columns of one block
    static constexpr int NW = N / 16;              // waves, one column tile each
    static constexpr int NT = NW * 64;             // threads
    static constexpr int JP = J == 3 ? 4 : J;      // lanes per output dim in phase B
    static constexpr int IT = DK / 16;             // 16-row tiles of W^T
    static constexpr int KP = DK + 4;              // padded K/Q row (bf16)
    static constexpr int TP = kC + 4;              // padded K^T row (bf16)
    static constexpr int NP = N + 4;               // padded fp32 column row
    static constexpr int KQ_PIECES = kC * DK / 8;  // 16-byte pieces of one K (or Q) chunk
    static constexpr int KQ_PER = (KQ_PIECES + NT - 1) / NT;
    static constexpr int PAIRS = kC * DB;          // (token, output dim) pairs per chunk
    static constexpr int PAIR_PER = (PAIRS + NT - 1) / NT;
    static_assert(N % 16 == 0 && N <= 64, "column block");
    static_assert(DB * JP <= 64, "phase B runs in one wave");
};

template <int DK, int J, int DB>
struct Smem {
    using C = Cfg<DK, J, DB>;
    uint16_t k[kC][C::KP];
    uint16_t q[kC][C::KP];
    uint16_t kt[DK][C::TP];
    float g[kC][kC + 4];      // K K^T
    float a[kC][kC + 4];      // Q K^T
    float c[kC][C::NP];       // coefficients beta r delta
    float py[kC][C::NP];      // phase A->B: predictions U; phase C->D: pi^q * y
    float beta[kC][C::NP];
    float lk[kC][C::NP];      // key-prior logit * log2(e)
    float pq[kC][C::NP];      // query prior
    float v[kC][DB + 4];
};

// Next chunk's inputs as raw bf16 bits, held in registers between the HBM
// fetch (start of a chunk) and the LDS store (end of it).  Every load is
// unconditional with an in-range address (tokens past T re-read the last
// token and are zeroed when staged), so nothing consumes a loaded register
// before the store and the loads stay in flight across the chunk.
template <int DK, int J, int DB>
struct Prefetch {
    using C = Cfg<DK, J, DB>;
    uint4 k[C::KQ_PER], q[C::KQ_PER];
    uint32_t v[C::PAIR_PER], lb[C::PAIR_PER][J], lk[C::PAIR_PER][J], lq[C::PAIR_PER][J];
};

template <int DK, int J, int DB>
__device__ __forceinline__ void fetch(const LayerArgs &a, int b, int h, int d0, int t0, int tid,
                                      Prefetch<DK, J, DB> &pf) {
    using C = Cfg<DK, J, DB>;
    const int T = a.T, H = a.H, Dv = a.Dv;
    const uint16_t *kp = static_cast<const uint16_t *>(a.k);
    const uint16_t *qp = static_cast<const uint16_t *>(a.q);
#pragma unroll
    for (int m = 0; m < C::KQ_PER; ++m) {
        int g = tid + m * C::NT;
        g = g < C::KQ_PIECES ? g : 0;
        const int t = min(t0 + g / (DK / 8), T - 1), i = (g % (DK / 8)) * 8;
        const size_t off = ((size_t)(b * T + t) * H + h) * DK + i;
        pf.k[m] = *reinterpret_cast<const uint4 *>(kp + off);
        pf.q[m] = *reinterpret_cast<const uint4 *>(qp + off);
    }
    const uint16_t *vp = static_cast<const uint16_t *>(a.v);
    const uint16_t *lbp = static_cast<const uint16_t *>(a.lb);
    const uint16_t *lkp = static_cast<const uint16_t *>(a.lk);
    const uint16_t *lqp = static_cast<const uint16_t *>(a.lq);
#pragma unroll
    for (int m = 0; m < C::PAIR_PER; ++m) {
        int g = tid + m * C::NT;
        g = g < C::PAIRS ? g : 0;
        const int t = min(t0 + g / DB, T - 1), dl = g % DB;
        const size_t row = (size_t)(b * T + t) * H + h;
        pf.v[m] = vp[row * Dv + d0 + dl];
        const size_t base = row * J * Dv + d0 + dl;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            pf.lb[m][j] = lbp[base + (size_t)j * Dv];
            pf.lk[m][j] = lkp[base + (size_t)j * Dv];
            pf.lq[m][j] = lqp[base + (size_t)j * Dv];
        }
    }
}

// Store the fetched chunk starting at token t0 into LDS: K and Q as bf16 (and
// K transposed), and per (token, column) beta = sigmoid, lk * log2(e) and
// pi^q = softmax over j.  Tokens at or past T become zeros (K = Q = 0,
// beta = 0), which leaves the state unchanged.
template <int DK, int J, int DB>
__device__ __forceinline__ void stage(const Prefetch<DK, J, DB> &pf, int t0, int T, int tid,
                                      Smem<DK, J, DB> &sm) {
    using C = Cfg<DK, J, DB>;
#pragma unroll
    for (int m = 0; m < C::KQ_PER; ++m) {
        const int g = tid + m * C::NT;
        if (g < C::KQ_PIECES) {
            const int t = g / (DK / 8), i = (g % (DK / 8)) * 8;
            const bool ok = t0 + t < T;
            const uint4 kk = ok ? pf.k[m] : make_uint4(0, 0, 0, 0);
            const uint4 qq = ok ? pf.q[m] : make_uint4(0, 0, 0, 0);
            *reinterpret_cast<uint2 *>(&sm.k[t][i]) = make_uint2(kk.x, kk.y);
            *reinterpret_cast<uint2 *>(&sm.k[t][i + 4]) = make_uint2(kk.z, kk.w);
            *reinterpret_cast<uint2 *>(&sm.q[t][i]) = make_uint2(qq.x, qq.y);
            *reinterpret_cast<uint2 *>(&sm.q[t][i + 4]) = make_uint2(qq.z, qq.w);
            const uint32_t w[4] = {kk.x, kk.y, kk.z, kk.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sm.kt[i + 2 * e][t] = (uint16_t)(w[e] & 0xffffu);
                sm.kt[i + 2 * e + 1][t] = (uint16_t)(w[e] >> 16);
            }
        }
    }
#pragma unroll
    for (int m = 0; m < C::PAIR_PER; ++m) {
        const int g = tid + m * C::NT;
        if (g < C::PAIRS) {
            const int t = g / DB, dl = g % DB;
            const bool ok = t0 + t < T;
            sm.v[t][dl] = ok ? bf16_bits_to_f32(pf.v[m]) : 0.f;
            float lq[J];
            float mq = -INFINITY;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                lq[j] = bf16_bits_to_f32(pf.lq[m][j]);
                mq = fmaxf(mq, lq[j]);
            }
            float z = 0.f;
#pragma unroll
            for (int j = 0; j < J; ++j) {
                lq[j] = exp_fast(lq[j] - mq);
                z += lq[j];
            }
            const float iz = rcp_fast(z);
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const float beta = rcp_fast(1.0f + exp_fast(-bf16_bits_to_f32(pf.lb[m][j])));
                sm.beta[t][j * DB + dl] = ok ? beta : 0.f;
                sm.lk[t][j * DB + dl] = bf16_bits_to_f32(pf.lk[m][j]) * kLog2e;
                sm.pq[t][j * DB + dl] = lq[j] * iz;
            }
        }
    }
}

template <int DK, int J, int DB>
__global__ __launch_bounds__(256) void scan_chunk_kernel(LayerArgs a) {
    using C = Cfg<DK, J, DB>;
    constexpr int IT = C::IT, N = C::N, JP = C::JP;
    __shared__ Smem<DK, J, DB> sm;

    const int tid = threadIdx.x;
    const int w = tid / 64, lane = tid % 64;
    const int tl = lane % 16, lg = lane / 16;
    const int d0 = blockIdx.x * DB;
    const int h = blockIdx.y, b = blockIdx.z;
    const int H = a.H, T = a.T, Dv = a.Dv;

    // W^T tile of this wave: rows i = 16 it + 4 lg + r, column col = 16 w + tl
    const int col = 16 * w + tl;
    const int jc = col / DB, dc = d0 + col % DB;
    const size_t sbase = (((size_t)b * H + h) * J + jc) * DK * Dv + dc;
    floatx4 W[IT];
#pragma unroll
    for (int it = 0; it < IT; ++it) W[it] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (a.state_in) {
#pragma unroll
        for (int it = 0; it < IT; ++it)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                W[it][r] = a.state_in[sbase + (size_t)(16 * it + 4 * lg + r) * Dv];
    }

    // phase B identity: lanes of one output dim are adjacent
    const int bdl = (tid / JP) % DB, bj = tid % JP;
    const bool bact = tid < DB * JP && bj < J;
    const int bcol = bact ? bj * DB + bdl : 0;

    Prefetch<DK, J, DB> pf;
    fetch<DK, J, DB>(a, b, h, d0, 0, tid, pf);
    stage<DK, J, DB>(pf, 0, T, tid, sm);
    __syncthreads();

    for (int t0 = 0; t0 < T; t0 += kC) {
        if (t0 + kC < T) fetch<DK, J, DB>(a, b, h, d0, t0 + kC, tid, pf);

        // ---- A: U = K W^T, Y = Q W^T for this wave's tile; wave 0: G, A
        floatx4 U = {0.f, 0.f, 0.f, 0.f}, Y = U, G = U, AQ = U;
        if constexpr (DK == 16) {
            short4v ak, aq, whi, wlo;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                ak[m] = (short)sm.k[tl][4 * lg + m];
                aq[m] = (short)sm.q[tl][4 * lg + m];
                __bf16 hi, lo;
                split(W[0][m], hi, lo);
                whi[m] = bf16_bits(hi);
                wlo[m] = bf16_bits(lo);
            }
            U = mfma16(ak, whi, U);
            U = mfma16(ak, wlo, U);
            Y = mfma16(aq, whi, Y);
            Y = mfma16(aq, wlo, Y);
            if (w == 0) {
                G = mfma16(ak, ak, G);
                AQ = mfma16(aq, ak, AQ);
            }
        } else {
#pragma unroll
            for (int s = 0; s < DK / 32; ++s) {
                // slot 8 lg + m <-> key index 32 s + 4 lg + m (m < 4), 32 s + 16 + 4 lg + m - 4
                const uint2 k0 = *reinterpret_cast<const uint2 *>(&sm.k[tl][32 * s + 4 * lg]);
                const uint2 k1 = *reinterpret_cast<const uint2 *>(&sm.k[tl][32 * s + 16 + 4 * lg]);
                const uint2 q0 = *reinterpret_cast<const uint2 *>(&sm.q[tl][32 * s + 4 * lg]);
                const uint2 q1 = *reinterpret_cast<const uint2 *>(&sm.q[tl][32 * s + 16 + 4 * lg]);
                const uint4 ku = make_uint4(k0.x, k0.y, k1.x, k1.y);
                const uint4 qu = make_uint4(q0.x, q0.y, q1.x, q1.y);
                const bf16x8 ak = __builtin_bit_cast(bf16x8, ku);
                const bf16x8 aq = __builtin_bit_cast(bf16x8, qu);
                bf16x8 whi, wlo;
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    __bf16 hi, lo;
                    split(W[2 * s][m], hi, lo);
                    whi[m] = hi;
                    wlo[m] = lo;
                    split(W[2 * s + 1][m], hi, lo);
                    whi[4 + m] = hi;
                    wlo[4 + m] = lo;
                }
                U = mfma32(ak, whi, U);
                U = mfma32(ak, wlo, U);
                Y = mfma32(aq, whi, Y);
                Y = mfma32(aq, wlo, Y);
                if (w == 0) {
                    G = mfma32(ak, ak, G);
                    AQ = mfma32(aq, ak, AQ);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) sm.py[4 * lg + r][col] = U[r];
        if (w == 0) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sm.g[4 * lg + r][tl] = G[r];
                sm.a[4 * lg + r][tl] = AQ[r];
            }
        }
        block_sync_lds();

        // ---- B: the sequential recurrence of the coefficients over the chunk
        if (w == 0) {
            float P[kC], vv[kC], lkv[kC], bev[kC];
#pragma unroll
            for (int t = 0; t < kC; ++t) {
                P[t] = sm.py[t][bcol];
                vv[t] = sm.v[t][bdl];
                lkv[t] = bact ? sm.lk[t][bcol] : -INFINITY;
                bev[t] = bact ? sm.beta[t][bcol] : 0.f;
            }
            float grow[kC];  // row t of G, fetched one token ahead
#pragma unroll
            for (int u = 1; u < kC; ++u) grow[u] = sm.g[0][u];
#pragma unroll
            for (int t = 0; t < kC; ++t) {
                float gnext[kC];
#pragma unroll
                for (int u = t + 2; u < kC; ++u) gnext[u] = sm.g[t + 1][u];
                const float delta = vv[t] - P[t];
                const float bd = bev[t] * delta;
                const float e = fmaf(-0.5f * kLog2e * delta, delta, lkv[t]);
                const float mx = group_max<JP>(e);
                const float ex = __builtin_amdgcn_exp2f(e - mx);
                const float z = group_sum<JP>(ex);
                const float r = ex * rcp_fast(z);
                const float c = bd * r;
#pragma unroll
                for (int u = t + 1; u < kC; ++u) P[u] = fmaf(grow[u], c, P[u]);
                if (bact) {
                    sm.c[t][bcol] = c;
                    if (a.resp && t0 + t < T)
                        a.resp[(((size_t)(b * T + t0 + t) * H + h) * J + bj) * Dv + d0 + bdl] = r;
                }
#pragma unroll
                for (int u = t + 2; u < kC; ++u) grow[u] = gnext[u];
            }
        }
        block_sync_lds();

        // ---- C: W += K^T C;  Y += tril(A) C;  stage pi^q * y
        {
            short4v chi, clo;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                __bf16 hi, lo;
                split(sm.c[4 * lg + m][col], hi, lo);
                chi[m] = bf16_bits(hi);
                clo[m] = bf16_bits(lo);
            }
#pragma unroll
            for (int it = 0; it < IT; ++it) {
                const uint2 kt = *reinterpret_cast<const uint2 *>(&sm.kt[16 * it + tl][4 * lg]);
                const short4v ak = __builtin_bit_cast(short4v, kt);
                W[it] = mfma16(ak, chi, W[it]);
                W[it] = mfma16(ak, clo, W[it]);
            }
            short4v ahi, alo;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int s = 4 * lg + m;
                __bf16 hi, lo;
                split(s <= tl ? sm.a[tl][s] : 0.f, hi, lo);
                ahi[m] = bf16_bits(hi);
                alo[m] = bf16_bits(lo);
            }
            Y = mfma16(ahi, chi, Y);
            Y = mfma16(ahi, clo, Y);
            Y = mfma16(alo, chi, Y);
#pragma unroll
            for (int r = 0; r < 4; ++r) sm.py[4 * lg + r][col] = Y[r] * sm.pq[4 * lg + r][col];
        }
        block_sync_lds();

        // ---- D: outputs of this chunk; inputs of the next one into LDS
        for (int g = tid; g < kC * DB; g += C::NT) {
            const int t = g / DB, dl = g % DB;
            if (t0 + t < T) {
                float o = 0.f;
#pragma unroll
                for (int j = 0; j < J; ++j) o += sm.py[t][j * DB + dl];
                store1(a.o, ((size_t)(b * T + t0 + t) * H + h) * Dv + d0 + dl, o, a.out_bf16);
            }
        }
        if (t0 + kC < T) stage<DK, J, DB>(pf, t0 + kC, T, tid, sm);
        block_sync_lds();
    }

    if (a.state_out) {
#pragma unroll
        for (int it = 0; it < IT; ++it)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                a.state_out[sbase + (size_t)(16 * it + 4 * lg + r) * Dv] = W[it][r];
    }
}

template <int DK, int J, int DB>
hipError_t launch_cfg(const LayerArgs &a, hipStream_t stream) {
    using C = Cfg<DK, J, DB>;
    dim3 grid(a.Dv / DB, a.H, a.B);
    hipLaunchKernelGGL((scan_chunk_kernel<DK, J, DB>), grid, dim3(C::NT), 0, stream, a);
    return hipGetLastError();
}

template <int DK>
hipError_t launch_dk(const LayerArgs &a, hipStream_t stream) {
    // DB = min(Dv, 64 / JP): at most 64 columns and one wave of phase-B lanes.
    switch (a.J) {
        case 1:
            if (a.Dv >= 64) return launch_cfg<DK, 1, 64>(a, stream);
            if (a.Dv == 32) return launch_cfg<DK, 1, 32>(a, stream);
            return launch_cfg<DK, 1, 16>(a, stream);
        case 2:
            if (a.Dv >= 32) return launch_cfg<DK, 2, 32>(a, stream);
            return launch_cfg<DK, 2, 16>(a, stream);
        case 3: return launch_cfg<DK, 3, 16>(a, stream);
        case 4: return launch_cfg<DK, 4, 16>(a, stream);
        case 8: return launch_cfg<DK, 8, 8>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_scan_chunk(const LayerArgs &a, hipStream_t stream) {
    if (!a.in_bf16) return hipErrorInvalidValue;
    switch (a.Dk) {
        case 16: return launch_dk<16>(a, stream);
        case 32: return launch_dk<32>(a, stream);
        case 64: return launch_dk<64>(a, stream);
        case 128: return launch_dk<128>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace swila
