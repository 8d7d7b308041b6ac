// One-token SwiLA decode step (Sec. 3.2 with T = 1): the state is read once
// from HBM, updated in registers and written once, so the step is bound by HBM
// bandwidth (state bytes dominate: 2 x J x Dk x Dv x 4 per head and token).
//
// Work split.  A block owns one head's block of DB = min(32, Dv) output
// columns for every component j and key index i: a J x Dk x DB fp32 tile.
// CL = DB / 4 lanes cover one 128-byte row segment (float4 per lane), so
// consecutive lanes read consecutive addresses.  Each thread holds 16 rows
// (i = ig + IG * m, m < 16) of one component j: IG = Dk / 16 row groups per
// component, J * IG * CL threads per block (at least DB; any extra threads
// hold no rows and only serve the per-column step).  Per token:
//   1. every thread forms partial k- and q-dots of its 16 rows for 4 columns;
//      lanes of the same component and column reduce over row groups;
//   2. DB threads (one per column) run the E-step over j and the retrieval;
//   3. every thread applies w += c k to its rows and stores them.
// state_out may alias state_in: each block reads its whole tile before any
// write, and tiles of different blocks are disjoint.
//
// Temporal SwiLA (TP; App. B.3): the column threads also read the prior state
// (r_{t-1}, rhobar_{t-1}) of their column, use rbar = (1 - g^k) r_{t-1} +
// g^k pi^k as the key prior and rhobar = (1 - g^q) rhobar_{t-1} + g^q pi^q as
// the query prior, and write the new pair (r, rhobar); prior_out may alias
// prior_in for the same reason as the state.
//
// Gated SwiLA (GT; App. B.4, eq. pre-decay): every thread scales its rows by
// the decay of its component and key index, a = sigmoid(decay logit), before
// the dots, so the E-step, update and retrieval all see the decayed state.
#include "device_common.hpp"
#include "launch.hpp"

namespace swila {
namespace {

constexpr int kRows = 16;  // state rows per thread

// The state streams through once per step: non-temporal loads and stores keep it
// from displacing lines that are reused (the token's inputs).
typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 stream_load(const float *p) {
    const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stream_store(float *p, float4 x) {
    f32x4 v = {x.x, x.y, x.z, x.w};
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4 *>(p));
}

template <int DK, int J, bool TP, bool GT>
__global__ __launch_bounds__(512) void decode_kernel(LayerArgs a, int DB) {
    constexpr int IG = DK / kRows;
    const int CL = DB / 4;
    const int tid = threadIdx.x;
    const int cl = tid % CL;
    const int ig = (tid / CL) % IG;
    const bool has_rows = tid < J * IG * CL;
    const int j = has_rows ? tid / (CL * IG) : 0;
    // Workgroups go to the eight XCDs round-robin by linear index.  The column
    // blocks of a head read interleaved pieces of the same state rows (and the
    // same k, q and decay row); they are all placed on one XCD.
    const int NDB = gridDim.x, NH = gridDim.y * gridDim.z;
    const int lin = blockIdx.x + NDB * (blockIdx.y + gridDim.y * blockIdx.z);
    int hh = blockIdx.y + gridDim.y * blockIdx.z, db = blockIdx.x;
    if (NDB > 1 && NH % 8 == 0) {
        const int xs = lin / 8;
        hh = 8 * (xs / NDB) + lin % 8;
        db = xs % NDB;
    }
    const int d0 = db * DB;
    const int h = hh % gridDim.y, b = hh / gridDim.y;
    const int H = a.H, Dv = a.Dv;
    const bool ibf = a.in_bf16;

    __shared__ float sk[DK], sq[DK];
    __shared__ float sP[J][32], sY[J][32], sC[J][32];
    __shared__ float sKQ;

    // state tile rows of this thread
    const size_t sbase = ((size_t)b * H + h) * J * DK * Dv + (size_t)j * DK * Dv + d0 + cl * 4;
    float4 st[kRows];
    if (a.state_in && has_rows) {
#pragma unroll
        for (int m = 0; m < kRows; ++m)
            st[m] = stream_load(a.state_in + sbase + (size_t)(ig + IG * m) * Dv);
    } else {
#pragma unroll
        for (int m = 0; m < kRows; ++m) st[m] = make_float4(0.f, 0.f, 0.f, 0.f);
    }

    // per-column inputs, fetched early by the column threads
    const size_t row = (size_t)b * H + h;
    float vd = 0.f, lb[J], lk[J], lq[J];
    float gk = 0.f, gq = 0.f, rprev[J], rho[J];   // temporal
    const size_t pbase = row * 2 * J * Dv + d0 + tid;
    if (tid < DB) {
        vd = load1(a.v, row * Dv + d0 + tid, ibf);
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            const size_t idx = (row * J + jj) * Dv + d0 + tid;
            lb[jj] = load1(a.lb, idx, ibf);
            lk[jj] = load1(a.lk, idx, ibf);
            lq[jj] = load1(a.lq, idx, ibf);
        }
        if constexpr (TP) {
            gk = 1.0f / (1.0f + exp_fast(-load1(a.gk, row * Dv + d0 + tid, ibf)));
            gq = 1.0f / (1.0f + exp_fast(-load1(a.gq, row * Dv + d0 + tid, ibf)));
#pragma unroll
            for (int jj = 0; jj < J; ++jj) {
                rprev[jj] = a.prior_in ? a.prior_in[pbase + (size_t)jj * Dv] : 1.0f / J;
                rho[jj] = a.prior_in ? a.prior_in[pbase + (size_t)(J + jj) * Dv] : 1.0f / J;
            }
        }
    }
    for (int i = tid; i < DK; i += blockDim.x) {
        sk[i] = load1(a.k, row * DK + i, ibf);
        sq[i] = load1(a.q, row * DK + i, ibf);
    }
    if constexpr (GT) {
        // eq. pre-decay: w_j (.)= a_j, one gate per key index
        if (has_rows) {
#pragma unroll
            for (int m = 0; m < kRows; ++m) {
                const float g = sigmoid(load1(a.decay, (row * J + j) * DK + ig + IG * m, ibf));
                st[m].x *= g, st[m].y *= g, st[m].z *= g, st[m].w *= g;
            }
        }
    }
    __syncthreads();

    // 1. partial dots over this thread's rows
    float p[4] = {0.f, 0.f, 0.f, 0.f}, y[4] = {0.f, 0.f, 0.f, 0.f}, kq = 0.f;
#pragma unroll
    for (int m = 0; m < kRows; ++m) {
        const float ki = sk[ig + IG * m], qi = sq[ig + IG * m];
        p[0] = fmaf(st[m].x, ki, p[0]); y[0] = fmaf(st[m].x, qi, y[0]);
        p[1] = fmaf(st[m].y, ki, p[1]); y[1] = fmaf(st[m].y, qi, y[1]);
        p[2] = fmaf(st[m].z, ki, p[2]); y[2] = fmaf(st[m].z, qi, y[2]);
        p[3] = fmaf(st[m].w, ki, p[3]); y[3] = fmaf(st[m].w, qi, y[3]);
        kq = fmaf(ki, qi, kq);
    }
    for (int off = CL; off < CL * IG; off *= 2) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            p[c] += __shfl_xor(p[c], off);
            y[c] += __shfl_xor(y[c], off);
        }
        kq += __shfl_xor(kq, off);
    }
    if (ig == 0 && has_rows) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            sP[j][cl * 4 + c] = p[c];
            sY[j][cl * 4 + c] = y[c];
        }
        if (j == 0 && cl == 0) sKQ = kq;
    }
    __syncthreads();

    // 2. E-step and retrieval, one thread per column
    if (tid < DB) {
        float delta[J], e[J];
        float m = -INFINITY, mq = -INFINITY, mk = -INFINITY;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            delta[jj] = vd - sP[jj][tid];
            e[jj] = (TP ? 0.0f : lk[jj]) - 0.5f * delta[jj] * delta[jj];
            m = fmaxf(m, e[jj]);
            mq = fmaxf(mq, lq[jj]);
            mk = fmaxf(mk, lk[jj]);
        }
        float z = 0.f, zq = 0.f, zk = 0.f;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            e[jj] = exp_fast(e[jj] - m);
            lq[jj] = exp_fast(lq[jj] - mq);
            zq += lq[jj];
            if constexpr (TP) {
                lk[jj] = exp_fast(lk[jj] - mk);
                zk += lk[jj];
            }
        }
        const float izk = TP ? 1.0f / zk : 1.0f;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            // temporal key prior: (1 - g^k) r_{t-1} + g^k pi^k
            if constexpr (TP) e[jj] *= fmaf(gk, lk[jj] * izk - rprev[jj], rprev[jj]);
            z += e[jj];
        }
        const float iz = rcp_fast(z), izq = 1.0f / zq, kqv = sKQ;
        float o = 0.f;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            const float beta = 1.0f / (1.0f + exp_fast(-lb[jj]));
            const float r = e[jj] * iz;
            const float c = beta * r * delta[jj];
            sC[jj][tid] = c;
            float pq = lq[jj] * izq;
            if constexpr (TP) {
                rprev[jj] = r;
                rho[jj] = fmaf(gq, pq - rho[jj], rho[jj]);   // (1 - g^q) rhobar + g^q pi^q
                pq = rho[jj];
            }
            o = fmaf(pq, fmaf(c, kqv, sY[jj][tid]), o);
        }
        store1(a.o, row * Dv + d0 + tid, o, a.out_bf16);
        if constexpr (TP) {
            if (a.prior_out) {
#pragma unroll
                for (int jj = 0; jj < J; ++jj) {
                    a.prior_out[pbase + (size_t)jj * Dv] = rprev[jj];
                    a.prior_out[pbase + (size_t)(J + jj) * Dv] = rho[jj];
                }
            }
        }
    }
    __syncthreads();

    // 3. rank-one update of this thread's rows
    if (a.state_out && has_rows) {
        const float4 c4 = make_float4(sC[j][cl * 4], sC[j][cl * 4 + 1], sC[j][cl * 4 + 2],
                                      sC[j][cl * 4 + 3]);
        float *dst = a.state_out + sbase;
#pragma unroll
        for (int m = 0; m < kRows; ++m) {
            const float ki = sk[ig + IG * m];
            float4 s = st[m];
            s.x = fmaf(c4.x, ki, s.x);
            s.y = fmaf(c4.y, ki, s.y);
            s.z = fmaf(c4.z, ki, s.z);
            s.w = fmaf(c4.w, ki, s.w);
            stream_store(dst + (size_t)(ig + IG * m) * Dv, s);
        }
    }
}

template <int DK, int J>
hipError_t launch_dk_j(const LayerArgs &a, hipStream_t stream) {
    // DB columns per block: 32, or fewer where J * (Dk / 16) * (DB / 4) row
    // threads would exceed the 512-thread block (J = 16, Dk = 128: 16 columns)
    constexpr int kMaxDB = 4 * 512 / (J * (DK / kRows)) < 32 ? 4 * 512 / (J * (DK / kRows)) : 32;
    static_assert(kMaxDB >= 4, "block of at least one float4 column group");
    const int DB = a.Dv < kMaxDB ? a.Dv : kMaxDB;
    int threads = J * (DK / kRows) * (DB / 4);
    if (threads < DB) threads = DB;
    dim3 grid(a.Dv / DB, a.H, a.B);
    if (a.decay && a.gk)
        hipLaunchKernelGGL((decode_kernel<DK, J, true, true>), grid, dim3(threads), 0, stream, a, DB);
    else if (a.decay)
        hipLaunchKernelGGL((decode_kernel<DK, J, false, true>), grid, dim3(threads), 0, stream, a, DB);
    else if (a.gk)
        hipLaunchKernelGGL((decode_kernel<DK, J, true, false>), grid, dim3(threads), 0, stream, a, DB);
    else
        hipLaunchKernelGGL((decode_kernel<DK, J, false, false>), grid, dim3(threads), 0, stream, a, DB);
    return hipGetLastError();
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

__global__ void fill_kernel(float *dst, const float *src, size_t n, float value) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        dst[i] = src ? src[i] : value;
}

}  // namespace

hipError_t launch_decode(const LayerArgs &a, hipStream_t stream) {
    switch (a.Dk) {
        case 16: return launch_dk<16>(a, stream);
        case 32: return launch_dk<32>(a, stream);
        case 64: return launch_dk<64>(a, stream);
        case 128: return launch_dk<128>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_fill(float *dst, const float *src, size_t n, float value, hipStream_t stream) {
    if (n == 0 || dst == src) return hipSuccess;
    size_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    hipLaunchKernelGGL(fill_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, dst, src, n,
                       value);
    return hipGetLastError();
}

hipError_t launch_state_fill(float *state, const float *src, size_t n, hipStream_t stream) {
    return launch_fill(state, src, n, 0.0f, stream);
}

}  // namespace swila
